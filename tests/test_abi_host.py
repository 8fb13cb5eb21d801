"""The C ABI without a GPU: the library loads, exports every declared entry
point, and its host-only planning matches the oracle's layout (CPU only)."""
import os
import re

import numpy as np
import pytest

import oracle as O

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "ckpt.h")


def declared_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(ckpt_[a-z_]+)\s*\(", src)))


@pytest.fixture(scope="module")
def P():
    import paper_2607_01646_amd as P

    P.lib()
    return P


def test_header_declares_the_boundary():
    names = declared_functions()
    for f in ["ckpt_register_tensors", "ckpt_snapshot_async", "ckpt_wait", "ckpt_restore", "ckpt_verify"]:
        assert f in names


def test_library_exports_every_declared_symbol(P):
    L = P.lib()
    missing = [f for f in declared_functions() if not hasattr(L, f)]
    assert not missing, missing


def test_no_cpu_fallback_in_binding():
    """The binding never reaches for the oracle or a host implementation."""
    pkg = os.path.join(ROOT, "paper_2607_01646_amd")
    for name in os.listdir(pkg):
        if name.endswith(".py"):
            text = open(os.path.join(pkg, name)).read()
            assert "oracle" not in text.replace("no fallback", ""), name


def test_plan_matches_oracle_layout(P):
    rng = np.random.default_rng(3)
    for A, C in [(256, 4 << 20), (256, 768), (16, 64), (4096, 8192), (64, 1 << 16)]:
        for _ in range(20):
            n = int(rng.integers(1, 300))
            sizes = [int(s) for s in rng.integers(0, 5000, n)]
            sizes[-1] = max(sizes[-1], 1)
            want = O.layout(sizes, A, C)
            got = P.ckpt_plan(sizes, C, A)
            assert [int(x) for x in got[0]] == [int(x) for x in want[0]]
            assert got[1:] == want[1:]


def test_plan_workload_sizes(P):
    import workloads as W

    for wid in [1, 2, 3, 5, 6]:
        plan = W.fragment_plan(wid)
        sizes = [p[1] for p in plan]
        C = W.WORKLOADS[wid]["chunk"]
        got = P.ckpt_plan(sizes, C, 256)
        want = O.layout(sizes, 256, C)
        assert np.array_equal(got[0], want[0]) and got[1:] == want[1:]


def test_tile_plan_brute_force(P):
    """Each tile's first/last fragment really holds the tile's first/last byte
    (checked by brute force over the oracle's layout)."""
    rng = np.random.default_rng(4)
    for C in [256, 768, 4096, 1 << 17]:
        sizes = [int(s) for s in rng.integers(0, 3000, 200)]
        sizes[10:14] = [0, 0, 0, 0]
        sizes[0] = 0
        sizes[-1] = 0
        tb, tf, tl = P.ckpt_debug_tile_plan(sizes, C, 256)
        assert C % tb == 0 and tb & (tb - 1) == 0 and tb <= 8192
        off, I, nc = O.layout(sizes, 256, C)
        nonempty = [i for i, s in enumerate(sizes) if s]

        def holder(x):  # last non-empty fragment starting at or before x
            return max(i for i in nonempty if int(off[i]) <= x)

        assert len(tf) == -(-I // tb)
        for t in range(len(tf)):
            x0, x1 = t * tb, min((t + 1) * tb, I) - 1
            assert sizes[tf[t]] > 0 and sizes[tl[t]] > 0
            assert tf[t] == holder(x0), (t, tf[t], holder(x0))
            assert tl[t] == holder(x1)


def test_plan_rejects_bad_geometry(P):
    with pytest.raises(P.CkptError):
        P.ckpt_plan([10, 20], 1000, 256)  # chunk not a multiple of the alignment
    with pytest.raises(P.CkptError):
        P.ckpt_plan([10, 20], 4096, 8)  # alignment below 16
    with pytest.raises(P.CkptError):
        P.ckpt_plan([0, 0], 4096, 256)  # nothing to pack


def test_create_without_gpu_fails_cleanly(P):
    import torch

    if torch.cuda.is_available():
        pytest.skip("a GPU is present")
    with pytest.raises(P.CkptError):
        P.ckpt_create(device=0)
