"""The C ABI without a GPU: the library loads, exports every declared entry
point, and its host-only planning matches the oracle's layout (CPU only)."""
import os
import re

import numpy as np
import pytest
from hypothesis import HealthCheck, given, settings
from hypothesis import strategies as st

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


def check_direct_plan(P, sizes, C, A, G):
    """The copy plan of direct D2H for one layout, byte by byte (see
    test_direct_plan_brute_force)."""
    pieces, gaps, pf, gf = P.ckpt_debug_direct_plan(sizes, C, A, G)
    off, I, nc = O.layout(sizes, A, C)
    unit = max(1, (G or (1 << 30)) // C) * C
    n_groups = -(-I // unit)
    assert len(pf) == len(gf) == n_groups + 1
    owner = np.full(I, -1, dtype=np.int64)  # fragment holding each image byte, -1 = padding
    pos = np.zeros(I, dtype=np.int64)       # its offset inside that fragment
    for i, (o, s) in enumerate(zip(off, sizes)):
        owner[int(o):int(o) + s] = i
        pos[int(o):int(o) + s] = np.arange(s)
    for g in range(n_groups):
        lo, hi = g * unit, min((g + 1) * unit, I)
        ps = pieces[int(pf[g]):int(pf[g + 1])]
        gs = gaps[int(gf[g]):int(gf[g + 1])]
        assert len(ps) >= 1
        spans = sorted([(int(p[2]), int(p[3]), int(p[0]), int(p[1])) for p in ps] +
                       [(int(r[0]), int(r[1]), -1, 0) for r in gs])
        x = lo
        for a, n, frag, src in spans:
            assert a == x and n > 0, (g, a, x, n)
            if frag >= 0:
                assert np.all(owner[a:a + n] == frag) and np.array_equal(pos[a:a + n], np.arange(src, src + n))
            else:
                assert np.all(owner[a:a + n] == -1)
            x = a + n
        assert x == hi
        assert np.all(np.diff(ps[:, 2].astype(np.int64)) > 0)  # pieces in image order
    for i, s in enumerate(sizes):  # every fragment byte in exactly one piece
        assert int(pieces[pieces[:, 0] == i][:, 3].sum()) == s


def test_direct_plan_brute_force(P):
    """The copy plan of direct D2H, checked byte by byte over the oracle's
    layout: in every chunk group the fragment pieces and the padding runs tile
    the group exactly, in image order; each piece is the fragment's own bytes
    at the fragment's own offset (so the engines copy every fragment byte once,
    to its place); each run is padding, which no fragment byte lies in."""
    rng = np.random.default_rng(6)
    geometries = [(256, 256, 0), (4096, 256, 4096), (4096, 16, 3 * 4096), (768, 256, 2 * 768), (1 << 17, 256, 0)]
    for (C, A, G), tail in [(g, t) for g in geometries for t in ([1], [0, 0], [5 * 4096, 0])]:
        sizes = [int(s) for s in rng.integers(0, 9000, 150)]
        sizes[7:11] = [0, 0, 0, 0]
        sizes[0] = 0
        sizes[-len(tail):] = tail  # the image ends on a byte, on empty fragments, or on a long one
        sizes[20] = 5 * C + 3  # spans several groups
        check_direct_plan(P, sizes, C, A, G)


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


def test_noalloc_pack_sizes_its_image_like_the_oracle(P):
    """ckpt_pack_noalloc computes its layout in two passes without any table;
    with capacities of zero it stops before touching a device and reports
    the image size and chunk count, which must be the oracle's."""
    import ctypes as C

    rng = np.random.default_rng(11)
    fake = 0x10000  # never dereferenced: the call returns before any device work
    for A, Cb in [(256, 4 << 20), (256, 768), (16, 64), (4096, 8192)]:
        for _ in range(10):
            n = int(rng.integers(1, 200))
            sizes = [int(s) for s in rng.integers(0, 9000, n)]
            sizes[0] = max(sizes[0], 1)
            arr = (P.ckpt_tensor * n)()
            for i, s in enumerate(sizes):
                arr[i].dev_ptr = fake if s else None
                arr[i].nbytes = s
            ib, nc = C.c_uint64(), C.c_uint64()
            rc = P.lib().ckpt_pack_noalloc(arr, n, Cb, A, 0, C.c_void_p(fake), 0, C.c_void_p(fake), 0, None,
                                           C.byref(ib), C.byref(nc))
            assert rc == P.CKPT_EINVAL and b"needs" in P.lib().ckpt_last_error(None)
            _, I, n_chunks = O.layout(sizes, A, Cb)
            assert (ib.value, nc.value) == (I, n_chunks)


def test_noalloc_pack_refuses_what_exceeds_its_scratch(P):
    import ctypes as C

    fake = 0x10000
    arr = (P.ckpt_tensor * 65537)()
    ib, nc = C.c_uint64(), C.c_uint64()
    args = (C.c_void_p(fake), 1 << 40, C.c_void_p(fake), 1 << 30, None, C.byref(ib), C.byref(nc))
    assert P.lib().ckpt_pack_noalloc(arr, 65537, 0, 0, 0, *args) == P.CKPT_EINVAL
    assert b"at most 65536" in P.lib().ckpt_last_error(None)
    arr[0].dev_ptr, arr[0].nbytes = fake, 100
    assert P.lib().ckpt_pack_noalloc(arr, 1, 2 << 30, 0, 0, *args) == P.CKPT_EINVAL
    assert b"1 GiB" in P.lib().ckpt_last_error(None)
    assert P.lib().ckpt_pack_noalloc(arr, 1, 1000, 256, 0, *args) == P.CKPT_EINVAL  # chunk not a multiple of 256
    assert P.lib().ckpt_pack_noalloc(arr, 1, 0, 0, 0, C.c_void_p(fake + 8), 1 << 40, C.c_void_p(fake), 1 << 30, None,
                                     C.byref(ib), C.byref(nc)) == P.CKPT_EINVAL
    assert b"aligned" in P.lib().ckpt_last_error(None)


def test_canary_of_the_header_and_the_binding_agree(P):
    import codecs

    line = [l for l in open(HEADER) if l.startswith("#define CKPT_CANARY")][0]
    pieces = re.findall(r'"((?:[^"\\]|\\.)*)"', line)
    value = b"".join(codecs.escape_decode(p.encode())[0] for p in pieces)
    assert value == P.CKPT_CANARY and len(value) == 16


@st.composite
def layouts(draw):
    """A fragment list and a geometry: alignment 16..4096, chunk a multiple of
    it, group a multiple of the chunk (0 = the default), fragment sizes mixing
    empty, tiny, sub-chunk and multi-chunk ones, at least one byte in all."""
    A = 1 << draw(st.integers(4, 12))
    C = A * draw(st.integers(1, max(1, (64 << 10) // A)))
    G = C * draw(st.integers(0, 5))
    size = st.one_of(st.just(0), st.integers(1, 300), st.integers(1, 5000), st.integers(1, 2 * C))
    sizes = draw(st.lists(size, min_size=1, max_size=40).filter(any))
    return sizes, C, A, G


@settings(max_examples=150, deadline=None, suppress_health_check=[HealthCheck.too_slow])
@given(layouts())
def test_direct_plan_properties(P, layout):
    """The direct D2H copy plan over random layouts, with the same byte-by-byte
    check as the fixed cases."""
    sizes, C, A, G = layout
    check_direct_plan(P, sizes, C, A, G)


@settings(max_examples=150, deadline=None, suppress_health_check=[HealthCheck.too_slow])
@given(layouts())
def test_layout_and_tile_plan_properties(P, layout):
    """Layout and tile table over random layouts: offsets, image size and chunk
    count equal the oracle's, and each tile's first and last fragment hold its
    first and last byte."""
    sizes, C, A, _ = layout
    off, I, nc = O.layout(sizes, A, C)
    poff, pI, pnc = P.ckpt_plan(sizes, C, A)
    assert [int(o) for o in poff] == [int(o) for o in off] and (pI, pnc) == (I, nc)
    tb, tf, tl = P.ckpt_debug_tile_plan(sizes, C, A)
    assert C % tb == 0 and tb & (tb - 1) == 0 and 16 <= tb <= 8192
    nonempty = [i for i, n in enumerate(sizes) if n]
    starts = np.array([int(off[i]) for i in nonempty])

    def holder(x):  # last non-empty fragment starting at or before x
        return nonempty[int(np.searchsorted(starts, x, side="right")) - 1]

    assert len(tf) == -(-I // tb)
    for t in range(len(tf)):
        x0, x1 = t * tb, min((t + 1) * tb, I) - 1
        assert tf[t] == holder(x0) and tl[t] == holder(x1), t
