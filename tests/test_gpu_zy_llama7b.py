"""The 7B LLaMA shard (94.3 GB of state; needs an MI355X and about 200 GB of
free host RAM).

Two 94.3 GB host images do not fit in the pinned memory the host grants (on
the 295 GB MI355X host used here, 16 GiB pinned blocks were refused after
64 GiB, and a second 94.3 GB image after a first one), so this shard runs
with pageable images behind 4 GiB pinned bounce rings.  Runs after the other
GPU tests; skips when the host has too little free memory for both images.
"""
import gc

import numpy as np
import pytest
import torch

import workloads as W
from gpu_util import host_bytes
from test_gpu_fullsize import check_shard

pytestmark = pytest.mark.gpu

if torch.cuda.is_available():
    import paper_2607_01646_amd as P


def _host_mem_gib(key="MemAvailable:"):
    try:
        for line in open("/proc/meminfo"):
            if line.startswith(key):
                return int(line.split()[1]) / (1 << 20)
    except OSError:
        pass
    return 0.0


@pytest.mark.timeout(900)
def test_llama7b_shard_pageable_images():
    """7B LLaMA: 1164 fragments, 94.3 GB, 64 MiB chunks, full device staging,
    1 GiB groups through two 4 GiB pinned rings.  Every one of the 1406
    chunks is compared byte for byte with the oracle's pack of the live
    fragments and every stored sum with the oracle's sum; every chunk then
    verifies on the GPU; after the tensors are trashed, the restore brings
    back every fragment (torch digests taken before the snapshot), and a few
    fragments are also compared byte for byte with host copies."""
    need = 2 * W.payload_bytes(4) / (1 << 30) + 8 + 16
    if _host_mem_gib() < need:
        pytest.skip("two pageable 94.3 GB images need about %.0f GiB of free host memory; %.0f GiB available"
                    % (need, _host_mem_gib()))
    pick = [0, 1, 2, 3, 577, 1160, 1161, 1162, 1163]
    tensors, _ = W.make_state(4, device="cuda")
    keep = {i: host_bytes(tensors[i]) for i in pick}
    del tensors
    gc.collect()
    torch.cuda.empty_cache()
    ck, tensors, plan, snap = check_shard(4, full_restore=False, bounce=4 << 30, digests=True)
    assert ck.n_chunks == 1406
    for i in pick:  # the same seeded state, restored byte for byte
        assert np.array_equal(host_bytes(tensors[i]), keep[i]), "fragment %d" % i
    ck.close()
    del tensors
    gc.collect()
    torch.cuda.empty_cache()


@pytest.mark.timeout(900)
def test_llama7b_shard_direct_d2h():
    """The same shard in direct D2H mode, as the benchmark's overlap leg runs
    it: no device staging (the engines copy the 1164 fragments from the
    tensors into 4 GiB pinned rings, host threads move them into the pageable
    images).  Every chunk and sum against the oracle, every chunk verified,
    every fragment restored through the four-group restore ring (digests)."""
    need = 2 * W.payload_bytes(4) / (1 << 30) + 8 + 16
    if _host_mem_gib() < need:
        pytest.skip("two pageable 94.3 GB images need about %.0f GiB of free host memory; %.0f GiB available"
                    % (need, _host_mem_gib()))
    ck, tensors, plan, snap = check_shard(4, full_restore=False, bounce=4 << 30, digests=True, direct=True)
    assert ck.n_chunks == 1406
    ck.close()
    del tensors
    gc.collect()
    torch.cuda.empty_cache()
