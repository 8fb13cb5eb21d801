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
    1 GiB groups through two 4 GiB pinned rings; sampled chunks against the
    oracle, verify of every chunk, and a sampled restore."""
    need = 2 * W.payload_bytes(4) / (1 << 30) + 8 + 16
    if _host_mem_gib() < need:
        pytest.skip("two pageable 94.3 GB images need about %.0f GiB of free host memory; %.0f GiB available"
                    % (need, _host_mem_gib()))
    ck, tensors, plan, snap = check_shard(4, full_restore=False, all_sums=False, bounce=4 << 30)
    assert ck.n_chunks == 1406
    pick = [0, 1, 2, 3, 577, 1160, 1161, 1162, 1163]
    keep = {i: host_bytes(tensors[i]) for i in pick}
    for i in pick:
        tensors[i].view(-1).view(torch.uint8).fill_(0x77)
    assert ck.restore(snap) == []
    torch.cuda.synchronize()
    for i in pick:
        assert np.array_equal(host_bytes(tensors[i]), keep[i])
    ck.close()
    del tensors
    gc.collect()
    torch.cuda.empty_cache()
