"""The 7B LLaMA shard (94.3 GB of state) through a ring of device staging
slots (needs an MI355X and room for two pinned host images of 94.3 GB).

Runs after the other GPU tests.  Pinned host memory comes from a driver pool
that is much smaller than host RAM: on the 295 GB MI355X host used here,
16 GiB pinned blocks were refused after 64 GiB, and a second 94.3 GB image
after a first one.  The test runs only when half of the host RAM covers both
images, and skips with that reason otherwise.
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


def _host_mem_gib(key="MemTotal:"):
    try:
        for line in open("/proc/meminfo"):
            if line.startswith(key):
                return int(line.split()[1]) / (1 << 20)
    except OSError:
        pass
    return 0.0


@pytest.mark.timeout(600)
def test_llama7b_shard_ring_staging():
    """7B LLaMA: 1164 fragments, 94.3 GB, 64 MiB chunks through a ring of 8
    staging slots (512 MiB of device staging); sampled chunks and a sampled
    restore."""
    need = 2 * W.payload_bytes(4) / (1 << 30) + 8
    if _host_mem_gib() / 2 < need:
        pytest.skip("two pinned images need %.0f GiB; the driver's pinned pool on a %.0f GiB host is smaller "
                    "(64 GiB in 16 GiB blocks was measured on such a host)" % (need, _host_mem_gib()))
    ck, tensors, plan, snap = check_shard(4, staging=8 * (64 << 20), full_restore=False, all_sums=False)
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
