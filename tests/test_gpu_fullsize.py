"""Full-size shards against the oracle (needs an MI355X; tens of seconds each).

Every chunk of the committed host image is compared byte for byte with the
oracle's pack of the live fragments, and every stored sum with the oracle's
sum of that chunk, streamed chunk by chunk over a pool of host threads
(gpu_util.check_image_against_oracle).  The restore is compared with device
copies taken before the snapshot where device memory allows, else with
per-fragment digests taken by torch before the snapshot.
"""
import gc

import numpy as np
import pytest
import torch

import oracle as O
import workloads as W
from gpu_util import assert_located, check_image_against_oracle, fragment_digests

pytestmark = pytest.mark.gpu

if torch.cuda.is_available():
    import paper_2607_01646_amd as P


@pytest.fixture(autouse=True)
def release_memory():
    yield
    gc.collect()
    if torch.cuda.is_available():
        torch.cuda.empty_cache()


def check_shard(wid, staging=0, full_restore=True, bounce=0, digests=False, direct=False):
    """Snapshot workload wid, check every chunk and sum against the oracle,
    verify, then trash the tensors, restore and check every fragment: against
    device copies (full_restore) or against torch digests taken before the
    snapshot (digests; for shards too large to copy on the device)."""
    tensors, plan = W.make_state(wid, device="cuda")
    sizes = [p[1] for p in plan]
    chunk = W.WORKLOADS[wid]["chunk"]
    torch.cuda.synchronize()
    before = [t.clone() for t in tensors] if full_restore else None
    dig = fragment_digests(tensors) if digests else None
    ck = P.Checkpointer(tensors, [p[2] for p in plan], [p[3] for p in plan], chunk_bytes=chunk,
                        device_staging_bytes=staging, bounce_bytes=bounce, direct=direct)
    off, I, nc = O.layout(sizes, 256, chunk)
    assert np.array_equal(ck.offsets, off) and (ck.image_bytes, ck.n_chunks) == (I, nc)
    snap = ck.snapshot(step=wid)
    ck.wait_committed(snap)
    img, sums = ck.host_image(snap)
    assert check_image_against_oracle(tensors, off, sizes, img, sums, chunk) == nc
    assert ck.verify(snap) == []
    if full_restore or digests:
        for t in tensors:
            t.view(-1).view(torch.uint8).fill_(0x3C)
        assert ck.restore(snap) == []
        torch.cuda.synchronize()
    if full_restore:
        for i, (t, b) in enumerate(zip(tensors, before)):
            assert torch.equal(t.view(-1).view(torch.uint8), b.view(-1).view(torch.uint8)), "fragment %d" % i
    if digests:
        after = fragment_digests(tensors)
        wrong = [i for i, (a, b) in enumerate(zip(dig, after)) if a != b]
        assert not wrong, "%d fragments not restored, first %d" % (len(wrong), wrong[0])
    return ck, tensors, plan, snap


def test_gpt_1_3b_shard():
    """24 layers, hidden 2048: 1168 fragments, 18.42 GB, 64 MiB chunks."""
    ck, *_ = check_shard(2)
    assert ck.n_chunks == 275
    ck.close()


def test_llama65b_tp8pp8_rank_shard():
    """One rank of a 65B LLaMA under TP=8 x PP=8: 360 fragments, 14.17 GB."""
    ck, *_ = check_shard(3)
    assert ck.n_chunks == 212
    ck.close()


@pytest.mark.parametrize("bounce", [0, 4 << 30])
def test_llama65b_tp8pp8_rank_shard_direct(bounce):
    """The same rank with direct D2H (no device staging; the engines copy the
    fragments, pinned images or pageable ones behind 4 GiB rings): every
    chunk and sum against the oracle, every fragment restored through the
    four-group restore ring."""
    ck, *_ = check_shard(3, bounce=bounce, direct=True)
    assert ck.n_chunks == 212
    ck.close()


@pytest.mark.parametrize("staging,bounce", [(1 << 30, 0), (256 << 20, 4 << 30)])
def test_llama65b_tp8pp8_rank_shard_ring_staging(staging, bounce):
    """The same rank through a bounded device staging ring (1 GiB of four
    256 MiB slots, or four one-chunk slots with pageable images behind 4 GiB
    rings): the packs follow the copies out of each slot, and every chunk,
    sum and restored fragment still matches."""
    ck, *_ = check_shard(3, staging=staging, bounce=bounce)
    assert ck.n_chunks == 212
    ck.close()


def test_llama65b_rank_shard_in_full_precision():
    """The same rank with every tensor in fp32, the paper's training setting:
    360 fragments, 16.19 GB (16 bytes per parameter)."""
    ck, tensors, plan, _ = check_shard(6)
    assert ck.n_chunks == 242 and sum(p[1] for p in plan) == 16_192_634_880
    assert all(p[2] == W.DT_FP32 for p in plan)
    assert torch.equal(tensors[0], tensors[1])  # the parameter equals its master copy
    ck.close()


def test_stress_4096_fragments_with_flips():
    """4096 fragments (8 GiB, bf16/fp32 alternating, 1 KiB .. ~21 MiB) with 32
    seeded single-bit flips in distinct chunks: all reported and located."""
    ck, tensors, plan, snap = check_shard(5)
    sizes = [p[1] for p in plan]
    chunk = W.WORKLOADS[5]["chunk"]
    img, sums = ck.host_image(snap)
    stored = sums.copy()
    ranges = [(c * chunk, min((c + 1) * chunk, img.size)) for c in range(ck.n_chunks)]
    flips = W.flip_positions(ranges, n_flips=32, seed=2005)
    for c, byte, bit in flips:
        img[byte] ^= np.uint8(1 << bit)
    bad = ck.restore(snap)
    assert bad == sorted(c for c, _, _ in flips)
    recomputed = P.ckpt_last_sums(ck.ctx)
    for c, byte, bit in flips:
        k = 8 * (byte % 8) + bit
        was_set = (int(img[byte]) >> bit) & 1 == 0
        assert (int(recomputed[c]) - int(stored[c])) % (1 << 64) == ((-(1 << k)) % (1 << 64) if was_set else 1 << k)
        assert assert_located(ck, c, chunk, sizes)
    ck.close()


@pytest.mark.parametrize("shift", [0, 3])
def test_fragment_beyond_4_gib(shift):
    """One 4.5 GiB fragment (16-byte aligned, or a view 3 bytes into its
    buffer) between two small ones: image offsets, tile offsets and the
    funnel-shifted reads all pass 2^32 bytes within the fragment."""
    n = (9 << 29) + 5  # 4.5 GiB + 5 bytes
    flat = torch.empty(n + 16, dtype=torch.uint8, device="cuda")
    g = torch.Generator(device="cuda").manual_seed(4242)
    flat.copy_(torch.randint(0, 256, (n + 16,), generator=g, device="cuda", dtype=torch.uint8))
    small_a = torch.arange(777, dtype=torch.int32, device="cuda")
    small_b = torch.full((1001,), 0xA7, dtype=torch.uint8, device="cuda")
    tensors = [small_a, flat[shift:shift + n], small_b]
    sizes = [777 * 4, n, 1001]
    chunk = 64 << 20
    torch.cuda.synchronize()
    before = [t.clone() for t in tensors]
    outside = torch.cat([flat[:shift], flat[shift + n:]]).clone()  # bytes of the buffer outside the view
    ck = P.Checkpointer(tensors, chunk_bytes=chunk)
    off, I, nc = O.layout(sizes, 256, chunk)
    assert np.array_equal(ck.offsets, off) and (ck.image_bytes, ck.n_chunks) == (I, nc)
    snap = ck.snapshot(step=1)
    ck.wait_committed(snap)
    img, sums = ck.host_image(snap)
    # every chunk, including those around the big fragment's byte 2^32
    assert check_image_against_oracle(tensors, off, sizes, img, sums, chunk) == nc
    assert ck.verify(snap) == []
    for t in tensors:
        t.view(-1).view(torch.uint8).fill_(0x3C)
    assert ck.restore(snap) == []
    torch.cuda.synchronize()
    for i, (t, b) in enumerate(zip(tensors, before)):
        assert torch.equal(t.view(-1).view(torch.uint8), b.view(-1).view(torch.uint8)), "fragment %d" % i
    # the scatter never writes outside the view
    assert torch.equal(torch.cat([flat[:shift], flat[shift + n:]]), outside)
    ck.close()
