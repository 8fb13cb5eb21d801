"""Pageable host images behind pinned bounce rings, against the CPU oracle
(needs an MI355X).

Same bar as the pinned path: image bytes, chunk sums, restored tensors and
bad-chunk lists are compared byte for byte with the oracle.  The rings are
kept small (two or three chunk groups) so that every snapshot reuses each
slot several times, also across consecutive snapshots.
"""
import numpy as np
import pytest
import torch

import oracle as O
import workloads as W
from gpu_util import EDGE_SIZES, garbage_fill, host_bytes, random_byte_fragments, snapshot_and_check
from test_gpu_parity import check_committed_image_survives

pytestmark = pytest.mark.gpu

if torch.cuda.is_available():
    import paper_2607_01646_amd as P


@pytest.mark.parametrize("chunk,staging,group,bounce,threads", [
    (4096, 0, 4096, 2 * 4096, 0),             # one-chunk groups, two slots
    (4096, 0, 3 * 4096, 6 * 4096, 3),         # three-chunk groups, two slots, three threads
    (8192, 4 * 8192, 0, 3 * 8192, 1),         # device ring of four slots, bounce ring of three
    (1 << 16, 0, 1 << 16, 5 << 16, 16),       # more slots than needed, more threads than parts
])
def test_edge_sizes_through_bounce_rings(chunk, staging, group, bounce, threads):
    tensors, host = random_byte_fragments(EDGE_SIZES, seed=chunk + bounce)
    ck, _ = snapshot_and_check(tensors, host, chunk, staging=staging, group=group, bounce=bounce, threads=threads)
    ck.close()


@pytest.mark.parametrize("group,launch,bounce", [
    (4096, 4 * 4096, 2 * 4096),          # four one-chunk groups per pack launch, a ring of two groups
    (2 * 4096, 8 * 4096, 3 * 2 * 4096),  # four two-chunk groups per launch, a ring of three
])
def test_several_groups_per_pack_launch_through_bounce_rings(group, launch, bounce):
    """Pack launches of several groups, each group its own DMA request into the
    bounce ring (the layout the benchmark uses for pageable images)."""
    tensors, host = random_byte_fragments(EDGE_SIZES, seed=group + launch)
    ck, first = snapshot_and_check(tensors, host, 4096, group=group, bounce=bounce, launch=launch)
    # a second snapshot reuses the ring slots and fills the other image
    snap = ck.snapshot(step=4)
    ck.wait_committed(snap)
    img, sums = ck.host_image(snap)
    want, _, _ = O.pack(host, 256, 4096)
    assert np.array_equal(img, want)
    assert np.array_equal(sums, O.chunk_sums(want, 0, want.size, 4096))
    assert ck.state(first) == P.CKPT_SNAP_COMMITTED and ck.verify(first) == []  # the other image still holds it
    ck.close()


def test_large_groups_use_the_copy_pool():
    """Groups of 32 MiB, so that each ring-to-image copy is cut into parts
    run by several threads."""
    sizes = [int(s) for s in np.random.default_rng(3).integers(1 << 20, 24 << 20, 12)]
    tensors, host = random_byte_fragments(sizes, seed=4)
    ck, _ = snapshot_and_check(tensors, host, 1 << 22, group=32 << 20, bounce=64 << 20, threads=8)
    ck.close()


def test_consecutive_snapshots_reuse_slots_and_images():
    """Six snapshots of changing state through a two-slot ring, each issued
    right after the previous one committed: each committed image equals the
    oracle's pack of the state it captured, and the older image keeps its own
    snapshot."""
    torch.manual_seed(5)
    tensors = [torch.randn(n, device="cuda") for n in (70_001, 1 << 18, 3, 1 << 19, 12_345)]
    chunk = 1 << 16
    ck = P.Checkpointer(tensors, chunk_bytes=chunk, group_bytes=chunk, bounce_bytes=2 * chunk, host_threads=2)
    states, snaps = [], []
    for step in range(6):
        states.append([host_bytes(t) for t in tensors])
        s = ck.snapshot(step=step)
        ck.wait_captured(s)
        for t in tensors:
            t.mul_(-1.5).add_(0.25)
        snaps.append(s)
        ck.wait_committed(s)
        if step % 2 == 1:
            for k in (step - 1, step):
                img, sums = ck.host_image(snaps[k])
                want, _, _ = O.pack(states[k], 256, chunk)
                assert np.array_equal(img, want), "snapshot %d" % k
                assert np.array_equal(sums, O.chunk_sums(want, 0, want.size, chunk))
    assert ck.restore(snaps[4]) == []
    torch.cuda.synchronize()
    for t, h in zip(tensors, states[4]):
        assert np.array_equal(host_bytes(t), h)
    ck.close()


def test_flips_in_the_pageable_image_are_located():
    sizes = [int(s) for s in np.random.default_rng(31).integers(1000, 300_000, 64)]
    tensors, host = random_byte_fragments(sizes, seed=32)
    chunk = 65536
    ck = P.Checkpointer(tensors, chunk_bytes=chunk, group_bytes=chunk, bounce_bytes=3 * chunk)
    snap = ck.snapshot()
    ck.wait_committed(snap)
    img, sums = ck.host_image(snap)
    ranges = [(c * chunk, min((c + 1) * chunk, img.size)) for c in range(ck.n_chunks)]
    flips = W.flip_positions(ranges, n_flips=32, seed=2005)
    for c, byte, bit in flips:
        img[byte] ^= np.uint8(1 << bit)
    want_bad = sorted(c for c, _, _ in flips)
    assert ck.verify(snap) == want_bad
    flipped = img.copy()
    assert np.array_equal(P.ckpt_last_sums(ck.ctx), O.chunk_sums(flipped, 0, flipped.size, chunk))
    garbage_fill(tensors)
    assert ck.restore(snap) == want_bad
    torch.cuda.synchronize()
    back = O.restore_window(flipped, 0, flipped.size, ck.offsets, sizes)
    for t, b in zip(tensors, back):
        assert np.array_equal(host_bytes(t), b)
    ck.close()


def test_interrupted_snapshot_through_bounce_ring():
    """Invariant I4 with pageable images: the interrupted snapshot stays
    ABORTED, the previous one restores, and the next one commits."""
    torch.manual_seed(6)
    tensors = [torch.randn(1 << 18, device="cuda") for _ in range(16)]
    chunk = 1 << 18
    ck = P.Checkpointer(tensors, chunk_bytes=chunk, group_bytes=chunk, bounce_bytes=2 * chunk)
    s1 = ck.snapshot(step=1)
    ck.wait_committed(s1)
    good = [host_bytes(t) for t in tensors]
    for t in tensors:
        t.add_(3.0)
    P.ckpt_debug_interrupt_next(ck.ctx, 3)
    s2 = ck.snapshot(step=2)
    torch.cuda.synchronize()
    assert ck.state(s2) == P.CKPT_SNAP_ABORTED
    garbage_fill(tensors)
    assert ck.restore(0) == []
    torch.cuda.synchronize()
    for t, h in zip(tensors, good):
        assert np.array_equal(host_bytes(t), h)
    s3 = ck.snapshot(step=3)
    ck.wait_committed(s3)
    img, _ = ck.host_image(s3)
    want, _, _ = O.pack(good, 256, chunk)
    assert np.array_equal(img, want)
    ck.close()


def test_verify_beside_an_inflight_bounce_snapshot():
    torch.manual_seed(7)
    tensors = [torch.randn(1 << 20, device="cuda") for _ in range(64)]  # 256 MiB
    chunk = 1 << 22
    ck = P.Checkpointer(tensors, chunk_bytes=chunk, group_bytes=1 << 24, bounce_bytes=1 << 25)
    host1 = [host_bytes(t) for t in tensors]
    s1 = ck.snapshot(step=1)
    ck.wait_committed(s1)
    for t in tensors:
        t.mul_(-1.0)
    host2 = [host_bytes(t) for t in tensors]
    s2 = ck.snapshot(step=2)
    assert ck.verify(s1) == []
    ck.wait_committed(s2)
    for s, h in ((s1, host1), (s2, host2)):
        img, sums = ck.host_image(s)
        want, _, _ = O.pack(h, 256, chunk)
        assert np.array_equal(img, want)
        assert np.array_equal(sums, O.chunk_sums(want, 0, want.size, chunk))
    ck.close()


def test_a_committed_image_exists_while_a_bounce_snapshot_is_in_flight():
    check_committed_image_survives(1 << 25)


def test_bounce_configuration_errors():
    t = [torch.zeros(1 << 20, device="cuda")]
    with pytest.raises(P.CkptError) as e:  # smaller than two chunks: rejected at create
        P.Checkpointer(t, chunk_bytes=1 << 16, bounce_bytes=1 << 16)
    assert e.value.code == P.CKPT_EINVAL
    with pytest.raises(P.CkptError) as e:  # fewer than two groups of 1 MiB
        P.Checkpointer(t, chunk_bytes=1 << 16, group_bytes=1 << 20, bounce_bytes=1 << 20)
    assert e.value.code == P.CKPT_EINVAL
    with pytest.raises(P.CkptError) as e:
        P.Checkpointer(t, chunk_bytes=1 << 16, bounce_bytes=1 << 20, host_threads=1000)
    assert e.value.code == P.CKPT_EINVAL
