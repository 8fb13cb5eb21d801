"""GPU path against the CPU oracle, bit for bit (needs an MI355X).

Every comparison is byte-exact: the snapshot image, the chunk sums, the
restored tensors, the bad-chunk lists and the envelope.  Inputs come from the
seeded generators in `workloads` or numpy; expected values come only from
`oracle`.
"""
import struct

import numpy as np
import pytest
import torch

import oracle as O
import workloads as W
from gpu_util import (EDGE_SIZES, ENDS_EMPTY, assert_located, garbage_fill, host_bytes, pick_stream,
                      random_byte_fragments, snapshot_and_check)

pytestmark = pytest.mark.gpu

if torch.cuda.is_available():
    import paper_2607_01646_amd as P


@pytest.mark.parametrize("chunk,align,staging,group,launch", [
    (4096, 256, 0, 4096, 3 * 4096),    # pack launches of three one-chunk groups, each group its own copy
    (8192, 256, 0, 2 * 8192, 5 * 8192),  # launch size rounded down to two groups of two chunks
    (4096, 16, 0, 4096, 1),            # launch smaller than a group: one group per launch
])
def test_edge_sizes_multi_group_launches(chunk, align, staging, group, launch):
    tensors, host = random_byte_fragments(EDGE_SIZES, seed=chunk + launch)
    ck, _ = snapshot_and_check(tensors, host, chunk, align, staging, group, launch=launch)
    ck.close()


@pytest.mark.parametrize("chunk,align,staging,group", [
    (4096, 256, 0, 0),                 # many chunks, one launch
    (4096, 256, 0, 3 * 4096),          # three chunks per launch and copy
    (768, 256, 0, 0),                  # chunk not a power of two (256-byte tiles)
    (1 << 20, 256, 0, 0),              # chunk larger than most fragments
    (65536, 16, 0, 65536),             # 16-byte alignment, one chunk per group
    (8192, 256, 4 * 8192, 0),          # ring of four device slots
    (4096, 256, 12 * 4096, 3 * 4096),  # ring of four slots of three chunks each
    (4096, 256, 4 * 4096, 8 * 4096),   # ring slot size capped at half the ring: two slots of two chunks
    (4096, 256, 16 * 4096, 0),         # default ring slots: a quarter of the ring, four slots of four chunks
    (1 << 16, 4096, 2 * (1 << 16), 0), # ring of two slots, 4 KiB alignment
    (16, 16, 0, 0),                    # chunk = alignment = one 16-byte vector: 16-byte tiles
    (48, 16, 0, 1 << 16),              # three-vector chunks, 1365 per group
])
def test_edge_sizes_all_geometries(chunk, align, staging, group):
    tensors, host = random_byte_fragments(EDGE_SIZES, seed=chunk + align)
    ck, _ = snapshot_and_check(tensors, host, chunk, align, staging, group)
    ck.close()


@pytest.mark.parametrize("staging,group,bounce", [
    (0, 0, 0),                  # full device image, pinned host images
    (4 * 4096, 4096, 0),        # ring of four one-chunk slots
    (0, 4096, 2 * 4096),        # pageable images behind a ring of two one-chunk groups
])
def test_empty_fragments_at_both_ends(staging, group, bounce):
    """Empty fragments first and last take no image space: the image starts
    with the first non-empty fragment and ends on the last one's padding."""
    tensors, host = random_byte_fragments(ENDS_EMPTY, seed=41 + staging + bounce)
    ck, _ = snapshot_and_check(tensors, host, 4096, 256, staging, group, bounce=bounce)
    ck.close()


def test_capped_grid_walks_tiles_grid_stride():
    """With the workgroup count capped, each workgroup loops over many tiles
    (pack, scatter and verify)."""
    tensors, host = random_byte_fragments(EDGE_SIZES, seed=5)
    for grid in [1, 7, 64]:
        ck, _ = snapshot_and_check(tensors, host, 1 << 16, grid=grid)
        ck.close()


def test_single_fragment_and_ragged_tail():
    for n in [1, 16, 17, 4 << 20, (4 << 20) + 3]:
        tensors, host = random_byte_fragments([n], seed=n)
        ck, _ = snapshot_and_check(tensors, host, 1 << 20)
        ck.close()


def test_many_small_fragments_in_one_tile():
    # 600 fragments of 1..40 bytes: 32 fragments per 8 KiB tile
    rng = np.random.default_rng(21)
    sizes = [int(s) for s in rng.integers(1, 41, 600)]
    tensors, host = random_byte_fragments(sizes, seed=22)
    ck, _ = snapshot_and_check(tensors, host, 1 << 20)
    ck.close()
    # more fragments in a tile than the LDS offset cache holds (empty ones are free)
    sizes = [0] * 3000 + [5, 0, 9] + [0] * 1500 + [300]
    tensors, host = random_byte_fragments(sizes, seed=23)
    ck, _ = snapshot_and_check(tensors, host, 1 << 16)
    ck.close()


@pytest.mark.parametrize("align", [256, 16])
def test_dense_tiny_fragments_at_odd_offsets(align):
    """60,000 fragments of 1..1199 bytes at arbitrary byte offsets in one
    buffer: nearly every tile holds several fragments with misaligned sources,
    so the multi-fragment path of pack and scatter carries the whole image.
    The restore must write every fragment back and leave the gaps between
    them untouched."""
    rng = np.random.default_rng(4242 + align)
    n = 60_000
    sizes = rng.integers(1, 1200, n)
    gaps = rng.integers(0, 64, n)
    offs = np.cumsum(gaps + np.concatenate(([0], sizes[:-1])))
    total = int(offs[-1] + sizes[-1] + 64)
    host_all = rng.integers(0, 256, total, dtype=np.uint8)
    dev_all = torch.from_numpy(host_all.copy()).cuda()
    frags = [dev_all[int(o):int(o) + int(z)] for o, z in zip(offs, sizes)]
    host = [host_all[int(o):int(o) + int(z)] for o, z in zip(offs, sizes)]
    chunk = 1 << 20
    ck = P.Checkpointer(frags, chunk_bytes=chunk, align_bytes=align)
    snap = ck.snapshot(step=1)
    ck.wait_committed(snap)
    img, sums = ck.host_image(snap)
    want, off, nc = O.pack(host, align, chunk)
    assert np.array_equal(ck.offsets, off) and img.size == want.size
    diff = np.flatnonzero(img != want)
    assert diff.size == 0, "image differs at %d bytes, first at %d" % (diff.size, diff[0])
    assert np.array_equal(sums, O.chunk_sums(want, 0, want.size, chunk))
    dev_all.fill_(0x5A)
    assert ck.restore(snap) == []
    torch.cuda.synchronize()
    got = dev_all.cpu().numpy()
    in_frag = np.zeros(total, dtype=bool)
    starts, ends = offs, offs + sizes
    marks = np.zeros(total + 1, dtype=np.int64)
    np.add.at(marks, starts, 1)
    np.add.at(marks, ends, -1)
    in_frag = np.cumsum(marks[:-1]) > 0
    assert np.array_equal(got[in_frag], host_all[in_frag]), "a fragment byte was not restored"
    assert np.all(got[~in_frag] == 0x5A), "the restore wrote outside the fragments"
    ck.close()


def test_tiny_gpt_shard_bit_exact():
    """Workload 1: 4-layer GPT shard (208 fragments, 238.9 MB), 4 MiB chunks."""
    tensors, plan = W.make_state(1, device="cuda")
    torch.cuda.synchronize()
    host = [host_bytes(t) for t in tensors]
    ck, snap = snapshot_and_check(tensors, host, W.WORKLOADS[1]["chunk"], dtypes=[p[2] for p in plan],
                                  classes=[p[3] for p in plan])
    assert ck.n_chunks == 57 and sum(p[1] for p in plan) == 238_938_112
    ck.close()


def test_adversarial_bit_patterns_pass_unchanged():
    frags = W.adversarial_fragments("cuda")
    host = [host_bytes(t) for t in frags]
    ck, _ = snapshot_and_check(frags, host, 4096)
    ck.close()


def test_misaligned_views_restore_without_touching_neighbours():
    views, flats = W.misaligned_views("cuda")
    torch.cuda.synchronize()
    host = [host_bytes(v) for v in views]
    flat_before = [host_bytes(f) for f in flats]
    ck = P.Checkpointer(views, chunk_bytes=1 << 16)
    snap = ck.snapshot()
    ck.wait_committed(snap)
    img, sums = ck.host_image(snap)
    want, off, nc = O.pack(host, 256, 1 << 16)
    assert np.array_equal(img, want)
    assert np.array_equal(sums, O.chunk_sums(want, 0, want.size, 1 << 16))
    for v in views:  # trash only the registered views
        v.view(torch.uint8).fill_(0xEE) if v.dtype == torch.uint8 else v.view(torch.int16 if v.element_size() == 2
                                                                              else torch.int32).fill_(-7)
    assert ck.restore(snap) == []
    torch.cuda.synchronize()
    for f, b in zip(flats, flat_before):  # views restored, bytes between them untouched
        assert np.array_equal(host_bytes(f), b)
    ck.close()


def test_single_bit_flips_are_reported_and_located():
    """Seeded flips, one per chunk, in the committed pinned image: restore and
    verify report exactly those chunks; the recomputed sums equal the oracle's
    sums of the flipped image, and each delta is +-2^k as the closed form says."""
    sizes = [int(s) for s in np.random.default_rng(31).integers(1000, 300_000, 64)]
    tensors, host = random_byte_fragments(sizes, seed=32)
    chunk = 65536
    ck = P.Checkpointer(tensors, chunk_bytes=chunk)
    snap = ck.snapshot()
    ck.wait_committed(snap)
    img, sums = ck.host_image(snap)
    stored = sums.copy()
    ranges = [(c * chunk, min((c + 1) * chunk, img.size)) for c in range(ck.n_chunks)]
    flips = W.flip_positions(ranges, n_flips=32, seed=2005)
    for c, byte, bit in flips:
        img[byte] ^= np.uint8(1 << bit)
    want_bad = sorted(c for c, _, _ in flips)
    assert ck.verify(snap) == want_bad
    flipped = img.copy()
    recomputed = P.ckpt_last_sums(ck.ctx)
    assert np.array_equal(recomputed, O.chunk_sums(flipped, 0, flipped.size, chunk))
    for c, byte, bit in flips:
        k = 8 * (byte % 8) + bit
        was_set = (int(flipped[byte]) >> bit) & 1 == 0  # bit value before the flip
        delta = (int(recomputed[c]) - int(stored[c])) % (1 << 64)
        assert delta == ((-(1 << k)) % (1 << 64) if was_set else (1 << k))
        assert assert_located(ck, c, chunk, sizes)
    garbage_fill(tensors)
    assert ck.restore(snap) == want_bad  # every byte is still written back
    torch.cuda.synchronize()
    back = O.restore_window(flipped, 0, flipped.size, ck.offsets, sizes)
    for t, b in zip(tensors, back):
        assert np.array_equal(host_bytes(t), b)
    ck.close()


def _step_state(n_frag=48, numel=1 << 20, seed=41):
    g = torch.Generator(device="cuda").manual_seed(seed)
    return [torch.randn(numel, generator=g, device="cuda") for _ in range(n_frag)]


def _hold(stream, ms=40.0):
    """Keep `stream` busy for about `ms` milliseconds (a chain of fp32
    matmuls), so that a snapshot triggered after it starts packing late."""
    a = torch.randn(4096, 4096, device="cuda")
    with torch.cuda.stream(stream):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        b = a @ a
        e1.record()
    e1.synchronize()
    n = max(1, int(ms / max(e0.elapsed_time(e1), 1e-3)))
    with torch.cuda.stream(stream):
        for _ in range(n):
            b = a @ b
    return b


# Staging modes of the gate tests: the full device image (the gate waits for
# the pack only) and a ring of four 4 MiB slots over the 384 MiB state (each
# slot is reused only after its previous group has been copied to the host,
# so the capture of the later chunks is paced by the D2H).
GATE_STAGING = [0, 16 << 20]
GATE_CHUNK = 1 << 20


@pytest.mark.parametrize("launch", [3 << 20, 8 << 20])
def test_gate_with_multi_group_launches(launch):
    """Full-image staging with one-chunk groups packed several per launch:
    the gate on fragments [0, 8) waits for the launch holding their last
    chunk; an update of those fragments right after it stays out of the
    image, and so does an update of everything after a whole-range wait."""
    tensors = _step_state(n_frag=96)
    ck = P.Checkpointer(tensors, chunk_bytes=GATE_CHUNK, group_bytes=GATE_CHUNK, pack_launch_bytes=launch)
    main, side = torch.cuda.current_stream(), torch.cuda.Stream()
    for lo, hi in [(0, 8), (0, len(tensors))]:
        torch.cuda.synchronize()
        before = [host_bytes(t) for t in tensors]
        keep = _hold(main)
        s = ck.snapshot(step=hi, stream=main)
        ck.wait_captured(s, lo, hi, stream=side)
        with torch.cuda.stream(side):
            for t in tensors[lo:hi]:
                t.mul_(-1.0)
        ck.wait_committed(s)
        img, sums = ck.host_image(s)
        want, _, _ = O.pack(before, 256, GATE_CHUNK)
        off = ck.offsets
        end = int(off[hi - 1]) + before[hi - 1].size
        assert np.array_equal(img[:end], want[:end])
        if hi == len(tensors):
            assert np.array_equal(sums, O.chunk_sums(want, 0, want.size, GATE_CHUNK))
        torch.cuda.synchronize()
        del keep
    ck.close()


@pytest.mark.parametrize("staging", GATE_STAGING)
def test_gate_orders_optimizer_after_capture(staging):
    """The wait before the optimizer step: an in-place update launched on
    another stream right after ckpt_wait(CAPTURED) must not leak into the
    snapshot, although the snapshot's trigger sits behind ~40 ms of work on
    the training stream, so its pack starts long after the update could.
    Whole range, then a partial range [0, 8) that protects only those."""
    tensors = _step_state(n_frag=96)
    ck = P.Checkpointer(tensors, chunk_bytes=GATE_CHUNK, device_staging_bytes=staging)
    main, side = torch.cuda.current_stream(), torch.cuda.Stream()
    torch.cuda.synchronize()
    before = [host_bytes(t) for t in tensors]
    keep = _hold(main)
    s = ck.snapshot(step=1, stream=main)
    ck.wait_captured(s, 0, len(tensors), stream=side)
    with torch.cuda.stream(side):
        for t in tensors:
            t.add_(1.0)  # the "optimizer step"
    ck.wait_committed(s)
    img, sums = ck.host_image(s)
    want, _, _ = O.pack(before, 256, GATE_CHUNK)
    assert np.array_equal(img, want)
    assert np.array_equal(sums, O.chunk_sums(want, 0, want.size, GATE_CHUNK))
    torch.cuda.synchronize()
    before = [host_bytes(t) for t in tensors]
    keep = _hold(main)
    s = ck.snapshot(step=2, stream=main)
    ck.wait_captured(s, 0, 8, stream=side)
    with torch.cuda.stream(side):
        for t in tensors[:8]:
            t.mul_(2.0)
    ck.wait_committed(s)
    img, _ = ck.host_image(s)
    off = ck.offsets
    for i in range(8):
        o = int(off[i])
        assert np.array_equal(img[o:o + before[i].size], before[i])
    torch.cuda.synchronize()
    del keep
    ck.close()


@pytest.mark.parametrize("staging", GATE_STAGING)
def test_gate_negative_control_detects_the_race(staging):
    """Same without the wait: the update on the other stream runs while the
    pack still waits for its trigger, so the snapshot holds updated values.
    Shows the gate test can see a missing wait.  The pack runs on a stream
    of the test's, and the update on one probed to run beside it and the
    training stream (streams that share a hardware queue would run in
    submission order and hide the race)."""
    tensors = _step_state(n_frag=96)
    main = torch.cuda.current_stream()
    pk = pick_stream(main)
    side = pick_stream(main, pk)
    ck = P.Checkpointer(tensors, chunk_bytes=GATE_CHUNK, device_staging_bytes=staging, side_stream=pk)
    torch.cuda.synchronize()
    before = [host_bytes(t) for t in tensors]
    keep = _hold(main)
    s = ck.snapshot(step=1, stream=main)
    with torch.cuda.stream(side):
        for t in tensors:
            t.add_(1.0)  # no ckpt_wait: runs before the delayed pack
    ck.wait_committed(s)
    img, _ = ck.host_image(s)
    want, _, _ = O.pack(before, 256, GATE_CHUNK)
    assert not np.array_equal(img, want)
    torch.cuda.synchronize()
    del keep
    ck.close()


def test_ring_gate_covers_only_its_range():
    """Ring staging: the capture of the last chunks waits for ring slots to
    come back from the host link, so a wait on fragments [0, 8) (captured
    first) does not cover the last eight fragments.  Updating those after
    that wait races the D2H-paced pack and reaches the image; updating them
    after a wait on their own range does not.  Shows that in ring mode the
    gate's range decides what is protected.  The update runs on a stream
    probed to run beside the pack's."""
    tensors = _step_state(n_frag=96)
    pk = pick_stream(torch.cuda.current_stream())
    side = pick_stream(pk)
    ck = P.Checkpointer(tensors, chunk_bytes=GATE_CHUNK, device_staging_bytes=16 << 20, side_stream=pk)
    n = len(tensors)
    for lo, hi, leaks in [(0, 8, True), (n - 8, n, False)]:
        torch.cuda.synchronize()
        before = [host_bytes(t) for t in tensors]
        s = ck.snapshot(step=lo)
        ck.wait_captured(s, lo, hi, stream=side)
        with torch.cuda.stream(side):
            for t in tensors[n - 8:]:
                t.add_(1.0)
        ck.wait_committed(s)
        torch.cuda.synchronize()
        img, _ = ck.host_image(s)
        off = ck.offsets
        same = all(np.array_equal(img[int(off[i]):int(off[i]) + before[i].size], before[i]) for i in range(n - 8, n))
        assert same != leaks, "gate on [%d, %d): last fragments %s" % (lo, hi, "protected" if same else "updated")
        # the chunks before the updated fragments hold the state of the trigger either way
        o = int(off[n - 8])
        want, _, _ = O.pack(before, 256, GATE_CHUNK)
        assert np.array_equal(img[:o], want[:o])
    ck.close()


@pytest.mark.parametrize("staging", GATE_STAGING)
def test_trigger_captures_writes_queued_before_it(staging):
    """The trigger (row a2): a snapshot issued on after_stream is ordered after
    the work already enqueued there.  An in-place update of every registered
    tensor is queued on the training stream behind ~40 ms of other work; the
    snapshot call returns while that update is still pending, and the
    committed image must equal the oracle's pack of the updated bytes."""
    tensors = _step_state(n_frag=96)
    ck = P.Checkpointer(tensors, chunk_bytes=GATE_CHUNK, device_staging_bytes=staging)
    main = torch.cuda.current_stream()
    torch.cuda.synchronize()
    before = [host_bytes(t) for t in tensors]
    keep = _hold(main)
    for t in tensors:
        t.add_(1.0)  # queued on main behind the hold
    updated = torch.cuda.Event()
    updated.record(main)
    s = ck.snapshot(step=1, stream=main)
    assert not updated.query(), "the update ran before the snapshot call returned; the test proves nothing"
    ck.wait_committed(s)
    torch.cuda.synchronize()
    after = [host_bytes(t) for t in tensors]
    img, sums = ck.host_image(s)
    want, _, _ = O.pack(after, 256, GATE_CHUNK)
    assert np.array_equal(img, want)
    assert np.array_equal(sums, O.chunk_sums(want, 0, want.size, GATE_CHUNK))
    assert not np.array_equal(want, O.pack(before, 256, GATE_CHUNK)[0])
    del keep
    ck.close()


def test_trigger_negative_control_on_an_idle_stream():
    """Same, with the snapshot issued on an idle stream: nothing orders it
    after the update pending on the training stream, so it packs the bytes
    from before the update.  Shows the trigger test can see a missing order.
    Both the idle stream and the pack's are probed to run beside the
    training stream."""
    tensors = _step_state(n_frag=96)
    main = torch.cuda.current_stream()
    pk = pick_stream(main)
    idle = pick_stream(main)
    ck = P.Checkpointer(tensors, chunk_bytes=GATE_CHUNK, side_stream=pk)
    torch.cuda.synchronize()
    before = [host_bytes(t) for t in tensors]
    keep = _hold(main)
    for t in tensors:
        t.add_(1.0)
    s = ck.snapshot(step=1, stream=idle)
    ck.wait_committed(s)
    img, _ = ck.host_image(s)
    want, _, _ = O.pack(before, 256, GATE_CHUNK)
    assert np.array_equal(img, want)
    torch.cuda.synchronize()
    del keep
    ck.close()


@pytest.mark.parametrize("staging,bounce", [(16 << 20, 0), (0, 0), (16 << 20, 8 << 20)])
def test_poison_canary_never_reaches_an_image(staging, bounce):
    """ckpt_config.poison: each staging area is filled with the canary after
    its previous copy and before it is packed again.  Over several snapshots
    (each gated update changing every fragment) every committed image equals
    the oracle's pack and holds no 16-byte-aligned copy of the canary: the
    pack always overwrites the canary before a copy reads the area.  Ring
    staging (pinned and pageable images) and the full-size image."""
    tensors = _step_state(n_frag=96)
    ck = P.Checkpointer(tensors, chunk_bytes=GATE_CHUNK, device_staging_bytes=staging, bounce_bytes=bounce,
                        poison=True)
    canary = np.frombuffer(P.CKPT_CANARY, dtype=np.uint8)
    for k in range(3):
        torch.cuda.synchronize()
        before = [host_bytes(t) for t in tensors]
        s = ck.snapshot(step=k)
        ck.wait_captured(s, 0, len(tensors))
        for t in tensors:
            t.mul_(-1.0)  # the gated update
        ck.wait_committed(s)
        img, sums = ck.host_image(s)
        want, _, _ = O.pack(before, 256, GATE_CHUNK)
        assert np.array_equal(img, want), "snapshot %d" % k
        assert np.array_equal(sums, O.chunk_sums(want, 0, want.size, GATE_CHUNK))
        assert not np.any(np.all(img.reshape(-1, 16) == canary, axis=1))
        assert ck.verify(s) == []
    ck.close()


def test_side_stream_carries_the_pack():
    """ckpt_config.side_stream: the pack runs on the caller's stream, behind
    what the caller queued there.  With ~40 ms of work on that stream, the
    pack comes after an (ungated) update queued 5 ms later on the training
    stream, so the image holds the updated bytes; with the library's own
    stream the pack ran at once and holds the bytes from before.  The
    caller's stream outlives the context."""
    tensors = _step_state(n_frag=48)
    main = torch.cuda.current_stream()
    for use_side in (False, True):
        side = torch.cuda.Stream()
        ck = P.Checkpointer(tensors, chunk_bytes=GATE_CHUNK, side_stream=side if use_side else None)
        torch.cuda.synchronize()
        before = [host_bytes(t) for t in tensors]
        keep_side = _hold(side)
        s = ck.snapshot(step=1, stream=main)
        keep_main = _hold(main, 5.0)
        for t in tensors:
            t.add_(1.0)  # not gated: ordered only by where the pack runs
        ck.wait_committed(s)
        torch.cuda.synchronize()
        after = [host_bytes(t) for t in tensors]
        img, sums = ck.host_image(s)
        want, _, _ = O.pack(after if use_side else before, 256, GATE_CHUNK)
        assert np.array_equal(img, want), "side stream %s" % use_side
        assert np.array_equal(sums, O.chunk_sums(want, 0, want.size, GATE_CHUNK))
        ck.close()
        with torch.cuda.stream(side):  # still the caller's
            keep_side = keep_side + 1.0
        side.synchronize()
        del keep_side, keep_main


@pytest.mark.parametrize("launch", [0, 3 << 18])
def test_interrupted_snapshot_is_never_restored(launch):
    """Invariant I4: an offload interrupted after two chunk groups stays
    ABORTED; restore returns the previous committed snapshot.  With three
    groups per pack launch the interruption falls inside a launch."""
    tensors = _step_state(n_frag=16, numel=1 << 18)
    ck = P.Checkpointer(tensors, chunk_bytes=1 << 18, group_bytes=1 << 18, pack_launch_bytes=launch)
    s1 = ck.snapshot(step=1)
    ck.wait_committed(s1)
    good = [host_bytes(t) for t in tensors]
    for t in tensors:
        t.add_(3.0)
    P.ckpt_debug_interrupt_next(ck.ctx, 2)
    s2 = ck.snapshot(step=2)
    torch.cuda.synchronize()
    assert ck.state(s2) == P.CKPT_SNAP_ABORTED
    assert ck.state(s1) == P.CKPT_SNAP_COMMITTED
    with pytest.raises(P.CkptError) as e:
        ck.wait_committed(s2)
    assert e.value.code == P.CKPT_ESTATE
    garbage_fill(tensors)
    assert ck.restore(0) == []
    torch.cuda.synchronize()
    for t, h in zip(tensors, good):
        assert np.array_equal(host_bytes(t), h)
    # The next snapshot reuses the aborted image, never s1's.
    s3 = ck.snapshot(step=3)
    ck.wait_committed(s3)
    assert ck.state(s1) == P.CKPT_SNAP_COMMITTED and ck.state(s3) == P.CKPT_SNAP_COMMITTED
    assert ck.restore(s1) == []
    ck.close()


def test_ping_pong_roles_and_busy():
    tensors = _step_state(n_frag=64, numel=1 << 20)  # 256 MiB: copies take ~5 ms
    ck = P.Checkpointer(tensors, chunk_bytes=1 << 22)
    s1 = ck.snapshot(step=1)
    with pytest.raises(P.CkptError) as e:  # one snapshot in flight at a time
        ck.snapshot(step=2)
    assert e.value.code == P.CKPT_EBUSY
    ck.wait_committed(s1)
    s2 = ck.snapshot(step=2)  # the other image
    ck.wait_committed(s2)
    assert ck.state(s1) == P.CKPT_SNAP_COMMITTED and ck.state(s2) == P.CKPT_SNAP_COMMITTED
    s3 = ck.snapshot(step=3)  # takes s1's image
    ck.wait_committed(s3)
    assert ck.state(s1) == P.CKPT_SNAP_SUPERSEDED
    with pytest.raises(P.CkptError) as e:
        ck.restore(s1)
    assert e.value.code == P.CKPT_ENOSNAP
    assert ck.restore(s2) == [] and ck.restore(0) == []
    # A corrupted newest image: the other buffer still restores cleanly.
    img, _ = ck.host_image(s3)
    img[12345] ^= 0x40
    assert ck.verify(s3) == [12345 // (1 << 22)]
    assert ck.restore(s2) == []
    ck.close()


def check_committed_image_survives(bounce):
    """The ping-pong guarantee (Sec. VI-A; invariant I4): while a snapshot is
    in flight the newest committed one stays in its own image, restorable and
    verify-clean, and a further snapshot is refused until the first commits."""
    tensors = _step_state(n_frag=256, numel=1 << 20)  # 1 GiB: ~19 ms of D2H
    ck = P.Checkpointer(tensors, chunk_bytes=1 << 22, group_bytes=1 << 24, bounce_bytes=bounce)
    s1 = ck.snapshot(step=1)
    ck.wait_committed(s1)
    img1, _ = ck.host_image(s1)
    watch = 2 << 24
    head = img1[:watch].copy()
    for t in tensors:
        t.mul_(-1.0)
    s2 = ck.snapshot(step=2)
    with pytest.raises(P.CkptError) as e:
        ck.snapshot(step=3)
    assert e.value.code == P.CKPT_EBUSY
    polls = 0
    while ck.state(s2) != P.CKPT_SNAP_COMMITTED:
        assert ck.latest() == (s1, 1) and ck.state(s1) == P.CKPT_SNAP_COMMITTED
        assert np.array_equal(img1[:watch], head)
        polls += 1
    assert polls >= 1
    assert ck.verify(s1) == [] and ck.latest() == (s2, 2)
    ck.close()


def test_a_committed_image_exists_while_a_snapshot_is_in_flight():
    check_committed_image_survives(0)


def test_verify_runs_beside_an_inflight_snapshot():
    """Verify reads only the committed image, through its own staging ring,
    so it runs while a newer snapshot streams into the other image; both
    results match the oracle."""
    tensors = _step_state(n_frag=64, numel=1 << 20)  # 256 MiB
    ck = P.Checkpointer(tensors, chunk_bytes=1 << 22, group_bytes=1 << 24)
    host1 = [host_bytes(t) for t in tensors]
    s1 = ck.snapshot(step=1)
    ck.wait_committed(s1)
    for t in tensors:
        t.mul_(-1.0)
    host2 = [host_bytes(t) for t in tensors]
    s2 = ck.snapshot(step=2)
    assert ck.verify(s1) == []  # while s2's copies are in flight
    want1, _, _ = O.pack(host1, 256, 1 << 22)
    assert np.array_equal(P.ckpt_last_sums(ck.ctx), O.chunk_sums(want1, 0, want1.size, 1 << 22))
    ck.wait_committed(s2)
    img2, sums2 = ck.host_image(s2)
    want2, _, _ = O.pack(host2, 256, 1 << 22)
    assert np.array_equal(img2, want2) and np.array_equal(sums2, O.chunk_sums(want2, 0, want2.size, 1 << 22))
    img1, _ = ck.host_image(s1)
    assert np.array_equal(img1, want1)
    ck.close()


def test_envelope_matches_oracle():
    sizes = [100, 0, 4096, 33, 70_000]
    tensors, host = random_byte_fragments(sizes, seed=51)
    dtypes = [1, 2, 2, 0, 1]
    classes = [0, 1, 2, 3, 0]
    meta = b"tp=8;pp=8;dp=4;rng=" + struct.pack("<Q", 123456789)
    ck, snap = snapshot_and_check(tensors, host, 4096, dtypes=dtypes, classes=classes, meta=meta, step=77)
    env = ck.envelope(snap)
    img, sums = ck.host_image(snap)
    want = O.envelope(77, 256, 4096, ck.image_bytes, ck.offsets, sizes, dtypes, classes,
                      O.chunk_sums(O.pack(host, 256, 4096)[0], 0, ck.image_bytes, 4096), meta)
    assert env == want
    ck.close()


def test_error_codes():
    tensors, _ = random_byte_fragments([1000], seed=61)
    ctx = P.ckpt_create(chunk_bytes=4096)
    with pytest.raises(P.CkptError) as e:
        P.ckpt_snapshot_async(ctx)
    assert e.value.code == P.CKPT_ESTATE
    P.ckpt_register_tensors(ctx, tensors)
    with pytest.raises(P.CkptError) as e:
        P.ckpt_register_tensors(ctx, tensors)
    assert e.value.code == P.CKPT_ESTATE
    with pytest.raises(P.CkptError) as e:
        P.ckpt_restore(ctx, 0)
    assert e.value.code == P.CKPT_ENOSNAP
    with pytest.raises(P.CkptError) as e:
        P.ckpt_wait(ctx, 99, P.CKPT_WAIT_CAPTURED, None, 0, 1)
    assert e.value.code == P.CKPT_ERANGE
    P.ckpt_destroy(ctx)
    with pytest.raises(P.CkptError):
        P.ckpt_create(chunk_bytes=1000)  # not a multiple of the alignment


def test_registration_rejects_memory_the_kernels_cannot_read():
    """Only device memory of the context's GPU, inside one allocation, can be
    registered; anything else fails at registration (no kernel runs here)."""
    import ctypes as C

    def register_raw(ptr, nbytes):
        ctx = P.ckpt_create(chunk_bytes=1 << 20)
        arr = (P.ckpt_tensor * 1)()
        arr[0].dev_ptr = ptr
        arr[0].nbytes = nbytes
        rc = P.lib().ckpt_register_tensors(ctx, arr, 1)
        msg = P.ckpt_last_error(ctx)
        P.ckpt_destroy(ctx)
        return rc, msg

    host = np.zeros(1 << 16, dtype=np.uint8)  # pageable host memory
    rc, msg = register_raw(host.ctypes.data, host.size)
    assert rc == P.CKPT_EINVAL, msg
    pinned = torch.zeros(1 << 16, dtype=torch.uint8, pin_memory=True)  # host memory the GPU can reach
    rc, msg = register_raw(pinned.data_ptr(), pinned.numel())
    assert rc == P.CKPT_EINVAL and "not device memory" in msg, msg
    dev = torch.zeros(1 << 20, dtype=torch.uint8, device="cuda")
    rc, msg = register_raw(dev.data_ptr(), 1 << 40)  # far past the end of its allocation
    assert rc == P.CKPT_EINVAL and "past the end" in msg, msg
    rc, msg = register_raw(dev.data_ptr() + 4096, (1 << 20) - 4096)  # a view inside the allocation
    assert rc == P.CKPT_OK, msg
    rc, msg = register_raw(dev.data_ptr(), 1 << 20)
    assert rc == P.CKPT_OK, msg
    torch.cuda.synchronize()


def test_timing_levels():
    """ckpt_set_timing: level 1 times every pack launch; level 2 only the
    first launch and the pack stream's end (span and trigger-to-commit
    still reported, per-launch sums not), and the image is the same."""
    tensors = _step_state(n_frag=32)
    ck = P.Checkpointer(tensors, chunk_bytes=GATE_CHUNK, group_bytes=4 * GATE_CHUNK)
    host = [host_bytes(t) for t in tensors]
    want, _, _ = O.pack(host, 256, GATE_CHUNK)
    for level in (1, 2):
        P.ckpt_set_timing(ck.ctx, level)
        s = ck.snapshot(step=level)
        ck.wait_committed(s)
        t = P.ckpt_last_timing(ck.ctx, P.CKPT_OP_SNAPSHOT)
        assert t["kernels"] == t["copies"] == ck.n_chunks // 4
        assert t["span_ms"] > 0 and t["total_ms"] > t["copy_ms"] > 0
        assert np.array_equal(ck.host_image(s)[0], want)
        if level == 1:
            assert 0 < t["kernel_ms"] <= t["span_ms"]
            assert P.ckpt_last_timing(ck.ctx, P.CKPT_OP_PACK)["kernel_ms"] > 0
        else:
            assert t["kernel_ms"] == -1
            with pytest.raises(P.CkptError) as e:
                P.ckpt_last_timing(ck.ctx, P.CKPT_OP_PACK)
            assert e.value.code == P.CKPT_ESTATE
    ck.close()
