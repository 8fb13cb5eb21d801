"""Direct D2H (ckpt_config.direct_d2h) against the CPU oracle, bit for bit
(needs an MI355X).

In this mode nothing is staged on the device: the DMA engines copy every
fragment piece from the live tensors straight into the host image (pinned,
or through the bounce ring), the padding is zeroed on the host, the kernel
only computes the chunk sums, and the gate waits for the copies.  Images,
sums, restored tensors and bad lists are compared with values from `oracle`
alone; inputs come from numpy and torch generators.
"""
import numpy as np
import pytest
import torch

import oracle as O
from gpu_util import (EDGE_SIZES, ENDS_EMPTY, assert_located, garbage_fill, hold, host_bytes, pick_stream,
                      random_byte_fragments, snapshot_and_check)

pytestmark = pytest.mark.gpu

if torch.cuda.is_available():
    import paper_2607_01646_amd as P


@pytest.mark.parametrize("chunk,align,group,bounce", [
    (4096, 256, 0, 0),                    # one group over every chunk
    (4096, 256, 4096, 0),                 # one-chunk groups: fragments cut at many group boundaries
    (4096, 16, 3 * 4096, 0),              # 16-byte alignment, three-chunk groups
    (768, 256, 768, 0),                   # chunk not a power of two
    (1 << 20, 256, 1 << 20, 0),           # chunks larger than most fragments
    (1 << 16, 4096, 1 << 16, 0),          # 4 KiB alignment: padding runs of up to 4095 bytes
    (4096, 256, 4096, 4 * 4096),          # pageable images behind a ring of four groups
    (8192, 16, 2 * 8192, 2 * 2 * 8192),   # ... and of two groups of two chunks
])
def test_edge_sizes(chunk, align, group, bounce):
    tensors, host = random_byte_fragments(EDGE_SIZES, seed=chunk + align + group + bounce)
    ck, _ = snapshot_and_check(tensors, host, chunk, align, group=group, bounce=bounce, direct=True)
    ck.close()


@pytest.mark.parametrize("bounce", [0, 2 * 4096])
def test_empty_fragments_at_both_ends(bounce):
    """Empty fragments first and last: no piece and no padding run for them,
    and the copies end on the last non-empty fragment's padding."""
    tensors, host = random_byte_fragments(ENDS_EMPTY, seed=43 + bounce)
    ck, _ = snapshot_and_check(tensors, host, 4096, 256, group=4096, bounce=bounce, direct=True)
    ck.close()


def test_capped_grid_strides_over_tiles():
    """With the workgroup count capped, the sums kernel's workgroups loop
    over many tiles (the per-tile path instead of the two-tile runs)."""
    tensors, host = random_byte_fragments(EDGE_SIZES, seed=55)
    for grid in [1, 7, 64]:
        ck, _ = snapshot_and_check(tensors, host, 1 << 16, group=1 << 16, grid=grid, direct=True)
        ck.close()


def test_many_small_fragments_in_one_tile():
    """32 fragments per 8 KiB tile (the multi-fragment sums path with its LDS
    search), then more fragments in one tile than the LDS offset cache holds
    (the search in global memory)."""
    rng = np.random.default_rng(31)
    sizes = [int(s) for s in rng.integers(1, 41, 600)]
    tensors, host = random_byte_fragments(sizes, seed=32)
    ck, _ = snapshot_and_check(tensors, host, 1 << 20, direct=True)
    ck.close()
    sizes = [0] * 3000 + [5, 0, 9] + [0] * 1500 + [300]
    tensors, host = random_byte_fragments(sizes, seed=33)
    ck, _ = snapshot_and_check(tensors, host, 1 << 16, direct=True)
    ck.close()


def test_dense_tiny_fragments_at_odd_offsets():
    """20,000 fragments of 1..1199 bytes at arbitrary byte offsets in one
    buffer, 16-byte alignment: nearly every tile holds several misaligned
    fragments, so the sums kernel's general path carries the image and the
    engines copy 20,000 small pieces.  The restore writes every fragment
    back and leaves the bytes between them untouched."""
    rng = np.random.default_rng(4343)
    n = 20_000
    sizes = rng.integers(1, 1200, n)
    gaps = rng.integers(0, 64, n)
    offs = np.cumsum(gaps + np.concatenate(([0], sizes[:-1])))
    total = int(offs[-1] + sizes[-1] + 64)
    host_all = rng.integers(0, 256, total, dtype=np.uint8)
    dev_all = torch.from_numpy(host_all.copy()).cuda()
    frags = [dev_all[int(o):int(o) + int(z)] for o, z in zip(offs, sizes)]
    host = [host_all[int(o):int(o) + int(z)] for o, z in zip(offs, sizes)]
    chunk = 1 << 20
    ck = P.Checkpointer(frags, chunk_bytes=chunk, align_bytes=16, group_bytes=2 * chunk, direct=True)
    snap = ck.snapshot(step=1)
    ck.wait_committed(snap)
    img, sums = ck.host_image(snap)
    want, off, nc = O.pack(host, 16, chunk)
    assert np.array_equal(ck.offsets, off) and img.size == want.size
    diff = np.flatnonzero(img != want)
    assert diff.size == 0, "image differs at %d bytes, first at %d" % (diff.size, diff[0])
    assert np.array_equal(sums, O.chunk_sums(want, 0, want.size, chunk))
    dev_all.fill_(0x5A)
    assert ck.restore(snap) == []
    torch.cuda.synchronize()
    got = dev_all.cpu().numpy()
    marks = np.zeros(total + 1, dtype=np.int64)
    np.add.at(marks, offs, 1)
    np.add.at(marks, offs + sizes, -1)
    in_frag = np.cumsum(marks[:-1]) > 0
    assert np.array_equal(got[in_frag], host_all[in_frag]), "a fragment byte was not restored"
    assert np.all(got[~in_frag] == 0x5A), "the restore wrote outside the fragments"
    ck.close()


@pytest.mark.parametrize("bounce", [0, 4 * 8192])
def test_misaligned_views_and_bit_patterns(bounce):
    """Views at odd byte offsets of one buffer, with NaN payloads, -0,
    subnormals and all-ones words: the engines copy any alignment, the sums
    kernel funnel-shifts, and the restore leaves the bytes between the views
    untouched."""
    rng = np.random.default_rng(77)
    raw = rng.integers(0, 256, 1 << 20, dtype=np.uint8)
    special = np.array([0x7FC00001, 0x80000000, 0x00000001, 0xFFFFFFFF, 0x7F800000], dtype=np.uint32)
    raw[:special.nbytes] = special.view(np.uint8)
    buf = torch.from_numpy(raw.copy()).cuda()
    cuts = [(0, 20), (21, 4093), (4120, 1), (4123, 65539), (70001, 300000), (370003, 17), (370030, 600000)]
    views = [buf[a:a + n] for a, n in cuts]
    host = [raw[a:a + n].copy() for a, n in cuts]
    ck, snap = snapshot_and_check(views, host, 8192, 256, group=8192, bounce=bounce, direct=True)
    torch.cuda.synchronize()
    got = buf.cpu().numpy()
    assert np.array_equal(got, raw), "the restore wrote outside the views"
    ck.close()


@pytest.mark.parametrize("bounce", [0, 1 << 20])
def test_repeated_snapshots_alternate_images(bounce):
    """Five snapshots, each after every fragment changed: each commits into
    the other image and equals the oracle's pack of the bytes at its trigger;
    the older snapshot stays restorable."""
    tensors, host = random_byte_fragments(EDGE_SIZES * 3, seed=5)
    chunk = 1 << 16
    ck = P.Checkpointer(tensors, chunk_bytes=chunk, group_bytes=2 * chunk, bounce_bytes=bounce, direct=True)
    prev = None
    for k in range(5):
        for t in tensors:
            if t.numel():
                t.add_(k + 1)
        torch.cuda.synchronize()
        now = [host_bytes(t) for t in tensors]
        s = ck.snapshot(step=k)
        ck.wait_committed(s)
        img, sums = ck.host_image(s)
        want, _, _ = O.pack(now, 256, chunk)
        assert np.array_equal(img, want), "snapshot %d" % k
        assert np.array_equal(sums, O.chunk_sums(want, 0, want.size, chunk))
        if prev is not None:
            assert ck.state(prev[0]) == P.CKPT_SNAP_COMMITTED
        prev = (s, now)
    garbage_fill(tensors)
    assert ck.restore(prev[0]) == []
    torch.cuda.synchronize()
    for t, h in zip(tensors, prev[1]):
        assert np.array_equal(host_bytes(t), h)
    ck.close()


@pytest.mark.parametrize("bounce", [0, 1 << 20])
def test_padding_is_rewritten(bounce):
    """The engines never write the padding between fragments; the library
    zeroes it on the host before each group's copies.  Bytes planted in the
    padding of a committed image are gone when a later snapshot reuses that
    image."""
    tensors, host = random_byte_fragments([1, 300, 17, 4097, 255, 100_003], seed=9)
    chunk = 4096
    ck = P.Checkpointer(tensors, chunk_bytes=chunk, group_bytes=chunk, bounce_bytes=bounce, direct=True)
    s1 = ck.snapshot(step=1)
    ck.wait_committed(s1)
    img, _ = ck.host_image(s1)
    off = [int(o) for o in ck.offsets]
    ends = [o + h.size for o, h in zip(off, host)]
    starts = off[1:] + [ck.image_bytes]
    pad = [(e, s) for e, s in zip(ends, starts) if s > e]
    assert pad, "no padding to plant in"
    for e, s in pad:
        img[e:s] = 0xA7
    s2 = ck.snapshot(step=2)
    ck.wait_committed(s2)
    s3 = ck.snapshot(step=3)  # back into s1's image
    ck.wait_committed(s3)
    img3, sums3 = ck.host_image(s3)
    want, _, _ = O.pack(host, 256, chunk)
    assert np.array_equal(img3, want)
    assert np.array_equal(sums3, O.chunk_sums(want, 0, want.size, chunk))
    ck.close()


def _state(n_frag=96, numel=1 << 20, seed=43):
    g = torch.Generator(device="cuda").manual_seed(seed)
    return [torch.randn(numel, generator=g, device="cuda") for _ in range(n_frag)]


CHUNK = 1 << 20


@pytest.mark.parametrize("bounce", [0, 16 << 20])
def test_gate_orders_update_after_the_copies(bounce):
    """The update of every fragment, on another stream right after
    ckpt_wait(CAPTURED) on the whole range, waits for the engines: the image
    holds the bytes of the trigger, although the trigger sits behind ~40 ms
    of work and the update would otherwise run first."""
    tensors = _state()
    ck = P.Checkpointer(tensors, chunk_bytes=CHUNK, group_bytes=CHUNK, bounce_bytes=bounce, direct=True)
    main, side = torch.cuda.current_stream(), torch.cuda.Stream()
    torch.cuda.synchronize()
    before = [host_bytes(t) for t in tensors]
    keep = hold(main)
    s = ck.snapshot(step=1, stream=main)
    ck.wait_captured(s, 0, len(tensors), stream=side)
    with torch.cuda.stream(side):
        for t in tensors:
            t.add_(1.0)
    ck.wait_committed(s)
    img, sums = ck.host_image(s)
    want, _, _ = O.pack(before, 256, CHUNK)
    assert np.array_equal(img, want)
    assert np.array_equal(sums, O.chunk_sums(want, 0, want.size, CHUNK))
    torch.cuda.synchronize()
    del keep
    ck.close()


def test_gate_negative_control_detects_the_race():
    """Same without the wait: the update runs while the snapshot still waits
    for its trigger, and the image holds updated values.  Shows the gate test
    can see a missing wait."""
    tensors = _state()
    main = torch.cuda.current_stream()
    pk = pick_stream(main)
    side = pick_stream(main, pk)
    ck = P.Checkpointer(tensors, chunk_bytes=CHUNK, group_bytes=CHUNK, direct=True, side_stream=pk)
    torch.cuda.synchronize()
    before = [host_bytes(t) for t in tensors]
    keep = hold(main)
    s = ck.snapshot(step=1, stream=main)
    with torch.cuda.stream(side):
        for t in tensors:
            t.add_(1.0)
    ck.wait_committed(s)
    img, _ = ck.host_image(s)
    want, _, _ = O.pack(before, 256, CHUNK)
    assert not np.array_equal(img, want)
    torch.cuda.synchronize()
    del keep
    ck.close()


def test_gate_covers_only_its_range():
    """One-chunk groups copied in order over ~7 ms of host link: a wait on
    fragments [0, 8) (copied first) does not cover the last eight fragments,
    so updating those right after it reaches the image; after a wait on
    their own range it does not.  The chunks before them hold the trigger's
    bytes either way."""
    tensors = _state()
    pk = pick_stream(torch.cuda.current_stream())
    side = pick_stream(pk)
    ck = P.Checkpointer(tensors, chunk_bytes=CHUNK, group_bytes=CHUNK, direct=True, side_stream=pk)
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
        o = int(off[n - 8])
        want, _, _ = O.pack(before, 256, CHUNK)
        assert np.array_equal(img[:o], want[:o])
    ck.close()


@pytest.mark.parametrize("bounce", [0, 16 << 20])
def test_trigger_captures_writes_queued_before_it(bounce):
    """An in-place update of every fragment queued on the training stream
    behind ~40 ms of work, before the snapshot call: the engines copy the
    updated bytes (they start only after the trigger)."""
    tensors = _state()
    ck = P.Checkpointer(tensors, chunk_bytes=CHUNK, group_bytes=CHUNK, bounce_bytes=bounce, direct=True)
    main = torch.cuda.current_stream()
    torch.cuda.synchronize()
    keep = hold(main)
    for t in tensors:
        t.add_(1.0)
    updated = torch.cuda.Event()
    updated.record(main)
    s = ck.snapshot(step=1, stream=main)
    assert not updated.query(), "the update ran before the snapshot call returned; the test proves nothing"
    ck.wait_committed(s)
    torch.cuda.synchronize()
    after = [host_bytes(t) for t in tensors]
    img, sums = ck.host_image(s)
    want, _, _ = O.pack(after, 256, CHUNK)
    assert np.array_equal(img, want)
    assert np.array_equal(sums, O.chunk_sums(want, 0, want.size, CHUNK))
    del keep
    ck.close()


@pytest.mark.parametrize("bounce", [0, 1 << 20])
def test_interrupted_snapshot_gate_and_restore(bounce):
    """An offload cut after two groups stays ABORTED; a gate on its whole
    range returns (the groups never copied wait only for their sums), the
    previous snapshot restores, and the next snapshot, into the cut one's
    image, equals the oracle."""
    tensors = _state(n_frag=16, numel=1 << 18)
    chunk = 1 << 18
    ck = P.Checkpointer(tensors, chunk_bytes=chunk, group_bytes=chunk, bounce_bytes=bounce, direct=True)
    s1 = ck.snapshot(step=1)
    ck.wait_committed(s1)
    good = [host_bytes(t) for t in tensors]
    for t in tensors:
        t.add_(3.0)
    P.ckpt_debug_interrupt_next(ck.ctx, 2)
    s2 = ck.snapshot(step=2)
    side = torch.cuda.Stream()
    ck.wait_captured(s2, 0, len(tensors), stream=side)
    with torch.cuda.stream(side):
        for t in tensors:
            t.add_(1.0)
    torch.cuda.synchronize()
    assert ck.state(s2) == P.CKPT_SNAP_ABORTED
    with pytest.raises(P.CkptError) as e:
        ck.wait_committed(s2)
    assert e.value.code == P.CKPT_ESTATE
    now = [host_bytes(t) for t in tensors]
    garbage_fill(tensors)
    assert ck.restore(0) == []
    torch.cuda.synchronize()
    for t, h in zip(tensors, good):
        assert np.array_equal(host_bytes(t), h)
    for t, h in zip(tensors, now):
        t.view(torch.uint8).copy_(torch.from_numpy(h).cuda())
    s3 = ck.snapshot(step=3)
    ck.wait_committed(s3)
    img, sums = ck.host_image(s3)
    want, _, _ = O.pack(now, 256, chunk)
    assert np.array_equal(img, want)
    assert np.array_equal(sums, O.chunk_sums(want, 0, want.size, chunk))
    assert ck.restore(s1) == []
    ck.close()


def test_flips_are_reported_and_located():
    """Single-bit flips in a committed image (one per chunk, in three
    chunks): restore through the direct mode's device ring reports exactly
    those chunks, the recomputed sums differ by the closed-form +-2^b, and
    each is located to the oracle's fragments."""
    tensors, host = random_byte_fragments(EDGE_SIZES * 2, seed=12)
    chunk = 4096
    sizes = [h.size for h in host]
    ck = P.Checkpointer(tensors, chunk_bytes=chunk, group_bytes=chunk, direct=True)
    s = ck.snapshot(step=1)
    ck.wait_committed(s)
    img, sums = ck.host_image(s)
    stored = sums.copy()
    rng = np.random.default_rng(3)
    picks = sorted(rng.choice(ck.n_chunks, 3, replace=False).tolist())
    delta = {}
    for c in picks:
        lo = c * chunk
        n_words = (min(lo + chunk, ck.image_bytes) - lo) // 8
        w = int(rng.integers(0, n_words))
        b = int(rng.integers(0, 64))
        word = int(np.frombuffer(img[lo + 8 * w:lo + 8 * w + 8].tobytes(), "<u8")[0])
        delta[c] = ((1 << b) if not (word >> b) & 1 else -(1 << b)) % (1 << 64)
        img[lo + 8 * w + b // 8] ^= np.uint8(1 << (b % 8))
    assert ck.verify(s) == picks
    garbage_fill(tensors)
    assert ck.restore(s) == picks
    recomputed = P.ckpt_last_sums(ck.ctx)
    for c in picks:
        assert (int(recomputed[c]) - int(stored[c])) % (1 << 64) == delta[c]
        assert_located(ck, c, chunk, sizes)
    ck.close()


def test_timing_counts_the_sums_bytes():
    tensors, host = random_byte_fragments([1 << 20, 3 << 20, 12345], seed=2)
    ck = P.Checkpointer(tensors, chunk_bytes=1 << 20, group_bytes=1 << 20, direct=True)
    P.ckpt_set_timing(ck.ctx, True)
    s = ck.snapshot(step=1)
    ck.wait_committed(s)
    t = P.ckpt_last_timing(ck.ctx, P.CKPT_OP_SNAPSHOT)
    assert t["kernel_bytes"] == sum(h.size for h in host)
    assert t["kernels"] == ck.n_chunks and t["copies"] == ck.n_chunks
    assert t["kernel_ms"] > 0 and t["copy_ms"] > 0 and t["total_ms"] > 0
    ck.close()


def test_configuration_errors():
    t = [torch.zeros(1024, device="cuda")]
    for kw in ({"device_staging_bytes": 8 << 20}, {"poison": True}):
        with pytest.raises(P.CkptError) as e:
            P.Checkpointer(t, chunk_bytes=1 << 20, direct=True, **kw)
        assert e.value.code == P.CKPT_EINVAL
    # more than 65536 fragment pieces
    buf = torch.zeros(70_000 * 2, dtype=torch.uint8, device="cuda")
    views = [buf[2 * i:2 * i + 1] for i in range(70_000)]
    with pytest.raises(P.CkptError) as e:
        P.Checkpointer(views, chunk_bytes=1 << 20, align_bytes=16, direct=True)
    assert e.value.code == P.CKPT_EINVAL
