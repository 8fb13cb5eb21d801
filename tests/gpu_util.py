"""Shared helpers of the GPU tests: inputs, host copies, and the
snapshot -> oracle -> restore check used across geometries."""
import numpy as np
import torch

import oracle as O

EDGE_SIZES = [1, 2, 3, 15, 16, 17, 255, 256, 257, 0, 4095, 4096, 4097, 100_003, 0, 0, 65536, 65537, 1 << 20, 7]
# Empty fragments before the first byte and after the last one.
ENDS_EMPTY = [0, 0, 5, 4096, 0, 3 * 4096 + 1, 17, 0, 0]


def host_bytes(t):
    """The tensor's bytes as a host numpy uint8 array (through torch, outside
    the library)."""
    if t.numel() == 0:
        return np.zeros(0, dtype=np.uint8)
    return t.detach().contiguous().cpu().reshape(-1).view(torch.uint8).numpy().copy()


def random_byte_fragments(sizes, seed, device="cuda"):
    rng = np.random.default_rng(seed)
    host = [rng.integers(0, 256, s, dtype=np.uint8) for s in sizes]
    dev = [torch.from_numpy(h.copy()).to(device) for h in host]
    return dev, host


def garbage_fill(tensors, value=0x5A):
    for t in tensors:
        if t.numel():
            t.view(-1).view(torch.uint8).fill_(value) if t.dtype != torch.uint8 else t.fill_(value)


def snapshot_and_check(tensors, host, chunk, align=256, staging=0, group=0, dtypes=None, classes=None,
                       meta=b"", step=3, grid=0, bounce=0, threads=0, launch=0, direct=False):
    """Snapshot, compare image and sums with the oracle, trash the tensors,
    restore and compare them; returns the Checkpointer and snapshot id."""
    import paper_2607_01646_amd as P

    ck = P.Checkpointer(tensors, dtypes, classes, chunk_bytes=chunk, align_bytes=align,
                        device_staging_bytes=staging, group_bytes=group, grid_blocks=grid, bounce_bytes=bounce,
                        host_threads=threads, pack_launch_bytes=launch, direct=direct)
    snap = ck.snapshot(step=step, meta=meta)
    ck.wait_committed(snap)
    assert ck.state(snap) == P.CKPT_SNAP_COMMITTED
    img, sums = ck.host_image(snap)
    want, off, nc = O.pack(host, align, chunk)
    assert np.array_equal(ck.offsets, off)
    assert (ck.image_bytes, ck.n_chunks) == (want.size, nc)
    assert img.size == want.size
    diff = np.flatnonzero(img != want)
    assert diff.size == 0, "image differs at %d bytes, first at %d" % (diff.size, diff[0])
    want_sums = O.chunk_sums(want, 0, want.size, chunk)
    assert np.array_equal(sums, want_sums)
    assert ck.verify(snap) == []
    garbage_fill(tensors)
    assert ck.restore(snap) == []
    torch.cuda.synchronize()
    for i, (t, h) in enumerate(zip(tensors, host)):
        assert np.array_equal(host_bytes(t), h), "fragment %d not restored" % i
    assert np.array_equal(P.ckpt_last_sums(ck.ctx), want_sums)
    return ck, snap


def class_major(tensors, plan):
    """The same state registered class by class: parameters first, then master
    weights and the two moments, so the optimizer classes fill a run of chunks."""
    order = sorted(range(len(plan)), key=lambda i: (plan[i][3], i))
    return [tensors[i] for i in order], [plan[i][2] for i in order], [plan[i][3] for i in order]


def expected_replica(host, dtypes, classes, chunk, mask, step, meta=b""):
    """From the oracle alone: the chunk ids holding a byte of a fragment of a
    class in mask, their bytes, their sums, and the snapshot's envelope."""
    sizes = [h.size for h in host]
    img, off, nc = O.pack(host, 256, chunk)
    I = img.size
    ids = [c for c in range(nc) if any((mask >> classes[i]) & 1 for i in O.locate(c, chunk, I, off, sizes)[1])]
    data = np.concatenate([img[c * chunk:min((c + 1) * chunk, I)] for c in ids])
    sums = O.chunk_sums(img, 0, I, chunk)
    env = O.envelope(step, 256, chunk, I, off, sizes, dtypes, classes, sums, meta)
    return np.array(ids, dtype=np.uint64), data, sums[ids], env


def expected_after_restore(failed_host, before_host, ids, chunk):
    """A replacement's fragments after restoring the chunks `ids` of the
    failed rank's image (oracle pack of failed_host): the image bytes inside
    those chunks, the replacement's own bytes (before_host) elsewhere."""
    sizes = [h.size for h in failed_host]
    img, off, _ = O.pack(failed_host, 256, chunk)
    out = [b.copy() for b in before_host]
    for c in ids:
        lo, hi = int(c) * chunk, min((int(c) + 1) * chunk, img.size)
        for i, o in enumerate(off):
            a, b = max(lo, int(o)), min(hi, int(o) + sizes[i])
            if a < b:
                out[i][a - int(o):b - int(o)] = img[a:b]
    return out


def assert_located(ck, c, chunk, sizes):
    """Locate (definition 5): the library's byte range of chunk c and its
    fragment range [f0, f1] must give exactly the oracle's list -- the
    non-empty fragments inside the range are the fragments overlapping the
    chunk, no more and no fewer."""
    lo, hi, f0, f1 = ck.chunk_fragments(c)
    (olo, ohi), ids = O.locate(c, chunk, ck.image_bytes, ck.offsets, sizes)
    assert (lo, hi) == (olo, ohi), "chunk %d: byte range %s, oracle %s" % (c, (lo, hi), (olo, ohi))
    got = [i for i in range(f0, f1 + 1) if sizes[i]]
    assert got == ids, "chunk %d: fragments %s, oracle %s" % (c, got, ids)
    return ids


def window_slices(tensors, off, sizes, lo, hi):
    """Host copies of the live fragments' bytes that fall in image bytes
    [lo, hi), with their image offsets (fragment i's bytes [a, b) sit at
    image offset off[i] + a).  Copied by torch, outside the library."""
    import bisect

    offs = [int(o) for o in off]
    frags, at = [], []
    i = max(0, bisect.bisect_right(offs, lo) - 1)
    while i < len(sizes) and offs[i] < hi:
        o, s = offs[i], int(sizes[i])
        a, b = max(o, lo) - o, min(o + s, hi) - o
        if b > a:
            frags.append(tensors[i].reshape(-1).view(torch.uint8)[a:b].cpu().numpy())
            at.append(o + a)
        i += 1
    return frags, at


def check_image_against_oracle(tensors, off, sizes, img, sums, chunk, threads=16):
    """Every chunk of a committed host image, byte for byte, against the
    oracle's pack of the live fragments, and every stored sum against the
    oracle's sum of that chunk.  Streams chunk by chunk (the main thread
    copies the fragment bytes of a chunk to the host, a pool of threads runs
    the oracle and compares; the oracle's C calls release the interpreter
    lock), so it needs no second copy of a shard of tens of GB.  Returns the
    number of chunks checked."""
    import os
    from concurrent.futures import ThreadPoolExecutor

    I = img.size
    nc = (I + chunk - 1) // chunk
    assert sums.size == nc

    def check(c, frags, at):
        lo, hi = c * chunk, min((c + 1) * chunk, I)
        want = O.pack_window(frags, at, lo, hi)
        if not np.array_equal(img[lo:hi], want):
            d = np.flatnonzero(img[lo:hi] != want)
            return "chunk %d differs from the oracle at %d bytes, first at image byte %d" % (c, d.size, lo + d[0])
        s = int(O.chunk_sums(want, lo, hi, chunk)[0])
        if s != int(sums[c]):
            return "chunk %d: stored sum %#x, oracle %#x" % (c, int(sums[c]), s)
        return None

    workers = max(1, min(threads, os.cpu_count() or 1))
    pending = []
    errors = []
    with ThreadPoolExecutor(workers) as ex:
        for c in range(nc):
            lo, hi = c * chunk, min((c + 1) * chunk, I)
            frags, at = window_slices(tensors, off, sizes, lo, hi)
            pending.append(ex.submit(check, c, frags, at))
            if len(pending) >= 2 * workers:  # bound the host memory in flight
                r = pending.pop(0).result()
                if r:
                    errors.append(r)
        errors += [r for r in (f.result() for f in pending) if r]
    assert not errors, "%d chunks wrong; %s" % (len(errors), "; ".join(errors[:4]))
    return nc


def fragment_digests(tensors, piece=1 << 26):
    """Per-fragment digest computed by torch on the GPU (independent of the
    library): byte count, the sum of the fragment's 32-bit words (bytes when
    its length is not a multiple of 4) and their sum weighted by position
    (weights 1..65521, so moved or swapped words change it).  int64
    arithmetic wraps the same way every time, so equal bytes give equal
    digests."""
    out = []
    for t in tensors:
        b = t.reshape(-1).view(torch.uint8)
        n = b.numel()
        if n == 0:
            out.append((0, 0, 0))
            continue
        w = b.view(torch.int32) if n % 4 == 0 else b
        s1 = torch.zeros((), dtype=torch.int64, device=b.device)
        s2 = torch.zeros((), dtype=torch.int64, device=b.device)
        for k in range(0, w.numel(), piece):
            x = w[k:k + piece].to(torch.int64)
            pos = torch.arange(k, k + x.numel(), dtype=torch.int64, device=b.device) % 65521 + 1
            s1 += x.sum()
            s2 += (x * pos).sum()
        out.append((n, int(s1), int(s2)))
    return out


def hold(stream, ms=40.0):
    """Keep `stream` busy for about `ms` milliseconds (a chain of fp32
    matmuls); returns the result, which the caller keeps alive until the
    chain has run."""
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


def runs_beside(a, b):
    """Whether work on stream b runs while stream a is busy.  HIP maps
    streams onto a limited set of hardware queues; two streams that share
    one run in submission order, so a race test that needs two streams to
    overlap has to check that they do.  Probe: while a holds ~30 ms of
    matmuls, a marker on b must finish first."""
    import time

    torch.cuda.synchronize()
    keep = hold(a, 30.0)
    done_a = torch.cuda.Event()
    done_a.record(a)
    with torch.cuda.stream(b):
        torch.empty(1, device="cuda").fill_(1.0)
    done_b = torch.cuda.Event()
    done_b.record(b)
    t0 = time.monotonic()
    while not done_b.query() and time.monotonic() - t0 < 0.01:
        time.sleep(0.0002)
    ok = done_b.query() and not done_a.query()
    torch.cuda.synchronize()
    del keep
    return ok


def pick_stream(*others, tries=40):
    """A torch stream that runs beside every stream in `others` (probed with
    runs_beside); torch hands out streams from a pool of 32 in turn."""
    for _ in range(tries):
        c = torch.cuda.Stream()
        if all(c.cuda_stream != o.cuda_stream and runs_beside(o, c) for o in others):
            return c
    raise RuntimeError("no stream runs beside %d given streams" % len(others))
