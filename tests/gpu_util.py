"""Shared helpers of the GPU tests: inputs, host copies, and the
snapshot -> oracle -> restore check used across geometries."""
import numpy as np
import torch

import oracle as O

EDGE_SIZES = [1, 2, 3, 15, 16, 17, 255, 256, 257, 0, 4095, 4096, 4097, 100_003, 0, 0, 65536, 65537, 1 << 20, 7]


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
                       meta=b"", step=3, grid=0, bounce=0, threads=0):
    """Snapshot, compare image and sums with the oracle, trash the tensors,
    restore and compare them; returns the Checkpointer and snapshot id."""
    import paper_2607_01646_amd as P

    ck = P.Checkpointer(tensors, dtypes, classes, chunk_bytes=chunk, align_bytes=align,
                        device_staging_bytes=staging, group_bytes=group, grid_blocks=grid, bounce_bytes=bounce,
                        host_threads=threads)
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
