"""Python binding of libckpt (include/ckpt.h): argument marshalling only.

Every step of the snapshot path -- pack and chunk sums, the D2H pipeline,
the gate before the optimizer step, restore and verify -- runs in the
library's HIP kernels and DMA queues; this module converts torch tensors and
streams to pointers and handles and turns status codes into exceptions.
The functions keep the C names; `Checkpointer` bundles them for a training
loop (paper Sec. V-B D2H phase, Sec. VI-A ping-pong buffers and the single
wait before the optimizer step).
"""
import ctypes as C
import os

import numpy as np
import torch  # loaded before libckpt so that both use torch's HIP runtime

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libckpt.so")

CKPT_OK = 0
CKPT_EINVAL = -1
CKPT_ESTATE = -2
CKPT_ENOMEM = -3
CKPT_EHIP = -4
CKPT_ECORRUPT = -5
CKPT_ENOSNAP = -6
CKPT_EBUSY = -7
CKPT_ERANGE = -8
CKPT_WAIT_CAPTURED = 0
CKPT_WAIT_COMMITTED = 1
CKPT_WAIT_REPLICATED = 2
REPLICA_PENDING, REPLICA_OK, REPLICA_CORRUPT, REPLICA_FAILED = 0, 1, 2, 3
CKPT_FILE_CREATE = 0
CKPT_FILE_ADOPT = 1
CKPT_SNAP_IN_FLIGHT = 0
CKPT_SNAP_COMMITTED = 1
CKPT_SNAP_ABORTED = 2
CKPT_SNAP_SUPERSEDED = 3
CKPT_OP_SNAPSHOT = 0
CKPT_OP_RESTORE = 1
CKPT_OP_VERIFY = 2
CKPT_OP_PACK = 3
CKPT_CANARY = bytes([0xDE, 0xAD, 0xC0, 0xDE, 0x5A, 0x5A, 0xA5, 0xA5]) + b"CKPTPOIS"

_NAMES = {v: k for k, v in dict(globals()).items() if k.startswith("CKPT_E")}


class ckpt_config(C.Structure):
    _fields_ = [("chunk_bytes", C.c_uint64), ("align_bytes", C.c_uint32), ("host_buffers", C.c_uint32),
                ("device_staging_bytes", C.c_uint64), ("group_bytes", C.c_uint64), ("device", C.c_int32),
                ("grid_blocks", C.c_uint32), ("bounce_bytes", C.c_uint64), ("host_threads", C.c_uint32),
                ("side_stream", C.c_void_p), ("pack_launch_bytes", C.c_uint64), ("d2h_engines", C.c_uint32),
                ("poison", C.c_uint32), ("direct_d2h", C.c_uint32)]


class ckpt_tensor(C.Structure):
    _fields_ = [("dev_ptr", C.c_void_p), ("nbytes", C.c_uint64), ("dtype", C.c_uint32), ("cls", C.c_uint32)]


class ckpt_timing(C.Structure):
    _fields_ = [("kernel_ms", C.c_float), ("kernels", C.c_uint32), ("copies", C.c_uint32), ("copy_ms", C.c_float),
                ("total_ms", C.c_float), ("kernel_bytes", C.c_uint64), ("copy_bytes", C.c_uint64),
                ("span_ms", C.c_float)]


class CkptError(RuntimeError):
    def __init__(self, code, msg):
        super().__init__("%s (%d): %s" % (_NAMES.get(code, "CKPT_E?"), code, msg))
        self.code = code


_lib = None


def lib():
    """The loaded libckpt.  Raises if it has not been built: there is no
    fallback implementation."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError("libckpt.so is not built; run `python -c 'import __graft_entry__ as g; g.build()'`")
        L = C.CDLL(LIB_PATH)
        vp, u64, u32, i32 = C.c_void_p, C.c_uint64, C.c_uint32, C.c_int32
        P = C.POINTER
        sig = {
            "ckpt_create": ([P(ckpt_config), P(vp)], i32),
            "ckpt_destroy": ([vp], i32),
            "ckpt_register_tensors": ([vp, P(ckpt_tensor), u32], i32),
            "ckpt_snapshot_async": ([vp, vp, u64, vp, u32, P(u64)], i32),
            "ckpt_wait": ([vp, u64, u32, vp, u32, u32], i32),
            "ckpt_snapshot_state": ([vp, u64, P(u32)], i32),
            "ckpt_restore": ([vp, u64, vp, P(u32), u32, P(u32)], i32),
            "ckpt_verify": ([vp, u64, P(u32), u32, P(u32)], i32),
            "ckpt_layout": ([vp, P(u64), P(u64), P(u64)], i32),
            "ckpt_chunk_fragments": ([vp, u64, P(u64), P(u64), P(u32), P(u32)], i32),
            "ckpt_host_image": ([vp, u64, P(vp), P(u64), P(P(u64))], i32),
            "ckpt_last_sums": ([vp, P(u64), u64], i32),
            "ckpt_envelope": ([vp, u64, vp, u64, P(u64)], i32),
            "ckpt_debug_interrupt_next": ([vp, i32], i32),
            "ckpt_set_timing": ([vp, i32], i32),
            "ckpt_last_timing": ([vp, u32, P(ckpt_timing)], i32),
            "ckpt_plan": ([P(u64), u32, u64, u32, P(u64), P(u64), P(u64)], i32),
            "ckpt_debug_tile_plan": ([P(u64), u32, u64, u32, P(u64), P(u64), P(u32), P(u32)], i32),
            "ckpt_debug_direct_plan": ([P(u64), u32, u64, u32, u64, P(u64), P(u64), P(u64), P(u64), P(u64)], i32),
            "ckpt_last_error": ([vp], C.c_char_p),
            "ckpt_image_file": ([vp, C.c_char_p, u32], i32),
            "ckpt_latest": ([vp, P(u64), P(u64)], i32),
            "ckpt_replicate_to": ([vp, C.c_char_p, u32, u64], i32),
            "ckpt_replica_chunks": ([vp, P(u64), u64, P(u64), P(u64)], i32),
            "ckpt_replica_result": ([vp, u64, P(i32), P(u64), u32, P(u32)], i32),
            "ckpt_replica_timing": ([vp, P(C.c_double), P(C.c_double)], i32),
            "ckpt_debug_h2h_fault": ([vp, i32, u64, u64], i32),
            "ckpt_debug_h2h_fault_peer": ([vp, u32, i32, u64, u64], i32),
            "ckpt_replica_peer_result": ([vp, u32, u64, P(i32), P(u64), u32, P(u32)], i32),
            "ckpt_replica_peers": ([vp, P(u32)], i32),
            "ckpt_replicate_remove": ([vp, u32], i32),
            "ckpt_peer_create": ([P(ckpt_config), u32, P(vp)], i32),
            "ckpt_peer_port": ([vp, P(u32)], i32),
            "ckpt_peer_destroy": ([vp], i32),
            "ckpt_peer_wait": ([vp, u64, i32, P(i32)], i32),
            "ckpt_peer_replica": ([vp, P(u64), P(u64), P(vp), P(u64), P(P(u64)), P(P(u64)), P(u64), P(vp), P(u64)],
                                  i32),
            "ckpt_peer_last_bad": ([vp, P(u64), u32, P(u32)], i32),
            "ckpt_peer_timing": ([vp, P(C.c_double), P(C.c_double)], i32),
            "ckpt_peer_last_error": ([vp], C.c_char_p),
            "ckpt_restore_from_peer": ([vp, C.c_char_p, u32, vp, P(u64), P(u64), P(u32), u32, P(u32)], i32),
            "ckpt_peer_restore_info": ([vp, P(u64), u64, P(u64), vp, u64, P(u64), P(C.c_double), P(C.c_double)],
                                       i32),
            "ckpt_pack_noalloc": ([P(ckpt_tensor), u32, u64, u32, i32, vp, u64, vp, u64, vp, P(u64), P(u64)], i32),
        }
        for name, (args, res) in sig.items():
            f = getattr(L, name)
            f.argtypes = args
            f.restype = res
        _lib = L
    return _lib


def _check(ctx, rc):
    if rc != CKPT_OK:
        raise CkptError(rc, (lib().ckpt_last_error(ctx) or b"").decode())
    return rc


def _stream(s):
    """hipStream_t handle of a torch stream, an int handle, or (None) torch's
    current stream."""
    if s is None:
        s = torch.cuda.current_stream()
    if isinstance(s, int):
        return C.c_void_p(s)
    return C.c_void_p(s.cuda_stream)


def _u64p(a):
    return a.ctypes.data_as(C.POINTER(C.c_uint64))


def _u32p(a):
    return a.ctypes.data_as(C.POINTER(C.c_uint32))


def ckpt_create(chunk_bytes=0, align_bytes=0, device_staging_bytes=0, group_bytes=0, device=None, grid_blocks=0,
                bounce_bytes=0, host_threads=0, side_stream=None, pack_launch_bytes=0, d2h_engines=0, poison=False,
                direct=False):
    """side_stream: a torch stream (or raw handle) for the pack kernels; None =
    the library's own.  The caller keeps it alive while the context lives.
    direct: ckpt_config.direct_d2h."""
    if device is None:
        device = torch.cuda.current_device()
    cfg = ckpt_config(chunk_bytes, align_bytes, 0, device_staging_bytes, group_bytes, device, grid_blocks,
                      bounce_bytes, host_threads, _stream(side_stream).value if side_stream is not None else None,
                      pack_launch_bytes, d2h_engines, 1 if poison else 0, 1 if direct else 0)
    ctx = C.c_void_p()
    rc = lib().ckpt_create(C.byref(cfg), C.byref(ctx))
    if rc != CKPT_OK:
        raise CkptError(rc, "ckpt_create rejected the configuration")
    return ctx


def ckpt_destroy(ctx):
    return _check(ctx, lib().ckpt_destroy(ctx))


def tensor_bytes(t):
    if not t.is_contiguous():
        raise ValueError("fragment tensors must be contiguous (got strides %s)" % (t.stride(),))
    return t.numel() * t.element_size()


def ckpt_register_tensors(ctx, tensors, dtypes=None, classes=None):
    n = len(tensors)
    arr = (ckpt_tensor * n)()
    for i, t in enumerate(tensors):
        if not t.is_cuda:
            raise ValueError("fragment %d is not a device tensor" % i)
        nb = tensor_bytes(t)
        arr[i].dev_ptr = t.data_ptr() if nb else None
        arr[i].nbytes = nb
        arr[i].dtype = dtypes[i] if dtypes is not None else 0
        arr[i].cls = classes[i] if classes is not None else 0
    return _check(ctx, lib().ckpt_register_tensors(ctx, arr, n))


def ckpt_snapshot_async(ctx, after_stream=None, step=0, meta=b""):
    sid = C.c_uint64()
    meta = bytes(meta)
    buf = C.create_string_buffer(meta, len(meta)) if meta else None
    _check(ctx, lib().ckpt_snapshot_async(ctx, _stream(after_stream), step, buf, len(meta), C.byref(sid)))
    return sid.value


def ckpt_wait(ctx, snap_id, mode=CKPT_WAIT_CAPTURED, stream=None, frag_lo=0, frag_hi=None, n_frags=None):
    if frag_hi is None:
        frag_hi = n_frags if n_frags is not None else 0xFFFFFFFF
    if mode == CKPT_WAIT_COMMITTED:
        frag_lo, frag_hi = 0, 0
    return _check(ctx, lib().ckpt_wait(ctx, snap_id, mode, _stream(stream), frag_lo, frag_hi))


def ckpt_snapshot_state(ctx, snap_id):
    st = C.c_uint32()
    _check(ctx, lib().ckpt_snapshot_state(ctx, snap_id, C.byref(st)))
    return st.value


def _bad_list_call(ctx, fn, n_chunks):
    cap = max(int(n_chunks), 1)
    bad = np.zeros(cap, dtype=np.uint32)
    nb = C.c_uint32()
    rc = fn(_u32p(bad), cap, C.byref(nb))
    if rc not in (CKPT_OK, CKPT_ECORRUPT):
        _check(ctx, rc)
    return [int(x) for x in bad[:min(nb.value, cap)]]


def ckpt_restore(ctx, snap_id=0, stream=None):
    """Returns the list of chunks whose sum failed ([] = every chunk verified)."""
    _, _, nc = ckpt_layout(ctx, offsets=False)
    s = _stream(stream)
    return _bad_list_call(ctx, lambda b, cap, n: lib().ckpt_restore(ctx, snap_id, s, b, cap, n), nc)


def ckpt_verify(ctx, snap_id=0):
    _, _, nc = ckpt_layout(ctx, offsets=False)
    return _bad_list_call(ctx, lambda b, cap, n: lib().ckpt_verify(ctx, snap_id, b, cap, n), nc)


def ckpt_layout(ctx, n_frags=None, offsets=True):
    I = C.c_uint64()
    nc = C.c_uint64()
    off = None
    if offsets:
        if n_frags is None:
            raise ValueError("n_frags needed for offsets")
        off = np.zeros(max(n_frags, 1), dtype=np.uint64)
        _check(ctx, lib().ckpt_layout(ctx, _u64p(off), C.byref(I), C.byref(nc)))
        off = off[:n_frags]
    else:
        _check(ctx, lib().ckpt_layout(ctx, None, C.byref(I), C.byref(nc)))
    return off, I.value, nc.value


def ckpt_chunk_fragments(ctx, c):
    lo, hi = C.c_uint64(), C.c_uint64()
    f0, f1 = C.c_uint32(), C.c_uint32()
    _check(ctx, lib().ckpt_chunk_fragments(ctx, c, C.byref(lo), C.byref(hi), C.byref(f0), C.byref(f1)))
    return lo.value, hi.value, f0.value, f1.value


def ckpt_host_image(ctx, snap_id):
    """(image, sums): numpy views of the snapshot's pinned host image and its
    stored chunk sums.  Borrowed: valid until the image is reused."""
    img = C.c_void_p()
    nbytes = C.c_uint64()
    sums = C.POINTER(C.c_uint64)()
    _check(ctx, lib().ckpt_host_image(ctx, snap_id, C.byref(img), C.byref(nbytes), C.byref(sums)))
    _, _, nc = ckpt_layout(ctx, offsets=False)
    image = np.ctypeslib.as_array(C.cast(img, C.POINTER(C.c_uint8)), shape=(nbytes.value,))
    s = np.ctypeslib.as_array(sums, shape=(nc,))
    return image, s


def ckpt_last_sums(ctx):
    _, _, nc = ckpt_layout(ctx, offsets=False)
    out = np.zeros(nc, dtype=np.uint64)
    _check(ctx, lib().ckpt_last_sums(ctx, _u64p(out), nc))
    return out


def ckpt_envelope(ctx, snap_id):
    n = C.c_uint64()
    rc = lib().ckpt_envelope(ctx, snap_id, None, 0, C.byref(n))
    if rc not in (CKPT_OK, CKPT_EINVAL) or n.value == 0:
        _check(ctx, rc)
    buf = C.create_string_buffer(n.value)
    _check(ctx, lib().ckpt_envelope(ctx, snap_id, buf, n.value, C.byref(n)))
    return buf.raw[:n.value]


def ckpt_debug_interrupt_next(ctx, groups):
    return _check(ctx, lib().ckpt_debug_interrupt_next(ctx, groups))


def ckpt_set_timing(ctx, enable=True):
    """enable: False/0 off, True/1 events around every launch and copy, 2 a
    snapshot's first pack launch and pack-stream end only."""
    level = 2 if enable == 2 and not isinstance(enable, bool) else (1 if enable else 0)
    return _check(ctx, lib().ckpt_set_timing(ctx, level))


def ckpt_last_timing(ctx, which=CKPT_OP_SNAPSHOT):
    t = ckpt_timing()
    _check(ctx, lib().ckpt_last_timing(ctx, which, C.byref(t)))
    return {k: getattr(t, k) for k, _ in ckpt_timing._fields_}


def ckpt_plan(nbytes, chunk_bytes=0, align_bytes=0):
    nb = np.ascontiguousarray(np.asarray(nbytes, dtype=np.uint64))
    off = np.zeros(max(nb.size, 1), dtype=np.uint64)
    I = C.c_uint64()
    nc = C.c_uint64()
    _check(None, lib().ckpt_plan(_u64p(nb), nb.size, chunk_bytes, align_bytes, _u64p(off), C.byref(I),
                                 C.byref(nc)))
    return off[:nb.size], I.value, nc.value


def ckpt_debug_tile_plan(nbytes, chunk_bytes=0, align_bytes=0):
    nb = np.ascontiguousarray(np.asarray(nbytes, dtype=np.uint64))
    tb = C.c_uint64()
    nt = C.c_uint64()
    _check(None, lib().ckpt_debug_tile_plan(_u64p(nb), nb.size, chunk_bytes, align_bytes, C.byref(tb),
                                            C.byref(nt), None, None))
    tf = np.zeros(nt.value, dtype=np.uint32)
    tl = np.zeros(nt.value, dtype=np.uint32)
    _check(None, lib().ckpt_debug_tile_plan(_u64p(nb), nb.size, chunk_bytes, align_bytes, C.byref(tb),
                                            C.byref(nt), _u32p(tf), _u32p(tl)))
    return tb.value, tf, tl


def ckpt_debug_direct_plan(nbytes, chunk_bytes=0, align_bytes=0, group_bytes=0):
    """The direct D2H copy plan: (pieces [k, 4]: fragment, offset in it, image
    offset, bytes; gaps [k, 2]: image offset, bytes; piece_first; gap_first)."""
    nb = np.ascontiguousarray(np.asarray(nbytes, dtype=np.uint64))
    counts = np.zeros(3, dtype=np.uint64)
    _check(None, lib().ckpt_debug_direct_plan(_u64p(nb), nb.size, chunk_bytes, align_bytes, group_bytes,
                                              _u64p(counts), None, None, None, None))
    ng, npc, ngp = (int(x) for x in counts)
    pieces = np.zeros((max(npc, 1), 4), dtype=np.uint64)
    gaps = np.zeros((max(ngp, 1), 2), dtype=np.uint64)
    pf = np.zeros(ng + 1, dtype=np.uint64)
    gf = np.zeros(ng + 1, dtype=np.uint64)
    _check(None, lib().ckpt_debug_direct_plan(_u64p(nb), nb.size, chunk_bytes, align_bytes, group_bytes,
                                              _u64p(counts), _u64p(pieces), _u64p(gaps), _u64p(pf), _u64p(gf)))
    return pieces[:npc], gaps[:ngp], pf, gf


def ckpt_last_error(ctx):
    return (lib().ckpt_last_error(ctx) or b"").decode()


def ckpt_image_file(ctx, path, mode=CKPT_FILE_CREATE):
    return _check(ctx, lib().ckpt_image_file(ctx, path.encode(), mode))


def ckpt_latest(ctx):
    """(snapshot id, step) of the newest committed snapshot still held; id 0 if none."""
    sid, step = C.c_uint64(), C.c_uint64()
    _check(ctx, lib().ckpt_latest(ctx, C.byref(sid), C.byref(step)))
    return sid.value, step.value


def ckpt_replicate_to(ctx, host, port, cls_mask):
    return _check(ctx, lib().ckpt_replicate_to(ctx, host.encode(), port, cls_mask))


def ckpt_replica_chunks(ctx):
    """(chunk ids uint64[m], replica bytes) of the replicated chunk set."""
    n = C.c_uint64()
    rb = C.c_uint64()
    _check(ctx, lib().ckpt_replica_chunks(ctx, None, 0, C.byref(n), C.byref(rb)))
    ids = np.zeros(max(n.value, 1), dtype=np.uint64)
    _check(ctx, lib().ckpt_replica_chunks(ctx, _u64p(ids), n.value, C.byref(n), C.byref(rb)))
    return ids[:n.value], rb.value


def ckpt_replica_result(ctx, snap_id):
    """(state, [bad chunk ids]) of a snapshot's replication."""
    st = C.c_int32()
    nb = C.c_uint32()
    _check(ctx, lib().ckpt_replica_result(ctx, snap_id, C.byref(st), None, 0, C.byref(nb)))
    bad = np.zeros(max(nb.value, 1), dtype=np.uint64)
    _check(ctx, lib().ckpt_replica_result(ctx, snap_id, C.byref(st), _u64p(bad), nb.value, C.byref(nb)))
    return st.value, [int(x) for x in bad[:nb.value]]


def ckpt_replica_peer_result(ctx, peer, snap_id):
    """(state, [bad chunk ids]) of a snapshot's replication to one peer."""
    st = C.c_int32()
    nb = C.c_uint32()
    _check(ctx, lib().ckpt_replica_peer_result(ctx, peer, snap_id, C.byref(st), None, 0, C.byref(nb)))
    bad = np.zeros(max(nb.value, 1), dtype=np.uint64)
    _check(ctx, lib().ckpt_replica_peer_result(ctx, peer, snap_id, C.byref(st), _u64p(bad), nb.value, C.byref(nb)))
    return st.value, [int(x) for x in bad[:nb.value]]


def ckpt_replicate_remove(ctx, peer):
    return _check(ctx, lib().ckpt_replicate_remove(ctx, peer))


def ckpt_replica_peers(ctx):
    n = C.c_uint32()
    _check(ctx, lib().ckpt_replica_peers(ctx, C.byref(n)))
    return n.value


def ckpt_debug_h2h_fault_peer(ctx, peer, kind, a=0, b=0):
    return _check(ctx, lib().ckpt_debug_h2h_fault_peer(ctx, peer, kind, a, b))


def ckpt_replica_timing(ctx):
    a, b = C.c_double(), C.c_double()
    _check(ctx, lib().ckpt_replica_timing(ctx, C.byref(a), C.byref(b)))
    return a.value, b.value


def ckpt_debug_h2h_fault(ctx, kind, a=0, b=0):
    return _check(ctx, lib().ckpt_debug_h2h_fault(ctx, kind, a, b))


def ckpt_restore_from_peer(ctx, host, port, stream=None):
    """A replacement rank's restore from its ring peer's newest committed
    replica: (snap_id, step, [chunk ids whose sum failed])."""
    _, _, nc = ckpt_layout(ctx, offsets=False)
    s = _stream(stream)
    sid, step = C.c_uint64(), C.c_uint64()
    bad = _bad_list_call(ctx, lambda b, cap, n: lib().ckpt_restore_from_peer(ctx, host.encode(), port, s,
                                                                              C.byref(sid), C.byref(step), b, cap,
                                                                              n), nc)
    return sid.value, step.value, bad


def ckpt_peer_restore_info(ctx):
    """What the last restore from a peer received: {"chunk_ids", "envelope",
    "fetch_ms", "check_ms"}."""
    n, elen = C.c_uint64(), C.c_uint64()
    fetch, check = C.c_double(), C.c_double()
    _check(ctx, lib().ckpt_peer_restore_info(ctx, None, 0, C.byref(n), None, 0, C.byref(elen), None, None))
    ids = np.zeros(max(n.value, 1), dtype=np.uint64)
    env = C.create_string_buffer(max(elen.value, 1))
    _check(ctx, lib().ckpt_peer_restore_info(ctx, _u64p(ids), n.value, C.byref(n), env, elen.value, C.byref(elen),
                                             C.byref(fetch), C.byref(check)))
    return {"chunk_ids": ids[:n.value], "envelope": env.raw[:elen.value], "fetch_ms": fetch.value,
            "check_ms": check.value}


def ckpt_pack_noalloc(tensors, image, sums, chunk_bytes=0, align_bytes=0, stream=None, device=None):
    """Allocation-free pack of `tensors` into the device tensors `image`
    (uint8) and `sums` (int64/uint64, one per chunk) on `stream`; returns
    (image_bytes, n_chunks).  Asynchronous like a kernel launch."""
    if device is None:
        device = torch.cuda.current_device()
    n = len(tensors)
    arr = (ckpt_tensor * max(n, 1))()
    for i, t in enumerate(tensors):
        if not t.is_cuda:
            raise ValueError("fragment %d is not a device tensor" % i)
        nb = tensor_bytes(t)
        arr[i].dev_ptr = t.data_ptr() if nb else None
        arr[i].nbytes = nb
    ib, nc = C.c_uint64(), C.c_uint64()
    rc = lib().ckpt_pack_noalloc(arr, n, chunk_bytes, align_bytes, device, C.c_void_p(image.data_ptr()),
                                 image.numel() * image.element_size(), C.c_void_p(sums.data_ptr()),
                                 sums.numel() * sums.element_size() // 8, _stream(stream), C.byref(ib), C.byref(nc))
    if rc != CKPT_OK:
        raise CkptError(rc, (lib().ckpt_last_error(None) or b"").decode())
    return ib.value, nc.value


class PeerError(RuntimeError):
    def __init__(self, code, msg):
        super().__init__("%s (%d): %s" % (_NAMES.get(code, "CKPT_E?"), code, msg))
        self.code = code


class Peer:
    """The receiving ring peer of H2H replication (include/ckpt.h,
    ckpt_peer_*): listens on 127.0.0.1, re-checks every received chunk sum on
    the GPU, keeps two alternating replica buffers."""

    def __init__(self, port=0, device=None, group_bytes=0):
        if device is None:
            device = torch.cuda.current_device()
        cfg = ckpt_config(0, 0, 0, 0, group_bytes, device, 0, 0, 0, None, 0, 0, 0)
        self.p = C.c_void_p()
        rc = lib().ckpt_peer_create(C.byref(cfg), port, C.byref(self.p))
        if rc != CKPT_OK:
            raise PeerError(rc, "ckpt_peer_create failed")
        pt = C.c_uint32()
        lib().ckpt_peer_port(self.p, C.byref(pt))
        self.port = pt.value

    def _err(self, rc):
        return PeerError(rc, (lib().ckpt_peer_last_error(self.p) or b"").decode())

    def wait(self, snap_id, timeout_ms=120_000):
        """Result code of the sender's snapshot snap_id (CKPT_OK, CKPT_ECORRUPT,
        CKPT_EHIP ...); raises on timeout."""
        r = C.c_int32()
        rc = lib().ckpt_peer_wait(self.p, snap_id, timeout_ms, C.byref(r))
        if rc != CKPT_OK:
            raise self._err(rc)
        return r.value

    def replica(self):
        """Newest committed replica: dict with snap_id, step, data (uint8 view),
        chunk_ids, sums, envelope (bytes)."""
        sid, step, nbytes, n, elen = C.c_uint64(), C.c_uint64(), C.c_uint64(), C.c_uint64(), C.c_uint64()
        data, env = C.c_void_p(), C.c_void_p()
        ids, sums = C.POINTER(C.c_uint64)(), C.POINTER(C.c_uint64)()
        rc = lib().ckpt_peer_replica(self.p, C.byref(sid), C.byref(step), C.byref(data), C.byref(nbytes),
                                     C.byref(ids), C.byref(sums), C.byref(n), C.byref(env), C.byref(elen))
        if rc != CKPT_OK:
            raise self._err(rc)
        return {"snap_id": sid.value, "step": step.value,
                "data": np.ctypeslib.as_array(C.cast(data, C.POINTER(C.c_uint8)), shape=(nbytes.value,)),
                "chunk_ids": np.ctypeslib.as_array(ids, shape=(n.value,)).copy(),
                "sums": np.ctypeslib.as_array(sums, shape=(n.value,)),
                "envelope": C.string_at(env, elen.value) if elen.value else b""}

    def last_bad(self):
        n = C.c_uint32()
        lib().ckpt_peer_last_bad(self.p, None, 0, C.byref(n))
        out = np.zeros(max(n.value, 1), dtype=np.uint64)
        lib().ckpt_peer_last_bad(self.p, _u64p(out), n.value, C.byref(n))
        return [int(x) for x in out[:n.value]]

    def timing(self):
        a, b = C.c_double(), C.c_double()
        lib().ckpt_peer_timing(self.p, C.byref(a), C.byref(b))
        return a.value, b.value

    def last_error(self):
        """Text of the receiver's last error ("" if none)."""
        return (lib().ckpt_peer_last_error(self.p) or b"").decode()

    def close(self):
        if self.p:
            lib().ckpt_peer_destroy(self.p)
            self.p = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


class Checkpointer:
    """One rank's in-memory snapshot context over a list of device tensors.

    The tensors (any dtype, contiguous, possibly views into flat buffers)
    are registered in order; they must stay allocated and unmoved while the
    Checkpointer lives (it keeps references).  Typical step:

        snap = ck.snapshot(step)            # right after optimizer step k-1
        ... forward / backward ...
        ck.wait_captured(snap, lo, hi)      # before overwriting fragments [lo, hi)
        ... optimizer step ...

    Recovery: ck.restore() (newest committed snapshot) or ck.verify().
    Replication: ck.replicate_to(port, cls_mask) once per peer, then
    ck.wait_replicated(snap).  A replacement rank registered with the same
    layout calls restore_from_peer(port) on the peer holding its replica.
    """

    def __init__(self, tensors, dtypes=None, classes=None, chunk_bytes=0, align_bytes=0, device_staging_bytes=0,
                 group_bytes=0, grid_blocks=0, device=None, bounce_bytes=0, host_threads=0, image_file=None,
                 image_file_mode=CKPT_FILE_CREATE, side_stream=None, pack_launch_bytes=0, d2h_engines=0,
                 poison=False, direct=False):
        self.tensors = list(tensors)
        self.side_stream = side_stream  # kept alive with the context
        self.ctx = ckpt_create(chunk_bytes, align_bytes, device_staging_bytes, group_bytes, device, grid_blocks,
                               bounce_bytes, host_threads, side_stream, pack_launch_bytes, d2h_engines, poison,
                               direct)
        try:
            if image_file is not None:
                ckpt_image_file(self.ctx, image_file, image_file_mode)
            ckpt_register_tensors(self.ctx, self.tensors, dtypes, classes)
        except Exception:
            ckpt_destroy(self.ctx)
            self.ctx = None
            raise
        self.offsets, self.image_bytes, self.n_chunks = ckpt_layout(self.ctx, len(self.tensors))

    def snapshot(self, step=0, meta=b"", stream=None):
        return ckpt_snapshot_async(self.ctx, stream, step, meta)

    def wait_captured(self, snap, frag_lo=0, frag_hi=None, stream=None):
        hi = len(self.tensors) if frag_hi is None else frag_hi
        return ckpt_wait(self.ctx, snap, CKPT_WAIT_CAPTURED, stream, frag_lo, hi)

    def wait_committed(self, snap):
        return ckpt_wait(self.ctx, snap, CKPT_WAIT_COMMITTED)

    def state(self, snap):
        return ckpt_snapshot_state(self.ctx, snap)

    def restore(self, snap=0, stream=None):
        return ckpt_restore(self.ctx, snap, stream)

    def verify(self, snap=0):
        return ckpt_verify(self.ctx, snap)

    def host_image(self, snap):
        return ckpt_host_image(self.ctx, snap)

    def envelope(self, snap):
        return ckpt_envelope(self.ctx, snap)

    def chunk_fragments(self, c):
        return ckpt_chunk_fragments(self.ctx, c)

    def latest(self):
        return ckpt_latest(self.ctx)

    def replicate_to(self, port, cls_mask, host="127.0.0.1"):
        return ckpt_replicate_to(self.ctx, host, port, cls_mask)

    def wait_replicated(self, snap):
        return ckpt_wait(self.ctx, snap, CKPT_WAIT_REPLICATED)

    def replica_result(self, snap):
        return ckpt_replica_result(self.ctx, snap)

    def replica_peer_result(self, peer, snap):
        return ckpt_replica_peer_result(self.ctx, peer, snap)

    def replicate_remove(self, peer):
        return ckpt_replicate_remove(self.ctx, peer)

    def restore_from_peer(self, port, host="127.0.0.1", stream=None):
        """Take the failed rank's replicated chunks back from its ring peer:
        (snap_id, step, [bad chunk ids])."""
        return ckpt_restore_from_peer(self.ctx, host, port, stream)

    def peer_restore_info(self):
        return ckpt_peer_restore_info(self.ctx)

    def close(self):
        if self.ctx is not None:
            ckpt_destroy(self.ctx)
            self.ctx = None

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
