"""ctypes binding of the plain-C oracle (ckpt_oracle.c).

Test infrastructure only: the definitions it implements (layout, pack,
checksum, restore, verify, locate, envelope) are stated in the header of
ckpt_oracle.c, following Sec. V-B (D2H paragraph) and Sec. VI-A of the paper
plus a per-chunk word-sum integrity check, which the paper does not have.  Arrays are numpy;
fragment bytes are numpy uint8 arrays or bytes objects.
"""
import ctypes as C
import os

import numpy as np

from .build_oracle import LIB, SRC, build

__all__ = ["layout", "pack", "pack_window", "chunk_sums", "restore_window", "verify", "locate",
           "envelope", "envelope_bytes", "lib", "use_library", "restore_library"]

_lib = None


def lib():
    """Load the oracle library, compiling it first when missing or stale."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB) or os.path.getmtime(LIB) < os.path.getmtime(SRC):
            build()
        _lib = _load(LIB)
    return _lib


def use_library(path):
    """Point this module at another build of ckpt_oracle.c (the mutation tests
    load copies with a planted mistake); returns the previous library."""
    global _lib
    prev = _lib
    _lib = _load(path) if path is not None else None
    return prev


def restore_library(prev):
    global _lib
    _lib = prev


def _load(path):
    if True:
        L = C.CDLL(path)
        u64p = C.POINTER(C.c_uint64)
        u32p = C.POINTER(C.c_uint32)
        u8p = C.POINTER(C.c_uint8)
        L.oracle_layout.argtypes = [C.c_uint32, u64p, C.c_uint64, C.c_uint64, u64p, u64p, u64p]
        L.oracle_layout.restype = C.c_int
        L.oracle_pack_window.argtypes = [C.c_uint32, C.POINTER(u8p), u64p, u64p, C.c_uint64, C.c_uint64, u8p]
        L.oracle_pack_window.restype = C.c_int
        L.oracle_chunk_sums.argtypes = [u8p, C.c_uint64, C.c_uint64, C.c_uint64, u64p]
        L.oracle_chunk_sums.restype = C.c_int
        L.oracle_restore_window.argtypes = [u8p, C.c_uint64, C.c_uint64, C.c_uint32, u64p, u64p, C.POINTER(u8p)]
        L.oracle_restore_window.restype = C.c_int
        L.oracle_verify.argtypes = [u8p, C.c_uint64, C.c_uint64, C.c_uint64, u64p, u32p, C.c_uint32]
        L.oracle_verify.restype = C.c_int64
        L.oracle_locate.argtypes = [C.c_uint64, C.c_uint64, C.c_uint64, C.c_uint32, u64p, u64p, u64p, u64p,
                                    u32p, C.c_uint32]
        L.oracle_locate.restype = C.c_int64
        L.oracle_envelope_bytes.argtypes = [C.c_uint32, C.c_uint64, C.c_uint32]
        L.oracle_envelope_bytes.restype = C.c_uint64
        L.oracle_envelope.argtypes = [C.c_uint64, C.c_uint64, C.c_uint64, C.c_uint64, C.c_uint64, C.c_uint32,
                                      u64p, u64p, u32p, u32p, u64p, u8p, C.c_uint32, u8p, C.c_uint64]
        L.oracle_envelope.restype = C.c_uint64
        return L


def _p(a, ct):
    return a.ctypes.data_as(C.POINTER(ct))


def _u64(a):
    return np.ascontiguousarray(np.asarray(a, dtype=np.uint64))


def _u8(b):
    if isinstance(b, (bytes, bytearray, memoryview)):
        return np.frombuffer(bytes(b), dtype=np.uint8)
    return np.ascontiguousarray(np.asarray(b).view(np.uint8).reshape(-1))


def layout(nbytes, align=256, chunk=4 << 20):
    """Definition 1: returns (off[n] uint64, image_bytes, n_chunks)."""
    nb = _u64(nbytes)
    n = len(nb)
    off = np.zeros(max(n, 1), dtype=np.uint64)
    I = C.c_uint64()
    nc = C.c_uint64()
    rc = lib().oracle_layout(n, _p(nb, C.c_uint64), align, chunk, _p(off, C.c_uint64), C.byref(I), C.byref(nc))
    if rc != 0:
        raise ValueError("oracle_layout: invalid alignment/chunk (%d, %d)" % (align, chunk))
    return off[:n].copy(), int(I.value), int(nc.value)


def _frag_ptrs(frags):
    arrs = [_u8(f) for f in frags]
    ptrs = (C.POINTER(C.c_uint8) * max(len(arrs), 1))()
    for i, a in enumerate(arrs):
        ptrs[i] = _p(a, C.c_uint8)
    return arrs, ptrs


def pack_window(frags, off, lo, hi):
    """Definition 2 restricted to image bytes [lo, hi): returns a uint8 array."""
    arrs, ptrs = _frag_ptrs(frags)
    nb = _u64([a.size for a in arrs])
    off = _u64(off)
    out = np.empty(hi - lo, dtype=np.uint8)
    rc = lib().oracle_pack_window(len(arrs), ptrs, _p(nb, C.c_uint64), _p(off, C.c_uint64), lo, hi,
                                  _p(out, C.c_uint8))
    if rc != 0:
        raise ValueError("oracle_pack_window")
    return out


def pack(frags, align=256, chunk=4 << 20):
    """Definitions 1 and 2: returns (image uint8[I], off, n_chunks)."""
    arrs = [_u8(f) for f in frags]
    off, I, nc = layout([a.size for a in arrs], align, chunk)
    return pack_window(arrs, off, 0, I), off, nc


def chunk_sums(window, lo, hi, chunk):
    """Definition 3 for the chunks of image bytes [lo, hi) (window = those bytes)."""
    w = _u8(window)
    assert w.size == hi - lo
    n = (hi - lo + chunk - 1) // chunk
    sums = np.zeros(max(n, 1), dtype=np.uint64)
    rc = lib().oracle_chunk_sums(_p(w, C.c_uint8), lo, hi, chunk, _p(sums, C.c_uint64))
    if rc != 0:
        raise ValueError("oracle_chunk_sums: window not chunk-aligned")
    return sums[:n].copy()


def restore_window(window, lo, hi, off, nbytes):
    """Definition 4 restricted to [lo, hi): returns a list of uint8 arrays, one
    per fragment, holding the window's bytes at the fragment positions it
    covers (bytes outside the window are left zero)."""
    w = _u8(window)
    nb = _u64(nbytes)
    off = _u64(off)
    outs = [np.zeros(int(b), dtype=np.uint8) for b in nb]
    arrs, ptrs = _frag_ptrs(outs)
    rc = lib().oracle_restore_window(_p(w, C.c_uint8), lo, hi, len(outs), _p(off, C.c_uint64),
                                     _p(nb, C.c_uint64), ptrs)
    if rc != 0:
        raise ValueError("oracle_restore_window")
    return arrs


def verify(window, lo, hi, chunk, stored):
    """Definition 4 (verify): sorted list of chunk indices whose sum differs."""
    w = _u8(window)
    st = _u64(stored)
    n = (hi - lo + chunk - 1) // chunk
    assert st.size == n
    bad = np.zeros(max(n, 1), dtype=np.uint32)
    cnt = lib().oracle_verify(_p(w, C.c_uint8), lo, hi, chunk, _p(st, C.c_uint64), _p(bad, C.c_uint32), n)
    if cnt < 0:
        raise ValueError("oracle_verify")
    return [int(x) for x in bad[:cnt]]


def locate(c, chunk, image_bytes, off, nbytes):
    """Definition 5: ((lo, hi), [fragment ids]) for chunk c."""
    off = _u64(off)
    nb = _u64(nbytes)
    lo = C.c_uint64()
    hi = C.c_uint64()
    cap = max(len(nb), 1)
    fr = np.zeros(cap, dtype=np.uint32)
    cnt = lib().oracle_locate(c, chunk, image_bytes, len(nb), _p(off, C.c_uint64), _p(nb, C.c_uint64),
                              C.byref(lo), C.byref(hi), _p(fr, C.c_uint32), cap)
    if cnt < 0:
        raise ValueError("oracle_locate: chunk out of range")
    return (int(lo.value), int(hi.value)), [int(x) for x in fr[:cnt]]


def envelope_bytes(n_frag, n_chunks, meta_len):
    return int(lib().oracle_envelope_bytes(n_frag, n_chunks, meta_len))


def envelope(step, align, chunk, image_bytes, off, nbytes, dtype, cls, sums, meta=b""):
    """The metadata envelope bytes (format in ckpt_oracle.c)."""
    off = _u64(off)
    nb = _u64(nbytes)
    dt = np.ascontiguousarray(np.asarray(dtype, dtype=np.uint32))
    cl = np.ascontiguousarray(np.asarray(cls, dtype=np.uint32))
    sm = _u64(sums)
    mt = np.frombuffer(bytes(meta) + b"\0", dtype=np.uint8)
    n = len(nb)
    total = envelope_bytes(n, sm.size, len(meta))
    out = np.zeros(total, dtype=np.uint8)
    got = lib().oracle_envelope(step, align, chunk, image_bytes, sm.size, n, _p(off, C.c_uint64),
                                _p(nb, C.c_uint64), _p(dt, C.c_uint32), _p(cl, C.c_uint32),
                                _p(sm, C.c_uint64), _p(mt, C.c_uint8), len(meta), _p(out, C.c_uint8), total)
    if got != total:
        raise ValueError("oracle_envelope")
    return out.tobytes()
