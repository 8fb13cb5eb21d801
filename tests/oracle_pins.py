"""Pins of the CPU oracle: checks it against facts fixed by mathematics or by
hand-worked values, never against itself.

Each check raises AssertionError on failure.  test_oracle_pins.py runs them
against the oracle; test_oracle_mutants.py runs them against copies of the
oracle with a planted mistake and expects at least one to fail.
"""
import os
import struct

import numpy as np

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")
M64 = (1 << 64) - 1


def _golden_lines(name):
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.strip()
            if line and not line.startswith("#"):
                yield line


def pin_checksum_hand_vectors(O):
    n = 0
    for line in _golden_lines("checksum_vectors.txt"):
        hexbytes, want = [s.strip() for s in line.split("|")]
        data = bytes.fromhex(hexbytes.replace(" ", ""))
        got = O.chunk_sums(data, 0, len(data), len(data))
        assert int(got[0]) == int(want, 16), (hexbytes, hex(int(got[0])), want)
        n += 1
    assert n >= 7


def pin_checksum_vs_numpy(O, seed=11):
    """numpy's uint64 reduction is a separate implementation of the same
    modular sum (it wraps modulo 2^64)."""
    rng = np.random.default_rng(seed)
    assert int(np.array([M64, 2], dtype=np.uint64).sum(dtype=np.uint64)) == 1
    for chunk, nbytes in [(256, 256 * 7), (1024, 4096 + 512), (4096, 4096 * 3 + 256), (64, 64 * 5 + 8)]:
        img = rng.integers(0, 256, nbytes, dtype=np.uint8)
        got = O.chunk_sums(img, 0, nbytes, chunk)
        want = [int(np.frombuffer(img[c:c + chunk].tobytes(), dtype="<u8").sum(dtype=np.uint64))
                for c in range(0, nbytes, chunk)]
        assert [int(x) for x in got] == want


def pin_checksum_closed_forms(O, seed=12):
    rng = np.random.default_rng(seed)
    for n in [1, 2, 3, 31, 32, 257]:
        w = int(rng.integers(0, 1 << 63)) * 2 + 1  # odd, high bits set
        data = struct.pack("<Q", w) * n
        got = int(O.chunk_sums(data, 0, len(data), len(data))[0])
        assert got == (n * w) & M64
    # A chunk of zeros sums to zero; one non-zero word anywhere gives that word.
    for pos in [0, 8, 248]:
        data = bytearray(256)
        data[pos:pos + 8] = struct.pack("<Q", 0xDEADBEEFCAFEF00D)
        assert int(O.chunk_sums(bytes(data), 0, 256, 256)[0]) == 0xDEADBEEFCAFEF00D


def pin_single_flip_delta(O, seed=13):
    """Flipping bit k of a word adds 2^k if it was 0 and subtracts 2^k if it
    was 1 (mod 2^64); only the flipped chunk changes."""
    rng = np.random.default_rng(seed)
    chunk = 512
    img = rng.integers(0, 256, chunk * 4, dtype=np.uint8)
    base = [int(x) for x in O.chunk_sums(img, 0, img.size, chunk)]
    for _ in range(64):
        byte = int(rng.integers(0, img.size))
        bit = int(rng.integers(0, 8))
        was = (int(img[byte]) >> bit) & 1
        flipped = img.copy()
        flipped[byte] ^= np.uint8(1 << bit)
        got = [int(x) for x in O.chunk_sums(flipped, 0, img.size, chunk)]
        k = 8 * (byte % 8) + bit
        c = byte // chunk
        delta = (-(1 << k) if was else (1 << k)) & M64
        for j in range(len(base)):
            want = (base[j] + delta) & M64 if j == c else base[j]
            assert got[j] == want
        assert O.verify(flipped, 0, img.size, chunk, base) == [c]


def pin_exhaustive_single_flips(O):
    """Brute force on a tiny image: every one of its 4096 bits, flipped alone,
    is reported in exactly its own chunk."""
    chunk = 256
    rng = np.random.default_rng(14)
    img = rng.integers(0, 256, 512, dtype=np.uint8)
    stored = O.chunk_sums(img, 0, 512, chunk)
    assert O.verify(img, 0, 512, chunk, stored) == []
    for byte in range(512):
        for bit in range(8):
            img[byte] ^= np.uint8(1 << bit)
            assert O.verify(img, 0, 512, chunk, stored) == [byte // chunk]
            img[byte] ^= np.uint8(1 << bit)


def pin_cancelling_flips(O):
    """A known blind spot, predicted exactly: the same bit flipped 0->1 in one
    word and 1->0 in another word of the same chunk cancels."""
    data = bytearray(256)
    data[8] = 0x10  # word 1 has bit 4 set
    stored = O.chunk_sums(bytes(data), 0, 256, 256)
    data[8] = 0x00  # 1->0 in word 1
    data[16] = 0x10  # 0->1 in word 2
    assert O.verify(bytes(data), 0, 256, 256, stored) == []


def pin_layout_golden(O):
    n = 0
    for line in _golden_lines("layout_cases.txt"):
        head, sizes, offs, tail = [s.strip() for s in line.split("|")]
        A, C = [int(x) for x in head.split()]
        sizes = [int(x) for x in sizes.split()]
        offs = [int(x) for x in offs.split()]
        I, nc = [int(x) for x in tail.split()]
        off, gotI, gotnc = O.layout(sizes, A, C)
        assert [int(x) for x in off] == offs, (sizes, off, offs)
        assert (gotI, gotnc) == (I, nc)
        n += 1
    assert n >= 5


def pin_layout_invariants(O, seed=15):
    rng = np.random.default_rng(seed)
    for A, C in [(256, 256), (256, 4096), (512, 1 << 20), (64, 192)]:
        sizes = [int(s) for s in rng.integers(0, 3000, 200)]
        sizes[5] = 0
        sizes[6] = A
        off, I, nc = O.layout(sizes, A, C)
        prev_end = 0
        for i, (o, s) in enumerate(zip(off, sizes)):
            o = int(o)
            assert o % A == 0
            assert o >= prev_end and o - prev_end < A  # no overlap, minimal padding
            prev_end = o + s
        assert I % A == 0 and prev_end <= I < prev_end + A
        assert nc == -(-I // C)
    assert O.layout([], 256, 256)[1:] == (0, 0)


def _fragments(rng, sizes):
    return [rng.integers(0, 256, s, dtype=np.uint8) for s in sizes]


def pin_pack_places_bytes(O, seed=16):
    rng = np.random.default_rng(seed)
    sizes = [1, 2, 255, 256, 257, 0, 1000, 3, 4096, 7]
    frags = _fragments(rng, sizes)
    img, off, nc = O.pack(frags, 256, 1024)
    mask = np.zeros(img.size, dtype=bool)
    for f, o in zip(frags, off):
        o = int(o)
        assert np.array_equal(img[o:o + f.size], f)
        mask[o:o + f.size] = True
    assert not img[~mask].any()  # every padding byte is zero


def pin_round_trip(O, seed=17):
    rng = np.random.default_rng(seed)
    sizes = [int(s) for s in rng.integers(0, 5000, 60)] + [0, 1, 2, 3]
    frags = _fragments(rng, sizes)
    C = 2048
    img, off, nc = O.pack(frags, 256, C)
    back = O.restore_window(img, 0, img.size, off, sizes)
    for a, b in zip(frags, back):
        assert np.array_equal(a, b)
    # The window forms agree with the whole-image forms, chunk by chunk.
    sums = O.chunk_sums(img, 0, img.size, C)
    acc = [np.zeros(s, dtype=np.uint8) for s in sizes]
    for c in range(nc):
        lo, hi = c * C, min((c + 1) * C, img.size)
        win = O.pack_window(frags, off, lo, hi)
        assert np.array_equal(win, img[lo:hi])
        assert int(O.chunk_sums(win, lo, hi, C)[0]) == int(sums[c])
        part = O.restore_window(win, lo, hi, off, sizes)
        for i in range(len(sizes)):
            a, b = int(off[i]), int(off[i]) + sizes[i]
            s0, s1 = max(a, lo) - a, min(b, hi) - a
            if s1 > s0:
                acc[i][s0:s1] = part[i][s0:s1]
    for a, b in zip(frags, acc):
        assert np.array_equal(a, b)


def pin_chunk_sum_additive(O, seed=18):
    """The chunk sum equals the sum over its 256-byte pieces (segments start on
    the alignment, so a chunk splits into whole words)."""
    rng = np.random.default_rng(seed)
    img = rng.integers(0, 256, 8192, dtype=np.uint8)
    whole = int(O.chunk_sums(img, 0, 8192, 8192)[0])
    parts = sum(int(x) for x in O.chunk_sums(img, 0, 8192, 256)) & M64
    assert whole == parts


def pin_locate_by_markers(O, seed=19):
    """Which fragments overlap a chunk, found independently: fill fragment i
    with the marker byte pattern of i+1 and read the markers back out of the
    packed chunk."""
    rng = np.random.default_rng(seed)
    sizes = [int(s) for s in rng.integers(0, 700, 120)]
    sizes[3] = 0
    sizes[4] = 0
    frags = [np.full(s, 0, dtype=np.uint8) for s in sizes]
    # 2-byte marker of i+1 in every even/odd byte pair, never all-zero
    for i, s in enumerate(sizes):
        m = np.frombuffer(struct.pack("<H", i + 1), dtype=np.uint8)
        frags[i] = np.resize(m, s).astype(np.uint8)
    C = 512
    img, off, nc = O.pack(frags, 256, C)
    for c in range(nc):
        (lo, hi), ids = O.locate(c, C, img.size, off, sizes)
        assert (lo, hi) == (c * C, min((c + 1) * C, img.size))
        seen = set()
        for i, s in enumerate(sizes):
            o = int(off[i])
            if s and o < hi and o + s > lo:
                # the marker bytes of fragment i really are inside the chunk
                a = max(o, lo)
                seen.add(i)
                x = img[a]
                assert x == frags[i][a - o]
        assert sorted(ids) == sorted(seen)


def pin_envelope(O):
    """Parse the envelope with struct (a separate reader) and check fields."""
    off = [0, 256, 1024]
    nb = [3, 700, 16]
    dt = [1, 2, 2]
    cl = [0, 1, 3]
    sums = [5, M64, 0x0123456789ABCDEF]
    meta = b"rng:42;tp=8"
    env = O.envelope(7, 256, 512, 1280, off, nb, dt, cl, sums, meta)
    assert len(env) == 56 + 24 * 3 + 8 * 3 + 16 + 8
    assert env[:8] == b"CKPTENV1"
    ver, A, step, C, I, nc, nf, ml = struct.unpack_from("<IIQQQQII", env, 8)
    assert (ver, A, step, C, I, nc, nf, ml) == (1, 256, 7, 512, 1280, 3, 3, len(meta))
    p = 56
    for i in range(3):
        assert struct.unpack_from("<QQII", env, p) == (off[i], nb[i], dt[i], cl[i])
        p += 24
    assert list(struct.unpack_from("<3Q", env, p)) == sums
    p += 24
    assert env[p:p + len(meta)] == meta and env[p + len(meta):p + 16] == b"\0" * (16 - len(meta))
    p += 16
    words = np.frombuffer(env[:p], dtype="<u8")
    assert struct.unpack_from("<Q", env, p)[0] == int(words.sum(dtype=np.uint64))


ALL_PINS = [
    pin_checksum_hand_vectors,
    pin_checksum_vs_numpy,
    pin_checksum_closed_forms,
    pin_single_flip_delta,
    pin_exhaustive_single_flips,
    pin_cancelling_flips,
    pin_layout_golden,
    pin_layout_invariants,
    pin_pack_places_bytes,
    pin_round_trip,
    pin_chunk_sum_additive,
    pin_locate_by_markers,
    pin_envelope,
]
