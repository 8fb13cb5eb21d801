"""The oracle over random layouts (CPU only), against facts computed here by
other means: the image is each fragment's bytes at its offset with zeros
elsewhere, a chunk sum is the sum of the chunk's little-endian 64-bit words
as Python integers modulo 2^64, the restore gives every fragment back, and
one flipped bit is reported in exactly its own chunk."""
import numpy as np
from hypothesis import HealthCheck, given, settings
from hypothesis import strategies as st

import oracle as O


@st.composite
def shards(draw):
    A = 1 << draw(st.integers(4, 12))
    C = A * draw(st.integers(1, max(1, (16 << 10) // A)))
    size = st.one_of(st.just(0), st.integers(1, 64), st.integers(1, 3000), st.integers(1, 3 * C))
    sizes = draw(st.lists(size, min_size=1, max_size=24).filter(any))
    seed = draw(st.integers(0, 2**32 - 1))
    rng = np.random.default_rng(seed)
    frags = [rng.integers(0, 256, n, dtype=np.uint8) for n in sizes]
    return frags, sizes, A, C, seed


def word_sum(b):
    total = 0
    for k in range(0, len(b), 8):
        total += int.from_bytes(bytes(b[k:k + 8]), "little")
    return total % (1 << 64)


@settings(max_examples=120, deadline=None, suppress_health_check=[HealthCheck.too_slow])
@given(shards())
def test_pack_sums_restore_and_a_flip(shard):
    frags, sizes, A, C, seed = shard
    img, off, nc = O.pack(frags, A, C)
    I = img.size
    assert I % A == 0 and nc == -(-I // C)
    # bytes at their offsets, in registration order, without overlap; zeros elsewhere
    covered = np.zeros(I, dtype=bool)
    for f, o in zip(frags, off):
        o = int(o)
        assert o % A == 0
        assert np.array_equal(img[o:o + f.size], f)
        assert not covered[o:o + f.size].any()
        covered[o:o + f.size] = True
    assert not img[~covered].any()
    last = max(int(o) + n for o, n in zip(off, sizes) if n)
    assert I - last < A  # the image ends on the padding of its last byte
    # chunk sums as Python integers
    sums = O.chunk_sums(img, 0, I, C)
    assert [int(s) for s in sums] == [word_sum(img[c * C:min((c + 1) * C, I)]) for c in range(nc)]
    # restore gives back every fragment
    back = O.restore_window(img, 0, I, off, sizes)
    assert all(np.array_equal(a, b) for a, b in zip(frags, back))
    # one flipped bit of a fragment byte: exactly its chunk fails
    rng = np.random.default_rng(seed + 1)
    x = int(rng.choice(np.flatnonzero(covered)))
    bad = img.copy()
    bad[x] ^= np.uint8(1 << int(rng.integers(0, 8)))
    assert O.verify(bad, 0, I, C, sums) == [x // C]
