"""The GPU tests' full-image checker and restore digests, exercised on the
CPU: each must pass on correct data and fail on a planted mistake, so a
green full-size parity test means what it says."""
import numpy as np
import pytest
import torch

import oracle as O
from gpu_util import check_image_against_oracle, fragment_digests, window_slices


def _state(seed=3):
    rng = np.random.default_rng(seed)
    sizes = [int(s) for s in rng.integers(0, 70_000, 40)] + [0, 5, 3 << 16]
    frags = [torch.from_numpy(rng.integers(0, 256, s, dtype=np.uint8)) for s in sizes]
    return frags, sizes


@pytest.mark.parametrize("chunk", [4096, 1 << 16])
def test_full_image_check_passes_and_catches_planted_mistakes(chunk):
    frags, sizes = _state()
    host = [f.numpy() for f in frags]
    img, off, nc = O.pack(host, 256, chunk)
    sums = O.chunk_sums(img, 0, img.size, chunk)
    assert check_image_against_oracle(frags, off, sizes, img, sums, chunk, threads=4) == nc
    bad = img.copy()
    k = img.size // 2 + 7
    bad[k] ^= 0x10
    with pytest.raises(AssertionError, match="chunk %d differs" % (k // chunk)):
        check_image_against_oracle(frags, off, sizes, bad, sums, chunk, threads=4)
    wrong = sums.copy()
    wrong[nc - 1] += np.uint64(1)
    with pytest.raises(AssertionError, match="chunk %d: stored sum" % (nc - 1)):
        check_image_against_oracle(frags, off, sizes, img, wrong, chunk, threads=4)
    # a fragment placed one alignment step late
    shifted = img.copy()
    i = 10
    o = int(off[i])
    shifted[o + 256:o + 256 + sizes[i]] = host[i]
    if sizes[i]:
        with pytest.raises(AssertionError):
            check_image_against_oracle(frags, off, sizes, shifted, sums, chunk, threads=4)


def test_window_slices_cover_each_fragment_byte_once():
    frags, sizes = _state(5)
    off, I, nc = O.layout(sizes, 256, 4096)
    seen = [np.zeros(s, dtype=np.int32) for s in sizes]
    for c in range(nc):
        lo, hi = c * 4096, min((c + 1) * 4096, I)
        for piece, at in zip(*window_slices(frags, off, sizes, lo, hi)):
            assert lo <= at and at + piece.size <= hi
            i = max(j for j in range(len(sizes)) if int(off[j]) <= at and sizes[j])
            a = at - int(off[i])
            assert np.array_equal(piece, frags[i].numpy()[a:a + piece.size])
            seen[i][a:a + piece.size] += 1
    assert all(np.all(s == 1) for s in seen)


def test_digests_see_changed_and_moved_bytes():
    frags, _ = _state(7)
    d0 = fragment_digests(frags, piece=1000)
    assert d0 == fragment_digests([f.clone() for f in frags], piece=777)
    t = frags[-1].clone()
    t[100] ^= 1
    assert fragment_digests([t])[0] != d0[-1]
    w = frags[-1].clone().view(torch.int32)
    w[[3, 9]] = w[[9, 3]]  # two words swapped: same plain sum, different weighted sum
    dw = fragment_digests([w.view(torch.uint8)])[0]
    assert dw[1] == d0[-1][1] and dw[2] != d0[-1][2]
    odd = torch.arange(13, dtype=torch.uint8)
    assert fragment_digests([odd])[0] == (13, int(odd.sum()), sum(int(x) * (k + 1) for k, x in enumerate(odd)))
