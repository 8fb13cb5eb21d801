"""ckpt_pack_noalloc (the allocation-free pack) against the snapshot entry
point it varies, ckpt_snapshot_async, and against the oracle: bit-exact
image bytes and chunk sums, on two calls in a row (the second smaller), on
images of several scratch groups, and on misaligned views and adversarial
bit patterns.  Needs an MI355X; goes through the C ABI."""
import numpy as np
import pytest
import torch

import oracle as O
import workloads as W
from gpu_util import EDGE_SIZES, host_bytes, random_byte_fragments

pytestmark = pytest.mark.gpu

if torch.cuda.is_available():
    import paper_2607_01646_amd as P

PATTERN = 0xC3


def _outputs(sets, chunk, align):
    """Output buffers with room for the largest of the fragment sets, plus a
    margin that must stay untouched."""
    I, nc = 0, 0
    for tensors in sets:
        _, i, n = P.ckpt_plan([t.numel() * t.element_size() for t in tensors], chunk, align)
        I, nc = max(I, i), max(nc, n)
    image = torch.full((I + 4096,), PATTERN, dtype=torch.uint8, device="cuda")
    sums = torch.full((nc + 8,), -1, dtype=torch.int64, device="cuda")
    return image, sums


def _snapshot(tensors, chunk, align):
    """The existing entry point: image and sums of a committed snapshot."""
    with P.Checkpointer(tensors, chunk_bytes=chunk, align_bytes=align) as ck:
        s = ck.snapshot(step=1)
        ck.wait_committed(s)
        img, sums = ck.host_image(s)
        return img.copy(), sums.copy()


def _noalloc(tensors, chunk, align, image, sums, stream=None):
    I, nc = P.ckpt_pack_noalloc(tensors, image, sums, chunk_bytes=chunk, align_bytes=align, stream=stream)
    torch.cuda.synchronize()
    return I, nc, image.cpu().numpy(), sums.cpu().numpy().view(np.uint64)


def _check(tensors, chunk, align, image, sums, stream=None):
    host = [host_bytes(t) for t in tensors]
    want, _, nc_o = O.pack(host, align, chunk)
    want_sums = O.chunk_sums(want, 0, want.size, chunk)
    ref_img, ref_sums = _snapshot(tensors, chunk, align)
    I, nc, img, got_sums = _noalloc(tensors, chunk, align, image, sums, stream)
    assert (I, nc) == (want.size, nc_o)
    assert np.array_equal(img[:I], ref_img) and np.array_equal(img[:I], want)
    assert np.array_equal(got_sums[:nc], ref_sums) and np.array_equal(got_sums[:nc], want_sums)
    assert np.all(img[I:] == PATTERN), "bytes past the image were written"
    assert np.all(got_sums[nc:] == np.uint64(0xFFFFFFFFFFFFFFFF)), "sums past the chunk count were written"
    return I, nc


@pytest.mark.parametrize("chunk,align", [(4096, 256), (768, 256), (65536, 16), (16, 16)])
def test_two_calls_in_a_row_match_the_snapshot_entry_point(chunk, align):
    """A larger call, then a smaller one into the same output buffers (the
    scratch keeps the first call's contents)."""
    big, _ = random_byte_fragments(EDGE_SIZES + [3 << 20, 5, 0, 1 << 16], seed=chunk + align)
    small, _ = random_byte_fragments([7, 4097, 300, 0, 65537], seed=chunk + align + 1)
    image, sums = _outputs([big, small], chunk, align)
    I1, nc1 = _check(big, chunk, align, image, sums)
    image.fill_(PATTERN)
    sums.fill_(-1)
    I2, nc2 = _check(small, chunk, align, image, sums)
    assert I2 < I1 and nc2 <= nc1


def test_several_scratch_groups():
    """768-byte chunks have 256-byte tiles, so the scratch's 131072 tiles
    cover 32 MiB per group: a 100 MB state is packed in four groups that
    reuse the scratch, then a smaller one in one group."""
    rng = np.random.default_rng(9)
    sizes = [int(s) for s in rng.integers(1, 3 << 20, 60)] + [40 << 20]
    tensors, _ = random_byte_fragments(sizes, seed=10)
    image, sums = _outputs([tensors], 768, 256)
    I, nc = _check(tensors, 768, 256, image, sums)
    assert I > 96 << 20
    image.fill_(PATTERN)
    sums.fill_(-1)
    _check(tensors[:5], 768, 256, image, sums)


def test_shard_views_and_bit_patterns_on_a_side_stream():
    tensors, _ = W.make_state(1, device="cuda")
    views, _ = W.misaligned_views("cuda")
    frags = tensors[:24] + views + W.adversarial_fragments("cuda")
    torch.cuda.synchronize()
    image, sums = _outputs([frags], 1 << 20, 256)
    side = torch.cuda.Stream()
    _check(frags, 1 << 20, 256, image, sums, stream=side)


def test_allocates_no_device_memory():
    tensors, _ = random_byte_fragments([1 << 20, 12345, 1 << 22], seed=4)
    image, sums = _outputs([tensors], 1 << 20, 256)
    P.ckpt_pack_noalloc(tensors, image, sums, chunk_bytes=1 << 20)  # first call on the device: scratch lookup
    torch.cuda.synchronize()
    free0 = torch.cuda.mem_get_info()[0]
    for _ in range(3):
        P.ckpt_pack_noalloc(tensors, image, sums, chunk_bytes=1 << 20)
    torch.cuda.synchronize()
    assert torch.cuda.mem_get_info()[0] == free0


def test_limits_and_bad_arguments_are_errors():
    tensors, _ = random_byte_fragments([5000, 70000], seed=6)
    image = torch.zeros(1 << 20, dtype=torch.uint8, device="cuda")
    sums = torch.zeros(4, dtype=torch.int64, device="cuda")

    def code(**kw):
        with pytest.raises(P.CkptError) as e:
            P.ckpt_pack_noalloc(**kw)
        return e.value.code, str(e.value)

    c, msg = code(tensors=tensors, image=image, sums=sums[:1], chunk_bytes=4096)
    assert c == P.CKPT_EINVAL and "sums" in msg
    c, msg = code(tensors=tensors, image=image[:1000], sums=sums, chunk_bytes=1 << 20)
    assert c == P.CKPT_EINVAL and "image" in msg
    c, msg = code(tensors=tensors, image=image[1:], sums=sums, chunk_bytes=1 << 20)
    assert c == P.CKPT_EINVAL and "aligned" in msg
    many = [tensors[0][:0]] * 65537
    c, msg = code(tensors=many, image=image, sums=sums, chunk_bytes=1 << 20)
    assert c == P.CKPT_EINVAL and "65536" in msg
    c, msg = code(tensors=tensors, image=image, sums=sums, chunk_bytes=2 << 30)
    assert c == P.CKPT_EINVAL and "1 GiB" in msg
    pinned = torch.zeros(4096, dtype=torch.uint8, pin_memory=True)
    with pytest.raises(ValueError):
        P.ckpt_pack_noalloc([pinned], image, sums)  # the binding refuses host tensors itself
    # below the binding: a host pointer is refused by the library
    arr = (P.ckpt_tensor * 1)()
    arr[0].dev_ptr = pinned.data_ptr()
    arr[0].nbytes = 4096
    import ctypes as C

    ib, nc = C.c_uint64(), C.c_uint64()
    rc = P.lib().ckpt_pack_noalloc(arr, 1, 1 << 20, 0, torch.cuda.current_device(), C.c_void_p(image.data_ptr()),
                                   image.numel(), C.c_void_p(sums.data_ptr()), 4, None, C.byref(ib), C.byref(nc))
    assert rc == P.CKPT_EINVAL and b"not device memory" in P.lib().ckpt_last_error(None)
    torch.cuda.synchronize()
