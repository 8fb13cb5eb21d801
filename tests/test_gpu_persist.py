"""Crash-surviving local snapshots: host images in a shared file mapping
(needs an MI355X).  A process takes snapshots and dies; a new process with
the same layout adopts the file and restores.  Expected bytes come from the
seeded input generator (numpy) and the oracle, never from the library.
"""
import multiprocessing as mp
import os
import struct
import uuid

import numpy as np
import pytest
import torch

import oracle as O
from gpu_util import garbage_fill, host_bytes

pytestmark = pytest.mark.gpu

if torch.cuda.is_available():
    import paper_2607_01646_amd as P

SIZES = [70_001, 4096, 3, 1 << 20, 0, 257, 300_000, 65_536, 12_345, 1 << 19]
CHUNK = 1 << 16
BOUNCE = 4 * CHUNK


def state(k):
    """Host bytes of the state at snapshot k (k = 1, 2, 3): seeded numpy."""
    rng = np.random.default_rng(1000 + k)
    return [rng.integers(0, 256, s, dtype=np.uint8) for s in SIZES]


@pytest.fixture
def path():
    d = "/dev/shm" if os.path.isdir("/dev/shm") else "/tmp"
    p = os.path.join(d, "ckpt_test_%s.img" % uuid.uuid4().hex)
    yield p
    if os.path.exists(p):
        os.unlink(p)


def load(tensors, host):
    for t, h in zip(tensors, host):
        if h.size:
            t.copy_(torch.from_numpy(h.copy()).to(t.device))
    torch.cuda.synchronize()


def writer(path, crash_mid_snapshot):
    """Snapshots of states 1 and 2 committed; state 3's snapshot is cut after
    one chunk group (it never commits); then the process dies without any
    cleanup."""
    import time

    import paper_2607_01646_amd as PP

    tensors = [torch.zeros(s, dtype=torch.uint8, device="cuda") for s in SIZES]
    ck = PP.Checkpointer(tensors, chunk_bytes=CHUNK, group_bytes=CHUNK, bounce_bytes=BOUNCE, image_file=path)
    for k in (1, 2):
        load(tensors, state(k))
        s = ck.snapshot(step=k, meta=b"state-%d" % k)
        ck.wait_committed(s)
    load(tensors, state(3))
    if crash_mid_snapshot:
        PP.ckpt_debug_interrupt_next(ck.ctx, 1)
        ck.snapshot(step=3)
        time.sleep(0.5)  # its first group lands in the image of state 1
    os._exit(0)  # no destroy, no flush: the file is all that is left


def run_writer(path, crash_mid_snapshot=True):
    ctx = mp.get_context("spawn")
    proc = ctx.Process(target=writer, args=(path, crash_mid_snapshot))
    proc.start()
    proc.join(timeout=120)
    assert proc.exitcode == 0


def adopt(path):
    tensors = [torch.zeros(s, dtype=torch.uint8, device="cuda") for s in SIZES]
    ck = P.Checkpointer(tensors, chunk_bytes=CHUNK, group_bytes=CHUNK, bounce_bytes=BOUNCE, image_file=path,
                        image_file_mode=P.CKPT_FILE_ADOPT)
    return ck, tensors


def expected_image(k):
    img, off, nc = O.pack(state(k), 256, CHUNK)
    return img, off, O.chunk_sums(img, 0, img.size, CHUNK)


def test_restore_after_the_writer_died_mid_snapshot(path):
    run_writer(path)
    ck, tensors = adopt(path)
    sid, step = ck.latest()
    assert sid != 0 and step == 2  # the cut snapshot never became the recovery point
    img, off, sums = expected_image(2)
    got, got_sums = ck.host_image(sid)
    assert np.array_equal(got, img) and np.array_equal(got_sums, sums)
    want_env = O.envelope(2, 256, CHUNK, img.size, off, SIZES, [0] * len(SIZES), [0] * len(SIZES), sums, b"state-2")
    assert ck.envelope(sid) == want_env
    garbage_fill(tensors)
    assert ck.restore(0) == []
    torch.cuda.synchronize()
    for t, h in zip(tensors, state(2)):
        assert np.array_equal(host_bytes(t), h)
    # the adopted context goes on: its next snapshot takes the other image
    load(tensors, state(1))
    s = ck.snapshot(step=4)
    ck.wait_committed(s)
    assert ck.latest() == (s, 4)
    ck.close()


def test_restore_after_a_clean_exit_between_snapshots(path):
    run_writer(path, crash_mid_snapshot=False)
    ck, tensors = adopt(path)
    assert ck.latest()[1] == 2
    assert ck.restore(0) == []
    torch.cuda.synchronize()
    for t, h in zip(tensors, state(2)):
        assert np.array_equal(host_bytes(t), h)
    ck.close()


def head_and_records(path):
    with open(path, "rb") as f:
        raw = f.read(4096 + 1024)
    head = struct.unpack_from("<8sII3QII Q 2Q 2Q 2Q Q", raw, 0)
    recs = [struct.unpack_from("<6Q", raw, 4096 + 512 * b) for b in range(2)]
    return head, recs


def test_file_format_matches_its_description(path):
    """The head and records of the written file, parsed from the format in
    include/ckpt.h, against the oracle."""
    run_writer(path, crash_mid_snapshot=False)
    head, recs = head_and_records(path)
    magic, version, align, chunk, image, nc, nfrag, _, table_sum = head[:9]
    img, off, sums = expected_image(2)
    assert (magic, version, align, chunk, image, nc, nfrag) == (b"CKPTFIL1", 1, 256, CHUNK, img.size,
                                                                 sums.size, len(SIZES))
    assert table_sum == sum(int(o) + s for o, s in zip(off, SIZES)) % (1 << 64)
    image_off, sums_off, meta_off = head[9:11], head[11:13], head[13:15]
    states = sorted((r[1], b) for b, r in enumerate(recs) if r[0] == 1)
    assert len(states) == 2  # both images committed (states 1 and 2)
    b = states[-1][1]  # the newest
    state_, seq, snap_id, step, meta_len, rec_sum = recs[b]
    assert step == 2 and meta_len == 7
    raw = np.fromfile(path, dtype=np.uint8)
    assert np.array_equal(raw[image_off[b]:image_off[b] + img.size], img)
    file_sums = raw[sums_off[b]:sums_off[b] + 8 * nc].view("<u8")
    assert np.array_equal(file_sums, sums)
    blob = raw[meta_off[b]:meta_off[b] + 8].tobytes()
    assert blob == b"state-2\0"
    want = (seq + snap_id + step + meta_len + int(sums.sum(dtype=np.uint64))
            + int(np.frombuffer(blob, "<u8").sum(dtype=np.uint64))) % (1 << 64)
    assert rec_sum == want


def test_torn_newest_record_falls_back_to_the_older_image(path):
    run_writer(path, crash_mid_snapshot=False)
    head, recs = head_and_records(path)
    b = max(range(2), key=lambda i: recs[i][1])
    sums_off = head[11:13]
    with open(path, "r+b") as f:  # one byte of the newest image's stored sums
        f.seek(sums_off[b] + 3)
        x = f.read(1)
        f.seek(sums_off[b] + 3)
        f.write(bytes([x[0] ^ 0x01]))
    ck, tensors = adopt(path)
    assert ck.latest()[1] == 1
    assert ck.restore(0) == []
    torch.cuda.synchronize()
    for t, h in zip(tensors, state(1)):
        assert np.array_equal(host_bytes(t), h)
    ck.close()


def test_flipped_image_byte_in_the_file_is_located(path):
    run_writer(path)
    ck, tensors = adopt(path)
    sid, _ = ck.latest()
    img, _ = ck.host_image(sid)  # the shared mapping of the file
    img[5 * CHUNK + 17] ^= 0x80
    assert ck.verify(sid) == [5]
    assert ck.restore(sid) == [5]
    ck.close()


def test_adopting_a_file_of_another_layout_is_refused(path):
    run_writer(path, crash_mid_snapshot=False)
    tensors = [torch.zeros(s + 1, dtype=torch.uint8, device="cuda") for s in SIZES]
    with pytest.raises(P.CkptError) as e:
        P.Checkpointer(tensors, chunk_bytes=CHUNK, group_bytes=CHUNK, bounce_bytes=BOUNCE, image_file=path,
                       image_file_mode=P.CKPT_FILE_ADOPT)
    assert e.value.code == P.CKPT_EINVAL
    with pytest.raises(P.CkptError) as e:  # pinned images cannot live in a file
        P.Checkpointer(tensors, chunk_bytes=CHUNK, image_file=path)
    assert e.value.code == P.CKPT_EINVAL
