"""A replacement rank takes its optimizer state back from the ring peer's
replica (Sec. V-C, third recovery stage), against the CPU oracle (needs an
MI355X; ranks and peer talk over TCP on 127.0.0.1).

The expected tensors come from the oracle alone: the failed rank's image
(oracle pack of its state at the snapshot), the replicated chunk ids
(oracle locate of the optimizer classes), and the replacement's own bytes
wherever no replicated chunk reaches.
"""
import multiprocessing as mp
import os
import sys

import numpy as np
import pytest
import torch

import oracle as O
import workloads as W
from gpu_util import class_major, expected_after_restore, expected_replica, garbage_fill, host_bytes

pytestmark = pytest.mark.gpu

if torch.cuda.is_available():
    import paper_2607_01646_amd as P

OPT = (1 << W.CLS_MASTER) | (1 << W.CLS_ADAM_M) | (1 << W.CLS_ADAM_V)
CHUNK = 1 << 20


def state():
    tensors, plan = W.make_state(1, device="cuda")
    tensors, dtypes, classes = class_major(tensors, plan)
    torch.cuda.synchronize()
    return tensors, dtypes, classes


def replacement_like(tensors, value=0x3C):
    """Fresh tensors of the failed rank's shapes, filled with a byte pattern."""
    out = [torch.empty_like(t) for t in tensors]
    garbage_fill(out, value)
    torch.cuda.synchronize()
    return out


def expected_after(failed_host, before_host, classes, ids):
    return expected_after_restore(failed_host, before_host, ids, CHUNK)


def assert_tensors(tensors, want):
    torch.cuda.synchronize()
    for i, (t, w) in enumerate(zip(tensors, want)):
        assert np.array_equal(host_bytes(t), w), "fragment %d differs" % i


@pytest.mark.parametrize("bounce, staging, direct", [(0, 0, False), (2 << 20, 0, False), (0, 3 << 20, False),
                                                     (0, 0, True), (2 << 20, 0, True)])
def test_replacement_takes_the_optimizer_state_back(bounce, staging, direct):
    """Rank A replicates snapshot (step 7) to the peer and is lost; replacement
    B, registered with A's layout, restores from the peer: the optimizer
    fragments equal A's at step 7, parameter-only fragments keep B's bytes.
    With direct D2H both ranks stage nothing and B restores through its
    device ring."""
    tensors, dtypes, classes = state()
    peer = P.Peer()
    a = P.Checkpointer(tensors, dtypes, classes, chunk_bytes=CHUNK, direct=direct)
    a.replicate_to(peer.port, OPT)
    failed_host = [host_bytes(t) for t in tensors]
    s = a.snapshot(step=7, meta=b"rng")
    a.wait_replicated(s)
    fresh = replacement_like(tensors)
    a.close()  # rank A is gone
    del tensors
    ids, _, _, env = expected_replica(failed_host, dtypes, classes, CHUNK, OPT, 7, b"rng")

    before = [host_bytes(t) for t in fresh]
    b = P.Checkpointer(fresh, dtypes, classes, chunk_bytes=CHUNK, group_bytes=CHUNK, bounce_bytes=bounce,
                       device_staging_bytes=staging, direct=direct)
    sid, step, bad = b.restore_from_peer(peer.port)
    assert (sid, step, bad) == (s, 7, [])
    assert_tensors(fresh, expected_after(failed_host, before, classes, ids))
    info = b.peer_restore_info()
    assert np.array_equal(info["chunk_ids"], ids) and info["envelope"] == env
    # every optimizer-class fragment is whole again; parameters are not touched
    for i, c in enumerate(classes):
        if c != W.CLS_PARAM:
            assert np.array_equal(host_bytes(fresh[i]), failed_host[i])
    # the replacement snapshots and restores as usual afterwards
    s2 = b.snapshot(step=8)
    b.wait_committed(s2)
    garbage_fill(fresh, 0x11)
    assert b.restore(s2) == []
    assert_tensors(fresh, expected_after(failed_host, before, classes, ids))
    b.close()
    peer.close()


def test_fetch_between_two_snapshots_of_a_connected_sender():
    """The peer answers a fetch while the sender stays connected, and keeps
    taking the sender's snapshots afterwards."""
    tensors, dtypes, classes = state()
    peer = P.Peer()
    a = P.Checkpointer(tensors, dtypes, classes, chunk_bytes=CHUNK)
    a.replicate_to(peer.port, OPT)
    host1 = [host_bytes(t) for t in tensors]
    s1 = a.snapshot(step=1)
    a.wait_replicated(s1)
    fresh = replacement_like(tensors)
    before = [host_bytes(t) for t in fresh]
    b = P.Checkpointer(fresh, dtypes, classes, chunk_bytes=CHUNK)
    assert b.restore_from_peer(peer.port) == (s1, 1, [])
    ids = expected_replica(host1, dtypes, classes, CHUNK, OPT, 1)[0]
    assert_tensors(fresh, expected_after(host1, before, classes, ids))
    for t in tensors:
        t.add_(1.0)
    host2 = [host_bytes(t) for t in tensors]
    s2 = a.snapshot(step=2)
    a.wait_replicated(s2)
    assert peer.wait(s2) == P.CKPT_OK
    assert b.restore_from_peer(peer.port) == (s2, 2, [])
    assert_tensors(fresh, expected_after(host2, before, classes, ids))
    a.close()
    b.close()
    peer.close()


def test_corrupt_replica_chunk_is_located():
    """A bit flipped in the peer's committed replica: the replacement's GPU
    check names exactly that chunk; every other chunk is restored."""
    tensors, dtypes, classes = state()
    peer = P.Peer()
    a = P.Checkpointer(tensors, dtypes, classes, chunk_bytes=CHUNK)
    a.replicate_to(peer.port, OPT)
    failed_host = [host_bytes(t) for t in tensors]
    s = a.snapshot(step=3)
    a.wait_replicated(s)
    a.close()
    r = peer.replica()
    j = 2  # third replicated chunk
    r["data"][j * CHUNK + 4321] ^= 0x10
    fresh = replacement_like(tensors)
    before = [host_bytes(t) for t in fresh]
    b = P.Checkpointer(fresh, dtypes, classes, chunk_bytes=CHUNK)
    sid, step, bad = b.restore_from_peer(peer.port)
    ids = r["chunk_ids"]
    assert (sid, step) == (s, 3) and bad == [int(ids[j])]
    # the flipped byte landed; all else is the failed rank's state
    want = expected_after(failed_host, before, classes, ids)
    _, off, _ = O.pack(failed_host, 256, CHUNK)
    x = int(ids[j]) * CHUNK + 4321
    i = max(k for k in range(len(off)) if int(off[k]) <= x)
    if x - int(off[i]) < failed_host[i].size:  # padding is never written back
        want[i][x - int(off[i])] ^= 0x10
    assert_tensors(fresh, want)
    b.close()
    peer.close()


def test_layout_mismatch_and_empty_peer_are_refused():
    tensors, dtypes, classes = state()
    peer = P.Peer()
    fresh = replacement_like(tensors)
    b = P.Checkpointer(fresh, dtypes, classes, chunk_bytes=CHUNK)
    with pytest.raises(P.CkptError) as e:
        b.restore_from_peer(peer.port)  # nothing replicated yet
    assert e.value.code == P.CKPT_ENOSNAP
    a = P.Checkpointer(tensors, dtypes, classes, chunk_bytes=CHUNK)
    a.replicate_to(peer.port, OPT)
    s = a.snapshot(step=5)
    a.wait_replicated(s)
    # one fragment fewer: another layout
    other = replacement_like(tensors[:-1])
    before = [host_bytes(t) for t in other]
    c = P.Checkpointer(other, dtypes[:-1], classes[:-1], chunk_bytes=CHUNK)
    with pytest.raises(P.CkptError) as e:
        c.restore_from_peer(peer.port)
    assert e.value.code == P.CKPT_EINVAL
    assert_tensors(other, before)
    # same sizes, one class tag changed: the envelope differs too
    cls2 = list(classes)
    cls2[-1] = W.CLS_PARAM
    d = P.Checkpointer(other + [replacement_like(tensors[-1:])[0]], dtypes, cls2, chunk_bytes=CHUNK)
    with pytest.raises(P.CkptError) as e:
        d.restore_from_peer(peer.port)
    assert e.value.code == P.CKPT_EINVAL
    assert b.restore_from_peer(peer.port)[:2] == (s, 5)
    for x in (a, b, c, d):
        x.close()
    peer.close()


def test_peer_restore_supersedes_the_older_local_snapshot():
    """The replica lands in the image the next snapshot would fill: the older
    of two committed local snapshots there becomes SUPERSEDED, the newer one
    stays restorable, and snapshots alternate as before."""
    tensors, dtypes, classes = state()
    peer = P.Peer()
    a = P.Checkpointer(tensors, dtypes, classes, chunk_bytes=CHUNK)
    a.replicate_to(peer.port, OPT)
    host_a = [host_bytes(t) for t in tensors]
    sa = a.snapshot(step=9)
    a.wait_replicated(sa)
    fresh = replacement_like(tensors)
    b = P.Checkpointer(fresh, dtypes, classes, chunk_bytes=CHUNK)
    s1 = b.snapshot(step=1)
    b.wait_committed(s1)
    garbage_fill(fresh, 0x77)
    torch.cuda.synchronize()
    host_b2 = [host_bytes(t) for t in fresh]
    s2 = b.snapshot(step=2)
    b.wait_committed(s2)
    assert b.state(s1) == P.CKPT_SNAP_COMMITTED and b.state(s2) == P.CKPT_SNAP_COMMITTED
    assert b.restore_from_peer(peer.port) == (sa, 9, [])
    assert b.state(s1) == P.CKPT_SNAP_SUPERSEDED and b.state(s2) == P.CKPT_SNAP_COMMITTED
    assert b.latest() == (s2, 2)
    ids = expected_replica(host_a, dtypes, classes, CHUNK, OPT, 9)[0]
    assert_tensors(fresh, expected_after(host_a, host_b2, classes, ids))
    assert b.restore(s2) == []
    assert_tensors(fresh, host_b2)
    s3 = b.snapshot(step=3)
    b.wait_committed(s3)
    assert b.state(s2) == P.CKPT_SNAP_COMMITTED and b.state(s3) == P.CKPT_SNAP_COMMITTED
    for x in (a, b):
        x.close()
    peer.close()


def _failed_rank(conn, device, port):
    sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
    sys.path.insert(0, os.path.dirname(os.path.abspath(__file__)))
    import paper_2607_01646_amd as PP
    import workloads as WW
    from gpu_util import class_major as cm, host_bytes as hb

    torch.cuda.set_device(device)
    tensors, plan = WW.make_state(1, device="cuda")
    tensors, dtypes, classes = cm(tensors, plan)
    torch.cuda.synchronize()
    ck = PP.Checkpointer(tensors, dtypes, classes, chunk_bytes=CHUNK)
    ck.replicate_to(port, OPT)
    host = [hb(t) for t in tensors]
    s = ck.snapshot(step=21, meta=b"dp=3")
    ck.wait_replicated(s)
    conn.send((s, dtypes, classes, [h.tobytes() for h in host]))
    conn.recv()
    os._exit(0)  # the rank dies without closing anything


def test_failed_rank_in_another_process():
    """The failed rank is a process that dies after its replica committed;
    the replacement in this process restores from the peer."""
    peer = P.Peer()
    ctx = mp.get_context("spawn")
    a_end, b_end = ctx.Pipe()
    proc = ctx.Process(target=_failed_rank, args=(b_end, torch.cuda.current_device(), peer.port))
    proc.start()
    try:
        s, dtypes, classes, raw = a_end.recv()
        a_end.send("die")
        proc.join(timeout=60)
        assert proc.exitcode == 0
        failed_host = [np.frombuffer(x, dtype=np.uint8).copy() for x in raw]
        fresh = replacement_like(state()[0])
        before = [host_bytes(t) for t in fresh]
        b = P.Checkpointer(fresh, dtypes, classes, chunk_bytes=CHUNK)
        assert b.restore_from_peer(peer.port) == (s, 21, [])
        ids, _, _, env = expected_replica(failed_host, dtypes, classes, CHUNK, OPT, 21, b"dp=3")
        assert_tensors(fresh, expected_after(failed_host, before, classes, ids))
        assert b.peer_restore_info()["envelope"] == env
        b.close()
    finally:
        if proc.is_alive():
            proc.kill()
        peer.close()


def _fake_peer(replies):
    """A listening socket on 127.0.0.1 whose thread answers one fetch with
    the bytes of `replies` (then closes): (port, thread)."""
    import socket
    import threading

    srv = socket.socket()
    srv.bind(("127.0.0.1", 0))
    srv.listen(1)

    def run():
        conn, _ = srv.accept()
        with conn:
            got = b""
            while len(got) < 32:
                got += conn.recv(32 - len(got))
            assert got[:8] == b"CKPTGET1"
            for part in replies:
                conn.sendall(part)
        srv.close()

    th = threading.Thread(target=run, daemon=True)
    th.start()
    return srv.getsockname()[1], th


def _ack(snap):
    """The peer's answer to a fetch (wire format of csrc/ckpt_wire.h):
    magic, snapshot id, status, bad count, reserved."""
    import struct

    return struct.pack("<8sQiIQ", b"CKPTACK1", snap, P.CKPT_OK, 0, 0)


def test_transfer_cut_midway_leaves_the_earlier_chunks_written():
    """A peer that closes the stream inside the fourth replicated chunk: the
    restore fails with EHIP, the three chunks before the cut are written
    (and checked), nothing after them is; the context stays usable."""
    import struct

    tensors, dtypes, classes = state()
    host = [host_bytes(t) for t in tensors]
    ids, data, sums, env = expected_replica(host, dtypes, classes, CHUNK, OPT, 4, b"x")
    I = O.pack(host, 256, CHUNK)[0].size
    ack = _ack(17)
    head = struct.pack("<8s7Q", b"CKPTH2H1", 17, 4, CHUNK, I, len(ids), data.size, len(env))
    cut = 3 * CHUNK + 100
    port, th = _fake_peer([ack, head, ids.tobytes(), sums.tobytes(), env, data[:cut].tobytes()])
    fresh = replacement_like(tensors)
    before = [host_bytes(t) for t in fresh]
    b = P.Checkpointer(fresh, dtypes, classes, chunk_bytes=CHUNK, group_bytes=CHUNK)
    with pytest.raises(P.CkptError) as e:
        b.restore_from_peer(port)
    assert e.value.code == P.CKPT_EHIP
    th.join(timeout=30)
    assert_tensors(fresh, expected_after(host, before, classes, ids[:3]))
    s = b.snapshot(step=1)
    b.wait_committed(s)
    assert b.verify(s) == []
    b.close()


def test_malformed_replies_are_refused_before_anything_is_written():
    import struct

    tensors, dtypes, classes = state()
    host = [host_bytes(t) for t in tensors]
    ids, data, sums, env = expected_replica(host, dtypes, classes, CHUNK, OPT, 4)
    I = O.pack(host, 256, CHUNK)[0].size
    ack = _ack(5)
    head = struct.pack("<8s7Q", b"CKPTH2H1", 5, 4, CHUNK, I, len(ids), data.size, len(env))
    bad_env = bytearray(env)
    bad_env[64] ^= 1  # the envelope's own word-sum no longer holds
    bad_sums = sums.copy()
    bad_sums[1] += np.uint64(1)  # sums that disagree with the envelope
    cases = [
        [b"CKPTNAK1" + ack[8:]],
        [ack, struct.pack("<8s7Q", b"CKPTH2H1", 5, 4, CHUNK * 2, I, len(ids), data.size, len(env))],
        [ack, head, ids[::-1].tobytes(), sums.tobytes(), env],
        [ack, head, ids.tobytes(), sums.tobytes(), bytes(bad_env)],
        [ack, head, ids.tobytes(), bad_sums.tobytes(), env],
        [ack, struct.pack("<8s7Q", b"CKPTH2H1", 5, 5, CHUNK, I, len(ids), data.size, len(env)),
         ids.tobytes(), sums.tobytes(), env],
    ]
    fresh = replacement_like(tensors)
    before = [host_bytes(t) for t in fresh]
    b = P.Checkpointer(fresh, dtypes, classes, chunk_bytes=CHUNK)
    for k, parts in enumerate(cases):
        port, th = _fake_peer(parts)
        with pytest.raises(P.CkptError) as e:
            b.restore_from_peer(port)
        assert e.value.code == P.CKPT_EINVAL, (k, e.value)
        th.join(timeout=30)
    assert_tensors(fresh, before)
    # a well-formed reply from the same kind of peer goes through
    port, th = _fake_peer([ack, head, ids.tobytes(), sums.tobytes(), env, data.tobytes()])
    assert b.restore_from_peer(port) == (5, 4, [])
    th.join(timeout=30)
    assert_tensors(fresh, expected_after(host, before, classes, ids))
    b.close()


def test_owner_and_one_replica_holder_lost_the_other_serves():
    """k = 2: the owner and its first replica holder fail in the same step;
    the replacement restores from the second holder."""
    tensors, dtypes, classes = state()
    peers = [P.Peer(), P.Peer()]
    a = P.Checkpointer(tensors, dtypes, classes, chunk_bytes=CHUNK)
    for p in peers:
        a.replicate_to(p.port, OPT)
    failed_host = [host_bytes(t) for t in tensors]
    s = a.snapshot(step=13, meta=b"two")
    a.wait_replicated(s)
    fresh = replacement_like(tensors)
    a.close()
    peers[0].close()  # the first holder is gone too
    before = [host_bytes(t) for t in fresh]
    b = P.Checkpointer(fresh, dtypes, classes, chunk_bytes=CHUNK)
    with pytest.raises(P.CkptError) as e:
        b.restore_from_peer(peers[0].port)  # nobody listens there any more
    assert e.value.code == P.CKPT_EHIP
    assert b.restore_from_peer(peers[1].port) == (s, 13, [])
    ids, _, _, env = expected_replica(failed_host, dtypes, classes, CHUNK, OPT, 13, b"two")
    assert_tensors(fresh, expected_after(failed_host, before, classes, ids))
    assert b.peer_restore_info()["envelope"] == env
    b.close()
    peers[1].close()
