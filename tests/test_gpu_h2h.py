"""Host-to-host replication to a ring peer, against the CPU oracle (needs an
MI355X; sender and peer talk over TCP on 127.0.0.1).

The expected replica is computed from the oracle alone: the chunks that hold
a byte of a fragment of a selected class (oracle locate), their bytes from the
oracle's pack, their sums, and the oracle's envelope of the snapshot.
"""
import multiprocessing as mp
import os
import sys

import numpy as np
import pytest
import torch

import workloads as W
from gpu_util import class_major, expected_replica, host_bytes

pytestmark = pytest.mark.gpu

if torch.cuda.is_available():
    import paper_2607_01646_amd as P

OPT = (1 << W.CLS_MASTER) | (1 << W.CLS_ADAM_M) | (1 << W.CLS_ADAM_V)


def tiny_state():
    tensors, plan = W.make_state(1, device="cuda")
    tensors, dtypes, classes = class_major(tensors, plan)
    torch.cuda.synchronize()
    return tensors, dtypes, classes


@pytest.mark.parametrize("bounce,direct", [(0, False), (2 << 20, False), (0, True), (2 << 20, True)])
def test_replica_of_the_optimizer_state_matches_the_oracle(bounce, direct):
    """Workload 1 registered class-major, 1 MiB chunks: the peer's committed
    replica equals the oracle's chunks, sums and envelope, and leaves out the
    chunks that hold parameters only (also with direct D2H, whose host
    image the replication reads the same way)."""
    tensors, dtypes, classes = tiny_state()
    chunk = 1 << 20
    peer = P.Peer()
    ck = P.Checkpointer(tensors, dtypes, classes, chunk_bytes=chunk, group_bytes=chunk, bounce_bytes=bounce,
                        direct=direct)
    ck.replicate_to(peer.port, OPT)
    host = [host_bytes(t) for t in tensors]
    s = ck.snapshot(step=7, meta=b"rng")
    ck.wait_replicated(s)
    assert peer.wait(s) == P.CKPT_OK
    ids, data, sums, env = expected_replica(host, dtypes, classes, chunk, OPT, 7, b"rng")
    got_ids, nbytes = P.ckpt_replica_chunks(ck.ctx)
    assert np.array_equal(got_ids, ids) and nbytes == data.size
    assert data.size < ck.image_bytes  # parameter-only chunks stay home
    r = peer.replica()
    assert (r["snap_id"], r["step"]) == (s, 7)
    assert np.array_equal(r["chunk_ids"], ids)
    assert np.array_equal(r["data"], data)
    assert np.array_equal(r["sums"], sums)
    assert r["envelope"] == env
    assert ck.replica_result(s) == (P.REPLICA_OK, [])
    ck.close()
    peer.close()


def test_param_major_layout_replicates_every_mixed_chunk():
    """Parameter-major registration interleaves classes: every chunk holding a
    byte of master weights or moments is sent; the replica still matches."""
    tensors, plan = W.make_state(1, device="cuda")
    dtypes, classes = [p[2] for p in plan], [p[3] for p in plan]
    torch.cuda.synchronize()
    chunk = 1 << 20
    peer = P.Peer()
    ck = P.Checkpointer(tensors, dtypes, classes, chunk_bytes=chunk)
    ck.replicate_to(peer.port, OPT)
    host = [host_bytes(t) for t in tensors]
    s = ck.snapshot(step=1)
    ck.wait_replicated(s)
    ids, data, sums, env = expected_replica(host, dtypes, classes, chunk, OPT, 1)
    r = peer.replica()
    assert np.array_equal(r["chunk_ids"], ids) and np.array_equal(r["data"], data)
    assert np.array_equal(r["sums"], sums) and r["envelope"] == env
    ck.close()
    peer.close()


def test_flip_in_transit_is_caught_and_the_previous_replica_stays():
    tensors, dtypes, classes = tiny_state()
    chunk = 1 << 20
    peer = P.Peer()
    ck = P.Checkpointer(tensors, dtypes, classes, chunk_bytes=chunk)
    ck.replicate_to(peer.port, OPT)
    host1 = [host_bytes(t) for t in tensors]
    s1 = ck.snapshot(step=1)
    ck.wait_replicated(s1)
    for t in tensors:
        t.mul_(2)
    ids, _ = P.ckpt_replica_chunks(ck.ctx)
    at = 3 * chunk + 12345  # replica byte in the fourth replicated chunk
    P.ckpt_debug_h2h_fault(ck.ctx, 1, at, 5)
    s2 = ck.snapshot(step=2)
    with pytest.raises(P.CkptError) as e:
        ck.wait_replicated(s2)
    assert e.value.code == P.CKPT_ECORRUPT
    assert ck.replica_result(s2) == (P.REPLICA_CORRUPT, [int(ids[3])])
    assert peer.wait(s2) == P.CKPT_ECORRUPT and peer.last_bad() == [int(ids[3])]
    r = peer.replica()  # still snapshot 1, byte for byte
    want1 = expected_replica(host1, dtypes, classes, chunk, OPT, 1)
    assert r["snap_id"] == s1 and np.array_equal(r["data"], want1[1])
    assert ck.verify(s2) == []  # the local snapshot itself is intact
    host3 = [host_bytes(t) for t in tensors]
    s3 = ck.snapshot(step=3)
    ck.wait_replicated(s3)
    r = peer.replica()
    assert r["snap_id"] == s3 and np.array_equal(r["data"], expected_replica(host3, dtypes, classes, chunk, OPT, 3)[1])
    ck.close()
    peer.close()


def test_cut_stream_keeps_the_previous_replica():
    tensors, dtypes, classes = tiny_state()
    chunk = 1 << 20
    peer = P.Peer()
    ck = P.Checkpointer(tensors, dtypes, classes, chunk_bytes=chunk)
    ck.replicate_to(peer.port, OPT)
    host1 = [host_bytes(t) for t in tensors]
    s1 = ck.snapshot(step=1)
    ck.wait_replicated(s1)
    P.ckpt_debug_h2h_fault(ck.ctx, 2, 5 * chunk + 7)  # stream closed 5 MiB into the replica
    s2 = ck.snapshot(step=2)
    with pytest.raises(P.CkptError) as e:
        ck.wait_replicated(s2)
    assert e.value.code == P.CKPT_EHIP
    assert peer.wait(s2) == P.CKPT_EHIP
    r = peer.replica()
    assert r["snap_id"] == s1 and np.array_equal(r["data"], expected_replica(host1, dtypes, classes, chunk, OPT, 1)[1])
    # the connection is gone: later snapshots still commit locally, replication fails fast
    s3 = ck.snapshot(step=3)
    ck.wait_committed(s3)
    with pytest.raises(P.CkptError) as e:
        ck.wait_replicated(s3)
    assert e.value.code == P.CKPT_EHIP
    ck.close()
    peer.close()


def test_ping_pong_on_the_peer_over_several_snapshots():
    """Four snapshots of changing state, each waited for before the next
    update (the paper's single wait before the optimizer step): the peer's
    replica always equals the newest one."""
    tensors, dtypes, classes = tiny_state()
    chunk = 1 << 20
    peer = P.Peer(group_bytes=4 << 20)
    ck = P.Checkpointer(tensors, dtypes, classes, chunk_bytes=chunk)
    ck.replicate_to(peer.port, OPT)
    for step in range(4):
        host = [host_bytes(t) for t in tensors]
        s = ck.snapshot(step=step)
        ck.wait_replicated(s)
        r = peer.replica()
        want = expected_replica(host, dtypes, classes, chunk, OPT, step)
        assert r["snap_id"] == s and np.array_equal(r["data"], want[1]) and r["envelope"] == want[3]
        for t in tensors:
            t.add_(0.5)
    ck.close()
    peer.close()


def _peer_process(conn, device):
    sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
    import paper_2607_01646_amd as PP

    peer = PP.Peer(device=device)
    conn.send(peer.port)
    snap = conn.recv()
    rc = peer.wait(snap)
    r = peer.replica()
    conn.send((rc, r["snap_id"], r["chunk_ids"].tolist(), r["sums"].tolist(), bytes(r["data"]), r["envelope"]))
    conn.recv()
    peer.close()


def test_peer_in_another_process():
    """The ring peer as its own process (its own HIP context on the same GPU)."""
    tensors, dtypes, classes = tiny_state()
    chunk = 1 << 20
    ctx = mp.get_context("spawn")
    a, b = ctx.Pipe()
    proc = ctx.Process(target=_peer_process, args=(b, torch.cuda.current_device()))
    proc.start()
    try:
        port = a.recv()
        ck = P.Checkpointer(tensors, dtypes, classes, chunk_bytes=chunk)
        ck.replicate_to(port, OPT)
        host = [host_bytes(t) for t in tensors]
        s = ck.snapshot(step=11)
        a.send(s)
        ck.wait_replicated(s)
        rc, sid, ids, sums, data, env = a.recv()
        want = expected_replica(host, dtypes, classes, chunk, OPT, 11)
        assert rc == P.CKPT_OK and sid == s
        assert ids == want[0].tolist() and sums == want[2].tolist()
        assert np.array_equal(np.frombuffer(data, dtype=np.uint8), want[1]) and env == want[3]
        a.send("done")
        ck.close()
    finally:
        proc.join(timeout=60)
        if proc.is_alive():
            proc.kill()
    assert proc.exitcode == 0


def test_replication_errors():
    tensors, dtypes, classes = tiny_state()
    ck = P.Checkpointer(tensors, dtypes, classes, chunk_bytes=1 << 20)
    with pytest.raises(P.CkptError) as e:
        ck.wait_replicated(1)
    assert e.value.code == P.CKPT_ESTATE
    with pytest.raises(P.CkptError) as e:
        ck.replicate_to(1, 1 << 9)  # no fragment has class 9
    assert e.value.code == P.CKPT_EINVAL
    with pytest.raises(P.CkptError) as e:
        ck.replicate_to(1, OPT)  # nothing listens on port 1
    assert e.value.code == P.CKPT_EHIP
    ck.close()


def test_two_peers_hold_the_same_replica_and_fail_separately():
    """k = 2 (Sec. V-C): both peers commit the oracle's replica; a bit flipped
    on the way to the first peer only is reported by that peer, the second
    commits, and the combined result lists the chunk."""
    tensors, dtypes, classes = tiny_state()
    chunk = 1 << 20
    peers = [P.Peer(), P.Peer()]
    ck = P.Checkpointer(tensors, dtypes, classes, chunk_bytes=chunk)
    for p in peers:
        ck.replicate_to(p.port, OPT)
    assert P.ckpt_replica_peers(ck.ctx) == 2
    host1 = [host_bytes(t) for t in tensors]
    s1 = ck.snapshot(step=4, meta=b"k2")
    ck.wait_replicated(s1)
    want1 = expected_replica(host1, dtypes, classes, chunk, OPT, 4, b"k2")
    for k, p in enumerate(peers):
        r = p.replica()
        assert r["snap_id"] == s1 and np.array_equal(r["data"], want1[1]) and r["envelope"] == want1[3]
        assert np.array_equal(r["sums"], want1[2])
        assert ck.replica_peer_result(k, s1) == (P.REPLICA_OK, [])
    for t in tensors:
        t.mul_(3)
    host2 = [host_bytes(t) for t in tensors]
    ids = want1[0]
    P.ckpt_debug_h2h_fault_peer(ck.ctx, 0, 1, 5 * chunk + 99, 2)
    s2 = ck.snapshot(step=5)
    with pytest.raises(P.CkptError) as e:
        ck.wait_replicated(s2)
    assert e.value.code == P.CKPT_ECORRUPT
    assert ck.replica_peer_result(0, s2) == (P.REPLICA_CORRUPT, [int(ids[5])])
    assert ck.replica_peer_result(1, s2) == (P.REPLICA_OK, [])
    assert ck.replica_result(s2) == (P.REPLICA_CORRUPT, [int(ids[5])])
    assert peers[0].replica()["snap_id"] == s1  # kept its previous replica
    r = peers[1].replica()
    assert r["snap_id"] == s2 and np.array_equal(r["data"], expected_replica(host2, dtypes, classes, chunk, OPT, 5)[1])
    ck.close()
    for p in peers:
        p.close()


def test_peer_added_later_and_removed():
    tensors, dtypes, classes = tiny_state()
    chunk = 1 << 20
    a, b = P.Peer(), P.Peer()
    ck = P.Checkpointer(tensors, dtypes, classes, chunk_bytes=chunk)
    ck.replicate_to(a.port, OPT)
    s1 = ck.snapshot(step=1)
    ck.wait_replicated(s1)
    ck.replicate_to(b.port, OPT)
    with pytest.raises(P.PeerError):
        b.replica()  # nothing yet
    host2 = [host_bytes(t) for t in tensors]
    s2 = ck.snapshot(step=2)
    ck.wait_replicated(s2)
    ck.wait_replicated(s1)  # s1 went to the first peer only, and still counts as replicated
    assert ck.replica_result(s1) == (P.REPLICA_OK, [])
    want = expected_replica(host2, dtypes, classes, chunk, OPT, 2)
    for p in (a, b):
        assert p.replica()["snap_id"] == s2 and np.array_equal(p.replica()["data"], want[1])
    with pytest.raises(P.CkptError) as e:
        ck.replica_peer_result(1, s1)
    assert e.value.code == P.CKPT_ERANGE
    # dropping the first peer: s1 went to it alone and no longer counts as replicated
    ck.replicate_remove(0)
    assert P.ckpt_replica_peers(ck.ctx) == 1
    with pytest.raises(P.CkptError) as e:
        ck.wait_replicated(s1)
    assert e.value.code == P.CKPT_ERANGE
    ck.wait_replicated(s2)
    s3 = ck.snapshot(step=3)
    ck.wait_replicated(s3)
    assert b.replica()["snap_id"] == s3 and a.replica()["snap_id"] == s2
    with pytest.raises(P.CkptError) as e:
        ck.replicate_remove(1)
    assert e.value.code == P.CKPT_ESTATE
    ck.close()
    a.close()
    b.close()


def test_peer_list_errors():
    tensors, dtypes, classes = tiny_state()
    peers = [P.Peer() for _ in range(9)]
    ck = P.Checkpointer(tensors, dtypes, classes, chunk_bytes=1 << 20)
    ck.replicate_to(peers[0].port, OPT)
    with pytest.raises(P.CkptError) as e:
        ck.replicate_to(peers[1].port, 1 << W.CLS_MASTER)  # another class mask
    assert e.value.code == P.CKPT_EINVAL
    for p in peers[1:8]:
        ck.replicate_to(p.port, OPT)
    assert P.ckpt_replica_peers(ck.ctx) == 8
    with pytest.raises(P.CkptError) as e:
        ck.replicate_to(peers[8].port, OPT)  # a ninth
    assert e.value.code == P.CKPT_EINVAL
    with pytest.raises(P.CkptError) as e:
        ck.replica_peer_result(8, 1)
    assert e.value.code == P.CKPT_ESTATE
    s = ck.snapshot(step=1)
    ck.wait_replicated(s)
    assert all(p.wait(s) == P.CKPT_OK for p in peers[:8])
    ck.close()
    for p in peers:
        p.close()


def test_sender_idle_after_connecting_keeps_its_connection():
    """A sender may connect long before its first snapshot; meanwhile the peer
    answers a fetch on another connection (regression: the peer used to drop
    a connection that sent nothing for 10 s)."""
    import time

    tensors, dtypes, classes = tiny_state()
    peer = P.Peer()
    ck = P.Checkpointer(tensors, dtypes, classes, chunk_bytes=1 << 20)
    ck.replicate_to(peer.port, OPT)
    other = P.Checkpointer([torch.empty_like(t) for t in tensors], dtypes, classes, chunk_bytes=1 << 20)
    with pytest.raises(P.CkptError) as e:
        other.restore_from_peer(peer.port)  # answered while the sender is still silent
    assert e.value.code == P.CKPT_ENOSNAP
    time.sleep(11)
    host = [host_bytes(t) for t in tensors]
    s = ck.snapshot(step=1)
    ck.wait_replicated(s)
    assert np.array_equal(peer.replica()["data"], expected_replica(host, dtypes, classes, 1 << 20, OPT, 1)[1])
    other.close()
    ck.close()
    peer.close()


def _raw_stream(port, data):
    import socket

    s = socket.create_connection(("127.0.0.1", port))
    s.sendall(data)
    return s


def _await_error(peer, text, timeout=30.0):
    import time

    end = time.time() + timeout
    while time.time() < end:
        if text in peer.last_error():
            return
        time.sleep(0.05)
    raise AssertionError("peer error %r, expected %r" % (peer.last_error(), text))


def test_malformed_sender_streams_are_dropped_and_the_peer_keeps_serving():
    """Streams no sender writes are refused before the peer allocates anything
    for them, and a real sender is served afterwards (regression: a header
    claiming 2^32 chunks made the peer allocate room for their ids up front)."""
    import struct

    C = 1 << 20

    def head(snap, chunk, image, m, replica, env_len=0):
        return struct.pack("<8s7Q", b"CKPTH2H1", snap, 1, chunk, image, m, replica, env_len)

    def ids(*k):
        return np.array(k, dtype=np.uint64).tobytes()

    peer = P.Peer()
    # 2^32 chunks of 256 bytes in a 1 TiB image: consistent, but the ids never come
    s = _raw_stream(peer.port, head(1, 256, 1 << 40, 1 << 32, 1 << 40))
    s.close()
    assert peer.wait(1, 30_000) == P.CKPT_EHIP
    cases = [
        (head(2, 100, 4 * C, 2, 2 * C), None, "malformed replica header"),  # chunk not a multiple of 256
        (head(3, C, 4 * C, 2, 2 * C) + ids(1, 0), P.CKPT_EINVAL, "malformed replica chunk list"),  # out of order
        (head(4, C, 4 * C, 5, 5 * C), None, "malformed replica header"),  # more chunks than the image has
        (head(5, C, 4 * C, 2, 2 * C) + ids(3, 4), P.CKPT_EINVAL, "malformed replica chunk list"),  # beyond the image
        (head(6, C, 4 * C, 2, 2 * C - 256) + ids(0, 1), P.CKPT_EINVAL, "malformed replica size"),
        (head(7, C, 1 << 50, 2, 2 * C), None, "malformed replica header"),  # image above 2^48 bytes
    ]
    for data, result, text in cases:
        s = _raw_stream(peer.port, data)
        if result is not None:
            snap = struct.unpack_from("<Q", data, 8)[0]
            assert peer.wait(snap, 30_000) == result
        _await_error(peer, text)
        s.close()
    with pytest.raises(P.PeerError) as e:
        peer.replica()
    assert e.value.code == P.CKPT_ENOSNAP

    tensors, dtypes, classes = tiny_state()
    ck = P.Checkpointer(tensors, dtypes, classes, chunk_bytes=C)
    ck.replicate_to(peer.port, OPT)
    host = [host_bytes(t) for t in tensors]
    s = ck.snapshot(step=9, meta=b"after")
    ck.wait_replicated(s)
    ids_want, data_want, _, env_want = expected_replica(host, dtypes, classes, C, OPT, 9, b"after")
    rep = peer.replica()
    assert (rep["snap_id"], rep["step"]) == (s, 9)
    assert np.array_equal(rep["chunk_ids"], ids_want) and np.array_equal(rep["data"], data_want)
    assert rep["envelope"] == env_want
    ck.close()
    peer.close()
