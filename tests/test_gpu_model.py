"""A seeded random walk over the library's operations, checked against a
model of the ping-pong images (needs an MI355X).

Operations: change the tensors, snapshot and commit, snapshot with the
offload cut after a random number of groups (invariant I4: never committed),
restore the newest or the older held snapshot, verify, and flip a bit in a
committed host image.  The model holds, per host image, which snapshot it
keeps and the tensor bytes of that snapshot; a snapshot goes to the image
that does not hold the newest committed one (Sec. VI-A).  After every
operation the library's snapshot states and newest snapshot must match the
model; every restore must give back the model's bytes; every committed image
must equal the oracle's pack of those bytes, with the oracle's sums.
"""
import numpy as np
import pytest
import torch

import oracle as O
import workloads as W
from gpu_util import garbage_fill, host_bytes

pytestmark = pytest.mark.gpu

if torch.cuda.is_available():
    import paper_2607_01646_amd as P

CHUNK = 1 << 20
GROUP = 2 << 20


class Image:
    def __init__(self, snap, step, data):
        self.snap, self.step, self.data = snap, step, data  # data None: interrupted


@pytest.mark.parametrize("bounce, staging, file, threads, direct", [
    (0, 0, False, 0, False), (4 << 20, 0, False, 0, False), (0, 3 * GROUP, False, 0, False),
    (4 << 20, 3 * GROUP, False, 0, False), (4 << 20, 0, True, 0, False),
    (4 << 20, 3 * GROUP, False, 1, False),  # one host copy thread: the drainer lags far behind the engines
    (0, 0, False, 0, True), (4 << 20, 0, False, 0, True), (4 << 20, 0, True, 0, True),  # direct D2H
    (4 << 20, 0, False, 1, True),
])
def test_random_walk_against_the_ping_pong_model(bounce, staging, file, threads, direct, tmp_path):
    rng = np.random.default_rng(1234 + bounce + staging + file + threads + 7 * direct)
    tensors, plan = W.make_state(1, device="cuda")
    tensors, plan = tensors[:72], plan[:72]  # the first 18 parameter tensors with their optimizer state
    torch.cuda.synchronize()
    sizes = [p[1] for p in plan]
    ck = P.Checkpointer(tensors, [p[2] for p in plan], [p[3] for p in plan], chunk_bytes=CHUNK, group_bytes=GROUP,
                        bounce_bytes=bounce, device_staging_bytes=staging, host_threads=threads,
                        image_file=str(tmp_path / "images") if file else None, direct=direct)
    _, I, nc = O.layout(sizes, 256, CHUNK)
    n_groups = -(-I // GROUP)
    hold = [None, None]
    newest = None  # index of the image holding the newest committed snapshot
    seen = {}      # snap id -> (image index, committed?)
    step = 0

    def current():
        torch.cuda.synchronize()
        return [host_bytes(t) for t in tensors]

    def target():
        if newest is not None:
            return 1 - newest
        for b in (0, 1):
            if hold[b] is None or hold[b].data is None:
                return b
        raise AssertionError("unreachable")

    def check_states():
        for sid, (b, committed) in seen.items():
            try:
                st = ck.state(sid)
            except P.CkptError as e:  # old records may be dropped
                assert e.code == P.CKPT_ERANGE
                continue
            if not committed:
                assert st == P.CKPT_SNAP_ABORTED, (sid, st)
            elif hold[b] is not None and hold[b].snap == sid:
                assert st == P.CKPT_SNAP_COMMITTED, (sid, st)
            else:
                assert st == P.CKPT_SNAP_SUPERSEDED, (sid, st)
        if newest is None:
            assert ck.latest()[0] == 0
        else:
            assert ck.latest() == (hold[newest].snap, hold[newest].step)

    def assert_tensors(data):
        torch.cuda.synchronize()
        for i, (t, d) in enumerate(zip(tensors, data)):
            assert np.array_equal(host_bytes(t), d), "fragment %d" % i

    ops = ["mutate", "commit", "commit", "abort", "restore", "restore_older", "verify", "flip"]
    if file:
        ops.append("reopen")
    done = {op: 0 for op in ops}
    for it in range(120):
        op = ops[int(rng.integers(0, len(ops)))]
        done[op] += 1
        if op == "mutate":
            for i in rng.choice(len(tensors), size=8, replace=False):
                t = tensors[int(i)]
                if rng.random() < 0.5:
                    t.add_(float(rng.integers(1, 9)))
                else:
                    u = t.view(-1).view(torch.uint8)
                    u.copy_(torch.randint(0, 256, u.shape, dtype=torch.uint8, device=u.device))
        elif op == "commit":
            step += 1
            data = current()
            b = target()
            s = ck.snapshot(step=step, meta=b"walk %d" % it)
            ck.wait_committed(s)
            hold[b] = Image(s, step, data)
            newest = b
            seen[s] = (b, True)
            img, sums = ck.host_image(s)
            want, _, _ = O.pack(data, 256, CHUNK)
            assert np.array_equal(img, want), "image of snapshot %d" % s
            assert np.array_equal(sums, O.chunk_sums(want, 0, I, CHUNK))
        elif op == "abort":
            step += 1
            b = target()
            P.ckpt_debug_interrupt_next(ck.ctx, int(rng.integers(0, n_groups)))
            s = ck.snapshot(step=step)
            torch.cuda.synchronize()
            assert ck.state(s) == P.CKPT_SNAP_ABORTED
            hold[b] = Image(s, step, None)
            seen[s] = (b, False)
        elif op == "restore":
            garbage_fill(tensors, int(rng.integers(0, 256)))
            if newest is None:
                with pytest.raises(P.CkptError) as e:
                    ck.restore(0)
                assert e.value.code == P.CKPT_ENOSNAP
                continue
            assert ck.restore(0) == []
            assert_tensors(hold[newest].data)
        elif op == "restore_older":
            older = None if newest is None else hold[1 - newest]
            if older is None or older.data is None:
                continue
            garbage_fill(tensors, 0x42)
            assert ck.restore(older.snap) == []
            assert_tensors(older.data)
        elif op == "verify":
            for img in hold:
                if img is not None and img.data is not None:
                    assert ck.verify(img.snap) == []
        elif op == "reopen":  # a restarted process adopts the image file: the newest committed snapshot survives
            ck.close()
            ck = P.Checkpointer(tensors, [p[2] for p in plan], [p[3] for p in plan], chunk_bytes=CHUNK,
                                group_bytes=GROUP, bounce_bytes=bounce, device_staging_bytes=staging,
                                host_threads=threads, image_file=str(tmp_path / "images"),
                                image_file_mode=P.CKPT_FILE_ADOPT, direct=direct)
            seen = {}
            if newest is None:
                hold = [None, None]
            else:
                sid, st = ck.latest()
                assert st == hold[newest].step
                kept = Image(sid, st, hold[newest].data)
                hold = [None, None]
                hold[newest] = kept
                seen[sid] = (newest, True)
        elif op == "flip":
            if newest is None:
                continue
            s = hold[newest].snap
            img, _ = ck.host_image(s)
            x = int(rng.integers(0, I))
            bit = 1 << int(rng.integers(0, 8))
            img[x] ^= bit
            assert ck.verify(s) == [x // CHUNK]
            img[x] ^= bit
            assert ck.verify(s) == []
        check_states()
    assert min(done.values()) >= 5, done  # every kind of operation ran several times
    ck.close()


def test_random_walk_with_a_peer():
    """The same walk with replication to a peer: every committed snapshot is
    replicated and waited for; some streams carry a flipped bit (the peer
    rejects them and keeps its previous replica); a replacement context
    restores from the peer now and then and must get exactly the replica the
    model says the peer holds."""
    from gpu_util import class_major, expected_after_restore

    opt = (1 << W.CLS_MASTER) | (1 << W.CLS_ADAM_M) | (1 << W.CLS_ADAM_V)
    rng = np.random.default_rng(99)
    full, plan = W.make_state(1, device="cuda")
    tensors, dtypes, classes = class_major(full[:72], plan[:72])
    del full
    torch.cuda.synchronize()
    sizes = [int(t.numel() * t.element_size()) for t in tensors]
    _, I, nc = O.layout(sizes, 256, CHUNK)
    peer = P.Peer()
    ck = P.Checkpointer(tensors, dtypes, classes, chunk_bytes=CHUNK, group_bytes=GROUP)
    ck.replicate_to(peer.port, opt)
    ids, rbytes = P.ckpt_replica_chunks(ck.ctx)
    fresh = [torch.empty_like(t) for t in tensors]
    rk = P.Checkpointer(fresh, dtypes, classes, chunk_bytes=CHUNK, group_bytes=GROUP)
    peer_state = None  # (snap, step, tensor bytes) of the peer's committed replica
    step = 0
    ops = ["mutate", "replicate", "replicate", "replicate_flip", "abort", "fetch"]
    done = {op: 0 for op in ops}
    for it in range(60):
        op = ops[int(rng.integers(0, len(ops)))]
        done[op] += 1
        if op == "mutate":
            for i in rng.choice(len(tensors), size=6, replace=False):
                tensors[int(i)].add_(float(rng.integers(1, 9)))
        elif op in ("replicate", "replicate_flip"):
            step += 1
            torch.cuda.synchronize()
            data = [host_bytes(t) for t in tensors]
            if op == "replicate_flip":
                at = int(rng.integers(0, rbytes))
                P.ckpt_debug_h2h_fault(ck.ctx, 1, at, int(rng.integers(0, 8)))
            s = ck.snapshot(step=step)
            ck.wait_committed(s)
            if op == "replicate":
                ck.wait_replicated(s)
                peer_state = (s, step, data)
            else:
                with pytest.raises(P.CkptError) as e:
                    ck.wait_replicated(s)
                assert e.value.code == P.CKPT_ECORRUPT
                assert ck.replica_result(s) == (P.REPLICA_CORRUPT, [int(ids[at // CHUNK])])
        elif op == "abort":
            step += 1
            P.ckpt_debug_interrupt_next(ck.ctx, int(rng.integers(0, -(-I // GROUP))))
            ck.snapshot(step=step)
            torch.cuda.synchronize()
        elif op == "fetch":
            garbage_fill(fresh, int(rng.integers(0, 256)))
            torch.cuda.synchronize()
            before = [host_bytes(t) for t in fresh]
            if peer_state is None:
                with pytest.raises(P.CkptError) as e:
                    rk.restore_from_peer(peer.port)
                assert e.value.code == P.CKPT_ENOSNAP
                continue
            s, st, data = peer_state
            assert rk.restore_from_peer(peer.port) == (s, st, [])
            want = expected_after_restore(data, before, ids, CHUNK)
            torch.cuda.synchronize()
            for i, t in enumerate(fresh):
                assert np.array_equal(host_bytes(t), want[i]), "fragment %d" % i
        if peer_state is not None:
            r = peer.replica()
            assert (r["snap_id"], r["step"]) == peer_state[:2]
    assert min(done.values()) >= 4, done
    rk.close()
    ck.close()
    peer.close()


def test_random_walk_with_changing_peers():
    """Peers join and leave (1 to 3 at a time, Sec. V-C k-peer replication and
    ring repair); a flipped bit goes to one chosen peer only; fetches go to a
    random live peer.  The model keeps each peer's committed replica: a peer
    takes only snapshots issued after it joined, and keeps its previous
    replica when it rejects one."""
    from gpu_util import class_major, expected_after_restore

    opt = (1 << W.CLS_MASTER) | (1 << W.CLS_ADAM_M) | (1 << W.CLS_ADAM_V)
    rng = np.random.default_rng(7)
    full, plan = W.make_state(1, device="cuda")
    tensors, dtypes, classes = class_major(full[:72], plan[:72])
    del full
    torch.cuda.synchronize()
    ck = P.Checkpointer(tensors, dtypes, classes, chunk_bytes=CHUNK, group_bytes=GROUP)
    fresh = [torch.empty_like(t) for t in tensors]
    rk = P.Checkpointer(fresh, dtypes, classes, chunk_bytes=CHUNK, group_bytes=GROUP)
    peers = []  # [Peer, committed replica (snap, step, bytes) or None], in the order added
    retired = []
    ids = rbytes = None
    step = 0

    def add_peer():
        nonlocal ids, rbytes
        p = P.Peer()
        ck.replicate_to(p.port, opt)
        peers.append([p, None])
        ids, rbytes = P.ckpt_replica_chunks(ck.ctx)

    add_peer()
    ops = ["mutate", "snap", "snap", "snap_flip", "add", "remove", "fetch"]
    done = {op: 0 for op in ops}
    for it in range(80):
        op = ops[int(rng.integers(0, len(ops)))]
        if op == "add" and len(peers) >= 3 or op == "remove" and len(peers) <= 1:
            continue
        done[op] += 1
        if op == "mutate":
            for i in rng.choice(len(tensors), size=6, replace=False):
                tensors[int(i)].add_(float(rng.integers(1, 9)))
        elif op == "add":
            add_peer()
        elif op == "remove":
            j = int(rng.integers(0, len(peers)))
            ck.replicate_remove(j)
            retired.append(peers.pop(j)[0])  # its node stays up; it just leaves the ring
            assert P.ckpt_replica_peers(ck.ctx) == len(peers)
        elif op in ("snap", "snap_flip"):
            step += 1
            torch.cuda.synchronize()
            data = [host_bytes(t) for t in tensors]
            bad_peer = None
            if op == "snap_flip":
                bad_peer = int(rng.integers(0, len(peers)))
                at = int(rng.integers(0, rbytes))
                P.ckpt_debug_h2h_fault_peer(ck.ctx, bad_peer, 1, at, int(rng.integers(0, 8)))
            s = ck.snapshot(step=step)
            if bad_peer is None:
                ck.wait_replicated(s)
            else:
                with pytest.raises(P.CkptError) as e:
                    ck.wait_replicated(s)
                assert e.value.code == P.CKPT_ECORRUPT
                assert ck.replica_result(s) == (P.REPLICA_CORRUPT, [int(ids[at // CHUNK])])
            for j, entry in enumerate(peers):
                want_state = P.REPLICA_CORRUPT if j == bad_peer else P.REPLICA_OK
                assert ck.replica_peer_result(j, s)[0] == want_state
                if j != bad_peer:
                    entry[1] = (s, step, data)
        elif op == "fetch":
            j = int(rng.integers(0, len(peers)))
            p, rep = peers[j]
            garbage_fill(fresh, int(rng.integers(0, 256)))
            torch.cuda.synchronize()
            before = [host_bytes(t) for t in fresh]
            if rep is None:
                with pytest.raises(P.CkptError) as e:
                    rk.restore_from_peer(p.port)
                assert e.value.code == P.CKPT_ENOSNAP
                continue
            assert rk.restore_from_peer(p.port) == (rep[0], rep[1], [])
            want = expected_after_restore(rep[2], before, ids, CHUNK)
            torch.cuda.synchronize()
            for i, t in enumerate(fresh):
                assert np.array_equal(host_bytes(t), want[i]), "fragment %d" % i
        for p, rep in peers:
            if rep is not None:
                r = p.replica()
                assert (r["snap_id"], r["step"]) == rep[:2]
    assert min(done.values()) >= 4, done
    rk.close()
    ck.close()
    for p, _ in peers:
        p.close()
    for p in retired:
        p.close()
