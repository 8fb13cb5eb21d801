"""Eight ranks of one data-parallel ring on one GPU with k = 2 (Sec. V-C:
each optimizer-state shard goes to two distinct DP peers, so any two
failures in the same step leave a copy of every shard).  Two adjacent ranks
die together; both replacements restore from survivors.  Needs an MI355X.

Each rank is a process with its own shard (the tiny GPT state offset by its
rank), two peers holding its two predecessors' replicas, and streams to its
two successors' peers.  Expected values come from the oracle over states
rebuilt in this process from the same seeded generators.
"""
import multiprocessing as mp
import os
import sys

import numpy as np
import pytest
import torch

import workloads as W
from gpu_util import class_major, expected_after_restore, expected_replica, garbage_fill, host_bytes

pytestmark = pytest.mark.gpu

if torch.cuda.is_available():
    import paper_2607_01646_amd as P

OPT = (1 << W.CLS_MASTER) | (1 << W.CLS_ADAM_M) | (1 << W.CLS_ADAM_V)
CHUNK = 1 << 20
D = 8
K = 2


def rank_state(r):
    tensors, plan = W.make_state(1, device="cuda")
    tensors, dtypes, classes = class_major(tensors, plan)
    for t in tensors:
        t.add_(r)
    torch.cuda.synchronize()
    return tensors, dtypes, classes


def _rank(r, conn, device):
    here = os.path.dirname(os.path.abspath(__file__))
    sys.path.insert(0, os.path.dirname(here))
    sys.path.insert(0, here)
    import paper_2607_01646_amd as PP

    torch.cuda.set_device(device)
    # peer j holds the replica of rank r - 1 - j
    peers = [PP.Peer(device=device) for _ in range(K)]
    conn.send([p.port for p in peers])
    tensors, dtypes, classes = rank_state(r)
    ck = PP.Checkpointer(tensors, dtypes, classes, chunk_bytes=CHUNK)
    for port in conn.recv():
        ck.replicate_to(port, OPT)
    while True:
        cmd = conn.recv()
        if cmd[0] == "snap":
            s = ck.snapshot(step=cmd[1], meta=b"rank%d" % r)
            ck.wait_replicated(s)
            conn.send(s)
        elif cmd[0] == "die":
            os._exit(0)
        else:
            ck.close()
            for p in peers:
                p.close()
            conn.send("closed")
            return


@pytest.mark.timeout(300)
def test_two_adjacent_ranks_lost_in_one_step():
    ctx = mp.get_context("spawn")
    dev = torch.cuda.current_device()
    pipes, procs = [], []
    for r in range(D):
        a, b = ctx.Pipe()
        p = ctx.Process(target=_rank, args=(r, b, dev))
        p.start()
        pipes.append(a)
        procs.append(p)
    try:
        ports = [a.recv() for a in pipes]  # ports[r][j]: rank r's peer for rank r - 1 - j
        for r in range(D):
            # rank r sends to rank r+1+j's peer number j
            pipes[r].send([ports[(r + 1 + j) % D][j] for j in range(K)])
        for a in pipes:
            a.send(("snap", 30))
        snaps = [a.recv() for a in pipes]

        lost = (3, 4)  # two adjacent ranks, in the same step
        for r in lost:
            pipes[r].send(("die",))
        for r in lost:
            procs[r].join(timeout=60)
            assert procs[r].exitcode == 0

        # rank 3's replicas live on ranks 4 (gone) and 5; rank 4's on ranks 5 and 6
        sources = {3: [(4, 0), (5, 1)], 4: [(5, 0), (6, 1)]}
        for r in lost:
            state, dtypes, classes = rank_state(r)
            failed_host = [host_bytes(t) for t in state]
            fresh = [torch.empty_like(t) for t in state]
            garbage_fill(fresh, 0x6D)
            del state
            torch.cuda.synchronize()
            before = [host_bytes(t) for t in fresh]
            ck = P.Checkpointer(fresh, dtypes, classes, chunk_bytes=CHUNK)
            done = False
            for holder, j in sources[r]:
                if holder in lost:
                    with pytest.raises(P.CkptError) as e:  # that node is gone
                        ck.restore_from_peer(ports[holder][j])
                    assert e.value.code == P.CKPT_EHIP
                    continue
                assert ck.restore_from_peer(ports[holder][j]) == (snaps[r], 30, [])
                done = True
                break
            assert done
            ids, _, _, env = expected_replica(failed_host, dtypes, classes, CHUNK, OPT, 30, b"rank%d" % r)
            assert ck.peer_restore_info()["envelope"] == env
            want = expected_after_restore(failed_host, before, ids, CHUNK)
            for i, t in enumerate(fresh):
                assert np.array_equal(host_bytes(t), want[i]), "rank %d fragment %d" % (r, i)
                if classes[i] != W.CLS_PARAM:
                    assert np.array_equal(want[i], failed_host[i])
            ck.close()
            del fresh
            torch.cuda.empty_cache()

        for r in range(D):
            if r not in lost:
                pipes[r].send(("close",))
                assert pipes[r].recv() == "closed"
    finally:
        for p in procs:
            p.join(timeout=60)
            if p.is_alive():
                p.kill()
    assert all(p.exitcode == 0 for p in procs)
