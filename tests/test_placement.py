"""Replica placement for k peers (Sec. V-C) against the paper's printed loss
bounds, and its survival properties checked by brute force (CPU only)."""
import itertools
import math

import pytest

from paper_2607_01646_amd import disruption as M
from paper_2607_01646_amd import placement as PL

D = 128


def racks(D, per):
    """Contiguous ranks share a rack: ranks 0..per-1 in rack 0, and so on."""
    return [r // per for r in range(D)]


def test_ring_placement_reproduces_the_independent_failure_bounds():
    # D = 128 shards, p = 1e-6 per node per step: 1.28e-10 (k=1); over 1e5 steps 1.28e-5 (k=1), 1.28e-11 (k=2)
    for k, per_step, run in ((1, 1.28e-10, 1.28e-5), (2, 1.28e-16, 1.28e-11)):
        pl = PL.ring_peers(D, k)
        assert math.isclose(PL.node_loss_per_step(pl, 1e-6), per_step, rel_tol=1e-9)
        assert math.isclose(PL.node_loss_per_step(pl, 1e-6) * 1e5, run, rel_tol=1e-9)
        assert math.isclose(PL.node_loss_per_step(pl, 1e-6), M.shard_loss_per_step(D, 1e-6, k), rel_tol=1e-12)


def test_topology_aware_placement_reproduces_the_domain_bounds():
    # q = 1e-4 per domain per step, replicas in distinct domains: 0.128 (k=1) and 1.28e-5 (k=2) over 1e5 steps
    dom = racks(D, 4)
    for k, run in ((1, 0.128), (2, 1.28e-5)):
        pl = PL.topology_aware_peers(dom, k)
        assert math.isclose(PL.domain_loss_per_step(pl, dom, 1e-4) * 1e5, run, rel_tol=1e-9)
        assert math.isclose(PL.domain_loss_per_step(pl, dom, 1e-4), M.shard_loss_per_step(D, 1e-4, k), rel_tol=1e-12)


def test_topology_unaware_ring_shares_domains():
    """The ring's next rank usually sits in the owner's rack: most shards have
    a single domain holding both copies, so a rack failure can take both."""
    dom = racks(D, 4)
    pl = PL.ring_peers(D, 1)
    same = sum(dom[r] == dom[p[0]] for r, p in enumerate(pl))
    assert same == 96  # 3 of every 4 ranks
    q = 1e-4
    assert math.isclose(PL.domain_loss_per_step(pl, dom, q), 96 * q + 32 * q * q, rel_tol=1e-12)
    assert PL.domain_loss_per_step(pl, dom, q) > 700 * PL.domain_loss_per_step(PL.topology_aware_peers(dom, 1), dom, q)
    lost = [d for d in range(32) if not PL.survives(pl, [r for r in range(D) if dom[r] == d])]
    assert lost == list(range(32))  # every rack failure loses a shard


@pytest.mark.parametrize("per, k", [(4, 1), (4, 2), (8, 3), (16, 1), (1, 2)])
def test_topology_aware_structure(per, k):
    dom = racks(D, per)
    pl = PL.topology_aware_peers(dom, k)
    for r, peers in enumerate(pl):
        assert len(peers) == k and r not in peers and len(set(peers)) == k
        doms = [dom[r]] + [dom[p] for p in peers]
        assert len(set(doms)) == k + 1  # k + 1 distinct domains hold the copies
    # equal domains: every rank holds exactly k replicas
    assert all(len(h) == k for h in PL.holders(pl))


def test_topology_aware_survives_any_k_domain_failures_brute_force():
    dom = racks(32, 4)  # 8 racks
    for k in (1, 2):
        pl = PL.topology_aware_peers(dom, k)
        for failed in itertools.combinations(range(8), k):
            ranks = [r for r in range(32) if dom[r] in failed]
            assert PL.survives(pl, ranks), failed
        # k + 1 racks can take every copy of some shard
        assert any(not PL.survives(pl, [r for r in range(32) if dom[r] in f]) for f in itertools.combinations(range(8), k + 1))


def test_ring_survives_any_k_node_failures_brute_force():
    n = 12
    for k in (1, 2, 3):
        pl = PL.ring_peers(n, k)
        for failed in itertools.combinations(range(n), k):
            assert PL.survives(pl, failed)
        assert not PL.survives(pl, range(k + 1))  # owner 0 and its k peers


def test_uneven_domains_and_errors():
    dom = ["a"] * 5 + ["b"] * 3 + ["c"] * 2
    pl = PL.topology_aware_peers(dom, 2)
    for r, peers in enumerate(pl):
        assert len({dom[r]} | {dom[p] for p in peers}) == 3
    with pytest.raises(ValueError):
        PL.topology_aware_peers(["a", "a", "b"], 2)  # needs 3 domains
    with pytest.raises(ValueError):
        PL.ring_peers(4, 4)
    assert PL.ring_peers(3, 0) == [[], [], []]
    assert PL.node_loss_per_step(PL.ring_peers(3, 0), 0.5) == 1.5
