"""Where each rank's optimizer-state replicas go (paper Sec. V-C, replication
to k distinct data-parallel peers), and what a placement risks.

Every rank of one tensor/pipeline coordinate owns one shard; its replicas go
to k other ranks of the same coordinate.  Without topology information the
peers are the next k ranks of the data-parallel ring.  With a failure-domain
label per rank (the rack, switch or power feed of its node) the k peers are
taken in k distinct domains, none of them the owner's, so a single
infrastructure event removes at most one copy of any shard.

The risk figures are the section's union bounds, evaluated on the actual
placement: a shard is lost in a step only if every node (or every domain)
holding one of its copies fails in that step.
"""


def ring_peers(D, k):
    """Topology-unaware placement: rank r's replicas go to ranks r+1 .. r+k
    (mod D).  Returns a list of D peer lists."""
    if not 0 <= k < D:
        raise ValueError("need 0 <= k < D")
    return [[(r + j) % D for j in range(1, k + 1)] for r in range(D)]


def _interleaved(domains):
    """Ranks ordered so that consecutive ones come from different domains
    where possible: the first rank of every domain, then the second of
    every domain, and so on (domains in order of first appearance)."""
    groups = {}
    for r, d in enumerate(domains):
        groups.setdefault(d, []).append(r)
    cols = list(groups.values())
    order = []
    for i in range(max(len(c) for c in cols)):
        order.extend(c[i] for c in cols if i < len(c))
    return order


def topology_aware_peers(domains, k):
    """Placement over failure domains: domains[r] labels rank r's domain.
    Each rank's k peers lie in k distinct domains other than its own.  The
    ranks are walked along a ring that interleaves the domains, and each
    rank takes the next ranks on that ring whose domains it does not hold
    yet; with domains of equal size every rank then holds exactly k
    replicas.  Raises ValueError with fewer than k + 1 domains."""
    D = len(domains)
    if k < 0 or D == 0:
        raise ValueError("need k >= 0 and at least one rank")
    if len(set(domains)) < k + 1:
        raise ValueError("k = %d needs at least %d failure domains" % (k, k + 1))
    order = _interleaved(domains)
    pos = {r: i for i, r in enumerate(order)}
    out = [None] * D
    for r in range(D):
        used = {domains[r]}
        peers = []
        i = pos[r]
        while len(peers) < k:
            i = (i + 1) % D
            cand = order[i]
            if domains[cand] not in used:
                used.add(domains[cand])
                peers.append(cand)
        out[r] = peers
    return out


def holders(placement):
    """Per rank, the shards whose replicas it holds."""
    held = [[] for _ in placement]
    for r, peers in enumerate(placement):
        for p in peers:
            held[p].append(r)
    return held


def survives(placement, failed):
    """Whether every shard keeps a copy when the ranks in `failed` are lost
    together (owner and every replica holder gone = lost)."""
    failed = set(failed)
    return all(r not in failed or any(p not in failed for p in peers) for r, peers in enumerate(placement))


def node_loss_per_step(placement, p):
    """Union bound over shards for independent node failures with
    probability p per node per step: sum of p ** (copies on distinct nodes)."""
    return sum(p ** (1 + len(set(peers) - {r})) for r, peers in enumerate(placement))


def domain_loss_per_step(placement, domains, q):
    """Union bound over shards when whole failure domains fail, each with
    probability q per step: a shard whose copies sit in m distinct domains
    is lost with probability q ** m."""
    total = 0.0
    for r, peers in enumerate(placement):
        m = len({domains[r]} | {domains[x] for x in peers})
        total += q ** m
    return total
