"""The paper's analytic disruption and shard-loss models (Sec. IV, Sec. V-C),
as a calculator for sizing checkpoint intervals and replication degree.

Sec. IV: per-failure disruption of checkpoint-restart is overhead + restart
time + replayed steps x step time; with a uniform failure position the
expected replay is about half an interval; training efficiency alternates
failure-free stretches of MTTF with disruption intervals.  The in-memory
scheme replaces restart with hot-swap and bounds replay by the interrupted
step (fraction phi).

Sec. V-C: a shard is lost only if its owner and all k replica holders fail
in the same step; a union bound over D data-parallel shards gives the loss
probability per step (independent node failures, probability p each) or
(replicas in distinct failure domains, probability q each) D * q^(k+1).
"""


def expected_replay_steps(K, worked_example=False):
    """Expected steps since the last checkpoint under uniform failures: the
    model states (K - 1) / 2; the worked example of Sec. IV computes K / 2
    (100 steps of 20 s -> 16.7 min), which `worked_example` reproduces."""
    return K / 2.0 if worked_example else (K - 1) / 2.0


def expected_replay_steps_empirical(dist):
    """E[R] = sum r * Pr(R = r) for an empirical replay distribution given as
    {r: probability} (probabilities summing to 1)."""
    total = sum(dist.values())
    if abs(total - 1.0) > 1e-9:
        raise ValueError("probabilities sum to %r, not 1" % total)
    return sum(r * p for r, p in dist.items())


def disruption_checkpoint_restart(overhead_s, restart_s, step_s, replay_steps):
    """E[C_ckpt] = C_overhead + E[T_restart] + t_step * E[R] (seconds)."""
    return overhead_s + restart_s + step_s * replay_steps


def disruption_in_memory(overhead_s, hotswap_s, step_s, phi):
    """E[C] of the in-memory scheme = C_overhead + E[T_hotswap] + t_step * E[phi],
    phi in [0, 1) the fraction of the interrupted step."""
    if not 0.0 <= phi < 1.0:
        raise ValueError("phi must lie in [0, 1)")
    return overhead_s + hotswap_s + step_s * phi


def disruption_rate(mttf_s, disruption_s):
    """E[C_rate] = lambda * E[C], lambda = 1 / MTTF_sys (seconds of disruption per second)."""
    return disruption_s / mttf_s


def efficiency(mttf_s, disruption_s):
    """eta ~= MTTF / (MTTF + E[C])."""
    return mttf_s / (mttf_s + disruption_s)


def per_node_step_failure(mttf_sys_s, step_s, nodes):
    """Per-node per-step failure probability from a system MTTF: the
    system fails in a step with probability about t_step / MTTF, spread over
    `nodes` nodes."""
    return step_s / mttf_sys_s / nodes


def shard_loss_per_step(D, prob, k):
    """Union bound on the per-step probability that some shard loses its
    owner and all k replicas: D * prob^(k+1) (prob = p for independent nodes,
    q for replicas in distinct failure domains)."""
    if k < 0 or D < 0 or not 0.0 <= prob <= 1.0:
        raise ValueError("need D >= 0, k >= 0 and prob in [0, 1]")
    return D * prob ** (k + 1)


def shard_loss_over_run(D, prob, k, steps):
    """Cumulative union bound over a run of `steps` steps."""
    return steps * shard_loss_per_step(D, prob, k)
