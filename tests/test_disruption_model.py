"""The analytic models of Sec. IV and Sec. V-C against the numbers the paper
prints (CPU only)."""
import math

import pytest

from paper_2607_01646_amd import disruption as M


def close(a, b, rel=1e-9):
    return math.isclose(a, b, rel_tol=rel)


def test_worked_example_replay_of_sec_iv():
    # checkpoints every 100 steps of ~20 s: expected replay ~16.7 minutes
    replay = M.expected_replay_steps(100, worked_example=True) * 20.0
    assert round(replay / 60.0, 1) == 16.7
    # the model's own formula gives half a step less
    assert M.expected_replay_steps(100) == 49.5


def test_empirical_replay_reduces_to_the_uniform_case():
    K = 100
    uniform = {r: 1.0 / K for r in range(K)}
    assert close(M.expected_replay_steps_empirical(uniform), M.expected_replay_steps(K))
    with pytest.raises(ValueError):
        M.expected_replay_steps_empirical({1: 0.5})


def test_disruption_and_efficiency_at_the_sec_iv_operating_point():
    # failures every 18 min, 10 min restart stall, replay 16.7 min
    mttf = 18 * 60.0
    c = M.disruption_checkpoint_restart(0.0, 10 * 60.0, 20.0, M.expected_replay_steps(100, worked_example=True))
    assert close(c, 600.0 + 1000.0)
    assert close(M.efficiency(mttf, c), mttf / (mttf + 1600.0))
    assert close(M.disruption_rate(mttf, c), 1600.0 / 1080.0)
    # the in-memory scheme: replay bounded by the interrupted step
    d = M.disruption_in_memory(0.0, 30.0, 20.0, 0.5)
    assert close(d, 40.0) and M.efficiency(mttf, d) > 0.96
    with pytest.raises(ValueError):
        M.disruption_in_memory(0.0, 30.0, 20.0, 1.0)


def test_per_node_failure_probability_is_order_1e_minus_6():
    # one interruption per ~18 min over ~100K GPUs (8 per node), 20 s steps
    p = M.per_node_step_failure(18 * 60.0, 20.0, 100_000 / 8)
    assert 1e-6 <= p < 1e-5 and round(math.log10(p)) == -6


def test_independent_failure_bounds_of_sec_v_c():
    assert close(M.shard_loss_per_step(128, 1e-6, 1), 1.28e-10)
    assert close(M.shard_loss_over_run(128, 1e-6, 1, 10**5), 1.28e-5)
    assert close(M.shard_loss_over_run(128, 1e-6, 2, 10**5), 1.28e-11)


def test_failure_domain_bounds_of_sec_v_c():
    assert close(M.shard_loss_over_run(128, 1e-4, 1, 10**5), 0.128)
    assert close(M.shard_loss_over_run(128, 1e-4, 2, 10**5), 1.28e-5)


def test_loss_bound_edge_cases():
    assert M.shard_loss_per_step(128, 0.0, 1) == 0.0
    assert M.shard_loss_per_step(1, 1.0, 3) == 1.0
    assert M.shard_loss_per_step(0, 0.5, 1) == 0.0
    with pytest.raises(ValueError):
        M.shard_loss_per_step(128, 1.5, 1)
