"""The placement ILP (Eq. 4-10) with the cost model of Eq. 2-3 and the
replica cap of Eq. 8: exact optimum against brute-force enumeration on small
instances, closed-form cases, infeasibility, and the cost-model helpers."""
import math

import numpy as np
import pytest

from oracle.placement import brute_force_makespan
from paper_2606_03014_amd.placement import (ModelCost, fit_session_model, output_stats, session_time,
                                            solve_placement)


def _check_constraints(models, N, K, p):
    M = len(models)
    assert p.X.sum(axis=1).tolist() == [m.n_prompts for m in models]                     # Eq. 5
    assert np.all(p.X <= np.array([[m.n_prompts] for m in models]) * p.Y)                 # Eq. 6
    reps = p.Y.sum(axis=1)
    assert np.all(reps >= 1) and all(reps[i] <= models[i].replica_cap(N) for i in range(M))  # Eq. 7-8
    assert np.all(p.Y.sum(axis=0) <= K)                                                   # Eq. 9
    t = np.array([m.load for m in models]) @ p.Y + np.array([m.tau for m in models]) @ p.X
    assert np.allclose(t, p.worker_time) and math.isclose(p.makespan, t.max())            # Eq. 4, 10


@pytest.mark.parametrize("seed", range(40))
def test_ilp_optimum_equals_brute_force(seed):
    rng = np.random.default_rng([seed, 77])
    M, N = int(rng.integers(1, 4)), int(rng.integers(1, 4))
    K = int(rng.integers(1, M + 1))
    models = []
    for i in range(M):
        n = int(rng.integers(1, 6))
        load = float(rng.choice([0.0, rng.uniform(0.5, 5.0)]))
        models.append(ModelCost(f"m{i}", n, load, float(rng.uniform(1.0, 40.0))))
    want = brute_force_makespan([(m.n_prompts, m.load, m.tau,
                                  N if m.load <= 0 else max(1, min(N, math.floor(m.T_hat / m.load))))
                                 for m in models], N, K)
    if want is None:
        with pytest.raises(ValueError):
            solve_placement(models, N, K)
        return
    p = solve_placement(models, N, K)
    _check_constraints(models, N, K, p)
    assert math.isclose(p.makespan, want, rel_tol=1e-9, abs_tol=1e-9)


def test_single_model_splits_evenly():
    """One model, no load cost, N workers: ceil(N_m / N) prompts on the busiest worker."""
    for n_prompts, N in ((10, 4), (7, 7), (3, 5), (1, 3)):
        m = ModelCost("a", n_prompts, 0.0, 6.0 * n_prompts)
        p = solve_placement([m], N, 1)
        assert math.isclose(p.makespan, math.ceil(n_prompts / N) * m.tau)


def test_capacity_one_pins_each_model_to_a_worker():
    """K = 1 and loads as large as the sessions (cap 1): every model alone on one worker."""
    models = [ModelCost(f"m{i}", 4, 10.0 * (i + 1), 10.0 * (i + 1)) for i in range(3)]
    p = solve_placement(models, 3, 1)
    assert p.Y.sum(axis=1).tolist() == [1, 1, 1] and p.Y.sum(axis=0).tolist() == [1, 1, 1]
    assert math.isclose(p.makespan, max(m.load + m.T_hat for m in models))


def test_infeasible_capacity_raises():
    models = [ModelCost(f"m{i}", 2, 1.0, 5.0) for i in range(5)]
    with pytest.raises(ValueError):
        solve_placement(models, 2, 2)          # K * N = 4 < M = 5


def test_replica_cap_formula():
    assert ModelCost("r", 10, 2.0, 9.0).replica_cap(8) == 4        # floor(9 / 2)
    assert ModelCost("r", 10, 20.0, 9.0).replica_cap(8) == 1       # clamped below
    assert ModelCost("r", 10, 0.5, 90.0).replica_cap(8) == 8       # clamped above
    assert ModelCost("r", 10, 0.0, 9.0).replica_cap(3) == 3        # no load cost: any worker


def test_cost_model_helpers():
    assert output_stats([3, 5, 10]) == (6.0, 10.0)
    samples = [(n, om, ox, session_time(n, om, ox, 0.0125, 3e-5))
               for n, om, ox in ((10, 300, 900), (50, 800, 4000), (7, 120, 200), (200, 1500, 8000))]
    t_step, t_token = fit_session_model(samples)
    assert math.isclose(t_step, 0.0125, rel_tol=1e-6) and math.isclose(t_token, 3e-5, rel_tol=1e-6)
