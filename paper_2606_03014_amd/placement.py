"""Placement of experts on N workers: the paper's scheduling ILP.

Host-side policy (no device work). It decides which workers load which
experts and how many of each expert's prompts every worker serves, from a
per-model cost model:

* Eq. 2: per-model output statistics Obar_m (mean) and O_m^max (max output
  tokens per call) from a calibration set of calls.
* T_m(N_m, Obar_m, O_m^max): predicted wall time of one session that serves
  the model's N_m prompts (Section "Workload Characterisation"). The paper
  fits a regression to a profiling sweep of its serving engine. On this
  engine a session is continuous batching of all its calls, so its time is
  the longest call's decode steps times the per-step cost, plus the marginal
  cost of every generated token: T = t_step * O^max + t_token * N * Obar,
  with t_step and t_token fitted by least squares to measured sessions
  (fit_session_model) or taken from a bandwidth model.
* Eq. 3: per-prompt cost tau_m = T_m / N_m.
* Eq. 8: replica cap R_m^max = clamp(1, floor(T_m / l_m), N), l_m the load cost.
* Eq. 4-10: binary Y[m][n] (worker n loads m), integer X[m][n] (prompts of m
  on n), worker time T_n = sum_m l_m Y + sum_m tau_m X; minimise the makespan
  C >= T_n subject to coverage (sum_n X = N_m), linkage (X <= N_m Y), replica
  bounds (1 <= sum_n Y <= R_m^max) and capacity (sum_m Y <= K). Solved exactly
  by a mixed-integer solver (scipy / HiGHS).

Eq. 9 is applied as a hard constraint, as written; the evaluation text calls
K a soft budget, a reading this module does not take.

On one MI355X every expert is resident (no load cost, N = 1: the placement
is trivial); the solver plans multi-GPU deployments of this engine.
"""
from dataclasses import dataclass, field
import math

import numpy as np


def output_stats(lengths):
    """Eq. 2: (mean, max) output tokens of a model over its calibration calls."""
    a = np.asarray(lengths, dtype=np.float64)
    if a.size == 0:
        raise ValueError("no calibration calls")
    return float(a.mean()), float(a.max())


def session_time(n_prompts, o_mean, o_max, t_step, t_token):
    """T_m(N_m, Obar_m, O_m^max) of one continuous-batching session."""
    return t_step * o_max + t_token * n_prompts * o_mean


def fit_session_model(samples):
    """Least-squares (t_step, t_token) from measured sessions
    [(n_prompts, o_mean, o_max, seconds)], both constrained to be >= 0."""
    A = np.array([[s[2], s[0] * s[1]] for s in samples], dtype=np.float64)
    y = np.array([s[3] for s in samples], dtype=np.float64)
    from scipy.optimize import nnls
    coef, _ = nnls(A, y)
    return float(coef[0]), float(coef[1])


@dataclass
class ModelCost:
    name: str
    n_prompts: int        # N_m
    load: float           # l_m, seconds to start a session of the model on a worker
    T_hat: float          # T_m(N_m, ...), seconds for all N_m prompts in one session

    @property
    def tau(self):
        """Eq. 3: per-prompt scheduling cost."""
        return self.T_hat / self.n_prompts

    def replica_cap(self, n_workers):
        """Eq. 8: as many workers as the session time amortises loads, in [1, N]."""
        if self.load <= 0:
            return n_workers
        return max(1, min(n_workers, int(math.floor(self.T_hat / self.load))))


@dataclass
class Placement:
    Y: np.ndarray                 # [M, N] 0/1
    X: np.ndarray                 # [M, N] prompts
    worker_time: np.ndarray       # [N] seconds (Eq. 4)
    makespan: float               # C
    caps: list = field(default_factory=list)   # R_m^max used


def solve_placement(models, n_workers, capacity):
    """Exact solution of Eq. 4-10 for `models` (list of ModelCost) on
    `n_workers` workers with per-worker capacity K = `capacity`.
    Raises ValueError when no placement satisfies the constraints."""
    from scipy.optimize import Bounds, LinearConstraint, milp
    M, N = len(models), n_workers
    if M == 0 or N < 1 or capacity < 1:
        raise ValueError("need at least one model, one worker and capacity >= 1")
    caps = [m.replica_cap(N) for m in models]
    # variable layout: Y (M*N), X (M*N), C
    nv = 2 * M * N + 1
    yi = lambda m, n: m * N + n
    xi = lambda m, n: M * N + m * N + n
    ci = 2 * M * N
    rows, lo, hi = [], [], []

    def row(coefs, a, b):
        r = np.zeros(nv)
        for i, v in coefs:
            r[i] += v
        rows.append(r)
        lo.append(a)
        hi.append(b)

    for n in range(N):          # Eq. 4 / 10: T_n - C <= 0
        row([(yi(m, n), models[m].load) for m in range(M)] + [(xi(m, n), models[m].tau) for m in range(M)]
            + [(ci, -1.0)], -np.inf, 0.0)
    for m in range(M):          # Eq. 5: coverage
        row([(xi(m, n), 1.0) for n in range(N)], models[m].n_prompts, models[m].n_prompts)
    for m in range(M):          # Eq. 6: linkage
        for n in range(N):
            row([(xi(m, n), 1.0), (yi(m, n), -float(models[m].n_prompts))], -np.inf, 0.0)
    for m in range(M):          # Eq. 7-8: replicas
        row([(yi(m, n), 1.0) for n in range(N)], 1.0, float(caps[m]))
    for n in range(N):          # Eq. 9: capacity
        row([(yi(m, n), 1.0) for m in range(M)], -np.inf, float(capacity))
    c = np.zeros(nv)
    c[ci] = 1.0
    integrality = np.ones(nv)
    integrality[ci] = 0
    ub = np.concatenate([np.ones(M * N), np.repeat([float(mm.n_prompts) for mm in models], N), [np.inf]])
    res = milp(c, constraints=LinearConstraint(np.array(rows), lo, hi), integrality=integrality,
               bounds=Bounds(np.zeros(nv), ub), options={"mip_rel_gap": 0.0})
    if res.status != 0 or res.x is None:
        raise ValueError(f"no feasible placement ({res.message})")
    Y = np.rint(res.x[: M * N]).astype(np.int64).reshape(M, N)
    X = np.rint(res.x[M * N: 2 * M * N]).astype(np.int64).reshape(M, N)
    loads = np.array([mm.load for mm in models])
    taus = np.array([mm.tau for mm in models])
    worker_time = loads @ Y + taus @ X
    return Placement(Y=Y, X=X, worker_time=worker_time, makespan=float(worker_time.max()), caps=caps)
