"""Brute-force optimum of the paper's placement ILP (Section "Scheduling
Algorithm Formulation", Eq. 4-10) on small instances.

TEST INFRASTRUCTURE ONLY; the product package never imports this.

Every 0/1 placement Y is enumerated; the ones that respect the replica caps
(Eq. 7-8: 1 <= sum_n Y[m][n] <= R_m) and the worker capacity (Eq. 9:
sum_m Y[m][n] <= K) are kept; for each, every way of splitting each model's
N_m prompts over the workers that load it (Eq. 5-6) is enumerated, and the
worker times T_n = sum_m l_m Y[m][n] + sum_m tau_m X[m][n] (Eq. 4) give the
makespan (Eq. 10). The minimum over everything is the optimum.

models: list of (n_prompts, load, tau, cap).
"""
import itertools


def _splits(total, slots):
    """All ways to write `total` as an ordered sum of `slots` non-negative integers."""
    if slots == 1:
        yield (total,)
        return
    for first in range(total + 1):
        for rest in _splits(total - first, slots - 1):
            yield (first,) + rest


def brute_force_makespan(models, n_workers, capacity):
    """Optimal makespan, or None when no placement is feasible."""
    M, N = len(models), n_workers
    best = None
    worker_sets = []
    for (n_p, load, tau, cap) in models:
        opts = [s for r in range(1, min(cap, N) + 1) for s in itertools.combinations(range(N), r)]
        worker_sets.append(opts)
    for choice in itertools.product(*worker_sets):
        per_worker = [0] * N
        for s in choice:
            for n in s:
                per_worker[n] += 1
        if max(per_worker) > capacity:
            continue
        base = [0.0] * N
        for (n_p, load, tau, cap), s in zip(models, choice):
            for n in s:
                base[n] += load
        splits = [list(_splits(models[m][0], len(choice[m]))) for m in range(M)]
        for split in itertools.product(*splits):
            t = list(base)
            for m, parts in enumerate(split):
                for n, k in zip(choice[m], parts):
                    t[n] += models[m][2] * k
            c = max(t)
            if best is None or c < best:
                best = c
    return best
