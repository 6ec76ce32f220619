"""Cost evaluator polynomials and RolloutDP, from their definitions.

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__``).

Sec. 4.5 and App. B.1: the cost evaluator predicts an operator's time at sequence
length L with a polynomial fitted to measured timings; attention is quadratic,
T(L) = gamma L^2 + eta L + theta.  Sec. 7.5 scores the fit by MAPE.  Sec. 4.2 and
Alg. 1 (RolloutDP) split the rollout GPUs into instances of TP degrees from a set and
give each a contiguous run of the length-sorted requests, minimising the makespan
through dp[g][i] = min over (tp <= g, 0 <= x <= i) of
max(dp[g - tp][i - x], Cost(tp, i - x + 1, i)).

Readings (the paper leaves them open):
* The fit minimises squared relative error, the quantity MAPE averages.
* Cost(tp, a, b), the evaluator's RolloutTime of one instance, is modelled as continuous
  batching of all its requests: as many decode steps as the longest request, each
  paying a per-step non-attention time at that TP, plus every request's own trajectory
  attention, sum over its decode steps l = 1 .. len of T_attn_step(l), scaled per TP.
* Requests are sorted by (length, original index); ties among equal makespans are
  broken by the first candidate in (tp in the given order, x ascending).
"""
from __future__ import annotations

import functools
import math

import numpy as np

TP_SLOTS = {1: 0, 2: 1, 4: 2, 8: 3}


def poly_eval(poly, L):
    g, e, t = poly
    return g * L * L + e * L + t


def ce_fit_ref(lengths, times):
    """Least squares in relative error: minimise sum ((T(L_i) - t_i) / t_i)^2.

    Written as an ordinary least-squares problem with rows (L^2, L, 1) / t_i and
    target 1, solved by numpy's lstsq.
    """
    L = np.asarray(lengths, dtype=np.float64)
    t = np.asarray(times, dtype=np.float64)
    A = np.stack([L * L / t, L / t, 1.0 / t], axis=1)
    coef, *_ = np.linalg.lstsq(A, np.ones_like(t), rcond=None)
    return tuple(float(c) for c in coef)


def mape_ref(poly, lengths, times):
    """Mean absolute percentage error of the polynomial against measured times (Sec. 7.5)."""
    errs = [abs(poly_eval(poly, float(L)) - float(t)) / float(t) for L, t in zip(lengths, times)]
    return 100.0 * sum(errs) / len(errs)


def poly_sum_ref(poly, a: int, b: int):
    """sum of T(l) for l = a .. b, one term at a time."""
    return sum(poly_eval(poly, float(l)) for l in range(int(a), int(b) + 1))


@functools.lru_cache(maxsize=None)
def trajectory_attention(poly, length: int):
    """A request's attention time over its decode steps l = 1 .. length."""
    return poly_sum_ref(poly, 1, length)


def instance_cost(model, tp: int, seg_lengths):
    """RolloutTime of one instance of degree tp serving the given requests (the reading
    above): per-step non-attention time times the longest request, plus the scaled sum
    of the requests' trajectory attention.  Empty: 0."""
    if len(seg_lengths) == 0:
        return 0.0
    s = TP_SLOTS[tp]
    attn = sum(trajectory_attention(tuple(model["attn_step"]), int(x)) for x in seg_lengths)
    return model["linear_step"][s] * max(seg_lengths) + model["attn_scale"][s] * attn


def sorted_order(lengths):
    return sorted(range(len(lengths)), key=lambda j: (lengths[j], j))


def rollout_dp_ref(lengths, n_gpus: int, tp_set, model):
    """Alg. 1, RolloutDP, with 1-based request indices as in the paper.

    Returns (makespan, order, instances): instances are (tp, first sorted position
    (0-based), count), last-added first, recovered by backtracking.
    """
    order = sorted_order(lengths)
    ls = [int(lengths[j]) for j in order]
    n = len(ls)
    inf = math.inf
    dp = [[inf] * (n + 1) for _ in range(n_gpus + 1)]
    pick = [[None] * (n + 1) for _ in range(n_gpus + 1)]
    dp[0][0] = 0.0

    def cost(tp, a, b):          # requests a .. b (1-based, inclusive); empty when b < a
        return instance_cost(model, tp, ls[a - 1:b])

    for g in range(1, n_gpus + 1):
        for i in range(0, n + 1):
            for tp in tp_set:
                if tp > g:
                    continue
                for x in range(0, i + 1):
                    t_inst = cost(tp, i - x + 1, i)
                    cand = max(dp[g - tp][i - x], t_inst)
                    if cand < dp[g][i]:
                        dp[g][i] = cand
                        pick[g][i] = (tp, x)
    ms = dp[n_gpus][n]
    inst = []
    if math.isfinite(ms):
        g, i = n_gpus, n
        while g > 0:
            tp, x = pick[g][i]
            inst.append((tp, i - x, x))
            g -= tp
            i -= x
    return ms, order, inst


def partition_makespan(lengths, order, instances, model):
    """Makespan of a given partition (instances over sorted positions), for checking
    that any partition a solver returns is valid and achieves its claimed value."""
    ls = [int(lengths[j]) for j in order]
    return max((instance_cost(model, tp, ls[f:f + c]) for tp, f, c in instances), default=0.0)
