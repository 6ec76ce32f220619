"""Pins for the cost-evaluator and RolloutDP oracle (Sec. 4.2, Sec. 4.5, Alg. 1).

* The fit: noise-free data of a known quadratic gives back its coefficients; the
  weighted residual is orthogonal to every weighted column (the normal equations,
  checked without the solver); scaling every time scales the coefficients.
* The trajectory sum: textbook sums of l and l^2, in exact integer arithmetic.
* RolloutDP: a brute force over every way of writing the GPU count as an ordered
  sequence of TP degrees and every cut of the sorted requests into that many contiguous
  runs, plus closed-form special cases.
"""
import itertools
import math

import numpy as np
import pytest

import oracle.cost_model as ocm
from oracle.cost_model import (ce_fit_ref, instance_cost, mape_ref, partition_makespan,
                               poly_eval, poly_sum_ref, rollout_dp_ref, sorted_order)


def test_fit_recovers_exact_quadratic():
    true = (3.5e-9, 2.0e-5, 0.011)
    L = np.array([256, 1024, 4096, 8192, 16384, 32768, 40960], dtype=np.float64)
    t = np.array([poly_eval(true, x) for x in L])
    got = ce_fit_ref(L, t)
    for a, b in zip(got, true):
        assert abs(a - b) <= 1e-9 * abs(b)
    assert mape_ref(got, L, t) < 1e-9


def test_fit_normal_equations_hold():
    rng = np.random.default_rng(0)
    L = np.sort(rng.uniform(100, 40000, size=30))
    t = (2e-9 * L * L + 1e-5 * L + 0.02) * rng.lognormal(0, 0.05, size=30)
    g, e, th = ce_fit_ref(L, t)
    r = (g * L * L + e * L + th - t) / t
    for col in (L * L / t, L / t, 1.0 / t):
        assert abs(float(np.dot(r, col))) <= 1e-9 * float(np.linalg.norm(col)) * max(1.0, float(np.linalg.norm(r)))


def test_fit_scales_with_times():
    rng = np.random.default_rng(1)
    L = np.linspace(500, 30000, 12)
    t = (1e-9 * L * L + 3e-5 * L + 0.05) * rng.lognormal(0, 0.03, size=12)
    a = ce_fit_ref(L, t)
    b = ce_fit_ref(L, 7.0 * t)
    for x, y in zip(a, b):
        assert abs(7.0 * x - y) <= 1e-9 * abs(y)


def test_mape_by_hand():
    # T(L) = L: predictions 1, 2 against times 2, 2 -> errors 50% and 0% -> MAPE 25%
    assert mape_ref((0.0, 1.0, 0.0), [1, 2], [2, 2]) == pytest.approx(25.0, abs=1e-12)


@pytest.mark.parametrize("a,b", [(1, 1), (1, 10), (3, 77), (0, 5), (1000, 2000), (5, 4)])
def test_trajectory_sum_textbook(a, b):
    s1 = lambda n: n * (n + 1) // 2
    s2 = lambda n: n * (n + 1) * (2 * n + 1) // 6
    am = max(a - 1, 0)
    want_sq = s2(b) - s2(am) if b >= a else 0
    want_lin = s1(b) - s1(am) if b >= a else 0
    count = max(0, b - a + 1)
    assert poly_sum_ref((1, 0, 0), a, b) == want_sq
    assert poly_sum_ref((0, 1, 0), a, b) == want_lin
    assert poly_sum_ref((0, 0, 1), a, b) == count
    assert poly_sum_ref((3, -2, 5), a, b) == 3 * want_sq - 2 * want_lin + 5 * count


MODEL = {"attn_step": (2e-9, 1e-6, 0.0),
         "linear_step": [1.0e-3, 0.6e-3, 0.36e-3, 0.25e-3],
         "attn_scale": [1.0, 0.52, 0.27, 0.15]}


# Hand-sized model for the by-hand pins below: T_attn_step(l) = l + 2, per-step
# non-attention time 10 at TP 1 and 6 at TP 2, attention scaled by 1 at TP 1 and 0.5 at TP 2.
HAND = {"attn_step": (0.0, 1.0, 2.0), "linear_step": [10.0, 6.0, 0.0, 0.0],
        "attn_scale": [1.0, 0.5, 0.0, 0.0]}


def test_instance_cost_by_hand():
    """Cost(tp, a, b) of Alg. 1 under the library's reading (an instance batches all its
    requests: as many decode steps as its longest request, each paying the TP's
    per-step time, plus every request's trajectory attention sum_{l=1..len} T(l),
    scaled per TP), worked out by hand for requests of 2, 3 and 5 tokens:

      trajectory attention: len 2 -> (1+2) + (2+2) = 7
                            len 3 -> 3 + 4 + 5     = 12
                            len 5 -> 3+4+5+6+7     = 25      total 44
      TP 1: 10 * max(2, 3, 5) + 1.0 * 44 = 50 + 44 = 94
      TP 2:  6 * 5            + 0.5 * 44 = 30 + 22 = 52
      one request of 5 at TP 1: 10 * 5 + 25 = 75; of 2 and 3: 10 * 3 + 19 = 49
    """
    assert ocm.instance_cost(HAND, 1, [2, 3, 5]) == 94.0
    assert ocm.instance_cost(HAND, 2, [2, 3, 5]) == 52.0
    assert ocm.instance_cost(HAND, 1, [5]) == 75.0
    assert ocm.instance_cost(HAND, 1, [2, 3]) == 49.0
    assert ocm.instance_cost(HAND, 2, []) == 0.0


def test_rollout_dp_by_hand():
    """Two GPUs, degrees {1, 2}, requests 5, 2, 3 (sorted: 2, 3, 5), by hand from the costs
    of test_instance_cost_by_hand: one TP-2 instance costs 52; two TP-1 instances with
    contiguous runs cost max(0, 94) = 94, max(27, 87) = 87 (runs [2] and [3, 5]:
    10 * 2 + 7 = 27, 10 * 5 + 12 + 25 = 87) or max(49, 75) = 75.  Best: 52, TP 2."""
    ms, order, inst = ocm.rollout_dp_ref([5, 2, 3], 2, [1, 2], HAND)
    assert ms == 52.0
    assert order == [1, 2, 0] and inst == [(2, 0, 3)]
    ms1, _, inst1 = ocm.rollout_dp_ref([5, 2, 3], 2, [1], HAND)
    assert ms1 == 75.0 and sorted(inst1) == [(1, 0, 2), (1, 2, 1)]


def compositions(n, parts):
    """Every ordered sequence of degrees from ``parts`` summing to n."""
    if n == 0:
        yield ()
        return
    for p in parts:
        if p <= n:
            for rest in compositions(n - p, parts):
                yield (p,) + rest


def brute_force(lengths, n_gpus, tp_set, model):
    ls = [lengths[j] for j in sorted_order(lengths)]
    n = len(ls)
    best = math.inf
    for comp in compositions(n_gpus, tp_set):
        m = len(comp)
        # cut points 0 <= c_1 <= ... <= c_{m-1} <= n
        for cuts in itertools.combinations_with_replacement(range(n + 1), m - 1):
            bounds = (0,) + cuts + (n,)
            ms = max(instance_cost(model, comp[k], ls[bounds[k]:bounds[k + 1]]) for k in range(m))
            best = min(best, ms)
    return best


@pytest.mark.parametrize("seed", range(6))
def test_rollout_dp_equals_brute_force(seed):
    rng = np.random.default_rng(seed)
    n = int(rng.integers(1, 7))
    lengths = rng.choice([30, 200, 900, 2500, 6000], size=n).tolist()
    n_gpus = int(rng.integers(1, 7))
    tp_set = [1, 2, 4] if seed % 2 else [1, 2, 4, 8]
    ms, order, inst = rollout_dp_ref(lengths, n_gpus, tp_set, MODEL)
    want = brute_force(lengths, n_gpus, tp_set, MODEL)
    assert ms == pytest.approx(want, rel=1e-12)
    assert partition_makespan(lengths, order, inst, MODEL) == pytest.approx(ms, rel=1e-12)
    assert sum(tp for tp, _, _ in inst) == n_gpus
    assert sum(c for _, _, c in inst) == n


def test_rollout_dp_special_cases():
    ls = [100, 40, 900]
    # one GPU, TP 1 only: a single instance holds everything
    ms, order, inst = rollout_dp_ref(ls, 1, [1], MODEL)
    assert inst == [(1, 0, 3)] and ms == instance_cost(MODEL, 1, sorted(ls))
    # GPUs that no degree can fill exactly: no partition
    ms, _, inst = rollout_dp_ref(ls, 3, [2, 4], MODEL)
    assert ms == math.inf and inst == []
    # no requests: makespan 0
    ms, _, _ = rollout_dp_ref([], 4, [1, 2], MODEL)
    assert ms == 0.0
    # sorted by (length, index)
    assert sorted_order([5, 3, 5, 1]) == [3, 1, 0, 2]


def test_more_gpus_never_hurt_with_tp1():
    ls = [50, 700, 3000, 3000, 12000]
    prev = math.inf
    for g in range(1, 7):
        ms, _, _ = rollout_dp_ref(ls, g, [1, 2, 4, 8], MODEL)
        assert ms <= prev + 1e-15
        prev = ms


def _partitions(n):
    """Number of integer partitions of n, by the textbook recurrence over the largest part."""
    table = [1] + [0] * n
    for part in range(1, n + 1):
        for total in range(part, n + 1):
            table[total] += table[total - part]
    return table[n]


def _tp_multisets(n, degrees=(1, 2, 4, 8)):
    """Number of ways to split n GPUs into instances of the given TP degrees (as multisets)."""
    table = [1] + [0] * n
    for d in degrees:
        for total in range(d, n + 1):
            table[total] += table[total - d]
    return table[n]


def test_partition_count_matches_the_paper():
    """Golden value: Sec. 4.2 prints p(64) ~ 1.7e6 for the search space RolloutDP avoids."""
    import os
    path = os.path.join(os.path.dirname(__file__), "golden", "partition_count.txt")
    rows = [line.split() for line in open(path) if line.strip() and not line.startswith("#")]
    for n, printed, rtol in rows:
        assert abs(_partitions(int(n)) - float(printed)) <= float(rtol) * float(printed)
    assert _partitions(5) == 7 and _partitions(10) == 42          # textbook values
    # with TP degrees restricted to {1, 2, 4, 8} the instance multisets are far fewer, and
    # RolloutDP also chooses the contiguous request runs; its brute-force pins above
    # enumerate both
    assert _tp_multisets(8) == 10 and _tp_multisets(64) < _partitions(64) / 1000
