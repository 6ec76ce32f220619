"""The library's host cost evaluator, RolloutDP, prefix tree and routing against the
oracle (no GPU involved: all of it is host arithmetic behind the C-ABI)."""
import math

import numpy as np
import pytest

from oracle.cost_model import (ce_fit_ref, mape_ref, partition_makespan, poly_sum_ref,
                               rollout_dp_ref)
from oracle.scheduler import PrefixTreeRef, route_ref
from paper_2606_03077_amd import libra
from paper_2606_03077_amd import workloads as wl


@pytest.mark.parametrize("seed", range(5))
def test_ce_fit_matches_oracle(seed):
    rng = np.random.default_rng(seed)
    n = int(rng.integers(3, 40))
    L = np.sort(rng.uniform(0, 40960, size=n))
    L[:3] = [16.0, 2048.0, 40960.0]
    g, e, t = 10 ** rng.uniform(-10, -8), 10 ** rng.uniform(-6, -4), 10 ** rng.uniform(-3, -1)
    T = (g * L * L + e * L + t) * rng.lognormal(0, 0.05 * (seed % 3), size=n)
    got = libra.libra_ce_fit(L, T)
    want = ce_fit_ref(L, T)
    # compare predictions (what the coefficients are for) over the measured range
    grid = np.linspace(0, 40960, 50)
    pg = got[0] * grid ** 2 + got[1] * grid + got[2]
    pw = want[0] * grid ** 2 + want[1] * grid + want[2]
    assert np.max(np.abs(pg - pw) / np.abs(pw)) <= 1e-7
    # the library's solution is at least as good in the objective both minimise
    obj = lambda c: float(np.sum(((c[0] * L * L + c[1] * L + c[2]) - T) ** 2 / T ** 2))
    assert obj(got) <= obj(want) * (1 + 1e-9) + 1e-24
    assert libra.libra_ce_mape(want, L, T) == pytest.approx(mape_ref(want, L, T), rel=1e-12)


def test_ce_fit_validation():
    with pytest.raises(libra.LibraError):
        libra.libra_ce_fit([1, 2], [1, 2])                    # too few points
    with pytest.raises(libra.LibraError):
        libra.libra_ce_fit([1, 1, 2, 2], [1, 2, 3, 4])        # two distinct lengths
    with pytest.raises(libra.LibraError):
        libra.libra_ce_fit([1, 2, 3], [1, 0, 3])              # a non-positive time
    with pytest.raises(libra.LibraError):
        libra.libra_ce_poly_sum((1, 0, 0), -1, 3)


@pytest.mark.parametrize("poly", [(1.0, 0.0, 0.0), (3.0, -2.0, 5.0), (2e-9, 1e-6, 3e-5)])
@pytest.mark.parametrize("ab", [(1, 1), (1, 100), (0, 7), (500, 40960), (9, 3), (40000, 40960)])
def test_poly_sum_matches_oracle(poly, ab):
    got = libra.libra_ce_poly_sum(poly, *ab)
    want = poly_sum_ref(poly, *ab)
    assert got == pytest.approx(want, rel=1e-12, abs=1e-12)


MODEL = {"attn_step": (2e-9, 1e-6, 0.0),
         "linear_step": [1.0e-3, 0.6e-3, 0.36e-3, 0.25e-3],
         "attn_scale": [1.0, 0.52, 0.27, 0.15]}


def lib_model(m):
    return libra.rollout_model(m["attn_step"], dict(zip([1, 2, 4, 8], m["linear_step"])),
                               dict(zip([1, 2, 4, 8], m["attn_scale"])))


@pytest.mark.parametrize("seed", range(8))
def test_rollout_dp_matches_oracle(seed):
    rng = np.random.default_rng(100 + seed)
    n = int(rng.integers(0, 14))
    lengths = rng.choice([0, 16, 300, 300, 2500, 9000, 40000], size=n).tolist()
    n_gpus = int(rng.integers(0, 10))
    tp_set = [[1, 2, 4, 8], [1, 2, 4], [2, 4], [8, 4, 2, 1]][seed % 4]
    want, want_order, _ = rollout_dp_ref(lengths, n_gpus, tp_set, MODEL)
    for exact in (True, False):
        ms, order, inst = libra.libra_rollout_dp(lengths, n_gpus, tp_set, lib_model(MODEL), exact)
        assert order.tolist() == want_order
        if math.isinf(want):
            assert math.isinf(ms) and inst == []
            continue
        assert ms == pytest.approx(want, rel=1e-12, abs=1e-15)
        # the returned partition is valid and achieves the makespan
        assert sum(tp for tp, _, _ in inst) == n_gpus
        assert all(tp in tp_set for tp, _, _ in inst)
        covered = sorted(p for _, f, c in inst for p in range(f, f + c))
        assert covered == list(range(n))
        assert partition_makespan(lengths, order.tolist(), inst, MODEL) == pytest.approx(ms, rel=1e-12, abs=1e-15)


def test_rollout_dp_fast_equals_literal_at_scale():
    """The crossing search returns the literal recurrence's makespan bit for bit."""
    rng = np.random.default_rng(7)
    lengths = np.minimum(rng.pareto(1.2, size=400) * 2000 + 200, 65536).astype(np.int64)
    m = lib_model(MODEL)
    a = libra.libra_rollout_dp(lengths, 32, [1, 2, 4, 8], m, exact=True)
    b = libra.libra_rollout_dp(lengths, 32, [1, 2, 4, 8], m, exact=False)
    assert a[0] == b[0]


def test_rollout_dp_validation():
    m = lib_model(MODEL)
    with pytest.raises(libra.LibraError):
        libra.libra_rollout_dp([1, 2], 4, [3], m)           # degree outside {1,2,4,8}
    with pytest.raises(libra.LibraError):
        libra.libra_rollout_dp([1, 2], 4, [2, 2], m)        # repeated degree
    with pytest.raises(libra.LibraError):
        libra.libra_rollout_dp([-1], 4, [1], m)             # negative length
    with pytest.raises(libra.LibraError):
        libra.libra_rollout_dp([1] * 60000, 4096, [1], m)   # state table too large


def test_prefix_tree_matches_oracle_on_synthetic_traces():
    traces = wl.synthetic_traces(40, 8, seed=5)
    edges = [1024, 4096, 16384]
    lib = libra.PrefixTree(edges)
    ref = PrefixTreeRef(edges)
    for p, st, res in traces[:250]:
        lib.insert(p, st, res)
        ref.insert(p, st, res)
    rng = np.random.default_rng(1)
    queries = [(p, st[:k]) for p, st, _ in traces for k in range(len(st) + 1)]
    queries += [(p, st + [int(rng.integers(64))]) for p, st, _ in traces[:50]]
    queries += [(999, []), (998, [1, 2, 3])]
    for p, st in queries:
        h, d = lib.lookup(p, st)
        rh, rd = ref.lookup(p, st)
        assert d == rd and h.tolist() == rh, (p, st)
    lib.close()


def test_prefix_tree_validation():
    with pytest.raises(libra.LibraError):
        libra.PrefixTree([4096, 1024])                      # not increasing
    t = libra.PrefixTree([10])
    with pytest.raises(libra.LibraError):
        t.lookup(1, [])                                     # empty tree
    with pytest.raises(libra.LibraError):
        t.insert(1, [2], [5, -1])                           # negative residual
    t.close()


@pytest.mark.parametrize("seed", range(6))
def test_route_matches_oracle(seed):
    rng = np.random.default_rng(seed)
    M, K = int(rng.integers(1, 6)), int(rng.integers(1, 8))
    hist = rng.dirichlet(np.ones(K))
    t_dec = rng.uniform(1, 100, size=(M, K))
    c_mig = rng.uniform(0, 20, size=(M, M))
    cur = int(rng.integers(M))
    b, c = libra.libra_route_bucket(hist, t_dec, c_mig, cur)
    rb, rc = route_ref(hist.tolist(), t_dec.tolist(), c_mig.tolist(), cur)
    assert c == pytest.approx(rc, rel=1e-12)
    costs = [sum(hist[k] * t_dec[x][k] for k in range(K)) + (0 if x == cur else c_mig[cur][x])
             for x in range(M)]
    second = sorted(costs)[1] if M > 1 else math.inf
    if second - min(costs) > 1e-9 * abs(min(costs)):
        assert b == rb                                      # unique minimum
    else:
        assert costs[b] == pytest.approx(min(costs), rel=1e-12)
