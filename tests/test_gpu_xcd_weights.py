"""XCD read-rate calibration and decode plans placed with per-XCD weights (MI355X).

The weights only move units between compute-unit slots; every placement must give the
oracle's result within the attention tolerances (and the same plan bit for bit as the
oracle's plan rule, which the host tests cover).
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2606_03077_amd import libra
from paper_2606_03077_amd import workloads as wl

import gpu_harness as H

pytestmark = pytest.mark.gpu


def test_xcd_read_weights_are_sane():
    buf = torch.empty(1 << 30, dtype=torch.uint8, device="cuda")
    H.say("[case] xcd read weights, 1 GiB")
    w = libra.libra_xcd_read_weights(buf, reps=3)
    H.say(f"[xcd] weights {w}")
    assert len(w) == 8
    assert all(1 <= x <= 1000 for x in w), w    # MI355X: 8 XCDs, each ran workgroups
    assert max(w) == 1000


def test_hbm_read_rate_is_sane():
    """Both read rates are positive, below the 8 TB/s peak plus slack, and the
    fixed-interval rate (no ramp or tail) is not below the completion-timed one by much."""
    buf = torch.empty(1 << 30, dtype=torch.uint8, device="cuda")
    H.say("[case] HBM read rate, 1 GiB")
    interval, completion = libra.libra_hbm_read_rate(buf, reps=3)
    H.say(f"[hbm] interval {interval:.0f} GB/s, completion {completion:.0f} GB/s")
    assert 1000 < completion < 9000 and 1000 < interval < 9000
    assert interval > 0.8 * completion


@pytest.mark.parametrize("weights", [None, (1000, 1, 1000, 1, 1000, 1, 1000, 1),
                                     (1, 10, 100, 1000, 1000000, 7, 0, 910), "measured"])
def test_weighted_one_wave_decode_matches_oracle(weights):
    # 12 rows on 16 CUs x 3 units, Hkv = 2: the one-wave apportionment applies and step 11
    # places 48 units on 16 slots.
    lens = [4000, 37, 1500, 900, 16, 2500, 700, 1200, 3100, 64, 511, 2049]
    H.say(f"[case] weighted one-wave decode weights={weights}")
    b = wl.custom_batch(lens, num_q_heads=8, num_kv_heads=2, seed=51)
    cache = H.DeviceCache(b)
    if weights == "measured":
        buf = torch.empty(1 << 30, dtype=torch.uint8, device="cuda")
        weights = libra.libra_xcd_read_weights(buf, reps=1)
        del buf
    params = dict(num_cus=16, units_per_cu=3, min_split_pages=2)
    if weights is not None:
        params["xcd_weight"] = list(weights)
    plan = H.plan_for(b, **params)
    info = libra.libra_plan_get_info(plan)
    assert info["balanced"] == 1 and info["n_single"] <= 48
    op = oracle.PlanParams(num_cus=16, units_per_cu=3, min_split_pages=2,
                           xcd_weight=tuple(weights) if weights is not None else (0,) * 8)
    ref_units, _ = oracle.plan_ref(lens, None, 2, 4, op)
    assert np.array_equal(libra.libra_plan_get_units(plan),
                          np.array(ref_units, np.int32).reshape(-1, 12))
    libra.libra_plan_destroy(plan)
    o, lse, _, _ = H.run(b, cache, plan_params=params)
    ro, rl = oracle.decode_ref(b.q, b.k_pages, b.v_pages, b.block_table, b.seq_lens, b.scale)
    H.assert_parity(o, lse, ro, rl, label=f"weights {weights}")
    cache.close()


@pytest.mark.parametrize("weights", [(1000, 850, 1000, 850, 1000, 850, 1000, 850),
                                     (1, 1000000, 3, 999, 0, 500, 1000, 2)])
def test_weighted_xcd_queue_decode_matches_oracle(weights):
    # 40 rows on 4 CUs x 3 units, Hkv = 2: more rows than a wave, so the chunk rule cuts
    # them (the 20,000-token row into pieces) and step 11 deals the units to the 8 XCD
    # queues.
    rng = np.random.default_rng(52)
    lens = rng.integers(1, 3000, size=40).tolist()
    lens[7] = 20000  # one row long enough for the chunk rule to split
    H.say(f"[case] weighted XCD-queue decode weights={weights}")
    b = wl.custom_batch(lens, num_q_heads=8, num_kv_heads=2, seed=53)
    cache = H.DeviceCache(b)
    params = dict(num_cus=4, units_per_cu=3, min_split_pages=4, xcd_weight=list(weights))
    plan = H.plan_for(b, **params)
    info = libra.libra_plan_get_info(plan)
    assert info["balanced"] == 0 and info["n_merge_groups"] > 0
    ref_units, _ = oracle.plan_ref(lens, None, 2, 4,
                                   oracle.PlanParams(num_cus=4, units_per_cu=3, min_split_pages=4,
                                                     xcd_weight=tuple(weights)))
    assert np.array_equal(libra.libra_plan_get_units(plan),
                          np.array(ref_units, np.int32).reshape(-1, 12))
    libra.libra_plan_destroy(plan)
    o, lse, _, _ = H.run(b, cache, plan_params=params)
    ro, rl = oracle.decode_ref(b.q, b.k_pages, b.v_pages, b.block_table, b.seq_lens, b.scale)
    H.assert_parity(o, lse, ro, rl, label=f"xcd queues, weights {weights}")
    cache.close()
