"""Pins for the plan oracle: hand-derived tables and the invariants the rule promises."""
import dataclasses

import numpy as np
import pytest

from oracle.plan import PlanParams, plan_ref, UNIT_FIELDS

F = {name: i for i, name in enumerate(UNIT_FIELDS)}


def test_hand_derived_decode_example():
    # L = [40, 0, 100] -> pages [3, 0, 7]; W = 10, target = 1 * 2 = 2,
    # chunk = max(2, ceil(10 / 2)) = 5; n = [1, 1, 2].  Sequence 2 splits into pages
    # [0, 3) and [3, 7), i.e. tokens [0, 48) and [48, 100); its two slots start at 0.
    # Step 11 deals the four units to XCD queues 0-3 in step 9's order (one each).
    units, info = plan_ref([40, 0, 100], None, 1, 4,
                           PlanParams(num_cus=1, units_per_cu=2, min_split_pages=2, max_splits=8))
    assert units == [
        (2, 0, 48, 100, 0, 1, 1, 2, 0, 2, 0, 99),
        (2, 0, 0, 48, 0, 1, 0, 2, 0, 2, 0, 99),
        (0, 0, 0, 40, 0, 1, 0, 1, -1, 0, 0, 39),
        (1, 0, 0, 0, 0, 1, 0, 1, -1, 1, 0, -1),
    ]
    assert info["n_partial_slots"] == 2 and info["chunk_pages"] == 5


def test_hand_derived_append_example():
    # L = [10, 100], C = [1, 70], Hkv = 2, G = 8 -> T = floor(256 / 8) = 32.
    # Single row 0: one page, W = 2, target = 4, chunk = 1, n = 1.
    # Chunk row 1: P = 30, tiles [0,32) [32,64) [64,70) with keys [0,62) [0,94) [0,100);
    # costs in 64-key steps ceil(62/64) = 1, ceil(94/64) = 2, ceil(100/64) = 2; each
    # KV-head group costs 5 of a total 10, so F = ceil(10 / 8) = 2 and each group is cut
    # into n = min(3, ceil(5 / 2)) = 3 parts: tile i goes to part floor(S_i * 3 / 5) with
    # S = 0, 1, 3 -> parts 0, 0, 1 (part 2 is empty and dropped).  Parts by descending
    # cost, ties (b, g, part): (1,0,0) (1,1,0) cost 3, (1,0,1) (1,1,1) cost 2, dealt to the
    # empty queues 0..3 in that order; queues 0 and 1 list the [32,64) tile (cost 2)
    # before the [0,32) tile (cost 1).
    units, info = plan_ref([10, 100], [1, 70], 2, 8,
                           PlanParams(num_cus=4, units_per_cu=1, min_split_pages=1, max_splits=4))
    assert units == [
        (0, 0, 0, 10, 0, 1, 0, 1, -1, 0, 0, 9),
        (0, 1, 0, 10, 0, 1, 0, 1, -1, 0, 0, 9),
        (1, 0, 0, 94, 32, 64, 0, 1, -1, 1, 1, 30),
        (1, 0, 0, 62, 0, 32, 0, 1, -1, 1, 1, 30),
        (1, 1, 0, 94, 32, 64, 0, 1, -1, 1, 1, 30),
        (1, 1, 0, 62, 0, 32, 0, 1, -1, 1, 1, 30),
        (1, 0, 0, 100, 64, 70, 0, 1, -1, 1, 1, 30),
        (1, 1, 0, 100, 64, 70, 0, 1, -1, 1, 1, 30),
    ]
    assert info["xcd_queue_lens"] == [2, 2, 1, 1, 0, 0, 0, 0]
    assert info["n_single"] == 2 and info["n_chunk"] == 6 and info["q_tile"] == 32


def test_hand_derived_group_parts():
    # One 256-token chunk with no prior, Hkv = 1, G = 16 -> T = 16: tiles k = 0..15 with
    # keys 16 (k + 1) and costs ceil((k + 1) / 4) = 1,1,1,1, 2,2,2,2, 3,3,3,3, 4,4,4,4
    # (total 40, F = 5).  The group is cut into n = min(16, ceil(40 / 5)) = 8 parts at
    # floor(S_k * 8 / 40), S = 0,1,2,3,4,6,8,10,12,15,18,21,24,28,32,36 -> parts
    # 0,0,0,0,0, 1,1, 2,2, 3,3, 4,4, 5, 6, 7 of costs 6, 4, 5, 6, 7, 4, 4, 4.  By
    # descending cost (ties by part index): p4 p0 p3 p2 p1 p5 p6 p7 -> queues 0..7.
    # Each queue by descending cost, ties ascending q_begin: queue 0 = tiles 12, 11;
    # queue 1 = tile 4 (cost 2), then tiles 0, 1, 2, 3; queue 2 = tiles 9, 10; queue 3 =
    # tiles 8 (cost 3), 7 (cost 2); queue 4 = tiles 5, 6; queues 5-7 = tiles 13, 14, 15.
    units, info = plan_ref([256], [256], 1, 16, PlanParams())
    tile = lambda k: (0, 16 * (k + 1), 16 * k, 16 * (k + 1))
    assert [(u[2], u[3], u[4], u[5]) for u in units] == [
        tile(k) for k in (12, 11, 4, 0, 1, 2, 3, 9, 10, 8, 7, 5, 6, 13, 14, 15)]
    assert info["xcd_queue_lens"] == [2, 5, 2, 2, 2, 1, 1, 1]


def test_few_groups_fill_every_queue():
    # A recompute prefill with 4 KV heads has 4 (b, g) groups; each is larger than an
    # eighth of the work and is cut into parts, so all 8 XCD queues get tiles and their
    # costs differ by at most the largest single part.
    units, info = plan_ref([40960], [40960], 4, 7, PlanParams())
    lens = info["xcd_queue_lens"]
    assert all(n > 0 for n in lens)
    chunks = units[info["n_single"]:]
    cost = [-(-(u[3] - u[2]) // 64) for u in chunks]
    qcost, pos = [], 0
    for n in lens:
        qcost.append(sum(cost[pos:pos + n]))
        pos += n
    assert max(qcost) - min(qcost) <= 0.02 * sum(cost)


def check_slot_placement(singles, params, S):
    """Step 11 read off the output: position w belongs to slot w % num_cus; slot c holds
    exactly the positions w < n with w % num_cus = c; replaying the units in step 9's
    order (descending KV tokens, ties (b, g, j)), each unit's slot had room and no slot
    with room had a smaller (load + cost) / weight, nor an equal one with a smaller
    index; and a slot's units keep step 9's order across its positions."""
    from fractions import Fraction
    n = len(singles)
    w8 = [x if x > 0 else 1000 for x in params.xcd_weight]
    slot_of = {}
    for w, u in enumerate(singles):
        slot_of.setdefault(u, []).append(w % S)
    order = sorted(singles, key=lambda u: (-(u[3] - u[2]), u[0], u[1], u[6]))
    cap = [len(range(c, n, S)) for c in range(S)]
    load, used, seq = [0] * S, [0] * S, [[] for _ in range(S)]
    for u in order:
        c = slot_of[u].pop(0)
        cost = -(-u[3] // 16) - u[2] // 16
        assert used[c] < cap[c]
        mine = Fraction(load[c] + cost, w8[c % 8])
        for d in range(S):
            if used[d] < cap[d]:
                other = Fraction(load[d] + cost, w8[d % 8])
                assert other > mine or (other == mine and d >= c), (u, c, d)
        load[c] += cost
        used[c] += 1
        seq[c].append(u)
    assert used == cap
    for c in range(S):
        assert [singles[w] for w in range(c, n, S)] == seq[c]


def test_hand_derived_slot_placement():
    # Six one-page-multiple rows, Hkv = 1, 2 CUs x 3 units: S = 6 = R, so step 4 keeps one
    # split each (pages 6, 5, 5, 4, 4, 3; 2 * 6 * 6 = 72 <= 3 * 27 = 81: balanced) and
    # step 9 lists b = 0..5.  Equal weights: 6 -> slot 0; 5 -> slot 1; 5 -> slot 1 (5 + 5
    # = 10 < 6 + 5); 4 -> slot 0 (10 < 14); 4 -> tie at 14, slot 0 (now full); 3 -> slot
    # 1.  Slot 0 holds b0, b3, b4 at positions 0, 2, 4, slot 1 holds b1, b2, b5 at 1, 3, 5.
    lens = [96, 80, 80, 64, 64, 48]
    unit = lambda b: (b, 0, 0, lens[b], 0, 1, 0, 1, -1, b, 0, lens[b] - 1)
    par = dict(num_cus=2, units_per_cu=3, min_split_pages=1)
    units, info = plan_ref(lens, None, 1, 4, PlanParams(**par))
    assert info["balanced"]
    assert units == [unit(b) for b in (0, 1, 3, 2, 4, 5)]
    # Slot 1 at half speed (weight 500): 6 -> slot 0 (6/1000 < 6/500); 5 -> slot 1
    # (5/500 = 0.010 < 11/1000); 5 -> slot 0 (11/1000 < 10/500); 4 -> slot 0 (15/1000 <
    # 9/500), which is then full; 4 and 3 -> slot 1.  Slot 0: b0, b2, b3; slot 1: b1, b4, b5.
    units, _ = plan_ref(lens, None, 1, 4, PlanParams(**par, xcd_weight=(1000, 500, 0, 0, 0, 0, 0, 0)))
    assert units == [unit(b) for b in (0, 1, 2, 4, 3, 5)]


def test_hand_derived_xcd_queue_placement():
    # Ten rows of 10, 9, ..., 1 pages, Hkv = 1, one CU x 2 units: more rows than R = 2, so
    # the chunk rule keeps one split each (chunk = ceil(55 / 2) = 28 pages) and step 11
    # deals the ten units to the 8 XCD queues: queues 0 and 1 take positions {0, 8} and
    # {1, 9}, queues 2-7 one position each.  Equal weights: 10, 9, ..., 3 go to queues
    # 0..7 in turn; 2 -> queue 1 (9 + 2 < 10 + 2); 1 -> queue 0, the only one with room.
    pages = list(range(10, 0, -1))
    lens = [16 * p for p in pages]
    unit = lambda b: (b, 0, 0, lens[b], 0, 1, 0, 1, -1, b, 0, lens[b] - 1)
    par = dict(num_cus=1, units_per_cu=2, min_split_pages=1)
    units, info = plan_ref(lens, None, 1, 4, PlanParams(**par))
    assert not info["balanced"]
    assert units == [unit(b) for b in (0, 1, 2, 3, 4, 5, 6, 7, 9, 8)]
    # Odd XCDs at half weight: 10, 9, 8, 7 -> even queues 0, 2, 4, 6 (x / 1000 < x / 500);
    # 6 -> queue 1 (6 / 500 = 0.012 < 16 / 1000); 5, 4, 3 -> queues 3, 5, 7 (below 15, 14,
    # 13 / 1000 on queue 0); 2 -> queue 0 (12 / 1000 < 8 / 500); 1 -> queue 1, the last room.
    units, _ = plan_ref(lens, None, 1, 4,
                        PlanParams(**par, xcd_weight=(1000, 500) * 4))
    assert units == [unit(b) for b in (0, 4, 1, 5, 2, 6, 3, 7, 8, 9)]


def test_slot_placement_catches_a_planted_mistake(monkeypatch):
    # A placement that ignores the weights breaks the replay check.
    import oracle.plan as op
    lens = [96, 80, 80, 64, 64, 48]
    params = PlanParams(num_cus=2, units_per_cu=3, min_split_pages=1,
                        xcd_weight=(1000, 500, 0, 0, 0, 0, 0, 0))
    real = op._place_on_slots
    monkeypatch.setattr(op, "_place_on_slots",
                        lambda units, p, S: real(units, dataclasses.replace(p, xcd_weight=(0,) * 8), S))
    units, _ = op.plan_ref(lens, None, 1, 4, params)
    with pytest.raises(AssertionError):
        check_slot_placement(units, params, 2)


def check_invariants(seq_lens, q_lens, hkv, group, params):
    units, info = plan_ref(seq_lens, q_lens, hkv, group, params)
    B = len(seq_lens)
    C = [1] * B if q_lens is None else list(q_lens)
    singles = units[:info["n_single"]]
    chunks = units[info["n_single"]:]
    assert all(u[F["kind"]] == 0 for u in singles) and all(u[F["kind"]] == 1 for u in chunks)
    # ordering: step 11's slots (CUs for a one-wave plan, else XCD queues), each slot's
    # units in step 9's descending KV order
    if singles:
        S = params.num_cus if info["balanced"] else 8
        check_slot_placement(singles, params, S)
        for c in range(S):
            kv = [u[3] - u[2] for u in singles[c::S]]
            assert kv == sorted(kv, reverse=True)
    # chunk units: per-XCD queues, each uncut (b, g) group inside one queue and contiguous
    # in it, longest tiles of the queue's parts first (costs in 64-key steps)
    cost = lambda u: -(-(u[3] - u[2]) // 64)
    lens = info["xcd_queue_lens"]
    assert sum(lens) == len(chunks)
    seen = {}
    pos = 0
    qcost = []
    for n in lens:
        q = chunks[pos:pos + n]
        pos += n
        qcost.append(sum(cost(u) for u in q))
        for u in q:
            seen.setdefault(u[:2], []).append((len(qcost) - 1, pos - n + q.index(u)))
    if chunks:
        total = sum(cost(u) for u in chunks)
        fair = -(-total // 8)
        for key, where in seen.items():
            gcost = sum(cost(u) for u in chunks if u[:2] == key)
            if gcost <= fair:
                # an uncut group: one queue, contiguous, its tiles by descending cost
                assert len({x for x, _ in where}) == 1
                idx = sorted(i for _, i in where)
                assert idx == list(range(idx[0], idx[0] + len(idx)))
                c = [cost(chunks[i]) for i in idx]
                assert c == sorted(c, reverse=True)
        pos = 0
        for n in lens:
            q = chunks[pos:pos + n]
            pos += n
            # runs of one (b, g): each run opens with its longest tile, and the runs open
            # in non-increasing cost
            heads = [cost(u) for i, u in enumerate(q) if i == 0 or q[i - 1][:2] != u[:2]]
            assert heads == sorted(heads, reverse=True)
        # dealing bound: queues differ by at most one part, and a part costs at most
        # F plus one tile
        assert max(qcost) - min(qcost) <= fair + max(cost(u) for u in chunks)
    # single rows: splits tile [0, L) exactly, page aligned, non-empty unless L = 0
    slots = set()
    for b in range(B):
        if C[b] != 1:
            continue
        for g in range(hkv):
            us = sorted((u for u in singles if u[0] == b and u[1] == g), key=lambda u: u[6])
            n = us[0][F["n_splits"]]
            assert len(us) == n and 1 <= n <= params.max_splits
            assert [u[6] for u in us] == list(range(n))
            assert us[0][2] == 0 and us[-1][3] == seq_lens[b]
            for a, c in zip(us[:-1], us[1:]):
                assert a[3] == c[2] and c[2] % 16 == 0
            if seq_lens[b] > 0:
                assert all(u[3] > u[2] for u in us)
            for u in us:
                if n > 1:
                    s = u[F["part_base"]] + u[6]
                    assert 0 <= s < info["n_partial_slots"] and s not in slots
                    slots.add(s)
                else:
                    assert u[F["part_base"]] == -1
    assert len(slots) == info["n_partial_slots"]
    # chunk rows: tiles cover [0, C) and see keys up to P + q_end
    row0 = np.concatenate([[0], np.cumsum(C)])
    for b in range(B):
        if C[b] == 1:
            continue
        for g in range(hkv):
            us = sorted((u for u in chunks if u[0] == b and u[1] == g), key=lambda u: u[4])
            assert us[0][4] == 0 and us[-1][5] == C[b]
            for a, c in zip(us[:-1], us[1:]):
                assert a[5] == c[4]
            for u in us:
                P = seq_lens[b] - C[b]
                assert u[F["prior"]] == P and u[3] == P + u[5] and u[2] == 0
                assert u[F["row0"]] == row0[b] and u[5] - u[4] <= info["q_tile"]
    total = sum(u[3] - u[2] for u in singles)
    assert total == hkv * sum(seq_lens[b] for b in range(B) if C[b] == 1)
    if info["balanced"]:
        # one wave: at most S units, and the largest piece within 1.5x the mean share
        S = params.num_cus * params.units_per_cu
        R = S // hkv
        assert len(singles) <= R * hkv <= S
        pages = [-(-(u[3] - u[2]) // 16) for u in singles]
        wp = sum(-(-seq_lens[b] // 16) for b in range(B) if C[b] == 1)
        assert 2 * max(pages) * R <= 3 * wp
    return units, info


@pytest.mark.parametrize("seed", range(8))
def test_plan_invariants_random(seed):
    rng = np.random.default_rng(seed)
    B = int(rng.integers(1, 40))
    lens = rng.choice([0, 1, 15, 16, 17, 31, 33, 500, 4096, 131072], size=B).tolist()
    lens += rng.integers(1, 70000, size=3).tolist()
    params = PlanParams(num_cus=int(rng.integers(1, 300)), units_per_cu=int(rng.integers(1, 4)),
                        min_split_pages=int(rng.integers(1, 64)), max_splits=int(rng.integers(1, 100)))
    check_invariants(lens, None, int(rng.choice([1, 2, 8])), 4, params)
    C = rng.choice([1, 1, 1, 2, 64, 1000], size=len(lens)).tolist()
    lens2 = [max(L, c) for L, c in zip(lens, C)]
    check_invariants(lens2, C, 2, int(rng.choice([1, 4, 7, 8, 16])), params)


def test_longtail_batch_splits_only_the_tail():
    from paper_2606_03077_amd import workloads as wl
    lens, _ = wl.draw_lengths(wl.WORKLOADS["longtail"], np.random.default_rng(26063))
    units, info = check_invariants(lens.tolist(), None, 8, 4, PlanParams())
    split_rows = {u[0] for u in units if u[F["n_splits"]] > 1}
    assert split_rows and all(lens[b] > 16 * info["chunk_pages"] for b in split_rows)


def test_straggler_batch_splits_every_row():
    lens = [98304, 131072, 100000, 120000]
    units, info = check_invariants(lens, None, 8, 8, PlanParams())
    assert all(u[F["n_splits"]] >= 8 for u in units)
    assert len(units) >= 256


def test_hand_derived_one_wave_apportionment():
    # L = [160, 48, 1600] -> pages [10, 3, 100]; Hkv = 2, S = 4 * 4 = 16, R = 8.
    # Three rows fit.  Greedy from n = [1, 1, 1]: row 2's share 100 > 10 > 3 takes splits
    # until n = [1, 1, 6] (shares 10, 3, 16.7; sum 8 = R).  Largest piece ceil(100/6) = 17
    # and 2 * 17 * 8 = 272 <= 3 * 113 = 339, so it is kept (the chunk rule would have cut
    # row 2 into ceil(100 / 15) = 7).  Row 2's pages split at floor(j * 100 / 6) =
    # 0, 16, 33, 50, 66, 83, 100: tokens 256, 272, 272, 256, 272, 272.
    units, info = plan_ref([160, 48, 1600], None, 2, 4,
                           PlanParams(num_cus=4, units_per_cu=4, min_split_pages=2, max_splits=8))
    cut = [0, 16, 33, 50, 66, 83, 100]

    def u(b, g, j):
        if b == 2:
            return (2, g, 16 * cut[j], 16 * cut[j + 1], 0, 1, j, 6, 6 * g, 2, 0, 1599)
        L = [160, 48][b]
        return (b, g, 0, L, 0, 1, 0, 1, -1, b, 0, L - 1)

    expect = ([u(2, g, j) for g in (0, 1) for j in (1, 2, 4, 5)]
              + [u(2, g, j) for g in (0, 1) for j in (0, 3)]
              + [u(0, 0, 0), u(0, 1, 0), u(1, 0, 0), u(1, 1, 0)])
    expect = sorted(expect, key=lambda x: (-(x[3] - x[2]), x[0], x[1], x[6]))
    assert expect[:8] == [u(2, 0, 1), u(2, 0, 2), u(2, 0, 4), u(2, 0, 5),
                          u(2, 1, 1), u(2, 1, 2), u(2, 1, 4), u(2, 1, 5)]
    assert units == expect
    assert info["balanced"] and info["n_partial_slots"] == 12 and info["chunk_pages"] == 15


def test_hand_derived_unbalanced_falls_back_to_chunk_rule():
    # pages [40, 1, 1], Hkv = 1, S = R = 4, min_split 16.  Greedy: n = [2, 1, 1], largest
    # piece 20, and 2 * 20 * 4 = 160 > 3 * 42 = 126: not balanced.  Chunk rule:
    # chunk = max(16, ceil(42 / 4)) = 16, n = [ceil(40 / 16), 1, 1] = [3, 1, 1]; row 0's
    # pages split at floor(j * 40 / 3) = 0, 13, 26, 40.
    units, info = plan_ref([640, 16, 16], None, 1, 1,
                           PlanParams(num_cus=1, units_per_cu=4, min_split_pages=16, max_splits=8))
    assert units == [
        (0, 0, 416, 640, 0, 1, 2, 3, 0, 0, 0, 639),
        (0, 0, 0, 208, 0, 1, 0, 3, 0, 0, 0, 639),
        (0, 0, 208, 416, 0, 1, 1, 3, 0, 0, 0, 639),
        (1, 0, 0, 16, 0, 1, 0, 1, -1, 1, 0, 15),
        (2, 0, 0, 16, 0, 1, 0, 1, -1, 2, 0, 15),
    ]
    assert not info["balanced"] and info["chunk_pages"] == 16


@pytest.mark.parametrize("seed", range(40))
def test_apportionment_is_optimal_by_brute_force(seed):
    """The greedy attains the smallest possible largest piece over every admissible
    choice of split counts with the same budget (exhaustive search on tiny inputs)."""
    import itertools
    from oracle.plan import _apportion, _ceil_div
    rng = np.random.default_rng(1000 + seed)
    B = int(rng.integers(1, 5))
    pages = [int(x) for x in rng.integers(0, 13, size=B)]
    params = PlanParams(num_cus=1, units_per_cu=1, min_split_pages=int(rng.integers(1, 4)),
                        max_splits=int(rng.integers(1, 5)))
    R = int(rng.integers(B, 3 * B + 3))
    single = list(range(B))
    n = _apportion(pages, single, R, params)
    ub = [max(1, min(params.max_splits, p // params.min_split_pages)) for p in pages]
    assert all(1 <= n[b] <= ub[b] for b in single)
    assert sum(n.values()) == min(R, sum(ub))
    best = min(max(_ceil_div(p, k) for p, k in zip(pages, ks))
               for ks in itertools.product(*[range(1, u + 1) for u in ub]) if sum(ks) <= R)
    assert max(_ceil_div(pages[b], n[b]) for b in single) == best
