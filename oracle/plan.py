"""The library's split-KV work partition, re-implemented in plain Python integers.

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__``).  The library builds its plan in host
C++; this file re-derives the same table from the written rule so that the two can be
compared entry by entry.

Why a partition at all: the paper finds that the longest tenth of trajectories takes
over half of rollout time (Sec. 2.2, "Long-tailed Rollout") and that stragglers set the
makespan (Sec. 1).  On one GPU the same imbalance appears inside a decode step: a few
very long sequences next to many short ones.  The rule below cuts long sequences into
page-aligned KV ranges so that all compute units stay busy, and merges the pieces by
their log-sum-exps.  The paper does not describe this step; the rule is the library's.

The rule
--------
Inputs: per-sequence KV length L_b (after this step's new tokens), query tokens C_b
(1 for decode), KV heads Hkv, group size G = Hq / Hkv, and parameters (compute units,
units per CU, minimum split size in pages, maximum splits, chunk query tile).

1. pages_b = ceil(L_b / 16).
2. Rows with C_b = 1 are *single* rows; rows with C_b > 1 are *chunk* rows.
3. S = num_cus * units_per_cu (units_per_cu is meant to be the number of decode
   workgroups that are resident on one compute unit at a time, so that S units form a
   single wave); R = floor(S / Hkv) split budget per KV head.
4. One-wave apportionment.  If the number of single rows is at most R, every single row
   starts with n_b = 1 split, and while sum n_b < R one more split goes to the single row
   with the largest pages_b / n_b (compared exactly, ties to the smallest b) among the
   rows that can still be split: n_b < max_splits and pages_b >= (n_b + 1) *
   min_split_pages.  It stops early when no row can be split.  This gives the smallest
   possible largest piece, max ceil(pages_b / n_b), for that many splits.  The result is
   kept when it is balanced, 2 * max_b ceil(pages_b / n_b) * R <= 3 * sum_b pages_b (the
   largest piece at most 1.5 times the mean share of a unit); otherwise, and whenever
   there are more single rows than R, step 5 decides instead.
5. Chunk rule: W = sum over single rows of pages_b * Hkv; chunk = max(min_split_pages,
   ceil(W / S)) (min_split_pages when W = 0);
   n_b = min(max_splits, max(1, ceil(pages_b / chunk))).
6. Split j of a single row covers pages [floor(j pages_b / n_b), floor((j+1) pages_b /
   n_b)), i.e. tokens [16 p0, min(16 p1, L_b)).  An empty sequence gets one empty unit.
7. A chunk row is cut into query tiles of T tokens (T = q_tile, or floor(256 / G) when
   q_tile = 0): tile k holds new tokens [kT, min(kT + T, C_b)) and keys
   [0, P_b + min(kT + T, C_b)), where P_b = L_b - C_b.  Tiles are not split along KV.
8. Every unit is repeated for each KV head g.
9. Single units are ordered by descending KV token count, ties by ascending (b, g, j).
   Chunk units are grouped per (b, g); a tile costs its key-loop steps,
   ceil((kv_end - kv_begin) / 64), and a group the sum of its tiles.  With
   F = ceil(total cost / 8), a group of cost c and m tiles is cut into
   n = min(m, ceil(c / F)) parts: its tile i (ascending q_begin) goes to part
   floor(S_i * n / c), S_i being the cost of the group's tiles before it; empty parts are
   dropped.  Parts, by descending cost (ties ascending (b, g, part)), are dealt to 8
   queues (one per XCD), each to the queue with the least accumulated cost (ties to the
   lowest queue).  Each queue then lists its parts by descending cost of their longest
   tile (ties ascending (b, g, part)), a part's tiles together by descending cost (ties
   ascending q_begin).
   The table lists all single units, then queue 0's tiles, queue 1's, ... queue 7's.
10. Single rows with n_b > 1 own n_b partial-result slots per KV head, allotted in
    ascending (b, g) order: part_base(b, g) = (slots of earlier split rows) + g * n_b.
    Units with n_b = 1 have part_base = -1.
11. The single units are placed on S slots.  The decode launch puts workgroup w on XCD
    w mod 8; when step 4 decided, every unit is resident at once and workgroups w,
    w + num_cus, ... share one CU, so S = num_cus; otherwise each XCD runs its workgroups
    as its CUs free up, so S = 8.  With n single units, slot c holds the positions w < n
    with w mod S = c; its weight is xcd_weight[c mod 8] (1000 for 0).  A unit costs
    ceil(kv_end / 16) - floor(kv_begin / 16) pages.  Taking the units in step 9's order,
    each goes to the slot with room whose (load + cost) / weight is smallest (exact
    comparison, ties to the smaller c); the r-th unit of slot c is listed at position
    c + r * S.

Each unit is 12 int32 fields, in the order of ``UNIT_FIELDS``.
"""
from __future__ import annotations

import dataclasses

UNIT_FIELDS = ("b", "g", "kv_begin", "kv_end", "q_begin", "q_end", "split", "n_splits",
               "part_base", "row0", "kind", "prior")
KIND_SINGLE = 0
KIND_CHUNK = 1
PAGE = 16
NUM_XCDS = 8
CHUNK_STEP_KEYS = 64   # keys per step of the chunk kernel's key loop (step 9's tile cost)


@dataclasses.dataclass(frozen=True)
class PlanParams:
    num_cus: int = 256
    units_per_cu: int = 3
    min_split_pages: int = 16
    max_splits: int = 64
    q_tile: int = 0
    xcd_weight: tuple = (0, 0, 0, 0, 0, 0, 0, 0)


def _ceil_div(a: int, b: int) -> int:
    return -(-a // b)


def _apportion(pages, single, R, params):
    """Step 4's greedy: split counts n_b (sum at most R) of the single rows."""
    n = {b: 1 for b in single}
    total = len(single)

    def can_split(b):
        return n[b] < params.max_splits and pages[b] >= (n[b] + 1) * params.min_split_pages

    while total < R:
        best = None
        for b in single:   # ascending b, replaced only on a strictly larger share
            if can_split(b) and (best is None or pages[b] * n[best] > pages[best] * n[b]):
                best = b
        if best is None:
            break
        n[best] += 1
        total += 1
    return n


def _one_wave_splits(pages, single, R, params):
    """Step 4: split counts of the single rows for one wave of R units per KV head, or
    None when there are no single rows, they do not fit, or the result is unbalanced."""
    if not single or len(single) > R:
        return None
    n = _apportion(pages, single, R, params)
    largest = max(_ceil_div(pages[b], n[b]) for b in single)
    if 2 * largest * R > 3 * sum(pages[b] for b in single):
        return None
    return n


def _place_on_slots(units, params, S):
    """Step 11: deal the units to S slots, each to the slot with room that minimises
    (load + cost) / weight, scanning every slot."""
    n = len(units)
    weight = [x if x > 0 else 1000 for x in params.xcd_weight]
    cap = [len(range(c, n, S)) for c in range(S)]
    load = [0] * S
    placed = [[] for _ in range(S)]
    for u in units:
        cost = _ceil_div(u[3], PAGE) - u[2] // PAGE
        best = None
        for c in range(S):
            if len(placed[c]) == cap[c]:
                continue
            # (load_c + cost) / w_c < (load_best + cost) / w_best, cross-multiplied
            if best is None or ((load[c] + cost) * weight[best % NUM_XCDS]
                                < (load[best] + cost) * weight[c % NUM_XCDS]):
                best = c
        placed[best].append(u)
        load[best] += cost
    out = [None] * n
    for c in range(S):
        for r, u in enumerate(placed[c]):
            out[c + r * S] = u
    return out


def plan_ref(seq_lens, q_lens, num_kv_heads: int, group: int, params: PlanParams):
    """Returns (units: list of 12-tuples, info: dict) following the rule above."""
    L = [int(x) for x in seq_lens]
    B = len(L)
    C = [1] * B if q_lens is None else [int(x) for x in q_lens]
    Hkv = int(num_kv_heads)
    pages = [_ceil_div(x, PAGE) for x in L]
    row0 = [0] * B
    acc = 0
    for b in range(B):
        row0[b] = acc
        acc += C[b]

    single = [b for b in range(B) if C[b] == 1]
    chunked = [b for b in range(B) if C[b] > 1]

    S = params.num_cus * params.units_per_cu
    R = S // Hkv
    n_split = _one_wave_splits(pages, single, R, params)
    balanced = n_split is not None
    W = sum(pages[b] * Hkv for b in single)
    chunk = max(params.min_split_pages, _ceil_div(W, S)) if W > 0 else params.min_split_pages
    if not balanced:
        n_split = {}
        for b in single:
            n_split[b] = min(params.max_splits, max(1, _ceil_div(pages[b], chunk)))

    part_base = {}
    slots = 0
    for b in range(B):
        if b in n_split and n_split[b] > 1:
            for g in range(Hkv):
                part_base[(b, g)] = slots + g * n_split[b]
            slots += n_split[b] * Hkv

    singles = []
    for b in single:
        n = n_split[b]
        for g in range(Hkv):
            for j in range(n):
                p0 = (j * pages[b]) // n
                p1 = ((j + 1) * pages[b]) // n
                t0 = PAGE * p0
                t1 = min(PAGE * p1, L[b])
                singles.append((b, g, t0, t1, 0, 1, j, n, part_base.get((b, g), -1),
                                row0[b], KIND_SINGLE, L[b] - 1))
    singles.sort(key=lambda u: (-(u[3] - u[2]), u[0], u[1], u[6]))
    if singles:
        singles = _place_on_slots(singles, params, params.num_cus if balanced else NUM_XCDS)

    T = params.q_tile if params.q_tile > 0 else 256 // group
    chunks = []
    for b in chunked:
        P = L[b] - C[b]
        for g in range(Hkv):
            for k in range(_ceil_div(C[b], T)):
                q0 = k * T
                q1 = min(q0 + T, C[b])
                chunks.append((b, g, 0, P + q1, q0, q1, 0, 1, -1, row0[b], KIND_CHUNK, P))
    def cost(u):
        return _ceil_div(u[3] - u[2], CHUNK_STEP_KEYS)

    groups = {}
    for u in chunks:                      # built in ascending (b, g, q_begin)
        groups.setdefault((u[0], u[1]), []).append(u)
    fair = _ceil_div(sum(cost(u) for u in chunks), NUM_XCDS) if chunks else 1
    parts = {}
    for (b, g), tiles in groups.items():
        c = sum(cost(u) for u in tiles)
        n = min(len(tiles), _ceil_div(c, fair))
        before = 0
        for u in tiles:
            parts.setdefault((b, g, before * n // c), []).append(u)
            before += cost(u)
    order = sorted(parts, key=lambda k: (-sum(cost(u) for u in parts[k]), k))
    qparts = [[] for _ in range(NUM_XCDS)]
    qcost = [0] * NUM_XCDS
    for k in order:
        x = min(range(NUM_XCDS), key=lambda i: (qcost[i], i))
        qcost[x] += sum(cost(u) for u in parts[k])
        qparts[x].append(k)
    tiles = {k: sorted(parts[k], key=lambda u: (-cost(u), u[4])) for k in parts}
    queues = []
    for ks in qparts:
        ks = sorted(ks, key=lambda k: (-cost(tiles[k][0]), k))
        queues.append([u for k in ks for u in tiles[k]])
    chunks = [u for q in queues for u in q]

    info = {"n_single": len(singles), "n_chunk": len(chunks), "n_partial_slots": slots,
            "chunk_pages": chunk, "q_tile": T, "work_pages": W, "balanced": balanced,
            "xcd_queue_lens": [len(q) for q in queues]}
    return singles + chunks, info
