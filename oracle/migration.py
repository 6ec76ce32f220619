"""Request migration across tensor-parallel degrees: the head reshard of offloaded KV.

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__``).

Sec. 5 (migration Steps 1-3): a paused request's KV pages are copied to host memory
(Step 1), regrouped along the attention-head axis for the target bucket's TP degree
while the tool runs (Step 2), and each target GPU loads its own head shard when the
tool returns (Step 3).  Step 2 is stated for both directions: raising TP k-fold cuts
each source partition into k pieces of contiguous heads, lowering it k-fold joins k
adjacent partitions.  Both are the same operation on the full head axis: join all
source partitions in order, then cut the result into equal contiguous ranges.  Steps
1 and 3 only move bytes, so the oracle's view of them is "same values, other pages".

Arrays here are the logical page format [pages][heads][16][128] (uint16 bf16 bits), or
any array whose axis 1 is the head axis.
"""
from __future__ import annotations

import numpy as np


def reshard_heads(shards, n_dst: int):
    """Sec. 5, Step 2: join the source shards along heads, cut into n_dst equal ranges.

    ``shards`` lists arrays with the head axis at position 1, in head order (shard i holds
    the heads after those of shard i - 1).  Returns n_dst arrays; output j holds heads
    [j * H / n_dst, (j + 1) * H / n_dst) of the H joined heads.
    """
    full = np.concatenate([np.asarray(s) for s in shards], axis=1)
    H = full.shape[1]
    if n_dst <= 0 or H % n_dst:
        raise ValueError(f"{n_dst} shards do not divide {H} heads")
    h = H // n_dst
    return [full[:, j * h:(j + 1) * h].copy() for j in range(n_dst)]


def request_pages(pages, block_table_row, n_tokens: int):
    """The pages a request of n_tokens occupies, in token order (Step 1's payload)."""
    n = -(-int(n_tokens) // 16)
    return np.asarray(pages)[np.asarray(block_table_row[:n], dtype=np.int64)]


def query_heads_of_shard(j: int, n_dst: int, num_q_heads: int):
    """Query heads that travel with KV shard j: with query head h reading KV head h // G
    (grouped-query attention), the KV heads [j H / n, (j + 1) H / n) serve exactly the
    query heads [j Hq / n, (j + 1) Hq / n)."""
    h = num_q_heads // n_dst
    return slice(j * h, (j + 1) * h)
