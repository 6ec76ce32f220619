"""Plain float64 softmax attention over a paged KV cache (test infrastructure only).

Inputs are the generator's logical format: bf16 bit patterns (uint16) with pages laid
out ``[num_pages, Hkv, 16, 128]``; token ``t`` of sequence ``b`` sits in page
``block_table[b, t // 16]`` at slot ``t % 16``.  Nothing here models the library's device
layout, its blocking, its splitting or its online rescaling: the library must reach the
same numbers by its own route.

Readings of what the paper leaves open (the paper names KV caches and attention
operators, Sec. 4.5 and Sec. 5, but never defines them):

* softmax scale ``s`` is the float32 value passed by the caller, widened to float64;
* query head ``h`` reads KV head ``h // G`` with ``G = Hq / Hkv`` (contiguous groups);
* decode: ``seq_lens[b]`` counts the current token, whose K/V is already cached, so the
  query attends keys ``[0, L_b)``;
* append: sequence ``b`` holds ``P_b = L_b - C_b`` cached tokens; new token ``i``
  (position ``P_b + i``) is written to the cache and attends keys ``[0, P_b + i]``,
  itself included;
* an empty key set gives ``o = 0`` and ``LSE = -inf``;
* LSE is the natural logarithm of the softmax denominator including the running
  maximum, ``LSE = m + log(sum_j exp(z_j - m))``.
"""
from __future__ import annotations

import numpy as np

PAGE = 16


def bf16_bits_to_f64(bits) -> np.ndarray:
    """Exact value of bf16 bit patterns as float64 (bf16 is the top half of a float32)."""
    b = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
    return b.view(np.float32).astype(np.float64)


def gather_tokens(pages, block_table_row, kv_head: int, n_tokens: int) -> np.ndarray:
    """Logical K (or V) rows 0..n_tokens-1 of one sequence and one KV head.

    Follows the paged-cache indirection: token t is slot t % 16 of page
    block_table_row[t // 16].  Returns the raw bf16 bit patterns, shape [n_tokens, 128].
    """
    out = np.empty((n_tokens, pages.shape[-1]), dtype=np.uint16)
    for t in range(0, n_tokens, PAGE):
        page = int(block_table_row[t // PAGE])
        n = min(PAGE, n_tokens - t)
        out[t:t + n] = pages[page, kv_head, :n, :]
    return out


def attend(q_rows: np.ndarray, keys: np.ndarray, values: np.ndarray, scale: float,
           visible: np.ndarray | None = None):
    """Softmax attention of query rows over keys, straight from the definition.

    q_rows [R, d], keys [N, d], values [N, d] in float64; ``visible`` [R, N] bool marks
    which keys each row may see (all, if None).  Two passes: the maximum logit m, then
    the exponentials relative to it.  Returns (o [R, d], lse [R]).
    """
    q_rows = np.asarray(q_rows, dtype=np.float64)
    R, d = q_rows.shape
    N = keys.shape[0]
    o = np.zeros((R, d), dtype=np.float64)
    lse = np.full(R, -np.inf, dtype=np.float64)
    if N == 0 or R == 0:
        return o, lse
    z = float(scale) * (q_rows @ np.asarray(keys, np.float64).T)          # [R, N]
    if visible is not None:
        z = np.where(visible, z, -np.inf)
    m = z.max(axis=1)                                                     # [R]
    ok = np.isfinite(m)
    zs = np.where(ok[:, None], z - np.where(ok, m, 0.0)[:, None], -np.inf)
    e = np.exp(zs)                                                        # exp(-inf) = 0
    l = e.sum(axis=1)
    o[ok] = (e[ok] @ np.asarray(values, np.float64)) / l[ok, None]
    lse[ok] = m[ok] + np.log(l[ok])
    return o, lse


def decode_ref(q, k_pages, v_pages, block_table, seq_lens, scale, batch_rows=None):
    """One query token per sequence over its whole paged KV history.

    q: uint16 [B, Hq, d]; pages uint16 [P, Hkv, 16, d]; block_table int [B, *];
    seq_lens int [B].  Returns (o float64 [B, Hq, d], lse float64 [B, Hq]).
    ``batch_rows`` restricts the work to a subset of sequences (others stay zero / -inf).
    """
    B, Hq, d = q.shape
    Hkv = k_pages.shape[1]
    G = Hq // Hkv
    o = np.zeros((B, Hq, d), dtype=np.float64)
    lse = np.full((B, Hq), -np.inf, dtype=np.float64)
    rows = range(B) if batch_rows is None else batch_rows
    for b in rows:
        L = int(seq_lens[b])
        for g in range(Hkv):
            K = bf16_bits_to_f64(gather_tokens(k_pages, block_table[b], g, L))
            V = bf16_bits_to_f64(gather_tokens(v_pages, block_table[b], g, L))
            heads = slice(g * G, (g + 1) * G)
            ob, lb = attend(bf16_bits_to_f64(q[b, heads]), K, V, scale)
            o[b, heads] = ob
            lse[b, heads] = lb
    return o, lse


def write_new_tokens(k_pages, v_pages, k_new, v_new, block_table, seq_lens, q_lens):
    """Cache write of an append step: new token i of sequence b goes to position P_b + i.

    Returns new page arrays (inputs untouched).  Position t maps to page
    block_table[b, t // 16], slot t % 16.
    """
    k_out = np.array(k_pages, copy=True)
    v_out = np.array(v_pages, copy=True)
    row = 0
    for b in range(len(seq_lens)):
        C = int(q_lens[b])
        P = int(seq_lens[b]) - C
        for i in range(C):
            t = P + i
            page = int(block_table[b, t // PAGE])
            k_out[page, :, t % PAGE, :] = k_new[row + i]
            v_out[page, :, t % PAGE, :] = v_new[row + i]
        row += C
    return k_out, v_out


def append_ref(q, k_new, v_new, k_pages, v_pages, block_table, seq_lens, q_lens, scale,
               batch_rows=None):
    """Causal attention of appended tokens (a tool-output chunk, or one decode token).

    Sequence b appends C_b = q_lens[b] tokens after P_b = seq_lens[b] - C_b cached ones.
    Query rows are packed: sequence b's rows start at sum(q_lens[:b]).  New token i sees
    keys [0, P_b + i] (itself included).  Returns (o [sum C, Hq, d], lse [sum C, Hq],
    k_pages_after, v_pages_after).
    """
    n_rows, Hq, d = q.shape
    Hkv = k_pages.shape[1]
    G = Hq // Hkv
    k_after, v_after = write_new_tokens(k_pages, v_pages, k_new, v_new, block_table,
                                        seq_lens, q_lens)
    o = np.zeros((n_rows, Hq, d), dtype=np.float64)
    lse = np.full((n_rows, Hq), -np.inf, dtype=np.float64)
    starts = np.concatenate([[0], np.cumsum(np.asarray(q_lens, np.int64))])
    rows = range(len(seq_lens)) if batch_rows is None else batch_rows
    for b in rows:
        L = int(seq_lens[b])
        C = int(q_lens[b])
        P = L - C
        r0 = int(starts[b])
        # visible[i, j]: key j is at or before the query's own position P + i
        visible = np.arange(L)[None, :] <= (P + np.arange(C))[:, None]
        for g in range(Hkv):
            K = bf16_bits_to_f64(gather_tokens(k_after, block_table[b], g, L))
            V = bf16_bits_to_f64(gather_tokens(v_after, block_table[b], g, L))
            for j in range(G):
                h = g * G + j
                ob, lb = attend(bf16_bits_to_f64(q[r0:r0 + C, h]), K, V, scale, visible)
                o[r0:r0 + C, h] = ob
                lse[r0:r0 + C, h] = lb
    return o, lse, k_after, v_after


def merge_ref(o_parts, lse_parts):
    """Combine attention results over disjoint key subsets by their log-sum-exps.

    o_parts [n, ..., d] (each normalised over its own subset), lse_parts [n, ...].
    With M = max_j lse_j: lse = M + log(sum_j exp(lse_j - M)) and
    o = sum_j exp(lse_j - lse) o_j.  Subsets with lse_j = -inf (no keys) contribute
    nothing; if every subset is empty, o = 0 and lse = -inf.
    """
    o_parts = np.asarray(o_parts, dtype=np.float64)
    lse_parts = np.asarray(lse_parts, dtype=np.float64)
    M = lse_parts.max(axis=0)
    ok = np.isfinite(M)
    Ms = np.where(ok, M, 0.0)
    w = np.where(np.isfinite(lse_parts), np.exp(lse_parts - Ms), 0.0)
    s = w.sum(axis=0)
    lse = np.where(ok, Ms + np.log(np.where(ok, s, 1.0)), -np.inf)
    coef = np.where(ok, w / np.where(ok, s, 1.0), 0.0)
    o = (coef[..., None] * o_parts).sum(axis=0)
    return o, lse
