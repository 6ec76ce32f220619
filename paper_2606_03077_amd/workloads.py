"""Seeded synthetic rollout batches for ragged paged-KV decode / append attention.

This module only draws inputs: lengths, a shuffled block table, bf16 query / key /
value values and NaN sentinels.  It holds none of the attention arithmetic; both the
fp64 oracle (test infrastructure) and the HIP path consume what it returns.

Workload shapes stand in for the paper's agentic-RL rollout traffic: long-tailed
trajectory lengths where the longest tenth dominates rollout time (Sec. 2.2, "Long-tailed
Rollout"), a 40,960-token context ceiling (Sec. 7, Setup) that the straggler batches
deliberately exceed, and tool outputs appended mid-trajectory (Sec. 1; Sec. 5, Phase 2
and Step 3).  The paper's datasets (Search-R1, R2E-Gym, DAPO-Math-17K) are not used;
these distributions replace them.

Logical paged-KV format used for every returned cache (the library converts it to its
own device layout with its pack entry point):

* ``k_pages`` / ``v_pages``: uint16 bf16 bit patterns, shape ``[num_pages, Hkv, 16, 128]``
  (page, kv head, slot within page, channel).
* token ``t`` of sequence ``b`` lives in page ``block_table[b, t // 16]``, slot ``t % 16``.
* slots that hold no token, and every spare page, contain bf16 NaN (0x7FC0).
* unused block-table entries point at a spare (all-NaN) page.

Recipe (fixed, so that every stored number can be regenerated):

* seed = 26060 + config index (1..6), numpy PCG64 (``numpy.random.default_rng``);
* draw order: lengths, chunk lengths, mixture positions, page permutation, q, K, V,
  k_new, v_new;
* value draws: standard normal in float32, rounded to bf16 with round-to-nearest-even;
  each array draws one child seed from the batch generator and fills chunks of 2**22
  elements from PCG64(SeedSequence([child seed, chunk index]));
* "uniform in [a, b]" is inclusive; lognormal lengths are
  ``clip(rint(exp(ln(median) + sigma * z)), lo, hi)``; Pareto lengths are
  ``min(floor(xm * U ** (-1 / alpha)), cap)`` with ``U = 1 - uniform[0, 1)`` in (0, 1];
* mixture counts are exact (not Bernoulli) and placed by a seeded permutation;
* the physical page pool has ``ceil(0.01 * needed)`` (at least one) spare pages; physical
  page ids are a seeded permutation of the pool, handed out in logical order.
"""
from __future__ import annotations

import dataclasses
import math
import os
from typing import Optional

import numpy as np

PAGE = 16
HEAD_DIM = 128
BF16_NAN = np.uint16(0x7FC0)


@dataclasses.dataclass(frozen=True)
class Workload:
    """Shape recipe of one synthetic batch."""

    name: str
    index: int
    batch: int
    num_q_heads: int
    num_kv_heads: int
    description: str
    append: bool = False

    @property
    def seed(self) -> int:
        return 26060 + self.index

    @property
    def group(self) -> int:
        return self.num_q_heads // self.num_kv_heads


WORKLOADS = {
    "tiny": Workload("tiny", 1, 8, 8, 2,
                     "decode, B=8, Hq=8, Hkv=2, lengths U[16,512]"),
    "7b": Workload("7b", 2, 64, 28, 4,
                   "decode, B=64, Hq=28, Hkv=4, lengths lognormal(median 2048, sigma 1) "
                   "clipped to [64,32768]"),
    "longtail": Workload("longtail", 3, 256, 32, 8,
                         "decode, B=256, Hq=32, Hkv=8, 90% U[512,4096], 10% "
                         "Pareto(1.2) from 16384 capped at 65536"),
    "straggler": Workload("straggler", 4, 4, 64, 8,
                          "decode, B=4, Hq=64, Hkv=8, lengths U[98304,131072]"),
    "append": Workload("append", 5, 128, 32, 8,
                       "append, B=128, Hq=32, Hkv=8, prior lognormal(median 4096, "
                       "sigma 1) clipped to [256,32768]; 25% append U[64,1024] tokens, "
                       "75% append 1 token", append=True),
    # Recompute of a migrated request's KV on its target bucket: a full-context prefill
    # (empty prior) at the paper's 40,960-token maximum model length, with the 40 query /
    # 8 KV heads of its 14B policy (Sec. 5, cross-node migration; Sec. 7, Setup).
    "prefill": Workload("prefill", 6, 1, 40, 8,
                        "recompute prefill, B=1, Hq=40, Hkv=8, prior 0, 40960 new tokens",
                        append=True),
}


@dataclasses.dataclass
class Batch:
    """One generated batch (all host numpy arrays)."""

    workload: Workload
    seq_lens: np.ndarray        # int32 [B]: KV length after this step's tokens
    q_lens: np.ndarray          # int32 [B]: query tokens per sequence (1 for decode)
    cu_q_lens: np.ndarray       # int32 [B+1]: prefix sum of q_lens
    block_table: np.ndarray     # int32 [B, max_pages]
    k_pages: np.ndarray         # uint16 [num_pages, Hkv, 16, 128]
    v_pages: np.ndarray         # uint16 [num_pages, Hkv, 16, 128]
    q: np.ndarray               # uint16 [sum q_lens, Hq, 128]
    k_new: Optional[np.ndarray]  # uint16 [sum q_lens, Hkv, 128] (append only)
    v_new: Optional[np.ndarray]
    scale: float

    @property
    def prior_lens(self) -> np.ndarray:
        return (self.seq_lens - self.q_lens).astype(np.int32)

    @property
    def num_pages(self) -> int:
        return int(self.k_pages.shape[0])


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 to bf16 (round-to-nearest-even); returns the uint16 bit patterns."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    rounded = u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))
    out = (rounded >> np.uint32(16)).astype(np.uint16)
    nan = np.isnan(x)
    if nan.any():
        out[nan] = BF16_NAN
    return out


def bf16_bits_to_f32(bits: np.ndarray) -> np.ndarray:
    """Exact widening of bf16 bit patterns to float32."""
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


_CHUNK = 1 << 22


def _fill_chunk(child_seed: int, index: int, out: np.ndarray) -> None:
    g = np.random.Generator(np.random.PCG64(np.random.SeedSequence([child_seed, index])))
    out[:] = f32_to_bf16_bits(g.standard_normal(out.shape[0], dtype=np.float32))


def normal_bf16(rng: np.random.Generator, shape) -> np.ndarray:
    """N(0,1) float32 draws rounded to bf16, for one array of the batch.

    One 63-bit child seed is drawn from ``rng``; element chunk i (2**22 elements) comes
    from PCG64(SeedSequence([child_seed, i])).  The values therefore depend only on the
    seed and the shape, not on how many threads fill the chunks.
    """
    n = int(np.prod(shape))
    out = np.empty(n, dtype=np.uint16)
    child = int(rng.integers(0, 2 ** 63 - 1))
    starts = range(0, n, _CHUNK)
    if n > 4 * _CHUNK:
        import concurrent.futures as cf
        workers = min(16, len(os.sched_getaffinity(0)))
        with cf.ThreadPoolExecutor(max_workers=workers) as ex:
            list(ex.map(lambda i: _fill_chunk(child, i, out[i * _CHUNK:(i + 1) * _CHUNK]),
                        range(len(starts))))
    else:
        for i, s0 in enumerate(starts):
            _fill_chunk(child, i, out[s0:s0 + _CHUNK])
    return out.reshape(shape)


def _uniform_int(rng, lo, hi, n):
    return rng.integers(lo, hi, size=n, endpoint=True).astype(np.int64)


def _lognormal_len(rng, median, sigma, lo, hi, n):
    z = rng.standard_normal(n)
    return np.clip(np.rint(np.exp(math.log(median) + sigma * z)), lo, hi).astype(np.int64)


def _pareto_len(rng, xm, alpha, cap, n):
    u = 1.0 - rng.random(n)  # (0, 1]
    return np.minimum(np.floor(xm * u ** (-1.0 / alpha)), cap).astype(np.int64)


def draw_lengths(w: Workload, rng: np.random.Generator):
    """Returns (seq_lens, q_lens) as int64 arrays, following the recipe order."""
    B = w.batch
    if w.name == "tiny":
        return _uniform_int(rng, 16, 512, B), np.ones(B, np.int64)
    if w.name == "7b":
        return _lognormal_len(rng, 2048, 1.0, 64, 32768, B), np.ones(B, np.int64)
    if w.name == "longtail":
        n_tail = int(round(0.1 * B))
        body = _uniform_int(rng, 512, 4096, B - n_tail)
        tail = _pareto_len(rng, 16384, 1.2, 65536, n_tail)
        pos = rng.permutation(B)
        lens = np.empty(B, np.int64)
        lens[pos[:n_tail]] = tail
        lens[pos[n_tail:]] = body
        return lens, np.ones(B, np.int64)
    if w.name == "straggler":
        return _uniform_int(rng, 98304, 131072, B), np.ones(B, np.int64)
    if w.name == "prefill":
        return np.full(B, 40960, np.int64), np.full(B, 40960, np.int64)
    if w.name == "append":
        prior = _lognormal_len(rng, 4096, 1.0, 256, 32768, B)
        n_chunk = B // 4
        chunk = _uniform_int(rng, 64, 1024, n_chunk)
        pos = rng.permutation(B)
        q_lens = np.ones(B, np.int64)
        q_lens[pos[:n_chunk]] = chunk
        return prior + q_lens, q_lens
    raise KeyError(w.name)


def build_batch(w: Workload, seq_lens, q_lens, rng: np.random.Generator,
                spare_frac: float = 0.01, poison: bool = True) -> Batch:
    """Allocate pages, draw values and place NaN sentinels for given lengths.

    ``seq_lens`` is the KV length after the new tokens; the cache holds the first
    ``seq_lens - q_lens`` tokens (all of them for decode, where the current token's K/V
    has already been written).  For append, the slots of the new tokens are NaN until
    the library writes ``k_new`` / ``v_new`` there.
    """
    seq_lens = np.asarray(seq_lens, dtype=np.int64)
    q_lens = np.asarray(q_lens, dtype=np.int64)
    B = len(seq_lens)
    Hq, Hkv = w.num_q_heads, w.num_kv_heads
    pages_per_seq = (seq_lens + PAGE - 1) // PAGE
    needed = int(pages_per_seq.sum())
    spare = max(1, int(math.ceil(spare_frac * needed)))
    pool = needed + spare
    perm = rng.permutation(pool).astype(np.int64)
    max_pages = max(1, int(pages_per_seq.max()) if B else 1)
    spare_ids = perm[needed:]
    block_table = np.full((B, max_pages), spare_ids[0], dtype=np.int32)
    off = 0
    for b in range(B):
        n = int(pages_per_seq[b])
        block_table[b, :n] = perm[off:off + n]
        off += n

    n_q = int(q_lens.sum())
    q = normal_bf16(rng, (n_q, Hq, HEAD_DIM))
    k_pages = normal_bf16(rng, (pool, Hkv, PAGE, HEAD_DIM))
    v_pages = normal_bf16(rng, (pool, Hkv, PAGE, HEAD_DIM))
    k_new = v_new = None
    if w.append:
        k_new = normal_bf16(rng, (n_q, Hkv, HEAD_DIM))
        v_new = normal_bf16(rng, (n_q, Hkv, HEAD_DIM))

    if poison:
        cached = seq_lens - q_lens if w.append else seq_lens
        for b in range(B):
            first_empty = int(cached[b])
            n = int(pages_per_seq[b])
            for p in range(first_empty // PAGE, n):
                lo = max(0, first_empty - p * PAGE)
                k_pages[block_table[b, p], :, lo:, :] = BF16_NAN
                v_pages[block_table[b, p], :, lo:, :] = BF16_NAN
        k_pages[spare_ids] = BF16_NAN
        v_pages[spare_ids] = BF16_NAN

    cu = np.zeros(B + 1, dtype=np.int32)
    cu[1:] = np.cumsum(q_lens)
    return Batch(workload=w, seq_lens=seq_lens.astype(np.int32), q_lens=q_lens.astype(np.int32),
                 cu_q_lens=cu, block_table=block_table, k_pages=k_pages, v_pages=v_pages,
                 q=q, k_new=k_new, v_new=v_new, scale=float(np.float32(1.0 / math.sqrt(HEAD_DIM))))


def make_batch(name: str, seed: Optional[int] = None, **overrides) -> Batch:
    """Generate the named workload with its recipe seed (or ``seed``).

    ``overrides`` may replace ``batch`` (keeping the first sequences' lengths from the
    full draw is not attempted: a smaller batch re-draws with the same distributions).
    """
    w = WORKLOADS[name]
    if overrides:
        w = dataclasses.replace(w, **overrides)
    rng = np.random.default_rng(w.seed if seed is None else seed)
    seq_lens, q_lens = draw_lengths(w, rng)
    return build_batch(w, seq_lens, q_lens, rng)


def custom_batch(seq_lens, q_lens=None, num_q_heads=8, num_kv_heads=2, seed=0,
                 append=None, spare_frac=0.01, poison=True) -> Batch:
    """A batch with explicit lengths (edge cases, small parity cases)."""
    seq_lens = np.asarray(seq_lens, dtype=np.int64)
    if q_lens is None:
        q_lens = np.ones(len(seq_lens), np.int64)
    q_lens = np.asarray(q_lens, dtype=np.int64)
    if append is None:
        append = bool((q_lens != 1).any())
    w = Workload("custom", 0, len(seq_lens), num_q_heads, num_kv_heads, "explicit lengths",
                 append=append)
    rng = np.random.default_rng(seed)
    return build_batch(w, seq_lens, q_lens, rng, spare_frac=spare_frac, poison=poison)


def unit_batch(batch: Batch, b: int, g: int) -> Batch:
    """Sequence b with KV head g (and the G query heads that read it) as a batch of its
    own, its pages renamed 0..n-1 in logical order.  Pure data movement (no arithmetic):
    a renamed page pool and a head slice hold the same tokens, so attention over the unit
    equals that slice of attention over the batch.  Used to run the oracle on a batch in
    parallel host processes."""
    w = batch.workload
    G = w.num_q_heads // w.num_kv_heads
    L = int(batch.seq_lens[b])
    n = (L + PAGE - 1) // PAGE
    if n:
        ids = batch.block_table[b, :n]
        kp = np.ascontiguousarray(batch.k_pages[ids, g:g + 1])
        vp = np.ascontiguousarray(batch.v_pages[ids, g:g + 1])
    else:
        kp = np.full((1, 1, PAGE, HEAD_DIM), BF16_NAN, np.uint16)
        vp = kp.copy()
    bt = np.arange(max(n, 1), dtype=np.int32)[None, :]
    heads = slice(g * G, (g + 1) * G)
    if w.append:
        r0, r1 = int(batch.cu_q_lens[b]), int(batch.cu_q_lens[b + 1])
        q = np.ascontiguousarray(batch.q[r0:r1, heads])
        kn = np.ascontiguousarray(batch.k_new[r0:r1, g:g + 1])
        vn = np.ascontiguousarray(batch.v_new[r0:r1, g:g + 1])
    else:
        q = np.ascontiguousarray(batch.q[b:b + 1, heads])
        kn = vn = None
    sub = dataclasses.replace(w, batch=1, num_q_heads=G, num_kv_heads=1)
    C = int(batch.q_lens[b])
    return Batch(sub, batch.seq_lens[b:b + 1].copy(), batch.q_lens[b:b + 1].copy(),
                 np.array([0, C], np.int32), bt, kp, vp, q, kn, vn, batch.scale)


# --- synthetic agentic trajectories (stand-ins for the paper's rollout logs) ---------

def tool_state(tool_type: int, large: bool, failure: bool) -> int:
    """Composite tool-return state: tool type x payload size class x outcome."""
    return (int(tool_type) << 2) | (2 if large else 0) | (1 if failure else 0)


def synthetic_traces(n_prompts: int, per_prompt: int, seed: int = 2606, n_tool_types: int = 4):
    """Seeded multi-turn trajectories: (prompt_id, states, residual) per trace.

    Each prompt has a base difficulty; a trajectory alternates reasoning segments and
    tool calls until it stops.  Failed tools make another call more likely and add
    tokens (retries), large payloads add a long appended output, mirroring the paper's
    observation that payload size and tool failures drive length (Sec. 1, Sec. 2.2).
    ``residual[k]`` is the number of tokens still to come after the k-th tool return
    (``residual[0]`` counts from the prompt on).
    """
    rng = np.random.default_rng(seed)
    traces = []
    for p in range(n_prompts):
        difficulty = rng.lognormal(0.0, 0.6)
        p_fail = min(0.8, 0.15 * difficulty)
        for _ in range(per_prompt):
            segments = [int(rng.lognormal(6.0, 0.5) * difficulty)]
            states = []
            p_more = 0.7
            while rng.random() < p_more and len(states) < 24:
                t = int(rng.integers(n_tool_types))
                large = bool(rng.random() < 0.3)
                fail = bool(rng.random() < p_fail)
                states.append(tool_state(t, large, fail))
                seg = int(rng.lognormal(5.5, 0.6) * difficulty)
                if large:
                    seg += int(rng.lognormal(7.5, 0.4))
                if fail:
                    seg += int(rng.lognormal(6.5, 0.5))
                    p_more = min(0.95, p_more + 0.1)
                else:
                    p_more = max(0.2, p_more - 0.15)
                segments.append(seg)
            total = int(sum(segments))
            done = np.cumsum([0] + segments[:-1])[:len(states) + 1]
            residual = [total - int(d) for d in done]
            traces.append((p, states, residual))
    return traces
