"""Moves generator batches onto the GPU and runs them through the C-ABI (tests only)."""
from __future__ import annotations

import sys

import numpy as np
import torch

from paper_2606_03077_amd import libra
from paper_2606_03077_amd import workloads as wl

TOL_ABS = 2e-2      # max |gpu - oracle| over all output elements
TOL_ROW_REL = 1e-2  # max over rows of ||gpu - oracle||_inf / ||oracle||_inf
TOL_LSE = 1e-3      # max |lse_gpu - lse_oracle| (natural log)
BF16_NAN_I16 = 0x7FC0


def say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def u16_to_dev(a: np.ndarray) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).cuda()


def dev_to_u16(t: torch.Tensor) -> np.ndarray:
    return t.cpu().numpy().view(np.uint16)


def bf16_dev_to_f64(t: torch.Tensor) -> np.ndarray:
    return wl.bf16_bits_to_f32(dev_to_u16(t)).astype(np.float64)


class DeviceCache:
    """The batch's logical pages packed into the library layout on the GPU."""

    def __init__(self, batch: wl.Batch):
        P, Hkv = batch.k_pages.shape[0], batch.k_pages.shape[1]
        self.num_pages, self.hkv = P, Hkv
        self.k = torch.empty(P * Hkv * 2048, dtype=torch.int16, device="cuda")
        self.v = torch.empty_like(self.k)
        self.layout = libra.libra_kv_layout_create(self.k, self.v, P, Hkv)
        k_log = u16_to_dev(batch.k_pages)
        v_log = u16_to_dev(batch.v_pages)
        libra.libra_kv_pack_pages(self.layout, k_log, v_log, 0, P)
        torch.cuda.synchronize()
        del k_log, v_log
        self.bt = torch.from_numpy(batch.block_table).cuda()
        self.bt_stride = batch.block_table.shape[1]

    def unpack(self):
        k = torch.empty(self.num_pages * self.hkv * 2048, dtype=torch.int16, device="cuda")
        v = torch.empty_like(k)
        libra.libra_kv_unpack_pages(self.layout, k, v, 0, self.num_pages)
        torch.cuda.synchronize()
        shape = (self.num_pages, self.hkv, 16, 128)
        return dev_to_u16(k).reshape(shape), dev_to_u16(v).reshape(shape)

    def close(self):
        libra.libra_kv_layout_destroy(self.layout)


def plan_for(batch: wl.Batch, **params):
    w = batch.workload
    mode = libra.LIBRA_MODE_APPEND if w.append else libra.LIBRA_MODE_DECODE
    q_lens = batch.q_lens.tolist() if w.append else None
    return libra.libra_splitkv_plan(mode, len(batch.seq_lens), w.num_q_heads, w.num_kv_heads,
                                    batch.seq_lens.tolist(), q_lens, **params)


def run(batch: wl.Batch, cache: DeviceCache = None, plan_params=None, repeat: int = 1):
    """Runs decode or append; returns (out f64 [rows,Hq,128], lse f64 [rows,Hq], cache, raw)."""
    cache = cache or DeviceCache(batch)
    w = batch.workload
    plan = plan_for(batch, **(plan_params or {}))
    try:
        ws = libra.alloc_workspace(plan)
        q = u16_to_dev(batch.q)
        rows = batch.q.shape[0]
        # NaN before every call: a row that no kernel writes stays NaN and fails parity
        out = torch.empty((rows, w.num_q_heads, 128), dtype=torch.int16, device="cuda")
        lse = torch.empty((rows, w.num_q_heads), dtype=torch.float32, device="cuda")
        for _ in range(repeat):
            out.fill_(BF16_NAN_I16)
            lse.fill_(float("nan"))
            if w.append:
                kn, vn = u16_to_dev(batch.k_new), u16_to_dev(batch.v_new)
                libra.libra_append_attn(cache.layout, plan, q, kn, vn, cache.bt, cache.bt_stride,
                                        len(batch.seq_lens), w.num_q_heads, batch.scale, ws, out, lse)
            else:
                libra.libra_decode_attn(cache.layout, plan, q, cache.bt, cache.bt_stride,
                                        len(batch.seq_lens), w.num_q_heads, batch.scale, ws, out,
                                        lse)
        torch.cuda.synchronize()
        raw_out = dev_to_u16(out)
        o = wl.bf16_bits_to_f32(raw_out).astype(np.float64)
        l = lse.cpu().numpy().astype(np.float64)
        return o, l, cache, raw_out
    finally:
        libra.libra_plan_destroy(plan)


def errors(o, lse, ro, rl, rows=None):
    """(max-abs, max row-relative, max lse-abs) of GPU vs oracle over the given rows."""
    if rows is not None:
        o, lse, ro, rl = o[rows], lse[rows], ro[rows], rl[rows]
    assert np.isfinite(o).all(), "non-finite output"
    d = np.abs(o - ro)
    max_abs = float(d.max()) if d.size else 0.0
    ref_inf = np.abs(ro).max(axis=-1)
    row_rel = d.max(axis=-1) / np.maximum(ref_inf, 1e-30)
    row_rel = np.where(ref_inf > 0, row_rel, d.max(axis=-1))
    max_rel = float(row_rel.max()) if row_rel.size else 0.0
    assert not np.isnan(lse).any(), "LSE left unwritten (NaN)"
    both_inf = np.isneginf(lse) & np.isneginf(rl)
    with np.errstate(invalid="ignore"):
        dl = np.where(both_inf, 0.0, np.abs(lse - rl))
    max_lse = float(dl.max()) if dl.size else 0.0
    return max_abs, max_rel, max_lse


def allclose_fraction(o, ro, rows=None, atol=TOL_ABS, rtol=TOL_ROW_REL):
    """Diagnostic only: share of elements within elementwise allclose(atol, rtol)."""
    if rows is not None:
        o, ro = o[rows], ro[rows]
    if o.size == 0:
        return 1.0
    return float(np.mean(np.abs(o - ro) <= atol + rtol * np.abs(ro)))


def assert_parity(o, lse, ro, rl, rows=None, label=""):
    ea, er, el = errors(o, lse, ro, rl, rows)
    say(f"[parity] {label}: max_abs={ea:.3e} max_row_rel={er:.3e} max_lse={el:.3e} "
        f"allclose={allclose_fraction(o, ro, rows):.6f}")
    assert ea <= TOL_ABS, f"{label}: max abs error {ea} > {TOL_ABS}"
    assert er <= TOL_ROW_REL, f"{label}: row-relative error {er} > {TOL_ROW_REL}"
    assert el <= TOL_LSE, f"{label}: lse error {el} > {TOL_LSE}"


# --- the oracle over a whole batch, in parallel host processes ----------------------

_POOL_BATCH = None


def _unit_task(bg):
    from threadpoolctl import threadpool_limits
    import oracle
    b, g = bg
    u = wl.unit_batch(_POOL_BATCH, b, g)
    with threadpool_limits(1):
        if u.workload.append:
            o, l, _, _ = oracle.append_ref(u.q, u.k_new, u.v_new, u.k_pages, u.v_pages,
                                           u.block_table, u.seq_lens, u.q_lens, u.scale)
        else:
            o, l = oracle.decode_ref(u.q, u.k_pages, u.v_pages, u.block_table, u.seq_lens,
                                     u.scale)
    return b, g, o, l


def oracle_whole_batch(batch: wl.Batch, workers: int = 0):
    """Oracle output and LSE of every query row of the batch, computed per (sequence, KV
    head) in a pool of forked host processes (BLAS single-threaded in each).  Returns
    (o [rows, Hq, 128], lse [rows, Hq], seconds, workers)."""
    import multiprocessing as mp
    import os
    import time
    global _POOL_BATCH
    w = batch.workload
    G = w.num_q_heads // w.num_kv_heads
    rows = batch.q.shape[0]
    o = np.full((rows, w.num_q_heads, 128), np.nan)
    lse = np.full((rows, w.num_q_heads), np.nan)
    cost = batch.seq_lens.astype(np.int64) * batch.q_lens.astype(np.int64)
    tasks = [(int(b), g) for b in np.argsort(-cost, kind="stable")
             for g in range(w.num_kv_heads)]
    workers = workers or max(1, min(16, len(os.sched_getaffinity(0))))
    _POOL_BATCH = batch
    t0 = time.perf_counter()
    try:
        with mp.get_context("fork").Pool(workers) as pool:
            for b, g, ob, lb in pool.imap_unordered(_unit_task, tasks):
                heads = slice(g * G, (g + 1) * G)
                r0 = int(batch.cu_q_lens[b]) if w.append else b
                o[r0:r0 + ob.shape[0], heads] = ob
                lse[r0:r0 + ob.shape[0], heads] = lb
    finally:
        _POOL_BATCH = None
    el = time.perf_counter() - t0
    assert not np.isnan(lse).any(), "the oracle left rows uncomputed"
    return o, lse, el, workers
