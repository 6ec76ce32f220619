"""Benchmark of ragged paged-KV decode and append attention on one MI355X.

    python bench.py [--gpus 1] [--steps 50] [--warmup 5] [--workload longtail]

One step = one decode-attention call (the split-KV decode kernel, then the log-sum-exp
merge of split rows) over the whole synthetic batch, or one append call (cache write,
decode rows, causal chunk tiles, merge), inputs resident in HBM.  Before each timed step
an untimed 1 GiB fill evicts L2 and the 256 MB MALL, so every step reads its KV from HBM.
Each step is bracketed by HIP events on the stream the kernels run on.  The host-side
split plan is built once per batch step and shared by all layers of a model; its time is
reported separately (``plan_ms``) and is not part of a step.  Before planning, the
per-XCD HBM read weights that the plan's slot placement takes are measured once on the
flush buffer (``libra_xcd_read_weights``; ``--xcd-weights equal`` skips it).

Prints one JSON line (rank 0, N = 1).  The headline is the long-tailed rollout batch
(256 sequences, 32 query / 8 KV heads, 90% U[512, 4096] and 10% Pareto tails up to
65,536 tokens):
  value = algorithmic KV bytes / mean step time (TB/s), plus decode tokens/s, the
  roofline of the dominant kernel (decode_kernel against 8 TB/s HBM; chunk_kernel
  against 2.5 PFLOP/s bf16 for append workloads), and the fp64 oracle timed on the
  host cores (``cpu_baseline``).  The dominant kernel's average duration comes from a
  second timed pass in which the library brackets each of its kernels with HIP events.
  ``configs`` holds the same figures for the 7B-class batch, the straggler bucket, the
  tool-output append batch (with its combined HBM / matrix-core roofline fraction) and
  the 40,960-token recompute prefill, timed in the same run.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import math
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
HBM_PEAK_GBS = 8000.0
MFMA_BF16_PEAK_TFLOPS = 2500.0
PROFILE_COUNTERS = os.path.join(ROOT, "profiles", "counters.json")


def log(msg):
    print(msg, file=sys.stderr, flush=True)


def algorithmic_bytes(batch) -> dict:
    """Bytes the method must move for one decode call (per-unit figures in the design notes)."""
    w = batch.workload
    L = batch.seq_lens.astype(np.int64)
    kv = int(L.sum()) * w.num_kv_heads * 128 * 2 * 2          # K and V, bf16
    rows = int(batch.q_lens.sum())
    q = rows * w.num_q_heads * 128 * 2
    o = rows * w.num_q_heads * 128 * 2
    lse = rows * w.num_q_heads * 4
    bt = int(((L + 15) // 16).sum()) * 4
    kv_write = rows * w.num_kv_heads * 128 * 2 * 2 if w.append else 0   # new K and V
    return {"kv": kv, "q": q, "o": o, "lse": lse, "block_table": bt, "kv_write": kv_write,
            "total": kv + q + o + lse + bt + kv_write}


def flops(batch) -> int:
    w = batch.workload
    L = batch.seq_lens.astype(np.int64)
    C = batch.q_lens.astype(np.int64)
    P = L - C
    pairs = int((w.num_q_heads * (C * P + C * (C + 1) // 2)).sum())
    return 4 * 128 * pairs


# The device code of each kernel: its source and the table formats it reads.
KERNEL_SOURCES = {"decode_kernel": ("decode.hip", "tables.h"),
                  "chunk_kernel": ("chunk.hip", "tables.h")}


def kernel_source_sha(kernel: str = "decode_kernel") -> str:
    h = hashlib.sha256()
    for f in KERNEL_SOURCES[kernel]:
        with open(os.path.join(ROOT, "paper_2606_03077_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def plan_sha(units: np.ndarray) -> str:
    """Hash of a plan's units as far as a kernel's traffic depends on them: the set of
    single (decode) units, whose order the slot placement sets from XCD weights measured on
    the device, and the chunk tiles in their queue order, which is fixed by the lengths and
    decides which tiles share an XCD's L2 at a time."""
    u = np.ascontiguousarray(units, dtype=np.int32).reshape(-1, 12)
    single = u[u[:, 10] == 0]
    single = single[np.lexsort(single.T[::-1])]
    chunk = u[u[:, 10] != 0]
    return hashlib.sha256(np.ascontiguousarray(np.concatenate([single, chunk])).tobytes()).hexdigest()[:16]


def counter_from_profile(kernel: str, workload: str, units_sha: str,
                         field: str = "hbm_bytes_per_launch"):
    """A committed rocprofv3 figure for `kernel` on `workload` (HBM bytes per launch, or
    the matrix-core busy fraction).

    Null unless profiles/counters.json was taken on the current kernel source and on a
    plan with the same unit table.
    """
    try:
        with open(PROFILE_COUNTERS) as f:
            c = json.load(f)
    except (OSError, ValueError):
        return None
    e = c.get(kernel, {}).get(workload)
    if not e or e.get("source_sha") != kernel_source_sha(kernel) or e.get("plan_sha") != units_sha:
        return None
    return e.get(field)


_ORACLE_BATCH = None


def _oracle_unit(bg):
    """The fp64 oracle on one (sequence, KV head) unit of the batch; returns its K/V bytes."""
    from threadpoolctl import threadpool_limits
    import oracle
    from paper_2606_03077_amd import workloads as wl
    b, g = bg
    u = wl.unit_batch(_ORACLE_BATCH, b, g)
    with threadpool_limits(1):
        if u.workload.append:
            oracle.append_ref(u.q, u.k_new, u.v_new, u.k_pages, u.v_pages, u.block_table,
                              u.seq_lens, u.q_lens, u.scale)
        else:
            oracle.decode_ref(u.q, u.k_pages, u.v_pages, u.block_table, u.seq_lens, u.scale)
    return int(u.seq_lens[0]) * 128 * 2 * 2, int(u.q_lens[0])


def cpu_baseline(batch, min_seconds: float = 10.0) -> dict:
    """The fp64 oracle on the host cores over a bounded sample of the batch.

    Units are (sequence, KV head) pairs in a seeded random order, one per task, on a pool
    of forked processes (BLAS single-threaded in each), until at least min_seconds have
    passed; the rate is the K/V bytes of the finished units over the elapsed time."""
    import multiprocessing as mp
    global _ORACLE_BATCH
    _ORACLE_BATCH = batch
    w = batch.workload
    visible = len(os.sched_getaffinity(0))
    # at most 16 worker processes: the host cores one GPU's jobs may use, whatever the
    # affinity mask shows
    workers = max(1, min(visible, 16))
    units = [(b, g) for b in range(len(batch.seq_lens)) for g in range(w.num_kv_heads)]
    order = np.random.default_rng(0).permutation(len(units))
    tasks = [units[i] for i in order]
    done_bytes = done_units = done_rows = 0
    t0 = time.perf_counter()
    pool = mp.get_context("fork").Pool(workers)
    try:
        for _ in range(64):                      # passes over the batch, bounded
            for nbytes, rows in pool.imap_unordered(_oracle_unit, tasks):
                done_bytes += nbytes
                done_units += 1
                done_rows += rows
                if time.perf_counter() - t0 >= min_seconds:
                    break
            if time.perf_counter() - t0 >= min_seconds:
                break
    finally:
        pool.terminate()
        pool.join()
        _ORACLE_BATCH = None
    el = time.perf_counter() - t0
    kind = "append" if w.append else "decode"
    return {"value": round(done_bytes / el / 1e12, 6), "unit": "TB/s", "cores": workers,
            "kind": "oracle",
            "host_cores_visible": visible,
            "sample": f"{done_units} of {len(units)} (sequence, KV head) units of the "
                      f"{w.name} batch in seeded random order ({done_units / len(units):.2f} "
                      f"passes), {el:.1f} s, fp64 numpy {kind} oracle, one process per "
                      f"core ({workers} of {visible} visible cores, at most 16)",
            "kv_bytes": done_bytes}


PCIE_GEN5_X16_GBS = 64.0   # per direction, before protocol overhead


def bench_migrate(args, torch, libra, wl) -> dict:
    """Migration of one paused request between TP degrees (Sec. 5, Steps 1-3), per layer.

    The request holds ``--migrate-tokens`` tokens of a 40-query-head / 8-KV-head model
    (one layer's K and V).  Step 1: page gather into a packed device run, then a copy to
    pinned host memory.  Step 2: host reshard from TP_src to TP_dst head shards.  Step 3:
    each target shard's run is copied to the device and scattered into fresh pages (all
    target caches live on this one GPU).  Device phases are timed with HIP events on
    one stream, the host reshard with the wall clock.
    """
    tp_src, tp_dst = (int(x) for x in args.migrate_tp.split(","))
    hq, hkv, L = 40, 8, args.migrate_tokens
    if hkv % tp_src or hkv % tp_dst:
        raise SystemExit("TP degrees must divide the 8 KV heads")
    n = -(-L // 16)
    tile = 2048
    log(f"[bench] migrate: {L} tokens, TP {tp_src} -> {tp_dst}")
    batch = wl.custom_batch([L], num_q_heads=hq, num_kv_heads=hkv, seed=L, poison=False)
    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream()
    # TP_src source caches, each holding its head range of the request's pages
    full_k = batch.k_pages
    full_v = batch.v_pages
    P = full_k.shape[0]
    hs = hkv // tp_src
    src = []
    for i in range(tp_src):
        k = torch.empty(P * hs * tile, dtype=torch.int16, device=dev)
        v = torch.empty_like(k)
        lay = libra.libra_kv_layout_create(k, v, P, hs)
        kl = torch.from_numpy(np.ascontiguousarray(full_k[:, i * hs:(i + 1) * hs]).view(np.int16))
        vl = torch.from_numpy(np.ascontiguousarray(full_v[:, i * hs:(i + 1) * hs]).view(np.int16))
        libra.libra_kv_pack_pages(lay, kl.to(dev), vl.to(dev), 0, P)
        src.append((lay, k, v))
    ids = torch.from_numpy(np.ascontiguousarray(batch.block_table[0, :n])).to(dev)
    hd = hkv // tp_dst
    rng = np.random.default_rng(7)
    dst = []
    for j in range(tp_dst):
        k = torch.empty((n + 64) * hd * tile, dtype=torch.int16, device=dev)
        v = torch.empty_like(k)
        lay = libra.libra_kv_layout_create(k, v, n + 64, hd)
        tid = torch.from_numpy(rng.permutation(n + 64)[:n].astype(np.int32)).to(dev)
        dst.append((lay, k, v, tid))
    run_k = [torch.empty(n * hs * tile, dtype=torch.int16, device=dev) for _ in range(tp_src)]
    run_v = [torch.empty_like(r) for r in run_k]
    host_k = [torch.empty(r.shape, dtype=torch.int16, pin_memory=True) for r in run_k]
    host_v = [torch.empty(r.shape, dtype=torch.int16, pin_memory=True) for r in run_k]
    out_k = [torch.empty(n * hd * tile, dtype=torch.int16, pin_memory=True) for _ in range(tp_dst)]
    out_v = [torch.empty(r.shape, dtype=torch.int16, pin_memory=True) for r in out_k]
    dev_k = [torch.empty(r.shape, dtype=torch.int16, device=dev) for r in out_k]
    dev_v = [torch.empty_like(r) for r in dev_k]
    torch.cuda.synchronize()

    def ev():
        return torch.cuda.Event(enable_timing=True)

    phases = {"copy_out_kernel": [], "d2h": [], "reshard_host": [], "h2d": [],
              "copy_in_kernel": []}
    iters = max(1, args.steps)
    for it in range(args.warmup + iters):
        e = [ev() for _ in range(6)]
        e[0].record(stream)
        for i, (lay, _, _) in enumerate(src):
            libra.libra_kv_copy_out(lay, ids, n, run_k[i], run_v[i], stream=stream)
        e[1].record(stream)
        for i in range(tp_src):
            host_k[i].copy_(run_k[i], non_blocking=True)
            host_v[i].copy_(run_v[i], non_blocking=True)
        e[2].record(stream)
        stream.synchronize()
        t0 = time.perf_counter()
        libra.libra_kv_reshard_host(host_k, hs, out_k, n)
        libra.libra_kv_reshard_host(host_v, hs, out_v, n)
        t_reshard = (time.perf_counter() - t0) * 1e3
        e[3].record(stream)
        for j in range(tp_dst):
            dev_k[j].copy_(out_k[j], non_blocking=True)
            dev_v[j].copy_(out_v[j], non_blocking=True)
        e[4].record(stream)
        for j, (lay, _, _, tid) in enumerate(dst):
            libra.libra_kv_copy_in(lay, tid, n, dev_k[j], dev_v[j], stream=stream)
        e[5].record(stream)
        stream.synchronize()
        if it >= args.warmup:
            phases["copy_out_kernel"].append(e[0].elapsed_time(e[1]))
            phases["d2h"].append(e[1].elapsed_time(e[2]))
            phases["reshard_host"].append(t_reshard)
            phases["h2d"].append(e[3].elapsed_time(e[4]))
            phases["copy_in_kernel"].append(e[4].elapsed_time(e[5]))
        log(f"[bench] migrate iteration {it} done")

    def check_targets(what):
        """The target pages hold exactly the resharded runs (bit-exact)."""
        for j, (lay, _, _, tid) in enumerate(dst):
            kk = torch.empty(n * hd * tile, dtype=torch.int16, device=dev)
            vv = torch.empty_like(kk)
            libra.libra_kv_copy_out(lay, tid, n, kk, vv, stream=stream)
            stream.synchronize()
            if not (torch.equal(kk.cpu(), out_k[j]) and torch.equal(vv.cpu(), out_v[j])):
                raise RuntimeError(f"{what}: migrated pages differ from the resharded run")

    check_targets("staged")
    for lay, k, v, tid in dst:
        k.fill_(0)
        v.fill_(0)
    # Direct variant: the copy kernels read / write the pinned host runs themselves, so
    # each of offload and reload is one kernel crossing PCIe (no device staging buffer).
    direct = {"copy_out_direct": [], "copy_in_direct": []}
    for it in range(args.warmup + iters):
        e = [ev() for _ in range(4)]
        e[0].record(stream)
        for i, (lay, _, _) in enumerate(src):
            libra.libra_kv_copy_out(lay, ids, n, host_k[i], host_v[i], stream=stream)
        e[1].record(stream)
        stream.synchronize()
        libra.libra_kv_reshard_host(host_k, hs, out_k, n)
        libra.libra_kv_reshard_host(host_v, hs, out_v, n)
        e[2].record(stream)
        for j, (lay, _, _, tid) in enumerate(dst):
            libra.libra_kv_copy_in(lay, tid, n, out_k[j], out_v[j], stream=stream)
        e[3].record(stream)
        stream.synchronize()
        if it >= args.warmup:
            direct["copy_out_direct"].append(e[0].elapsed_time(e[1]))
            direct["copy_in_direct"].append(e[2].elapsed_time(e[3]))
    log("[bench] migrate direct variant done")
    check_targets("direct")
    med = {k: float(np.median(v)) for k, v in phases.items()}
    med_direct = {k: float(np.median(v)) for k, v in direct.items()}
    layer_bytes = n * hkv * tile * 2 * 2          # K and V of one layer, whole pages
    gbs = lambda ms, b: b / (ms * 1e-3) / 1e9
    offload_ms = med["copy_out_kernel"] + med["d2h"]
    reload_ms = med["h2d"] + med["copy_in_kernel"]
    total_ms = offload_ms + med["reshard_host"] + reload_ms
    copy_kernel_gbs = gbs(med["copy_out_kernel"], 2 * layer_bytes)
    for lay, _, _ in src:
        libra.libra_kv_layout_destroy(lay)
    for lay, _, _, _ in dst:
        libra.libra_kv_layout_destroy(lay)
    result = {
        "metric": "KV migration latency per layer (offload + head reshard + reload)",
        "value": round(total_ms, 4),
        "unit": "ms/layer",
        "n_gpus": 1, "steps": iters, "warmup": args.warmup,
        "ms_per_step": round(total_ms, 4),
        "higher_is_better": False, "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16", "data": "synthetic (seeded normal bf16 pages)",
        "config": {"workload": f"migrate: one {L}-token request, 40 query / 8 KV heads, "
                               f"head_dim 128, TP {tp_src} -> {tp_dst}, one layer",
                   "pages": n, "layer_kv_bytes": layer_bytes},
        "phases_ms_median": {k: round(v, 4) for k, v in med.items()},
        "direct_ms_median": {k: round(v, 4) for k, v in med_direct.items()},
        "direct_GBps": {k: round(gbs(v, layer_bytes), 2) for k, v in med_direct.items()},
        "offload_ms": round(offload_ms, 4),
        "reload_ms": round(reload_ms, 4),
        "d2h_GBps": round(gbs(med["d2h"], layer_bytes), 2),
        "h2d_GBps": round(gbs(med["h2d"], layer_bytes), 2),
        "reshard_host_GBps": round(gbs(med["reshard_host"], layer_bytes), 2),
        "pcie_peak_GBps_per_direction": PCIE_GEN5_X16_GBS,
        "roofline": {"bound": "hbm", "achieved": round(copy_kernel_gbs, 2), "peak": HBM_PEAK_GBS,
                     "unit": "GB/s", "frac": round(copy_kernel_gbs / HBM_PEAK_GBS, 4),
                     "traffic": None, "kernel": "page_copy_kernel (copy_out)",
                     "algorithmic_bytes_per_launch": 2 * layer_bytes // tp_src,
                     "kernel_avg_ms": round(med["copy_out_kernel"] / tp_src, 5)},
    }
    if not args.no_cpu_baseline:
        import oracle.migration as om
        req_k = om.request_pages(batch.k_pages, batch.block_table[0], L)
        req_v = om.request_pages(batch.v_pages, batch.block_table[0], L)
        srcs_k = om.reshard_heads([req_k], tp_src)
        srcs_v = om.reshard_heads([req_v], tp_src)
        reps, t0 = 0, time.perf_counter()
        while time.perf_counter() - t0 < min(args.cpu_seconds, 5.0):
            om.reshard_heads(srcs_k, tp_dst)
            om.reshard_heads(srcs_v, tp_dst)
            reps += 1
        el = time.perf_counter() - t0
        result["cpu_baseline"] = {
            "value": round(layer_bytes * reps / el / 1e9, 3), "unit": "GB/s", "cores": 1,
            "kind": "oracle",
            "sample": f"numpy head reshard of the request's pages (one layer) x {reps}, {el:.1f} s"}
    return result


CE_DECODE_LENS = [256, 512, 1024, 2048, 4096, 8192, 12288, 16384, 24576, 32768, 40960]
CE_PREFILL_LENS = [1024, 2048, 4096, 8192, 12288, 16384, 24576, 32768, 40960]


def bench_ce(args, torch, libra) -> dict:
    """Cost-evaluator calibration from this library's own attention timings (Sec. 4.5;
    App. B.1; Sec. 7.5).

    Per layer of a 40-query / 8-KV-head model: (a) a decode step over 32 sequences all
    at context L, (b) the recompute prefill of one L-token sequence (append with empty
    prior).  Each is timed with HIP events (median of --steps, L2 / MALL flushed before
    every call).  T(L) = gamma L^2 + eta L + theta is fitted to every other length and
    scored by MAPE on the lengths left out, then refitted on all of them.
    """
    hq, hkv, B = 40, 8, 32
    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream()
    gen = torch.Generator(device=dev)
    gen.manual_seed(2606)

    def randn_i16(n):
        return torch.randn(n, generator=gen, device=dev, dtype=torch.bfloat16).view(torch.int16)

    flush = torch.empty(args.flush_mib * (1 << 20) // 4, dtype=torch.float32, device=dev)
    reps = max(3, args.steps)

    def timed(call):
        ts = []
        for r in range(args.warmup + reps):
            flush.fill_(float(r))
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record(stream)
            call()
            b.record(stream)
            stream.synchronize()
            if r >= args.warmup:
                ts.append(a.elapsed_time(b))
        return float(np.median(ts))

    rng = np.random.default_rng(2606)
    max_pages = 40960 // 16
    # (a) decode steps
    P = B * max_pages + 1
    log(f"[bench] ce: filling a {P}-page cache on the device")
    k = randn_i16(P * hkv * 2048)
    v = randn_i16(P * hkv * 2048)
    layout = libra.libra_kv_layout_create(k, v, P, hkv)
    bt = torch.from_numpy(rng.permutation(P)[:B * max_pages].astype(np.int32)
                          .reshape(B, max_pages)).to(dev)
    q = randn_i16(B * hq * 128)
    out = torch.empty(B * hq * 128, dtype=torch.int16, device=dev)
    lse = torch.empty(B * hq, dtype=torch.float32, device=dev)
    dec = []
    for L in CE_DECODE_LENS:
        plan = libra.libra_splitkv_plan(libra.LIBRA_MODE_DECODE, B, hq, hkv, [L] * B)
        ws = libra.alloc_workspace(plan)
        libra.libra_plan_upload(plan, ws, stream=stream)
        ms = timed(lambda: libra.libra_decode_attn(layout, plan, q, bt, max_pages, B, hq,
                                                   0.088, ws, out, lse, stream=stream))
        libra.libra_plan_destroy(plan)
        dec.append(ms)
        log(f"[bench] ce decode L={L}: {ms:.4f} ms")
    libra.libra_kv_layout_destroy(layout)
    del k, v
    # (b) recompute prefill
    P2 = max_pages + 1
    k2 = randn_i16(P2 * hkv * 2048)
    v2 = randn_i16(P2 * hkv * 2048)
    layout2 = libra.libra_kv_layout_create(k2, v2, P2, hkv)
    bt2 = torch.from_numpy(rng.permutation(P2)[:max_pages].astype(np.int32)[None, :]).to(dev)
    qp = randn_i16(40960 * hq * 128)
    kn = randn_i16(40960 * hkv * 128)
    vn = randn_i16(40960 * hkv * 128)
    outp = torch.empty(40960 * hq * 128, dtype=torch.int16, device=dev)
    lsep = torch.empty(40960 * hq, dtype=torch.float32, device=dev)
    pf, pf_chunk = [], []
    for L in CE_PREFILL_LENS:
        plan = libra.libra_splitkv_plan(libra.LIBRA_MODE_APPEND, 1, hq, hkv, [L], [L])
        ws = libra.alloc_workspace(plan)
        libra.libra_plan_upload(plan, ws, stream=stream)
        call = lambda: libra.libra_append_attn(layout2, plan, qp, kn, vn, bt2, max_pages, 1, hq,
                                               0.088, ws, outp, lsep, stream=stream)
        ms = timed(call)
        libra.libra_profile_enable(True)
        libra.libra_profile_collect()
        for _ in range(3):
            call()
        stream.synchronize()
        kt = libra.libra_profile_collect()
        libra.libra_profile_enable(False)
        libra.libra_plan_destroy(plan)
        pf.append(ms)
        pf_chunk.append(kt["chunk"][0] / max(1, kt["chunk"][1]))
        log(f"[bench] ce prefill L={L}: {ms:.4f} ms")
    libra.libra_kv_layout_destroy(layout2)

    def fit_report(lens, times):
        lens = np.asarray(lens, dtype=np.float64)
        times = np.asarray(times, dtype=np.float64)
        train, held = lens[0::2], lens[1::2]
        tt, th = times[0::2], times[1::2]
        c_train = libra.libra_ce_fit(train, tt)
        c_all = libra.libra_ce_fit(lens, times)
        pred = c_all[0] * lens ** 2 + c_all[1] * lens + c_all[2]
        return {"gamma_eta_theta": list(c_all),
                "mape_heldout_pct": round(libra.libra_ce_mape(c_train, held, th), 3),
                "mape_all_pct": round(libra.libra_ce_mape(c_all, lens, times), 3),
                "points": [[int(L), round(float(t), 5), round(float(p), 5)]
                           for L, t, p in zip(lens, times, pred)]}

    d = fit_report(CE_DECODE_LENS, dec)
    f = fit_report(CE_PREFILL_LENS, pf)
    L = 40960
    fl = 4 * 128 * hq * (L * (L + 1) // 2)
    achieved = fl / (pf_chunk[-1] * 1e-3) / 1e12
    # per-sequence attention of one decode step at context l (the rollout model's input)
    per_seq = [c / B for c in d["gamma_eta_theta"]]
    result = {
        "metric": "cost-evaluator attention polynomial MAPE on held-out lengths",
        "value": round(max(d["mape_heldout_pct"], f["mape_heldout_pct"]), 3),
        "unit": "%", "n_gpus": 1, "steps": reps, "warmup": args.warmup,
        "ms_per_step": round(pf[-1], 4),
        "higher_is_better": False, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic (device-seeded normal bf16)",
        "config": {"workload": "ce: per-layer attention of a 40-query / 8-KV-head model; decode "
                               f"steps of {B} sequences at L in {CE_DECODE_LENS}; recompute "
                               f"prefill of one sequence at L in {CE_PREFILL_LENS}"},
        "decode_step": d, "prefill": f,
        "attn_step_per_sequence": per_seq,
        "roofline": {"bound": "mfma", "achieved": round(achieved, 2),
                     "peak": MFMA_BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
                     "frac": round(achieved / MFMA_BF16_PEAK_TFLOPS, 4), "traffic": None,
                     "kernel": "chunk_kernel (prefill, L = 40960)",
                     "kernel_avg_ms": round(pf_chunk[-1], 5)},
    }
    if not args.no_cpu_baseline:
        import oracle.cost_model as ocm
        n, t0 = 0, time.perf_counter()
        while time.perf_counter() - t0 < 1.0:
            ocm.ce_fit_ref(CE_PREFILL_LENS, pf)
            n += 1
        el = time.perf_counter() - t0
        result["cpu_baseline"] = {"value": round(n / el, 1), "unit": "fits/s", "cores": 1,
                                  "kind": "oracle",
                                  "sample": f"numpy least-squares fit of the prefill points x {n}"}
    return result


def bench_planner(args) -> dict:
    """Host-side planner pieces: RolloutDP (Alg. 1) search time at cluster scale, literal
    recurrence against the crossing search, and prefix-tree insert / lookup rates on
    synthetic trajectories (Sec. 4.2, Sec. 5)."""
    from paper_2606_03077_amd import libra
    from paper_2606_03077_amd import workloads as wl
    traces = wl.synthetic_traces(2000, 8, seed=26060)
    lengths = np.array([r[0] for _, _, r in traces], dtype=np.int64)
    # Model inputs, in seconds for a 40-layer model: the per-sequence decode attention
    # step is 40 x the per-layer fit of the ce workload on MI355X (eta 6.87e-10 s per
    # context token, theta 2.5e-7 s; its tiny negative gamma clipped to 0); the per-step
    # non-attention time stands in for reading a 14B model's bf16 weights at each TP.
    model = libra.rollout_model((0.0, 2.75e-8, 1.0e-5),
                                {1: 3.5e-3, 2: 1.9e-3, 4: 1.05e-3, 8: 0.62e-3},
                                {1: 1.0, 2: 0.52, 4: 0.27, 8: 0.15})
    rows = []
    for n_gpus, n_req, exact in [(8, 256, True), (8, 256, False), (64, 1024, True),
                                 (64, 1024, False), (128, 1024, False), (128, 4096, False)]:
        sub = lengths[:n_req]
        t0 = time.perf_counter()
        ms, _, inst = libra.libra_rollout_dp(sub, n_gpus, [1, 2, 4, 8], model, exact)
        el = time.perf_counter() - t0
        rows.append({"n_gpus": n_gpus, "n_req": n_req, "exact": exact, "search_s": round(el, 4),
                     "makespan_s": round(ms, 3),
                     "instances_per_tp": {str(t): sum(1 for tp, _, c in inst if tp == t)
                                          for t in (8, 4, 2, 1)}})
        log(f"[bench] planner {rows[-1]}")
    tree = libra.PrefixTree([2048, 8192, 32768])
    t0 = time.perf_counter()
    for p, st, res in traces:
        tree.insert(p, st, res)
    ins = len(traces) / (time.perf_counter() - t0)
    queries = [(p, st) for p, st, _ in traces]
    t0 = time.perf_counter()
    for p, st in queries:
        tree.lookup(p, st)
    look = len(queries) / (time.perf_counter() - t0)
    tree.close()
    big = next(r for r in rows if r["n_gpus"] == 128 and r["n_req"] == 1024)
    result = {
        "metric": "RolloutDP search time (128 GPUs, 1024 requests, TP set {1,2,4,8})",
        "value": big["search_s"], "unit": "s", "n_gpus": 0, "steps": 1, "warmup": 0,
        "ms_per_step": round(big["search_s"] * 1e3, 3),
        "higher_is_better": False, "scaling": "strong", "vs_baseline": None, "dtype": "f64",
        "data": "synthetic trajectories (workloads.synthetic_traces)",
        "config": {"workload": "planner: host RolloutDP and prefix tree"},
        "dp": rows,
        "trie_inserts_per_s": round(ins, 1), "trie_lookups_per_s_python": round(look, 1),
        "roofline": None,
    }
    if not args.no_cpu_baseline:
        import oracle.cost_model as ocm
        m = {"attn_step": (0.0, 2.75e-8, 1.0e-5),
             "linear_step": [3.5e-3, 1.9e-3, 1.05e-3, 0.62e-3],
             "attn_scale": [1.0, 0.52, 0.27, 0.15]}
        sub = lengths[:24].tolist()
        t0 = time.perf_counter()
        ocm.rollout_dp_ref(sub, 8, [1, 2, 4, 8], m)
        el = time.perf_counter() - t0
        t1 = time.perf_counter()
        libra.libra_rollout_dp(sub, 8, [1, 2, 4, 8], model, True)
        el_lib = time.perf_counter() - t1
        result["cpu_baseline"] = {"value": round(el, 4), "unit": "s", "cores": 1,
                                  "kind": "oracle",
                                  "sample": f"Alg. 1 in Python, 8 GPUs x 24 requests "
                                            f"(library, same case: {el_lib:.5f} s)"}
    return result


EXTRA_CONFIGS = ("7b", "straggler", "append", "prefill")


def measure(name, args, torch, libra, wl, flush, xcd_weight, steps, warmup, cpu_seconds=0.0):
    """Times one decode / append workload; returns its result fields (see the module
    docstring) and, when cpu_seconds > 0, the oracle's rate on a sample of the same batch."""
    dev = torch.device("cuda:0")
    log(f"[bench] generating workload {name}")
    t = time.perf_counter()
    batch = wl.make_batch(name)
    log(f"[bench] generated {name} in {time.perf_counter() - t:.1f} s")
    w = batch.workload
    P, Hkv = batch.k_pages.shape[0], batch.k_pages.shape[1]

    k_cache = torch.empty(P * Hkv * 2048, dtype=torch.int16, device=dev)
    v_cache = torch.empty_like(k_cache)
    layout = libra.libra_kv_layout_create(k_cache, v_cache, P, Hkv)
    k_log = torch.from_numpy(batch.k_pages.view(np.int16)).to(dev)
    v_log = torch.from_numpy(batch.v_pages.view(np.int16)).to(dev)
    libra.libra_kv_pack_pages(layout, k_log, v_log, 0, P)
    torch.cuda.synchronize()
    del k_log, v_log
    bt = torch.from_numpy(batch.block_table).to(dev)
    q = torch.from_numpy(batch.q.view(np.int16)).to(dev)
    rows = batch.q.shape[0]
    out = torch.empty((rows, w.num_q_heads, 128), dtype=torch.int16, device=dev)
    lse = torch.empty((rows, w.num_q_heads), dtype=torch.float32, device=dev)
    kn = vn = None
    if w.append:
        kn = torch.from_numpy(batch.k_new.view(np.int16)).to(dev)
        vn = torch.from_numpy(batch.v_new.view(np.int16)).to(dev)

    mode = libra.LIBRA_MODE_APPEND if w.append else libra.LIBRA_MODE_DECODE
    ql = batch.q_lens.tolist() if w.append else None
    B = len(batch.seq_lens)
    plan_kw = dict(units_per_cu=args.units_per_cu, min_split_pages=args.min_split_pages,
                   max_splits=args.max_splits, xcd_weight=xcd_weight)
    plan_times = []
    for _ in range(5):
        t = time.perf_counter()
        plan = libra.libra_splitkv_plan(mode, B, w.num_q_heads, Hkv, batch.seq_lens.tolist(),
                                        ql, **plan_kw)
        plan_times.append((time.perf_counter() - t) * 1e3)
        libra.libra_plan_destroy(plan)
    plan = libra.libra_splitkv_plan(mode, B, w.num_q_heads, Hkv, batch.seq_lens.tolist(), ql,
                                    **plan_kw)
    info = libra.libra_plan_get_info(plan)
    ws = libra.alloc_workspace(plan)
    stream = torch.cuda.current_stream()
    libra.libra_plan_upload(plan, ws, stream=stream)

    def step(p=plan):
        if w.append:
            libra.libra_append_attn(layout, p, q, kn, vn, bt, bt.shape[1], B, w.num_q_heads,
                                    batch.scale, ws, out, lse, stream=stream)
        else:
            libra.libra_decode_attn(layout, p, q, bt, bt.shape[1], B, w.num_q_heads,
                                    batch.scale, ws, out, lse, stream=stream)

    log(f"[bench] {name}: warmup {warmup}")
    for i in range(warmup):
        flush.fill_(float(i))
        step()
    torch.cuda.synchronize()

    starts = [torch.cuda.Event(enable_timing=True) for _ in range(steps)]
    ends = [torch.cuda.Event(enable_timing=True) for _ in range(steps)]
    log(f"[bench] {name}: timing {steps} steps")
    torch.cuda.synchronize()
    wall0 = time.perf_counter()
    for i in range(steps):
        flush.fill_(float(i))           # untimed: evicts L2 / MALL
        starts[i].record(stream)
        step()
        ends[i].record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - wall0
    times_ms = np.array([s.elapsed_time(e) for s, e in zip(starts, ends)])
    mean_ms = float(times_ms.mean())
    p10, p50, p90 = (float(x) for x in np.percentile(times_ms, [10, 50, 90]))

    # Second timed pass: the library brackets each of its kernels with HIP events on the
    # same stream, giving the dominant kernel's own average duration.
    libra.libra_profile_enable(True)
    libra.libra_profile_collect()
    for i in range(steps):
        flush.fill_(float(i))
        step()
    torch.cuda.synchronize()
    ktimes = libra.libra_profile_collect()
    libra.libra_profile_enable(False)
    kernel_avg_ms = {k: ms / n for k, (ms, n) in ktimes.items() if n}

    # A step that also builds, uploads and destroys its plan (host wall clock, synchronised):
    # the per-step cost of a plan when every layer of a model shares it is plan_ms / layers.
    with_plan = []
    for i in range(min(steps, 10)):
        flush.fill_(float(i))
        torch.cuda.synchronize()
        t = time.perf_counter()
        p2 = libra.libra_splitkv_plan(mode, B, w.num_q_heads, Hkv, batch.seq_lens.tolist(), ql,
                                      **plan_kw)
        libra.libra_plan_upload(p2, ws, stream=stream)
        step(p2)
        libra.libra_plan_destroy(p2)
        torch.cuda.synchronize()
        with_plan.append((time.perf_counter() - t) * 1e3)
    libra.libra_plan_upload(plan, ws, stream=stream)

    # The chunk kernel alone: when the append batch also has single-token rows, its chunk
    # tiles share the device with the decode rows during a step (see the design notes), so
    # its duration inside a step is not its own.  Time a plan of the chunk rows only, on
    # the same cache (the cache write rewrites the same values), to give its roofline.
    chunk_alone_ms = None
    if w.append and info["n_single"] > 0 and info["n_chunk"] > 0:
        ch = np.nonzero(batch.q_lens > 1)[0]
        rows_ch = np.concatenate([np.arange(batch.cu_q_lens[b], batch.cu_q_lens[b + 1])
                                  for b in ch]).astype(np.int64)
        idx = torch.from_numpy(rows_ch).to(dev)
        q_c, kn_c, vn_c = q.view(rows, -1)[idx].contiguous(), kn.view(rows, -1)[idx].contiguous(), \
            vn.view(rows, -1)[idx].contiguous()
        out_c = torch.empty_like(q_c)
        lse_c = torch.empty((len(rows_ch), w.num_q_heads), dtype=torch.float32, device=dev)
        bt_c = bt[torch.from_numpy(ch).to(dev)].contiguous()
        plan_c = libra.libra_splitkv_plan(mode, len(ch), w.num_q_heads, Hkv,
                                          batch.seq_lens[ch].tolist(), batch.q_lens[ch].tolist(),
                                          **plan_kw)
        ws_c = libra.alloc_workspace(plan_c)
        libra.libra_plan_upload(plan_c, ws_c, stream=stream)
        libra.libra_profile_enable(True)
        libra.libra_profile_collect()
        for i in range(max(3, min(steps, 20))):
            flush.fill_(float(i))
            libra.libra_append_attn(layout, plan_c, q_c, kn_c, vn_c, bt_c, bt_c.shape[1], len(ch),
                                    w.num_q_heads, batch.scale, ws_c, out_c, lse_c, stream=stream)
        torch.cuda.synchronize()
        kt = libra.libra_profile_collect()
        libra.libra_profile_enable(False)
        chunk_alone_ms = kt["chunk"][0] / kt["chunk"][1]
        libra.libra_plan_destroy(plan_c)
        del q_c, kn_c, vn_c, out_c, lse_c, bt_c, ws_c
    ab = algorithmic_bytes(batch)
    fl = flops(batch)
    kv_tbs = ab["kv"] / (mean_ms * 1e-3) / 1e12
    tokens_per_s = rows / (mean_ms * 1e-3)
    units_sha = plan_sha(libra.libra_plan_get_units(plan))
    if w.append:
        # chunk rows dominate: a matrix-core bound contraction
        ch = batch.q_lens > 1
        sub = wl.Batch(w, batch.seq_lens[ch], batch.q_lens[ch], None, None, None, None, None,
                       None, None, batch.scale)
        kern = "chunk"
        work = flops(sub)
        achieved = work / (kernel_avg_ms[kern] * 1e-3) / 1e12
        roof = {"bound": "mfma", "achieved": round(achieved, 2), "peak": MFMA_BF16_PEAK_TFLOPS,
                "unit": "TFLOP/s", "frac": round(achieved / MFMA_BF16_PEAK_TFLOPS, 4),
                "traffic": counter_from_profile("chunk_kernel", name, units_sha),
                "kernel": "chunk_kernel",
                "algorithmic_flops_per_launch": work,
                "mfma_busy": counter_from_profile("chunk_kernel", name, units_sha, "mfma_busy")}
        if chunk_alone_ms is not None:
            a = work / (chunk_alone_ms * 1e-3) / 1e12
            roof["chunk_kernel_alone"] = {
                "kernel_avg_ms": round(chunk_alone_ms, 5), "achieved": round(a, 2),
                "frac": round(a / MFMA_BF16_PEAK_TFLOPS, 4),
                "note": "same chunk tiles in a plan of the chunk rows only; within a step "
                        "they share the device with the decode rows"}
    else:
        kern = "decode"
        achieved = ab["total"] / (kernel_avg_ms[kern] * 1e-3) / 1e9
        roof = {"bound": "hbm", "achieved": round(achieved, 2), "peak": HBM_PEAK_GBS,
                "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4),
                "traffic": counter_from_profile("decode_kernel", name, units_sha),
                "kernel": "decode_kernel",
                "algorithmic_bytes_per_launch": ab["total"]}
    roof["kernel_avg_ms"] = round(kernel_avg_ms[kern], 5)
    roof["other_kernels_avg_ms"] = {k: round(v, 5) for k, v in kernel_avg_ms.items() if k != kern}
    # Whole-step roofline: the step cannot beat both its HBM bytes at 8 TB/s and its
    # matrix-core flops at 2.5 PFLOP/s, whichever takes longer.
    t_hbm = ab["total"] / (HBM_PEAK_GBS * 1e9) * 1e3
    t_mfma = fl / (MFMA_BF16_PEAK_TFLOPS * 1e12) * 1e3
    combined = {"t_roofline_ms": round(max(t_hbm, t_mfma), 5),
                "t_hbm_ms": round(t_hbm, 5), "t_mfma_ms": round(t_mfma, 5),
                "bound": "hbm" if t_hbm >= t_mfma else "mfma",
                "t_step_ms": round(mean_ms, 5), "frac": round(max(t_hbm, t_mfma) / mean_ms, 4)}

    result = {
        "value": round(kv_tbs, 4),
        "ms_per_step": round(mean_ms, 5),
        "config": {"workload": f"{name}: {w.description}", "batch": B,
                   "num_q_heads": w.num_q_heads, "num_kv_heads": Hkv, "head_dim": 128,
                   "page_size": 16, "kv_tokens": int(batch.seq_lens.sum()),
                   "query_rows": rows, "seed": w.seed},
        "hbm_peak_frac": round(kv_tbs * 1e3 / HBM_PEAK_GBS, 4),
        "decode_tokens_per_s": round(tokens_per_s, 1),
        "step_ms_p10_p50_p90": [round(p10, 5), round(p50, 5), round(p90, 5)],
        "timed_wall_s": round(wall, 4),
        "plan_ms": round(float(np.median(plan_times)), 4),
        "step_with_plan_upload_destroy_ms": round(float(np.median(with_plan)), 4),
        "plan": dict({k: info[k] for k in ("n_units", "n_single", "n_chunk", "n_partial_slots",
                                           "balanced", "chunk_pages", "num_cus")}, **plan_kw),
        "algorithmic_bytes": ab["total"],
        "flops": fl,
        "roofline": roof,
        "step_roofline": combined,
    }
    if cpu_seconds > 0:
        log(f"[bench] {name}: timing the oracle on host cores (~{cpu_seconds:.0f} s)")
        result["cpu_baseline"] = cpu_baseline(batch, cpu_seconds)
    libra.libra_plan_destroy(plan)
    libra.libra_kv_layout_destroy(layout)
    del k_cache, v_cache, q, out, lse, kn, vn, bt, ws, batch
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    return result


def config_summary(r: dict) -> dict:
    """The per-config block: step time, KV rate, and the dominant kernel's roofline."""
    roof = r["roofline"]
    out = {"workload": r["config"]["workload"], "ms_per_step": r["ms_per_step"],
           "kv_TBps": r["value"], "hbm_peak_frac": r["hbm_peak_frac"],
           "decode_tokens_per_s": r["decode_tokens_per_s"],
           "step_ms_p10_p50_p90": r["step_ms_p10_p50_p90"],
           "kernel": roof["kernel"], "kernel_avg_ms": roof["kernel_avg_ms"],
           "kernel_frac": roof["frac"], "kernel_achieved": roof["achieved"],
           "kernel_unit": roof["unit"], "traffic": roof["traffic"],
           "other_kernels_avg_ms": roof["other_kernels_avg_ms"],
           "algorithmic_bytes": r["algorithmic_bytes"], "flops": r["flops"],
           "step_roofline": r["step_roofline"], "plan_ms": r["plan_ms"]}
    if "mfma_busy" in roof:
        out["mfma_busy"] = roof["mfma_busy"]
    if "chunk_kernel_alone" in roof:
        out["chunk_kernel_alone"] = roof["chunk_kernel_alone"]
    return out


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="longtail",
                    choices=["tiny", "7b", "longtail", "straggler", "append", "prefill",
                             "migrate", "ce", "planner"])
    ap.add_argument("--extra-configs", default=",".join(EXTRA_CONFIGS),
                    help="decode / append workloads timed after the headline one and reported "
                         "under 'configs' (comma-separated; empty for none)")
    ap.add_argument("--extra-steps", type=int, default=20)
    ap.add_argument("--migrate-tokens", type=int, default=40960,
                    help="migrate workload: prefix length of the migrated request")
    ap.add_argument("--migrate-tp", default="1,2",
                    help="migrate workload: source and target TP degree (head shards)")
    ap.add_argument("--flush-mib", type=int, default=1024)
    ap.add_argument("--units-per-cu", type=int, default=3)
    ap.add_argument("--min-split-pages", type=int, default=16)
    ap.add_argument("--max-splits", type=int, default=64)
    ap.add_argument("--xcd-weights", default="measure",
                    help="plan's per-XCD weights: 'measure' (libra_xcd_read_weights on the "
                         "flush buffer), 'equal', or 8 comma-separated integers")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run a plain 1 GiB device-to-device copy 3 times (the known-size "
                         "reference that rocprofv3 FETCH_SIZE / WRITE_SIZE are scaled by)")
    args = ap.parse_args()

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU: the library has no multi-GPU path "
              "(run with --gpus 1)", file=sys.stderr)
        sys.exit(2)

    if args.workload == "planner":
        sys.path.insert(0, ROOT)
        print(json.dumps(bench_planner(args)), flush=True)
        return

    import torch
    if args.copy_calibration:
        n = 1 << 30
        src = torch.empty(n // 4, dtype=torch.float32, device="cuda").fill_(1.0)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_calibration_bytes_read": n, "copy_calibration_bytes_written": n,
                          "launches": 3}))
        return
    sys.path.insert(0, ROOT)
    from paper_2606_03077_amd import libra
    from paper_2606_03077_amd import workloads as wl

    libra.load()
    if len(libra.hip_runtimes_mapped()) != 1:
        raise RuntimeError(f"expected one HIP runtime, found {libra.hip_runtimes_mapped()}")
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    if args.workload == "migrate":
        print(json.dumps(bench_migrate(args, torch, libra, wl)), flush=True)
        return
    if args.workload == "ce":
        print(json.dumps(bench_ce(args, torch, libra)), flush=True)
        return

    flush = torch.empty(args.flush_mib * (1 << 20) // 4, dtype=torch.float32, device=dev)
    if args.xcd_weights == "measure":
        calib = flush if flush.numel() * 4 >= (1 << 30) else torch.empty(1 << 30, dtype=torch.uint8, device=dev)
        xcd_weight = libra.libra_xcd_read_weights(calib, reps=10, stream=torch.cuda.current_stream())
        del calib
        log(f"[bench] measured XCD read weights {xcd_weight}")
    elif args.xcd_weights == "equal":
        xcd_weight = [0] * 8
    else:
        xcd_weight = [int(x) for x in args.xcd_weights.split(",")]

    head = measure(args.workload, args, torch, libra, wl, flush, xcd_weight, args.steps,
                   args.warmup, 0.0 if args.no_cpu_baseline else args.cpu_seconds)
    result = {
        "metric": "KV TB/s and % HBM peak for ragged paged decode attn; decode tokens/s",
        "value": head["value"],
        "unit": "TB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": head["ms_per_step"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded; lengths and values as documented in workloads.py)",
    }
    result.update({k: v for k, v in head.items() if k not in ("value", "ms_per_step")})
    # The chip's achievable streaming read rate over as many bytes as the headline step
    # reads, beside the 8 TB/s figure: one pass timed to completion (ramp and tail
    # included, like any kernel), and the rate while every CU reads (fixed interval).
    def read_ceiling(nbytes):
        """Achievable read rate over a buffer of the step's size (>= 256 MiB)."""
        nbytes = max(1 << 28, (int(nbytes) + (1 << 20) - 1) >> 20 << 20)
        rbuf = torch.empty(nbytes, dtype=torch.uint8, device=dev)
        interval, completion = libra.libra_hbm_read_rate(rbuf, reps=5,
                                                         stream=torch.cuda.current_stream())
        del rbuf
        torch.cuda.empty_cache()
        log(f"[bench] HBM read ceiling: {completion:.0f} GB/s to completion, {interval:.0f} "
            f"GB/s over a fixed interval ({nbytes / 1e9:.2f} GB)")
        return {"completion_GBps": round(completion, 1), "interval_GBps": round(interval, 1),
                "bytes": nbytes,
                "kernel": "16-byte non-temporal loads, 2048 workgroups (libra_hbm_read_rate)"}

    def with_ceiling(roof, ceiling):
        if roof["unit"] == "GB/s":
            roof["frac_of_measured_read_ceiling"] = round(
                roof["achieved"] / ceiling["completion_GBps"], 4)

    result["hbm_read_ceiling"] = read_ceiling(head["algorithmic_bytes"])
    with_ceiling(result["roofline"], result["hbm_read_ceiling"])
    extras = [x for x in args.extra_configs.split(",") if x and x != args.workload]
    if extras:
        result["configs"] = {}
        for name in extras:
            r = measure(name, args, torch, libra, wl, flush, xcd_weight, args.extra_steps,
                        min(args.warmup, 3))
            c = config_summary(r)
            if not wl.WORKLOADS[name].append:
                c["hbm_read_ceiling"] = read_ceiling(r["algorithmic_bytes"])
                c["kernel_frac_of_measured_read_ceiling"] = round(
                    c["kernel_achieved"] / c["hbm_read_ceiling"]["completion_GBps"], 4)
            result["configs"][name] = c
            log(f"[bench] {name}: {r['ms_per_step']:.4f} ms/step, {r['value']:.3f} KV TB/s")
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
