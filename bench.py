"""Benchmark of ragged paged-KV decode attention on one MI355X.

    python bench.py [--gpus 1] [--steps 50] [--warmup 5] [--workload 7b]

One step = one decode-attention call (the split-KV decode kernel, then the log-sum-exp
merge of split rows) over the whole synthetic batch, inputs resident in HBM.  Before each
timed step an untimed 1 GiB fill evicts L2 and the 256 MB MALL, so every step reads its
KV from HBM.  Each step is bracketed by HIP events on the stream the kernel runs on.
The host-side split plan is built once per batch step and shared by all layers of a
model; its time is reported separately (``plan_ms``) and is not part of a step.

Prints one JSON line (rank 0, N = 1):
  value = algorithmic KV bytes / mean step time (TB/s), plus decode tokens/s, the
  roofline of the dominant kernel (decode_kernel against 8 TB/s HBM; for the append
  workload chunk_kernel against 2.5 PFLOP/s bf16), and the fp64 oracle timed on the host
  cores (``cpu_baseline``).  The dominant kernel's average duration comes from a second
  timed pass in which the library brackets each of its kernels with HIP events.
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
    return {"kv": kv, "q": q, "o": o, "lse": lse, "block_table": bt,
            "total": kv + q + o + lse + bt}


def flops(batch) -> int:
    w = batch.workload
    L = batch.seq_lens.astype(np.int64)
    C = batch.q_lens.astype(np.int64)
    P = L - C
    pairs = int((w.num_q_heads * (C * P + C * (C + 1) // 2)).sum())
    return 4 * 128 * pairs


def kernel_source_sha() -> str:
    h = hashlib.sha256()
    for f in ("decode.hip", "internal.h"):
        with open(os.path.join(ROOT, "paper_2606_03077_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def traffic_from_profile(workload: str):
    """HBM bytes per launch of the decode kernel from committed rocprofv3 counters.

    Null unless profiles/counters.json was taken on the current kernel source.
    """
    try:
        with open(PROFILE_COUNTERS) as f:
            c = json.load(f)
    except (OSError, ValueError):
        return None
    e = c.get("decode_kernel", {}).get(workload)
    if not e or e.get("source_sha") != kernel_source_sha():
        return None
    return e.get("hbm_bytes_per_launch")


def _oracle_worker(args):
    rows, = args
    from threadpoolctl import threadpool_limits
    import oracle
    b = _ORACLE_BATCH
    with threadpool_limits(1):
        oracle.decode_ref(b.q, b.k_pages, b.v_pages, b.block_table, b.seq_lens, b.scale,
                          batch_rows=rows)
    return len(rows)


_ORACLE_BATCH = None


def cpu_baseline(batch, min_seconds: float = 10.0) -> dict:
    """The fp64 oracle on the host cores: the whole batch, repeated for >= min_seconds."""
    import multiprocessing as mp
    global _ORACLE_BATCH
    _ORACLE_BATCH = batch
    cores = len(os.sched_getaffinity(0))
    cores = max(1, min(cores, 16))
    B = len(batch.seq_lens)
    order = np.argsort(-batch.seq_lens)  # longest first, one sequence per task
    tasks = [([int(b)],) for b in order]
    ctx = mp.get_context("fork")
    kv_per_pass = algorithmic_bytes(batch)["kv"]
    passes = 0
    t0 = time.perf_counter()
    with ctx.Pool(cores) as pool:
        while True:
            list(pool.imap_unordered(_oracle_worker, tasks))
            passes += 1
            el = time.perf_counter() - t0
            if el >= min_seconds:
                break
    rate = kv_per_pass * passes / el
    return {"value": rate / 1e12, "unit": "TB/s", "cores": cores, "kind": "oracle",
            "sample": f"whole {batch.workload.name} batch ({B} sequences) x {passes} passes, "
                      f"{el:.1f} s, fp64 numpy, one process per core, one sequence per task",
            "decode_tokens_per_s": B * passes / el}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="7b",
                    choices=["tiny", "7b", "longtail", "straggler", "append", "prefill"])
    ap.add_argument("--flush-mib", type=int, default=1024)
    ap.add_argument("--units-per-cu", type=int, default=4)
    ap.add_argument("--min-split-pages", type=int, default=16)
    ap.add_argument("--max-splits", type=int, default=64)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=10.0)
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run a plain 1 GiB device-to-device copy 3 times (the known-size "
                         "reference that rocprofv3 FETCH_SIZE / WRITE_SIZE are scaled by)")
    args = ap.parse_args()

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU: this build has no multi-GPU path "
              "(run with --gpus 1)", file=sys.stderr)
        sys.exit(2)

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

    log(f"[bench] generating workload {args.workload}")
    t = time.perf_counter()
    batch = wl.make_batch(args.workload)
    log(f"[bench] generated in {time.perf_counter() - t:.1f} s")
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
    plan_kw = dict(units_per_cu=args.units_per_cu, min_split_pages=args.min_split_pages,
                   max_splits=args.max_splits)
    plan_times = []
    for _ in range(5):
        t = time.perf_counter()
        plan = libra.libra_splitkv_plan(mode, len(batch.seq_lens), w.num_q_heads, Hkv,
                                        batch.seq_lens.tolist(), ql, **plan_kw)
        plan_times.append((time.perf_counter() - t) * 1e3)
        libra.libra_plan_destroy(plan)
    plan = libra.libra_splitkv_plan(mode, len(batch.seq_lens), w.num_q_heads, Hkv,
                                    batch.seq_lens.tolist(), ql, **plan_kw)
    info = libra.libra_plan_get_info(plan)
    ws = libra.alloc_workspace(plan)
    stream = torch.cuda.current_stream()
    libra.libra_plan_upload(plan, ws, stream=stream)

    def step():
        if w.append:
            libra.libra_append_attn(layout, plan, q, kn, vn, bt, bt.shape[1], len(batch.seq_lens),
                                    w.num_q_heads, batch.scale, ws, out, lse, stream=stream)
        else:
            libra.libra_decode_attn(layout, plan, q, bt, bt.shape[1], len(batch.seq_lens),
                                    w.num_q_heads, batch.scale, ws, out, lse, stream=stream)

    flush = torch.empty(args.flush_mib * (1 << 20) // 4, dtype=torch.float32, device=dev)
    log(f"[bench] warmup {args.warmup}")
    for i in range(args.warmup):
        flush.fill_(float(i))
        step()
    torch.cuda.synchronize()

    starts = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps)]
    ends = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps)]
    log(f"[bench] timing {args.steps} steps")
    torch.cuda.synchronize()
    wall0 = time.perf_counter()
    for i in range(args.steps):
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
    for i in range(args.steps):
        flush.fill_(float(i))
        step()
    torch.cuda.synchronize()
    ktimes = libra.libra_profile_collect()
    libra.libra_profile_enable(False)
    kernel_avg_ms = {k: ms / n for k, (ms, n) in ktimes.items() if n}

    ab = algorithmic_bytes(batch)
    fl = flops(batch)
    kv_tbs = ab["kv"] / (mean_ms * 1e-3) / 1e12
    tokens_per_s = rows / (mean_ms * 1e-3)
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
                "traffic": None, "kernel": "chunk_kernel",
                "algorithmic_flops_per_launch": work}
    else:
        kern = "decode"
        achieved = ab["total"] / (kernel_avg_ms[kern] * 1e-3) / 1e9
        roof = {"bound": "hbm", "achieved": round(achieved, 2), "peak": HBM_PEAK_GBS,
                "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4),
                "traffic": traffic_from_profile(args.workload), "kernel": "decode_kernel",
                "algorithmic_bytes_per_launch": ab["total"]}
    roof["kernel_avg_ms"] = round(kernel_avg_ms[kern], 5)
    roof["other_kernels_avg_ms"] = {k: round(v, 5) for k, v in kernel_avg_ms.items() if k != kern}

    result = {
        "metric": "KV TB/s and % HBM peak for ragged paged decode attn; decode tokens/s",
        "value": round(kv_tbs, 4),
        "unit": "TB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(mean_ms, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded; lengths and values as documented in workloads.py)",
        "config": {"workload": f"{args.workload}: {w.description}", "batch": len(batch.seq_lens),
                   "num_q_heads": w.num_q_heads, "num_kv_heads": Hkv, "head_dim": 128,
                   "page_size": 16, "kv_tokens": int(batch.seq_lens.sum()),
                   "query_rows": rows, "seed": w.seed},
        "hbm_peak_frac": round(kv_tbs * 1e3 / HBM_PEAK_GBS, 4),
        "decode_tokens_per_s": round(tokens_per_s, 1),
        "step_ms_p10_p50_p90": [round(p10, 5), round(p50, 5), round(p90, 5)],
        "timed_wall_s": round(wall, 4),
        "plan_ms": round(float(np.median(plan_times)), 4),
        "plan": dict({k: info[k] for k in ("n_units", "n_single", "n_chunk", "n_partial_slots",
                                           "chunk_pages", "num_cus")}, **plan_kw),
        "algorithmic_bytes": ab["total"],
        "flops": fl,
        "roofline": roof,
    }
    if not args.no_cpu_baseline:
        log(f"[bench] timing the oracle on host cores (~{args.cpu_seconds:.0f} s)")
        result["cpu_baseline"] = cpu_baseline(batch, args.cpu_seconds)
    libra.libra_plan_destroy(plan)
    libra.libra_kv_layout_destroy(layout)
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
