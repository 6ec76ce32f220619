"""ctypes binding of liblibra.so: the C-ABI of include/libra.h, same names, same order.

Argument marshalling only.  torch supplies device memory and streams; every step of the
attention path runs in the library's HIP kernels.  There is no fallback: if the shared
library is missing or a call fails, an exception is raised.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence

import numpy as np

import torch  # loaded first, so that liblibra.so binds to the HIP runtime torch already mapped

_LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "liblibra.so")

LIBRA_OK = 0
STATUS_NAMES = {0: "LIBRA_OK", 1: "LIBRA_E_INVAL", 2: "LIBRA_E_UNSUPPORTED",
                3: "LIBRA_E_WORKSPACE", 4: "LIBRA_E_HIP", 5: "LIBRA_E_NOMEM"}
LIBRA_MODE_DECODE = 0
LIBRA_MODE_APPEND = 1
LIBRA_DTYPE_BF16 = 0
PAGE_SIZE = 16
HEAD_DIM = 128
UNIT_INTS = 12
UNIT_FIELDS = ("b", "g", "kv_begin", "kv_end", "q_begin", "q_end", "split", "n_splits",
               "part_base", "row0", "kind", "prior")

EXPORTS = ("libra_status_string", "libra_last_error", "libra_alloc_calls",
           "libra_kv_layout_create",
           "libra_kv_layout_destroy", "libra_kv_pack_pages", "libra_kv_unpack_pages",
           "libra_kv_gather", "libra_kv_copy_out", "libra_kv_copy_in", "libra_kv_reshard_host",
           "libra_xcd_read_weights", "libra_hbm_read_rate", "libra_splitkv_plan", "libra_plan_get_units",
           "libra_plan_get_info",
           "libra_plan_workspace_bytes", "libra_plan_upload", "libra_plan_destroy",
           "libra_decode_attn", "libra_decode_attn_noalloc", "libra_append_attn",
           "libra_profile_enable",
           "libra_profile_collect", "libra_ce_fit", "libra_ce_mape", "libra_ce_poly_sum",
           "libra_rollout_dp", "libra_trie_create", "libra_trie_destroy", "libra_trie_insert",
           "libra_trie_lookup", "libra_route_bucket")
TP_SLOTS = {1: 0, 2: 1, 4: 2, 8: 3}
KERNEL_KINDS = ("pack", "unpack", "gather", "cache_write", "decode", "merge", "chunk", "upload",
                "copy_out", "copy_in")


class LibraError(RuntimeError):
    def __init__(self, status: int, where: str, detail: str):
        super().__init__(f"{where}: {STATUS_NAMES.get(status, status)}: {detail}")
        self.status = status


class LayoutDesc(ctypes.Structure):
    _fields_ = [("num_pages", ctypes.c_int64), ("page_size", ctypes.c_int32),
                ("num_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32),
                ("dtype", ctypes.c_int32), ("k_cache", ctypes.c_void_p),
                ("v_cache", ctypes.c_void_p)]


class PlanParams(ctypes.Structure):
    _fields_ = [("num_cus", ctypes.c_int32), ("units_per_cu", ctypes.c_int32),
                ("min_split_pages", ctypes.c_int32), ("max_splits", ctypes.c_int32),
                ("q_tile", ctypes.c_int32), ("xcd_weight", ctypes.c_int32 * 8)]


class PlanDesc(ctypes.Structure):
    _fields_ = [("mode", ctypes.c_int32), ("batch", ctypes.c_int32),
                ("num_q_heads", ctypes.c_int32), ("num_kv_heads", ctypes.c_int32)]


class PlanInfo(ctypes.Structure):
    _fields_ = [("n_units", ctypes.c_int32), ("n_single", ctypes.c_int32),
                ("n_chunk", ctypes.c_int32), ("n_partial_slots", ctypes.c_int32),
                ("chunk_pages", ctypes.c_int64), ("q_tile", ctypes.c_int32),
                ("n_rows", ctypes.c_int32), ("n_write_tiles", ctypes.c_int32),
                ("num_cus", ctypes.c_int32), ("n_merge_groups", ctypes.c_int32),
                ("balanced", ctypes.c_int32)]


class CePoly(ctypes.Structure):
    _fields_ = [("gamma", ctypes.c_double), ("eta", ctypes.c_double), ("theta", ctypes.c_double)]


class RolloutModel(ctypes.Structure):
    _fields_ = [("attn_step", CePoly), ("linear_step", ctypes.c_double * 4),
                ("attn_scale", ctypes.c_double * 4)]


class KernelTimes(ctypes.Structure):
    _fields_ = [("ms", ctypes.c_double * len(KERNEL_KINDS)),
                ("launches", ctypes.c_int64 * len(KERNEL_KINDS))]


_lib = None


def library_path() -> str:
    return _LIB_PATH


def load() -> ctypes.CDLL:
    """Loads liblibra.so (once).  Raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH):
        raise RuntimeError(f"{_LIB_PATH} is missing: build it with "
                           "`python -m paper_2606_03077_amd.build` (no fallback exists)")
    lib = ctypes.CDLL(_LIB_PATH)
    P, I32, I64, SZ = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t
    I32P = ctypes.POINTER(ctypes.c_int32)
    I64P = ctypes.POINTER(ctypes.c_int64)
    DP = ctypes.POINTER(ctypes.c_double)
    sig = {
        "libra_status_string": (ctypes.c_char_p, [ctypes.c_int]),
        "libra_last_error": (ctypes.c_char_p, []),
        "libra_alloc_calls": (ctypes.c_uint64, []),
        "libra_kv_layout_create": (ctypes.c_int, [ctypes.POINTER(LayoutDesc), ctypes.POINTER(P)]),
        "libra_kv_layout_destroy": (None, [P]),
        "libra_kv_pack_pages": (ctypes.c_int, [P, P, P, I64, I64, P]),
        "libra_kv_unpack_pages": (ctypes.c_int, [P, P, P, I64, I64, P]),
        "libra_kv_gather": (ctypes.c_int, [P, P, I32, P, I32, I32, P, P, P]),
        "libra_kv_copy_out": (ctypes.c_int, [P, P, I64, P, P, P]),
        "libra_kv_copy_in": (ctypes.c_int, [P, P, I64, P, P, P]),
        "libra_kv_reshard_host": (ctypes.c_int, [ctypes.POINTER(P), I32, I32, ctypes.POINTER(P),
                                                 I32, I64]),
        "libra_splitkv_plan": (ctypes.c_int, [ctypes.POINTER(PlanDesc), I32P, I32P,
                                              ctypes.POINTER(PlanParams), ctypes.POINTER(P)]),
        "libra_xcd_read_weights": (ctypes.c_int, [P, SZ, I32, I32P, P]),
        "libra_hbm_read_rate": (ctypes.c_int, [P, SZ, I32, DP, DP, P]),
        "libra_plan_get_units": (ctypes.c_int, [P, ctypes.POINTER(I32P), I32P]),
        "libra_plan_get_info": (ctypes.c_int, [P, ctypes.POINTER(PlanInfo)]),
        "libra_plan_workspace_bytes": (SZ, [P]),
        "libra_plan_upload": (ctypes.c_int, [P, P, SZ, P]),
        "libra_plan_destroy": (None, [P]),
        "libra_decode_attn": (ctypes.c_int, [P, P, P, P, I32, I32, I32, ctypes.c_float, P, SZ,
                                             P, P, P]),
        "libra_decode_attn_noalloc": (ctypes.c_int, [P, P, P, P, I32, I32, I32, ctypes.c_float,
                                                     P, P, P]),
        "libra_append_attn": (ctypes.c_int, [P, P, P, P, P, P, I32, I32, I32, ctypes.c_float, P,
                                             SZ, P, P, P]),
        "libra_profile_enable": (ctypes.c_int, [ctypes.c_int]),
        "libra_profile_collect": (ctypes.c_int, [ctypes.POINTER(KernelTimes)]),
        "libra_ce_fit": (ctypes.c_int, [DP, DP, I32, ctypes.POINTER(CePoly)]),
        "libra_ce_mape": (ctypes.c_int, [ctypes.POINTER(CePoly), DP, DP, I32, DP]),
        "libra_ce_poly_sum": (ctypes.c_int, [ctypes.POINTER(CePoly), I64, I64, DP]),
        "libra_rollout_dp": (ctypes.c_int, [I64P, I32, I32, I32P, I32,
                                            ctypes.POINTER(RolloutModel), I32, DP, I32P, I32P,
                                            I32P]),
        "libra_trie_create": (ctypes.c_int, [I64P, I32, ctypes.POINTER(P)]),
        "libra_trie_destroy": (None, [P]),
        "libra_trie_insert": (ctypes.c_int, [P, I64, I32P, I32, I64P]),
        "libra_trie_lookup": (ctypes.c_int, [P, I64, I32P, I32, DP, I32P]),
        "libra_route_bucket": (ctypes.c_int, [DP, I32, DP, DP, I32, I32, I32P, DP]),
    }
    for name, (res, args) in sig.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    _lib = lib
    return lib


def hip_runtimes_mapped() -> list:
    """Paths of every libamdhip64 mapped into this process (there must be exactly one)."""
    with open("/proc/self/maps") as f:
        return sorted({line.split()[-1] for line in f if "libamdhip64" in line})


def _check(status: int, where: str):
    if status != LIBRA_OK:
        lib = load()
        raise LibraError(status, where, lib.libra_last_error().decode())


def _ptr(t) -> Optional[int]:
    if t is None:
        return None
    if isinstance(t, torch.Tensor):
        if t.device.type != "cuda":
            raise ValueError("device tensor expected")
        if not t.is_contiguous():
            raise ValueError("contiguous tensor expected")
        return t.data_ptr()
    return int(t)


def _host_ptr(t) -> Optional[int]:
    if t is None:
        return None
    if isinstance(t, torch.Tensor):
        if t.device.type != "cpu":
            raise ValueError("host tensor expected")
        if not t.is_contiguous():
            raise ValueError("contiguous tensor expected")
        return t.data_ptr()
    if isinstance(t, np.ndarray):
        if not t.flags.c_contiguous:
            raise ValueError("contiguous array expected")
        return t.ctypes.data
    return int(t)


def _run_ptr(t) -> Optional[int]:
    """A page run: a device tensor, or a host tensor / array (the library accepts pinned
    host memory and refuses pageable memory)."""
    if isinstance(t, torch.Tensor) and t.device.type == "cpu":
        return _host_ptr(t)
    if isinstance(t, np.ndarray):
        return _host_ptr(t)
    return _ptr(t)


def _stream(stream) -> Optional[int]:
    if stream is None:
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, torch.cuda.Stream):
        return stream.cuda_stream
    return int(stream)


def _i32_array(x) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(x, dtype=np.int32))


def libra_status_string(status: int) -> str:
    return load().libra_status_string(status).decode()


def libra_last_error() -> str:
    return load().libra_last_error().decode()


def libra_alloc_calls() -> int:
    """HIP allocate / free / event / stream creation calls the library has made so far."""
    return int(load().libra_alloc_calls())


def libra_kv_layout_create(k_cache, v_cache, num_pages: int, num_kv_heads: int,
                           page_size: int = PAGE_SIZE, head_dim: int = HEAD_DIM,
                           dtype: int = LIBRA_DTYPE_BF16) -> int:
    d = LayoutDesc(num_pages, page_size, num_kv_heads, head_dim, dtype, _ptr(k_cache),
                   _ptr(v_cache))
    h = ctypes.c_void_p()
    _check(load().libra_kv_layout_create(ctypes.byref(d), ctypes.byref(h)), "libra_kv_layout_create")
    return h.value


def libra_kv_layout_destroy(layout: int) -> None:
    load().libra_kv_layout_destroy(layout)


def libra_kv_pack_pages(layout: int, k_src, v_src, first_page: int, n_pages: int, stream=None):
    _check(load().libra_kv_pack_pages(layout, _ptr(k_src), _ptr(v_src), first_page, n_pages,
                                      _stream(stream)), "libra_kv_pack_pages")


def libra_kv_unpack_pages(layout: int, k_dst, v_dst, first_page: int, n_pages: int, stream=None):
    _check(load().libra_kv_unpack_pages(layout, _ptr(k_dst), _ptr(v_dst), first_page, n_pages,
                                        _stream(stream)), "libra_kv_unpack_pages")


def libra_kv_copy_out(layout: int, page_ids, n_pages: int, k_dst, v_dst, stream=None):
    """Gathers pages page_ids[:n_pages] (device int32) into packed runs k_dst / v_dst
    (device memory, or pinned host memory written directly over PCIe)."""
    _check(load().libra_kv_copy_out(layout, _ptr(page_ids), n_pages, _run_ptr(k_dst),
                                    _run_ptr(v_dst), _stream(stream)), "libra_kv_copy_out")


def libra_kv_copy_in(layout: int, page_ids, n_pages: int, k_src, v_src, stream=None):
    """Scatters packed runs k_src / v_src (device or pinned host memory) into pages
    page_ids[:n_pages] (distinct)."""
    _check(load().libra_kv_copy_in(layout, _ptr(page_ids), n_pages, _run_ptr(k_src),
                                   _run_ptr(v_src), _stream(stream)), "libra_kv_copy_in")


def libra_kv_reshard_host(src: Sequence, heads_per_src: int, dst: Sequence, n_pages: int):
    """Regroups host page runs along heads: len(src) shards of heads_per_src heads each
    become len(dst) shards of equal contiguous head ranges."""
    P = ctypes.c_void_p
    sp = (P * len(src))(*[_host_ptr(x) for x in src])
    dp = (P * len(dst))(*[_host_ptr(x) for x in dst])
    _check(load().libra_kv_reshard_host(sp, len(src), heads_per_src, dp, len(dst), n_pages),
           "libra_kv_reshard_host")


def libra_kv_gather(layout: int, block_table, bt_stride: int, cu_seq_lens, batch: int,
                    max_pages: int, k_out, v_out, stream=None):
    _check(load().libra_kv_gather(layout, _ptr(block_table), bt_stride, _ptr(cu_seq_lens), batch,
                                  max_pages, _ptr(k_out), _ptr(v_out), _stream(stream)),
           "libra_kv_gather")


def libra_splitkv_plan(mode: int, batch: int, num_q_heads: int, num_kv_heads: int,
                       seq_lens: Sequence[int], q_lens: Optional[Sequence[int]] = None,
                       num_cus: int = 0, units_per_cu: int = 3, min_split_pages: int = 16,
                       max_splits: int = 64, q_tile: int = 0,
                       xcd_weight: Optional[Sequence[int]] = None) -> int:
    """Builds a split plan (rule in include/libra.h).  xcd_weight: 8 relative HBM read rates
    of the XCDs for the slot placement (e.g. from libra_xcd_read_weights); None = equal."""
    d = PlanDesc(mode, batch, num_q_heads, num_kv_heads)
    w = list(xcd_weight) if xcd_weight is not None else [0] * 8
    if len(w) != 8:
        raise ValueError("xcd_weight needs 8 entries")
    p = PlanParams(num_cus, units_per_cu, min_split_pages, max_splits, q_tile,
                   (ctypes.c_int32 * 8)(*w))
    sl = _i32_array(seq_lens)
    ql = None if q_lens is None else _i32_array(q_lens)
    I32P = ctypes.POINTER(ctypes.c_int32)
    I64P = ctypes.POINTER(ctypes.c_int64)
    DP = ctypes.POINTER(ctypes.c_double)
    h = ctypes.c_void_p()
    _check(load().libra_splitkv_plan(ctypes.byref(d), sl.ctypes.data_as(I32P),
                                     None if ql is None else ql.ctypes.data_as(I32P),
                                     ctypes.byref(p), ctypes.byref(h)), "libra_splitkv_plan")
    return h.value


def libra_xcd_read_weights(buf, reps: int = 5, stream=None) -> list:
    """Per-XCD HBM read weights measured by streaming the device buffer `buf` (>= 1 GiB)."""
    w = (ctypes.c_int32 * 8)()
    nbytes = buf.numel() * buf.element_size()
    _check(load().libra_xcd_read_weights(_ptr(buf), nbytes, reps, w, _stream(stream)),
           "libra_xcd_read_weights")
    return list(w)


def libra_hbm_read_rate(buf, reps: int = 5, stream=None) -> tuple:
    """(fixed-interval GB/s, completion-timed GB/s) of streaming the device buffer `buf`
    (>= 1 GiB) with every CU reading."""
    iv, cp = ctypes.c_double(), ctypes.c_double()
    nbytes = buf.numel() * buf.element_size()
    _check(load().libra_hbm_read_rate(_ptr(buf), nbytes, reps, ctypes.byref(iv), ctypes.byref(cp),
                                      _stream(stream)), "libra_hbm_read_rate")
    return iv.value, cp.value


def libra_plan_get_units(plan: int) -> np.ndarray:
    ptr = ctypes.POINTER(ctypes.c_int32)()
    n = ctypes.c_int32()
    _check(load().libra_plan_get_units(plan, ctypes.byref(ptr), ctypes.byref(n)),
           "libra_plan_get_units")
    if n.value == 0:
        return np.zeros((0, UNIT_INTS), np.int32)
    return np.ctypeslib.as_array(ptr, shape=(n.value * UNIT_INTS,)).reshape(n.value, UNIT_INTS).copy()


def libra_plan_get_info(plan: int) -> dict:
    info = PlanInfo()
    _check(load().libra_plan_get_info(plan, ctypes.byref(info)), "libra_plan_get_info")
    return {name: getattr(info, name) for name, _ in PlanInfo._fields_}


def libra_plan_workspace_bytes(plan: int) -> int:
    return int(load().libra_plan_workspace_bytes(plan))


def libra_plan_upload(plan: int, workspace, ws_bytes: Optional[int] = None, stream=None):
    ws_bytes = workspace.numel() * workspace.element_size() if ws_bytes is None else ws_bytes
    _check(load().libra_plan_upload(plan, _ptr(workspace), ws_bytes, _stream(stream)),
           "libra_plan_upload")


def libra_plan_destroy(plan: int) -> None:
    load().libra_plan_destroy(plan)


def libra_decode_attn(layout: int, plan: int, q, block_table, bt_stride: int, batch: int,
                      num_q_heads: int, scale: float, workspace, out, lse=None, stream=None):
    ws_bytes = workspace.numel() * workspace.element_size()
    _check(load().libra_decode_attn(layout, plan, _ptr(q), _ptr(block_table), bt_stride, batch,
                                    num_q_heads, scale, _ptr(workspace), ws_bytes, _ptr(out),
                                    _ptr(lse), _stream(stream)), "libra_decode_attn")


def libra_decode_attn_noalloc(layout: int, plan: int, q, block_table, bt_stride: int,
                              batch: int, num_q_heads: int, scale: float, out, lse=None,
                              stream=None):
    _check(load().libra_decode_attn_noalloc(layout, plan, _ptr(q), _ptr(block_table), bt_stride,
                                            batch, num_q_heads, scale, _ptr(out), _ptr(lse),
                                            _stream(stream)), "libra_decode_attn_noalloc")


def libra_append_attn(layout: int, plan: int, q, k_new, v_new, block_table, bt_stride: int,
                      batch: int, num_q_heads: int, scale: float, workspace, out, lse=None,
                      stream=None):
    ws_bytes = workspace.numel() * workspace.element_size()
    _check(load().libra_append_attn(layout, plan, _ptr(q), _ptr(k_new), _ptr(v_new),
                                    _ptr(block_table), bt_stride, batch, num_q_heads, scale,
                                    _ptr(workspace), ws_bytes, _ptr(out), _ptr(lse),
                                    _stream(stream)), "libra_append_attn")


def libra_profile_enable(enable: bool = True) -> None:
    _check(load().libra_profile_enable(1 if enable else 0), "libra_profile_enable")


def libra_profile_collect() -> dict:
    """{kind: (total_ms, launches)} accumulated since the last collect."""
    t = KernelTimes()
    _check(load().libra_profile_collect(ctypes.byref(t)), "libra_profile_collect")
    return {k: (t.ms[i], t.launches[i]) for i, k in enumerate(KERNEL_KINDS)}


def alloc_workspace(plan: int, device="cuda") -> torch.Tensor:
    """A 256-byte aligned uint8 device buffer of the plan's workspace size."""
    n = max(256, libra_plan_workspace_bytes(plan))
    ws = torch.empty(n, dtype=torch.uint8, device=device)
    if ws.data_ptr() % 256:
        raise RuntimeError("torch returned a workspace that is not 256-byte aligned")
    return ws


# --- cost evaluator, rollout DP, prefix tree and routing (host only) ----------------

def _f64(x) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(x, dtype=np.float64))


def _i64(x) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(x, dtype=np.int64))


def _dp(a: np.ndarray):
    return a.ctypes.data_as(ctypes.POINTER(ctypes.c_double))


def _i32p(a: np.ndarray):
    return a.ctypes.data_as(ctypes.POINTER(ctypes.c_int32))


def _i64p(a: np.ndarray):
    return a.ctypes.data_as(ctypes.POINTER(ctypes.c_int64))


def _poly(p) -> CePoly:
    if isinstance(p, CePoly):
        return p
    g, e, t = p
    return CePoly(float(g), float(e), float(t))


def libra_ce_fit(lengths, times):
    """(gamma, eta, theta) of T(L) = gamma L^2 + eta L + theta, least squares in relative error."""
    L, T = _f64(lengths), _f64(times)
    if L.shape != T.shape:
        raise ValueError("lengths and times differ in size")
    out = CePoly()
    _check(load().libra_ce_fit(_dp(L), _dp(T), len(L), ctypes.byref(out)), "libra_ce_fit")
    return out.gamma, out.eta, out.theta


def libra_ce_mape(poly, lengths, times) -> float:
    L, T = _f64(lengths), _f64(times)
    m = ctypes.c_double()
    pp = _poly(poly)
    _check(load().libra_ce_mape(ctypes.byref(pp), _dp(L), _dp(T), len(L), ctypes.byref(m)),
           "libra_ce_mape")
    return m.value


def libra_ce_poly_sum(poly, a: int, b: int) -> float:
    out = ctypes.c_double()
    pp = _poly(poly)
    _check(load().libra_ce_poly_sum(ctypes.byref(pp), a, b, ctypes.byref(out)),
           "libra_ce_poly_sum")
    return out.value


def rollout_model(attn_step, linear_step: dict, attn_scale: dict) -> RolloutModel:
    """linear_step / attn_scale map a TP degree (1, 2, 4, 8) to its figure."""
    m = RolloutModel()
    m.attn_step = _poly(attn_step)
    for tp, slot in TP_SLOTS.items():
        m.linear_step[slot] = float(linear_step.get(tp, 0.0))
        m.attn_scale[slot] = float(attn_scale.get(tp, 0.0))
    return m


def libra_rollout_dp(lengths, n_gpus: int, tp_set, model: RolloutModel, exact: bool = True):
    """Returns (makespan, order, instances) with instances a list of (tp, first, count)."""
    L = _i64(lengths)
    tps = _i32_array(tp_set)
    order = np.zeros(max(1, len(L)), dtype=np.int32)
    inst = np.zeros(3 * max(1, n_gpus), dtype=np.int32)
    k = ctypes.c_int32()
    ms = ctypes.c_double()
    _check(load().libra_rollout_dp(_i64p(L), len(L), n_gpus, _i32p(tps), len(tps),
                                   ctypes.byref(model), int(bool(exact)), ctypes.byref(ms),
                                   _i32p(order), _i32p(inst), ctypes.byref(k)),
           "libra_rollout_dp")
    return ms.value, order[:len(L)].copy(), [tuple(int(v) for v in inst[3 * j:3 * j + 3])
                                              for j in range(k.value)]


class PrefixTree:
    """Owns a libra_trie handle (residual-length histograms over tool-return histories)."""

    def __init__(self, bin_edges):
        e = _i64(bin_edges)
        self.n_bins = len(e) + 1
        h = ctypes.c_void_p()
        _check(load().libra_trie_create(_i64p(e) if len(e) else None, len(e), ctypes.byref(h)),
               "libra_trie_create")
        self.handle = h

    def insert(self, prompt_id: int, states, residual):
        st, r = _i32_array(states), _i64(residual)
        if len(r) != len(st) + 1:
            raise ValueError("residual needs one entry per state plus one")
        _check(load().libra_trie_insert(self.handle, prompt_id, _i32p(st), len(st), _i64p(r)),
               "libra_trie_insert")

    def lookup(self, prompt_id: int, states):
        st = _i32_array(states)
        hist = np.zeros(self.n_bins, dtype=np.float64)
        d = ctypes.c_int32()
        _check(load().libra_trie_lookup(self.handle, prompt_id, _i32p(st), len(st), _dp(hist),
                                        ctypes.byref(d)), "libra_trie_lookup")
        return hist, d.value

    def close(self):
        if self.handle:
            load().libra_trie_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def libra_route_bucket(hist, t_dec, c_mig, current: int):
    """(best bucket, its cost); t_dec is [buckets][bins], c_mig [buckets][buckets]."""
    h, td, cm = _f64(hist), _f64(t_dec), _f64(c_mig)
    M = td.shape[0]
    if td.shape != (M, len(h)) or cm.shape != (M, M):
        raise ValueError("t_dec must be [buckets][bins] and c_mig [buckets][buckets]")
    best = ctypes.c_int32()
    cost = ctypes.c_double()
    _check(load().libra_route_bucket(_dp(h), len(h), _dp(td), _dp(cm), M, current,
                                     ctypes.byref(best), ctypes.byref(cost)),
           "libra_route_bucket")
    return best.value, cost.value
