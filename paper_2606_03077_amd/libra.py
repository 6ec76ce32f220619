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

EXPORTS = ("libra_status_string", "libra_last_error", "libra_kv_layout_create",
           "libra_kv_layout_destroy", "libra_kv_pack_pages", "libra_kv_unpack_pages",
           "libra_kv_gather", "libra_kv_copy_out", "libra_kv_copy_in", "libra_kv_reshard_host",
           "libra_splitkv_plan", "libra_plan_get_units", "libra_plan_get_info",
           "libra_plan_workspace_bytes", "libra_plan_upload", "libra_plan_destroy",
           "libra_decode_attn", "libra_append_attn", "libra_profile_enable",
           "libra_profile_collect")
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
                ("q_tile", ctypes.c_int32)]


class PlanDesc(ctypes.Structure):
    _fields_ = [("mode", ctypes.c_int32), ("batch", ctypes.c_int32),
                ("num_q_heads", ctypes.c_int32), ("num_kv_heads", ctypes.c_int32)]


class PlanInfo(ctypes.Structure):
    _fields_ = [("n_units", ctypes.c_int32), ("n_single", ctypes.c_int32),
                ("n_chunk", ctypes.c_int32), ("n_partial_slots", ctypes.c_int32),
                ("chunk_pages", ctypes.c_int64), ("q_tile", ctypes.c_int32),
                ("n_rows", ctypes.c_int32), ("n_write_tiles", ctypes.c_int32),
                ("num_cus", ctypes.c_int32), ("n_merge_groups", ctypes.c_int32)]


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
    sig = {
        "libra_status_string": (ctypes.c_char_p, [ctypes.c_int]),
        "libra_last_error": (ctypes.c_char_p, []),
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
        "libra_plan_get_units": (ctypes.c_int, [P, ctypes.POINTER(I32P), I32P]),
        "libra_plan_get_info": (ctypes.c_int, [P, ctypes.POINTER(PlanInfo)]),
        "libra_plan_workspace_bytes": (SZ, [P]),
        "libra_plan_upload": (ctypes.c_int, [P, P, SZ, P]),
        "libra_plan_destroy": (None, [P]),
        "libra_decode_attn": (ctypes.c_int, [P, P, P, P, I32, I32, I32, ctypes.c_float, P, SZ,
                                             P, P, P]),
        "libra_append_attn": (ctypes.c_int, [P, P, P, P, P, P, I32, I32, I32, ctypes.c_float, P,
                                             SZ, P, P, P]),
        "libra_profile_enable": (ctypes.c_int, [ctypes.c_int]),
        "libra_profile_collect": (ctypes.c_int, [ctypes.POINTER(KernelTimes)]),
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
                       num_cus: int = 0, units_per_cu: int = 4, min_split_pages: int = 16,
                       max_splits: int = 64, q_tile: int = 0) -> int:
    d = PlanDesc(mode, batch, num_q_heads, num_kv_heads)
    p = PlanParams(num_cus, units_per_cu, min_split_pages, max_splits, q_tile)
    sl = _i32_array(seq_lens)
    ql = None if q_lens is None else _i32_array(q_lens)
    I32P = ctypes.POINTER(ctypes.c_int32)
    h = ctypes.c_void_p()
    _check(load().libra_splitkv_plan(ctypes.byref(d), sl.ctypes.data_as(I32P),
                                     None if ql is None else ql.ctypes.data_as(I32P),
                                     ctypes.byref(p), ctypes.byref(h)), "libra_splitkv_plan")
    return h.value


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
