"""HIP graph capture of decode and append calls.

A call whose workspace already holds its plan's tables enqueues kernels only (no
allocation, host copy, memset or event), so it can be captured into a HIP graph.  The
graph is replayed several times, with eager library calls and synchronisations between
the replays, and every replay must reproduce the eager call's outputs bit for bit: the
kernels are deterministic (fixed unit tables, fixed merge order).
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2606_03077_amd import libra
from paper_2606_03077_amd import workloads as wl

import gpu_harness as H

pytestmark = pytest.mark.gpu

REPLAYS = 3


def _capture(fn) -> torch.cuda.CUDAGraph:
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        fn()
    torch.cuda.synchronize()
    return g


def _same_bits(a: torch.Tensor, b: torch.Tensor) -> bool:
    return torch.equal(a.view(torch.int32) if a.dtype == torch.float32 else a,
                       b.view(torch.int32) if b.dtype == torch.float32 else b)


def test_decode_of_two_layers_replays_from_a_graph():
    """Two layers (two caches, one plan, one workspace) with split rows, so each layer
    is decode_kernel + merge_kernel inside the graph."""
    lens = [3000, 17, 5000, 129, 2048]
    hq, hkv = 28, 4
    H.say(f"[case] graph decode lens={lens}")
    layers = [wl.custom_batch(lens, num_q_heads=hq, num_kv_heads=hkv, seed=s) for s in (41, 42)]
    caches = [H.DeviceCache(b) for b in layers]
    plan = libra.libra_splitkv_plan(libra.LIBRA_MODE_DECODE, len(lens), hq, hkv, lens, None,
                                    num_cus=64, units_per_cu=1, min_split_pages=2)
    assert libra.libra_plan_get_info(plan)["n_merge_groups"] > 0
    ws = libra.alloc_workspace(plan)
    qs = [H.u16_to_dev(b.q) for b in layers]
    shape_o, shape_l = (len(lens), hq, 128), (len(lens), hq)

    def call(i, out, lse):
        c = caches[i]
        libra.libra_decode_attn(c.layout, plan, qs[i], c.bt, c.bt_stride, len(lens), hq,
                                layers[i].scale, ws, out, lse)

    # Eager reference (this call also uploads the tables to ws).
    ref_o = [torch.empty(shape_o, dtype=torch.int16, device="cuda") for _ in layers]
    ref_l = [torch.empty(shape_l, dtype=torch.float32, device="cuda") for _ in layers]
    for i in range(2):
        call(i, ref_o[i], ref_l[i])
    torch.cuda.synchronize()
    ro, rl = oracle.decode_ref(layers[0].q, layers[0].k_pages, layers[0].v_pages,
                               layers[0].block_table, layers[0].seq_lens, layers[0].scale)
    H.assert_parity(H.bf16_dev_to_f64(ref_o[0]), ref_l[0].cpu().numpy().astype(np.float64),
                    ro, rl, label="eager layer 0")

    g_o = [torch.empty(shape_o, dtype=torch.int16, device="cuda") for _ in layers]
    g_l = [torch.empty(shape_l, dtype=torch.float32, device="cuda") for _ in layers]
    graph = _capture(lambda: [call(i, g_o[i], g_l[i]) for i in range(2)])
    scratch_o = torch.empty(shape_o, dtype=torch.int16, device="cuda")
    scratch_l = torch.empty(shape_l, dtype=torch.float32, device="cuda")
    for r in range(REPLAYS):
        for t in g_o:
            t.fill_(-1)
        for t in g_l:
            t.fill_(float("nan"))
        graph.replay()
        torch.cuda.synchronize()
        for i in range(2):
            assert _same_bits(g_o[i], ref_o[i]), f"replay {r} layer {i}: out differs"
            assert _same_bits(g_l[i], ref_l[i]), f"replay {r} layer {i}: lse differs"
        call(1 - r % 2, scratch_o, scratch_l)  # eager work on the same workspace in between
        torch.cuda.synchronize()
    H.say(f"[graph] decode: {REPLAYS} replays bit-identical to eager")
    del graph
    for c in caches:
        c.close()
    libra.libra_plan_destroy(plan)


def test_append_replays_from_a_graph():
    """Cache write + decode rows + chunk tiles + merge in one captured call.  Rewriting the
    new tokens on each replay stores the same bytes, so every replay sees the same cache."""
    seq_lens, q_lens = [600, 1500, 300, 2200], [1, 200, 64, 1]
    hq, hkv = 32, 8
    H.say(f"[case] graph append seq_lens={seq_lens} q_lens={q_lens}")
    b = wl.custom_batch(seq_lens, q_lens, num_q_heads=hq, num_kv_heads=hkv, seed=43)
    cache = H.DeviceCache(b)
    plan = H.plan_for(b, num_cus=32, units_per_cu=1, min_split_pages=2)
    info = libra.libra_plan_get_info(plan)
    assert info["n_chunk"] > 0 and info["n_single"] > 0
    ws = libra.alloc_workspace(plan)
    q, kn, vn = H.u16_to_dev(b.q), H.u16_to_dev(b.k_new), H.u16_to_dev(b.v_new)
    rows = b.q.shape[0]

    def call(out, lse):
        libra.libra_append_attn(cache.layout, plan, q, kn, vn, cache.bt, cache.bt_stride,
                                len(seq_lens), hq, b.scale, ws, out, lse)

    ref_o = torch.empty((rows, hq, 128), dtype=torch.int16, device="cuda")
    ref_l = torch.empty((rows, hq), dtype=torch.float32, device="cuda")
    call(ref_o, ref_l)
    torch.cuda.synchronize()
    ro, rl, _, _ = oracle.append_ref(b.q, b.k_new, b.v_new, b.k_pages, b.v_pages, b.block_table,
                                     b.seq_lens, b.q_lens, b.scale)
    H.assert_parity(H.bf16_dev_to_f64(ref_o), ref_l.cpu().numpy().astype(np.float64), ro, rl,
                    label="eager append")

    g_o = torch.empty_like(ref_o)
    g_l = torch.empty_like(ref_l)
    graph = _capture(lambda: call(g_o, g_l))
    scratch_o, scratch_l = torch.empty_like(ref_o), torch.empty_like(ref_l)
    for r in range(REPLAYS):
        g_o.fill_(-1)
        g_l.fill_(float("nan"))
        graph.replay()
        torch.cuda.synchronize()
        assert _same_bits(g_o, ref_o), f"replay {r}: out differs"
        assert _same_bits(g_l, ref_l), f"replay {r}: lse differs"
        call(scratch_o, scratch_l)
        torch.cuda.synchronize()
    H.say(f"[graph] append: {REPLAYS} replays bit-identical to eager")
    del graph
    cache.close()
    libra.libra_plan_destroy(plan)
