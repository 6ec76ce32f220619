"""The static-scratch decode entry point (for callers that cannot allocate) against the
workspace entry point, through the C-ABI: the same kernels on the same plan tables give
bit-identical outputs.  Two plans take turns on the scratch: a large batch twice (the
second call finds its tables already there), a smaller batch (its tables replace them),
then the large batch again (its tables must be copied back).  Outputs start as NaN, so a
row that no kernel wrote would show."""
import numpy as np
import pytest
import torch

import oracle
from paper_2606_03077_amd import libra
from paper_2606_03077_amd import workloads as wl

import gpu_harness as H

pytestmark = pytest.mark.gpu

LIBRA_E_WORKSPACE = 3


class _Case:
    def __init__(self, batch, params):
        self.batch = batch
        self.w = batch.workload
        self.B = len(batch.seq_lens)
        self.cache = H.DeviceCache(batch)
        self.plan = H.plan_for(batch, **params)
        self.q = H.u16_to_dev(batch.q)
        self.ws = libra.alloc_workspace(self.plan)
        self.oracle = oracle.decode_ref(batch.q, batch.k_pages, batch.v_pages,
                                        batch.block_table, batch.seq_lens, batch.scale)

    def run(self, noalloc: bool):
        out = torch.full((self.B, self.w.num_q_heads, 128), 0x7FC0, dtype=torch.int16,
                         device="cuda")
        lse = torch.full((self.B, self.w.num_q_heads), float("nan"), dtype=torch.float32,
                         device="cuda")
        args = (self.cache.layout, self.plan, self.q, self.cache.bt, self.cache.bt_stride,
                self.B, self.w.num_q_heads, self.batch.scale)
        if noalloc:
            libra.libra_decode_attn_noalloc(*args, out, lse)
        else:
            libra.libra_decode_attn(*args, self.ws, out, lse)
        torch.cuda.synchronize()
        return H.dev_to_u16(out), lse.cpu().numpy()

    def close(self):
        libra.libra_plan_destroy(self.plan)
        self.cache.close()


def test_noalloc_decode_equals_workspace_decode_on_calls_in_a_row():
    params = dict(num_cus=64, units_per_cu=2, min_split_pages=2)
    big = _Case(wl.custom_batch([3000, 17, 5000, 129, 2048, 1, 700, 4097], num_q_heads=28,
                                num_kv_heads=4, seed=41), params)
    small = _Case(wl.custom_batch([900, 33, 1500], num_q_heads=28, num_kv_heads=4, seed=42),
                  params)
    try:
        assert libra.libra_plan_get_info(big.plan)["n_partial_slots"] > 0
        for label, case in [("large batch (8 rows)", big), ("same plan again", big),
                            ("smaller batch (3 rows)", small),
                            ("large batch, tables copied back", big)]:
            H.say(f"[case] noalloc decode: {label}")
            ref_o, ref_l = case.run(noalloc=False)
            o, l = case.run(noalloc=True)
            assert np.array_equal(o, ref_o), f"{label}: outputs differ from the workspace call"
            assert np.array_equal(l, ref_l), f"{label}: LSE differs from the workspace call"
            H.assert_parity(wl.bf16_bits_to_f32(o).astype(np.float64), l.astype(np.float64),
                            case.oracle[0], case.oracle[1], label=f"noalloc {label}")
    finally:
        big.close()
        small.close()


def test_noalloc_decode_rejects_plans_beyond_the_scratch():
    H.say("[case] noalloc decode: plan larger than the scratch")
    plan = libra.libra_splitkv_plan(libra.LIBRA_MODE_DECODE, 40, 32, 8, [65536] * 40, None,
                                    num_cus=4096, min_split_pages=1)
    buf = torch.zeros(1 << 20, dtype=torch.int16, device="cuda")
    lay = libra.libra_kv_layout_create(buf, buf, 8, 8)
    try:
        assert libra.libra_plan_workspace_bytes(plan) > (8 << 20)
        # refused on the host, before anything is enqueued
        with pytest.raises(libra.LibraError) as e:
            libra.libra_decode_attn_noalloc(lay, plan, buf, buf.view(torch.int32), 4096, 40, 32,
                                            0.088, buf, None)
        assert e.value.status == LIBRA_E_WORKSPACE
    finally:
        libra.libra_kv_layout_destroy(lay)
        libra.libra_plan_destroy(plan)
