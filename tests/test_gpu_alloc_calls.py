"""Decode and append calls allocate nothing once their plan exists.

The library counts every HIP call it makes that allocates or frees memory or creates an
event or a stream (libra_alloc_calls).  Plan creation takes its pinned table image and
events from a pool; after that, decode calls (workspace and static-scratch entry points)
and append calls whose plan runs decode rows beside chunk tiles (fork / join events,
auxiliary stream) must leave the count unchanged, on the first call of a plan (which
uploads its tables) and on later ones.  A plan built after another of the same size was
destroyed reuses the pooled image and events, so its creation allocates nothing either.
"""
import pytest
import torch

from paper_2606_03077_amd import libra
from paper_2606_03077_amd import workloads as wl

import gpu_harness as H

pytestmark = pytest.mark.gpu


def test_decode_and_append_calls_make_no_allocation_calls():
    libra.libra_profile_enable(False)
    params = dict(num_cus=16, units_per_cu=2, min_split_pages=2)
    dec = wl.custom_batch([3000, 17, 900, 1, 4097], num_q_heads=28, num_kv_heads=4, seed=5)
    app = wl.custom_batch([700, 300, 2100, 64], q_lens=[1, 200, 1, 64], num_q_heads=32,
                          num_kv_heads=8, seed=6)
    dcache, acache = H.DeviceCache(dec), H.DeviceCache(app)
    dplan = H.plan_for(dec, **params)
    aplan = H.plan_for(app, **params)
    info = libra.libra_plan_get_info(aplan)
    assert info["n_single"] > 0 and info["n_chunk"] > 0, info
    assert libra.libra_plan_get_info(dplan)["n_partial_slots"] > 0
    try:
        dws, aws = libra.alloc_workspace(dplan), libra.alloc_workspace(aplan)
        dq = H.u16_to_dev(dec.q)
        aq, kn, vn = H.u16_to_dev(app.q), H.u16_to_dev(app.k_new), H.u16_to_dev(app.v_new)
        dout = torch.empty((len(dec.seq_lens), 28, 128), dtype=torch.int16, device="cuda")
        dlse = torch.empty((len(dec.seq_lens), 28), dtype=torch.float32, device="cuda")
        rows = app.q.shape[0]
        aout = torch.empty((rows, 32, 128), dtype=torch.int16, device="cuda")
        alse = torch.empty((rows, 32), dtype=torch.float32, device="cuda")
        torch.cuda.synchronize()
        # The first no-alloc call on the device looks up the static scratch's address
        # (hipGetSymbolAddress, not an allocation): it is counted in the loop too.
        before = libra.libra_alloc_calls()
        for _ in range(3):
            libra.libra_decode_attn(dcache.layout, dplan, dq, dcache.bt, dcache.bt_stride,
                                    len(dec.seq_lens), 28, dec.scale, dws, dout, dlse)
            libra.libra_decode_attn_noalloc(dcache.layout, dplan, dq, dcache.bt,
                                            dcache.bt_stride, len(dec.seq_lens), 28, dec.scale,
                                            dout, dlse)
            libra.libra_append_attn(acache.layout, aplan, aq, kn, vn, acache.bt,
                                    acache.bt_stride, len(app.seq_lens), 32, app.scale, aws,
                                    aout, alse)
        torch.cuda.synchronize()
        after = libra.libra_alloc_calls()
        H.say(f"alloc calls: {before} before, {after} after 9 decode / append calls")
        assert after == before

        # A second plan of the same size after the first is destroyed: pooled image and
        # events, no allocation.
        libra.libra_plan_destroy(aplan)
        aplan = None
        before = libra.libra_alloc_calls()
        again = H.plan_for(app, **params)
        created = libra.libra_alloc_calls() - before
        libra.libra_plan_destroy(again)
        assert created == 0, created
    finally:
        libra.libra_plan_destroy(dplan)
        if aplan is not None:
            libra.libra_plan_destroy(aplan)
        dcache.close()
        acache.close()
