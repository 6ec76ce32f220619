"""Request migration on the GPU (Sec. 5, Steps 1-3): offload, head reshard, reload.

Step 1 gathers a request's pages into a packed run (``libra_kv_copy_out``) and copies it
to pinned host memory; Step 2 regroups the run along heads on the host
(``libra_kv_reshard_host``); Step 3 copies each head shard back and scatters it into
fresh pages of a target cache with that shard's head count (``libra_kv_copy_in``).  On
one GPU the "target GPUs" are separate caches on the same device.

Parity: bytes are compared with the oracle's reshard of the request's logical pages
(bit-exact), and attention decoded on every target shard with the query heads that
travel with it is compared with the oracle's attention of the full model.
"""
import numpy as np
import pytest
import torch

from gpu_harness import assert_parity, dev_to_u16, say, u16_to_dev, DeviceCache
from oracle import decode_ref
from oracle.migration import query_heads_of_shard, request_pages, reshard_heads
from paper_2606_03077_amd import libra
from paper_2606_03077_amd import workloads as wl

pytestmark = pytest.mark.gpu

NAN_I16 = 0x7FC0   # bf16 quiet NaN: any page a reload misses poisons attention
TILE = 2048        # bf16 elements of one (page, head) tile


class Cache:
    """An empty library-layout cache, every element NaN."""

    def __init__(self, num_pages, hkv):
        self.num_pages, self.hkv = num_pages, hkv
        self.k = torch.full((num_pages * hkv * TILE,), NAN_I16, dtype=torch.int16, device="cuda")
        self.v = torch.full_like(self.k, NAN_I16)
        self.layout = libra.libra_kv_layout_create(self.k, self.v, num_pages, hkv)

    def unpack(self):
        k = torch.empty_like(self.k)
        v = torch.empty_like(self.v)
        libra.libra_kv_unpack_pages(self.layout, k, v, 0, self.num_pages)
        torch.cuda.synchronize()
        shape = (self.num_pages, self.hkv, 16, 128)
        return dev_to_u16(k).reshape(shape), dev_to_u16(v).reshape(shape)

    def close(self):
        libra.libra_kv_layout_destroy(self.layout)


def offload(layout, hkv, ids_dev, n):
    """Step 1: pages -> packed device run -> pinned host run (K and V)."""
    run_k = torch.empty(n * hkv * TILE, dtype=torch.int16, device="cuda")
    run_v = torch.empty_like(run_k)
    libra.libra_kv_copy_out(layout, ids_dev, n, run_k, run_v)
    host_k = torch.empty(run_k.shape, dtype=torch.int16, pin_memory=True)
    host_v = torch.empty(run_v.shape, dtype=torch.int16, pin_memory=True)
    host_k.copy_(run_k, non_blocking=True)
    host_v.copy_(run_v, non_blocking=True)
    torch.cuda.synchronize()
    return host_k, host_v


def reshard(host_runs, heads_per_src, n_dst, n):
    """Step 2 on the host: source runs -> n_dst runs of equal contiguous head ranges."""
    H = len(host_runs) * heads_per_src
    outs = [torch.empty(n * (H // n_dst) * TILE, dtype=torch.int16, pin_memory=True)
            for _ in range(n_dst)]
    libra.libra_kv_reshard_host(host_runs, heads_per_src, outs, n)
    return outs


def reload(cache, ids_dev, n, host_k, host_v):
    """Step 3: pinned host run -> device -> pages ids of the target cache."""
    dk = host_k.to("cuda", non_blocking=True)
    dv = host_v.to("cuda", non_blocking=True)
    libra.libra_kv_copy_in(cache.layout, ids_dev, n, dk, dv)
    torch.cuda.synchronize()


def migrate(src_layouts, src_hkv, src_ids, n, n_dst, dst_pages, seed):
    """Offloads one request from every source shard, reshards to n_dst, reloads each
    target shard into fresh (randomly placed) pages; returns (targets, their page ids)."""
    hk, hv = [], []
    for lay, ids in zip(src_layouts, src_ids):
        k, v = offload(lay, src_hkv, ids, n)
        hk.append(k)
        hv.append(v)
    H = len(src_layouts) * src_hkv
    ks = reshard(hk, src_hkv, n_dst, n)
    vs = reshard(hv, src_hkv, n_dst, n)
    rng = np.random.default_rng(seed)
    targets, ids_np = [], []
    for j in range(n_dst):
        c = Cache(dst_pages, H // n_dst)
        ids = rng.permutation(dst_pages)[:n].astype(np.int32)
        reload(c, torch.from_numpy(ids).cuda(), n, ks[j], vs[j])
        targets.append(c)
        ids_np.append(ids)
    return targets, ids_np


def decode_shard(cache, ids, L, q_rows, hq, scale):
    """Decode of the one migrated request on a target shard (its own block table)."""
    hkv = cache.hkv
    plan = libra.libra_splitkv_plan(libra.LIBRA_MODE_DECODE, 1, hq, hkv, [L], None)
    try:
        ws = libra.alloc_workspace(plan)
        bt = torch.from_numpy(np.ascontiguousarray(ids[None, :])).cuda()
        q = u16_to_dev(q_rows)
        out = torch.empty((1, hq, 128), dtype=torch.int16, device="cuda")
        lse = torch.empty((1, hq), dtype=torch.float32, device="cuda")
        libra.libra_decode_attn(cache.layout, plan, q, bt, bt.shape[1], 1, hq, scale, ws, out,
                                lse)
        torch.cuda.synchronize()
        o = wl.bf16_bits_to_f32(dev_to_u16(out)).astype(np.float64)
        return o, lse.cpu().numpy().astype(np.float64)
    finally:
        libra.libra_plan_destroy(plan)


@pytest.mark.parametrize("hq,hkv,n_dst", [(32, 8, 2), (32, 8, 8), (28, 4, 4), (8, 2, 1)])
def test_offload_reshard_reload(hq, hkv, n_dst):
    """TP 1 -> n_dst: target bytes equal the oracle's shards; decode on each shard
    equals the oracle's full-model attention for its query heads; TP n_dst -> 1 back
    restores the request's pages bit for bit."""
    say(f"[case] migrate TP1->TP{n_dst} hq={hq} hkv={hkv}")
    batch = wl.custom_batch([300, 1000, 47], num_q_heads=hq, num_kv_heads=hkv, seed=hkv + n_dst)
    src = DeviceCache(batch)
    b, L = 1, int(batch.seq_lens[1])
    n = -(-L // 16)
    ids = torch.from_numpy(np.ascontiguousarray(batch.block_table[b, :n])).cuda()
    targets, tids = migrate([src.layout], hkv, [ids], n, n_dst, dst_pages=n + 9, seed=n_dst)
    try:
        want_k = reshard_heads([request_pages(batch.k_pages, batch.block_table[b], L)], n_dst)
        want_v = reshard_heads([request_pages(batch.v_pages, batch.block_table[b], L)], n_dst)
        o_ref, l_ref = decode_ref(batch.q, batch.k_pages, batch.v_pages, batch.block_table,
                                  batch.seq_lens, batch.scale, batch_rows=[b])
        for j, (c, t) in enumerate(zip(targets, tids)):
            k, v = c.unpack()
            assert np.array_equal(k[t], want_k[j]) and np.array_equal(v[t], want_v[j])
            untouched = np.setdiff1d(np.arange(c.num_pages), t)
            assert (k[untouched] == NAN_I16).all() and (v[untouched] == NAN_I16).all()
            qh = query_heads_of_shard(j, n_dst, hq)
            o, lse = decode_shard(c, t, L, batch.q[b:b + 1, qh], hq // n_dst, batch.scale)
            assert_parity(o, lse, o_ref[b:b + 1, qh], l_ref[b:b + 1, qh],
                          label=f"shard {j}/{n_dst} decode after reload")
        # TP n_dst -> 1: join the shards back into one cache
        back, bids = migrate([c.layout for c in targets], hkv // n_dst,
                             [torch.from_numpy(t).cuda() for t in tids], n, 1,
                             dst_pages=n + 3, seed=99)
        k, v = back[0].unpack()
        assert np.array_equal(k[bids[0]], batch.k_pages[batch.block_table[b, :n]])
        assert np.array_equal(v[bids[0]], batch.v_pages[batch.block_table[b, :n]])
        back[0].close()
    finally:
        for c in targets:
            c.close()
        src.close()


def test_copy_edges():
    """Out-of-range ids are skipped, one side may be absent, an empty copy is a no-op."""
    say("[case] page copy edges")
    batch = wl.custom_batch([64], num_q_heads=8, num_kv_heads=2, seed=5)
    src = DeviceCache(batch)
    P = src.num_pages
    ids = torch.tensor([2, -1, P, 0], dtype=torch.int32, device="cuda")
    run = torch.full((4 * 2 * TILE,), 7, dtype=torch.int16, device="cuda")
    libra.libra_kv_copy_out(src.layout, ids, 4, None, run)      # V only
    torch.cuda.synchronize()
    r = dev_to_u16(run).reshape(4, 2, TILE)
    assert (r[1] == 7).all() and (r[2] == 7).all()               # skipped ids: untouched
    run_ref = torch.empty_like(run)
    libra.libra_kv_copy_out(src.layout, torch.tensor([2, 0], dtype=torch.int32, device="cuda"),
                            2, None, run_ref[:2 * 2 * TILE])
    torch.cuda.synchronize()
    rr = dev_to_u16(run_ref[:2 * 2 * TILE]).reshape(2, 2, TILE)
    assert np.array_equal(r[0], rr[0]) and np.array_equal(r[3], rr[1])
    # copy_in with an id past the cache writes nothing
    dst = Cache(3, 2)
    libra.libra_kv_copy_in(dst.layout, torch.tensor([3, 1], dtype=torch.int32, device="cuda"), 2,
                           run[:2 * 2 * TILE], run[2 * 2 * TILE:])
    libra.libra_kv_copy_in(dst.layout, torch.tensor([0], dtype=torch.int32, device="cuda"), 0,
                           run, run)
    torch.cuda.synchronize()
    k = dev_to_u16(dst.k).reshape(3, 2, TILE)
    v = dev_to_u16(dst.v).reshape(3, 2, TILE)
    assert np.array_equal(k[1], r[1]) and np.array_equal(v[1], r[3])
    assert (k[[0, 2]] == NAN_I16).all() and (v[[0, 2]] == NAN_I16).all()
    dst.close()
    src.close()


def test_migrate_40k_token_request_tp1_to_tp2():
    """A 40,960-token request of a 40-query-head / 8-KV-head model, TP 1 -> 2: every
    page bit-exact; decode on both shards against the oracle."""
    say("[case] migrate 40960-token request TP1->TP2")
    hq, hkv, L = 40, 8, 40960
    batch = wl.custom_batch([L], num_q_heads=hq, num_kv_heads=hkv, seed=40960)
    src = DeviceCache(batch)
    n = L // 16
    ids = torch.from_numpy(np.ascontiguousarray(batch.block_table[0, :n])).cuda()
    targets, tids = migrate([src.layout], hkv, [ids], n, 2, dst_pages=n + 64, seed=1)
    try:
        want_k = reshard_heads([request_pages(batch.k_pages, batch.block_table[0], L)], 2)
        want_v = reshard_heads([request_pages(batch.v_pages, batch.block_table[0], L)], 2)
        o_ref, l_ref = decode_ref(batch.q, batch.k_pages, batch.v_pages, batch.block_table,
                                  batch.seq_lens, batch.scale)
        for j, (c, t) in enumerate(zip(targets, tids)):
            k, v = c.unpack()
            assert np.array_equal(k[t], want_k[j]) and np.array_equal(v[t], want_v[j])
            qh = query_heads_of_shard(j, 2, hq)
            o, lse = decode_shard(c, t, L, batch.q[0:1, qh], hq // 2, batch.scale)
            assert_parity(o, lse, o_ref[:, qh], l_ref[:, qh], label=f"40K shard {j} decode")
    finally:
        for c in targets:
            c.close()
        src.close()


def test_direct_pcie_runs_match_staged():
    """Pinned host runs handed straight to the copy kernels (one kernel per direction,
    crossing PCIe) give the same bytes as the staged device-run + DMA path; pageable
    host memory is refused before any launch."""
    say("[case] direct pinned-host page runs")
    batch = wl.custom_batch([500, 77], num_q_heads=16, num_kv_heads=4, seed=11)
    src = DeviceCache(batch)
    n = -(-500 // 16)
    ids = torch.from_numpy(np.ascontiguousarray(batch.block_table[0, :n])).cuda()
    staged_k, staged_v = offload(src.layout, 4, ids, n)
    hk = torch.empty(staged_k.shape, dtype=torch.int16, pin_memory=True)
    hv = torch.empty(staged_v.shape, dtype=torch.int16, pin_memory=True)
    libra.libra_kv_copy_out(src.layout, ids, n, hk, hv)
    torch.cuda.synchronize()
    assert torch.equal(hk, staged_k) and torch.equal(hv, staged_v)
    dst = Cache(n + 5, 4)
    tid = torch.from_numpy(np.random.default_rng(3).permutation(n + 5)[:n].astype(np.int32)).cuda()
    libra.libra_kv_copy_in(dst.layout, tid, n, hk, hv)
    torch.cuda.synchronize()
    k, v = dst.unpack()
    t = tid.cpu().numpy()
    assert np.array_equal(k[t], batch.k_pages[batch.block_table[0, :n]])
    assert np.array_equal(v[t], batch.v_pages[batch.block_table[0, :n]])
    pageable = np.zeros(staged_k.shape[0], dtype=np.int16)
    with pytest.raises(libra.LibraError) as e:
        libra.libra_kv_copy_out(src.layout, ids, n, pageable, None)
    assert "pinned" in str(e.value)
    dst.close()
    src.close()


@pytest.mark.parametrize("n_dst", [1, 2, 4])
def test_decode_after_reload_equals_before(n_dst):
    """Decode on the migrated shards is bit-identical to decode on the source cache, for
    each shard's query heads, when both run one unit per (sequence, KV head): every head's
    unit then reads the same key tiles in the same order and does the same arithmetic."""
    say(f"[case] decode after reload equals before, TP1->TP{n_dst}")
    hq, hkv = 32, 8
    batch = wl.custom_batch([2000], num_q_heads=hq, num_kv_heads=hkv, seed=77 + n_dst)
    L = int(batch.seq_lens[0])
    n = -(-L // 16)
    src = DeviceCache(batch)
    no_split = dict(min_split_pages=1 << 20, max_splits=1)
    ids_np = np.ascontiguousarray(batch.block_table[0, :n])

    def decode(layout, heads_q, heads_kv, bt_row, q_rows):
        plan = libra.libra_splitkv_plan(libra.LIBRA_MODE_DECODE, 1, heads_q, heads_kv, [L], None,
                                        **no_split)
        try:
            assert libra.libra_plan_get_info(plan)["n_partial_slots"] == 0
            ws = libra.alloc_workspace(plan)
            bt = torch.from_numpy(np.ascontiguousarray(bt_row[None, :])).cuda()
            out = torch.empty((1, heads_q, 128), dtype=torch.int16, device="cuda")
            lse = torch.empty((1, heads_q), dtype=torch.float32, device="cuda")
            libra.libra_decode_attn(layout, plan, u16_to_dev(q_rows), bt, bt.shape[1], 1, heads_q,
                                    batch.scale, ws, out, lse)
            torch.cuda.synchronize()
            return dev_to_u16(out), lse.cpu().numpy()
        finally:
            libra.libra_plan_destroy(plan)

    o_before, l_before = decode(src.layout, hq, hkv, ids_np, batch.q[0:1])
    targets, tids = migrate([src.layout], hkv, [torch.from_numpy(ids_np).cuda()], n, n_dst,
                            dst_pages=n + 7, seed=3)
    try:
        for j, (c, t) in enumerate(zip(targets, tids)):
            qh = query_heads_of_shard(j, n_dst, hq)
            o, l = decode(c.layout, hq // n_dst, hkv // n_dst, t,
                          np.ascontiguousarray(batch.q[0:1, qh]))
            assert np.array_equal(o, o_before[:, qh]), f"shard {j}: output differs"
            assert np.array_equal(l, l_before[:, qh]), f"shard {j}: lse differs"
    finally:
        for c in targets:
            c.close()
        src.close()
