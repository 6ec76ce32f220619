"""Pins for the migration oracle (Sec. 5, Steps 1-3) and the library's host reshard.

The head reshard has a plain definition (join the source partitions along heads, cut
into equal contiguous ranges).  It is pinned by
  * a brute-force walk over every (page, head, element) of tiny inputs that states each
    direction of Step 2 separately (split one partition into k; join k partitions),
  * round trips through other TP degrees, which must return the input,
  * the property Step 3 relies on: decoding each target shard with the query heads that
    travel with it reproduces the full model's attention for those heads (grouped-query
    attention maps query head h to KV head h // G; a shard that broke that mapping would
    decode wrong values).
The library's ``libra_kv_reshard_host`` needs no GPU and is compared with the oracle
byte for byte here.
"""
import numpy as np
import pytest

from oracle import decode_ref
from oracle.migration import query_heads_of_shard, request_pages, reshard_heads
from paper_2606_03077_amd import workloads as wl


def _rand_pages(rng, n_pages, heads, inner=(4, 3)):
    return rng.integers(0, 1 << 16, size=(n_pages, heads, *inner), dtype=np.uint16)


def test_split_by_brute_force():
    # TP 1 -> 4 over 8 heads: target j holds source heads 2j, 2j + 1.
    rng = np.random.default_rng(1)
    src = _rand_pages(rng, 3, 8)
    out = reshard_heads([src], 4)
    assert len(out) == 4
    for j in range(4):
        assert out[j].shape == (3, 2, 4, 3)
        for p in range(3):
            for hh in range(2):
                for a in range(4):
                    for b in range(3):
                        assert out[j][p, hh, a, b] == src[p, 2 * j + hh, a, b]


def test_join_by_brute_force():
    # TP 4 -> 2 over 8 heads: target 0 joins sources 0, 1; target 1 joins sources 2, 3.
    rng = np.random.default_rng(2)
    srcs = [_rand_pages(rng, 2, 2) for _ in range(4)]
    out = reshard_heads(srcs, 2)
    for j in range(2):
        assert out[j].shape == (2, 4, 4, 3)
        for p in range(2):
            for hh in range(4):
                i, local = 2 * j + hh // 2, hh % 2
                for a in range(4):
                    for b in range(3):
                        assert out[j][p, hh, a, b] == srcs[i][p, local, a, b]


@pytest.mark.parametrize("path", [(1, 2, 1), (1, 8, 1), (2, 4, 2), (8, 2, 4, 1), (1, 4, 2, 8, 1)])
def test_round_trips_are_identity(path):
    rng = np.random.default_rng(3)
    full = _rand_pages(rng, 5, 8)
    shards = reshard_heads([full], path[0])
    for n in path[1:]:
        shards = reshard_heads(shards, n)
    assert len(shards) == path[-1]
    assert np.array_equal(np.concatenate(shards, axis=1), full)


def test_reshard_rejects_uneven_cut():
    with pytest.raises(ValueError):
        reshard_heads([np.zeros((1, 6, 1))], 4)


def test_request_pages_follow_the_block_table():
    pages = np.arange(10)[:, None] * np.ones((1, 2), dtype=np.int64)
    row = np.array([7, 2, 9, 9], dtype=np.int32)
    got = request_pages(pages, row, 33)    # 33 tokens -> 3 pages
    assert got[:, 0].tolist() == [7, 2, 9]
    assert request_pages(pages, row, 0).shape[0] == 0


@pytest.mark.parametrize("hq,hkv,n_dst", [(8, 2, 2), (32, 8, 4), (28, 4, 4), (16, 8, 8)])
def test_shard_decode_reproduces_full_heads(hq, hkv, n_dst):
    """Step 3: a target shard decodes its own query heads exactly as the full model."""
    batch = wl.custom_batch([37, 100, 5], num_q_heads=hq, num_kv_heads=hkv, seed=hq + n_dst)
    o, lse = decode_ref(batch.q, batch.k_pages, batch.v_pages, batch.block_table,
                        batch.seq_lens, batch.scale)
    ks = reshard_heads([batch.k_pages], n_dst)
    vs = reshard_heads([batch.v_pages], n_dst)
    for j in range(n_dst):
        qh = query_heads_of_shard(j, n_dst, hq)
        oj, lj = decode_ref(np.ascontiguousarray(batch.q[:, qh]), ks[j], vs[j],
                            batch.block_table, batch.seq_lens, batch.scale)
        assert np.array_equal(oj, o[:, qh]) and np.array_equal(lj, lse[:, qh])


# --- the library's host reshard against the oracle (no GPU involved) ---------------

@pytest.mark.parametrize("n_src,hps,n_dst", [(1, 8, 2), (1, 8, 8), (2, 4, 1), (4, 2, 2),
                                             (2, 4, 4), (1, 6, 3), (3, 2, 2), (8, 1, 1),
                                             (2, 3, 3)])
def test_library_reshard_host_matches_oracle(n_src, hps, n_dst):
    from paper_2606_03077_amd import libra
    rng = np.random.default_rng(n_src * 100 + hps * 10 + n_dst)
    n_pages = 7
    srcs = [_rand_pages(rng, n_pages, hps, (2048,)) for _ in range(n_src)]
    H = n_src * hps
    dsts = [np.full((n_pages, H // n_dst, 2048), 0xABCD, np.uint16) for _ in range(n_dst)]
    libra.libra_kv_reshard_host(srcs, hps, dsts, n_pages)
    for got, ref in zip(dsts, reshard_heads(srcs, n_dst)):
        assert np.array_equal(got, ref)


def test_library_reshard_host_threaded_run():
    """A 40 MiB run is split across host threads; the bytes must not change."""
    from paper_2606_03077_amd import libra
    rng = np.random.default_rng(9)
    src = _rand_pages(rng, 1280, 8, (2048,))
    dsts = [np.empty((1280, 4, 2048), np.uint16) for _ in range(2)]
    libra.libra_kv_reshard_host([src], 8, dsts, 1280)
    ref = reshard_heads([src], 2)
    assert all(np.array_equal(a, b) for a, b in zip(dsts, ref))
    back = np.empty_like(src)
    libra.libra_kv_reshard_host(dsts, 4, [back], 1280)
    assert np.array_equal(back, src)


def test_library_reshard_host_validation():
    from paper_2606_03077_amd import libra
    a = np.zeros((2, 6, 2048), np.uint16)
    outs = [np.zeros((2, 2, 2048), np.uint16) for _ in range(3)]
    bad4 = [np.zeros((2, 1, 2048), np.uint16) for _ in range(4)]
    with pytest.raises(libra.LibraError) as e:
        libra.libra_kv_reshard_host([a], 6, bad4, 2)      # 4 does not divide 6
    assert libra.STATUS_NAMES[e.value.status] == "LIBRA_E_INVAL"
    with pytest.raises(libra.LibraError):
        libra.libra_kv_reshard_host([a], 6, [a], 2)       # output overlaps input
    with pytest.raises(libra.LibraError):
        libra.libra_kv_reshard_host([a], 0, outs, 2)
    with pytest.raises(libra.LibraError):
        libra.libra_kv_reshard_host([a], 6, outs, -1)
    libra.libra_kv_reshard_host([a], 6, outs, 0)          # empty run: no-op
