"""Pins for the fp64 oracle: it must agree with things other than itself.

Each test ties the oracle to an independent fact: a library implementation of scaled
dot-product attention (torch CPU, float64) with its own causal-mask helper, closed
forms, or invariants that follow from the mathematics of softmax attention (page
permutation, key splitting with a log-sum-exp merge, head sharding).  The paper prints no
worked attention values, so these are the pins.
"""
import math

import numpy as np
import pytest
import scipy.special
import torch
import torch.nn.functional as F
from torch.nn.attention.bias import causal_lower_right

import oracle
import oracle.attention as oa
from oracle.attention import attend, gather_tokens
from paper_2606_03077_amd import workloads as wl

D = 128


def _torch_bf16(bits) -> np.ndarray:
    """bf16 bit patterns decoded by torch's own bfloat16 type, widened to float64.

    The SDPA references below take their inputs through this decoder, not the oracle's,
    so a slip in the oracle's bf16 decoding shows up as a disagreement."""
    a = np.ascontiguousarray(np.asarray(bits, dtype=np.uint16)).view(np.int16)
    return torch.from_numpy(a).view(torch.bfloat16).double().numpy()


def test_bf16_decoder_matches_torch_on_every_bit_pattern():
    """All 65,536 bf16 patterns decode to torch's bfloat16 values (NaN where torch gives
    NaN), plus closed forms read off the format: sign bit 15, 8 exponent bits with bias
    127, 7 fraction bits, subnormals below exponent 1."""
    bits = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16)
    got = oa.bf16_bits_to_f64(bits)
    ref = _torch_bf16(bits)
    nan = np.isnan(ref)
    assert np.array_equal(np.isnan(got), nan)
    assert np.array_equal(got[~nan], ref[~nan])
    assert np.array_equal(np.signbit(got[~nan]), np.signbit(ref[~nan]))   # -0.0 included
    closed = {0x0000: 0.0, 0x3F80: 1.0, 0xBF80: -1.0, 0x4000: 2.0, 0xC040: -3.0,
              0x3F81: 1.0 + 2.0 ** -7, 0x3E00: 0.125, 0x7F7F: (2.0 - 2.0 ** -7) * 2.0 ** 127,
              0x0080: 2.0 ** -126, 0x0001: 2.0 ** -133, 0x807F: -(127 * 2.0 ** -133),
              0x7F80: math.inf, 0xFF80: -math.inf}
    for b, v in closed.items():
        assert oa.bf16_bits_to_f64(np.array([b], np.uint16))[0] == v, hex(b)
    assert np.signbit(oa.bf16_bits_to_f64(np.array([0x8000], np.uint16))[0])
    assert np.isnan(oa.bf16_bits_to_f64(np.array([0x7FC0, 0xFFC1, 0x7F81], np.uint16))).all()


def _scatter_contiguous(K, block_table_row, pages, g):
    """Test-side placement of contiguous rows K [L, d] into pages (slot-major)."""
    for t in range(K.shape[0]):
        pages[block_table_row[t // 16], g, t % 16] = K[t]


def _sdpa(q, K, V, scale, mask=None):
    """torch float64 SDPA; q [Hq, R, d], K/V [Hq, N, d] -> o [Hq, R, d], lse [Hq, R]."""
    qt = torch.from_numpy(q)[None]
    kt = torch.from_numpy(K)[None]
    vt = torch.from_numpy(V)[None]
    o = F.scaled_dot_product_attention(qt, kt, vt, attn_mask=mask, scale=scale)[0].numpy()
    z = torch.einsum("hrd,hnd->hrn", qt[0], kt[0]) * scale
    if mask is not None:
        z = z.masked_fill(~mask, -math.inf)
    lse = torch.logsumexp(z, dim=-1).numpy()
    return o, lse


def _random_contig_batch(rng, lens, Hq, Hkv, q_lens=None):
    """Contiguous logical K/V drawn first, then placed into shuffled pages by the test."""
    B = len(lens)
    q_lens = [1] * B if q_lens is None else q_lens
    pages_per = [(L + 15) // 16 for L in lens]
    n_pages = sum(pages_per) + 3
    perm = rng.permutation(n_pages)
    bt = np.full((B, max(1, max(pages_per))), perm[-1], np.int32)
    off = 0
    for b, n in enumerate(pages_per):
        bt[b, :n] = perm[off:off + n]
        off += n
    kp = np.full((n_pages, Hkv, 16, D), wl.BF16_NAN, np.uint16)
    vp = kp.copy()
    Ks, Vs = [], []
    for b, L in enumerate(lens):
        K = wl.normal_bf16(rng, (Hkv, L, D))
        V = wl.normal_bf16(rng, (Hkv, L, D))
        for g in range(Hkv):
            _scatter_contiguous(K[g], bt[b], kp, g)
            _scatter_contiguous(V[g], bt[b], vp, g)
        Ks.append(K)
        Vs.append(V)
    q = wl.normal_bf16(rng, (sum(q_lens), Hq, D))
    return q, kp, vp, bt, Ks, Vs


@pytest.mark.parametrize("Hq,Hkv", [(8, 2), (28, 4), (4, 4), (16, 1)])
def test_decode_matches_torch_sdpa(Hq, Hkv):
    rng = np.random.default_rng(11)
    lens = [1, 15, 16, 17, 40, 64, 97]
    q, kp, vp, bt, Ks, Vs = _random_contig_batch(rng, lens, Hq, Hkv)
    scale = float(np.float32(1 / math.sqrt(D)))
    o, lse = oracle.decode_ref(q, kp, vp, bt, np.array(lens), scale)
    G = Hq // Hkv
    for b, L in enumerate(lens):
        # KV heads repeated G times in contiguous groups (torch repeat_interleave)
        K = np.repeat(_torch_bf16(Ks[b]), G, axis=0)
        V = np.repeat(_torch_bf16(Vs[b]), G, axis=0)
        qq = _torch_bf16(q[b])[:, None, :]
        ro, rl = _sdpa(qq, K, V, scale)
        np.testing.assert_allclose(o[b], ro[:, 0], rtol=0, atol=1e-12)
        np.testing.assert_allclose(lse[b], rl[:, 0], rtol=0, atol=1e-12)


@pytest.mark.parametrize("prior,chunk", [(0, 5), (7, 9), (16, 16), (33, 40), (50, 1)])
def test_append_matches_torch_sdpa_lower_right_causal(prior, chunk):
    rng = np.random.default_rng(prior * 100 + chunk)
    Hq, Hkv = 8, 2
    G = Hq // Hkv
    L = prior + chunk
    q, kp, vp, bt, Ks, Vs = _random_contig_batch(rng, [L], Hq, Hkv, q_lens=[chunk])
    # the cache holds only the prior; the new tokens come in k_new / v_new
    k_new = np.ascontiguousarray(Ks[0][:, prior:].transpose(1, 0, 2))
    v_new = np.ascontiguousarray(Vs[0][:, prior:].transpose(1, 0, 2))
    for t in range(prior, L):
        kp[bt[0, t // 16], :, t % 16] = wl.BF16_NAN
        vp[bt[0, t // 16], :, t % 16] = wl.BF16_NAN
    scale = 0.0883883461356163
    o, lse, kp2, vp2 = oracle.append_ref(q, k_new, v_new, kp, vp, bt, np.array([L]),
                                         np.array([chunk]), scale)
    K = np.repeat(_torch_bf16(Ks[0]), G, axis=0)
    V = np.repeat(_torch_bf16(Vs[0]), G, axis=0)
    qq = _torch_bf16(q).transpose(1, 0, 2)  # [Hq, chunk, d]
    mask = causal_lower_right(chunk, L)._materialize("cpu")
    ro, rl = _sdpa(qq, K, V, scale, mask)
    np.testing.assert_allclose(o.transpose(1, 0, 2), ro, rtol=0, atol=1e-12)
    np.testing.assert_allclose(lse.T, rl, rtol=0, atol=1e-12)
    # cache write: the written pages now hold exactly the new tokens
    for g in range(Hkv):
        np.testing.assert_array_equal(gather_tokens(kp2, bt[0], g, L), Ks[0][g])
        np.testing.assert_array_equal(gather_tokens(vp2, bt[0], g, L), Vs[0][g])


def test_single_key_returns_v_exactly():
    rng = np.random.default_rng(3)
    q, kp, vp, bt, Ks, Vs = _random_contig_batch(rng, [1, 1], 8, 2)
    scale = 0.125
    o, lse = oracle.decode_ref(q, kp, vp, bt, np.array([1, 1]), scale)
    for b in range(2):
        for h in range(8):
            g = h // 4
            assert np.array_equal(o[b, h], _torch_bf16(Vs[b][g, 0]))
            ref = scale * float(np.dot(_torch_bf16(q[b, h]), _torch_bf16(Ks[b][g, 0])))
            assert abs(lse[b, h] - ref) <= 1e-12 * max(1.0, abs(ref))


def test_identical_keys_give_mean_v_and_log_n():
    rng = np.random.default_rng(4)
    L = 37
    q, kp, vp, bt, Ks, Vs = _random_contig_batch(rng, [L], 4, 1)
    k0 = wl.normal_bf16(rng, (D,))
    for t in range(L):
        kp[bt[0, t // 16], 0, t % 16] = k0
    o, lse = oracle.decode_ref(q, kp, vp, bt, np.array([L]), 0.1)
    mean_v = _torch_bf16(Vs[0][0]).mean(axis=0)
    for h in range(4):
        np.testing.assert_allclose(o[0, h], mean_v, rtol=0, atol=1e-13)
        ref = 0.1 * np.dot(_torch_bf16(q[0, h]), _torch_bf16(k0)) + math.log(L)
        assert abs(lse[0, h] - ref) < 1e-12


def test_zero_query_gives_mean_v_and_log_n():
    rng = np.random.default_rng(5)
    L = 50
    q, kp, vp, bt, Ks, Vs = _random_contig_batch(rng, [L], 2, 2)
    q[:] = 0
    o, lse = oracle.decode_ref(q, kp, vp, bt, np.array([L]), 0.088)
    for h in range(2):
        np.testing.assert_allclose(o[0, h], _torch_bf16(Vs[0][h]).mean(axis=0), atol=1e-13, rtol=0)
        assert abs(lse[0, h] - math.log(L)) < 1e-13


def test_dominant_key_selects_its_value():
    rng = np.random.default_rng(6)
    L = 20
    q, kp, vp, bt, Ks, Vs = _random_contig_batch(rng, [L], 1, 1)
    q[0, 0] = wl.f32_to_bf16_bits(np.full(D, 1.0, np.float32))
    kp[bt[0, 0], 0, 7] = wl.f32_to_bf16_bits(np.full(D, 4.0, np.float32))  # logit 512 above the rest
    o, lse = oracle.decode_ref(q, kp, vp, bt, np.array([L]), 1.0)
    np.testing.assert_allclose(o[0, 0], _torch_bf16(Vs[0][0, 7]), atol=1e-12, rtol=0)


def test_lse_matches_scipy_logsumexp():
    rng = np.random.default_rng(7)
    K = rng.standard_normal((300, D))
    V = rng.standard_normal((300, D))
    qr = rng.standard_normal((3, D)) * 3
    o, lse = attend(qr, K, V, 0.3)
    z = 0.3 * qr @ K.T
    np.testing.assert_allclose(lse, scipy.special.logsumexp(z, axis=1), rtol=0, atol=1e-12)
    np.testing.assert_allclose(o, scipy.special.softmax(z, axis=1) @ V, rtol=0, atol=1e-12)


def test_page_permutation_invariance():
    b = wl.make_batch("tiny")
    o1, l1 = oracle.decode_ref(b.q, b.k_pages, b.v_pages, b.block_table, b.seq_lens, b.scale)
    rng = np.random.default_rng(99)
    perm = rng.permutation(b.num_pages)          # new physical id of old page p is perm[p]
    kp = np.empty_like(b.k_pages)
    vp = np.empty_like(b.v_pages)
    kp[perm] = b.k_pages
    vp[perm] = b.v_pages
    bt = perm[b.block_table].astype(np.int32)
    o2, l2 = oracle.decode_ref(b.q, kp, vp, bt, b.seq_lens, b.scale)
    assert np.array_equal(o1, o2) and np.array_equal(l1, l2)


@pytest.mark.parametrize("cuts", [[1], [16], [7, 8, 300], [0, 0, 5], [299], [100, 200]])
def test_split_anywhere_then_merge_equals_unsplit(cuts):
    rng = np.random.default_rng(len(cuts))
    N = 300
    K = rng.standard_normal((N, D))
    V = rng.standard_normal((N, D))
    qr = rng.standard_normal((4, D))
    full_o, full_l = attend(qr, K, V, 0.2)
    bounds = [0] + sorted(cuts) + [N]
    parts = [attend(qr, K[a:c], V[a:c], 0.2) for a, c in zip(bounds[:-1], bounds[1:])]
    mo, ml = oracle.merge_ref([p[0] for p in parts], [p[1] for p in parts])
    np.testing.assert_allclose(mo, full_o, rtol=0, atol=1e-12)
    np.testing.assert_allclose(ml, full_l, rtol=0, atol=1e-12)


def test_merge_degenerate_cases():
    o = np.arange(2 * 3 * 4, dtype=np.float64).reshape(2, 3, 4)
    lse = np.full((2, 3), -np.inf)
    mo, ml = oracle.merge_ref(o, lse)
    assert np.all(mo == 0) and np.all(ml == -np.inf)
    mo, ml = oracle.merge_ref(o[:1], np.zeros((1, 3)))
    assert np.array_equal(mo, o[0]) and np.all(ml == 0)


def test_empty_sequence_gives_zero_and_neg_inf():
    b = wl.custom_batch([0, 5], num_q_heads=4, num_kv_heads=2)
    o, lse = oracle.decode_ref(b.q, b.k_pages, b.v_pages, b.block_table, b.seq_lens, b.scale)
    assert np.all(o[0] == 0) and np.all(lse[0] == -np.inf)
    assert np.all(np.isfinite(o[1])) and np.all(np.isfinite(lse[1]))


def test_head_shard_equals_slice_of_full():
    # KV resharded along heads (Sec. 5, Step 2): a head subset is a slice of the result
    b = wl.make_batch("tiny")
    o, lse = oracle.decode_ref(b.q, b.k_pages, b.v_pages, b.block_table, b.seq_lens, b.scale)
    G = b.workload.group
    for g0, g1 in [(0, 1), (1, 2)]:
        os_, ls_ = oracle.decode_ref(b.q[:, g0 * G:g1 * G], b.k_pages[:, g0:g1],
                                     b.v_pages[:, g0:g1], b.block_table, b.seq_lens, b.scale)
        assert np.array_equal(os_, o[:, g0 * G:g1 * G]) and np.array_equal(ls_, lse[:, g0 * G:g1 * G])


def test_mha_equals_gqa_with_repeated_kv_heads():
    b = wl.custom_batch([20, 45, 3], num_q_heads=6, num_kv_heads=2, seed=8)
    o, lse = oracle.decode_ref(b.q, b.k_pages, b.v_pages, b.block_table, b.seq_lens, b.scale)
    kp = np.repeat(b.k_pages, 3, axis=1)
    vp = np.repeat(b.v_pages, 3, axis=1)
    o2, l2 = oracle.decode_ref(b.q, kp, vp, b.block_table, b.seq_lens, b.scale)
    np.testing.assert_allclose(o2, o, atol=1e-15, rtol=0)
    np.testing.assert_allclose(l2, lse, atol=1e-15, rtol=0)


def test_append_one_token_equals_decode_after_write():
    b = wl.custom_batch([30, 17, 64, 1], q_lens=[1, 1, 1, 1], num_q_heads=8, num_kv_heads=2,
                        seed=9, append=True)
    o, lse, kp, vp = oracle.append_ref(b.q, b.k_new, b.v_new, b.k_pages, b.v_pages,
                                       b.block_table, b.seq_lens, b.q_lens, b.scale)
    od, ld = oracle.decode_ref(b.q, kp, vp, b.block_table, b.seq_lens, b.scale)
    np.testing.assert_allclose(o, od, atol=1e-15, rtol=0)
    np.testing.assert_allclose(lse, ld, atol=1e-14, rtol=0)


def test_append_row_equals_decode_of_its_prefix():
    b = wl.custom_batch([70, 40], q_lens=[21, 3], num_q_heads=4, num_kv_heads=1, seed=10)
    o, lse, kp, vp = oracle.append_ref(b.q, b.k_new, b.v_new, b.k_pages, b.v_pages,
                                       b.block_table, b.seq_lens, b.q_lens, b.scale)
    row = 0
    for s in range(2):
        P = int(b.seq_lens[s] - b.q_lens[s])
        for i in range(int(b.q_lens[s])):
            od, ld = oracle.decode_ref(b.q[row + i][None], kp, vp, b.block_table[s][None],
                                       np.array([P + i + 1]), b.scale)
            np.testing.assert_allclose(o[row + i], od[0], atol=1e-15, rtol=0)
            np.testing.assert_allclose(lse[row + i], ld[0], atol=1e-15, rtol=0)
        row += int(b.q_lens[s])


def test_chunked_append_equals_two_successive_appends():
    b = wl.custom_batch([90], q_lens=[30], num_q_heads=4, num_kv_heads=2, seed=12)
    o, lse, kp, vp = oracle.append_ref(b.q, b.k_new, b.v_new, b.k_pages, b.v_pages,
                                       b.block_table, b.seq_lens, b.q_lens, b.scale)
    c1 = 11
    o1, l1, kp1, vp1 = oracle.append_ref(b.q[:c1], b.k_new[:c1], b.v_new[:c1], b.k_pages,
                                         b.v_pages, b.block_table, np.array([60 + c1]),
                                         np.array([c1]), b.scale)
    o2, l2, kp2, vp2 = oracle.append_ref(b.q[c1:], b.k_new[c1:], b.v_new[c1:], kp1, vp1,
                                         b.block_table, np.array([90]), np.array([30 - c1]),
                                         b.scale)
    np.testing.assert_allclose(np.concatenate([o1, o2]), o, atol=1e-15, rtol=0)
    np.testing.assert_allclose(np.concatenate([l1, l2]), lse, atol=1e-15, rtol=0)
    assert np.array_equal(kp2, kp) and np.array_equal(vp2, vp)


def test_generator_is_deterministic_and_poisoned():
    a = wl.make_batch("tiny")
    b = wl.make_batch("tiny")
    assert np.array_equal(a.k_pages, b.k_pages) and np.array_equal(a.block_table, b.block_table)
    # unused slots of the last page and spare pages hold NaN, used slots never do
    for s in range(a.workload.batch):
        L = int(a.seq_lens[s])
        toks = gather_tokens(a.k_pages, a.block_table[s], 0, L)
        assert not np.isnan(_torch_bf16(toks)).any()
        if L % 16:
            last = a.k_pages[a.block_table[s, (L - 1) // 16], 0, L % 16:]
            assert np.isnan(_torch_bf16(last)).all()
    lens = wl.draw_lengths(wl.WORKLOADS["longtail"], np.random.default_rng(26063))[0]
    assert (lens > 4096).sum() == 26 and lens.max() <= 65536 and lens.min() >= 512


def test_bf16_rounding_is_round_to_nearest_even():
    x = np.array([1.0, 1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, -2.5, 3.14159], np.float32)
    got = wl.bf16_bits_to_f32(wl.f32_to_bf16_bits(x))
    ref = torch.from_numpy(x).to(torch.bfloat16).to(torch.float32).numpy()
    assert np.array_equal(got, ref)
