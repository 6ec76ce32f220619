"""Online softmax over scores whose maximum keeps moving.

With N(0,1) inputs the running maximum of a row settles within its first keys, so the
kernels' rescale paths (the chunk kernel moves its maximum lazily, only when a page
pair's probabilities would exceed 2^8; decode rescales every page) are hardly exercised
by the other parity tests.  Here the keys of every sequence are scaled along the
sequence, so scores grow (or shrink) by about 2^15 in log2 units from the first key to
the last, and a few keys are scaled by 8 (spikes, late in the row), so the maximum jumps
several times per row.  Outputs and LSEs must match the fp64 oracle to the usual
tolerances; the oracle takes the same scaled inputs.
"""
import numpy as np
import pytest

import oracle
from paper_2606_03077_amd import workloads as wl

import gpu_harness as H

pytestmark = pytest.mark.gpu


def _scale_keys(batch, rising: bool):
    """Multiplies the K vector of token t of sequence b by f_b(t) in place (cached pages
    and new tokens alike): a ramp over the row, x8 at two spike positions."""
    k_pages = wl.bf16_bits_to_f32(batch.k_pages)
    k_new = wl.bf16_bits_to_f32(batch.k_new) if batch.k_new is not None else None
    for b, L in enumerate(batch.seq_lens.tolist()):
        t = np.arange(L, dtype=np.float64)
        f = 1.0 + 3.0 * t / max(L - 1, 1) if rising else 4.0 - 3.0 * t / max(L - 1, 1)
        for spike in (L // 3, L - 3):
            if 0 <= spike < L:
                f[spike] *= 8.0
        prior = L - int(batch.q_lens[b]) if batch.k_new is not None else L
        for tok in range(L):
            if tok < prior:
                page = batch.block_table[b, tok // 16]
                k_pages[page, :, tok % 16, :] *= f[tok]
            else:
                row = int(batch.cu_q_lens[b]) + tok - prior
                k_new[row] *= f[tok]
    batch.k_pages = wl.f32_to_bf16_bits(k_pages)
    if k_new is not None:
        batch.k_new = wl.f32_to_bf16_bits(k_new)


@pytest.mark.parametrize("rising", [True, False])
def test_append_with_moving_maximum(rising):
    prior = [0, 3000, 700, 40, 1200]
    chunk = [700, 300, 1, 64, 1]
    lens = [p + c for p, c in zip(prior, chunk)]
    H.say(f"[case] append, keys scaled {'up' if rising else 'down'} along the row")
    b = wl.custom_batch(lens, q_lens=chunk, num_q_heads=16, num_kv_heads=4, seed=77)
    _scale_keys(b, rising)
    o, lse, cache, _ = H.run(b, plan_params=dict(num_cus=8, units_per_cu=1, min_split_pages=2))
    ro, rl, _, _ = oracle.append_ref(b.q, b.k_new, b.v_new, b.k_pages, b.v_pages,
                                     b.block_table, b.seq_lens, b.q_lens, b.scale)
    spread = float(rl.max() - rl.min())
    H.say(f"  oracle LSE spread over rows {spread:.1f}")
    H.assert_parity(o, lse, ro, rl, label=f"append moving max rising={rising}")
    cache.close()


@pytest.mark.parametrize("rising", [True, False])
def test_decode_with_moving_maximum(rising):
    lens = [5000, 17, 900, 3001]
    H.say(f"[case] decode, keys scaled {'up' if rising else 'down'} along the row")
    b = wl.custom_batch(lens, num_q_heads=16, num_kv_heads=4, seed=78)
    _scale_keys(b, rising)
    o, lse, cache, _ = H.run(b, plan_params=dict(num_cus=8, units_per_cu=1, min_split_pages=2))
    ro, rl = oracle.decode_ref(b.q, b.k_pages, b.v_pages, b.block_table, b.seq_lens, b.scale)
    H.assert_parity(o, lse, ro, rl, label=f"decode moving max rising={rising}")
    cache.close()
