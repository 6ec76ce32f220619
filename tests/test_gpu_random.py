"""Randomised parity sweep: many small batches with random head shapes, lengths, chunk
sizes and plan parameters, each compared in full with the fp64 oracle (decode and append),
the append cache write compared bit for bit.  Sizes are kept small so that the oracle
finishes in seconds; together the cases cross page, split, tile and step boundaries many
times over."""
import numpy as np
import pytest

import oracle
from paper_2606_03077_amd import workloads as wl

import gpu_harness as H

pytestmark = pytest.mark.gpu

GROUPS = [1, 2, 3, 4, 5, 7, 8, 16]


def _case(seed):
    rng = np.random.default_rng(1000 + seed)
    hkv = int(rng.choice([1, 2, 4, 8]))
    g = int(rng.choice([x for x in GROUPS if x * hkv <= 64]))
    B = int(rng.integers(1, 10))
    lens = rng.choice([1, 2, 15, 16, 17, 63, 64, 65, 200, 1000, 2500], size=B)
    lens = np.maximum(1, lens + rng.integers(-3, 4, size=B)).tolist()
    append = bool(seed % 2)
    q_lens = None
    if append:
        q_lens = [int(min(L, rng.choice([1, 1, 2, 16, 17, 50, 130]))) for L in lens]

    params = dict(num_cus=int(rng.choice([4, 16, 64, 256])),
                  units_per_cu=int(rng.integers(1, 5)),
                  min_split_pages=int(rng.choice([1, 2, 4, 16])),
                  max_splits=int(rng.choice([1, 2, 8, 64])),
                  q_tile=int(rng.choice([0, 1, 16, 256 // g])))
    # drawn last so the earlier draws (and cases) stay as they were
    weights = [int(x) for x in rng.choice([0, 1, 500, 910, 1000, 1000000], size=8)]
    params["xcd_weight"] = weights if seed % 3 else [0] * 8
    return g * hkv, hkv, lens, q_lens, params


@pytest.mark.parametrize("seed", range(24))
def test_random_batch(seed):
    hq, hkv, lens, q_lens, params = _case(seed)
    H.say(f"[case] random seed={seed} hq={hq} hkv={hkv} lens={lens} q_lens={q_lens} {params}")
    b = wl.custom_batch(lens, q_lens=q_lens, num_q_heads=hq, num_kv_heads=hkv, seed=seed,
                        append=q_lens is not None)
    if q_lens is None:
        params.pop("q_tile")
    o, lse, cache, _ = H.run(b, plan_params=params)
    if q_lens is None:
        ro, rl = oracle.decode_ref(b.q, b.k_pages, b.v_pages, b.block_table, b.seq_lens, b.scale)
    else:
        ro, rl, k_after, v_after = oracle.append_ref(b.q, b.k_new, b.v_new, b.k_pages,
                                                     b.v_pages, b.block_table, b.seq_lens,
                                                     b.q_lens, b.scale)
        k2, v2 = cache.unpack()
        assert np.array_equal(k2, k_after) and np.array_equal(v2, v_after)
    cache.close()
    H.assert_parity(o, lse, ro, rl, label=f"random {seed}")
