"""The whole-batch oracle of the GPU parity tests (tests/gpu_harness.py) runs the oracle
per (sequence, KV head) on a renamed-page, head-sliced copy of the inputs, in forked host
processes.  On the CPU it must give what the oracle gives on the whole batch."""
import numpy as np
import pytest

import oracle
from paper_2606_03077_amd import workloads as wl

import gpu_harness as H


@pytest.mark.parametrize("append", [False, True])
def test_whole_batch_pool_equals_direct_oracle(append):
    lens = [0, 1, 17, 300, 1000, 45] if not append else [1, 18, 300, 1000, 45, 64]
    ql = [1] * 6 if not append else [1, 5, 1, 200, 45, 1]
    b = wl.custom_batch(lens, q_lens=ql, num_q_heads=12, num_kv_heads=4, seed=9, append=append)
    o, l, secs, workers = H.oracle_whole_batch(b, workers=3)
    if append:
        ro, rl, _, _ = oracle.append_ref(b.q, b.k_new, b.v_new, b.k_pages, b.v_pages,
                                         b.block_table, b.seq_lens, b.q_lens, b.scale)
    else:
        ro, rl = oracle.decode_ref(b.q, b.k_pages, b.v_pages, b.block_table, b.seq_lens,
                                   b.scale)
    np.testing.assert_allclose(o, ro, rtol=0, atol=1e-13)
    both = np.isneginf(l) & np.isneginf(rl)
    assert np.array_equal(np.isneginf(l), np.isneginf(rl))
    np.testing.assert_allclose(np.where(both, 0, l), np.where(both, 0, rl), rtol=0, atol=1e-13)
