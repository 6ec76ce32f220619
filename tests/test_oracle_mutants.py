"""Planted mistakes in the oracle must fail its pins (mutation check, CPU only).

Each mutant patches one piece of ``oracle.attention`` with a plausible slip (a wrong
scale, a dropped term, a wrong index, a swapped operand, an off-by-one causal bound) and
runs pins from ``test_oracle_pins``; every mutant has to be caught by at least one.
"""
import numpy as np
import pytest

import oracle.attention as oa
import test_oracle_pins as pins

_attend = oa.attend
_gather = oa.gather_tokens


def _scale_squared(q, K, V, s, visible=None):
    return _attend(q, K, V, s * s, visible)


def _lse_without_max(q, K, V, s, visible=None):
    o, lse = _attend(q, K, V, s, visible)
    if K.shape[0] == 0:
        return o, lse
    z = s * (np.asarray(q) @ np.asarray(K).T)
    if visible is not None:
        z = np.where(visible, z, -np.inf)
    return o, lse - z.max(axis=1)


def _values_are_keys(q, K, V, s, visible=None):
    return _attend(q, K, K, s, visible)


def _exclusive_causal(q, K, V, s, visible=None):
    if visible is not None:
        visible = np.roll(visible, 1, axis=1)
        visible[:, 0] = False
    return _attend(q, K, V, s, visible)


def _wrong_kv_head(pages, row, kv_head, n):
    return _gather(pages, row, (kv_head + 1) % pages.shape[1], n)


def _slot_page_swapped(pages, row, kv_head, n):
    out = np.empty((n, pages.shape[-1]), dtype=np.uint16)
    for t in range(n):
        out[t] = pages[int(row[t % 16 if t % 16 < len(row) else 0]), kv_head, (t // 16) % 16]
    return out


def _drops_last_token(pages, row, kv_head, n):
    if n <= 1:
        return _gather(pages, row, kv_head, n)
    g = _gather(pages, row, kv_head, n)
    g[-1] = g[-2]
    return g


ATTEND_MUTANTS = [_scale_squared, _lse_without_max, _values_are_keys]
GATHER_MUTANTS = [_wrong_kv_head, _slot_page_swapped, _drops_last_token]


def _caught(fn, *args):
    try:
        fn(*args)
    except AssertionError:
        return True
    return False


@pytest.mark.parametrize("mutant", ATTEND_MUTANTS, ids=lambda f: f.__name__)
def test_attend_mutants_are_caught(monkeypatch, mutant):
    monkeypatch.setattr(oa, "attend", mutant)
    assert _caught(pins.test_decode_matches_torch_sdpa, 8, 2)


@pytest.mark.parametrize("mutant", GATHER_MUTANTS, ids=lambda f: f.__name__)
def test_gather_mutants_are_caught(monkeypatch, mutant):
    monkeypatch.setattr(oa, "gather_tokens", mutant)
    assert _caught(pins.test_decode_matches_torch_sdpa, 8, 2)


def test_causal_off_by_one_is_caught(monkeypatch):
    monkeypatch.setattr(oa, "attend", _exclusive_causal)
    assert _caught(pins.test_append_matches_torch_sdpa_lower_right_causal, 7, 9)


def _bf16_shift_by_15(bits):
    b = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(15)
    return b.view(np.float32).astype(np.float64)


def _bf16_sign_dropped(bits):
    b = (np.asarray(bits, dtype=np.uint16) & np.uint16(0x7FFF)).astype(np.uint32) << np.uint32(16)
    return b.view(np.float32).astype(np.float64)


def _bf16_fraction_truncated(bits):
    b = (np.asarray(bits, dtype=np.uint16) & np.uint16(0xFFFE)).astype(np.uint32) << np.uint32(16)
    return b.view(np.float32).astype(np.float64)


@pytest.mark.parametrize("mutant", [_bf16_shift_by_15, _bf16_sign_dropped,
                                    _bf16_fraction_truncated], ids=lambda f: f.__name__)
def test_bf16_decoder_mutants_are_caught(monkeypatch, mutant):
    """A wrong bf16 decoder fails the exhaustive decoder pin, and, since the SDPA
    references decode their inputs with torch's own bfloat16, the attention pin too."""
    monkeypatch.setattr(oa, "bf16_bits_to_f64", mutant)
    assert _caught(pins.test_bf16_decoder_matches_torch_on_every_bit_pattern)
    assert _caught(pins.test_decode_matches_torch_sdpa, 8, 2)


def test_merge_sign_slip_is_caught(monkeypatch):
    real = oa.merge_ref

    def wrong(o_parts, lse_parts):
        return real(o_parts, -np.asarray(lse_parts))

    import oracle
    monkeypatch.setattr(oracle, "merge_ref", wrong)
    assert _caught(pins.test_split_anywhere_then_merge_equals_unsplit, [7, 8, 300])


# --- head reshard (Sec. 5, Step 2) --------------------------------------------------

def _interleaved_heads(shards, n_dst):
    full = np.concatenate([np.asarray(s) for s in shards], axis=1)
    return [full[:, j::n_dst].copy() for j in range(n_dst)]


def _reversed_targets(shards, n_dst):
    import oracle.migration as om
    return om.reshard_heads(shards, n_dst)[::-1]


def _sources_joined_backwards(shards, n_dst):
    import oracle.migration as om
    return om.reshard_heads(list(shards)[::-1], n_dst)


@pytest.mark.parametrize("mutant", [_interleaved_heads, _reversed_targets,
                                    _sources_joined_backwards], ids=lambda f: f.__name__)
def test_reshard_mutants_are_caught(monkeypatch, mutant):
    import test_migration_oracle as mig
    monkeypatch.setattr(mig, "reshard_heads", mutant)
    caught = [_caught(mig.test_split_by_brute_force), _caught(mig.test_join_by_brute_force),
              _caught(mig.test_shard_decode_reproduces_full_heads, 32, 8, 4)]
    assert any(caught), caught


# --- cost evaluator, RolloutDP, prefix tree, routing --------------------------------

def test_unweighted_fit_is_caught(monkeypatch):
    import test_cost_model_oracle as cm

    def absolute_fit(lengths, times):
        L = np.asarray(lengths, dtype=np.float64)
        A = np.stack([L * L, L, np.ones_like(L)], axis=1)
        coef, *_ = np.linalg.lstsq(A, np.asarray(times, dtype=np.float64), rcond=None)
        return tuple(float(c) for c in coef)

    monkeypatch.setattr(cm, "ce_fit_ref", absolute_fit)
    assert _caught(cm.test_fit_normal_equations_hold)


def _cost_sum_not_max(model, tp, seg_lengths):
    if len(seg_lengths) == 0:
        return 0.0
    import oracle.cost_model as ocm
    s = ocm.TP_SLOTS[tp]
    attn = sum(ocm.trajectory_attention(tuple(model["attn_step"]), int(x)) for x in seg_lengths)
    return model["linear_step"][s] * sum(seg_lengths) + model["attn_scale"][s] * attn


def _cost_attention_unscaled(model, tp, seg_lengths):
    if len(seg_lengths) == 0:
        return 0.0
    import oracle.cost_model as ocm
    s = ocm.TP_SLOTS[tp]
    attn = sum(ocm.trajectory_attention(tuple(model["attn_step"]), int(x)) for x in seg_lengths)
    return model["linear_step"][s] * max(seg_lengths) + attn


def _cost_attention_of_longest_only(model, tp, seg_lengths):
    if len(seg_lengths) == 0:
        return 0.0
    import oracle.cost_model as ocm
    s = ocm.TP_SLOTS[tp]
    attn = ocm.trajectory_attention(tuple(model["attn_step"]), int(max(seg_lengths)))
    return model["linear_step"][s] * max(seg_lengths) + model["attn_scale"][s] * attn


@pytest.mark.parametrize("mutant", [_cost_sum_not_max, _cost_attention_unscaled,
                                    _cost_attention_of_longest_only], ids=lambda f: f.__name__)
def test_instance_cost_mutants_are_caught(monkeypatch, mutant):
    """Plausible misreadings of Cost(tp, a, b) fail the hand-computed pins (the brute
    force and the DP both call instance_cost, so they cannot catch these)."""
    import oracle.cost_model as ocm
    import test_cost_model_oracle as cm
    monkeypatch.setattr(ocm, "instance_cost", mutant)
    assert _caught(cm.test_instance_cost_by_hand)
    assert _caught(cm.test_rollout_dp_by_hand)


def test_dp_segment_off_by_one_is_caught(monkeypatch):
    import oracle.cost_model as ocm
    import test_cost_model_oracle as cm
    real = ocm.instance_cost

    def dp_with_wrong_segment(lengths, n_gpus, tp_set, model):
        order = ocm.sorted_order(lengths)
        ls = [int(lengths[j]) for j in order]
        n = len(ls)
        dp = [[np.inf] * (n + 1) for _ in range(n_gpus + 1)]
        dp[0][0] = 0.0
        for g in range(1, n_gpus + 1):
            for i in range(n + 1):
                for tp in tp_set:
                    if tp > g:
                        continue
                    for x in range(i + 1):
                        seg = ls[max(0, i - x - 1):i] if x else []   # one request too many
                        dp[g][i] = min(dp[g][i], max(dp[g - tp][i - x], real(model, tp, seg)))
        return dp[n_gpus][n], order, []

    monkeypatch.setattr(cm, "rollout_dp_ref", dp_with_wrong_segment)
    assert any(_caught(cm.test_rollout_dp_equals_brute_force, s) for s in range(6))


def test_trie_back_off_to_root_is_caught(monkeypatch):
    import oracle.scheduler as osch
    import test_scheduler_oracle as so
    real = osch.PrefixTreeRef.lookup

    def lookup_root_on_miss(self, prompt_id, states):
        h, d = real(self, prompt_id, states)
        if d < len(states) and d >= 0:
            return real(self, -12345, [])
        return h, d

    monkeypatch.setattr(osch.PrefixTreeRef, "lookup", lookup_root_on_miss)
    assert _caught(so.test_back_off_to_parent)


def test_route_without_migration_cost_is_caught(monkeypatch):
    import test_scheduler_oracle as so

    def route_free_moves(hist, t_dec, c_mig, current):
        costs = [sum(h * t for h, t in zip(hist, row)) for row in t_dec]
        b = min(range(len(costs)), key=lambda i: (costs[i], i))
        return b, costs[b]

    monkeypatch.setattr(so, "route_ref", route_free_moves)
    assert _caught(so.test_route_by_hand)
