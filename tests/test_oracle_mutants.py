"""The oracle's pins catch plausible mistakes (no GPU).

Each case plants one mistake in the oracle (on the CPU, by swapping one of its functions
for a wrong variant) and checks that at least one of the pins in test_oracle_pins.py then
fails.  A pin set that let a dropped term, a wrong sign, an off-by-one window, a wrong
rounding or a transposed operand through would be no pin at all.
"""
import math

import numpy as np
import pytest

import test_oracle_pins as pins
from oracle import taskpress_oracle as o

_orig = {name: getattr(o, name) for name in dir(o) if callable(getattr(o, name))}


def _softmax_rows(x):
    e = np.exp(x - x.max(axis=1, keepdims=True))
    return e / e.sum(axis=1, keepdims=True)


# ----------------------------------------------------------------------------- mutants
def m_softmax_wrong_axis(q_rows, k_rows, scale, kg_rows=None):
    x = scale * (q_rows @ k_rows.T)
    e = np.exp(x - x.max(axis=0, keepdims=True))
    return e / e.sum(axis=0, keepdims=True)


def m_scale_dropped(q_rows, k_rows, scale, kg_rows=None):
    return _orig["attention_slice"](q_rows, k_rows, 1.0, kg_rows)


def m_transposed_logits(q_rows, k_rows, scale, kg_rows=None):
    x = scale * (q_rows @ k_rows.T)
    return _softmax_rows(x[:, ::-1])  # keys in the wrong order


def m_guide_key_not_causal_self(q_rows, k_rows, scale, kg_rows=None):
    if kg_rows is None:
        return _orig["attention_slice"](q_rows, k_rows, scale)
    g = q_rows.shape[0]
    x = scale * (q_rows @ k_rows.T)
    y = scale * (q_rows @ kg_rows.T)
    y = np.where(np.arange(g)[None, :] < np.arange(g)[:, None], y, -np.inf)  # t < j: own key left out
    m = np.maximum(x.max(axis=1, keepdims=True), np.max(np.where(np.isinf(y), -1e300, y), axis=1, keepdims=True))
    e = np.exp(x - m)
    return e / (e.sum(axis=1, keepdims=True) + np.exp(y - m).sum(axis=1, keepdims=True))


def m_sum_over_heads(q_group, k_rows, scale, kg_rows=None):
    return _orig["guide_attention_sum"](q_group, k_rows, scale, kg_rows) * q_group.shape[0]


def m_mean_over_guide(q_group, k_rows, scale, kg_rows=None):
    return _orig["guide_attention_sum"](q_group, k_rows, scale, kg_rows) / q_group.shape[1]


def m_pool_divide_by_count(raw, pool_k):
    n = raw.shape[0]
    h = pool_k // 2
    out = np.zeros(n)
    for i in range(n):
        lo, hi = max(0, i - h), min(n, i + h + 1)
        out[i] = raw[lo:hi].sum() / (hi - lo)
    return out


def m_pool_window_short(raw, pool_k):
    n = raw.shape[0]
    h = pool_k // 2
    acc = np.zeros(n)
    for t in range(-h, h):  # drops the last tap
        lo, hi = max(0, -t), min(n, n - t)
        if lo < hi:
            acc[lo:hi] += raw[lo + t:hi + t]
    return acc / pool_k


def m_qmax_off_by_one(qfmt, bits):
    return 448.0 if qfmt == o.QFMT_FP8_E4M3 else float(2 ** (bits - 1))


def m_round_half_up(v_rows, gamma, qfmt=o.QFMT_INT, bits=8):
    if qfmt != o.QFMT_INT:
        return _orig["quantize_values"](v_rows, gamma, qfmt, bits)
    g = np.asarray(gamma, dtype=np.float64)[:, None]
    safe = np.where(g == 0.0, 1.0, g)
    y = o.to_f32(v_rows / safe).astype(np.float64)
    y = np.where(g == 0.0, 0.0, y)
    qm = o.qmax_of(qfmt, bits)
    return np.clip(np.floor(y + 0.5), -qm, qm).astype(np.int8)


def m_quotient_in_f64(v_rows, gamma, qfmt=o.QFMT_INT, bits=8):
    if qfmt != o.QFMT_INT:
        return _orig["quantize_values"](v_rows, gamma, qfmt, bits)
    g = np.asarray(gamma, dtype=np.float64)[:, None]
    y = np.where(g == 0.0, 0.0, v_rows / np.where(g == 0.0, 1.0, g))  # no fl32 of the quotient
    qm = o.qmax_of(qfmt, bits)
    return np.clip(np.rint(y), -qm, qm).astype(np.int8)


def m_e4m3_truncate(y):
    vals = o.e4m3_positive_values()
    a = np.minimum(np.abs(np.asarray(y, dtype=np.float64)), 448.0)
    idx = np.searchsorted(vals, a, side="right") - 1  # round toward zero
    codes = np.asarray(idx, dtype=np.uint8)
    return np.where(np.signbit(y), codes | 0x80, codes).astype(np.uint8)


def m_select_ties_high(scores, k):
    s = np.asarray(scores)
    n = s.shape[0]
    order = np.lexsort((-np.arange(n), -s.astype(np.float64)))
    return np.sort(order[:k]).astype(np.int32)


def m_select_unsorted(scores, k):
    s = np.asarray(scores)
    n = s.shape[0]
    order = np.lexsort((np.arange(n), -s.astype(np.float64)))
    return order[:k].astype(np.int32)


def m_combine_f64(s_key, gamma, rule=o.COMBINE_MUL):
    if rule == o.COMBINE_MUL:
        return np.asarray(s_key, dtype=np.float64) * np.asarray(gamma, dtype=np.float64)
    return _orig["combine"](s_key, gamma, rule)


def m_keep_count_ceil(n, keep_ratio=None, keep_budget=None):
    if keep_ratio is not None:
        return max(1, int(math.ceil(float(n) * float(keep_ratio))))
    return _orig["keep_count"](n, keep_ratio, keep_budget)


def m_pack_high_nibble_first(q, qfmt, bits):
    if qfmt == o.QFMT_INT and bits <= 4:
        u = (q.astype(np.int16) & 0xF).astype(np.uint8)
        return (u[:, 1::2] | (u[:, 0::2] << 4)).astype(np.uint8)
    return _orig["pack_codes"](q, qfmt, bits)


def m_lse_added(q_group, k_rows, scale, lse):
    R = q_group.shape[0]
    raw = np.zeros(k_rows.shape[0])
    for r in range(R):
        raw += np.exp(scale * (q_group[r] @ k_rows.T) + np.asarray(lse[r])[:, None]).sum(axis=0)  # sign flipped
    return raw / R


def m_lse_base2(q_group, k_rows, scale, lse):
    R = q_group.shape[0]
    raw = np.zeros(k_rows.shape[0])
    for r in range(R):
        raw += np.exp2(scale * (q_group[r] @ k_rows.T) - np.asarray(lse[r])[:, None]).sum(axis=0)
    return raw / R


def m_lse_first_row_only(q_group, k_rows, scale, lse):
    lse = np.asarray(lse, dtype=np.float64)
    return _orig["guide_attention_sum_given_lse"](q_group, k_rows, scale, np.repeat(lse[:, :1], lse.shape[1], axis=1))


def m_lognorm_not_causal_self(q_rows, k_rows, scale, kg_rows=None):
    if kg_rows is None:
        return _orig["guide_log_normalisers"](q_rows, k_rows, scale)
    g = q_rows.shape[0]
    x = scale * (q_rows @ k_rows.T)
    y = scale * (q_rows @ kg_rows.T)
    y = np.where(np.arange(g)[None, :] < np.arange(g)[:, None], y, -np.inf)  # own key left out
    z = np.concatenate([x, y], axis=1)
    m = z.max(axis=1)
    return m + np.log(np.exp(z - m[:, None]).sum(axis=1))


def m_lognorm_log2(q_rows, k_rows, scale, kg_rows=None):
    return _orig["guide_log_normalisers"](q_rows, k_rows, scale, kg_rows) / math.log(2.0)


def m_bf16_shift_15(bits):
    bits = np.asarray(bits, dtype=np.uint16)
    return (bits.astype(np.uint32) << 15).view(np.float32).astype(np.float64)


def m_bf16_sign_dropped(bits):
    bits = np.asarray(bits, dtype=np.uint16) & np.uint16(0x7FFF)
    return (bits.astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def m_output_not_causal_self(q_rows, k_rows, v_rows, scale, kg_rows=None, vg_rows=None):
    if kg_rows is None:
        return _orig["guide_attention_output"](q_rows, k_rows, v_rows, scale)
    g = q_rows.shape[0]
    x = scale * (q_rows @ k_rows.T)
    y = scale * (q_rows @ kg_rows.T)
    y = np.where(np.arange(g)[None, :] < np.arange(g)[:, None], y, -np.inf)  # own key left out
    m = np.maximum(x.max(axis=1, keepdims=True), np.max(np.where(np.isinf(y), -1e300, y), axis=1, keepdims=True))
    e, eg = np.exp(x - m), np.exp(y - m)
    return (e @ v_rows + eg @ vg_rows) / (e.sum(axis=1, keepdims=True) + eg.sum(axis=1, keepdims=True))


def m_output_context_normaliser(q_rows, k_rows, v_rows, scale, kg_rows=None, vg_rows=None):
    if kg_rows is None:
        return _orig["guide_attention_output"](q_rows, k_rows, v_rows, scale)
    g = q_rows.shape[0]
    x = scale * (q_rows @ k_rows.T)
    y = scale * (q_rows @ kg_rows.T)
    y = np.where(np.arange(g)[None, :] <= np.arange(g)[:, None], y, -np.inf)
    m = np.maximum(x.max(axis=1, keepdims=True), y.max(axis=1, keepdims=True))
    e, eg = np.exp(x - m), np.exp(y - m)
    return (e @ v_rows + eg @ vg_rows) / e.sum(axis=1, keepdims=True)  # guide keys left out of the normaliser


def m_output_guide_values_shifted(q_rows, k_rows, v_rows, scale, kg_rows=None, vg_rows=None):
    if kg_rows is None:
        return _orig["guide_attention_output"](q_rows, k_rows, v_rows, scale)
    return _orig["guide_attention_output"](q_rows, k_rows, v_rows, scale, kg_rows, np.roll(vg_rows, 1, axis=0))


# ----------------------------------------------------------------------------- pins to run
P = pins
CASES = [
    ("bf16_to_f64", m_bf16_shift_15, [P.test_bf16_decode_every_pattern]),
    ("bf16_to_f64", m_bf16_sign_dropped, [P.test_bf16_decode_every_pattern]),
    ("attention_slice", m_softmax_wrong_axis, [P.test_softmax_rows_sum_to_one, P.test_textbook_softmax_reduction]),
    ("attention_slice", m_scale_dropped, [P.test_textbook_softmax_reduction]),
    ("attention_slice", m_transposed_logits, [P.test_textbook_softmax_reduction, P.test_permutation_equivariance]),
    ("attention_slice", m_guide_key_not_causal_self, [P.test_guide_keys_match_the_full_causal_map,
                                                      P.test_guide_keys_closed_form_and_mass]),
    ("guide_attention_sum", m_sum_over_heads, [P.test_gqa_group_mean, P.test_softmax_rows_sum_to_one]),
    ("guide_attention_sum", m_mean_over_guide, [P.test_sum_not_mean_over_guide_tokens]),
    ("avg_pool", m_pool_divide_by_count, [lambda: P.test_avg_pool_vs_convolution(10, 3),
                                          lambda: P.test_uniform_closed_form(5)]),
    ("avg_pool", m_pool_window_short, [lambda: P.test_avg_pool_vs_convolution(37, 11)]),
    ("qmax_of", m_qmax_off_by_one, [lambda: P.test_scales_exhaustive_closed_form(o.QFMT_INT, 8)]),
    ("quantize_values", m_round_half_up, [P.test_quant_int_exhaustive_at_unit_absmax]),
    ("quantize_values", m_quotient_in_f64, [lambda: P.test_quant_int_quotient_rounded_to_fp32_first(8)]),
    ("e4m3_encode", m_e4m3_truncate, [P.test_e4m3_golden_codes, P.test_e4m3_encoder_vs_torch]),
    ("select", m_select_ties_high, [P.test_select_brute_force_all_multisets]),
    ("select", m_select_unsorted, [P.test_select_brute_force_all_multisets]),
    ("combine", m_combine_f64, [P.test_combine_mul_is_fp32_product]),
    ("keep_count", m_keep_count_ceil, [P.test_keep_count_golden]),
    ("pack_codes", m_pack_high_nibble_first, [P.test_int4_packing]),
    ("guide_attention_sum_given_lse", m_lse_added, [P.test_given_lse_with_the_true_normaliser_is_the_softmax]),
    ("guide_attention_sum_given_lse", m_lse_base2, [P.test_given_lse_with_the_true_normaliser_is_the_softmax]),
    ("guide_attention_sum_given_lse", m_lse_first_row_only, [P.test_given_lse_shift_scales_each_row]),
    ("guide_log_normalisers", m_lognorm_not_causal_self, [P.test_log_normalisers_closed_form]),
    ("guide_log_normalisers", m_lognorm_log2, [P.test_log_normalisers_closed_form,
                                                P.test_log_normalisers_vs_scipy_logsumexp]),
    ("guide_attention_output", m_output_not_causal_self,
     [P.test_guide_attention_output_matches_the_full_causal_attention, P.test_guide_attention_output_closed_forms]),
    ("guide_attention_output", m_output_context_normaliser,
     [P.test_guide_attention_output_matches_the_full_causal_attention, P.test_guide_attention_output_closed_forms]),
    ("guide_attention_output", m_output_guide_values_shifted,
     [P.test_guide_attention_output_matches_the_full_causal_attention, P.test_guide_attention_output_closed_forms]),
]


@pytest.mark.parametrize("target,mutant,checks", CASES, ids=[f"{c[0]}-{c[1].__name__}" for c in CASES])
def test_pins_catch_mutant(monkeypatch, target, mutant, checks):
    monkeypatch.setattr(o, target, mutant)
    caught = 0
    for check in checks:
        try:
            check()
        except (AssertionError, ValueError, IndexError):
            caught += 1
    assert caught >= 1, f"no pin caught the planted mistake {mutant.__name__} in {target}"


def test_unmutated_oracle_passes_the_same_checks():
    for _, _, checks in CASES:
        for check in checks:
            check()
