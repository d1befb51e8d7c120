"""Pins of the CPU oracle to facts fixed by the paper and by mathematics (no GPU).

Each test checks the oracle against something other than itself: a closed form,
an invariant the paper states, a textbook/library routine, or brute force.
"""
import itertools
import math
import os

import numpy as np
import pytest
import scipy.special
import torch

from oracle import taskpress_oracle as o

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
rng = np.random.default_rng(20260803)


def _bf16_round(x):
    return torch.tensor(x, dtype=torch.float32).to(torch.bfloat16).to(torch.float64).numpy()


# ----------------------------------------------------------------------------- formats
def _bf16_from_definition(b):
    """Value of one bf16 bit pattern from the format's definition: 1 sign bit, 8 exponent
    bits with bias 127, 7 fraction bits; exponent 0 is subnormal (f/128 * 2^-126), 255 is
    infinity (f = 0) or NaN."""
    s, e, f = b >> 15, (b >> 7) & 0xFF, b & 0x7F
    sign = -1.0 if s else 1.0
    if e == 0xFF:
        return sign * math.inf if f == 0 else math.nan
    if e == 0:
        return sign * math.ldexp(f, -126 - 7)
    return sign * math.ldexp(128 + f, e - 127 - 7)


def test_bf16_decode_every_pattern():
    """The oracle's bf16 decoder gives, for all 65536 bit patterns (both zeros, subnormals,
    normals, infinities, NaNs), the value the format defines and the value torch's bfloat16
    conversion gives."""
    bits = np.arange(0, 1 << 16, dtype=np.uint32).astype(np.uint16)
    got = o.bf16_to_f64(bits)
    ref = np.array([_bf16_from_definition(int(b)) for b in bits.astype(np.int64)])
    tref = torch.from_numpy(bits.view(np.int16).copy()).view(torch.bfloat16).to(torch.float64).numpy()
    for r in (ref, tref):
        nan = np.isnan(r)
        assert np.array_equal(np.isnan(got), nan)
        assert np.array_equal(got[~nan], r[~nan])
        assert np.array_equal(np.signbit(got[~nan]), np.signbit(r[~nan]))  # -0 stays -0


# ----------------------------------------------------------------------------- stage 1
def test_softmax_rows_sum_to_one():
    """Sec. 6: the attention is softmax-normalised, so each guide row sums to 1 over the
    context and sum_i raw_i = G (for any number of query heads in the group)."""
    for R, G, N, d in [(1, 1, 7, 4), (4, 16, 300, 64), (2, 5, 1, 8)]:
        q = rng.standard_normal((R, G, d)) * 3
        k = rng.standard_normal((N, d)) * 3
        A = o.attention_slice(q[0], k, 0.3)
        assert np.allclose(A.sum(axis=1), 1.0, atol=1e-12)
        raw = o.guide_attention_sum(q, k, 0.3)
        assert abs(raw.sum() - G) < 1e-10 * G
        # pooling with K=1 is the identity
        assert np.array_equal(o.key_scores(q, k, 0.3, 1), raw)


@pytest.mark.parametrize("pool_k", [1, 3, 5, 9])
def test_uniform_closed_form(pool_k):
    """Q = 0 (or all keys equal) gives A = 1/N, so s_key_i = (G/N) c_i / K with c_i the number
    of window positions inside [0, N) (Eq. 1, zero padding)."""
    R, G, N, d = 3, 7, 23, 16
    h = pool_k // 2
    c = np.array([sum(1 for t in range(-h, h + 1) if 0 <= i + t < N) for i in range(N)], dtype=float)
    expect = (G / N) * c / pool_k
    s0 = o.key_scores(np.zeros((R, G, d)), rng.standard_normal((N, d)), 0.125, pool_k)
    np.testing.assert_allclose(s0, expect, rtol=1e-13, atol=0)
    k_eq = np.tile(rng.standard_normal((1, d)), (N, 1))
    s1 = o.key_scores(rng.standard_normal((R, G, d)), k_eq, 0.125, pool_k)
    np.testing.assert_allclose(s1, expect, rtol=1e-12, atol=0)


def test_textbook_softmax_reduction():
    """G = 1, R = 1, K = 1: s_key is exactly softmax(scale * K q) (scipy)."""
    for N, d, scale in [(1, 4, 1.0), (50, 64, 0.125), (1000, 128, 1 / math.sqrt(128))]:
        q = rng.standard_normal(d) * 2
        k = rng.standard_normal((N, d)) * 2
        s = o.key_scores(q[None, None, :], k, scale, 1)
        ref = scipy.special.softmax(scale * (k @ q))
        np.testing.assert_allclose(s, ref, rtol=1e-12, atol=1e-300)


def test_sum_not_mean_over_guide_tokens():
    """Eq. 1 sums over the guide tokens j: the score of a G-token guide is the sum of the
    G single-token scores (softmax per row, then sum)."""
    G, N, d = 6, 40, 8
    q = rng.standard_normal((1, G, d))
    k = rng.standard_normal((N, d))
    whole = o.guide_attention_sum(q, k, 0.5)
    parts = sum(scipy.special.softmax(0.5 * (k @ q[0, j])) for j in range(G))
    np.testing.assert_allclose(whole, parts, rtol=1e-12)


def test_gqa_group_mean():
    """The R query heads sharing a KV head are averaged: identical heads reproduce the
    single-head score; two different heads give the average of their scores."""
    G, N, d = 4, 33, 16
    q1 = rng.standard_normal((1, G, d))
    q2 = rng.standard_normal((1, G, d))
    k = rng.standard_normal((N, d))
    s1 = o.key_scores(q1, k, 0.25, 3)
    s2 = o.key_scores(q2, k, 0.25, 3)
    np.testing.assert_allclose(o.key_scores(np.concatenate([q1] * 4), k, 0.25, 3), s1, rtol=1e-13)
    np.testing.assert_allclose(o.key_scores(np.concatenate([q1, q2]), k, 0.25, 3), (s1 + s2) / 2, rtol=1e-13)


def test_permutation_equivariance():
    """With K = 1, permuting the context rows permutes the key scores."""
    R, G, N, d = 2, 5, 64, 16
    q = rng.standard_normal((R, G, d))
    k = rng.standard_normal((N, d))
    p = rng.permutation(N)
    np.testing.assert_allclose(o.key_scores(q, k[p], 0.2, 1), o.key_scores(q, k, 0.2, 1)[p], rtol=1e-12)


@pytest.mark.parametrize("n,pool_k", [(1, 1), (1, 5), (4, 7), (10, 3), (100, 5), (37, 11)])
def test_avg_pool_vs_convolution(n, pool_k):
    """Eq. 1's window with zero padding equals numpy's centred full convolution with a box
    of width K, divided by K (K odd); K >= N included."""
    raw = rng.random(n)
    h = pool_k // 2
    ref = np.convolve(raw, np.ones(pool_k), mode="full")[h:h + n] / pool_k
    np.testing.assert_allclose(o.avg_pool(raw, pool_k), ref, rtol=1e-14, atol=1e-16)


def test_even_pool_rejected():
    with pytest.raises(ValueError):
        o.avg_pool(np.ones(4), 4)


def test_attention_dilution():
    """App. B (dilution): planting more keys aligned with the guide spreads the softmax mass,
    so each planted token's key score falls as their number grows."""
    N, d = 512, 64
    q = rng.standard_normal((1, 8, d))
    base = rng.standard_normal((N, d)) * 0.5
    target = q[0].mean(axis=0)
    prev = None
    for m in [1, 4, 16, 64]:
        k = base.copy()
        k[:m] = target * 4.0
        s = o.key_scores(q, k, 1 / 8, 1)
        cur = s[0]
        if prev is not None:
            assert cur < prev
        prev = cur


# ----------------------------------------------------------------------------- stage 1, guide keys
def _full_causal_map(q_ctx, k_ctx, q_guide, k_guide, scale):
    """Brute force from Sec. 3.2's description: append the guide after the context, build
    the full causal attention map of size (N+G) x (N+G), softmax every row over the keys it
    may see, and return the guide rows' context columns (the slice A)."""
    qa = np.concatenate([q_ctx, q_guide])
    ka = np.concatenate([k_ctx, k_guide])
    n_all = qa.shape[0]
    out = np.zeros((n_all, n_all))
    for p in range(n_all):
        logits = [scale * float(np.dot(qa[p], ka[t])) for t in range(p + 1)]  # causal: keys 0..p
        m = max(logits)
        w = [math.exp(v - m) for v in logits]
        z = math.fsum(w)
        for t in range(p + 1):
            out[p, t] = w[t] / z
    n = q_ctx.shape[0]
    return out[n:, :n]


def _full_causal_outputs(q_ctx, k_ctx, v_ctx, q_guide, k_guide, v_guide, scale):
    """Brute force: the guide rows' outputs of the full causal attention over the context
    with the guide appended (softmax of each row over keys 0..p, times the values)."""
    qa = np.concatenate([q_ctx, q_guide])
    ka = np.concatenate([k_ctx, k_guide])
    va = np.concatenate([v_ctx, v_guide])
    n = q_ctx.shape[0]
    out = []
    for p in range(n, qa.shape[0]):
        logits = [scale * float(np.dot(qa[p], ka[t])) for t in range(p + 1)]
        m = max(logits)
        w = [math.exp(v - m) for v in logits]
        z = math.fsum(w)
        out.append([math.fsum(w[t] * va[t, c] for t in range(p + 1)) / z for c in range(va.shape[1])])
    return np.array(out)


def test_guide_attention_output_matches_the_full_causal_attention():
    """The prefill's attention output for the appended guide rows (Sec. 3.2): equal to the
    guide rows of the full causal attention over context + guide, built by brute force."""
    for N, G, d, scale in [(5, 3, 4, 0.7), (12, 6, 8, 0.35), (1, 4, 2, 1.1)]:
        q_ctx = rng.standard_normal((N, d))
        k_ctx, v_ctx = rng.standard_normal((N, d)) * 2, rng.standard_normal((N, d))
        q_g, k_g, v_g = rng.standard_normal((G, d)) * 2, rng.standard_normal((G, d)) * 2, rng.standard_normal((G, d))
        want = _full_causal_outputs(q_ctx, k_ctx, v_ctx, q_g, k_g, v_g, scale)
        got = o.guide_attention_output(q_g, k_ctx, v_ctx, scale, k_g, v_g)
        np.testing.assert_allclose(got, want, rtol=1e-12, atol=1e-13)


def test_guide_attention_output_closed_forms():
    """One row without guide keys is softmax(s K q) V (scipy); constant values come out
    unchanged (the weights sum to 1); Q = 0 averages the values each row sees."""
    N, G, d = 40, 5, 8
    k, v = rng.standard_normal((N, d)), rng.standard_normal((N, d))
    q = rng.standard_normal((1, d))
    np.testing.assert_allclose(o.guide_attention_output(q, k, v, 0.4)[0],
                               scipy.special.softmax(0.4 * (k @ q[0])) @ v, rtol=1e-12)
    c = rng.standard_normal(d)
    kg = rng.standard_normal((G, d))
    q5 = rng.standard_normal((G, d)) * 3
    out = o.guide_attention_output(q5, k, np.tile(c, (N, 1)), 0.5, kg, np.tile(c, (G, 1)))
    np.testing.assert_allclose(out, np.tile(c, (G, 1)), rtol=1e-12, atol=1e-12)
    vg = rng.standard_normal((G, d))
    out0 = o.guide_attention_output(np.zeros((G, d)), k, v, 0.5, kg, vg)
    for j in range(G):
        np.testing.assert_allclose(out0[j], (v.sum(axis=0) + vg[:j + 1].sum(axis=0)) / (N + j + 1), rtol=1e-12)


def test_guide_keys_match_the_full_causal_map():
    """With the guide's keys, A is the context slice of the causal attention map of the
    context with the guide appended (Sec. 3.2), checked by building that map."""
    for N, G, d, scale in [(5, 3, 4, 0.7), (12, 6, 8, 0.35), (1, 4, 2, 1.1)]:
        q_ctx = rng.standard_normal((N, d))
        k_ctx = rng.standard_normal((N, d)) * 2
        q_g = rng.standard_normal((G, d)) * 2
        k_g = rng.standard_normal((G, d)) * 2
        want = _full_causal_map(q_ctx, k_ctx, q_g, k_g, scale)
        got = o.attention_slice(q_g, k_ctx, scale, k_g)
        assert np.allclose(got, want, rtol=1e-12, atol=1e-15)


def test_guide_keys_closed_form_and_mass():
    """All logits equal (Q = 0): row j spreads its weight evenly over the N context keys and
    the j+1 guide keys it sees, so A[j, i] = 1/(N + j + 1); the context mass of every row is
    below 1 and the rest is the weight on the guide keys."""
    N, G, d = 40, 7, 16
    q = np.zeros((2, G, d))
    k = rng.standard_normal((N, d))
    kg = rng.standard_normal((G, d))
    A = o.attention_slice(q[0], k, 0.5, kg)
    for j in range(G):
        assert np.allclose(A[j], 1.0 / (N + j + 1), rtol=1e-13)
    raw = o.guide_attention_sum(q, k, 0.5, kg)
    assert np.allclose(raw, sum(1.0 / (N + j + 1) for j in range(G)), rtol=1e-13)
    q = rng.standard_normal((1, G, d)) * 2
    A = o.attention_slice(q[0], k, 0.5, kg)
    mass = A.sum(axis=1)
    assert np.all(mass < 1.0) and np.all(mass > 0.0)


def test_log_normalisers_closed_form():
    """All logits equal (Q = 0): row j's normaliser is the count of keys it sees, so its log is
    ln N over the context, ln(N + j + 1) with the guide keys 0..j."""
    N, G, d = 37, 6, 8
    q = np.zeros((G, d))
    k = rng.standard_normal((N, d))
    kg = rng.standard_normal((G, d))
    np.testing.assert_allclose(o.guide_log_normalisers(q, k, 0.3), np.full(G, math.log(N)), rtol=1e-14)
    np.testing.assert_allclose(o.guide_log_normalisers(q, k, 0.3, kg), np.log(N + np.arange(G) + 1.0), rtol=1e-14)


def test_log_normalisers_vs_scipy_logsumexp():
    """Random rows: the context-only normaliser is scipy's logsumexp of the scaled logits, and
    with guide keys it is the logsumexp over the context keys plus the visible guide keys."""
    N, G, d, scale = 300, 5, 32, 0.2
    q = rng.standard_normal((G, d)) * 3
    k = rng.standard_normal((N, d)) * 3
    kg = rng.standard_normal((G, d)) * 3
    ref = scipy.special.logsumexp(scale * (q @ k.T), axis=1)
    np.testing.assert_allclose(o.guide_log_normalisers(q, k, scale), ref, rtol=1e-13)
    ref_kg = [scipy.special.logsumexp(np.concatenate([scale * (k @ q[j]), scale * (kg[:j + 1] @ q[j])]))
              for j in range(G)]
    np.testing.assert_allclose(o.guide_log_normalisers(q, k, scale, kg), ref_kg, rtol=1e-13)


def test_given_lse_with_the_true_normaliser_is_the_softmax():
    """G = R = K = 1 and lse = scipy's logsumexp: the score is scipy's softmax; with a guide
    of G rows each given its own logsumexp, the raw scores sum to G (every row sums to 1)."""
    N, d, scale = 500, 64, 0.125
    q = rng.standard_normal(d) * 2
    k = rng.standard_normal((N, d)) * 2
    lse = np.array([[scipy.special.logsumexp(scale * (k @ q))]])
    s = o.key_scores_given_lse(q[None, None, :], k, scale, 1, lse)
    np.testing.assert_allclose(s, scipy.special.softmax(scale * (k @ q)), rtol=1e-12, atol=1e-300)
    G = 7
    qg = rng.standard_normal((2, G, d))
    lse = scipy.special.logsumexp(scale * (qg @ k.T), axis=2)
    raw = o.guide_attention_sum_given_lse(qg, k, scale, lse)
    assert abs(raw.sum() - G) < 1e-10


def test_given_lse_shift_scales_each_row():
    """Raising row j's lse by delta_j divides its weights by exp(delta_j): with one guide row
    per head the raw score scales by exp(-delta); rows with different deltas mix."""
    N, G, d, scale = 64, 3, 16, 0.25
    q = rng.standard_normal((1, G, d))
    k = rng.standard_normal((N, d))
    lse = scipy.special.logsumexp(scale * (q @ k.T), axis=2)
    delta = np.array([[0.5, -1.25, 2.0]])
    got = o.guide_attention_sum_given_lse(q, k, scale, lse + delta)
    want = sum(scipy.special.softmax(scale * (k @ q[0, j])) * math.exp(-delta[0, j]) for j in range(G))
    np.testing.assert_allclose(got, want, rtol=1e-12)


def test_guide_keys_reduce_to_context_softmax():
    """Guide keys whose logits lie 1000 below the context's leave A equal to the context-only
    softmax: their weight underflows to exactly 0 in float64."""
    N, G, d = 30, 5, 8
    q = rng.standard_normal((G, d))
    q[:, 0] = np.abs(q[:, 0]) + 1.0          # every guide query has a positive first component
    k = rng.standard_normal((N, d))
    kg = np.zeros((G, d))
    kg[:, 0] = -4000.0                       # so every guide logit is <= -2000
    y = 0.5 * (q @ kg.T)
    assert np.all(y <= -2000)
    assert np.array_equal(o.attention_slice(q, k, 0.5, kg), o.attention_slice(q, k, 0.5))


# ----------------------------------------------------------------------------- stage 2
ALL_POS_BF16 = np.arange(1, 0x7F80, dtype=np.uint16)  # every positive finite bf16


@pytest.mark.parametrize("qfmt,bits", [(o.QFMT_INT, 8), (o.QFMT_INT, 4), (o.QFMT_INT, 2), (o.QFMT_INT, 6),
                                       (o.QFMT_FP8_E4M3, 8)])
def test_scales_exhaustive_closed_form(qfmt, bits):
    """Eq. 2, gamma = absmax / (2^(b-1) - 1) (448 for E4M3), checked for every positive finite
    bf16 absmax against numpy's IEEE fp32 division."""
    absmax = o.bf16_to_f64(ALL_POS_BF16)
    v = np.stack([absmax, -absmax / 2], axis=1)
    g = o.value_scales(v, qfmt, bits)
    qmax = {8: 127.0, 4: 7.0, 2: 1.0, 6: 31.0}[bits] if qfmt == o.QFMT_INT else 448.0
    ref = absmax.astype(np.float32) / np.float32(qmax)
    assert np.array_equal(g.view(np.uint32), ref.view(np.uint32))


def test_quant_int_exhaustive_at_unit_absmax():
    """Every bf16 v in [-1, 1] with absmax 1: q equals RNE of the IEEE fp32 quotient, clamped;
    |v - q gamma| <= gamma/2 except where the fp32 quotient rounding decides a half."""
    bits16 = np.arange(0, 0x3F81, dtype=np.uint16)
    mags = o.bf16_to_f64(bits16)
    vals = np.concatenate([mags, -mags])
    rows = np.stack([np.full(vals.shape, 1.0), vals], axis=1)
    g = o.value_scales(rows, o.QFMT_INT, 8)
    q = o.quantize_values(rows, g, o.QFMT_INT, 8)
    y32 = rows.astype(np.float32) / g.astype(np.float32)[:, None]
    ref = np.clip(np.rint(y32.astype(np.float64)), -127, 127).astype(np.int8)
    assert np.array_equal(q, ref)
    assert np.all(q[:, 0] == 127)
    err = np.abs(rows - q.astype(np.float64) * g[:, None].astype(np.float64))
    assert np.all(err <= g[:, None].astype(np.float64) * (0.5 + 1e-6))


@pytest.mark.parametrize("bits", [8, 4])
def test_quant_int_quotient_rounded_to_fp32_first(bits):
    """q = RNE(fl32(v / gamma)): the quotient is rounded to fp32 before the integer rounding.
    For every bf16 absmax in [1, 2) and every bf16 v in [0, absmax] the codes equal numpy's
    IEEE fp32 division followed by RNE; this sweep includes the v = absmax/2 cases whose fp32
    quotient lands exactly on a half while the exact quotient does not."""
    qm = 2 ** (bits - 1) - 1
    pos = o.bf16_to_f64(np.arange(0, 0x7F80, dtype=np.uint16))
    for a_bits in range(0x3F80, 0x4000):
        a = float(o.bf16_to_f64(np.array([a_bits], dtype=np.uint16))[0])
        v = pos[pos <= a]
        rows = np.stack([np.full(v.shape, a), v], axis=1)
        g = o.value_scales(rows, o.QFMT_INT, bits)
        q = o.quantize_values(rows, g, o.QFMT_INT, bits)
        y32 = v.astype(np.float32) / g.astype(np.float32)
        ref = np.clip(np.rint(y32.astype(np.float64)), -qm, qm).astype(np.int8)
        assert np.array_equal(q[:, 1], ref), a


@pytest.mark.parametrize("qfmt,bits", [(o.QFMT_INT, 8), (o.QFMT_INT, 4), (o.QFMT_FP8_E4M3, 8)])
def test_quant_properties(qfmt, bits):
    """The absmax element maps to +-qmax; scaling a row by 2^e leaves q unchanged and scales
    gamma by 2^e; a zero row gives gamma = 0, q = 0."""
    d = 128
    v = _bf16_round(rng.standard_normal((500, d)) * 3)
    v[7] = 0.0
    g = o.value_scales(v, qfmt, bits)
    q = o.quantize_values(v, g, qfmt, bits)
    amax_pos = np.abs(v).argmax(axis=1)
    top = q[np.arange(500), amax_pos]
    if qfmt == o.QFMT_INT:
        qm = 2 ** (bits - 1) - 1
        rows = np.arange(500) != 7
        assert np.all(np.abs(top[rows].astype(int)) == qm)
    else:
        rows = np.arange(500) != 7
        assert np.all((top[rows] & 0x7F) == 0x7E)
    assert g[7] == 0 and np.all(q[7].view(np.uint8) == 0)
    for e in (-3, 5):
        g2 = o.value_scales(v * 2.0 ** e, qfmt, bits)
        q2 = o.quantize_values(v * 2.0 ** e, g2, qfmt, bits)
        assert np.array_equal(q2, q)
        assert np.array_equal(g2.astype(np.float64), g.astype(np.float64) * 2.0 ** e)


def test_e4m3_golden_codes():
    """Code table of the OCP OFP8 specification (fixture with citation)."""
    rows = [l.split() for l in open(os.path.join(GOLDEN, "e4m3_ocp_values.txt")) if not l.startswith("#")]
    for code_hex, val in rows:
        code = int(code_hex, 16)
        dec = o.e4m3_decode(np.array([code], dtype=np.uint8))[0]
        assert dec == float(val) and np.signbit(dec) == val.startswith("-")
        assert o.e4m3_encode(np.array([float(val)]))[0] == code
    assert np.isnan(o.e4m3_decode(np.array([0x7F], dtype=np.uint8))[0])


def test_e4m3_encoder_vs_torch():
    """Within [-448, 448] the encoder equals PyTorch's float32 -> float8_e4m3fn conversion
    (round to nearest even), including every midpoint between neighbouring codes."""
    vals = o.e4m3_positive_values()
    mids = (vals[:-1] + vals[1:]) / 2
    x = np.concatenate([rng.uniform(-448, 448, 100000), mids, -mids, vals, -vals, [2.0 ** -10, 2.0 ** -11]])
    x = x.astype(np.float32).astype(np.float64)
    ref = torch.tensor(x, dtype=torch.float32).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    assert np.array_equal(o.e4m3_encode(x), ref)
    assert np.all(o.e4m3_encode(np.array([449.0, 500.0, 1e30, -1e9])) == np.array([0x7E, 0x7E, 0x7E, 0xFE]))


def test_int4_packing():
    """b <= 4: two 4-bit two's-complement values per byte, even element in the low nibble."""
    q = np.array([[-1, 2, 7, -7, 0, -8 + 1]], dtype=np.int8)
    packed = o.pack_codes(q, o.QFMT_INT, 4)
    assert packed.tolist() == [[0x2F, 0x97, 0x90]]


# ----------------------------------------------------------------------------- stage 3
def test_keep_count_golden():
    rows = [l.split() for l in open(os.path.join(GOLDEN, "keep_counts.txt")) if not l.startswith("#")]
    for n, ratio, budget, k in rows:
        kk = o.keep_count(int(n), None if ratio == "-" else float(ratio), None if budget == "-" else int(budget))
        assert kk == int(k), (n, ratio, budget)


def _brute_select(S, k):
    order = sorted(range(len(S)), key=lambda i: (-float(S[i]), i))
    return sorted(order[:k])


def test_select_brute_force_all_multisets():
    """Every arrangement of small multisets with ties, every k: the highest k scores, ties to
    the lower index, ascending (pure-Python sort as the reference)."""
    for vals in [(1, 1, 2, 3, 3, 3), (0, 0, 0, 0), (5, 4, 3, 2, 1, 0, 0)]:
        for perm in set(itertools.permutations(vals)):
            S = np.array(perm, dtype=np.float32)
            for k in range(1, len(S) + 1):
                assert o.select(S, k).tolist() == _brute_select(S, k)


def test_select_random_ties():
    for _ in range(50):
        n = int(rng.integers(1, 200))
        S = rng.integers(0, 8, n).astype(np.float32) * np.float32(0.25)
        k = int(rng.integers(1, n + 1))
        assert o.select(S, k).tolist() == _brute_select(S, k)
    S = np.full(100, 3.0, dtype=np.float32)
    assert o.select(S, 17).tolist() == list(range(17))


def test_combine_mul_is_fp32_product():
    """Eq. 3 stored as fp32: equals numpy's IEEE fp32 multiply on fp32 inputs, bit for bit."""
    a = (rng.random(100000) * 10.0 ** rng.integers(-30, 5, 100000)).astype(np.float32)
    b = (rng.random(100000) * 10.0 ** rng.integers(-20, 3, 100000)).astype(np.float32)
    S = o.combine(a, b, o.COMBINE_MUL)
    assert np.array_equal(S.view(np.uint32), (a * b).view(np.uint32))


def test_combine_variants_properties():
    """Aggregation table variants: NORM_ADD of identical vectors has L2 norm 2 and is
    invariant to scaling either input; HARMONIC(a, a) = a, HARMONIC(a, 0) = 0, symmetric;
    KEY_ONLY equals MUL's ranking when gamma is constant."""
    a = rng.random(1000).astype(np.float32) + np.float32(0.01)
    b = rng.random(1000).astype(np.float32) + np.float32(0.01)
    S = o.combine(a, a, o.COMBINE_NORM_ADD).astype(np.float64)
    assert abs(np.linalg.norm(S) - 2.0) < 1e-6
    s1 = o.combine(a, b, o.COMBINE_NORM_ADD)
    s2 = o.combine(a * np.float32(8), b * np.float32(0.5), o.COMBINE_NORM_ADD)
    np.testing.assert_allclose(s1, s2, rtol=1e-6)
    h = o.combine(a, a, o.COMBINE_HARMONIC)
    np.testing.assert_allclose(h, a, rtol=1e-7)
    assert np.all(o.combine(a, np.zeros_like(a), o.COMBINE_HARMONIC) == 0)
    assert np.all(o.combine(np.zeros(3, np.float32), np.zeros(3, np.float32), o.COMBINE_HARMONIC) == 0)
    assert np.array_equal(o.combine(a, b, o.COMBINE_HARMONIC), o.combine(b, a, o.COMBINE_HARMONIC))
    g = np.full(1000, 0.37, dtype=np.float32)
    k = 100
    assert np.array_equal(o.select(o.combine(a, g, o.COMBINE_MUL), k), o.select(o.combine(a, g, o.COMBINE_KEY_ONLY), k))


# ----------------------------------------------------------------------------- stage 4
def test_compact_vs_index_select():
    rows = rng.integers(0, 2 ** 16, (300, 64)).astype(np.uint16)
    idx = np.sort(rng.choice(300, 70, replace=False)).astype(np.int32)
    ref = torch.index_select(torch.from_numpy(rows.astype(np.int32)), 0, torch.from_numpy(idx.astype(np.int64)))
    assert np.array_equal(o.compact(rows, idx), ref.numpy().astype(np.uint16))


# ----------------------------------------------------------------------------- whole segment
def test_evict_segment_consistency():
    R, G, N, d = 4, 16, 1024, 64
    bf = lambda x: torch.tensor(x, dtype=torch.float32).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    qb = bf(rng.standard_normal((R, G, d)))
    kb = bf(rng.standard_normal((N, d)))
    vb = bf(rng.standard_normal((N, d)))
    k = o.keep_count(N, 0.25)
    out = o.evict_segment(qb, kb, vb, softmax_scale=0.125, pool_k=5, qfmt=o.QFMT_INT, bits=8,
                          rule=o.COMBINE_MUL, k=k)
    idx = out["idx"]
    assert len(idx) == k and np.all(np.diff(idx) > 0)
    kept = np.zeros(N, bool)
    kept[idx] = True
    assert out["S"][kept].min() >= out["S"][~kept].max()
    assert abs(o.avg_pool(np.ones(N), 1).sum() - N) == 0
    assert np.array_equal(out["k_c"], kb[idx])
