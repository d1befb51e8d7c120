"""CPU oracle of the task-guided prefill-time KV eviction path (TaskPress,
arXiv 2608.03276).  TEST INFRASTRUCTURE ONLY: it exists to check the GPU path.
Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import it; the product path never does.

Plain, slow, direct definitions in float64 (numpy), one (sequence, layer,
KV head) segment at a time.  Where the output format is defined as fp32,
int-b or fp8-e4m3, the value is computed in float64 and rounded once to that
format; for a single +, -, *, / of fp32 operands that equals the correctly
rounded fp32 operation (53 >= 2*24 + 2: Figueroa, "When is double rounding
innocuous?", SIGNUM Newsletter 1995).

Sections cited are those of the paper:
  Sec. 3.1  problem statement: one kept index set per KV head, |I| << L_c.
  Sec. 3.2, Eq. 1  key score: sum over guide tokens of the guide->context
            attention, then 1-D average pooling with kernel K.
  Sec. 3.3, Eq. 2  value score: per-token quantisation scale
            gamma_i = max|v_i| / (2^(b-1) - 1).
  Sec. 3.4, Eq. 3  combined score s_i = s_key_i * s_value_i; keep the
            highest-scoring indices.
  Sec. 4 (setup)   uniform budget per KV head, chosen independently per head;
            the guide's own KV is dropped after prefill; int4 KV cache.
  Sec. 4.4 (aggregation table)  normalised-add and harmonic-mean variants.
  Sec. 6 (limitations)  the attention used is softmax-normalised.

Readings where the paper is silent (each listed in the design notes):
  - by default the softmax runs over the context keys only (the guide's own keys
    are not in the normaliser); given the guide keys, it is the paper-literal
    context slice of the causal attention over context + appended guide
    (Sec. 3.2); logits scaled by `softmax_scale`;
  - the R query heads of a GQA group are averaged;
  - pooling pads with zeros outside [0, N) and always divides by K;
  - gamma stored as fp32; q = clamp(RNE(fl32(v / gamma)), +-qmax); gamma = 0
    gives q = 0; fp8 is OCP E4M3 with RNE and saturation at 448;
  - the combined score is stored as fp32 and selection ranks those fp32
    values, ties going to the lower index; kept indices ascend;
  - k = max(1, floor(N * keep_ratio)) in binary64, or min(budget, N).
"""
from __future__ import annotations

import math

import numpy as np

QFMT_INT = 0
QFMT_FP8_E4M3 = 1

COMBINE_MUL = 0
COMBINE_NORM_ADD = 1
COMBINE_HARMONIC = 2
COMBINE_KEY_ONLY = 3


# --------------------------------------------------------------------------- formats
def bf16_to_f64(bits: np.ndarray) -> np.ndarray:
    """bf16 bit patterns (uint16) -> float64, exactly (bf16 is the top half of fp32)."""
    bits = np.asarray(bits, dtype=np.uint16)
    return (bits.astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def to_f32(x) -> np.ndarray:
    """Round float64 values once to fp32 (round to nearest even)."""
    return np.asarray(x, dtype=np.float64).astype(np.float32)


def e4m3_positive_values() -> np.ndarray:
    """Values of the 127 non-negative finite OCP E4M3 codes 0x00..0x7E, by code.

    Code c = (e << 3) | m: e = 0 is subnormal, m/8 * 2^-6; otherwise
    (1 + m/8) * 2^(e-7).  0x7F is NaN; there is no infinity."""
    vals = np.empty(127, dtype=np.float64)
    for c in range(127):
        e, m = c >> 3, c & 7
        vals[c] = (m / 8.0) * 2.0 ** -6 if e == 0 else (1.0 + m / 8.0) * 2.0 ** (e - 7)
    return vals


_E4M3 = e4m3_positive_values()


def e4m3_encode(y: np.ndarray) -> np.ndarray:
    """OCP E4M3 codes of fp32/float64 values: nearest value, ties to the even code
    (even mantissa), magnitudes >= 448 saturate to 448 (0x7E), sign bit kept."""
    y = np.asarray(y, dtype=np.float64)
    a = np.abs(y)
    hi = np.clip(np.searchsorted(_E4M3, a, side="left"), 1, 126)  # first value >= a
    lo = hi - 1
    dl = a - _E4M3[lo]
    dh = _E4M3[hi] - a
    take_lo = (dl < dh) | ((dl == dh) & (lo % 2 == 0))
    codes = np.where(take_lo, lo, hi)
    codes = np.where(a >= _E4M3[126], 126, codes).astype(np.uint8)
    return codes | np.where(np.signbit(y), np.uint8(0x80), np.uint8(0))


def e4m3_decode(codes: np.ndarray) -> np.ndarray:
    codes = np.asarray(codes, dtype=np.uint8)
    mag = codes & 0x7F
    out = np.where(mag == 0x7F, np.nan, _E4M3[np.minimum(mag, 126)])
    return np.where(codes & 0x80, -out, out)


def qmax_of(qfmt: int, bits: int) -> float:
    """Largest quantised magnitude: 2^(b-1) - 1 for b-bit integers (Eq. 2), 448 for E4M3."""
    if qfmt == QFMT_INT:
        if not 2 <= bits <= 8:
            raise ValueError("bits must be in [2, 8]")
        return float(2 ** (bits - 1) - 1)
    if qfmt == QFMT_FP8_E4M3:
        return 448.0
    raise ValueError("unknown qfmt")


# --------------------------------------------------------------------------- sizes
def keep_count(n: int, keep_ratio: float | None = None, keep_budget: int | None = None) -> int:
    """|I| for a head with n context tokens (Sec. 3.1; uniform per-head budget, Sec. 4 setup).

    keep_ratio is 1 - the paper's eviction ratio: k = max(1, floor(n * keep_ratio)) in
    binary64.  A budget gives k = min(budget, n)."""
    if (keep_ratio is None) == (keep_budget is None):
        raise ValueError("exactly one of keep_ratio / keep_budget")
    if keep_ratio is not None:
        if not 0.0 < keep_ratio <= 1.0:
            raise ValueError("keep_ratio must be in (0, 1]")
        return max(1, int(math.floor(float(n) * float(keep_ratio))))
    if keep_budget < 1:
        raise ValueError("keep_budget must be >= 1")
    return min(int(keep_budget), int(n))


# --------------------------------------------------------------------------- stage 1
def attention_slice(q_rows: np.ndarray, k_rows: np.ndarray, softmax_scale: float,
                    kg_rows: np.ndarray | None = None) -> np.ndarray:
    """A[j, i]: attention weight of guide token j on context token i (Sec. 3.2).

    Softmax-normalised (Sec. 6) attention of the logits softmax_scale * <q_j, k_i>.
    q_rows [G, d], k_rows [N, d], float64.  Without kg_rows the normaliser runs over the N
    context keys only (the default reading).  With kg_rows [G, d], the guide's own keys,
    A is the context slice of the full causal attention map of Sec. 3.2 with the guide
    appended after the context: row j's normaliser also covers guide keys 0..j."""
    x = softmax_scale * (q_rows @ k_rows.T)
    if kg_rows is None:
        m = x.max(axis=1, keepdims=True)
        e = np.exp(x - m)
        return e / e.sum(axis=1, keepdims=True)
    g = q_rows.shape[0]
    y = softmax_scale * (q_rows @ kg_rows.T)                      # [G, G] guide-key logits
    causal = np.arange(g)[None, :] <= np.arange(g)[:, None]        # key t visible to row j iff t <= j
    y = np.where(causal, y, -np.inf)
    m = np.maximum(x.max(axis=1, keepdims=True), y.max(axis=1, keepdims=True))
    e = np.exp(x - m)
    z = e.sum(axis=1, keepdims=True) + np.exp(y - m).sum(axis=1, keepdims=True)
    return e / z


def guide_attention_sum(q_group: np.ndarray, k_rows: np.ndarray, softmax_scale: float,
                        kg_rows: np.ndarray | None = None) -> np.ndarray:
    """Inner sum of Eq. 1, sum_j A[j, i], averaged over the R query heads that share the
    KV head.  q_group [R, G, d]; kg_rows: the KV head's guide keys [G, d] or None."""
    R = q_group.shape[0]
    raw = np.zeros(k_rows.shape[0], dtype=np.float64)
    for r in range(R):
        raw += attention_slice(q_group[r], k_rows, softmax_scale, kg_rows).sum(axis=0)
    return raw / R


def guide_log_normalisers(q_rows: np.ndarray, k_rows: np.ndarray, softmax_scale: float,
                          kg_rows: np.ndarray | None = None) -> np.ndarray:
    """ln of each guide row's softmax normaliser, ln sum over the row's keys of
    exp(softmax_scale * <q_j, key>): over the N context keys, plus guide keys 0..j when
    kg_rows is given (the causal map of Sec. 3.2).  This is the log-sum-exp a prefill
    attention kernel reports for the appended guide rows.  q_rows [G, d] -> [G]."""
    x = softmax_scale * (q_rows @ k_rows.T)
    if kg_rows is not None:
        g = q_rows.shape[0]
        y = softmax_scale * (q_rows @ kg_rows.T)
        y = np.where(np.arange(g)[None, :] <= np.arange(g)[:, None], y, -np.inf)
        x = np.concatenate([x, y], axis=1)
    m = x.max(axis=1)
    return m + np.log(np.exp(x - m[:, None]).sum(axis=1))


def guide_attention_output(q_rows: np.ndarray, k_rows: np.ndarray, v_rows: np.ndarray, softmax_scale: float,
                           kg_rows: np.ndarray | None = None, vg_rows: np.ndarray | None = None) -> np.ndarray:
    """Output of the prefill's attention for the guide rows (Sec. 3.2: the guide is appended
    after the context and attends causally): row j is the softmax-weighted sum of the values
    of the keys it sees, the N context keys, plus guide keys 0..j when kg_rows / vg_rows [G, d]
    are given.  q_rows [G, d], k_rows / v_rows [N, d] -> [G, d], float64.  Its normaliser is
    guide_log_normalisers' (the weights of the context keys are attention_slice's)."""
    x = softmax_scale * (q_rows @ k_rows.T)
    if kg_rows is None:
        m = x.max(axis=1, keepdims=True)
        e = np.exp(x - m)
        return (e @ v_rows) / e.sum(axis=1, keepdims=True)
    g = q_rows.shape[0]
    y = softmax_scale * (q_rows @ kg_rows.T)
    y = np.where(np.arange(g)[None, :] <= np.arange(g)[:, None], y, -np.inf)  # guide key t seen by row j iff t <= j
    m = np.maximum(x.max(axis=1, keepdims=True), y.max(axis=1, keepdims=True))
    e, eg = np.exp(x - m), np.exp(y - m)
    return (e @ v_rows + eg @ vg_rows) / (e.sum(axis=1, keepdims=True) + eg.sum(axis=1, keepdims=True))


def guide_attention_sum_given_lse(q_group: np.ndarray, k_rows: np.ndarray, softmax_scale: float,
                                  lse: np.ndarray) -> np.ndarray:
    """Inner sum of Eq. 1 with the normaliser supplied by the caller (Sec. 3.2 slices A from
    the prefill's attention map, whose kernel already has each guide row's log-sum-exp):
    A[j, i] = exp(softmax_scale * <q_j, k_i> - lse_j), summed over j and averaged over the
    R query heads.  q_group [R, G, d], lse [R, G] (natural log)."""
    R = q_group.shape[0]
    raw = np.zeros(k_rows.shape[0], dtype=np.float64)
    for r in range(R):
        x = softmax_scale * (q_group[r] @ k_rows.T)
        raw += np.exp(x - np.asarray(lse[r], dtype=np.float64)[:, None]).sum(axis=0)
    return raw / R


def avg_pool(raw: np.ndarray, pool_k: int) -> np.ndarray:
    """Outer part of Eq. 1: (1/K) sum_{t=-floor(K/2)}^{floor(K/2)} raw[i + t], with raw = 0
    outside [0, N).  K must be odd."""
    if pool_k < 1 or pool_k % 2 == 0:
        raise ValueError("pool_k must be odd and >= 1")
    n = raw.shape[0]
    h = pool_k // 2
    acc = np.zeros(n, dtype=np.float64)
    for t in range(-h, h + 1):
        lo, hi = max(0, -t), min(n, n - t)  # i with 0 <= i + t < n
        if lo < hi:
            acc[lo:hi] += raw[lo + t:hi + t]
    return acc / pool_k


def key_scores(q_group: np.ndarray, k_rows: np.ndarray, softmax_scale: float, pool_k: int,
               kg_rows: np.ndarray | None = None) -> np.ndarray:
    """s_key of Eq. 1 for one KV head: pooled guide-attention sum (float64, [N])."""
    return avg_pool(guide_attention_sum(q_group, k_rows, softmax_scale, kg_rows), pool_k)


def key_scores_given_lse(q_group: np.ndarray, k_rows: np.ndarray, softmax_scale: float, pool_k: int,
                         lse: np.ndarray) -> np.ndarray:
    """s_key of Eq. 1 with the guide rows' log-normalisers supplied (float64, [N])."""
    return avg_pool(guide_attention_sum_given_lse(q_group, k_rows, softmax_scale, lse), pool_k)


# --------------------------------------------------------------------------- stage 2
def value_scales(v_rows: np.ndarray, qfmt: int = QFMT_INT, bits: int = 8) -> np.ndarray:
    """gamma_i = max_c |v_ic| / qmax (Eq. 2), per token, stored as fp32.  v_rows [N, d]."""
    absmax = np.abs(v_rows).max(axis=1)
    return to_f32(absmax / qmax_of(qfmt, bits))


def quantize_values(v_rows: np.ndarray, gamma: np.ndarray, qfmt: int = QFMT_INT, bits: int = 8) -> np.ndarray:
    """Per-token symmetric quantisation with scale gamma (Sec. 3.3).

    y = fl32(v / gamma); integers: clamp(RNE(y), -qmax, qmax) as int8 values; E4M3: the
    code of y.  Rows with gamma = 0 quantise to 0."""
    g = np.asarray(gamma, dtype=np.float64)[:, None]
    safe = np.where(g == 0.0, 1.0, g)
    y = to_f32(v_rows / safe).astype(np.float64)
    y = np.where(g == 0.0, 0.0, y)
    if qfmt == QFMT_INT:
        qm = qmax_of(qfmt, bits)
        return np.clip(np.rint(y), -qm, qm).astype(np.int8)
    if qfmt == QFMT_FP8_E4M3:
        return e4m3_encode(y)
    raise ValueError("unknown qfmt")


def pack_codes(q: np.ndarray, qfmt: int, bits: int) -> np.ndarray:
    """Storage bytes of quantised rows [N, d]: one byte per value, except integers with
    b <= 4, two per byte (even element in the low nibble, 4-bit two's complement)."""
    if qfmt == QFMT_INT and bits <= 4:
        u = (q.astype(np.int16) & 0xF).astype(np.uint8)
        return (u[:, 0::2] | (u[:, 1::2] << 4)).astype(np.uint8)
    return q.view(np.uint8) if q.dtype == np.int8 else q.astype(np.uint8)


# --------------------------------------------------------------------------- stage 3
def combine(s_key: np.ndarray, gamma: np.ndarray, rule: int = COMBINE_MUL) -> np.ndarray:
    """Combined score s_i, stored as fp32.

    MUL: s_key * gamma (Eq. 3).  KEY_ONLY: s_key (key-score-only ablation, Sec. 4.3).
    NORM_ADD: s_key/||s_key||_2 + gamma/||gamma||_2 over the segment; HARMONIC:
    2 s_key gamma / (s_key + gamma), 0 where both are 0 (aggregation table, Sec. 4.4)."""
    a = np.asarray(s_key, dtype=np.float64)
    b = np.asarray(gamma, dtype=np.float64)
    if rule == COMBINE_MUL:
        return to_f32(a * b)
    if rule == COMBINE_KEY_ONLY:
        return to_f32(a)
    if rule == COMBINE_NORM_ADD:
        na = math.sqrt(float(np.sum(a * a)))
        nb = math.sqrt(float(np.sum(b * b)))
        ta = a / na if na > 0 else np.zeros_like(a)
        tb = b / nb if nb > 0 else np.zeros_like(b)
        return to_f32(ta + tb)
    if rule == COMBINE_HARMONIC:
        den = a + b
        with np.errstate(invalid="ignore", divide="ignore"):
            h = np.where(den > 0, 2.0 * a * b / np.where(den > 0, den, 1.0), 0.0)
        return to_f32(h)
    raise ValueError("unknown rule")


def select(scores: np.ndarray, k: int) -> np.ndarray:
    """Index set I (Sec. 3.4): the k highest scores, ties to the lower index, ascending."""
    s = np.asarray(scores)
    n = s.shape[0]
    order = np.lexsort((np.arange(n), -s.astype(np.float64)))  # score desc, then index asc
    return np.sort(order[:k]).astype(np.int32)


# --------------------------------------------------------------------------- stage 4
def compact(rows: np.ndarray, idx: np.ndarray) -> np.ndarray:
    """Kept rows of one KV head (Sec. 3.1: only I is kept; Sec. 4: evicted after prefill)."""
    return rows[np.asarray(idx, dtype=np.int64)]


# --------------------------------------------------------------------------- full path
def evict_segment(q_group_bits, k_bits, v_bits, *, softmax_scale, pool_k, qfmt, bits, rule, k, kg_bits=None):
    """All four stages for one (sequence, layer, KV head).

    q_group_bits [R, G, d], k_bits / v_bits [N, d] (bf16 bit patterns); kg_bits [G, d], the
    KV head's guide keys (bf16 bits), or None for the context-only normaliser.  Returns a dict
    with s_key (float64), gamma (fp32), q (quantised values, unpacked), vq (packed
    bytes), S (fp32 combined score), idx (int32, ascending), and the compact rows
    k_c (bf16 bits), vq_c (bytes), gamma_c (fp32)."""
    qg = bf16_to_f64(q_group_bits)
    kr = bf16_to_f64(k_bits)
    vr = bf16_to_f64(v_bits)
    kg = None if kg_bits is None else bf16_to_f64(kg_bits)
    s_key = key_scores(qg, kr, softmax_scale, pool_k, kg)
    gamma = value_scales(vr, qfmt, bits)
    q = quantize_values(vr, gamma, qfmt, bits)
    vq = pack_codes(q, qfmt, bits)
    S = combine(s_key, gamma, rule)
    idx = select(S, k)
    return dict(s_key=s_key, gamma=gamma, q=q, vq=vq, S=S, idx=idx,
                k_c=compact(np.asarray(k_bits), idx), vq_c=compact(vq, idx), gamma_c=compact(gamma, idx))
