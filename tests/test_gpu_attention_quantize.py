"""tp_guide_attention_quantize, through the C ABI: the guide rows' prefill attention with step 2
(Eq. 2, Sec. 3.3) taken from the same sweep over V.

  - Its attention outputs (o_guide, guide_lse) are bit-identical to tp_guide_attention's on
    the same inputs (that entry point is held to the oracle in test_gpu_guide_attention.py).
  - Its scales and codes are bit-identical to the oracle's Eq. 2 quantisation of every context
    token: the ragged tails of chunks and sequences, sequences whose guides need two row
    groups (where only one workgroup may write), and planted rows that take every path of the
    arithmetic (zero rows, and absmax near 2^-110, 2^-60 and 2^115).
  - tp_evict with v = NULL on those scales and codes gives bit-identical outputs to tp_evict
    with v, and both match the oracle.
"""
import numpy as np
import pytest
import torch

import synth
from oracle import taskpress_oracle as o
from paper_2608_03276_amd import binding as B
from synth import workloads as W

import parity_util as pu

pytestmark = pytest.mark.gpu

INT, E4M3 = B.TP_QFMT_INT, B.TP_QFMT_FP8_E4M3

CASES = [
    # (name, L, Hq, Hkv, d, lens, glens, guide keys, qfmt, bits)
    ("ragged-d128-int8", 2, 8, 2, 128, [1, 31, 33, 2049, 8191, 8193], [1, 3, 64, 100, 7, 33], True, INT, 8),
    ("two-row-groups-int4", 1, 16, 2, 128, [3000, 700], [40, 33], True, INT, 4),
    ("chunk-edges-e4m3", 1, 8, 2, 128, [8192, 16384, 16385], [64, 9, 40], False, E4M3, 8),
    ("d64-int6", 1, 8, 2, 64, [8193, 40, 1], [200, 1, 3], True, INT, 6),
    ("d64-e4m3-one-token", 2, 4, 4, 64, [1, 2, 33], [2, 1, 5], False, E4M3, 8),
]

# planted V rows (row index of [L*Hkv*N_tot] modulo p == r): a power-of-two factor keeps the
# bf16 values exact and moves the row's absmax into another range of the arithmetic
PLANTS = [(97, 5, 0.0), (89, 7, 2.0 ** -60), (83, 11, 2.0 ** 115), (79, 13, 2.0 ** -110)]


def _workload(case):
    name, L, Hq, Hkv, d, lens, glens, _, qfmt, bits = case
    return W.Workload(name, L, Hq, Hkv, d, tuple(lens), tuple(glens), synth.Stream(73, synth.TAG_Q),
                      synth.Stream(73, synth.TAG_K), synth.Stream(73, synth.TAG_V), keep_ratio=0.25, pool_k=5,
                      qfmt=qfmt, bits=bits)


def _plant(v, d):
    rows = v.view(-1, d)
    idx = torch.arange(rows.shape[0], device=v.device)
    for p, r, f in PLANTS:
        sel = idx % p == r
        rows[sel] = (rows[sel].float() * f).to(torch.bfloat16)


def _oracle_quant(v_bits, qfmt, bits):
    """fp32 scale bits and code bytes of every row of v_bits [rows, d] (bf16 bits), per the oracle."""
    vr = o.bf16_to_f64(v_bits)
    g = o.value_scales(vr, qfmt, bits)
    return g.view(np.uint32), o.pack_codes(o.quantize_values(vr, g, qfmt, bits), qfmt, bits)


def _run(w, q, k, v, kg, vg):
    d = B.dims(w.L, w.Hq, w.Hkv, w.d)
    bt = B.Batch(w.ctx_offsets(), w.guide_offsets())
    rb = B.row_bytes(w.qfmt, w.bits, w.d)
    rows = w.L * w.Hkv * w.n_tot
    nrow = w.L * w.Hq * w.g_tot
    o_ref = torch.full((nrow * w.d,), float("nan"), dtype=torch.float32, device="cuda")
    l_ref = torch.full((nrow,), float("nan"), dtype=torch.float32, device="cuda")
    B.tp_guide_attention(d, bt, q, k, v, w.softmax_scale, o_ref, l_ref, k_guide=kg, v_guide=vg)
    o_q = torch.full_like(o_ref, float("nan"))
    l_q = torch.full_like(l_ref, float("nan"))
    scales = torch.full((rows,), float("nan"), dtype=torch.float32, device="cuda")
    vq = torch.full((rows * rb,), 0x5A, dtype=torch.uint8, device="cuda")
    B.tp_guide_attention_quantize(d, bt, q, k, v, w.softmax_scale, w.qfmt, w.bits, o_q, l_q, scales, vq,
                                  k_guide=kg, v_guide=vg)
    torch.cuda.synchronize()
    return (o_ref, l_ref), (o_q, l_q), scales, vq


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_attention_quantize_parity(gpu_lib, case):
    w = _workload(case)
    guide_keys = case[7]
    pu.log(f"attention + quantisation {w.name}: {w.describe()}, qfmt {w.qfmt} bits {w.bits}")
    q, k, v = pu.device_inputs(w)
    _plant(v, w.d)
    kg = pu.device_guide_keys(w) if guide_keys else None
    vg = pu.device_guide_values(w) if guide_keys else None
    (o_ref, l_ref), (o_q, l_q), scales, vq = _run(w, q, k, v, kg, vg)
    assert torch.equal(o_q.view(torch.int32), o_ref.view(torch.int32)), "attention output differs"
    assert torch.equal(l_q.view(torch.int32), l_ref.view(torch.int32)), "normalisers differ"
    g_ref, c_ref = _oracle_quant(v.view(torch.int16).cpu().numpy().view(np.uint16).reshape(-1, w.d), w.qfmt, w.bits)
    g_gpu = scales.cpu().numpy().view(np.uint32)
    c_gpu = vq.cpu().numpy().reshape(g_gpu.shape[0], -1)
    bad = np.nonzero(g_gpu != g_ref)[0]
    assert bad.size == 0, f"{bad.size} scales differ, first rows {bad[:8].tolist()}"
    bad = np.nonzero(np.any(c_gpu != c_ref, axis=1))[0]
    assert bad.size == 0, f"{bad.size} code rows differ, first rows {bad[:8].tolist()}"
    pu.log(f"  {g_gpu.shape[0]} rows: scales and codes bit-exact, attention outputs bit-identical")


@pytest.mark.parametrize("case", [CASES[0], CASES[1]], ids=[CASES[0][0], CASES[1][0]])
def test_evict_after_attention_quantize(gpu_lib, case):
    """tp_evict(v = NULL) on the fused call's scales and codes, with its normalisers: the same
    outputs, bit for bit, as tp_evict(v) with those normalisers, and the oracle's."""
    w = _workload(case)
    pu.log(f"evict without V after attention + quantisation: {w.describe()}")
    q, k, v = pu.device_inputs(w)
    kg, vg = pu.device_guide_keys(w), pu.device_guide_values(w)
    d = B.dims(w.L, w.Hq, w.Hkv, w.d)
    bt = B.Batch(w.ctx_offsets(), w.guide_offsets())
    o_q = torch.empty(w.L * w.Hq * w.g_tot * w.d, dtype=torch.float32, device="cuda")
    lse = torch.empty(w.L * w.Hq * w.g_tot, dtype=torch.float32, device="cuda")
    kw = dict(softmax_scale=w.softmax_scale, pool_k=w.pool_k, qfmt=w.qfmt, bits=w.bits, rule=w.rule,
              keep_ratio=w.keep_ratio or 0.0, keep_budget=w.keep_budget or 0, guide_lse=lse)
    ko = B.kept_offsets_for(bt, w.keep_ratio or 0.0, w.keep_budget or 0)
    bufs = B.EvictBuffers(d, bt, w.qfmt, w.bits, ko, device=k.device)
    B.tp_guide_attention_quantize(d, bt, q, k, v, w.softmax_scale, w.qfmt, w.bits, o_q, lse, bufs.scales,
                                  bufs.v_q, k_guide=kg, v_guide=vg)
    ref = B.evict_fused(d, bt, q, k, v, **kw)
    B.evict_fused(d, bt, q, k, None, **kw, bufs=bufs)
    torch.cuda.synchronize()
    for name in ("s_key", "scales", "v_q", "s_comb", "kept_idx", "k_c", "v_q_c", "scales_c"):
        a, b = getattr(bufs, name), getattr(ref, name)
        assert torch.equal(a.view(torch.uint8), b.view(torch.uint8)), name + " differs"
    for b in range(w.batch):
        for l in range(w.L):
            for h in range(w.Hkv):
                pu.check_segment(w, bufs, b, l, h, guide_keys=True)


def test_attention_quantize_fullsize(gpu_lib):
    """The 128K workload in the launch configuration `bench.py --prefill-attention` times:
    attention outputs bit-identical to tp_guide_attention's, every scale and code equal to
    tp_quantize_v_scales's (itself held to the oracle), and sampled rows of two segments,
    across the chunk edges and at the end, against the oracle."""
    w = W.ALL["llama8b_128k"]()
    pu.log(f"attention + quantisation, full size: {w.describe()}")
    torch.cuda.empty_cache()
    q, k, v = pu.device_inputs(w)
    kg, vg = pu.device_guide_keys(w), pu.device_guide_values(w)
    (o_ref, l_ref), (o_q, l_q), scales, vq = _run(w, q, k, v, kg, vg)
    assert torch.equal(o_q.view(torch.int32), o_ref.view(torch.int32)), "attention output differs"
    assert torch.equal(l_q.view(torch.int32), l_ref.view(torch.int32)), "normalisers differ"
    del o_ref, l_ref, o_q, l_q
    d = B.dims(w.L, w.Hq, w.Hkv, w.d)
    bt = B.Batch(w.ctx_offsets(), w.guide_offsets())
    s2 = torch.empty_like(scales)
    vq2 = torch.empty_like(vq)
    B.tp_quantize_v_scales(d, bt, v, w.qfmt, w.bits, s2, vq2)
    torch.cuda.synchronize()
    assert torch.equal(scales.view(torch.int32), s2.view(torch.int32)), "scales differ from tp_quantize_v_scales"
    assert torch.equal(vq, vq2), "codes differ from tp_quantize_v_scales"
    del s2, vq2
    n = w.n_tot
    rb = B.row_bytes(w.qfmt, w.bits, w.d)
    for (l, h) in [(0, 0), (17, 3)]:
        seg = l * w.Hkv + h
        vb = synth.rows(w.v, 0, l, h, n, w.d)
        for t0, t1 in [(0, 512), (32768 - 256, 32768 + 256), (98304 - 64, 98304 + 64), (n - 300, n)]:
            g_ref, c_ref = _oracle_quant(vb[t0:t1], w.qfmt, w.bits)
            r0, r1 = seg * n + t0, seg * n + t1
            assert np.array_equal(scales[r0:r1].cpu().numpy().view(np.uint32), g_ref), (l, h, t0)
            assert np.array_equal(vq[r0 * rb:r1 * rb].cpu().numpy().reshape(t1 - t0, rb), c_ref), (l, h, t0)
    pu.log("  full-size scales and codes equal to tp_quantize_v_scales; sampled rows match the oracle")


@pytest.mark.parametrize("rule", [B.TP_COMBINE_NORM_ADD, B.TP_COMBINE_HARMONIC], ids=["norm-add", "harmonic"])
def test_evict_without_v_rules_and_pass1(gpu_lib, rule):
    """tp_evict(v = NULL) with step 2 from tp_quantize_v_scales and both score passes (no
    normalisers given), under the rules whose pooling runs in its own kernel (normalised add)
    or in the selection (harmonic): bit-identical to tp_evict(v), with the profile events."""
    w = _workload(CASES[0])
    pu.log(f"evict without V, both passes, rule {rule}: {w.describe()}")
    q, k, v = pu.device_inputs(w)
    d = B.dims(w.L, w.Hq, w.Hkv, w.d)
    bt = B.Batch(w.ctx_offsets(), w.guide_offsets())
    kw = dict(softmax_scale=w.softmax_scale, pool_k=w.pool_k, qfmt=w.qfmt, bits=w.bits, rule=rule,
              keep_ratio=w.keep_ratio or 0.0, keep_budget=w.keep_budget or 0)
    ref = B.evict_fused(d, bt, q, k, v, **kw)
    bufs = B.EvictBuffers(d, bt, w.qfmt, w.bits, ref.kept_offsets, device=k.device)
    B.tp_quantize_v_scales(d, bt, v, w.qfmt, w.bits, bufs.scales, bufs.v_q)
    events = [torch.cuda.Event(enable_timing=True) for _ in range(B.TP_EVICT_EVENTS)]
    B.evict_fused(d, bt, q, k, None, **kw, bufs=bufs, events=events)
    torch.cuda.synchronize()
    for name in ("s_key", "scales", "v_q", "s_comb", "kept_idx", "k_c", "v_q_c", "scales_c"):
        a, b = getattr(bufs, name), getattr(ref, name)
        assert torch.equal(a.view(torch.uint8), b.view(torch.uint8)), name + " differs"
    ms = [events[i].elapsed_time(events[i + 1]) for i in range(B.TP_EVICT_EVENTS - 1)]
    assert all(t >= 0.0 for t in ms), ms


@pytest.mark.parametrize("bits", [2, 3, 5, 7])
def test_attention_quantize_bit_widths(gpu_lib, bits):
    """The integer widths the cases above leave out (each has its own qmax and its own
    one-multiply multipliers or fallbacks): scales and codes bit-exact against the oracle,
    with the planted rows, on a batch with a ragged tail and two row groups."""
    case = (f"int{bits}", 1, 16, 2, 128, [3001, 64], [40, 3], False, INT, bits)
    w = _workload(case)
    pu.log(f"attention + quantisation, int{bits}: {w.describe()}")
    q, k, v = pu.device_inputs(w)
    _plant(v, w.d)
    (o_ref, l_ref), (o_q, l_q), scales, vq = _run(w, q, k, v, None, None)
    assert torch.equal(o_q.view(torch.int32), o_ref.view(torch.int32)), "attention output differs"
    g_ref, c_ref = _oracle_quant(v.view(torch.int16).cpu().numpy().view(np.uint16).reshape(-1, w.d), w.qfmt, w.bits)
    g_gpu = scales.cpu().numpy().view(np.uint32)
    c_gpu = vq.cpu().numpy().reshape(g_gpu.shape[0], -1)
    assert np.array_equal(g_gpu, g_ref), f"{int(np.sum(g_gpu != g_ref))} scales differ"
    bad = np.nonzero(np.any(c_gpu != c_ref, axis=1))[0]
    assert bad.size == 0, f"{bad.size} code rows differ, first rows {bad[:8].tolist()}"
