"""The guide rows' prefill attention (tp_guide_attention, through the C ABI) against the
oracle: the attention output and the log-normaliser of every guide row, and the eviction
driven by those normalisers against the oracle's key scores with the guide keys in the
normaliser (Sec. 3.2: A is the context slice of the prefill's causal attention map).

Tolerances: the normaliser within 1e-4 (absolute, natural log: a relative 1e-4 on every
weight); an output element within 2^-8 of the row's attention-weighted mean of |v| in that
column (the probabilities are rounded to bf16, relative error <= 2^-9, before the value
product, as flash attention does)."""
import numpy as np
import pytest
import torch

import synth
from oracle import taskpress_oracle as o
from paper_2608_03276_amd import binding as B
from synth import workloads as W

import parity_util as pu

pytestmark = pytest.mark.gpu

CASES = [
    # (name, L, Hq, Hkv, d, lens, glens, guide keys)
    ("tiny-d64", 1, 8, 2, 64, [1024], [16], False),
    ("tiny-d64-guide-keys", 1, 8, 2, 64, [1024], [16], True),
    ("ragged-d128-guide-keys", 2, 8, 2, 128, [1, 31, 33, 2049, 8191, 8193], [1, 3, 64, 100, 7, 33], True),
    ("chunk-edges", 1, 8, 2, 128, [8192, 16384, 16385], [64, 9, 40], True),
    ("two-row-groups", 1, 16, 2, 128, [3000, 700], [40, 33], True),
    ("outliers-no-guide-keys", 1, 8, 2, 128, [4500], [64], False),
    # degenerate: one query head per KV head, single guide tokens, a one-token context
    ("mha-one-row", 2, 2, 2, 64, [1, 5000, 33], [1, 1, 2], True),
    # head dim 64 with guide keys over the 8192-token chunk edge and a long guide
    ("d64-chunk-edge", 1, 8, 2, 64, [8193, 40], [200, 1], True),
]


def _workload(case):
    name, L, Hq, Hkv, d, lens, glens, _ = case
    k = synth.Stream(71, synth.TAG_K, synth.DIST_STUDENT_T3, 0.02, 30.0) if "outliers" in name else \
        synth.Stream(71, synth.TAG_K)
    return W.Workload(name, L, Hq, Hkv, d, tuple(lens), tuple(glens), synth.Stream(71, synth.TAG_Q), k,
                      synth.Stream(71, synth.TAG_V), keep_ratio=0.25, pool_k=5)


def _run_attention(w, guide_keys):
    q, k, v = pu.device_inputs(w)
    kg = pu.device_guide_keys(w) if guide_keys else None
    vg = pu.device_guide_values(w) if guide_keys else None
    d = B.dims(w.L, w.Hq, w.Hkv, w.d)
    bt = B.Batch(w.ctx_offsets(), w.guide_offsets())
    o_out = torch.full((w.L * w.Hq * w.g_tot * w.d,), float("nan"), dtype=torch.float32, device="cuda")
    lse = torch.full((w.L * w.Hq * w.g_tot,), float("nan"), dtype=torch.float32, device="cuda")
    B.tp_guide_attention(d, bt, q, k, v, w.softmax_scale, o_out, lse, k_guide=kg, v_guide=vg)
    torch.cuda.synchronize()
    return (q, k, v, kg, vg), o_out.cpu().numpy().reshape(w.L, w.Hq, w.g_tot, w.d), \
        lse.cpu().numpy().reshape(w.L, w.Hq, w.g_tot)


def _check_rows(w, b, l, h, qheads, o_gpu, lse_gpu, guide_keys):
    """The oracle's output and normaliser for the guide rows of query heads `qheads` (of KV
    head h) of sequence b, layer l, against the GPU's; returns the worst output error (as a
    fraction of the weighted |v|) and the worst normaliser error."""
    g = w.guide_lens[b]
    goff = w.guide_offsets()
    _, kb, vb = pu.host_segment(w, b, l, h)
    kr, vr = o.bf16_to_f64(kb), o.bf16_to_f64(vb)
    kg = o.bf16_to_f64(pu.host_guide_keys(w, b, l, h)) if guide_keys else None
    vg = o.bf16_to_f64(pu.host_guide_values(w, b, l, h)) if guide_keys else None
    worst_o = worst_l = 0.0
    for qh in qheads:
        qr = o.bf16_to_f64(synth.rows(w.q, b, l, qh, g, w.d))
        ref = o.guide_attention_output(qr, kr, vr, w.softmax_scale, kg, vg)
        mag = o.guide_attention_output(qr, kr, np.abs(vr), w.softmax_scale, kg, None if vg is None else np.abs(vg))
        got = o_gpu[l, qh, goff[b]:goff[b] + g].astype(np.float64)
        err = np.abs(got - ref)
        tag = f"{w.name} b={b} l={l} qh={qh}"
        assert np.all(np.isfinite(got)), tag
        assert np.all(err <= 2.0 ** -8 * mag + 1e-7), (tag, float((err / (mag + 1e-30)).max()))
        worst_o = max(worst_o, float((err / (mag + 1e-30)).max()))
        lref = o.guide_log_normalisers(qr, kr, w.softmax_scale, kg)
        lgot = lse_gpu[l, qh, goff[b]:goff[b] + g].astype(np.float64)
        assert np.all(np.abs(lgot - lref) <= 1e-4), (tag, float(np.abs(lgot - lref).max()))
        worst_l = max(worst_l, float(np.abs(lgot - lref).max()))
    return worst_o, worst_l


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_guide_attention_parity(gpu_lib, case):
    w = _workload(case)
    guide_keys = case[-1]
    pu.log(f"guide attention {w.name}: {w.describe()}, guide keys {guide_keys}")
    _, o_gpu, lse_gpu = _run_attention(w, guide_keys)
    worst_o = worst_l = 0.0
    for b in range(w.batch):
        for l in range(w.L):
            for h in range(w.Hkv):
                wo, wl = _check_rows(w, b, l, h, range(h * w.R, (h + 1) * w.R), o_gpu, lse_gpu, guide_keys)
                worst_o, worst_l = max(worst_o, wo), max(worst_l, wl)
    pu.log(f"  output error <= {worst_o:.3g} of the weighted |v|, normaliser error <= {worst_l:.3g}")


# The full-size workloads in the launch configuration `bench.py --prefill-attention` times,
# guide keys included (contexts of 131072 tokens or more take 32768-token chunks, shorter ones
# 8192): every output and normaliser finite, and sampled (sequence, layer, KV head, query
# head) rows against the oracle.
FULL = {
    "llama8b_128k": [(0, 0, 0, 0), (0, 17, 3, 14), (0, 31, 7, 31)],
    "llama8b_32k": [(0, 16, 3, 13)],
    "ragged8": [(2, 9, 2, 9), (7, 31, 7, 30)],
}


@pytest.mark.parametrize("name", list(FULL))
def test_guide_attention_fullsize_sampled(gpu_lib, name):
    w = W.ALL[name]()
    pu.log(f"guide attention, full size: {w.describe()}")
    torch.cuda.empty_cache()
    tensors, o_gpu, lse_gpu = _run_attention(w, True)
    del tensors
    torch.cuda.empty_cache()
    assert np.all(np.isfinite(o_gpu)) and np.all(np.isfinite(lse_gpu))
    for (b, l, h, qh) in FULL[name]:
        assert qh // w.R == h
        wo, wl = _check_rows(w, b, l, h, [qh], o_gpu, lse_gpu, True)
        pu.log(f"  b={b} l={l} qh={qh}: output error <= {wo:.3g} of the weighted |v|, normaliser error <= {wl:.3g}")


@pytest.mark.parametrize("case", [CASES[2], CASES[4]], ids=[CASES[2][0], CASES[4][0]])
def test_evict_with_prefill_attention_normalisers(gpu_lib, case):
    """tp_evict with the normalisers of tp_guide_attention (the prefill-integrated path: one
    sweep over K for the scores on top of the attention's) against the oracle's scores and
    kept sets with the guide keys in the normaliser."""
    w = _workload(case)
    pu.log(f"evict with the prefill attention's normalisers: {w.describe()}")
    (q, k, v, kg, vg), _, _ = _run_attention(w, True)
    d = B.dims(w.L, w.Hq, w.Hkv, w.d)
    bt = B.Batch(w.ctx_offsets(), w.guide_offsets())
    o_out = torch.empty(w.L * w.Hq * w.g_tot * w.d, dtype=torch.float32, device="cuda")
    lse = torch.empty(w.L * w.Hq * w.g_tot, dtype=torch.float32, device="cuda")
    B.tp_guide_attention(d, bt, q, k, v, w.softmax_scale, o_out, lse, k_guide=kg, v_guide=vg)
    bufs = B.evict_fused(d, bt, q, k, v, softmax_scale=w.softmax_scale, pool_k=w.pool_k, qfmt=w.qfmt, bits=w.bits,
                         rule=w.rule, keep_ratio=w.keep_ratio or 0.0, keep_budget=w.keep_budget or 0, guide_lse=lse)
    torch.cuda.synchronize()
    for b in range(w.batch):
        for l in range(w.L):
            for h in range(w.Hkv):
                pu.check_segment(w, bufs, b, l, h, guide_keys=True)
