"""The full-size workloads in the launch configuration the bench times, checked against the
oracle on sampled (sequence, layer, KV head) segments, plus size-independent properties of
every segment."""
import numpy as np
import pytest
import torch

from paper_2608_03276_amd import binding as B
from synth import workloads as W

import parity_util as pu

pytestmark = pytest.mark.gpu

# (sequence, layer, KV head) segments checked against the oracle: first, middle and last
# layers, spread over the KV heads (and over the sequences of the ragged batch)
SAMPLES = {
    "tiny": [(0, 0, 0), (0, 0, 1)],
    "llama8b_32k": [(0, 0, 0), (0, 16, 3), (0, 31, 7)],
    "llama8b_128k": [(0, 0, 0), (0, 16, 5), (0, 17, 3), (0, 31, 7)],
    "ragged8": [(0, 0, 0), (1, 9, 2), (3, 16, 5), (6, 31, 1), (7, 31, 7)],
    "widegqa_256k": [(0, 0, 0), (0, 24, 3), (0, 47, 5)],
}


def _properties_all_segments(w, bufs):
    """Every segment keeps exactly k ascending in-range indices."""
    ko = bufs.kept_offsets
    kt = ko[-1]
    kept = bufs.kept_idx[: w.L * w.Hkv * kt].view(w.L * w.Hkv, kt)
    for b in range(w.batch):
        part = kept[:, ko[b]:ko[b + 1]]
        if part.shape[1] > 1:
            assert bool((part[:, 1:] > part[:, :-1]).all()), f"b={b}: kept indices not ascending"
        assert int(part.min()) >= 0 and int(part.max()) < w.ctx_lens[b], f"b={b}: index out of range"
    s = bufs.s_key[: w.L * w.Hkv * w.n_tot]
    assert bool(torch.isfinite(s).all()) and bool((s >= 0).all())
    # each segment's raw attention sums to G per query head before pooling: with zero-padded
    # pooling the pooled sum is at most G and at least G * (1 - (K-1)/N) (edges only)
    per_seg = s.view(w.L * w.Hkv, w.n_tot).double()
    offs = w.ctx_offsets()
    for b in range(w.batch):
        tot = per_seg[:, offs[b]:offs[b + 1]].sum(dim=1)
        g = w.guide_lens[b]
        assert bool((tot <= g * (1 + 1e-3)).all()), f"b={b}: pooled mass above G"


@pytest.mark.parametrize("name", list(SAMPLES))
def test_fullsize_sampled(gpu_lib, name):
    w = W.ALL[name]()
    pu.log(f"full size: {w.describe()}")
    torch.cuda.empty_cache()
    q, k, v = pu.device_inputs(w)
    bufs = pu.run_gpu(w, q, k, v, fused=True)  # tp_evict, as the bench runs it
    _properties_all_segments(w, bufs)
    for (b, l, h) in SAMPLES[name]:
        pu.log(f"  oracle segment b={b} l={l} h={h}")
        diag = pu.check_segment(w, bufs, b, l, h)
        pu.log(f"    {diag}")
    del q, k, v, bufs
    torch.cuda.empty_cache()


def test_fullsize_lean_modes(gpu_lib):
    """The bench's 128K shape in the two other modes of tp_evict: without the code tensor of
    every token the compact cache is bit-identical, and with the normalisers supplied (fp32
    logsumexp from torch matmuls, standing in for what the prefill exports) sampled segments
    match the oracle."""
    import bench

    w = W.llama8b_128k()
    pu.log(f"full size, lean modes: {w.describe()}")
    torch.cuda.empty_cache()
    q, k, v = pu.device_inputs(w)
    d = B.dims(w.L, w.Hq, w.Hkv, w.d)
    bt = B.Batch(w.ctx_offsets(), w.guide_offsets())
    kw = dict(softmax_scale=w.softmax_scale, pool_k=w.pool_k, qfmt=w.qfmt, bits=w.bits, rule=w.rule,
              keep_ratio=w.keep_ratio or 0.0, keep_budget=w.keep_budget or 0)
    full = B.evict_fused(d, bt, q, k, v, **kw)
    lean = B.evict_fused(d, bt, q, k, v, full_codes=False, **kw)
    torch.cuda.synchronize()
    for n in ("kept_idx", "k_c", "v_q_c", "scales_c"):
        assert torch.equal(getattr(full, n).view(torch.uint8), getattr(lean, n).view(torch.uint8)), n
    del lean
    lse = bench.prefill_lse(w, q, k)
    given = B.evict_fused(d, bt, q, k, v, guide_lse=lse, bufs=full, **kw)
    torch.cuda.synchronize()
    for (b, l, h) in SAMPLES["llama8b_128k"]:
        pu.log(f"  oracle segment b={b} l={l} h={h} (normalisers supplied)")
        pu.log(f"    {pu.check_segment(w, given, b, l, h)}")
    del q, k, v, full, given, lse
    torch.cuda.empty_cache()
