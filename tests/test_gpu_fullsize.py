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

SAMPLES = {
    "tiny": [(0, 0, 0), (0, 0, 1)],
    "llama8b_32k": [(0, 0, 0), (0, 31, 7)],
    "llama8b_128k": [(0, 0, 0), (0, 17, 3)],
    "ragged8": [(0, 0, 0), (1, 9, 2), (7, 31, 7)],
    "widegqa_256k": [(0, 47, 5)],
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
    bufs = pu.run_gpu(w, q, k, v)
    _properties_all_segments(w, bufs)
    for (b, l, h) in SAMPLES[name]:
        pu.log(f"  oracle segment b={b} l={l} h={h}")
        diag = pu.check_segment(w, bufs, b, l, h)
        pu.log(f"    {diag}")
    del q, k, v, bufs
    torch.cuda.empty_cache()
