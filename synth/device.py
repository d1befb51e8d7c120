"""Seeded workload inputs drawn straight into device memory (torch tensors), bit-identical
to the host generator.  Input generation only: nothing here computes any step of the
eviction path."""
from __future__ import annotations

import torch

from . import TAG_KG, TAG_VG, Stream, device_fill


def device_inputs(w, device="cuda"):
    """Q/K/V of workload `w`: bf16 [L][Hq][G_tot][d], [L][Hkv][N_tot][d] twice."""
    lens = list(w.ctx_lens)
    glens = list(w.guide_lens)
    q = torch.empty(w.L * w.Hq * w.g_tot * w.d, dtype=torch.bfloat16, device=device)
    k = torch.empty(w.L * w.Hkv * w.n_tot * w.d, dtype=torch.bfloat16, device=device)
    v = torch.empty_like(k)
    s = torch.cuda.current_stream().cuda_stream
    device_fill(q.data_ptr(), w.q, w.L, w.Hq, glens, w.d, s)
    device_fill(k.data_ptr(), w.k, w.L, w.Hkv, lens, w.d, s)
    device_fill(v.data_ptr(), w.v, w.L, w.Hkv, lens, w.d, s)
    return q, k, v


def guide_key_stream(w):
    """The guide tokens' keys of workload w (N(0,1), same seed as its guide queries)."""
    return Stream(w.q.seed, TAG_KG)


def device_guide_keys(w, device="cuda"):
    """k_guide bf16 [L][Hkv][G_tot][d] of workload w."""
    kg = torch.empty(w.L * w.Hkv * w.g_tot * w.d, dtype=torch.bfloat16, device=device)
    device_fill(kg.data_ptr(), guide_key_stream(w), w.L, w.Hkv, list(w.guide_lens), w.d,
                torch.cuda.current_stream().cuda_stream)
    return kg


def guide_value_stream(w):
    """The guide tokens' values of workload w (N(0,1), same seed as its guide queries)."""
    return Stream(w.q.seed, TAG_VG)


def device_guide_values(w, device="cuda"):
    """v_guide bf16 [L][Hkv][G_tot][d] of workload w."""
    vg = torch.empty(w.L * w.Hkv * w.g_tot * w.d, dtype=torch.bfloat16, device=device)
    device_fill(vg.data_ptr(), guide_value_stream(w), w.L, w.Hkv, list(w.guide_lens), w.d,
                torch.cuda.current_stream().cuda_stream)
    return vg
