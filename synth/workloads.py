"""The synthetic workloads: shapes, value distributions and eviction settings.

Five workloads are defined, from a tiny parity case to a 256K-context wide-GQA
case; their shapes follow the paper's setting (Llama-3.1-8B-like GQA 32q/8kv,
head_dim 128, contexts of 32K-64K and beyond, guides of tens of tokens, keep
ratios of 5-25 %, per-token quantised V caches).  The paper's own benchmark
data (LongBench, RULER) is not used: seeded draws of the same shapes stand in.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field, replace

from . import DIST_NORMAL, DIST_STUDENT_T3, TAG_K, TAG_Q, TAG_V, Stream, host_lib

BASE_SEED = 20260803

QFMT_INT, QFMT_FP8_E4M3 = 0, 1
COMBINE_MUL, COMBINE_NORM_ADD, COMBINE_HARMONIC, COMBINE_KEY_ONLY = 0, 1, 2, 3


@dataclass(frozen=True)
class Workload:
    name: str
    L: int
    Hq: int
    Hkv: int
    d: int
    ctx_lens: tuple
    guide_lens: tuple
    q: Stream
    k: Stream
    v: Stream
    keep_ratio: float | None = None
    keep_budget: int | None = None
    qfmt: int = QFMT_INT
    bits: int = 8
    pool_k: int = 5
    rule: int = COMBINE_MUL
    softmax_scale: float = field(default=0.0)

    def __post_init__(self):
        if self.softmax_scale == 0.0:
            object.__setattr__(self, "softmax_scale", 1.0 / math.sqrt(self.d))

    @property
    def R(self) -> int:
        return self.Hq // self.Hkv

    @property
    def batch(self) -> int:
        return len(self.ctx_lens)

    @property
    def n_tot(self) -> int:
        return sum(self.ctx_lens)

    @property
    def g_tot(self) -> int:
        return sum(self.guide_lens)

    def ctx_offsets(self):
        out = [0]
        for n in self.ctx_lens:
            out.append(out[-1] + int(n))
        return out

    def guide_offsets(self):
        out = [0]
        for g in self.guide_lens:
            out.append(out[-1] + int(g))
        return out

    def with_(self, **kw) -> "Workload":
        return replace(self, **kw)

    def describe(self) -> str:
        dist = {DIST_NORMAL: "N(0,1)", DIST_STUDENT_T3: "Student-t(3)"}[self.k.dist]
        n = (f"N={self.ctx_lens[0]}" if self.batch == 1
             else f"{self.batch} seqs N_b in [{min(self.ctx_lens)},{max(self.ctx_lens)}] (sum {self.n_tot})")
        g = f"G={self.guide_lens[0]}" if len(set(self.guide_lens)) == 1 else f"G_b in {sorted(set(self.guide_lens))}"
        keep = f"keep ratio {self.keep_ratio}" if self.keep_ratio is not None else f"budget {self.keep_budget}"
        fmt = "int%d" % self.bits if self.qfmt == QFMT_INT else "fp8-e4m3"
        return (f"{self.name}: {self.L} layers, {self.Hq}q/{self.Hkv}kv, d={self.d}, {n}, {g}, "
                f"K/V bf16 {dist}, {keep}, {fmt} V scales, pool {self.pool_k}")


def _streams(seed, dist=DIST_NORMAL, k_out=(0.0, 1.0), v_out=(0.0, 1.0)):
    return (Stream(seed, TAG_Q, DIST_NORMAL),
            Stream(seed, TAG_K, dist, k_out[0], k_out[1]),
            Stream(seed, TAG_V, dist, v_out[0], v_out[1]))


def ragged_lengths(seed: int, batch: int, lo: int, hi: int):
    """Sequence lengths drawn uniformly in [lo, hi] from the SplitMix64 stream of `seed`."""
    lib = host_lib()
    key = lib.syn_probe_at(seed, 0xC0FFEE)
    return tuple(lo + int(lib.syn_probe_at(key, b) % (hi - lo + 1)) for b in range(batch))


def tiny() -> Workload:
    s = BASE_SEED + 1
    q, k, v = _streams(s)
    return Workload("tiny", 1, 8, 2, 64, (1024,), (16,), q, k, v, keep_ratio=0.25)


def llama8b_32k() -> Workload:
    s = BASE_SEED + 2
    q, k, v = _streams(s, DIST_NORMAL, (0.005, 20.0), (0.005, 20.0))
    return Workload("llama8b-32k", 32, 32, 8, 128, (32768,), (64,), q, k, v, keep_ratio=0.2)


def llama8b_128k() -> Workload:
    s = BASE_SEED + 3
    q, k, v = _streams(s, DIST_STUDENT_T3)
    return Workload("llama8b-128k", 32, 32, 8, 128, (131072,), (64,), q, k, v, keep_ratio=0.1)


def ragged8() -> Workload:
    s = BASE_SEED + 4
    q, k, v = _streams(s)
    lens = ragged_lengths(s, 8, 4096, 65536)
    glens = tuple(32 if b % 2 == 0 else 128 for b in range(8))
    return Workload("ragged8", 32, 32, 8, 128, lens, glens, q, k, v, keep_budget=2048)


def widegqa_256k() -> Workload:
    s = BASE_SEED + 5
    q, k, v = _streams(s, DIST_NORMAL, (0.0, 1.0), (0.01, 30.0))
    return Workload("widegqa-256k", 48, 64, 8, 128, (262144,), (256,), q, k, v, keep_ratio=0.05,
                    qfmt=QFMT_FP8_E4M3, bits=8)


ALL = {w.__name__: w for w in (tiny, llama8b_32k, llama8b_128k, ragged8, widegqa_256k)}
