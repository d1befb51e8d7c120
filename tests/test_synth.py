"""The seeded input generator (host build): published-definition checks, distribution
sanity and exact outlier counts.  The device build's bit-equality is a GPU test."""
import math
from fractions import Fraction

import numpy as np
import pytest

import synth
from synth import workloads

lib = synth.host_lib()


def test_splitmix64_reference_values():
    """SplitMix64 with seed 0: the first outputs of the published generator (Steele et al.
    2014; the same constants as java.util.SplittableRandom's mix64)."""
    expect = [0xE220A8397B1DCDAF, 0x6E789E6AA1B965F4, 0x06C45D188009454F]
    assert [lib.syn_probe_at(0, n) for n in range(3)] == expect


def test_log_and_cos_series_accuracy():
    rng = np.random.default_rng(5)
    for x in np.concatenate([rng.random(5000), 2.0 ** -rng.uniform(0, 53, 5000), [1.0, 0.5, 2.0 ** -53]]):
        ref = math.log(x)
        assert abs(lib.syn_probe_log(float(x)) - ref) <= 4e-16 * max(1.0, abs(ref))
    for w in rng.random(5000):
        assert abs(lib.syn_probe_cos_turns(float(w)) - math.cos(2 * math.pi * w)) <= 2e-15


def test_bf16_rounding_is_exact_rne():
    pos = (np.arange(0x7F80, dtype=np.uint32) << 16).view(np.float32).astype(np.float64)
    rng = np.random.default_rng(6)
    xs = list(rng.standard_normal(3000) * 10.0 ** rng.integers(-44, 38, 3000))
    for c in rng.integers(0, 0x7F7F, 1000):
        xs.append(float((Fraction(pos[c]) + Fraction(pos[c + 1])) / 2))  # exact ties
    for x in xs:
        a = abs(x)
        i = int(np.searchsorted(pos, a))
        cands = [c for c in (i - 1, i) if 0 <= c < len(pos)]
        best = min(cands, key=lambda c: (abs(Fraction(a) - Fraction(pos[c])), c & 1))
        assert lib.syn_probe_to_bf16(float(x)) == (best | (0x8000 if x < 0 else 0))


def test_normal_and_student_t_moments():
    n = 200000
    z = synth.bf16_bits_to_f64(synth.rows(synth.Stream(1, synth.TAG_K), 0, 0, 0, n // 100, 100))
    assert abs(z.mean()) < 0.01 and abs(z.std() - 1) < 0.01
    t = synth.bf16_bits_to_f64(synth.rows(synth.Stream(1, synth.TAG_V, synth.DIST_STUDENT_T3), 0, 0, 0, n // 100, 100))
    # Student-t(3): variance 3, heavy tails (P(|t| > 5) ~ 1.54 %)
    assert abs(t.var() - 3) < 0.6 and 0.01 < np.mean(np.abs(t) > 5) < 0.02


@pytest.mark.parametrize("n,frac", [(1, 0.5), (7, 0.3), (1000, 0.005), (32768, 0.005), (5000, 0.01)])
def test_outlier_perm_is_bijection_with_exact_count(n, frac):
    perm = [lib.syn_probe_perm(i, n, 1234567) for i in range(n)]
    assert sorted(perm) == list(range(n))
    s = synth.Stream(9, synth.TAG_V, synth.DIST_NORMAL, frac, 1000.0)
    x = np.abs(synth.bf16_bits_to_f64(synth.rows(s, 0, 3, 1, n, 8)))
    expect = int(math.floor(frac * n + 0.5))
    assert int((x.max(axis=1) > 30).sum()) == expect


def test_segments_regenerate_independently():
    s = synth.Stream(3, synth.TAG_K)
    full = synth.host_tensor(s, 2, 3, [50, 70], 16)
    seg = synth.rows(s, 1, 1, 2, 70, 16)
    assert np.array_equal(full[1, 2, 50:], seg)
    part = synth.rows(s, 1, 1, 2, 70, 16, t0=20, n=15)
    assert np.array_equal(part, seg[20:35])


def test_workload_shapes():
    w = workloads.ragged8()
    assert len(w.ctx_lens) == 8 and all(4096 <= n <= 65536 for n in w.ctx_lens)
    assert w.guide_lens == (32, 128, 32, 128, 32, 128, 32, 128)
    assert workloads.ragged8().ctx_lens == w.ctx_lens
    t = workloads.tiny()
    assert (t.L, t.Hq, t.Hkv, t.d, t.ctx_lens, t.guide_lens) == (1, 8, 2, 64, (1024,), (16,))
