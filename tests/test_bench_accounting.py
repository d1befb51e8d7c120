"""The algorithmic byte counts bench.py divides by the measured times (CPU only): the whole
path's bytes follow the compulsory-traffic formula per (layer, KV head, context token) at
d = 128 — read K and V once, write the 8-bit codes and the fp32 scale (644 B), plus per
kept token the re-read of its K row, codes and scale and the write of the compact cache and
index (780 B) — and the per-launch counts of step 2 add up over its launches."""
import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import bench  # noqa: E402
from synth import workloads as W  # noqa: E402


def _kept(w):
    from oracle import taskpress_oracle as o

    return sum(o.keep_count(n, w.keep_ratio, w.keep_budget) for n in w.ctx_lens)


def test_path_bytes_128k():
    w = W.llama8b_128k()
    k = _kept(w)
    assert k == 13107
    per, path = bench.algorithmic_bytes(w, k)
    LH, n = w.L * w.Hkv, w.n_tot
    q_bytes = w.L * w.Hq * w.g_tot * w.d * 2
    assert path == LH * (644 * n + 780 * k) + q_bytes
    assert abs(path / 1e9 - 24.24) < 0.01
    # step 2's launches (2/5 of the rows beside each score pass on the second stream, the rest
    # between the passes) cover every V row once
    row = 2 * w.d + w.d + 4
    assert per["k_quantize"] + 2 * per["k_quantize_lean"] == LH * n * row
    assert per["k_quantize_lean"] == (LH * n * 2 // 5 // 64 * 64) * row
    # with the normalisers given: the first half on the second stream, the rest between
    per_g, _ = bench.algorithmic_bytes(w, k, normalisers_given=True)
    assert per_g["k_quantize"] + per_g["k_quantize_lean"] == LH * n * row
    assert per_g["k_quantize_lean"] == (LH * n // 2 // 64 * 64) * row
    assert bench.LEAN_LAUNCHES == {False: 2, True: 1}
    # scales only: half beside each pass; with the normalisers given, 3/5 on the second stream
    per_s, _ = bench.algorithmic_bytes(w, k, full_codes=False)
    row_s = 2 * w.d + 4
    assert per_s["k_quantize"] + 2 * per_s["k_quantize_lean"] == LH * n * row_s
    assert per_s["k_quantize_lean"] == (LH * n // 2 // 64 * 64) * row_s
    per_gs, _ = bench.algorithmic_bytes(w, k, full_codes=False, normalisers_given=True)
    assert per_gs["k_quantize_lean"] == (LH * n * 3 // 5 // 64 * 64) * row_s


def test_path_bytes_scales_only_and_int4():
    w = W.llama8b_128k()
    k = _kept(w)
    LH, n = w.L * w.Hkv, w.n_tot
    q_bytes = w.L * w.Hq * w.g_tot * w.d * 2
    _, path = bench.algorithmic_bytes(w, k, full_codes=False)
    # scales only (516 B per token-head), the kept rows re-read in bf16 and quantised
    assert path == LH * (516 * n + k * (256 + 256 + 4 + 256 + 128 + 4)) + q_bytes
    w4 = w.with_(bits=4)
    _, path4 = bench.algorithmic_bytes(w4, k)
    assert path4 == LH * ((256 + 256 + 64 + 4) * n + k * (2 * (256 + 64 + 4) + 4)) + q_bytes


def test_kernel_source_lists_name_existing_files():
    """Every source a traffic summary is keyed on exists (a renamed file would otherwise leave
    every summary stale without notice)."""
    for kernel, names in bench.KERNEL_SOURCES.items():
        for name in names:
            assert os.path.exists(os.path.join(ROOT, "paper_2608_03276_amd", "csrc", name)), (kernel, name)


def test_attention_bytes_128k():
    """The guide rows' attention at 128K, counted by hand: K and V of the context
    (2 x 32 x 8 x 131072 x 128 x 2 B), Q (32 x 32 x 64 x 128 x 2 B) and O (x 4 B), the
    guide tokens' K and V (2 x 32 x 8 x 64 x 128 x 2 B); with step 2, int8 codes and a
    4-byte scale per context token-head."""
    w = W.llama8b_128k()
    plain = 17_179_869_184 + 16_777_216 + 33_554_432 + 8_388_608
    assert bench.attention_bytes(w, False) == plain
    assert bench.attention_bytes(w, True) == plain + 32 * 8 * 131072 * (128 + 4) == 21_667_774_464
    w4 = w.with_(bits=4)  # nibbles: 64 code bytes per row
    assert bench.attention_bytes(w4, True) == plain + 32 * 8 * 131072 * (64 + 4)
