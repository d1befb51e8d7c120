"""GPU path (through the C ABI) against the CPU oracle on the same seeded inputs.

Sizes span several tiles and ragged tails; the full-size workloads are checked on sampled
segments in test_gpu_fullsize.py.  Rules: see parity_util."""
import numpy as np
import pytest
import torch

import synth
from oracle import taskpress_oracle as o
from paper_2608_03276_amd import binding as B
from synth import workloads as W

import parity_util as pu

pytestmark = pytest.mark.gpu


def _bf16_tensor(bits: np.ndarray):
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16).cuda()


# ----------------------------------------------------------------------------- generator
def test_device_generator_matches_host(gpu_lib):
    for s, L, H, lens, d in [(synth.Stream(11, synth.TAG_K), 2, 3, [5, 300, 1], 64),
                             (synth.Stream(12, synth.TAG_V, synth.DIST_STUDENT_T3, 0.01, 30.0), 1, 2, [2000, 777], 128)]:
        pu.log(f"generator {s} L={L} H={H} lens={lens} d={d}")
        t = torch.empty(L * H * sum(lens) * d, dtype=torch.bfloat16, device="cuda")
        synth.device_fill(t.data_ptr(), s, L, H, lens, d, torch.cuda.current_stream().cuda_stream)
        torch.cuda.synchronize()
        host = synth.host_tensor(s, L, H, lens, d).reshape(-1)
        assert np.array_equal(t.view(torch.int16).cpu().numpy().view(np.uint16), host)


# ----------------------------------------------------------------------------- step 2
def _run_quant(vbits, L, Hkv, lens, d, qfmt, bits, with_vq=True):
    dd = B.dims(L, Hkv, Hkv, d)
    bt = B.Batch(np.concatenate([[0], np.cumsum(lens)]).tolist())
    v = _bf16_tensor(vbits.reshape(-1))
    n = L * Hkv * sum(lens)
    scales = torch.empty(n, dtype=torch.float32, device="cuda")
    vq = torch.empty(n * B.row_bytes(qfmt, bits, d), dtype=torch.uint8, device="cuda") if with_vq else None
    B.tp_quantize_v_scales(dd, bt, v, qfmt, bits, scales, vq)
    torch.cuda.synchronize()
    return scales.cpu().numpy(), None if vq is None else vq.cpu().numpy()


@pytest.mark.parametrize("qfmt,bits,d", [(0, 8, 128), (0, 8, 64), (0, 4, 128), (0, 4, 64), (0, 2, 128), (0, 6, 64),
                                         (1, 8, 128), (1, 8, 64)])
def test_quantize_parity(gpu_lib, qfmt, bits, d):
    pu.log(f"quantize qfmt={qfmt} bits={bits} d={d}")
    L, Hkv, lens = 2, 3, [1, 33, 1000]
    s = synth.Stream(21, synth.TAG_V, synth.DIST_STUDENT_T3, 0.02, 50.0)
    vb = synth.host_tensor(s, L, Hkv, lens, d)
    vb[0, 1, 5] = 0          # all-zero row
    vb[1, 2, 7] = 0x8000     # all -0.0 row
    vb[1, 0, 9, :3] = [0x7F7F, 0xFF7F, 0x0001]  # largest finite bf16 and a subnormal
    g, q = _run_quant(vb, L, Hkv, lens, d, qfmt, bits)
    rows = o.bf16_to_f64(vb.reshape(-1, d))
    gr = o.value_scales(rows, qfmt, bits)
    qr = o.pack_codes(o.quantize_values(rows, gr, qfmt, bits), qfmt, bits)
    assert np.array_equal(g.view(np.uint32), gr.view(np.uint32))
    assert np.array_equal(q.reshape(qr.shape), qr)
    g2, _ = _run_quant(vb, L, Hkv, lens, d, qfmt, bits, with_vq=False)
    assert np.array_equal(g2.view(np.uint32), gr.view(np.uint32))


@pytest.mark.parametrize("qfmt,bits", [(0, 8), (0, 4), (1, 8)])
def test_quantize_every_bf16_absmax(gpu_lib, qfmt, bits):
    """Every positive finite bf16 as a row's absmax, with 127 random values of smaller magnitude."""
    pu.log(f"quantize exhaustive absmax qfmt={qfmt} bits={bits}")
    rng = np.random.default_rng(31)
    amax = np.arange(1, 0x7F80, dtype=np.uint16)
    n = len(amax)
    mags = (rng.random((n, 127)) * (amax[:, None].astype(np.float64) + 1)).astype(np.uint16)
    signs = (rng.random((n, 127)) < 0.5).astype(np.uint16) << 15
    rows = np.concatenate([amax[:, None] | ((rng.random((n, 1)) < 0.5).astype(np.uint16) << 15), mags | signs], axis=1)
    for i in range(n):  # move the absmax element around
        j = i % 128
        rows[i, 0], rows[i, j] = rows[i, j], rows[i, 0]
    g, q = _run_quant(rows, 1, 1, [n], 128, qfmt, bits)
    vals = o.bf16_to_f64(rows)
    gr = o.value_scales(vals, qfmt, bits)
    qr = o.pack_codes(o.quantize_values(vals, gr, qfmt, bits), qfmt, bits)
    assert np.array_equal(g.view(np.uint32), gr.view(np.uint32))
    bad = np.nonzero(np.any(q.reshape(qr.shape) != qr, axis=1))[0]
    assert len(bad) == 0, f"{len(bad)} rows differ, first absmax bits {hex(int(amax[bad[0]]))}"


_EX_AMAX = np.arange(1, 0x7F80, dtype=np.int32)           # every positive finite bf16
_EX_PER = (_EX_AMAX + 1 + 126) // 127                      # rows per absmax and sign
_EX_END = np.cumsum(_EX_PER)                               # end row of each absmax (one sign)
_EX_ROWS = int(_EX_END[-1]) * 2


def _exhaustive_block(r0, r1):
    """Rows r0 .. r1-1 of the exhaustive table [A, v_1 .. v_127]: every (bf16 absmax A, bf16
    magnitude v <= A) pair once with each sign.  Row r of A (one sign) holds magnitudes
    127 r .. 127 r + 126, clipped to A (padding zeros); the second half repeats the table
    with the v's negated."""
    half = _EX_ROWS // 2
    idx = np.arange(r0, r1, dtype=np.int64)
    neg = idx >= half
    idx = np.where(neg, idx - half, idx)
    ai = np.searchsorted(_EX_END, idx, side="right")
    a = _EX_AMAX[ai]
    r_in_a = idx - (_EX_END[ai] - _EX_PER[ai])
    v = (r_in_a[:, None] * 127 + np.arange(127, dtype=np.int64)[None, :]).astype(np.int32)
    v = np.where(v <= a[:, None], v, 0).astype(np.uint16)
    v[neg] |= np.uint16(0x8000)
    return np.concatenate([a[:, None].astype(np.uint16), v], axis=1)


def _no_multiplier_significand(qmax):
    """A significand t (absmax 1 + t/128) that the one-multiply table marks as having no
    multiplier for this qmax, or None (read from the committed quant_recip_table.h)."""
    import os
    import re

    path = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "paper_2608_03276_amd", "csrc",
                        "quant_recip_table.h")
    text = open(path).read()
    qs = [float(x) for x in re.search(r"kRecipQmax\[\d+\] = \{([^}]*)\}", text).group(1).replace("f", "").split(",")]
    masks = re.findall(r"\{\{(0x[0-9a-f]+)ull, (0x[0-9a-f]+)ull\}, \{(0x[0-9a-f]+)ull, (0x[0-9a-f]+)ull\}, "
                       r"\{(0x[0-9a-f]+)ull, (0x[0-9a-f]+)ull\}\}", text)
    none = masks[qs.index(float(qmax))][4:6]
    for t in range(128):
        if (int(none[t >> 6], 16) >> (t & 63)) & 1:
            return t
    return None


def _with_poison_rows(rows, poison):
    """Every 4-row wave of the quantiser (d = 128) gets `poison` as its last row: rows are taken
    three at a time (the last group padded with zero rows).  Returns the new table and the
    positions of the original rows in it."""
    n = rows.shape[0]
    groups = -(-n // 3)
    out = np.zeros((groups, 4, rows.shape[1]), dtype=rows.dtype)
    flat = np.zeros((groups * 3, rows.shape[1]), dtype=rows.dtype)
    flat[:n] = rows
    out[:, :3] = flat.reshape(groups, 3, -1)
    out[:, 3] = poison
    pos = (np.arange(n) // 3) * 4 + np.arange(n) % 3
    return out.reshape(groups * 4, -1), pos


@pytest.mark.parametrize("qfmt,bits", [(0, 8), (0, 7), (0, 6), (0, 5), (0, 4), (0, 3), (0, 2), (1, 8)])
def test_quantize_every_pair(gpu_lib, qfmt, bits):
    """Every (absmax, |v| <= absmax) pair of bf16 values, both signs (about 1.07e9 values):
    codes and scales bit-exact against the oracle's definition, for every format (int2 ..
    int8 and E4M3; each has its own table of one-multiply multipliers).  The path of a row
    is chosen per wave of 4 rows, so every pair also runs in two more layouts: with an
    all-zero row in every wave (every row then takes the rescaled path), and with a row whose
    absmax significand has no one-multiply multiplier in every wave (every row of the common
    range then takes the corrected quotient; formats without such a significand skip it)."""
    qmax = 448.0 if qfmt == 1 else float(2 ** (bits - 1) - 1)
    t_none = _no_multiplier_significand(qmax)
    poisons = {"zero row": np.zeros(128, dtype=np.uint16)}
    if t_none is not None:
        p = np.zeros(128, dtype=np.uint16)
        p[0] = (127 << 7) | t_none  # absmax (1 + t/128), exponent field 127: the common range
        poisons["no-multiplier row"] = p
    pu.log(f"quantize every (absmax, v) pair, qfmt={qfmt} bits={bits}: {_EX_ROWS} rows of 128, "
           f"layouts: plain, {', '.join(poisons)}")
    rb = B.row_bytes(qfmt, bits, 128)
    for name, prow in poisons.items():  # the poison rows' own codes
        pv = o.bf16_to_f64(prow[None, :])
        pg = o.value_scales(pv, qfmt, bits)
        poisons[name] = (prow, pg, o.pack_codes(o.quantize_values(pv, pg, qfmt, bits), qfmt, bits)[0])
    group = 1 << 20
    for g0 in range(0, _EX_ROWS, group):
        rows = _exhaustive_block(g0, min(_EX_ROWS, g0 + group))
        n = rows.shape[0]
        vals = o.bf16_to_f64(rows)
        gr = o.value_scales(vals, qfmt, bits)
        qr = o.pack_codes(o.quantize_values(vals, gr, qfmt, bits), qfmt, bits)
        layouts = [("plain", rows, np.arange(n), None)]
        for name, (prow, pg, pq) in poisons.items():
            table, pos = _with_poison_rows(rows, prow)
            layouts.append((name, table, pos, (pg, pq)))
        for name, table, pos, poison in layouts:
            g, q = _run_quant(table, 1, 1, [table.shape[0]], 128, qfmt, bits)
            q = q.reshape(table.shape[0], rb)
            assert np.array_equal(g[pos].view(np.uint32), gr.view(np.uint32)), f"scales ({name}), rows {g0}+"
            bad = np.nonzero(np.any(q[pos] != qr, axis=1))[0]
            assert len(bad) == 0, (f"{name}: {len(bad)} rows differ from row {g0 + bad[0]} "
                                   f"(absmax bits {hex(int(rows[bad[0], 0]))})")
            if poison is not None:
                prow_pos = np.arange(3, table.shape[0], 4)
                assert np.all(g[prow_pos].view(np.uint32) == poison[0].view(np.uint32)[0]), name
                assert np.all(q[prow_pos] == poison[1][None, :]), name
        pu.log(f"  rows {g0} .. {g0 + n} match in every layout")


# ----------------------------------------------------------------------------- step 4
@pytest.mark.parametrize("qfmt,bits,d", [(0, 8, 128), (0, 4, 64), (1, 8, 64)])
def test_compact_parity(gpu_lib, qfmt, bits, d):
    pu.log(f"compact qfmt={qfmt} bits={bits} d={d}")
    rng = np.random.default_rng(41)
    L, Hkv, lens = 2, 2, [7, 300, 1]
    kept = [3, 41, 1]
    ntot, kt = sum(lens), sum(kept)
    rb = B.row_bytes(qfmt, bits, d)
    kb = rng.integers(0, 2 ** 16, (L * Hkv, ntot, d), dtype=np.uint16)
    vq = rng.integers(0, 256, (L * Hkv, ntot, rb), dtype=np.uint8)
    sc = rng.random((L * Hkv, ntot)).astype(np.float32)
    offs = np.concatenate([[0], np.cumsum(lens)])
    ko = np.concatenate([[0], np.cumsum(kept)])
    idx = np.zeros((L * Hkv, kt), dtype=np.int32)
    for s in range(L * Hkv):
        for b in range(len(lens)):
            idx[s, ko[b]:ko[b + 1]] = np.sort(rng.choice(lens[b], kept[b], replace=False))
    idx[1, 5] = -1            # out of range -> zero row
    idx[2, 10] = lens[1]      # out of range -> zero row
    dd = B.dims(L, Hkv, Hkv, d)
    bt = B.Batch(offs.tolist())
    k_out = torch.empty(L * Hkv * kt * d, dtype=torch.bfloat16, device="cuda")
    vq_out = torch.empty(L * Hkv * kt * rb, dtype=torch.uint8, device="cuda")
    sc_out = torch.empty(L * Hkv * kt, dtype=torch.float32, device="cuda")
    B.tp_compact_kv(dd, bt, ko.tolist(), torch.from_numpy(idx).cuda(), _bf16_tensor(kb), torch.from_numpy(vq).cuda(),
                    torch.from_numpy(sc).cuda(), qfmt, bits, k_out, vq_out, sc_out)
    torch.cuda.synchronize()
    ko_ = k_out.view(torch.int16).cpu().numpy().view(np.uint16).reshape(L * Hkv, kt, d)
    vo = vq_out.cpu().numpy().reshape(L * Hkv, kt, rb)
    so = sc_out.cpu().numpy().reshape(L * Hkv, kt)
    for s in range(L * Hkv):
        for b in range(len(lens)):
            for t in range(ko[b], ko[b + 1]):
                i = idx[s, t]
                if 0 <= i < lens[b]:
                    src = offs[b] + i
                    assert np.array_equal(ko_[s, t], kb[s, src]) and np.array_equal(vo[s, t], vq[s, src])
                    assert so[s, t] == sc[s, src]
                else:
                    assert not ko_[s, t].any() and not vo[s, t].any() and so[s, t] == 0


@pytest.mark.parametrize("qfmt,bits,d", [(0, 8, 128), (0, 4, 64), (0, 2, 128), (1, 8, 64), (1, 8, 128)])
def test_compact_quantize_parity(gpu_lib, qfmt, bits, d):
    """Quantise-while-gathering: the kept rows' codes and scales equal the oracle's
    quantisation of those rows, bit for bit; out-of-range indices give zero rows."""
    pu.log(f"compact+quantise qfmt={qfmt} bits={bits} d={d}")
    rng = np.random.default_rng(43)
    L, Hkv, lens = 2, 2, [7, 1300, 1]
    kept = [3, 401, 1]
    ntot, kt = sum(lens), sum(kept)
    rb = B.row_bytes(qfmt, bits, d)
    vb = synth.host_tensor(synth.Stream(23, synth.TAG_V, synth.DIST_STUDENT_T3, 0.02, 50.0), L, Hkv, lens, d)
    vb = vb.reshape(L * Hkv, ntot, d)
    vb[0, 8] = 0                                   # all-zero row (kept below)
    vb[1, 9, :3] = [0x7F7F, 0xFF7F, 0x0001]        # largest finite bf16 and a subnormal
    kb = rng.integers(0, 2 ** 16, (L * Hkv, ntot, d), dtype=np.uint16)
    offs = np.concatenate([[0], np.cumsum(lens)])
    ko = np.concatenate([[0], np.cumsum(kept)])
    idx = np.zeros((L * Hkv, kt), dtype=np.int32)
    for sg in range(L * Hkv):
        for b in range(len(lens)):
            pick = rng.choice(lens[b], kept[b], replace=False)
            if b == 1:
                pick[:2] = [1, 2]                  # rows 8 and 9 of the batch: the special rows
            idx[sg, ko[b]:ko[b + 1]] = np.sort(pick)
    idx[1, 5] = -1
    idx[2, 10] = lens[1]
    dd = B.dims(L, Hkv, Hkv, d)
    bt = B.Batch(offs.tolist())
    k_out = torch.empty(L * Hkv * kt * d, dtype=torch.bfloat16, device="cuda")
    vq_out = torch.empty(L * Hkv * kt * rb, dtype=torch.uint8, device="cuda")
    sc_out = torch.empty(L * Hkv * kt, dtype=torch.float32, device="cuda")
    B.tp_compact_quantize_kv(dd, bt, ko.tolist(), torch.from_numpy(idx).cuda(), _bf16_tensor(kb), _bf16_tensor(vb),
                             qfmt, bits, k_out, vq_out, sc_out)
    torch.cuda.synchronize()
    ko_ = k_out.view(torch.int16).cpu().numpy().view(np.uint16).reshape(L * Hkv, kt, d)
    vo = vq_out.cpu().numpy().reshape(L * Hkv, kt, rb)
    so = sc_out.cpu().numpy().reshape(L * Hkv, kt)
    rows = o.bf16_to_f64(vb.reshape(-1, d))
    gr = o.value_scales(rows, qfmt, bits).reshape(L * Hkv, ntot)
    qr = o.pack_codes(o.quantize_values(rows, gr.reshape(-1), qfmt, bits), qfmt, bits).reshape(L * Hkv, ntot, rb)
    for sg in range(L * Hkv):
        for b in range(len(lens)):
            for t in range(ko[b], ko[b + 1]):
                i = idx[sg, t]
                if 0 <= i < lens[b]:
                    src = offs[b] + i
                    assert np.array_equal(ko_[sg, t], kb[sg, src])
                    assert np.array_equal(vo[sg, t], qr[sg, src]), (sg, t)
                    assert so[sg, t].view(np.uint32) == gr[sg, src].view(np.uint32)
                else:
                    assert not ko_[sg, t].any() and not vo[sg, t].any() and so[sg, t] == 0


# ----------------------------------------------------------------------------- step 3
def _select_inputs(rng, L, Hkv, lens, tie_levels):
    n = L * Hkv * sum(lens)
    if tie_levels:
        sk = (rng.integers(0, tie_levels, n).astype(np.float32) * np.float32(0.125)).astype(np.float32)
        g = (rng.integers(1, 4, n).astype(np.float32) * np.float32(0.5)).astype(np.float32)
    else:
        sk = (rng.random(n) * 10.0 ** rng.integers(-30, 1, n)).astype(np.float32)
        g = (rng.random(n) * 10.0 ** rng.integers(-3, 1, n)).astype(np.float32)
    return sk, g


@pytest.mark.parametrize("rule", [0, 1, 2, 3])
@pytest.mark.parametrize("ties", [0, 5])
def test_select_parity(gpu_lib, rule, ties):
    pu.log(f"select rule={rule} ties={ties}")
    rng = np.random.default_rng(51 + rule + ties)
    L, Hkv, lens = 2, 3, [1, 5, 1000, 4099, 70000]
    for ratio, budget in [(0.1, 0), (1.0, 0), (0.0, 100), (0.0, 1)]:
        sk, g = _select_inputs(rng, L, Hkv, lens, ties)
        dd = B.dims(L, Hkv, Hkv, 64)
        bt = B.Batch(np.concatenate([[0], np.cumsum(lens)]).tolist())
        ko = B.kept_offsets_for(bt, ratio, budget)
        kt = ko[-1]
        kept = torch.empty(L * Hkv * kt, dtype=torch.int32, device="cuda")
        s_out = torch.empty(L * Hkv * sum(lens), dtype=torch.float32, device="cuda")
        B.tp_combine_select_topk(dd, bt, torch.from_numpy(sk).cuda(), torch.from_numpy(g).cuda(), rule, ratio,
                                 budget, ko, kept, s_out)
        torch.cuda.synchronize()
        kept_h = kept.cpu().numpy().reshape(L * Hkv, kt)
        S_h = s_out.cpu().numpy().reshape(L * Hkv, -1)
        skr, gr = sk.reshape(L * Hkv, -1), g.reshape(L * Hkv, -1)
        offs = bt.ctx_offsets
        for s in range(L * Hkv):
            for b in range(len(lens)):
                a, e = offs[b], offs[b + 1]
                S_ref = o.combine(skr[s, a:e], gr[s, a:e], rule)
                k = o.keep_count(lens[b], ratio or None, budget or None)
                got = kept_h[s, ko[b]:ko[b + 1]]
                tag = f"rule={rule} seg={s} b={b}"
                if rule == o.COMBINE_NORM_ADD:  # norms are sums in a different order: tolerance rules
                    pu.assert_scores_close(S_h[s, a:e], S_ref.astype(np.float64), tag)
                    pu.assert_keep_set(got, S_ref, k, tag)
                    pu.assert_topk_of_own_scores(got, S_h[s, a:e], tag)
                else:  # identical fp32 inputs: bit-exact
                    assert np.array_equal(S_h[s, a:e].view(np.uint32), S_ref.view(np.uint32)), tag
                    assert np.array_equal(got, o.select(S_ref, k)), tag


def test_select_all_equal_and_zero(gpu_lib):
    for val in [0.0, 1.5]:
        n = 5000
        sk = np.full(n, val, np.float32)
        g = np.ones(n, np.float32)
        dd = B.dims(1, 1, 1, 64)
        bt = B.Batch([0, n])
        ko = B.kept_offsets_for(bt, 0.3, 0)
        kept = torch.empty(ko[-1], dtype=torch.int32, device="cuda")
        B.tp_combine_select_topk(dd, bt, torch.from_numpy(sk).cuda(), torch.from_numpy(g).cuda(), 0, 0.3, 0, ko,
                                 kept, torch.empty(n, dtype=torch.float32, device="cuda"))
        torch.cuda.synchronize()
        assert np.array_equal(kept.cpu().numpy(), np.arange(ko[-1]))


def test_select_large_threshold_bucket(gpu_lib):
    """Keys of the threshold's top digit too many for the LDS candidate buffer (> 16384): the
    remaining digits are ranked from memory; also a bucket that just fits."""
    rng = np.random.default_rng(53)
    for n, levels in [(70000, 2), (40000, 3), (200000, 7)]:
        sk = (rng.integers(1, levels + 1, n).astype(np.float32) * np.float32(0.25)).astype(np.float32)
        sk[rng.integers(0, n, 50)] += np.float32(1e-3)   # a few distinct keys inside the buckets
        g = np.ones(n, np.float32)
        dd = B.dims(1, 1, 1, 64)
        bt = B.Batch([0, n])
        for ratio in (0.3, 0.61, 1.0):
            ko = B.kept_offsets_for(bt, ratio, 0)
            kept = torch.empty(ko[-1], dtype=torch.int32, device="cuda")
            B.tp_combine_select_topk(dd, bt, torch.from_numpy(sk).cuda(), torch.from_numpy(g).cuda(), 0, ratio, 0, ko,
                                     kept, torch.empty(n, dtype=torch.float32, device="cuda"))
            torch.cuda.synchronize()
            S = o.combine(sk, g, 0)
            assert np.array_equal(kept.cpu().numpy(), o.select(S, ko[-1])), (n, levels, ratio)


# ----------------------------------------------------------------------------- step 1
GUIDE_CASES = [
    # (name, L, Hq, Hkv, d, lens, glens, k-dist, pool)
    ("tiny-like", 1, 8, 2, 64, [1024], [16], synth.DIST_NORMAL, 5),
    ("ragged-d128", 2, 8, 2, 128, [1, 31, 32, 33, 2047, 2048, 2049, 5000], [1, 3, 64, 64, 100, 7, 64, 128],
     synth.DIST_NORMAL, 5),
    ("two-row-groups", 1, 16, 2, 128, [3000, 700], [40, 33], synth.DIST_NORMAL, 3),
    ("mha-g1-pool1", 1, 4, 4, 64, [777], [1], synth.DIST_NORMAL, 1),
    ("heavy-tail-outliers", 1, 8, 2, 128, [4500], [64], synth.DIST_STUDENT_T3, 7),
    ("pool-wider-than-seq", 1, 2, 1, 64, [1, 2, 3], [2, 1, 5], synth.DIST_NORMAL, 9),
    ("chunk-edges", 1, 8, 2, 128, [8191, 8192, 8193, 16385], [64, 9, 64, 33], synth.DIST_NORMAL, 5),
    ("wide-pool-staged", 1, 2, 1, 64, [2500, 40], [4, 2], synth.DIST_NORMAL, 1025),
    ("wide-pool-direct", 1, 2, 1, 64, [3000], [4], synth.DIST_NORMAL, 1027),
    # one launch per row-block class: 64, 128, 192 and 320 (= 256 + 64) guide rows
    ("row-classes", 2, 8, 2, 128, [9000, 1500, 20000, 4097], [16, 32, 48, 80], synth.DIST_NORMAL, 5),
    # rare keys scaled x100: their logits jump far above every row's running maximum in the
    # middle of a chunk, so pass 1 takes its exact re-update of the unit there
    ("extreme-outliers", 1, 8, 2, 128, [12000, 3000], [64, 16], synth.DIST_NORMAL, 5),
]
# (fraction, scale) of outlier key rows per case
GUIDE_OUTLIERS = {"heavy-tail-outliers": (0.02, 30.0), "extreme-outliers": (0.003, 100.0)}


def _guide_case(case, guide_keys):
    name, L, Hq, Hkv, d, lens, glens, dist, pool = case
    pu.log(f"guide scores case {name}{' with guide keys' if guide_keys else ''}")
    out_frac, out_scale = GUIDE_OUTLIERS.get(name, (0.0, 1.0))
    w = W.Workload(name, L, Hq, Hkv, d, tuple(lens), tuple(glens), synth.Stream(61, synth.TAG_Q),
                   synth.Stream(61, synth.TAG_K, dist, out_frac, out_scale), synth.Stream(61, synth.TAG_V),
                   keep_ratio=0.25, pool_k=pool)
    q, k, v = pu.device_inputs(w)
    kg = pu.device_guide_keys(w) if guide_keys else None
    dd = B.dims(L, Hq, Hkv, d)
    bt = B.Batch(w.ctx_offsets(), w.guide_offsets())
    s_key = torch.empty(L * Hkv * w.n_tot, dtype=torch.float32, device="cuda")
    ws = torch.empty(B.tp_workspace_size(B.TP_FN_GUIDE_SCORES, dd, bt), dtype=torch.uint8, device="cuda")
    B.tp_guide_scores(dd, bt, q, k, w.softmax_scale, pool, s_key, ws, k_guide=kg)
    torch.cuda.synchronize()
    got = s_key.cpu().numpy().reshape(L * Hkv, w.n_tot)
    offs = w.ctx_offsets()
    worst = 0.0
    for b in range(w.batch):
        for l in range(L):
            for h in range(Hkv):
                qg, kb, _ = pu.host_segment(w, b, l, h)
                kgr = o.bf16_to_f64(pu.host_guide_keys(w, b, l, h)) if guide_keys else None
                ref = o.key_scores(o.bf16_to_f64(qg), o.bf16_to_f64(kb), w.softmax_scale, pool, kgr)
                worst = max(worst, pu.assert_scores_close(got[l * Hkv + h, offs[b]:offs[b + 1]], ref,
                                                          f"{name} b={b} l={l} h={h}"))
    pu.log(f"  max rel err {worst:.3g}")


@pytest.mark.parametrize("case", GUIDE_CASES, ids=[c[0] for c in GUIDE_CASES])
def test_guide_scores_parity(gpu_lib, case):
    _guide_case(case, False)


@pytest.mark.parametrize("case", GUIDE_CASES[:5], ids=[c[0] for c in GUIDE_CASES[:5]])
def test_guide_scores_with_guide_keys(gpu_lib, case):
    """The paper-literal normaliser (guide keys 0..j of the appended guide included)."""
    _guide_case(case, True)


def _guide_lse_case(case, jitter_seed):
    name, L, Hq, Hkv, d, lens, glens, dist, pool = case
    pu.log(f"guide scores with supplied normalisers, case {name}, jitter {jitter_seed}")
    out_frac, out_scale = GUIDE_OUTLIERS.get(name, (0.0, 1.0))
    w = W.Workload(name, L, Hq, Hkv, d, tuple(lens), tuple(glens), synth.Stream(67, synth.TAG_Q),
                   synth.Stream(67, synth.TAG_K, dist, out_frac, out_scale), synth.Stream(67, synth.TAG_V),
                   keep_ratio=0.25, pool_k=pool)
    q, k, _ = pu.device_inputs(w)
    lse = pu.oracle_guide_lse(w, jitter_seed=jitter_seed)
    dd = B.dims(L, Hq, Hkv, d)
    bt = B.Batch(w.ctx_offsets(), w.guide_offsets())
    s_key = torch.empty(L * Hkv * w.n_tot, dtype=torch.float32, device="cuda")
    ws = torch.empty(B.tp_workspace_size(B.TP_FN_GUIDE_SCORES, dd, bt), dtype=torch.uint8, device="cuda")
    B.tp_guide_scores_lse(dd, bt, q, k, torch.from_numpy(lse.ravel()).cuda(), w.softmax_scale, pool, s_key, ws)
    torch.cuda.synchronize()
    got = s_key.cpu().numpy().reshape(L * Hkv, w.n_tot)
    offs, goff = w.ctx_offsets(), w.guide_offsets()
    worst = 0.0
    for b in range(w.batch):
        for l in range(L):
            for h in range(Hkv):
                qg, kb, _ = pu.host_segment(w, b, l, h)
                rows = lse[l, h * w.R:(h + 1) * w.R, goff[b]:goff[b + 1]].astype(np.float64)
                ref = o.key_scores_given_lse(o.bf16_to_f64(qg), o.bf16_to_f64(kb), w.softmax_scale, pool, rows)
                worst = max(worst, pu.assert_scores_close(got[l * Hkv + h, offs[b]:offs[b + 1]], ref,
                                                          f"{name} b={b} l={l} h={h}"))
    pu.log(f"  max rel err {worst:.3g}")


LSE_CASES = GUIDE_CASES[:5] + [GUIDE_CASES[-2]]


@pytest.mark.parametrize("jitter", [None, 5])
@pytest.mark.parametrize("case", LSE_CASES, ids=[c[0] for c in LSE_CASES])
def test_guide_scores_lse_parity(gpu_lib, case, jitter):
    """Step 1 with the normalisers supplied (as a prefill kernel exports them), exact and
    shifted per row."""
    _guide_lse_case(case, jitter)


# ----------------------------------------------------------------------------- whole path
@pytest.mark.parametrize("rule", [0, 3])
@pytest.mark.parametrize("fused", [False, True])
def test_end_to_end_tiny(gpu_lib, rule, fused):
    """Every rule against the oracle, through the four calls and through tp_evict (which pools
    inside the selection for every rule but NORM_ADD)."""
    w = W.tiny()
    pu.log(f"end-to-end {w.describe()} rule={rule} fused={fused}")
    q, k, v = pu.device_inputs(w)
    bufs = pu.run_gpu(w, q, k, v, rule=rule, fused=fused)
    for l in range(w.L):
        for h in range(w.Hkv):
            pu.check_segment(w, bufs, 0, l, h, rule=rule)


def test_end_to_end_ragged_int4_fp8(gpu_lib):
    base = W.ragged8()
    for qfmt, bits in [(0, 4), (1, 8)]:
        w = base.with_(name=f"ragged-small-{qfmt}-{bits}", L=2, ctx_lens=(3000, 1, 4097, 800),
                       guide_lens=(32, 128, 5, 64), keep_budget=700, qfmt=qfmt, bits=bits)
        pu.log(f"end-to-end {w.describe()}")
        q, k, v = pu.device_inputs(w)
        bufs = pu.run_gpu(w, q, k, v)
        for b in range(w.batch):
            for l in range(w.L):
                for h in (0, w.Hkv - 1):
                    pu.check_segment(w, bufs, b, l, h)


def test_deterministic(gpu_lib):
    w = W.llama8b_32k().with_(name="det", L=2, ctx_lens=(9000, 5001), guide_lens=(64, 17))
    q, k, v = pu.device_inputs(w)
    a = pu.run_gpu(w, q, k, v)
    snap = {n: getattr(a, n).clone() for n in ("s_key", "scales", "v_q", "s_comb", "kept_idx", "k_c", "v_q_c",
                                               "scales_c")}
    b = pu.run_gpu(w, q, k, v)
    for n, t in snap.items():
        assert torch.equal(t.view(torch.uint8), getattr(b, n).view(torch.uint8)), n


# ----------------------------------------------------------------------------- fused entry point
def _fused_vs_calls(w, with_events=False):
    d = B.dims(w.L, w.Hq, w.Hkv, w.d)
    bt = B.Batch(w.ctx_offsets(), w.guide_offsets())
    q, k, v = pu.device_inputs(w)
    sep = pu.run_gpu(w, q, k, v)
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(B.TP_EVICT_EVENTS)] if with_events else None
    fused = B.evict_fused(d, bt, q, k, v, softmax_scale=w.softmax_scale, pool_k=w.pool_k, qfmt=w.qfmt, bits=w.bits,
                          rule=w.rule, keep_ratio=w.keep_ratio or 0.0, keep_budget=w.keep_budget or 0, events=ev)
    torch.cuda.synchronize()
    for n in ("s_key", "scales", "v_q", "s_comb", "kept_idx", "k_c", "v_q_c", "scales_c"):
        assert torch.equal(getattr(sep, n).view(torch.uint8), getattr(fused, n).view(torch.uint8)), (w.name, n)
    return fused, ev


def test_evict_matches_the_four_calls(gpu_lib):
    """tp_evict gives bit-identical outputs to the separate calls."""
    for w in (W.tiny(),
              W.tiny().with_(name="tiny-d128-ragged-int4", d=128, ctx_lens=(1000, 33, 4200), guide_lens=(16, 3, 90),
                             bits=4, keep_ratio=None, keep_budget=100),
              W.ragged8().with_(name="ragged-fp8", L=2, ctx_lens=(9000, 1, 8193), guide_lens=(32, 128, 7),
                                keep_budget=500, qfmt=1),
              W.llama8b_32k().with_(name="two-row-groups", L=1, ctx_lens=(5000,), guide_lens=(100,)),
              # fewer than 192 V rows (the second stream's parts are empty), and a middle part
              # that is not a whole number of 64-row groups
              W.tiny().with_(name="tiny-61-rows", Hq=2, Hkv=1, ctx_lens=(1, 60), guide_lens=(3, 2)),
              W.tiny().with_(name="tiny-401-rows", Hq=4, Hkv=1, ctx_lens=(333, 68), guide_lens=(5, 7)),
              # the pooling fused into the selection: staged windows of the widest staged
              # half-width (512) and wider ones summed directly, a window wider than the
              # sequence, and sequences of several 32768-token parts of the selection
              W.tiny().with_(name="wide-pool-staged", ctx_lens=(2500, 40, 3), guide_lens=(4, 2, 9), pool_k=1025),
              W.tiny().with_(name="wide-pool-direct", ctx_lens=(3000, 2), guide_lens=(4, 6), pool_k=1027),
              W.tiny().with_(name="three-parts", ctx_lens=(70001, 5, 32768), guide_lens=(8, 3, 20), keep_ratio=0.3)):
        pu.log(f"tp_evict vs four calls: {w.describe()}")
        _fused_vs_calls(w)


def test_evict_against_oracle(gpu_lib):
    w = W.tiny().with_(name="tiny-evict", ctx_lens=(700, 1500), guide_lens=(9, 16), keep_ratio=0.3)
    d = B.dims(w.L, w.Hq, w.Hkv, w.d)
    bt = B.Batch(w.ctx_offsets(), w.guide_offsets())
    q, k, v = pu.device_inputs(w)
    bufs = B.evict_fused(d, bt, q, k, v, softmax_scale=w.softmax_scale, pool_k=w.pool_k, qfmt=w.qfmt, bits=w.bits,
                         rule=w.rule, keep_ratio=w.keep_ratio)
    torch.cuda.synchronize()
    for b in range(w.batch):
        for h in range(w.Hkv):
            pu.check_segment(w, bufs, b, 0, h)


def test_evict_with_guide_keys_against_oracle(gpu_lib):
    w = W.ragged8().with_(name="ragged-guide-keys", L=2, ctx_lens=(3000, 1, 700), guide_lens=(32, 5, 128),
                          keep_budget=300)
    d = B.dims(w.L, w.Hq, w.Hkv, w.d)
    bt = B.Batch(w.ctx_offsets(), w.guide_offsets())
    q, k, v = pu.device_inputs(w)
    kg = pu.device_guide_keys(w)
    bufs = B.evict_fused(d, bt, q, k, v, softmax_scale=w.softmax_scale, pool_k=w.pool_k, qfmt=w.qfmt, bits=w.bits,
                         rule=w.rule, keep_budget=w.keep_budget, k_guide=kg)
    torch.cuda.synchronize()
    for b in range(w.batch):
        for l in range(w.L):
            for h in (0, w.Hkv - 1):
                pu.check_segment(w, bufs, b, l, h, guide_keys=True)
    # the guide keys change the scores (the context mass of a row drops below 1)
    plain = pu.run_gpu(w, q, k, v)
    assert not torch.equal(plain.s_key, bufs.s_key)


def test_evict_with_supplied_normalisers_against_oracle(gpu_lib):
    """tp_evict given the guide rows' log-normalisers of the paper-literal map (context plus
    causal guide keys, as the prefill kernel would export them): same results as the oracle's
    guide-key path, and as tp_evict computing them itself from the guide keys."""
    w = W.ragged8().with_(name="ragged-lse", L=2, ctx_lens=(3000, 1, 700), guide_lens=(32, 5, 128),
                          keep_budget=300)
    d = B.dims(w.L, w.Hq, w.Hkv, w.d)
    bt = B.Batch(w.ctx_offsets(), w.guide_offsets())
    q, k, v = pu.device_inputs(w)
    lse = torch.from_numpy(pu.oracle_guide_lse(w, guide_keys=True).ravel()).cuda()
    bufs = B.evict_fused(d, bt, q, k, v, softmax_scale=w.softmax_scale, pool_k=w.pool_k, qfmt=w.qfmt, bits=w.bits,
                         rule=w.rule, keep_budget=w.keep_budget, guide_lse=lse)
    torch.cuda.synchronize()
    for b in range(w.batch):
        for l in range(w.L):
            for h in (0, w.Hkv - 1):
                pu.check_segment(w, bufs, b, l, h, guide_keys=True)
    kg = pu.device_guide_keys(w)
    own = B.evict_fused(d, bt, q, k, v, softmax_scale=w.softmax_scale, pool_k=w.pool_k, qfmt=w.qfmt, bits=w.bits,
                        rule=w.rule, keep_budget=w.keep_budget, k_guide=kg)
    torch.cuda.synchronize()
    pu.assert_scores_close(bufs.s_key.cpu().numpy(), own.s_key.cpu().numpy().astype(np.float64), "lse vs k_guide")


def test_evict_graph_capture(gpu_lib):
    """tp_evict captured into a graph (its second stream forks from and joins the capturing
    stream) and replayed several times, with eager work and synchronisations between the
    replays: every replay gives the eager outputs bit for bit."""
    w = W.ragged8().with_(name="graph-replay", L=2, ctx_lens=(3000, 1, 4097), guide_lens=(32, 5, 64),
                          keep_budget=300)
    pu.log(f"tp_evict graph capture and replay: {w.describe()}")
    q, k, v = pu.device_inputs(w)
    d = B.dims(w.L, w.Hq, w.Hkv, w.d)
    bt = B.Batch(w.ctx_offsets(), w.guide_offsets())
    kw = dict(softmax_scale=w.softmax_scale, pool_k=w.pool_k, qfmt=w.qfmt, bits=w.bits, rule=w.rule,
              keep_ratio=w.keep_ratio or 0.0, keep_budget=w.keep_budget or 0)
    eager = B.evict_fused(d, bt, q, k, v, **kw)  # also the first call on the device (outside capture)
    torch.cuda.synchronize()
    names = ("s_key", "scales", "v_q", "s_comb", "kept_idx", "k_c", "v_q_c", "scales_c")
    ref = {n: getattr(eager, n).clone() for n in names}
    ko = B.kept_offsets_for(bt, kw["keep_ratio"], kw["keep_budget"])
    bufs = B.EvictBuffers(d, bt, w.qfmt, w.bits, ko)
    graph = torch.cuda.CUDAGraph()
    cap = torch.cuda.Stream()
    cap.wait_stream(torch.cuda.current_stream())
    with torch.cuda.graph(graph, stream=cap):
        B.evict_fused(d, bt, q, k, v, bufs=bufs, **kw)
    torch.cuda.synchronize()
    for rep in range(3):
        for n in names:  # eager work between the replays
            getattr(bufs, n).zero_()
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        for n in names:
            assert torch.equal(getattr(bufs, n), ref[n]), (rep, n)
        pu.log(f"  replay {rep} matches the eager call")


def test_evict_concurrent_threads(gpu_lib):
    """Two host threads calling tp_evict at the same time, each on its own stream with its
    own buffers (the calls share the device's second stream and events, whose use is
    serialised by a lock while enqueueing): every result equals the serial call's."""
    import threading

    w = W.ragged8().with_(name="threads", L=2, ctx_lens=(3000, 1, 4097), guide_lens=(32, 5, 64), keep_budget=300)
    pu.log(f"tp_evict from two threads: {w.describe()}")
    q, k, v = pu.device_inputs(w)
    d = B.dims(w.L, w.Hq, w.Hkv, w.d)
    bt = B.Batch(w.ctx_offsets(), w.guide_offsets())
    kw = dict(softmax_scale=w.softmax_scale, pool_k=w.pool_k, qfmt=w.qfmt, bits=w.bits, rule=w.rule,
              keep_ratio=w.keep_ratio or 0.0, keep_budget=w.keep_budget or 0)
    names = ("s_key", "scales", "v_q", "s_comb", "kept_idx", "k_c", "v_q_c", "scales_c")
    ref = B.evict_fused(d, bt, q, k, v, **kw)
    torch.cuda.synchronize()
    ko = B.kept_offsets_for(bt, kw["keep_ratio"], kw["keep_budget"])
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    bufs = [B.EvictBuffers(d, bt, w.qfmt, w.bits, ko) for _ in streams]
    for st in streams:
        st.wait_stream(torch.cuda.current_stream())
    errors = []

    def worker(i):
        try:
            for _ in range(5):
                B.evict_fused(d, bt, q, k, v, bufs=bufs[i], stream=streams[i], **kw)
            streams[i].synchronize()
        except Exception as e:  # reported below
            errors.append(e)

    threads = [threading.Thread(target=worker, args=(i,)) for i in range(2)]
    for t in threads:
        t.start()
    for t in threads:
        t.join()
    assert not errors, errors
    torch.cuda.synchronize()
    for i in range(2):
        for n in names:
            assert torch.equal(getattr(bufs[i], n), getattr(ref, n)), (i, n)


def test_evict_without_full_codes(gpu_lib):
    """tp_evict with v_q = NULL (the kept rows are quantised during the compaction): the
    compact cache, kept set and scores are bit-identical to the run that writes every code,
    with the normalisers computed and with them supplied (each mode splits step 2 between the
    two streams differently)."""
    for w in (W.tiny().with_(name="tiny-int4", bits=4),
              W.ragged8().with_(name="ragged-fp8-nocodes", L=2, ctx_lens=(9000, 1, 8193), guide_lens=(32, 128, 7),
                                keep_budget=500, qfmt=1)):
        d = B.dims(w.L, w.Hq, w.Hkv, w.d)
        bt = B.Batch(w.ctx_offsets(), w.guide_offsets())
        q, k, v = pu.device_inputs(w)
        kw = dict(softmax_scale=w.softmax_scale, pool_k=w.pool_k, qfmt=w.qfmt, bits=w.bits, rule=w.rule,
                  keep_ratio=w.keep_ratio or 0.0, keep_budget=w.keep_budget or 0)
        lse = torch.from_numpy(pu.oracle_guide_lse(w).ravel()).cuda()
        for given in (None, lse):
            pu.log(f"tp_evict without the full code tensor{' (normalisers given)' if given is not None else ''}: "
                   f"{w.describe()}")
            full = B.evict_fused(d, bt, q, k, v, guide_lse=given, **kw)
            lean = B.evict_fused(d, bt, q, k, v, full_codes=False, guide_lse=given, **kw)
            torch.cuda.synchronize()
            for n in ("s_key", "scales", "s_comb", "kept_idx", "k_c", "v_q_c", "scales_c"):
                assert torch.equal(getattr(full, n).view(torch.uint8), getattr(lean, n).view(torch.uint8)), \
                    (w.name, given is not None, n)


def test_evict_profile_events(gpu_lib):
    w = W.llama8b_32k().with_(name="events", L=2, ctx_lens=(20000,), guide_lens=(64,))
    _, ev = _fused_vs_calls(w, with_events=True)
    stages = [ev[i].elapsed_time(ev[i + 1]) for i in range(B.TP_EVICT_EVENTS - 1)]
    assert all(t >= 0 for t in stages), stages
    assert stages[0] > 0 and stages[2] > 0 and stages[4] > 0, stages
    total = ev[0].elapsed_time(ev[-1])
    assert abs(sum(stages) - total) <= 1e-3 * total + 0.05, (stages, total)
