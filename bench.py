"""Throughput of the task-guided prefill-time eviction path on one MI355X.

A step is one pass of the whole path (guide scores, V scales + quantisation, combine +
top-k, compaction) over the workload, with inputs resident in HBM: one tp_evict call,
whose kernels are timed by events the library records between them.  Prints one JSON line.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload llama8b_128k]
"""
from __future__ import annotations

import argparse
import json
import os
import statistics
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "context tokens compressed/sec (all layers+heads); achieved HBM GB/s vs peak"
HBM_PEAK_GBS = 8000.0
MFMA_BF16_PEAK_TFLOPS = 2500.0  # MI355X dense bf16 matrix peak
FLUSH_BYTES = 512 << 20         # device write between timed steps (larger than every cache)

# The kernels of one tp_evict call, in launch order (the library records an event after each):
# with the product rule the pooling is part of the selection's first kernel (k_sel_score, which
# forms the combined scores) and "k_select" is the rest of the selection (four launches).
STAGES = ["k_guide_stats", "k_guide_lse", "k_quantize", "k_guide_attn", "k_sel_score", "k_select", "k_compact"]
KERNEL_SOURCES = {"k_guide_stats": ["guide_scores.hip", "tile_common.h", "tp_internal.h"],
                  "k_guide_lse": ["guide_scores.hip", "tile_common.h", "tp_internal.h"],
                  "k_guide_attn": ["guide_scores.hip", "tile_common.h", "tp_internal.h"],
                  "k_guide_pool": ["guide_scores.hip", "tile_common.h", "tp_internal.h"],
                  "k_guide_fwd": ["guide_attention.hip", "tile_common.h", "quant_row.h", "quant_recip_table.h",
                                  "tp_internal.h"],
                  # the rows each step-2 launch takes are set by tp_evict
                  "k_quantize": ["quantize.hip", "quant_row.h", "quant_recip_table.h", "tp_internal.h", "abi.cpp"],
                  "k_quantize_lean": ["quantize.hip", "quant_row.h", "quant_recip_table.h", "tp_internal.h", "abi.cpp"],
                  "k_sel_score": ["select.hip", "tp_internal.h", "abi.cpp"],
                  "k_select": ["select.hip", "tp_internal.h", "abi.cpp"],
                  "k_compact": ["compact.hip", "tp_internal.h"],
                  "k_compact_quant": ["compact.hip", "quant_row.h", "quant_recip_table.h", "tp_internal.h"],
                  "k_lse_import": ["guide_scores.hip", "tile_common.h", "tp_internal.h"]}


def algorithmic_bytes(w, kept_total_per_head, full_codes=True, normalisers_given=False):
    """Compulsory HBM bytes of each kernel launch of the step and of the whole path (see the
    design notes).  A kernel's bytes are what it must move itself; the path counts K once.
    Without full codes step 2 writes the scales only and the compaction re-reads the kept V
    rows.  Every kernel is launched once per step except k_quantize_lean (LEAN_LAUNCHES)."""
    from paper_2608_03276_amd import binding as B

    LH = w.L * w.Hkv
    n = w.n_tot
    d = w.d
    rb = B.row_bytes(w.qfmt, w.bits, d)
    kt = kept_total_per_head
    q_bytes = w.L * w.Hq * w.g_tot * d * 2
    rows = w.L * w.Hq * w.g_tot
    chunk = 16384 if min(w.ctx_lens) >= 65536 else 8192  # the score passes' chunk (tp_internal.h)
    nch = -(-max(w.ctx_lens) // chunk)
    per = {
        "k_guide_stats": LH * n * 2 * d + q_bytes + rows * nch * 8,     # read K, write chunk stats
        "k_guide_lse": rows * (nch * 8 + 4),                            # merge chunk stats
        "k_lse_import": rows * 8,                                       # supplied normalisers -> log2
        "k_guide_attn": LH * n * (2 * d + 4) + q_bytes,                 # read K, write raw
        "k_guide_pool": LH * n * (4 + 4),                               # read raw, write s_key
        "k_quantize": LH * n * (2 * d + rb + 4),                        # read V, write codes and scales
        "k_sel_score": LH * n * (4 + 4 + 4 + 4),                        # read raw, scales; write s_key, S
        "k_select": LH * (n * 4 + kt * 4),                              # read S once more, write kept idx
        "k_compact": LH * kt * (2 * (2 * d + rb + 4) + 4),              # read kept rows + idx, write them
        "k_compact_quant": LH * kt * (2 * d + 2 * d + 4 + 2 * d + rb + 4),  # read kept K, V, idx; write
    }
    path = LH * (n * (2 * d + 2 * d + rb + 4) + kt * (2 * d + rb + 4 + 2 * d + rb + 4 + 4)) + q_bytes
    if not full_codes:
        per["k_quantize"] = LH * n * (2 * d + 4)                        # read V, write scales
        path = LH * (n * (2 * d + 2 * d + 4) + kt * (2 * d + 2 * d + 4 + 2 * d + rb + 4)) + q_bytes
    # tp_evict quantises a part of the V rows (rounded down to 64 rows) on its second stream
    # beside each score pass (two k_quantize_lean launches), or, with the normalisers given,
    # one part beside the rest of the step (one launch); the k_quantize launch timed between
    # the events does the rest.  LEAN_PART gives the part as a fraction of the rows.
    rows = LH * n
    full = per["k_quantize"]
    num, den = LEAN_PART[(normalisers_given, full_codes)]
    r_lean = rows * num // den // 64 * 64
    launches = LEAN_LAUNCHES[normalisers_given]
    per["k_quantize"] = full * (rows - launches * r_lean) // rows
    per["k_quantize_lean"] = full * r_lean // rows
    return per, path


def attention_bytes(w, with_step2: bool) -> int:
    """Compulsory HBM bytes of the guide rows' attention (k_guide_fwd and its merge): K and V
    of the context and the guide tokens and Q read, O written (the normalisers are a rounding
    error), plus, with step 2 inside it, every context token's V codes and scale written."""
    from paper_2608_03276_amd import binding as B

    LH = w.L * w.Hkv
    b = (2 * LH * w.n_tot * w.d * 2 + w.L * w.Hq * w.g_tot * w.d * (2 + 4) + 2 * LH * w.g_tot * w.d * 2)
    if with_step2:
        b += LH * w.n_tot * (B.row_bytes(w.qfmt, w.bits, w.d) + 4)
    return b


# k_quantize_lean launches per tp_evict call, without / with the normalisers given, and the
# rows of each launch as a fraction of all rows, by (normalisers given, full codes)
LEAN_LAUNCHES = {False: 2, True: 1}
LEAN_PART = {(False, True): (2, 5), (False, False): (1, 2), (True, True): (1, 2), (True, False): (3, 5)}


def source_sha256(kernel: str) -> str:
    import hashlib

    h = hashlib.sha256()
    for name in KERNEL_SOURCES[kernel]:
        path = os.path.join(ROOT, "paper_2608_03276_amd", "csrc", name)
        if not os.path.exists(path):  # a listed source that is gone: no summary can match
            return "missing:" + name
        with open(path, "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def measured_traffic(kernel: str, workload: str):
    """HBM bytes per launch from the committed counter summary of this kernel and workload, or
    None when there is none or the kernel source has changed since the counters were taken."""
    path = os.path.join(ROOT, "profiles", f"{kernel}_{workload}_traffic.md")
    if not os.path.exists(path):
        return None
    kv = {}
    with open(path) as f:
        for line in f:
            if line.startswith("- ") and ": " in line:
                key, val = line[2:].split(": ", 1)
                kv[key.strip()] = val.strip().strip("`")
    if kv.get("source_sha256") != source_sha256(kernel):
        return None
    return int(kv["hbm_bytes_per_launch"])


def copy_calibration(gib: float = 1.0, reps: int = 3):
    """A plain device copy of known size, for scaling the FETCH_SIZE / WRITE_SIZE counters."""
    import torch

    n = int(gib * (1 << 30))
    src = torch.empty(n, dtype=torch.uint8, device="cuda").fill_(1)
    dst = torch.empty_like(src)
    for _ in range(reps):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_bytes_read": n, "copy_bytes_written": n, "reps": reps}), flush=True)


def _oracle_rate(w, seconds: float, seed: int, threads: int):
    """(context tokens/s, segments done, timed wall seconds) of the CPU oracle on a random
    sample of (sequence, layer, KV head) segments, `threads` segments at a time, each on its
    own host thread with BLAS limited to one thread (numpy releases the GIL in its array
    work).  Rounds of `threads` segments: their inputs are generated first (not timed), then
    the oracle runs on all of them in parallel and the round's wall time is counted, until
    `seconds` of wall time have been counted."""
    import concurrent.futures as cf

    import numpy as np
    import threadpoolctl

    from oracle import taskpress_oracle as o

    sys.path.insert(0, os.path.join(ROOT, "tests"))
    import parity_util as pu

    segs = [(b, l, h) for b in range(w.batch) for l in range(w.L) for h in range(w.Hkv)]
    order = [segs[i] for i in np.random.default_rng(seed).permutation(len(segs))]

    def run(inp):
        b, qg, kb, vb = inp
        o.evict_segment(qg, kb, vb, softmax_scale=w.softmax_scale, pool_k=w.pool_k, qfmt=w.qfmt, bits=w.bits,
                        rule=w.rule, k=o.keep_count(w.ctx_lens[b], w.keep_ratio, w.keep_budget))
        return w.ctx_lens[b]

    done_tokens = done = 0
    elapsed = 0.0
    with threadpoolctl.threadpool_limits(limits=1), cf.ThreadPoolExecutor(max_workers=threads) as ex:
        for r0 in range(0, len(order), threads):
            if elapsed >= seconds:
                break
            inputs = list(ex.map(lambda s: (s[0],) + pu.host_segment(w, *s), order[r0:r0 + threads]))
            t0 = time.perf_counter()
            done_tokens += sum(ex.map(run, inputs))
            elapsed += time.perf_counter() - t0
            done += len(inputs)
    # a context token counts once all L * Hkv segments of it are done
    return done_tokens / (w.L * w.Hkv) / elapsed, done, elapsed


def cpu_baseline(w, seconds: float):
    """The CPU oracle (test infrastructure) timed on a bounded sample of segments, spread over
    the host's cores (one segment per thread, at most 16 threads: a GPU machine's CPU share), and
    on one thread."""
    threads = max(1, min(16, os.cpu_count() or 1))
    segs = w.batch * w.L * w.Hkv
    rate, done, elapsed = _oracle_rate(w, seconds, 0, threads)
    rate1, done1, elapsed1 = _oracle_rate(w, seconds / 3, 1, 1)
    cpu = "unknown CPU"
    try:
        with open("/proc/cpuinfo") as f:
            cpu = next(l.split(":", 1)[1].strip() for l in f if l.startswith("model name"))
    except (OSError, StopIteration):
        pass
    return {"value": rate, "unit": "context tokens/s", "cores": threads, "kind": "oracle",
            "sample": f"{done} of {segs} (sequence, layer, KV head) segments in rounds of {threads}, one segment "
                      f"per thread, {elapsed:.1f} s of wall time (numpy float64, BLAS at 1 thread per segment; "
                      f"input generation not timed; {cpu}, {os.cpu_count()} logical CPUs visible)",
            "value_1_thread": rate1,
            "sample_1_thread": f"{done1} segments (another random order) on one thread, {elapsed1:.1f} s"}


def machine_rates():
    """Ceilings measured on this machine (microbenchmarks in libtprates.so): best streaming copy
    and read bandwidth over a few grid sizes, bf16 MFMA, v_exp_f32 and fp32 fma rates, and the
    shader clock while the MFMA loop runs.  Prints one JSON line."""
    import ctypes

    import torch

    lib = ctypes.CDLL(os.path.join(ROOT, "paper_2608_03276_amd", "lib", "libtprates.so"))
    P, I64, I32 = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int
    lib.mb_copy.argtypes = [P, P, I64, I32, P]
    lib.mb_read.argtypes = [P, I64, P, I32, P]
    lib.mb_two_pass.argtypes = [P, I64, I64, P, I32, P]
    lib.mb_exp.argtypes = [P, I32, I32, P]
    lib.mb_fma.argtypes = [P, I32, I32, P]
    lib.mb_mfma.argtypes = [P, P, I32, I32, P]
    torch.cuda.set_device(0)
    st = torch.cuda.current_stream()
    sp = ctypes.c_void_p(st.cuda_stream)

    def timed(fn, reps):
        for _ in range(2):
            assert fn() == 0
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(st)
        for _ in range(reps):
            assert fn() == 0
        b.record(st)
        torch.cuda.synchronize()
        return a.elapsed_time(b) * 1e-3 / reps

    nbytes = 4 << 30
    src = torch.ones(nbytes, dtype=torch.uint8, device="cuda")
    dst = torch.empty_like(src)
    sink = torch.zeros(4, dtype=torch.int32, device="cuda")
    n16 = nbytes // 16
    copy = {g: 2 * nbytes / timed(lambda g=g: lib.mb_copy(src.data_ptr(), dst.data_ptr(), n16, g, sp), 5) / 1e9
            for g in (1024, 4096, 16384)}
    read = {g: nbytes / timed(lambda g=g: lib.mb_read(src.data_ptr(), n16, sink.data_ptr(), g, sp), 5) / 1e9
            for g in (1024, 4096, 16384)}
    # A buffer read again by the next launch: the second read of X MB against the first (with
    # 1 GiB of other reads before the first, so it starts cold), median of 5.
    def once(fn):
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(st)
        assert fn() == 0
        b.record(st)
        torch.cuda.synchronize()
        return a.elapsed_time(b) * 1e-3

    reread = {}
    for xmb in (32, 64, 128, 192, 256):
        n = (xmb << 20) // 16
        first, second = [], []
        for _ in range(5):
            assert lib.mb_read(dst.data_ptr(), (1 << 30) // 16, sink.data_ptr(), 4096, sp) == 0
            first.append(once(lambda: lib.mb_read(src.data_ptr(), n, sink.data_ptr(), 4096, sp)))
            second.append(once(lambda: lib.mb_read(src.data_ptr(), n, sink.data_ptr(), 4096, sp)))
        reread[str(xmb)] = {"first_GBps": round((xmb << 20) / sorted(first)[2] / 1e9, 1),
                            "next_launch_GBps": round((xmb << 20) / sorted(second)[2] / 1e9, 1)}
    # Two read passes over 4 GiB: whole (the buffer twice) or chunk by chunk (each chunk read
    # twice in a row by two launches), as a schedule that re-reads K per group of segments would.
    two_pass = {}
    for cmb in (0, 32, 64, 128, 256):
        cb = nbytes if cmb == 0 else cmb << 20
        grid = 4096 if cmb == 0 else min(4096, cb // 16 // 256 // 4)
        t = timed(lambda: lib.mb_two_pass(src.data_ptr(), nbytes, cb, sink.data_ptr(), grid, sp), 3)
        two_pass["whole" if cmb == 0 else f"{cmb}MB_chunks"] = round(2 * nbytes / t / 1e9, 1)
    del src, dst
    blocks, iters = 2048, 4096
    out = torch.empty(blocks * 256, dtype=torch.float32, device="cuda")
    t_exp = timed(lambda: lib.mb_exp(out.data_ptr(), blocks, iters, sp), 3)
    t_fma = timed(lambda: lib.mb_fma(out.data_ptr(), blocks, iters, sp), 3)
    cyc = torch.zeros(blocks * 4 * 2, dtype=torch.int64, device="cuda")
    m_iters = 256
    t_mfma = timed(lambda: lib.mb_mfma(out.data_ptr(), cyc.data_ptr(), blocks, m_iters, sp), 3)
    c = cyc.view(-1, 2).double().cpu()
    clock = float((c[:, 0] / (c[:, 1] * 10.0)).median())  # s_memrealtime ticks at 100 MHz
    res = {
        "copy_GBps": {str(g): round(v, 1) for g, v in copy.items()},
        "read_GBps": {str(g): round(v, 1) for g, v in read.items()},
        "reread_next_launch_by_MB": reread,
        "two_read_passes_4GiB_GBps": two_pass,
        "exp2_Tps": round(blocks * 256 * iters * 8 / t_exp / 1e12, 2),
        "fma_f32_TFLOPs": round(2 * blocks * 256 * iters * 8 / t_fma / 1e12, 1),
        "mfma_bf16_TFLOPs": round(blocks * 4 * m_iters * 4 * 32768 / t_mfma / 1e12, 1),
        "shader_clock_GHz_during_mfma": round(clock, 3),
    }
    print(json.dumps({"rates": res}), flush=True)


def prefill_lse(w, q, k, kg=None):
    """The guide rows' natural-log normalisers that a prefill attention kernel exports (input
    preparation for --given-lse, outside the timed region): fp32 logits from torch matmuls,
    one (layer, KV head) at a time."""
    import torch

    out = torch.empty(w.L * w.Hq * w.g_tot, dtype=torch.float32, device=q.device)
    qv = q.view(w.L, w.Hq, w.g_tot, w.d)
    kv = k.view(w.L, w.Hkv, w.n_tot, w.d)
    kgv = kg.view(w.L, w.Hkv, w.g_tot, w.d) if kg is not None else None
    ov = out.view(w.L, w.Hq, w.g_tot)
    offs, goff = w.ctx_offsets(), w.guide_offsets()
    for b in range(w.batch):
        g0, g1, n0, n1 = goff[b], goff[b + 1], offs[b], offs[b + 1]
        for l in range(w.L):
            for h in range(w.Hkv):
                qs = qv[l, h * w.R:(h + 1) * w.R, g0:g1].float().reshape(-1, w.d)
                x = (qs @ kv[l, h, n0:n1].float().T) * w.softmax_scale
                if kgv is not None:
                    y = (qs @ kgv[l, h, g0:g1].float().T) * w.softmax_scale
                    j = torch.arange(g1 - g0, device=q.device)
                    y = y.masked_fill((j[None, :] > j[:, None]).repeat(w.R, 1), float("-inf"))
                    x = torch.cat([x, y], dim=1)
                ov[l, h * w.R:(h + 1) * w.R, g0:g1] = torch.logsumexp(x, dim=1).view(w.R, g1 - g0)
    torch.cuda.synchronize()
    return out


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="llama8b_128k")
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--guide-keys", action="store_true",
                    help="paper-literal normaliser: include the appended guide's own keys")
    ap.add_argument("--given-lse", action="store_true",
                    help="guide rows' log-normalisers supplied (as a prefill attention kernel exports them): "
                         "score pass 1 is skipped")
    ap.add_argument("--prefill-attention", action="store_true",
                    help="the prefill-integrated path: one step is the guide rows' prefill attention with step 2 "
                         "from the same sweep over V (tp_guide_attention_quantize over the context and the guide's "
                         "own keys and values: outputs, normalisers, V scales and codes) followed by tp_evict with "
                         "those normalisers, scales and codes (a secondary line)")
    ap.add_argument("--no-full-codes", action="store_true",
                    help="step 2 writes the scales only and the compaction quantises the kept V rows "
                         "(the codes of evicted rows are never written)")
    ap.add_argument("--bits", type=int, default=None,
                    help="integer code width b in [2, 8] instead of the workload's format (a b-sweep)")
    ap.add_argument("--fp8", action="store_true", help="E4M3 codes instead of the workload's format")
    ap.add_argument("--guide-tokens", type=int, default=None,
                    help="guide length G of every sequence instead of the workload's (a guide-length sweep)")
    ap.add_argument("--rates", action="store_true",
                    help="only run the machine-ceiling microbenchmarks and print them")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run a 1 GiB device copy (for counter calibration) and exit")
    args = ap.parse_args()
    if args.prefill_attention and args.no_full_codes:
        ap.error("--prefill-attention writes every token's codes with the attention: drop --no-full-codes")
    if args.gpus != 1:
        print(f"bench.py: measures one GPU only (asked for --gpus {args.gpus}); the path shards by "
              f"(layer, KV head, sequence) with no communication, so each GPU would run it on its own share.",
              file=sys.stderr)
        sys.exit(2)

    import torch

    if args.copy_calibration:
        copy_calibration()
        return
    if args.rates:
        machine_rates()
        return

    from paper_2608_03276_amd import binding as B
    from synth import device as SD
    from synth import workloads as W

    w = W.ALL[args.workload]()
    if args.bits is not None:
        w = w.with_(qfmt=B.TP_QFMT_INT, bits=args.bits)
    if args.fp8:
        w = w.with_(qfmt=B.TP_QFMT_FP8_E4M3, bits=8)
    if args.guide_tokens is not None:
        w = w.with_(guide_lens=tuple(args.guide_tokens for _ in w.ctx_lens))
    torch.cuda.set_device(0)
    q, k, v = SD.device_inputs(w)
    kg = SD.device_guide_keys(w) if (args.guide_keys or args.prefill_attention) else None
    vg = SD.device_guide_values(w) if args.prefill_attention else None
    lse = prefill_lse(w, q, k, kg) if args.given_lse else None
    if args.prefill_attention:  # written by tp_guide_attention_quantize inside every step
        lse = torch.empty(w.L * w.Hq * w.g_tot, dtype=torch.float32, device="cuda")
        o_guide = torch.empty(w.L * w.Hq * w.g_tot * w.d, dtype=torch.float32, device="cuda")
    kg_arg = None if lse is not None else kg
    d = B.dims(w.L, w.Hq, w.Hkv, w.d)
    bt = B.Batch(w.ctx_offsets(), w.guide_offsets())
    ko = B.kept_offsets_for(bt, w.keep_ratio or 0.0, w.keep_budget or 0)
    bufs = B.EvictBuffers(d, bt, w.qfmt, w.bits, ko)
    ws_attn = (torch.empty(B.tp_workspace_size(B.TP_FN_GUIDE_ATTENTION, d, bt), dtype=torch.uint8, device="cuda")
               if args.prefill_attention else None)
    torch.cuda.synchronize()

    def step(ev=None, att=None):
        if args.prefill_attention:
            if att is not None:
                att[0].record()
            B.tp_guide_attention_quantize(d, bt, q, k, v, w.softmax_scale, w.qfmt, w.bits, o_guide, lse,
                                          bufs.scales, bufs.v_q, ws_attn, k_guide=kg, v_guide=vg)
            if att is not None:
                att[1].record()
        B.tp_evict(d, bt, q, k, None if args.prefill_attention else v, w.softmax_scale, w.pool_k, w.qfmt, w.bits, w.rule, w.keep_ratio or 0.0,
                   w.keep_budget or 0, ko, bufs.s_key, bufs.scales, None if args.no_full_codes else bufs.v_q,
                   bufs.s_comb, bufs.kept_idx, bufs.k_c,
                   bufs.v_q_c, bufs.scales_c, bufs.ws_evict, events=ev, k_guide=kg_arg, guide_lse=lse)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    # Each step is timed by the events the library records at its start and end on this
    # stream; before each step a 512 MB device write (outside those events) evicts the caches
    # (4 MB of L2 per XCD, 256 MB Infinity Cache), so no step starts with the previous step's
    # data cached.  ms_per_step is the median over the K steps.
    flush = torch.empty(FLUSH_BYTES, dtype=torch.uint8, device="cuda")
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(B.TP_EVICT_EVENTS)] for _ in range(args.steps)]
    atts = [[torch.cuda.Event(enable_timing=True) for _ in range(2)] for _ in range(args.steps)]
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    start.record()
    for i in range(args.steps):
        flush.fill_(i & 0xFF)
        step(evs[i], atts[i])
    end.record()
    torch.cuda.synchronize()
    if args.prefill_attention:  # the step starts at the attention
        step_ms = sorted(a[0].elapsed_time(e[-1]) for a, e in zip(atts, evs))
    else:
        step_ms = sorted(e[0].elapsed_time(e[-1]) for e in evs)
    ms = statistics.median(step_ms)
    stages = STAGES if lse is None else ["pass1_skipped", "k_lse_import"] + STAGES[2:]
    if args.no_full_codes:
        stages = stages[:-1] + ["k_compact_quant"]
    if w.rule == B.TP_COMBINE_NORM_ADD:  # its norms need the pooled scores first: a pooling kernel
        stages[4] = "k_guide_pool"
    stage_ms = {n: statistics.median(e[j].elapsed_time(e[j + 1]) for e in evs) for j, n in enumerate(stages)}
    stage_ms.pop("pass1_skipped", None)
    if args.prefill_attention:  # step 2 ran inside the attention: no kernel between its events
        stage_ms.pop("k_quantize")
        stage_ms = dict({"k_guide_fwd": statistics.median(a[0].elapsed_time(a[1]) for a in atts)}, **stage_ms)
    timing = {"protocol": f"median of {args.steps} steps, each timed by events at its start and end on the "
                          f"stream it runs on, after {args.warmup} untimed warm-up steps; a {FLUSH_BYTES >> 20} MB "
                          f"device write before each step (outside its events) evicts the caches; stages_ms are "
                          f"per-kernel medians",
              "mean_ms": round(sum(step_ms) / len(step_ms), 4), "min_ms": round(step_ms[0], 4),
              "max_ms": round(step_ms[-1], 4),
              "bracket_ms_per_step": round(start.elapsed_time(end) / args.steps, 4)}

    per, path_bytes = algorithmic_bytes(w, ko[-1], not args.no_full_codes, lse is not None)
    # the two score passes are bf16 contractions (2 flop per guide-row x token x dim); the
    # other kernels stream HBM
    score_flops = 2 * w.L * w.Hq * sum(g * n for g, n in zip(w.guide_lens, w.ctx_lens)) * w.d

    # the guide rows' attention: the score contraction and the value product (twice the flops of
    # a score pass), over K and V once each
    attn_flops = 2 * score_flops + (4 * w.L * w.Hq * sum(g * (g + 1) // 2 for g in w.guide_lens) * w.d
                                    if args.prefill_attention else 0)
    per["k_guide_fwd"] = attention_bytes(w, args.prefill_attention)

    def roofline_of(kern):
        # the roof is whichever of HBM bytes and matrix flops takes longer at its peak; the
        # score passes sit just below the ridge point (about 250 flop/byte against 312)
        t = stage_ms[kern] * 1e-3
        hbm = {"bound": "hbm", "achieved": round(per[kern] / t / 1e9, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
               "frac": round(per[kern] / t / 1e9 / HBM_PEAK_GBS, 4), "algorithmic_bytes": per[kern]}
        if kern not in ("k_guide_stats", "k_guide_attn", "k_guide_fwd"):
            return hbm
        fl = attn_flops if kern == "k_guide_fwd" else score_flops
        mfma = {"bound": "mfma", "achieved": round(fl / t / 1e12, 1), "peak": MFMA_BF16_PEAK_TFLOPS,
                "unit": "TFLOP/s", "frac": round(fl / t / 1e12 / MFMA_BF16_PEAK_TFLOPS, 4), "flops": fl}
        hbm_s, mfma_s = per[kern] / (HBM_PEAK_GBS * 1e9), fl / (MFMA_BF16_PEAK_TFLOPS * 1e12)
        roof, other = (hbm, mfma) if hbm_s >= mfma_s else (mfma, hbm)
        return dict(roof, other_roof={k: other[k] for k in ("bound", "achieved", "unit", "frac")})

    kern = max(stage_ms, key=stage_ms.get)  # dominant kernel of the step
    # the committed counter summaries are of the workload's own format
    same_fmt = args.bits is None and not args.fp8 and args.guide_tokens is None
    roofline = dict(roofline_of(kern), traffic=measured_traffic(kern, args.workload) if same_fmt else None, kernel=kern,
                    avg_ms=round(stage_ms[kern], 4))
    path_gbs = path_bytes / (ms * 1e-3) / 1e9
    # the same path rate from the HBM bytes the counters measured for every kernel of the step
    # (second pass over K and re-reads included); only for the configuration the committed
    # summaries were taken on, and while every kernel's sources are unchanged
    measured_path = None
    if same_fmt and kg is None and lse is None and not args.no_full_codes:
        parts = [measured_traffic(kn, args.workload) for kn in STAGES + ["k_quantize_lean"]]
        if all(p is not None for p in parts):
            tot = sum(parts) + (LEAN_LAUNCHES[False] - 1) * parts[-1]
            measured_path = {"achieved": round(tot / (ms * 1e-3) / 1e9, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                             "frac": round(tot / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4), "traffic": tot}
    out = {
        "metric": METRIC,
        "value": round(w.n_tot / (ms * 1e-3), 1),
        "unit": "context tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded SplitMix64/Box-Muller draws of the workload's shapes and distributions)",
        "config": {"workload": w.describe()
                   + (", the guide rows' prefill attention (context and guide keys: outputs and normalisers) "
                      "with V's scales and codes from the same sweep, followed by the eviction from those"
                      if args.prefill_attention else "")
                   + (", guide keys in the normaliser" if kg is not None and not args.prefill_attention else "")
                   + (", row normalisers supplied by the prefill (score pass 1 skipped)"
                      if args.given_lse else "")
                   + (", codes written for the kept rows only" if args.no_full_codes else ""),
                   "layers": w.L, "q_heads": w.Hq, "kv_heads": w.Hkv, "head_dim": w.d,
                   "context_tokens": w.n_tot, "guide_tokens": w.g_tot, "kept_per_head": ko[-1]},
        "roofline": roofline,
        "path_hbm": {"achieved": round(path_gbs, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(path_gbs / HBM_PEAK_GBS, 4), "algorithmic_bytes": path_bytes},
        "path_hbm_measured": measured_path,
        "timing": timing,
        "stages_ms": {n: round(t, 4) for n, t in stage_ms.items()},
        "kernel_rooflines": {n: {k: v for k, v in roofline_of(n).items()
                                 if k in ("bound", "achieved", "unit", "frac", "other_roof")}
                             for n in stage_ms if n not in ("k_guide_lse", "k_lse_import")},
    }
    del q, k, v, kg, vg, bufs, flush, ws_attn
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(w, args.cpu_seconds)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
