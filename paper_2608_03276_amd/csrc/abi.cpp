// C-ABI layer of libtaskpress: synchronous host-side validation, workspace layout and
// kernel dispatch.  Nothing is enqueued unless every argument is valid.
#include <math.h>
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <algorithm>
#include <mutex>
#include <string>

#include "tp_internal.h"

namespace {

thread_local std::string g_err;

tp_status fail(tp_status s, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return s;
}

tp_status ok() {
  g_err.clear();
  return TP_OK;
}

bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

tp_status check_dims(const tp_dims* d) {
  if (!d) return fail(TP_ERR_NULL, "dims is NULL");
  if (d->num_layers < 1 || d->num_q_heads < 1 || d->num_kv_heads < 1 || d->head_dim < 1)
    return fail(TP_ERR_SHAPE, "dims must be positive (L=%d Hq=%d Hkv=%d d=%d)", d->num_layers,
                d->num_q_heads, d->num_kv_heads, d->head_dim);
  if (d->num_q_heads % d->num_kv_heads != 0)
    return fail(TP_ERR_SHAPE, "num_q_heads (%d) is not a multiple of num_kv_heads (%d)", d->num_q_heads,
                d->num_kv_heads);
  if (d->head_dim != 64 && d->head_dim != 128)
    return fail(TP_ERR_UNSUPPORTED, "head_dim %d not supported (64 or 128)", d->head_dim);
  if ((int64_t)d->num_layers * d->num_kv_heads > 65535)
    return fail(TP_ERR_UNSUPPORTED, "num_layers * num_kv_heads exceeds 65535");
  return TP_OK;
}

tp_status check_offsets(const int64_t* off, int32_t batch, const char* what, bool allow_empty_seq) {
  if (!off) return fail(TP_ERR_NULL, "%s is NULL", what);
  if (off[0] != 0) return fail(TP_ERR_SHAPE, "%s[0] must be 0", what);
  for (int b = 0; b < batch; ++b)  // compared, not subtracted: arbitrary entries cannot overflow
    if (off[b + 1] < off[b] || (!allow_empty_seq && off[b + 1] == off[b]))
      return fail(TP_ERR_SHAPE, "%s: entry %d is empty or negative (%lld -> %lld)", what, b, (long long)off[b],
                  (long long)off[b + 1]);
  return TP_OK;
}

// The batch's offsets (nondecreasing from 0, each sequence non-empty), and extents for which
// every size the layouts derive fits in 64 bits and every launch fits its grid (a dispatch
// holds fewer than 2^32 work-items per dimension): at most 2^30 context tokens per (layer,
// head) (the gather launches 4 work-items per kept token; kept indices are int32), at most
// 2^32 guide rows in all and 2^26 per sequence (the row merges launch a work-item per row and
// 64 per row), 2^31 - 1 guide tokens, and 2^60 bytes of per-chunk row partials (chunks of
// 8192 tokens, the smallest any kernel uses).  Far above any cache one GPU holds.  `d` has
// passed check_dims.
tp_status check_batch(const tp_dims* d, const tp_batch* bt, bool need_guides) {
  if (!bt) return fail(TP_ERR_NULL, "batch is NULL");
  if (bt->batch < 1) return fail(TP_ERR_SHAPE, "batch must be >= 1");
  if (bt->batch > TP_MAX_BATCH)
    return fail(TP_ERR_UNSUPPORTED, "batch %d exceeds TP_MAX_BATCH (%d)", bt->batch, TP_MAX_BATCH);
  tp_status s = check_offsets(bt->ctx_offsets, bt->batch, "ctx_offsets", false);
  if (s != TP_OK) return s;
  if (bt->ctx_offsets[bt->batch] > ((int64_t)1 << 30))
    return fail(TP_ERR_UNSUPPORTED, "context of %lld tokens too large (at most 2^30)",
                (long long)bt->ctx_offsets[bt->batch]);
  if (need_guides) {
    s = check_offsets(bt->guide_offsets, bt->batch, "guide_offsets", false);
    if (s != TP_OK) return s;
    int64_t max_nb = 0, max_gb = 0;
    for (int b = 0; b < bt->batch; ++b) {
      max_nb = std::max<int64_t>(max_nb, bt->ctx_offsets[b + 1] - bt->ctx_offsets[b]);
      max_gb = std::max<int64_t>(max_gb, bt->guide_offsets[b + 1] - bt->guide_offsets[b]);
    }
    const double g_tot = (double)bt->guide_offsets[bt->batch];
    const double heads = (double)d->num_layers * d->num_q_heads;
    const double rows = g_tot * heads;
    if (g_tot > 0x1p31 - 1 || rows > 0x1p32 || (double)max_gb * heads > 0x1p26 ||
        rows * ((double)max_nb / 8192.0 + 2.0) * (8.0 + 4.0 * d->head_dim) > 0x1p60)
      return fail(TP_ERR_UNSUPPORTED, "guide of %lld tokens too large for these dims and context",
                  (long long)bt->guide_offsets[bt->batch]);
  }
  return TP_OK;
}

tp::BatchArgs batch_args(const tp_batch* bt, bool with_guides) {
  tp::BatchArgs a;
  memset(&a, 0, sizeof a);
  a.batch = bt->batch;
  for (int b = 0; b <= bt->batch; ++b) {
    a.ctx_off[b] = bt->ctx_offsets[b];
    a.g_off[b] = with_guides ? bt->guide_offsets[b] : 0;
  }
  return a;
}

tp_status hip_fail(hipError_t e, const char* where) {
  return fail(TP_ERR_HIP, "%s: %s", where, hipGetErrorString(e));
}

size_t select_workspace(const tp_dims* d, const tp_batch* bt) {
  return tp::select_workspace_layout((int64_t)d->num_layers * d->num_kv_heads, bt->ctx_offsets, bt->batch).total;
}

// Largest quantised magnitude (Eq. 2): 2^(b-1) - 1 for b-bit integers, 448 for E4M3.
float qmax_of(int32_t qfmt, int32_t bits) { return qfmt == TP_QFMT_INT ? (float)((1 << (bits - 1)) - 1) : 448.0f; }

int row_bytes_of(int32_t qfmt, int32_t bits, int32_t d) {
  return (qfmt == TP_QFMT_INT && bits <= 4) ? d / 2 : d;
}

tp_status check_qfmt(int32_t qfmt, int32_t bits) {
  if (qfmt == TP_QFMT_INT) {
    if (bits < 2 || bits > 8) return fail(TP_ERR_PARAM, "bits %d outside [2, 8]", bits);
    return TP_OK;
  }
  if (qfmt == TP_QFMT_FP8_E4M3) return TP_OK;
  return fail(TP_ERR_PARAM, "unknown qfmt %d", qfmt);
}


// ------------------------------------------------------------------ argument preparation
// Each prepare_* validates one step's arguments and fills its kernel arguments without
// enqueueing anything, so the fused entry point can validate every step before launching.

tp_status prepare_guide(const tp_dims* dims, const tp_batch* batch, const void* q_guide, const void* k,
                        const void* k_guide, const float* guide_lse, float softmax_scale, int32_t pool_k,
                        float* s_key, void* workspace, size_t ws_bytes, tp::GuideArgs& a) {
  tp_status s = check_dims(dims);
  if (s != TP_OK) return s;
  s = check_batch(dims, batch, true);
  if (s != TP_OK) return s;
  if (!q_guide || !k || !s_key) return fail(TP_ERR_NULL, "q_guide, k and s_key must be non-NULL");
  if (!aligned16(q_guide) || !aligned16(k) || !aligned16(s_key) || (k_guide && !aligned16(k_guide)))
    return fail(TP_ERR_PARAM, "tensor pointers must be 16-byte aligned");
  if (k_guide && guide_lse)
    return fail(TP_ERR_PARAM, "k_guide and guide_lse are exclusive (supplied normalisers already cover the keys)");
  if (guide_lse && ((uintptr_t)guide_lse & 3u) != 0) return fail(TP_ERR_PARAM, "guide_lse must be 4-byte aligned");
  if (!(softmax_scale > 0.0f) || !isfinite(softmax_scale))
    return fail(TP_ERR_PARAM, "softmax_scale must be finite and > 0");
  if (pool_k < 1 || (pool_k & 1) == 0) return fail(TP_ERR_PARAM, "pool_k must be odd and >= 1 (got %d)", pool_k);
  const tp::GuideWorkspace lay = tp::guide_workspace_layout(
      dims->num_layers, dims->num_q_heads, dims->num_kv_heads, batch->ctx_offsets, batch->guide_offsets, batch->batch);
  if (!workspace || ws_bytes < lay.total)
    return fail(TP_ERR_WORKSPACE, "workspace needs %zu bytes (got %zu%s)", lay.total, ws_bytes,
                workspace ? "" : ", NULL");
  if (((uintptr_t)workspace & 255u) != 0) return fail(TP_ERR_WORKSPACE, "workspace must be 256-byte aligned");

  memset(&a, 0, sizeof a);
  a.bt = batch_args(batch, true);
  int64_t max_nb = 0, max_gb = 0;
  for (int b = 0; b < batch->batch; ++b) {
    max_nb = std::max<int64_t>(max_nb, batch->ctx_offsets[b + 1] - batch->ctx_offsets[b]);
    max_gb = std::max<int64_t>(max_gb, batch->guide_offsets[b + 1] - batch->guide_offsets[b]);
  }
  a.q = (const uint16_t*)q_guide;
  a.k = (const uint16_t*)k;
  a.kg = (const uint16_t*)k_guide;
  a.lse_in = guide_lse;
  a.s_key = s_key;
  a.stats = (float2*)((char*)workspace + lay.stats_off);
  a.lse2 = (float*)((char*)workspace + lay.lse_off);
  a.raw = (float*)((char*)workspace + lay.raw_off);
  a.L = dims->num_layers;
  a.Hq = dims->num_q_heads;
  a.Hkv = dims->num_kv_heads;
  a.R = dims->num_q_heads / dims->num_kv_heads;
  a.n_tot = batch->ctx_offsets[batch->batch];
  a.g_tot = batch->guide_offsets[batch->batch];
  a.c = (float)((double)softmax_scale * 1.4426950408889634);
  a.pool_inv = (float)(1.0 / ((double)a.R * pool_k));
  a.pool_half = pool_k / 2;
  a.chunk = tp::chunk_tokens(batch->ctx_offsets, batch->batch);
  a.nchunk_max = (int32_t)((max_nb + a.chunk - 1) / a.chunk);
  a.nrg_max = (int32_t)((a.R * max_gb + tp::kRowsPerGroup - 1) / tp::kRowsPerGroup);
  // workgroups of the score passes (the launcher splits them into row-block classes, each
  // with its own per-sequence ranges in wg_off); the total must fit one grid
  int64_t wg = 0;
  a.wg_off[0] = 0;
  for (int b = 0; b < batch->batch; ++b) {
    const int64_t nb = batch->ctx_offsets[b + 1] - batch->ctx_offsets[b];
    const int64_t gb = batch->guide_offsets[b + 1] - batch->guide_offsets[b];
    const int64_t units = (int64_t)a.L * a.Hkv * ((nb + a.chunk - 1) / a.chunk);
    wg += (units + 7) / 8 * 8 * ((a.R * gb + tp::kRowsPerGroup - 1) / tp::kRowsPerGroup);
    if (wg > 0x7FFFFFFF) return fail(TP_ERR_UNSUPPORTED, "context or guide too long for one launch");
    a.wg_off[b + 1] = (int32_t)wg;
  }
  return TP_OK;
}

tp_status prepare_quant(const tp_dims* dims, const tp_batch* batch, const void* v, int32_t qfmt, int32_t bits,
                        float* scales, void* v_q, tp::QuantArgs& a) {
  tp_status s = check_dims(dims);
  if (s != TP_OK) return s;
  s = check_batch(dims, batch, false);
  if (s != TP_OK) return s;
  s = check_qfmt(qfmt, bits);
  if (s != TP_OK) return s;
  if (!v || !scales) return fail(TP_ERR_NULL, "v and scales must be non-NULL");
  if (!aligned16(v) || !aligned16(scales) || (v_q && !aligned16(v_q)))
    return fail(TP_ERR_PARAM, "tensor pointers must be 16-byte aligned");
  a.v = (const uint16_t*)v;
  a.scales = scales;
  a.vq = (uint8_t*)v_q;
  a.rows = (int64_t)dims->num_layers * dims->num_kv_heads * batch->ctx_offsets[batch->batch];
  a.qfmt = qfmt;
  a.bits = bits;
  a.qmax = qmax_of(qfmt, bits);
  a.ro = tp::recip_offsets_for(a.qmax);
  return TP_OK;
}

tp_status prepare_select(const tp_dims* dims, const tp_batch* batch, const float* s_key, const float* scales,
                         int32_t rule, double keep_ratio, int64_t keep_budget, const int64_t* kept_offsets,
                         int32_t* kept_idx, float* s_out, void* workspace, size_t ws_bytes, tp::SelectArgs& a) {
  tp_status s = check_dims(dims);
  if (s != TP_OK) return s;
  s = check_batch(dims, batch, false);
  if (s != TP_OK) return s;
  if (!s_key || !scales || !kept_idx) return fail(TP_ERR_NULL, "s_key, scales and kept_idx must be non-NULL");
  if (!aligned16(s_key) || !aligned16(scales) || !aligned16(kept_idx) || (s_out && !aligned16(s_out)))
    return fail(TP_ERR_PARAM, "tensor pointers must be 16-byte aligned");
  if (rule < TP_COMBINE_MUL || rule > TP_COMBINE_KEY_ONLY) return fail(TP_ERR_PARAM, "unknown rule %d", rule);
  const bool use_ratio = keep_ratio > 0.0, use_budget = keep_budget >= 1;
  if (use_ratio == use_budget)
    return fail(TP_ERR_PARAM, "exactly one of keep_ratio in (0,1] and keep_budget >= 1 must be given");
  if (use_ratio && !(keep_ratio <= 1.0)) return fail(TP_ERR_PARAM, "keep_ratio must be in (0, 1]");
  if (!kept_offsets) return fail(TP_ERR_NULL, "kept_offsets is NULL");
  if (kept_offsets[0] != 0) return fail(TP_ERR_SHAPE, "kept_offsets[0] must be 0");
  memset(&a, 0, sizeof a);
  for (int b = 0; b < batch->batch; ++b) {
    const int64_t nb = batch->ctx_offsets[b + 1] - batch->ctx_offsets[b];
    const int64_t kb = tp_keep_count(nb, keep_ratio, keep_budget);
    if (kept_offsets[b + 1] < kept_offsets[b] || kept_offsets[b + 1] - kept_offsets[b] != kb)
      return fail(TP_ERR_SHAPE, "kept_offsets[%d+1]-kept_offsets[%d] = %lld, expected keep count %lld", b, b,
                  (long long)(kept_offsets[b + 1] - kept_offsets[b]), (long long)kb);
    a.k[b] = kb;
    a.kept_off[b] = kept_offsets[b];
  }
  a.kept_off[batch->batch] = kept_offsets[batch->batch];
  const int64_t segs = (int64_t)dims->num_layers * dims->num_kv_heads;
  const tp::SelectWorkspace lay = tp::select_workspace_layout(segs, batch->ctx_offsets, batch->batch);
  if (!workspace || ws_bytes < lay.total)
    return fail(TP_ERR_WORKSPACE, "workspace needs %zu bytes (got %zu%s)", lay.total, ws_bytes,
                workspace ? "" : ", NULL");
  if (((uintptr_t)workspace & 255u) != 0) return fail(TP_ERR_WORKSPACE, "workspace must be 256-byte aligned");
  char* ws = (char*)workspace;
  a.s_key = s_key;
  a.scales = scales;
  a.s_buf = s_out ? s_out : (float*)(ws + lay.s_off);
  a.hist = (uint32_t*)(ws + lay.hist_off);
  a.info = (uint4*)(ws + lay.info_off);
  a.thr = (uint2*)(ws + lay.thr_off);
  a.pcount = (uint2*)(ws + lay.pcount_off);
  a.pref = (uint2*)(ws + lay.pref_off);
  a.cstart = (uint32_t*)(ws + lay.cstart_off);
  a.cand = (uint32_t*)(ws + lay.cand_off);
  a.part_tot = lay.part_tot;
  a.cand_tot = lay.cand_tot;
  a.part_off[0] = a.cand_off[0] = 0;
  int64_t part_max = 0;
  for (int b = 0; b < batch->batch; ++b) {
    const int64_t nb = batch->ctx_offsets[b + 1] - batch->ctx_offsets[b];
    const int64_t np = (nb + tp::kSelPartTokens - 1) / tp::kSelPartTokens;
    part_max = std::max(part_max, np);
    a.part_off[b + 1] = a.part_off[b] + np;
    a.cand_off[b + 1] = a.cand_off[b] + std::min<int64_t>(nb, tp::kSelCandCap);
  }
  if (part_max > 65535) return fail(TP_ERR_UNSUPPORTED, "a sequence of more than %lld context tokens",
                                    (long long)65535 * tp::kSelPartTokens);
  a.part_max = (int32_t)part_max;
  a.raw = nullptr;  // the key score is read (tp_evict sets the fused pooling)
  a.s_key_out = nullptr;
  a.kept = kept_idx;
  a.n_tot = batch->ctx_offsets[batch->batch];
  a.k_tot = kept_offsets[batch->batch];
  a.rule = rule;
  a.bt = batch_args(batch, false);
  return TP_OK;
}

tp_status prepare_compact(const tp_dims* dims, const tp_batch* batch, const int64_t* kept_offsets,
                          const int32_t* kept_idx, const void* k, const void* v_q, const float* scales,
                          int32_t qfmt, int32_t bits, void* k_out, void* v_q_out, float* scales_out,
                          tp::CompactArgs& a) {
  tp_status s = check_dims(dims);
  if (s != TP_OK) return s;
  s = check_batch(dims, batch, false);
  if (s != TP_OK) return s;
  s = check_qfmt(qfmt, bits);
  if (s != TP_OK) return s;
  if (!kept_idx || !k || !k_out) return fail(TP_ERR_NULL, "kept_idx, k and k_out must be non-NULL");
  if ((v_q == nullptr) != (v_q_out == nullptr)) return fail(TP_ERR_NULL, "v_q and v_q_out must both be given or both NULL");
  if ((scales == nullptr) != (scales_out == nullptr))
    return fail(TP_ERR_NULL, "scales and scales_out must both be given or both NULL");
  if (!aligned16(kept_idx) || !aligned16(k) || !aligned16(k_out) || (v_q && (!aligned16(v_q) || !aligned16(v_q_out))) ||
      (scales && (!aligned16(scales) || !aligned16(scales_out))))
    return fail(TP_ERR_PARAM, "tensor pointers must be 16-byte aligned");
  if (!kept_offsets) return fail(TP_ERR_NULL, "kept_offsets is NULL");
  if (kept_offsets[0] != 0) return fail(TP_ERR_SHAPE, "kept_offsets[0] must be 0");
  memset(&a, 0, sizeof a);
  for (int b = 0; b < batch->batch; ++b) {
    const int64_t nb = batch->ctx_offsets[b + 1] - batch->ctx_offsets[b];
    if (kept_offsets[b + 1] < kept_offsets[b])  // entries from 0 up: their differences cannot overflow
      return fail(TP_ERR_SHAPE, "kept_offsets decrease at entry %d", b);
    const int64_t kb = kept_offsets[b + 1] - kept_offsets[b];
    if (kb > nb)
      return fail(TP_ERR_SHAPE, "kept count of sequence %d (%lld) outside [0, %lld]", b, (long long)kb, (long long)nb);
    a.kept_off[b] = kept_offsets[b];
  }
  a.kept_off[batch->batch] = kept_offsets[batch->batch];
  a.kept = kept_idx;
  a.k = (const uint16_t*)k;
  a.vq = (const uint8_t*)v_q;
  a.scales = scales;
  a.k_out = (uint16_t*)k_out;
  a.vq_out = (uint8_t*)v_q_out;
  a.scales_out = scales_out;
  a.n_tot = batch->ctx_offsets[batch->batch];
  a.k_tot = kept_offsets[batch->batch];
  a.row_bytes = row_bytes_of(qfmt, bits, dims->head_dim);
  a.qfmt = qfmt;
  a.bits = bits;
  a.qmax = qmax_of(qfmt, bits);
  a.ro = tp::recip_offsets_for(a.qmax);
  a.bt = batch_args(batch, false);
  return TP_OK;
}

// Compaction that quantises the kept V rows while gathering them (no full code tensor).
tp_status prepare_compact_quant(const tp_dims* dims, const tp_batch* batch, const int64_t* kept_offsets,
                                const int32_t* kept_idx, const void* k, const void* v, int32_t qfmt, int32_t bits,
                                void* k_out, void* v_q_out, float* scales_out, tp::CompactArgs& a) {
  if (!v || !v_q_out || !scales_out) return fail(TP_ERR_NULL, "v, v_q_out and scales_out must be non-NULL");
  if (!aligned16(v)) return fail(TP_ERR_PARAM, "tensor pointers must be 16-byte aligned");
  // the plain gather's checks, with the code and scale outputs fed from placeholders
  const tp_status s = prepare_compact(dims, batch, kept_offsets, kept_idx, k, v_q_out, scales_out, qfmt, bits, k_out,
                                      v_q_out, scales_out, a);
  if (s != TP_OK) return s;
  a.v = (const uint16_t*)v;
  a.vq = nullptr;
  a.scales = nullptr;
  return TP_OK;
}

size_t guide_workspace_bytes(const tp_dims* dims, const tp_batch* batch) {
  return tp::guide_workspace_layout(dims->num_layers, dims->num_q_heads, dims->num_kv_heads, batch->ctx_offsets,
                                    batch->guide_offsets, batch->batch)
      .total;
}

// tp_evict's workspace: the score pass's, then the selection's.
size_t evict_workspace_bytes(const tp_dims* dims, const tp_batch* batch) {
  return guide_workspace_bytes(dims, batch) + select_workspace(dims, batch);
}

// The second stream of tp_evict on one device and the events that fork it from, and join it
// to, the caller's stream (part1: the first part of step 2 on it is done): created by the first tp_evict call on that device and kept until
// the process ends.  `enqueue` is held while a call enqueues its work, so calls from several
// threads do not interleave their uses of the events.
struct AuxStream {
  std::mutex enqueue;
  bool ready = false;
  hipStream_t stream = nullptr;
  hipEvent_t fork = nullptr, fork2 = nullptr, join = nullptr, part1 = nullptr;
};
constexpr int kMaxDevices = 64;
AuxStream g_aux[kMaxDevices];
std::mutex g_aux_setup;

tp_status aux_stream_for(hipStream_t st, AuxStream*& out) {
  int dev = 0;
  hipError_t e = st ? hipStreamGetDevice(st, &dev) : hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "tp_evict: device of the stream");
  if (dev < 0 || dev >= kMaxDevices) return fail(TP_ERR_UNSUPPORTED, "tp_evict: device %d", dev);
  AuxStream& a = g_aux[dev];
  std::lock_guard<std::mutex> lk(g_aux_setup);
  if (!a.ready) {
    int cur = 0;
    e = hipGetDevice(&cur);
    if (e == hipSuccess && cur != dev) e = hipSetDevice(dev);
    // default priority (the caller's streams' priority is not inherited)
    if (e == hipSuccess && !a.stream) e = hipStreamCreateWithFlags(&a.stream, hipStreamNonBlocking);
    if (e == hipSuccess && !a.fork) e = hipEventCreateWithFlags(&a.fork, hipEventDisableTiming);
    if (e == hipSuccess && !a.fork2) e = hipEventCreateWithFlags(&a.fork2, hipEventDisableTiming);
    if (e == hipSuccess && !a.join) e = hipEventCreateWithFlags(&a.join, hipEventDisableTiming);
    if (e == hipSuccess && !a.part1) e = hipEventCreateWithFlags(&a.part1, hipEventDisableTiming);
    if (cur != dev) {
      const hipError_t e2 = hipSetDevice(cur);
      if (e == hipSuccess) e = e2;
    }
    if (e != hipSuccess) return hip_fail(e, "tp_evict: second stream");
    a.ready = true;
  }
  out = &a;
  return TP_OK;
}

// The selection's workspace pointers, laid out from `from`, moved to the same offsets from `to`.
char* const kPlaceholder = (char*)(uintptr_t)256;  // a 256-byte-aligned stand-in, never dereferenced
void rebase_select(tp::SelectArgs& a, char* from, char* to) {
  auto mv = [&](auto* p) { return (decltype(p))(to + ((char*)p - from)); };
  a.s_buf = mv(a.s_buf);
  a.hist = mv(a.hist);
  a.info = mv(a.info);
  a.thr = mv(a.thr);
  a.pcount = mv(a.pcount);
  a.pref = mv(a.pref);
  a.cstart = mv(a.cstart);
  a.cand = mv(a.cand);
}

// After a failed enqueue in tp_evict: record the join event on the second stream (it then
// completes once everything already queued there has run) and make `st` wait for it.  If the
// record itself fails, the stream is synchronised instead, so no queued part outlives the
// call's error return.  Errors here are not reported: the call already fails.
void join_after_failure(AuxStream* aux, hipStream_t st) {
  if (hipEventRecord(aux->join, aux->stream) == hipSuccess) {
    if (hipStreamWaitEvent(st, aux->join, 0) == hipSuccess) return;
  }
  (void)hipStreamSynchronize(aux->stream);
}

}  // namespace

extern "C" {

const char* tp_version(void) { return "taskpress-mi355x 0.1.0 (gfx950)"; }

const char* tp_status_string(tp_status s) {
  switch (s) {
    case TP_OK: return "TP_OK";
    case TP_ERR_NULL: return "TP_ERR_NULL";
    case TP_ERR_SHAPE: return "TP_ERR_SHAPE";
    case TP_ERR_PARAM: return "TP_ERR_PARAM";
    case TP_ERR_UNSUPPORTED: return "TP_ERR_UNSUPPORTED";
    case TP_ERR_WORKSPACE: return "TP_ERR_WORKSPACE";
    case TP_ERR_HIP: return "TP_ERR_HIP";
    default: return "TP_ERR_UNKNOWN";
  }
}

const char* tp_last_error(void) { return g_err.c_str(); }

int64_t tp_keep_count(int64_t n, double keep_ratio, int64_t keep_budget) {
  if (n < 1) return -1;
  const bool use_ratio = keep_ratio > 0.0;
  const bool use_budget = keep_budget >= 1;
  if (use_ratio == use_budget) return -1;
  if (use_ratio) {
    if (!(keep_ratio <= 1.0)) return -1;
    // k <= n; (double)n can round above n (to 2^63 at the top of the range), so compare
    // before converting back
    const double kd = floor((double)n * keep_ratio);
    if (kd >= (double)n) return n;
    const int64_t k = (int64_t)kd;
    return k < 1 ? 1 : k;
  }
  return keep_budget < n ? keep_budget : n;
}

tp_status tp_workspace_size(int32_t fn, const tp_dims* dims, const tp_batch* batch, size_t* bytes) {
  if (!bytes) return fail(TP_ERR_NULL, "bytes is NULL");
  tp_status s = check_dims(dims);
  if (s != TP_OK) return s;
  if (fn == TP_FN_GUIDE_SCORES) {
    s = check_batch(dims, batch, true);
    if (s != TP_OK) return s;
    *bytes = tp::guide_workspace_layout(dims->num_layers, dims->num_q_heads, dims->num_kv_heads,
                                        batch->ctx_offsets, batch->guide_offsets, batch->batch)
                 .total;
    return ok();
  }
  if (fn == TP_FN_COMBINE_SELECT_TOPK) {
    s = check_batch(dims, batch, false);
    if (s != TP_OK) return s;
    *bytes = select_workspace(dims, batch);
    return ok();
  }
  if (fn == TP_FN_GUIDE_ATTENTION) {
    s = check_batch(dims, batch, true);
    if (s != TP_OK) return s;
    *bytes = tp::attn_workspace_layout(dims->num_layers, dims->num_q_heads, dims->num_kv_heads, dims->head_dim,
                                       batch->ctx_offsets, batch->guide_offsets, batch->batch)
                 .total;
    return ok();
  }
  if (fn == TP_FN_EVICT) {
    s = check_batch(dims, batch, true);
    if (s != TP_OK) return s;
    *bytes = evict_workspace_bytes(dims, batch);
    return ok();
  }
  return fail(TP_ERR_PARAM, "unknown function id %d", fn);
}

tp_status tp_guide_scores(const tp_dims* dims, const tp_batch* batch, const void* q_guide, const void* k,
                          const void* k_guide, float softmax_scale, int32_t pool_k, float* s_key,
                          void* workspace, size_t ws_bytes, void* stream) {
  tp::GuideArgs a;
  const tp_status s =
      prepare_guide(dims, batch, q_guide, k, k_guide, nullptr, softmax_scale, pool_k, s_key, workspace, ws_bytes, a);
  if (s != TP_OK) return s;
  const hipError_t e = tp::launch_guide_scores(a, dims->head_dim, (hipStream_t)stream, nullptr);
  if (e != hipSuccess) return hip_fail(e, "tp_guide_scores launch");
  return ok();
}

tp_status tp_guide_scores_lse(const tp_dims* dims, const tp_batch* batch, const void* q_guide, const void* k,
                              const float* guide_lse, float softmax_scale, int32_t pool_k, float* s_key,
                              void* workspace, size_t ws_bytes, void* stream) {
  if (!guide_lse) return fail(TP_ERR_NULL, "guide_lse must be non-NULL");
  tp::GuideArgs a;
  const tp_status s = prepare_guide(dims, batch, q_guide, k, nullptr, guide_lse, softmax_scale, pool_k, s_key,
                                    workspace, ws_bytes, a);
  if (s != TP_OK) return s;
  const hipError_t e = tp::launch_guide_scores(a, dims->head_dim, (hipStream_t)stream, nullptr);
  if (e != hipSuccess) return hip_fail(e, "tp_guide_scores_lse launch");
  return ok();
}

}  // extern "C"

// The guide rows' attention; with qa (step 2 already validated) the kernel also quantises V.
static tp_status guide_attention(const tp_dims* dims, const tp_batch* batch, const void* q_guide, const void* k,
                                 const void* v, const void* k_guide, const void* v_guide, float softmax_scale,
                                 float* o_guide, float* guide_lse, const tp::QuantArgs* qa, void* workspace,
                                 size_t ws_bytes, void* stream) {
  tp_status s = check_dims(dims);
  if (s != TP_OK) return s;
  s = check_batch(dims, batch, true);
  if (s != TP_OK) return s;
  if (!q_guide || !k || !v || !o_guide || !guide_lse)
    return fail(TP_ERR_NULL, "q_guide, k, v, o_guide and guide_lse must be non-NULL");
  if ((k_guide == nullptr) != (v_guide == nullptr))
    return fail(TP_ERR_NULL, "k_guide and v_guide must both be given or both NULL");
  if (!aligned16(q_guide) || !aligned16(k) || !aligned16(v) || !aligned16(o_guide) ||
      (k_guide && (!aligned16(k_guide) || !aligned16(v_guide))))
    return fail(TP_ERR_PARAM, "tensor pointers must be 16-byte aligned");
  if (((uintptr_t)guide_lse & 3u) != 0) return fail(TP_ERR_PARAM, "guide_lse must be 4-byte aligned");
  if (!(softmax_scale > 0.0f) || !isfinite(softmax_scale))
    return fail(TP_ERR_PARAM, "softmax_scale must be finite and > 0");
  const tp::AttnWorkspace lay = tp::attn_workspace_layout(dims->num_layers, dims->num_q_heads, dims->num_kv_heads,
                                                          dims->head_dim, batch->ctx_offsets, batch->guide_offsets,
                                                          batch->batch);
  if (!workspace || ws_bytes < lay.total)
    return fail(TP_ERR_WORKSPACE, "workspace needs %zu bytes (got %zu%s)", lay.total, ws_bytes,
                workspace ? "" : ", NULL");
  if (((uintptr_t)workspace & 255u) != 0) return fail(TP_ERR_WORKSPACE, "workspace must be 256-byte aligned");
  tp::AttnArgs a;
  memset(&a, 0, sizeof a);
  a.bt = batch_args(batch, true);
  a.q = (const uint16_t*)q_guide;
  a.k = (const uint16_t*)k;
  a.v = (const uint16_t*)v;
  a.kg = (const uint16_t*)k_guide;
  a.vg = (const uint16_t*)v_guide;
  a.o = o_guide;
  a.lse = guide_lse;
  a.pstat = (float2*)((char*)workspace + lay.pstat_off);
  a.po = (float*)((char*)workspace + lay.po_off);
  a.L = dims->num_layers;
  a.Hq = dims->num_q_heads;
  a.Hkv = dims->num_kv_heads;
  a.R = dims->num_q_heads / dims->num_kv_heads;
  a.n_tot = batch->ctx_offsets[batch->batch];
  a.g_tot = batch->guide_offsets[batch->batch];
  a.c = (float)((double)softmax_scale * 1.4426950408889634);
  a.chunk = tp::attn_chunk_tokens(batch->ctx_offsets, batch->batch);
  int64_t max_nb = 0, max_gb = 0;
  for (int b = 0; b < batch->batch; ++b) {
    max_nb = std::max<int64_t>(max_nb, batch->ctx_offsets[b + 1] - batch->ctx_offsets[b]);
    max_gb = std::max<int64_t>(max_gb, batch->guide_offsets[b + 1] - batch->guide_offsets[b]);
  }
  const int64_t nchunk = (max_nb + a.chunk - 1) / a.chunk;
  const int64_t nrg = (a.R * max_gb + tp::kRowsPerGroup - 1) / tp::kRowsPerGroup;
  if (nchunk + 1 > 0x7FFFFFFF || (int64_t)batch->batch * nrg > 65535)
    return fail(TP_ERR_UNSUPPORTED, "context or guide too long for one launch");
  a.nchunk_max = (int32_t)nchunk;
  a.nrg_max = (int32_t)nrg;
  if (qa) {
    a.scales = qa->scales;
    a.vq = qa->vq;
    a.qfmt = qa->qfmt;
    a.bits = qa->bits;
    a.qmax = qa->qmax;
    a.ro = qa->ro;
  }
  const hipError_t e = tp::launch_guide_attention(a, dims->head_dim, (hipStream_t)stream);
  if (e != hipSuccess) return hip_fail(e, "tp_guide_attention launch");
  return ok();
}

extern "C" {

tp_status tp_guide_attention(const tp_dims* dims, const tp_batch* batch, const void* q_guide, const void* k,
                             const void* v, const void* k_guide, const void* v_guide, float softmax_scale,
                             float* o_guide, float* guide_lse, void* workspace, size_t ws_bytes, void* stream) {
  return guide_attention(dims, batch, q_guide, k, v, k_guide, v_guide, softmax_scale, o_guide, guide_lse, nullptr,
                         workspace, ws_bytes, stream);
}

tp_status tp_guide_attention_quantize(const tp_dims* dims, const tp_batch* batch, const void* q_guide,
                                      const void* k, const void* v, const void* k_guide, const void* v_guide,
                                      float softmax_scale, int32_t qfmt, int32_t bits, float* o_guide,
                                      float* guide_lse, float* scales, void* v_q, void* workspace, size_t ws_bytes,
                                      void* stream) {
  tp::QuantArgs qa;
  const tp_status s = prepare_quant(dims, batch, v, qfmt, bits, scales, v_q, qa);
  if (s != TP_OK) return s;
  if (!v_q) return fail(TP_ERR_NULL, "v_q must be non-NULL (the codes are written with the scales)");
  return guide_attention(dims, batch, q_guide, k, v, k_guide, v_guide, softmax_scale, o_guide, guide_lse, &qa,
                         workspace, ws_bytes, stream);
}

tp_status tp_quantize_v_scales(const tp_dims* dims, const tp_batch* batch, const void* v, int32_t qfmt,
                               int32_t bits, float* scales, void* v_q, void* stream) {
  tp::QuantArgs a;
  const tp_status s = prepare_quant(dims, batch, v, qfmt, bits, scales, v_q, a);
  if (s != TP_OK) return s;
  const hipError_t e = tp::launch_quantize(a, dims->head_dim, (hipStream_t)stream);
  if (e != hipSuccess) return hip_fail(e, "tp_quantize_v_scales launch");
  return ok();
}

tp_status tp_combine_select_topk(const tp_dims* dims, const tp_batch* batch, const float* s_key,
                                 const float* scales, int32_t rule, double keep_ratio, int64_t keep_budget,
                                 const int64_t* kept_offsets, int32_t* kept_idx, float* s_out, void* workspace,
                                 size_t ws_bytes, void* stream) {
  tp::SelectArgs a;
  const tp_status s = prepare_select(dims, batch, s_key, scales, rule, keep_ratio, keep_budget, kept_offsets,
                                     kept_idx, s_out, workspace, ws_bytes, a);
  if (s != TP_OK) return s;
  const hipError_t e = tp::launch_select(a, dims->num_layers * dims->num_kv_heads, (hipStream_t)stream);
  if (e != hipSuccess) return hip_fail(e, "tp_combine_select_topk launch");
  return ok();
}

tp_status tp_combine_select_topk_static(const tp_dims* dims, const tp_batch* batch, const float* s_key,
                                        const float* scales, int32_t rule, double keep_ratio, int64_t keep_budget,
                                        const int64_t* kept_offsets, int32_t* kept_idx, void* stream) {
  tp::SelectArgs a;
  // validated as tp_combine_select_topk with the combined scores staged in a buffer of the
  // static size (a placeholder address here; nothing is enqueued on failure)
  tp_status s = prepare_select(dims, batch, s_key, scales, rule, keep_ratio, keep_budget, kept_offsets, kept_idx,
                               nullptr, kPlaceholder, tp::kStaticScratchBytes, a);
  if (s != TP_OK) {
    if (s == TP_ERR_WORKSPACE)
      return fail(TP_ERR_WORKSPACE, "the selection needs %zu bytes of workspace, more than the static buffer's %zu",
                  select_workspace(dims, batch), (size_t)tp::kStaticScratchBytes);
    return s;
  }
  void* buf = nullptr;
  hipError_t e = tp::static_scratch((hipStream_t)stream, &buf);
  if (e != hipSuccess) return hip_fail(e, "tp_combine_select_topk_static: static buffer");
  rebase_select(a, kPlaceholder, (char*)buf);
  e = tp::launch_select(a, dims->num_layers * dims->num_kv_heads, (hipStream_t)stream);
  if (e != hipSuccess) return hip_fail(e, "tp_combine_select_topk_static launch");
  return ok();
}

tp_status tp_compact_kv(const tp_dims* dims, const tp_batch* batch, const int64_t* kept_offsets,
                        const int32_t* kept_idx, const void* k, const void* v_q, const float* scales, int32_t qfmt,
                        int32_t bits, void* k_out, void* v_q_out, float* scales_out, void* stream) {
  tp::CompactArgs a;
  const tp_status s = prepare_compact(dims, batch, kept_offsets, kept_idx, k, v_q, scales, qfmt, bits, k_out,
                                      v_q_out, scales_out, a);
  if (s != TP_OK) return s;
  const hipError_t e = tp::launch_compact(a, dims->num_layers * dims->num_kv_heads, dims->head_dim, (hipStream_t)stream);
  if (e != hipSuccess) return hip_fail(e, "tp_compact_kv launch");
  return ok();
}

tp_status tp_compact_quantize_kv(const tp_dims* dims, const tp_batch* batch, const int64_t* kept_offsets,
                                 const int32_t* kept_idx, const void* k, const void* v, int32_t qfmt, int32_t bits,
                                 void* k_out, void* v_q_out, float* scales_out, void* stream) {
  tp::CompactArgs a;
  const tp_status s = prepare_compact_quant(dims, batch, kept_offsets, kept_idx, k, v, qfmt, bits, k_out, v_q_out,
                                            scales_out, a);
  if (s != TP_OK) return s;
  const hipError_t e = tp::launch_compact(a, dims->num_layers * dims->num_kv_heads, dims->head_dim, (hipStream_t)stream);
  if (e != hipSuccess) return hip_fail(e, "tp_compact_quantize_kv launch");
  return ok();
}

}  // extern "C"

// tp_evict when step 2 was done beforehand: steps 1, 3 and 4 on the caller's stream only.
// Event [3] (after step 2) follows [2] with no kernel between them.
static tp_status evict_without_step2(const tp::GuideArgs& ga, const tp::SelectArgs& sa, const tp::CompactArgs& ca,
                                     bool fuse_pool, const tp_dims* dims, hipStream_t st, hipEvent_t* ev) {
  struct Rec {
    hipEvent_t done;
    hipStream_t st;
  } rec{ev ? ev[3] : nullptr, st};
  auto mark = [](void* c) -> hipError_t {
    const Rec* r = (const Rec*)c;
    return r->done ? hipEventRecord(r->done, r->st) : hipSuccess;
  };
  const int segs = dims->num_layers * dims->num_kv_heads;
  hipEvent_t gev[4] = {ev ? ev[1] : nullptr, ev ? ev[2] : nullptr, ev ? ev[4] : nullptr,
                       ev && !fuse_pool ? ev[5] : nullptr};
  hipError_t e = hipSuccess;
  if (ev) e = hipEventRecord(ev[0], st);
  if (e == hipSuccess) e = tp::launch_guide_scores(ga, dims->head_dim, st, ev ? gev : nullptr, mark, &rec);
  if (e == hipSuccess) e = tp::launch_select(sa, segs, st, ev && fuse_pool ? ev[5] : nullptr);
  if (e == hipSuccess && ev) e = hipEventRecord(ev[6], st);
  if (e == hipSuccess) e = tp::launch_compact(ca, segs, dims->head_dim, st);
  if (e == hipSuccess && ev) e = hipEventRecord(ev[7], st);
  if (e != hipSuccess) return hip_fail(e, "tp_evict launch");
  return ok();
}

extern "C" {

tp_status tp_evict(const tp_dims* dims, const tp_batch* batch, const void* q_guide, const void* k,
                   const void* k_guide, const float* guide_lse, const void* v, float softmax_scale, int32_t pool_k, int32_t qfmt, int32_t bits, int32_t rule, double keep_ratio,
                   int64_t keep_budget, const int64_t* kept_offsets, float* s_key, float* scales, void* v_q,
                   float* s_out, int32_t* kept_idx, void* k_out, void* v_q_out, float* scales_out, void* workspace,
                   size_t ws_bytes, const tp_profile* profile, void* stream) {
  if (profile && profile->num_events != 0) {
    if (profile->num_events < TP_EVICT_EVENTS)
      return fail(TP_ERR_PARAM, "profile->num_events must be 0 or %d", TP_EVICT_EVENTS);
    for (int i = 0; i < TP_EVICT_EVENTS; ++i)
      if (!profile->events[i]) return fail(TP_ERR_NULL, "profile->events[%d] is NULL", i);
  }
  tp_status s = check_dims(dims);
  if (s != TP_OK) return s;
  s = check_batch(dims, batch, true);
  if (s != TP_OK) return s;
  // workspace: the score pass's, then (without s_out) the combined scores
  const size_t gws = guide_workspace_bytes(dims, batch);
  const size_t ews = evict_workspace_bytes(dims, batch);
  if (!workspace || ws_bytes < ews) return fail(TP_ERR_WORKSPACE, "workspace needs %zu bytes (got %zu)", ews, ws_bytes);
  tp::GuideArgs ga;
  s = prepare_guide(dims, batch, q_guide, k, k_guide, guide_lse, softmax_scale, pool_k, s_key, workspace, gws, ga);
  if (s != TP_OK) return s;
  // v == NULL: step 2 is done (tp_guide_attention_quantize): scales and v_q are its results
  const bool step2 = v != nullptr;
  tp::QuantArgs qa;
  memset(&qa, 0, sizeof qa);
  if (step2) {
    s = prepare_quant(dims, batch, v, qfmt, bits, scales, v_q, qa);
    if (s != TP_OK) return s;
  } else if (!scales || !v_q) {
    return fail(TP_ERR_NULL, "without v, scales and v_q must hold step 2's results");
  }
  tp::SelectArgs sa;
  s = prepare_select(dims, batch, s_key, scales, rule, keep_ratio, keep_budget, kept_offsets, kept_idx, s_out,
                     (char*)workspace + gws, ews - gws, sa);
  if (s != TP_OK) return s;
  // Every rule but NORM_ADD (whose norms need the pooled scores first) pools score pass 2's
  // raw sums inside the selection's first kernel, which writes s_key: no pooling kernel.
  const bool fuse_pool = rule != TP_COMBINE_NORM_ADD;
  if (fuse_pool) {
    ga.skip_pool = 1;
    sa.raw = ga.raw;
    sa.s_key_out = s_key;
    sa.pool_inv = ga.pool_inv;
    sa.pool_half = ga.pool_half;
    for (int b = 0; b < batch->batch; ++b)
      sa.nrg[b] = (int32_t)((ga.R * (batch->guide_offsets[b + 1] - batch->guide_offsets[b]) + tp::kRowsPerGroup - 1) /
                            tp::kRowsPerGroup);
  }
  tp::CompactArgs ca;
  // without v_q the codes of the evicted rows are never written: the compaction quantises
  // the kept V rows itself (same codes and scales)
  if (v_q)
    s = prepare_compact(dims, batch, kept_offsets, kept_idx, k, v_q, scales, qfmt, bits, k_out, v_q_out, scales_out, ca);
  else
    s = prepare_compact_quant(dims, batch, kept_offsets, kept_idx, k, v, qfmt, bits, k_out, v_q_out, scales_out, ca);
  if (s != TP_OK) return s;

  const hipStream_t st = (hipStream_t)stream;
  hipEvent_t* ev = (profile && profile->num_events) ? (hipEvent_t*)profile->events : nullptr;
  if (!step2) return evict_without_step2(ga, sa, ca, fuse_pool, dims, st, ev);
  AuxStream* aux = nullptr;
  s = aux_stream_for(st, aux);
  if (s != TP_OK) return s;
  std::lock_guard<std::mutex> lk(aux->enqueue);

  // Step 2 is split by rows of V, each row quantised once, by one of three launches with the
  // same arithmetic.  The lean kernel, on the second stream, takes the first part while score
  // pass 1 runs (its workgroups leave one wave slot and 48 VGPRs per SIMD free, and it uses
  // HBM well below the copy rate) and the last part while pass 2 runs; the regular kernel
  // takes the middle part between the normalisers and pass 2, which then starts after a
  // memory-bound kernel instead of right after pass 1, at a higher power-limited clock.
  // With pass 1 each lean part is 2/5 of the rows (the middle fifth runs alone), or half
  // when only the scales are written (lighter, so all of it fits beside the passes); with the
  // normalisers given (no pass 1) the lean kernel takes the first half (3/5 for scales only)
  // and nothing runs beside pass 2.  Parts are rounded down to 64 rows.
  const bool pass1 = ga.lse_in == nullptr;
  const bool codes = qa.vq != nullptr;
  const int64_t num = pass1 ? (codes ? 2 : 1) : (codes ? 1 : 3), den = pass1 ? (codes ? 5 : 2) : (codes ? 2 : 5);
  const int64_t r_lean = qa.rows * num / den / 64 * 64;
  const int64_t r_mid_end = pass1 ? qa.rows - r_lean : qa.rows;
  const int64_t vrow = (int64_t)row_bytes_of(qfmt, bits, dims->head_dim);
  auto part = [&](int64_t r0, int64_t r1) {
    tp::QuantArgs p = qa;
    p.rows = r1 - r0;
    p.v += r0 * dims->head_dim;
    p.scales += r0;
    if (p.vq) p.vq += r0 * vrow;
    return p;
  };
  const tp::QuantArgs qa1 = part(0, r_lean), qa2 = part(r_lean, r_mid_end), qa3 = part(r_mid_end, qa.rows);
  hipError_t e = hipSuccess;
  if (ev) e = hipEventRecord(ev[0], st);
  if (e == hipSuccess) e = hipEventRecord(aux->fork, st);
  if (e == hipSuccess) e = hipStreamWaitEvent(aux->stream, aux->fork, 0);
  if (e == hipSuccess) e = tp::launch_quantize_lean(qa1, dims->head_dim, aux->stream);
  if (e == hipSuccess) e = hipEventRecord(aux->part1, aux->stream);  // the first part's scales are written
  // called by the score pass between the normalisers and pass 2 (exactly once on success)
  struct Mid {
    const tp::QuantArgs* mid;
    const tp::QuantArgs* last;
    int head_dim;
    hipStream_t st;
    hipEvent_t done;
    AuxStream* aux;
  } mid{&qa2, &qa3, dims->head_dim, st, ev ? ev[3] : nullptr, aux};
  auto quant_between = [](void* c) -> hipError_t {
    const Mid* m = (const Mid*)c;
    hipError_t r = tp::launch_quantize(*m->mid, m->head_dim, m->st);
    if (r == hipSuccess && m->done) r = hipEventRecord(m->done, m->st);
    if (r == hipSuccess && m->last->rows > 0) {
      r = hipEventRecord(m->aux->fork2, m->st);
      if (r == hipSuccess) r = hipStreamWaitEvent(m->aux->stream, m->aux->fork2, 0);
      if (r == hipSuccess) r = tp::launch_quantize_lean(*m->last, m->head_dim, m->aux->stream);
    }
    if (r == hipSuccess) r = hipEventRecord(m->aux->join, m->aux->stream);
    return r;
  };
  hipEvent_t gev[4] = {ev ? ev[1] : nullptr, ev ? ev[2] : nullptr, ev ? ev[4] : nullptr,
                       ev && !fuse_pool ? ev[5] : nullptr};
  if (e == hipSuccess)
    e = tp::launch_guide_scores(ga, dims->head_dim, st, ev ? gev : nullptr, quant_between, &mid);
  // The selection reads the scales.  Segments whose V rows all belong to parts of step 2
  // already done in this stream's order form their combined scores while the second stream
  // finishes its last part; the rest wait for it.  With pass 1 those are the rows before the
  // part beside pass 2 (the first part, on the second stream, is waited for by its own
  // event); with the normalisers given, the rows after the second stream's part.
  const int segs = dims->num_layers * dims->num_kv_heads;
  const int64_t n_tot = batch->ctx_offsets[batch->batch];
  int rb = 0, re = 0;  // segments [rb, re) scored before the join
  if (fuse_pool) {
    if (pass1) {
      re = (int)std::min<int64_t>(segs, r_mid_end / n_tot);
    } else {
      rb = (int)std::min<int64_t>(segs, (r_lean + n_tot - 1) / n_tot);
      re = segs;
    }
  }
  if (e == hipSuccess && re > rb && pass1) e = hipStreamWaitEvent(st, aux->part1, 0);
  if (e == hipSuccess) e = tp::launch_select_score(sa, rb, re, segs, st);
  if (e != hipSuccess) {
    // Work may already sit on the second stream (it was forked from `st` before the failure):
    // join it back, best effort, so nothing the caller's stream orders after this call can
    // overtake a quantisation part still writing the caller's buffers.
    join_after_failure(aux, st);
    return hip_fail(e, "tp_evict launch");
  }
  e = hipStreamWaitEvent(st, aux->join, 0);
  if (e == hipSuccess) e = tp::launch_select(sa, segs, st, ev && fuse_pool ? ev[5] : nullptr, rb, re);
  if (e == hipSuccess && ev) e = hipEventRecord(ev[6], st);
  if (e == hipSuccess) e = tp::launch_compact(ca, dims->num_layers * dims->num_kv_heads, dims->head_dim, st);
  if (e == hipSuccess && ev) e = hipEventRecord(ev[7], st);
  if (e != hipSuccess) return hip_fail(e, "tp_evict launch");
  return ok();
}

}  // extern "C"
