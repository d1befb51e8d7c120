// Internal declarations shared by the C-ABI layer and the gfx950 kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "quant_recip_table.h"
#include "taskpress.h"

namespace tp {

// Batch description passed by value in kernel arguments (no device staging).
struct BatchArgs {
  int32_t batch;
  int32_t pad_;
  int64_t ctx_off[TP_MAX_BATCH + 1];
  int64_t g_off[TP_MAX_BATCH + 1];
};

// ---------------------------------------------------------------- step 1 (guide scores)
constexpr int kGuideThreads = 512;       // 8 waves of 64, two per SIMD
constexpr int kGuideWaves = kGuideThreads / 64;
constexpr int kRowsPerGroup = 256;       // guide rows handled by one workgroup
// Context tokens of one segment per score-pass workgroup (a "chunk"): 16384 when every
// sequence of the batch has at least 65536 context tokens, so the per-workgroup query
// staging and statistics merge are spread over more tokens; else 8192, so short and ragged
// sequences keep enough workgroups and little padding.
constexpr int kChunkSmall = 8192;
constexpr int kChunkLarge = 16384;
constexpr int64_t kLongContext = 65536;
inline int32_t chunk_tokens(const int64_t* ctx_off, int32_t batch) {
  for (int b = 0; b < batch; ++b)
    if (ctx_off[b + 1] - ctx_off[b] < kLongContext) return kChunkSmall;
  return kChunkLarge;
}

struct GuideArgs {
  const uint16_t* q;  // bf16 [L][Hq][G_tot][d]
  const uint16_t* k;  // bf16 [L][Hkv][N_tot][d]
  const uint16_t* kg; // bf16 [L][Hkv][G_tot][d] guide keys, or nullptr (context-only normaliser)
  const float* lse_in;// fp32 [L][Hq][G_tot] caller's natural-log row normalisers, or nullptr
  float* s_key;       // fp32 [L][Hkv][N_tot]
  float2* stats;      // [nchunk_max + 1][L*Hq*G_tot] per-chunk (max, sum) in the log2 domain;
                      //   slot nchunk_max: the guide keys' terms (with kg)
  float* lse2;        // [L*Hq*G_tot]               log2-sum-exp2 of the row's normaliser
  float* raw;         // [nrg_max][L*Hkv][N_tot]    per row-group sums of normalised attention
  int32_t L, Hq, Hkv, R;
  int64_t n_tot, g_tot;
  float c;            // softmax_scale * log2(e)
  float pool_inv;     // 1 / (R * pool_k)
  int32_t pool_half;  // pool_k / 2
  int32_t chunk;      // context tokens per chunk (chunk_tokens of the batch)
  int32_t nchunk_max; // chunks of the longest sequence
  int32_t nrg_max;    // row groups of the largest R * G_b
  BatchArgs bt;
  // first workgroup of each sequence's range in the score passes: sequence b has
  // ceil(L * Hkv * nchunk_b / 8) * 8 * nrg_b workgroups
  int32_t wg_off[TP_MAX_BATCH + 1];
  // the pooling kernel is left out (the split selection pools the raw sums itself)
  int32_t skip_pool;
};

struct GuideWorkspace {
  size_t stats_off, lse_off, raw_off, total;
};
GuideWorkspace guide_workspace_layout(int32_t L, int32_t Hq, int32_t Hkv, const int64_t* ctx_off,
                                      const int64_t* g_off, int32_t batch);

// ev (optional): 4 events recorded after the stats, lse, attention and pooling kernels.
// between (optional): called with ctx once the row normalisers are enqueued and before
// pass 2, to put independent work on the stream there.
typedef hipError_t (*GuideBetween)(void* ctx);
hipError_t launch_guide_scores(const GuideArgs& a, int head_dim, hipStream_t stream, hipEvent_t* ev,
                               GuideBetween between = nullptr, void* ctx = nullptr);

// ---------------------------------------------------------------- step 2 (V scales)
// The one-multiply multipliers of the format with this qmax, per absmax significand t: the
// ulp offset from fl32(1/fl32(m/qmax)) (-1, 0, 1), or kNoMultiplier where there is none (also
// for every t of a qmax the table does not hold, which keeps the corrected quotient).
constexpr int8_t kNoMultiplier = 2;
struct RecipOffsets {
  int8_t off[128];
};
inline RecipOffsets recip_offsets_for(float qmax) {
  RecipOffsets r;
  const RecipMasks* m = nullptr;
  for (int f = 0; f < 8; ++f)
    if (kRecipQmax[f] == qmax) m = &kRecipMasks[f];
  for (int t = 0; t < 128; ++t) {
    const int w = t >> 6, b = t & 63;
    if (m == nullptr || ((m->none[w] >> b) & 1u))
      r.off[t] = kNoMultiplier;
    else
      r.off[t] = (int8_t)(((m->up[w] >> b) & 1u) ? 1 : ((m->down[w] >> b) & 1u) ? -1 : 0);
  }
  return r;
}

struct QuantArgs {
  const uint16_t* v;  // bf16 [rows][d]
  float* scales;      // fp32 [rows]
  uint8_t* vq;        // [rows][row_bytes] or nullptr
  int64_t rows;       // L * Hkv * N_tot
  int32_t qfmt, bits;
  float qmax;
  RecipOffsets ro;    // recip_offsets_for(qmax)
};
hipError_t launch_quantize(const QuantArgs& a, int head_dim, hipStream_t stream);

// The same quantisation in a form that stays resident beside a score-pass workgroup (one
// workgroup per CU, one wave per SIMD, at most 48 VGPRs), for running part of step 2 on a
// second stream concurrently with the score passes.
hipError_t launch_quantize_lean(const QuantArgs& a, int head_dim, hipStream_t stream);

// ---------------------------------------------------------------- guide rows' prefill attention
// Context tokens per workgroup of the guide rows' attention: 32768 when every sequence has at
// least 131072 (fewer partial outputs to merge), else 8192.
constexpr int kAttnChunkSmall = 8192;
constexpr int kAttnChunkLarge = 32768;
inline int32_t attn_chunk_tokens(const int64_t* ctx_off, int32_t batch) {
  for (int b = 0; b < batch; ++b)
    if (ctx_off[b + 1] - ctx_off[b] < 131072) return kAttnChunkSmall;
  return kAttnChunkLarge;
}

struct AttnArgs {
  const uint16_t* q;   // bf16 [L][Hq][G_tot][d]
  const uint16_t* k;   // bf16 [L][Hkv][N_tot][d]
  const uint16_t* v;   // bf16 [L][Hkv][N_tot][d]
  const uint16_t* kg;  // bf16 [L][Hkv][G_tot][d] the guide tokens' keys, or nullptr
  const uint16_t* vg;  // bf16 [L][Hkv][G_tot][d] their values (with kg)
  float* o;            // fp32 [L][Hq][G_tot][d]  attention output of the guide rows
  float* lse;          // fp32 [L][Hq][G_tot]     natural log of each row's normaliser
  float2* pstat;       // [nchunk_max + 1][L*Hq*G_tot] per chunk (max, sum), log2 domain; last slot: guide keys
  float* po;           // [nchunk_max + 1][L*Hq*G_tot][d] per chunk unnormalised output
  int32_t L, Hq, Hkv, R;
  int64_t n_tot, g_tot;
  float c;             // softmax_scale * log2(e)
  int32_t chunk;       // attn_chunk_tokens of the batch
  int32_t nchunk_max;  // chunks of the longest sequence
  int32_t nrg_max;     // row groups of the largest R * G_b
  BatchArgs bt;
  // Step 2 from the staged V sub-tiles (tp_guide_attention_quantize); vq == nullptr: none.
  float* scales;       // fp32 [L][Hkv][N_tot]
  uint8_t* vq;         // [L][Hkv][N_tot][row_bytes]
  int32_t qfmt, bits;
  float qmax;
  RecipOffsets ro;     // recip_offsets_for(qmax)
};

struct AttnWorkspace {
  size_t pstat_off, po_off, total;
};
AttnWorkspace attn_workspace_layout(int32_t L, int32_t Hq, int32_t Hkv, int32_t head_dim, const int64_t* ctx_off,
                                    const int64_t* g_off, int32_t batch);
hipError_t launch_guide_attention(const AttnArgs& a, int head_dim, hipStream_t stream);

// ---------------------------------------------------------------- step 3 (select)
// Every rule but NORM_ADD runs the split selection: each segment's tokens are cut into parts
// of kSelPartTokens, one workgroup per part in the passes over the scores.
constexpr int kSelPartTokens = 8192;
constexpr int kSelCandCap = 8192;  // keys of the threshold's top-digit bucket kept per segment

struct SelectArgs {
  const float* s_key;  // fp32 [L*Hkv][N_tot]  (read unless `raw` is set)
  const float* scales; // fp32 [L*Hkv][N_tot]
  float* s_buf;        // fp32 [L*Hkv][N_tot]   combined scores (s_out or workspace)
  int32_t* kept;       // int32 [L*Hkv][K_tot]
  int64_t n_tot, k_tot;
  int32_t rule;
  int32_t pad_;
  int64_t k[TP_MAX_BATCH];
  int64_t kept_off[TP_MAX_BATCH + 1];
  BatchArgs bt;
  // Pooling fused into the split selection (tp_evict): the key score is pooled here from score
  // pass 2's per-row-group sums and written to s_key_out; nullptr reads s_key instead.
  const float* raw;    // [nrg][L*Hkv][N_tot]
  float* s_key_out;    // fp32 [L*Hkv][N_tot]
  float pool_inv;      // 1 / (R * pool_k)
  int32_t pool_half;   // pool_k / 2
  int32_t nrg[TP_MAX_BATCH];  // row groups of sequence b
  // Workspace of the split selection (select_workspace_layout):
  uint32_t* hist;      // [L*Hkv][part_tot][kBins/2]  per-part top-digit counts, two 16-bit per word
  uint4* info;         // [L*Hkv][batch]  top digit of the k-th key, keys still needed, bucket size
  uint2* thr;          // [L*Hkv][batch]  threshold key T, keys equal to T to keep
  uint2* pcount;       // [L*Hkv][part_tot]  per part: keys above the top digit, keys in it
  uint2* pref;         // [L*Hkv][part_tot]  per part: keys > T and keys == T in earlier parts
  uint32_t* cstart;    // [L*Hkv][part_tot]  per part: its first slot in the candidate list
  uint32_t* cand;      // [L*Hkv][cand_tot]  the top-digit bucket's keys
  int64_t part_tot, cand_tot;
  int64_t part_off[TP_MAX_BATCH + 1];  // parts of the sequences before b
  int64_t cand_off[TP_MAX_BATCH + 1];  // candidate slots of the sequences before b
  int32_t part_max;    // parts of the longest sequence
  int32_t pad2_;
};

struct SelectWorkspace {
  size_t s_off, hist_off, info_off, thr_off, pcount_off, pref_off, cstart_off, cand_off, total;
  int64_t part_tot, cand_tot;
};
// Layout of the selection's workspace: the combined scores (unless s_out is given), then the
// split selection's buffers.  segments = L * Hkv.
SelectWorkspace select_workspace_layout(int64_t segments, const int64_t* ctx_off, int32_t batch);

// after_score (optional): recorded once the combined scores are formed (after the pooling
// fused into the split selection, when `raw` is set).  [scored_begin, scored_end): segments
// whose combined scores launch_select_score has already enqueued (the split selection only).
hipError_t launch_select(const SelectArgs& a, int segments, hipStream_t stream, hipEvent_t after_score = nullptr,
                         int scored_begin = 0, int scored_end = 0);
// The split selection's first kernel for segments [seg_begin, seg_end) of `segments` (none for
// NORM_ADD), so a caller can form the scores of segments whose inputs are ready early.
hipError_t launch_select_score(const SelectArgs& a, int seg_begin, int seg_end, int segments, hipStream_t stream);

// The library's static staging buffer for the selection (tp_combine_select_topk_static): the
// device address of the calling stream's GPU's copy, resolved on the first call on that GPU.
constexpr size_t kStaticScratchBytes = (size_t)TP_STATIC_SCRATCH_BYTES;
hipError_t static_scratch(hipStream_t stream, void** ptr);

// ---------------------------------------------------------------- step 4 (compaction)
struct CompactArgs {
  const int32_t* kept; // [L*Hkv][K_tot]
  const uint16_t* k;   // bf16 [L*Hkv][N_tot][d]
  const uint16_t* v;   // bf16 [L*Hkv][N_tot][d]: quantise the kept V rows while gathering, or nullptr
  const uint8_t* vq;   // [L*Hkv][N_tot][row_bytes] or nullptr
  const float* scales; // [L*Hkv][N_tot] or nullptr
  uint16_t* k_out;     // [L*Hkv][K_tot][d]
  uint8_t* vq_out;
  float* scales_out;
  int64_t n_tot, k_tot;
  int32_t row_bytes;
  int32_t qfmt, bits;  // format of the codes when v is set
  float qmax;
  RecipOffsets ro;     // recip_offsets_for(qmax)
  int64_t kept_off[TP_MAX_BATCH + 1];
  BatchArgs bt;
};
hipError_t launch_compact(const CompactArgs& a, int segments, int head_dim, hipStream_t stream);

}  // namespace tp
