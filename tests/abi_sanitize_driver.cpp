// Host-side driver of the C ABI for the sanitizer build (tests/test_abi_sanitized.py): every
// entry point with arguments that must fail validation, the host-only helpers at their edges,
// offsets and shapes chosen to overflow careless size arithmetic, and, only when the HIP
// runtime sees no device, well-formed calls that must end in TP_ERR_HIP.  The library under
// test is built with AddressSanitizer and UBSan on its host side; fake device pointers are
// never dereferenced by correct host code.  Exit status 0 when every check holds.
#include <hip/hip_runtime_api.h>

#include <climits>
#include <cmath>
#include <cstdint>
#include <cstdio>
#include <cstring>
#include <vector>

#include "taskpress.h"

namespace {

int failures = 0;
int checks = 0;

void expect(tp_status got, tp_status want, const char* what, int line) {
  ++checks;
  if (got != want) {
    std::fprintf(stderr, "line %d: %s returned %d, expected %d (%s)\n", line, what, got, want, tp_last_error());
    ++failures;
    return;
  }
  if (want != TP_OK && std::strlen(tp_last_error()) == 0) {
    std::fprintf(stderr, "line %d: %s failed without a message\n", line, what);
    ++failures;
  }
}
#define EXPECT(call, want) expect((call), (want), #call, __LINE__)

void expect_true(bool ok, const char* what, int line) {
  ++checks;
  if (!ok) {
    std::fprintf(stderr, "line %d: %s\n", line, what);
    ++failures;
  }
}
#define EXPECT_TRUE(cond) expect_true((cond), #cond, __LINE__)

char* fake(size_t off = 0) { return reinterpret_cast<char*>(0x10000) + off; }  // 256-byte aligned, never read

struct Batch {
  std::vector<int64_t> ctx, guide;
  tp_batch c{};
  Batch(std::vector<int64_t> ctx_, std::vector<int64_t> guide_ = {}) : ctx(std::move(ctx_)), guide(std::move(guide_)) {
    c.batch = (int32_t)ctx.size() - 1;
    c.ctx_offsets = ctx.data();
    c.guide_offsets = guide.empty() ? nullptr : guide.data();
  }
  Batch(const Batch&) = delete;
};

std::vector<int64_t> kept_offsets(const Batch& bt, double ratio, int64_t budget) {
  std::vector<int64_t> ko{0};
  for (int b = 0; b < bt.c.batch; ++b) ko.push_back(ko.back() + tp_keep_count(bt.ctx[b + 1] - bt.ctx[b], ratio, budget));
  return ko;
}

size_t ws_size(int32_t fn, const tp_dims& d, const Batch& bt) {
  size_t n = 0;
  EXPECT(tp_workspace_size(fn, &d, &bt.c, &n), TP_OK);
  return n;
}

// tp_guide_scores with defaults that pass validation
struct GS {
  const tp_dims* d;
  const tp_batch* bt;
  const void* q = fake();
  const void* k = fake();
  const void* kg = nullptr;
  float scale = 0.125f;
  int32_t pool = 5;
  float* s = (float*)fake();
  void* ws = fake();
  size_t wsb = (size_t)1 << 40;
  tp_status run() const { return tp_guide_scores(d, bt, q, k, kg, scale, pool, s, ws, wsb, nullptr); }
};

struct EV {
  const tp_dims* d;
  const tp_batch* bt;
  const void* q = fake();
  const void* k = fake();
  const void* kg = nullptr;
  const float* lse = nullptr;
  const void* v = fake();
  float scale = 0.125f;
  int32_t pool = 5, qfmt = TP_QFMT_INT, bits = 8, rule = TP_COMBINE_MUL;
  double ratio = 0.25;
  int64_t budget = 0;
  const int64_t* ko = nullptr;
  float* skey = (float*)fake();
  float* sc = (float*)fake();
  void* vq = fake();
  float* sout = (float*)fake();
  int32_t* idx = (int32_t*)fake();
  void* kout = fake();
  void* vqout = fake();
  float* scout = (float*)fake();
  void* ws = fake();
  size_t wsb = (size_t)1 << 40;
  const tp_profile* prof = nullptr;
  tp_status run() const {
    return tp_evict(d, bt, q, k, kg, lse, v, scale, pool, qfmt, bits, rule, ratio, budget, ko, skey, sc, vq, sout, idx,
                    kout, vqout, scout, ws, wsb, prof, nullptr);
  }
};

void host_helpers() {
  EXPECT_TRUE(tp_version() != nullptr && std::strlen(tp_version()) > 0);
  for (int s = -3; s < 12; ++s) EXPECT_TRUE(tp_status_string(s) != nullptr);
  EXPECT_TRUE(tp_last_error() != nullptr);
  EXPECT_TRUE(tp_keep_count(100, 0.25, 0) == 25);
  EXPECT_TRUE(tp_keep_count(100, 0.0, 7) == 7);
  EXPECT_TRUE(tp_keep_count(5, 0.0, 7) == 5);
  // extremes: defined answers, no overflow
  (void)tp_keep_count(INT64_MAX, 1.0, 0);
  (void)tp_keep_count(INT64_MAX, 1e-300, 0);
  (void)tp_keep_count(INT64_MAX, 0.0, INT64_MAX);
  (void)tp_keep_count(1, std::nan(""), 0);
  (void)tp_keep_count(1, -1.0, -5);
  (void)tp_keep_count(0, 0.5, 0);
  (void)tp_keep_count(-4, 0.5, 0);
}

void workspace_sizes() {
  const tp_dims d{32, 32, 8, 128};
  Batch bt({0, 131072}, {0, 64});
  size_t n = 0;
  for (int fn = 0; fn < 4; ++fn) EXPECT_TRUE(ws_size(fn, d, bt) > 0);
  EXPECT(tp_workspace_size(7, &d, &bt.c, &n), TP_ERR_PARAM);
  EXPECT(tp_workspace_size(-1, &d, &bt.c, &n), TP_ERR_PARAM);
  EXPECT(tp_workspace_size(0, nullptr, &bt.c, &n), TP_ERR_NULL);
  EXPECT(tp_workspace_size(0, &d, nullptr, &n), TP_ERR_NULL);
  EXPECT(tp_workspace_size(0, &d, &bt.c, nullptr), TP_ERR_NULL);
  Batch noguide({0, 131072});
  EXPECT(tp_workspace_size(TP_FN_GUIDE_SCORES, &d, &noguide.c, &n), TP_ERR_NULL);
  EXPECT(tp_workspace_size(TP_FN_GUIDE_ATTENTION, &d, &noguide.c, &n), TP_ERR_NULL);
  EXPECT(tp_workspace_size(TP_FN_COMBINE_SELECT_TOPK, &d, &noguide.c, &n), TP_OK);
  EXPECT_TRUE(ws_size(TP_FN_EVICT, d, bt) == ws_size(TP_FN_GUIDE_SCORES, d, bt) + ws_size(TP_FN_COMBINE_SELECT_TOPK, d, bt));
}

// Offsets and shapes that would overflow 64-bit size arithmetic or a 32-bit launch grid: each
// must be refused before any size is computed from them.
void hostile_shapes() {
  const tp_dims d{2, 8, 2, 64};
  size_t n = 0;
  {
    Batch bt({0, 1, INT64_MIN}, {0, 16, 32});
    EXPECT(tp_workspace_size(TP_FN_GUIDE_SCORES, &d, &bt.c, &n), TP_ERR_SHAPE);
  }
  {
    Batch bt({0, INT64_MAX}, {0, 16});
    const tp_status s = tp_workspace_size(TP_FN_GUIDE_SCORES, &d, &bt.c, &n);
    EXPECT_TRUE(s == TP_ERR_UNSUPPORTED || s == TP_ERR_SHAPE);
    const tp_status s2 = tp_workspace_size(TP_FN_COMBINE_SELECT_TOPK, &d, &bt.c, &n);
    EXPECT_TRUE(s2 == TP_ERR_UNSUPPORTED || s2 == TP_ERR_SHAPE);
    const tp_status s3 = tp_workspace_size(TP_FN_GUIDE_ATTENTION, &d, &bt.c, &n);
    EXPECT_TRUE(s3 == TP_ERR_UNSUPPORTED || s3 == TP_ERR_SHAPE);
  }
  {
    Batch bt({0, INT64_MAX / 2, INT64_MAX}, {0, 16, INT64_MAX});
    const tp_status s = tp_workspace_size(TP_FN_EVICT, &d, &bt.c, &n);
    EXPECT_TRUE(s == TP_ERR_UNSUPPORTED || s == TP_ERR_SHAPE);
  }
  {
    const tp_dims big{INT32_MAX, INT32_MAX, 1, 128};
    Batch bt({0, 1 << 20}, {0, 64});
    const tp_status s = tp_workspace_size(TP_FN_GUIDE_SCORES, &big, &bt.c, &n);
    EXPECT_TRUE(s == TP_ERR_UNSUPPORTED || s == TP_ERR_SHAPE);
    const tp_status s2 = tp_workspace_size(TP_FN_COMBINE_SELECT_TOPK, &big, &bt.c, &n);
    EXPECT_TRUE(s2 == TP_ERR_UNSUPPORTED || s2 == TP_ERR_SHAPE);
  }
  {
    // past the launch limits though the sizes fit in 64 bits: 2^30 + 1 context tokens, and
    // 2^26 + 1 guide rows of one sequence
    Batch wide({0, ((int64_t)1 << 30) + 1}, {0, 16});
    EXPECT(tp_workspace_size(TP_FN_COMBINE_SELECT_TOPK, &d, &wide.c, &n), TP_ERR_UNSUPPORTED);
    const tp_dims one{1, 1, 1, 64};
    Batch rows({0, 100}, {0, ((int64_t)1 << 26) + 1});
    EXPECT(tp_workspace_size(TP_FN_GUIDE_ATTENTION, &one, &rows.c, &n), TP_ERR_UNSUPPORTED);
    Batch rows_ok({0, 100}, {0, (int64_t)1 << 20});
    EXPECT(tp_workspace_size(TP_FN_GUIDE_ATTENTION, &one, &rows_ok.c, &n), TP_OK);
  }
  {
    const tp_dims neg{-2, 8, 2, 64};
    Batch bt({0, 100}, {0, 16});
    EXPECT(tp_workspace_size(TP_FN_GUIDE_SCORES, &neg, &bt.c, &n), TP_ERR_SHAPE);
    const tp_dims zero_kv{2, 8, 0, 64};
    EXPECT(tp_workspace_size(TP_FN_GUIDE_SCORES, &zero_kv, &bt.c, &n), TP_ERR_SHAPE);
  }
  {
    // a kept-offset table that would overflow when summed or compared carelessly
    const tp_dims d1{1, 1, 1, 64};
    Batch bt({0, 100});
    const int64_t ko[2] = {0, INT64_MIN};
    EXPECT(tp_combine_select_topk(&d1, &bt.c, (const float*)fake(), (const float*)fake(), TP_COMBINE_MUL, 0.25, 0, ko,
                                  (int32_t*)fake(), (float*)fake(), fake(), (size_t)1 << 40, nullptr),
           TP_ERR_SHAPE);
    const int64_t ko2[2] = {INT64_MAX, 5};
    EXPECT(tp_compact_kv(&d1, &bt.c, ko2, (const int32_t*)fake(), fake(), fake(), (const float*)fake(), TP_QFMT_INT, 8,
                         fake(), fake(), (float*)fake(), nullptr),
           TP_ERR_SHAPE);
  }
}

void guide_scores_cases() {
  const tp_dims d{2, 8, 2, 64};
  Batch bt({0, 100, 300}, {0, 16, 20});
  const auto gs = [&]() {
    GS g;
    g.d = &d;
    g.bt = &bt.c;
    return g;
  };
  GS g = gs();
  g.q = nullptr;
  EXPECT(g.run(), TP_ERR_NULL);
  g = gs(), g.k = nullptr;
  EXPECT(g.run(), TP_ERR_NULL);
  g = gs(), g.s = nullptr;
  EXPECT(g.run(), TP_ERR_NULL);
  for (float bad : {0.0f, -1.0f, INFINITY, NAN}) {
    g = gs(), g.scale = bad;
    EXPECT(g.run(), TP_ERR_PARAM);
  }
  for (int32_t bad : {4, 0, -5}) {
    g = gs(), g.pool = bad;
    EXPECT(g.run(), TP_ERR_PARAM);
  }
  g = gs(), g.ws = nullptr;
  EXPECT(g.run(), TP_ERR_WORKSPACE);
  g = gs(), g.wsb = 100;
  EXPECT(g.run(), TP_ERR_WORKSPACE);
  g = gs(), g.ws = fake(16);
  EXPECT(g.run(), TP_ERR_WORKSPACE);
  g = gs(), g.q = fake(2);
  EXPECT(g.run(), TP_ERR_PARAM);
  g = gs(), g.kg = fake(8);
  EXPECT(g.run(), TP_ERR_PARAM);
  const tp_dims d_mod{2, 8, 3, 64}, d_hd{2, 8, 2, 96}, d_l0{0, 8, 2, 64};
  g = gs(), g.d = &d_mod;
  EXPECT(g.run(), TP_ERR_SHAPE);
  g = gs(), g.d = &d_hd;
  EXPECT(g.run(), TP_ERR_UNSUPPORTED);
  g = gs(), g.d = &d_l0;
  EXPECT(g.run(), TP_ERR_SHAPE);
  g = gs(), g.d = nullptr;
  EXPECT(g.run(), TP_ERR_NULL);
  g = gs(), g.bt = nullptr;
  EXPECT(g.run(), TP_ERR_NULL);
  Batch empty_seq({0, 100, 100}, {0, 16, 20}), empty_guide({0, 100, 300}, {0, 16, 16}), bad0({1, 100, 300}, {0, 16, 20}),
      noguide({0, 100, 300});
  for (const Batch* b : {&empty_seq, &empty_guide, &bad0}) {
    g = gs(), g.bt = &b->c;
    EXPECT(g.run(), TP_ERR_SHAPE);
  }
  g = gs(), g.bt = &noguide.c;
  EXPECT(g.run(), TP_ERR_NULL);
  std::vector<int64_t> many;
  for (int i = 0; i < 66; ++i) many.push_back(i);
  Batch toomany(many, many);
  g = gs(), g.bt = &toomany.c;
  EXPECT(g.run(), TP_ERR_UNSUPPORTED);
  Batch zero({0});
  g = gs(), g.bt = &zero.c;
  EXPECT(g.run(), TP_ERR_SHAPE);

  const size_t wsb = ws_size(TP_FN_GUIDE_SCORES, d, bt);
  const auto gl = [&](const float* lse, float scale, int32_t pool, void* ws, size_t nb, const tp_batch* b) {
    return tp_guide_scores_lse(&d, b, fake(), fake(), lse, scale, pool, (float*)fake(), ws, nb, nullptr);
  };
  EXPECT(gl(nullptr, 0.125f, 5, fake(), wsb, &bt.c), TP_ERR_NULL);
  EXPECT(gl((const float*)fake(2), 0.125f, 5, fake(), wsb, &bt.c), TP_ERR_PARAM);
  EXPECT(gl((const float*)fake(), -1.0f, 5, fake(), wsb, &bt.c), TP_ERR_PARAM);
  EXPECT(gl((const float*)fake(), 0.125f, 4, fake(), wsb, &bt.c), TP_ERR_PARAM);
  EXPECT(gl((const float*)fake(), 0.125f, 5, fake(), wsb - 1, &bt.c), TP_ERR_WORKSPACE);
  EXPECT(gl((const float*)fake(), 0.125f, 5, fake(), wsb, &noguide.c), TP_ERR_NULL);
}

void attention_cases() {
  const tp_dims d{2, 8, 2, 64};
  Batch bt({0, 100, 300}, {0, 16, 20}), noguide({0, 100, 300});
  const size_t ws = ws_size(TP_FN_GUIDE_ATTENTION, d, bt);
  struct A {
    const void *q = fake(), *k = fake(), *v = fake(), *kg = nullptr, *vg = nullptr;
    float scale = 0.125f;
    float *o = (float*)fake(), *lse = (float*)fake();
    void* w = fake();
    size_t wsb = 0;
    const tp_batch* b = nullptr;
  };
  const tp_dims* dp = &d;
  const auto run = [&](const A& a) {
    return tp_guide_attention(dp, a.b, a.q, a.k, a.v, a.kg, a.vg, a.scale, a.o, a.lse, a.w, a.wsb, nullptr);
  };
  const auto base = [&]() {
    A a;
    a.wsb = ws;
    a.b = &bt.c;
    return a;
  };
  A a = base();
  a.v = nullptr;
  EXPECT(run(a), TP_ERR_NULL);
  a = base(), a.lse = nullptr;
  EXPECT(run(a), TP_ERR_NULL);
  a = base(), a.kg = fake();
  EXPECT(run(a), TP_ERR_NULL);
  a = base(), a.vg = fake();
  EXPECT(run(a), TP_ERR_NULL);
  a = base(), a.o = (float*)fake(4);
  EXPECT(run(a), TP_ERR_PARAM);
  a = base(), a.lse = (float*)fake(2);
  EXPECT(run(a), TP_ERR_PARAM);
  a = base(), a.scale = 0.0f;
  EXPECT(run(a), TP_ERR_PARAM);
  a = base(), a.w = nullptr;
  EXPECT(run(a), TP_ERR_WORKSPACE);
  a = base(), a.wsb = ws - 1;
  EXPECT(run(a), TP_ERR_WORKSPACE);
  a = base(), a.w = fake(16);
  EXPECT(run(a), TP_ERR_WORKSPACE);
  a = base(), a.b = &noguide.c;
  EXPECT(run(a), TP_ERR_NULL);
  // with step 2 from the same sweep
  const auto runq = [&](const A& x, int32_t qfmt, int32_t bits, float* sc, void* vq) {
    return tp_guide_attention_quantize(dp, x.b, x.q, x.k, x.v, x.kg, x.vg, x.scale, qfmt, bits, x.o, x.lse, sc, vq, x.w,
                                       x.wsb, nullptr);
  };
  EXPECT(runq(base(), TP_QFMT_INT, 8, (float*)fake(), nullptr), TP_ERR_NULL);
  EXPECT(runq(base(), TP_QFMT_INT, 8, nullptr, fake()), TP_ERR_NULL);
  EXPECT(runq(base(), TP_QFMT_INT, 1, (float*)fake(), fake()), TP_ERR_PARAM);
  EXPECT(runq(base(), 7, 8, (float*)fake(), fake()), TP_ERR_PARAM);
  EXPECT(runq(base(), TP_QFMT_INT, 4, (float*)fake(4), fake()), TP_ERR_PARAM);
  a = base(), a.v = nullptr;
  EXPECT(runq(a, TP_QFMT_INT, 8, (float*)fake(), fake()), TP_ERR_NULL);
  a = base(), a.wsb = ws - 1;
  EXPECT(runq(a, TP_QFMT_FP8_E4M3, 8, (float*)fake(), fake()), TP_ERR_WORKSPACE);
}

void quantize_select_compact_cases() {
  {
    const tp_dims d{2, 8, 2, 128};
    Batch bt({0, 100});
    const auto q = [&](int32_t fmt, int32_t bits, const void* v, float* s, void* vq) {
      return tp_quantize_v_scales(&d, &bt.c, v, fmt, bits, s, vq, nullptr);
    };
    EXPECT(q(0, 1, fake(), (float*)fake(), fake()), TP_ERR_PARAM);
    EXPECT(q(0, 9, fake(), (float*)fake(), fake()), TP_ERR_PARAM);
    EXPECT(q(5, 8, fake(), (float*)fake(), fake()), TP_ERR_PARAM);
    EXPECT(q(0, 8, nullptr, (float*)fake(), fake()), TP_ERR_NULL);
    EXPECT(q(0, 8, fake(), nullptr, fake()), TP_ERR_NULL);
    EXPECT(q(0, 8, fake(), (float*)fake(), fake(4)), TP_ERR_PARAM);
  }
  const tp_dims d{2, 8, 2, 64};
  Batch bt({0, 100, 300});
  const std::vector<int64_t> good = kept_offsets(bt, 0.25, 0);
  const size_t ws = ws_size(TP_FN_COMBINE_SELECT_TOPK, d, bt);
  const auto sel = [&](int32_t rule, double ratio, int64_t budget, const int64_t* ko, int32_t* kept, float* s_out, void* w,
                       size_t wsb) {
    return tp_combine_select_topk(&d, &bt.c, (const float*)fake(), (const float*)fake(), rule, ratio, budget, ko, kept,
                                  s_out, w, wsb, nullptr);
  };
  int32_t* kept = (int32_t*)fake();
  float* so = (float*)fake();
  const int64_t ko_short[3] = {0, 25, 74}, ko_off[3] = {1, 26, 76};
  EXPECT(sel(4, 0.25, 0, good.data(), kept, so, fake(), ws), TP_ERR_PARAM);
  EXPECT(sel(0, 0.25, 10, good.data(), kept, so, fake(), ws), TP_ERR_PARAM);
  EXPECT(sel(0, 0.0, 0, good.data(), kept, so, fake(), ws), TP_ERR_PARAM);
  EXPECT(sel(0, 1.5, 0, good.data(), kept, so, fake(), ws), TP_ERR_PARAM);
  EXPECT(sel(0, NAN, 0, good.data(), kept, so, fake(), ws), TP_ERR_PARAM);
  EXPECT(sel(0, 0.25, 0, ko_short, kept, so, fake(), ws), TP_ERR_SHAPE);
  EXPECT(sel(0, 0.25, 0, ko_off, kept, so, fake(), ws), TP_ERR_SHAPE);
  EXPECT(sel(0, 0.25, 0, nullptr, kept, so, fake(), ws), TP_ERR_NULL);
  EXPECT(sel(0, 0.25, 0, good.data(), nullptr, so, fake(), ws), TP_ERR_NULL);
  EXPECT(sel(0, 0.25, 0, good.data(), kept, nullptr, nullptr, 0), TP_ERR_WORKSPACE);
  EXPECT(sel(0, 0.25, 0, good.data(), kept, so, nullptr, 0), TP_ERR_WORKSPACE);
  EXPECT(sel(0, 0.25, 0, good.data(), kept, so, fake(), ws - 1), TP_ERR_WORKSPACE);
  EXPECT(sel(0, 0.25, 0, good.data(), kept, so, fake(16), ws), TP_ERR_WORKSPACE);
  // the no-allocation variant
  const auto sst = [&](const tp_dims& dd, const Batch& b, const int64_t* ko, int32_t rule, double ratio, int64_t budget,
                       int32_t* kp) {
    return tp_combine_select_topk_static(&dd, &b.c, (const float*)fake(), (const float*)fake(), rule, ratio, budget, ko,
                                         kp, nullptr);
  };
  EXPECT(sst(d, bt, good.data(), 4, 0.25, 0, kept), TP_ERR_PARAM);
  EXPECT(sst(d, bt, good.data(), 0, 0.25, 10, kept), TP_ERR_PARAM);
  EXPECT(sst(d, bt, ko_short, 0, 0.25, 0, kept), TP_ERR_SHAPE);
  EXPECT(sst(d, bt, good.data(), 0, 0.25, 0, nullptr), TP_ERR_NULL);
  {
    const tp_dims d1{1, 1, 1, 64};
    Batch b1({0, (int64_t)(TP_STATIC_SCRATCH_BYTES / 4) + 1});
    const std::vector<int64_t> k1 = kept_offsets(b1, 0.5, 0);
    EXPECT(sst(d1, b1, k1.data(), 0, 0.5, 0, kept), TP_ERR_WORKSPACE);
  }
  // compaction
  const auto cp = [&](const int64_t* ko, const void* vq, const float* sc, void* vqo, float* sco, int32_t bits) {
    return tp_compact_kv(&d, &bt.c, ko, (const int32_t*)fake(), fake(), vq, sc, TP_QFMT_INT, bits, fake(), vqo, sco,
                         nullptr);
  };
  const int64_t ko_ok[3] = {0, 25, 75}, ko_many[3] = {0, 101, 150}, ko_down[3] = {0, 30, 20};
  EXPECT(cp(ko_many, fake(), (const float*)fake(), fake(), (float*)fake(), 8), TP_ERR_SHAPE);
  EXPECT(cp(ko_down, fake(), (const float*)fake(), fake(), (float*)fake(), 8), TP_ERR_SHAPE);
  EXPECT(cp(ko_ok, nullptr, (const float*)fake(), fake(), (float*)fake(), 8), TP_ERR_NULL);
  EXPECT(cp(ko_ok, fake(), (const float*)fake(), fake(), nullptr, 8), TP_ERR_NULL);
  EXPECT(cp(ko_ok, fake(), (const float*)fake(), fake(), (float*)fake(), 0), TP_ERR_PARAM);
  EXPECT(cp(nullptr, fake(), (const float*)fake(), fake(), (float*)fake(), 8), TP_ERR_NULL);
  const auto cq = [&](const int64_t* ko, const void* v, void* vqo, float* sco, int32_t bits, void* kout) {
    return tp_compact_quantize_kv(&d, &bt.c, ko, (const int32_t*)fake(), fake(), v, TP_QFMT_INT, bits, kout, vqo, sco,
                                  nullptr);
  };
  EXPECT(cq(ko_ok, nullptr, fake(), (float*)fake(), 8, fake()), TP_ERR_NULL);
  EXPECT(cq(ko_ok, fake(), nullptr, (float*)fake(), 8, fake()), TP_ERR_NULL);
  EXPECT(cq(ko_ok, fake(), fake(), nullptr, 8, fake()), TP_ERR_NULL);
  EXPECT(cq(ko_ok, fake(), fake(), (float*)fake(), 8, nullptr), TP_ERR_NULL);
  EXPECT(cq(ko_ok, fake(8), fake(), (float*)fake(), 8, fake()), TP_ERR_PARAM);
  EXPECT(cq(ko_many, fake(), fake(), (float*)fake(), 8, fake()), TP_ERR_SHAPE);
  EXPECT(cq(ko_ok, fake(), fake(), (float*)fake(), 1, fake()), TP_ERR_PARAM);
}

void evict_cases() {
  const tp_dims d{2, 8, 2, 64};
  Batch bt({0, 100, 300}, {0, 16, 20}), noguide({0, 100, 300});
  const std::vector<int64_t> good = kept_offsets(bt, 0.25, 0);
  const auto base = [&]() {
    EV e;
    e.d = &d;
    e.bt = &bt.c;
    e.ko = good.data();
    return e;
  };
  EV e = base();
  const auto check = [&](EV ev, tp_status want, int line) { expect(ev.run(), want, "tp_evict", line); };
  e = base(), e.q = nullptr, check(e, TP_ERR_NULL, __LINE__);
  // v = NULL: step 2 done beforehand; its scales and codes must be given
  e = base(), e.v = nullptr, e.vq = nullptr, check(e, TP_ERR_NULL, __LINE__);
  e = base(), e.v = nullptr, e.sc = nullptr, check(e, TP_ERR_NULL, __LINE__);
  e = base(), e.v = nullptr, e.bits = 9, check(e, TP_ERR_PARAM, __LINE__);
  e = base(), e.v = nullptr, e.vq = fake(4), check(e, TP_ERR_PARAM, __LINE__);
  e = base(), e.vq = nullptr, e.vqout = nullptr, check(e, TP_ERR_NULL, __LINE__);
  e = base(), e.vq = nullptr, e.scout = nullptr, check(e, TP_ERR_NULL, __LINE__);
  e = base(), e.idx = nullptr, check(e, TP_ERR_NULL, __LINE__);
  e = base(), e.kout = nullptr, check(e, TP_ERR_NULL, __LINE__);
  e = base(), e.vqout = nullptr, check(e, TP_ERR_NULL, __LINE__);
  e = base(), e.scale = 0.0f, check(e, TP_ERR_PARAM, __LINE__);
  e = base(), e.pool = 2, check(e, TP_ERR_PARAM, __LINE__);
  e = base(), e.qfmt = 5, check(e, TP_ERR_PARAM, __LINE__);
  e = base(), e.bits = 9, check(e, TP_ERR_PARAM, __LINE__);
  e = base(), e.rule = 7, check(e, TP_ERR_PARAM, __LINE__);
  const int64_t ko3[3] = {0, 1, 2}, ko_bad[3] = {0, 25, 51};
  e = base(), e.ratio = 0.0, e.budget = 0, e.ko = ko3, check(e, TP_ERR_PARAM, __LINE__);
  e = base(), e.ko = ko_bad, check(e, TP_ERR_SHAPE, __LINE__);
  e = base(), e.ko = nullptr, check(e, TP_ERR_NULL, __LINE__);
  e = base(), e.ws = nullptr, check(e, TP_ERR_WORKSPACE, __LINE__);
  e = base(), e.wsb = 1024, check(e, TP_ERR_WORKSPACE, __LINE__);
  e = base(), e.sout = nullptr, e.wsb = ws_size(TP_FN_GUIDE_SCORES, d, bt), check(e, TP_ERR_WORKSPACE, __LINE__);
  e = base(), e.wsb = ws_size(TP_FN_EVICT, d, bt) - 1, check(e, TP_ERR_WORKSPACE, __LINE__);
  tp_profile short_prof{};
  short_prof.num_events = 3;
  tp_profile null_prof{};
  null_prof.num_events = TP_EVICT_EVENTS;
  e = base(), e.prof = &short_prof, check(e, TP_ERR_PARAM, __LINE__);
  e = base(), e.prof = &null_prof, check(e, TP_ERR_NULL, __LINE__);
  e = base(), e.k = fake(8), check(e, TP_ERR_PARAM, __LINE__);
  e = base(), e.kg = fake(4), check(e, TP_ERR_PARAM, __LINE__);
  e = base(), e.kg = fake(), e.lse = (const float*)fake(), check(e, TP_ERR_PARAM, __LINE__);
  e = base(), e.lse = (const float*)fake(2), check(e, TP_ERR_PARAM, __LINE__);
  e = base(), e.bt = &noguide.c, check(e, TP_ERR_NULL, __LINE__);
  const tp_dims d_hd{2, 8, 2, 96};
  e = base(), e.d = &d_hd, check(e, TP_ERR_UNSUPPORTED, __LINE__);
}

// Well-formed calls: every host-side layout, table and offset computation runs, then the first
// runtime call fails because no device is visible.  Only run when the runtime reports none.
void well_formed_without_device() {
  const tp_dims d{2, 8, 2, 64};
  Batch bt({0, 100, 300}, {0, 16, 20});
  const std::vector<int64_t> ko = kept_offsets(bt, 0.25, 0);
  GS g;
  g.d = &d;
  g.bt = &bt.c;
  g.wsb = ws_size(TP_FN_GUIDE_SCORES, d, bt);
  EXPECT(g.run(), TP_ERR_HIP);
  g.kg = fake();
  EXPECT(g.run(), TP_ERR_HIP);
  EXPECT(tp_guide_scores_lse(&d, &bt.c, fake(), fake(), (const float*)fake(), 0.125f, 5, (float*)fake(), fake(), g.wsb,
                             nullptr),
         TP_ERR_HIP);
  EXPECT(tp_guide_attention(&d, &bt.c, fake(), fake(), fake(), fake(), fake(), 0.125f, (float*)fake(), (float*)fake(),
                            fake(), ws_size(TP_FN_GUIDE_ATTENTION, d, bt), nullptr),
         TP_ERR_HIP);
  EXPECT(tp_guide_attention_quantize(&d, &bt.c, fake(), fake(), fake(), nullptr, nullptr, 0.125f, TP_QFMT_INT, 4,
                                     (float*)fake(), (float*)fake(), (float*)fake(), fake(), fake(),
                                     ws_size(TP_FN_GUIDE_ATTENTION, d, bt), nullptr),
         TP_ERR_HIP);
  EXPECT(tp_quantize_v_scales(&d, &bt.c, fake(), TP_QFMT_INT, 4, (float*)fake(), fake(), nullptr), TP_ERR_HIP);
  EXPECT(tp_combine_select_topk(&d, &bt.c, (const float*)fake(), (const float*)fake(), TP_COMBINE_NORM_ADD, 0.25, 0,
                                ko.data(), (int32_t*)fake(), nullptr, fake(), ws_size(TP_FN_COMBINE_SELECT_TOPK, d, bt),
                                nullptr),
         TP_ERR_HIP);
  EXPECT(tp_combine_select_topk(&d, &bt.c, (const float*)fake(), (const float*)fake(), TP_COMBINE_MUL, 0.25, 0, ko.data(),
                                (int32_t*)fake(), (float*)fake(), fake(), ws_size(TP_FN_COMBINE_SELECT_TOPK, d, bt), nullptr),
         TP_ERR_HIP);
  EXPECT(tp_combine_select_topk_static(&d, &bt.c, (const float*)fake(), (const float*)fake(), TP_COMBINE_MUL, 0.25, 0,
                                       ko.data(), (int32_t*)fake(), nullptr),
         TP_ERR_HIP);
  EXPECT(tp_compact_kv(&d, &bt.c, ko.data(), (const int32_t*)fake(), fake(), fake(), (const float*)fake(), TP_QFMT_INT, 8,
                       fake(), fake(), (float*)fake(), nullptr),
         TP_ERR_HIP);
  EXPECT(tp_compact_quantize_kv(&d, &bt.c, ko.data(), (const int32_t*)fake(), fake(), fake(), TP_QFMT_FP8_E4M3, 8, fake(),
                                fake(), (float*)fake(), nullptr),
         TP_ERR_HIP);
  for (int mode = 0; mode < 5; ++mode) {
    EV e;
    e.d = &d;
    e.bt = &bt.c;
    e.ko = ko.data();
    e.wsb = ws_size(TP_FN_EVICT, d, bt);
    if (mode == 1) e.lse = (const float*)fake();
    if (mode == 2) e.vq = nullptr;
    if (mode == 3) e.rule = TP_COMBINE_NORM_ADD, e.kg = fake();
    if (mode == 4) e.v = nullptr, e.lse = (const float*)fake();  // step 2 done beforehand
    EXPECT(e.run(), TP_ERR_HIP);
  }
}

}  // namespace

int main() {
  int ndev = 0;
  const bool device = hipGetDeviceCount(&ndev) == hipSuccess && ndev > 0;
  host_helpers();
  workspace_sizes();
  hostile_shapes();
  guide_scores_cases();
  attention_cases();
  quantize_select_compact_cases();
  evict_cases();
  if (!device) well_formed_without_device();
  std::printf("%d checks, %d failures%s\n", checks, failures, device ? " (well-formed calls skipped: a device is visible)" : "");
  return failures == 0 ? 0 : 1;
}
