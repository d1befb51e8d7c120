/*
 * Host (CPU) evaluation of the seeded input generator defined in synth_core.h.
 * Built with gcc -ffp-contract=off so that no multiply-add is fused and the
 * values agree bit for bit with the device build.
 */
#include <stdint.h>
#include "synth_core.h"

/* dst[t][c], t in [0, n), c in [0, d): rows of the (seq, layer, head) row set of a sequence
   with n_seq tokens, starting at token t0 (so dst row t is token t0 + t). */
void syn_host_rows(uint16_t* dst, const syn_spec* sp, int64_t seq, int64_t layer, int64_t head,
                   int64_t n_seq, int64_t t0, int64_t n, int64_t d) {
  uint64_t key = syn_key(sp->seed, (uint64_t)sp->tag, (uint64_t)seq, (uint64_t)layer, (uint64_t)head);
#pragma omp parallel for schedule(static)
  for (int64_t t = 0; t < n; ++t) {
    uint64_t tok = (uint64_t)(t0 + t);
    double f = syn_token_factor(sp, (uint64_t)seq, (uint64_t)layer, (uint64_t)head, (uint64_t)n_seq, tok);
    for (int64_t c = 0; c < d; ++c)
      dst[t * d + c] = syn_element(key, sp->dist, tok, (uint64_t)d, (uint64_t)c, f);
  }
}

/* Fill one sequence's tokens in a [L][H][ntot][d] tensor: tokens [off, off + n) of every
   (layer, head) receive the sequence's tokens 0..n-1. */
void syn_host_fill(uint16_t* dst, const syn_spec* sp, int64_t seq, int64_t L, int64_t H,
                   int64_t ntot, int64_t off, int64_t n, int64_t d) {
  for (int64_t l = 0; l < L; ++l)
    for (int64_t h = 0; h < H; ++h)
      syn_host_rows(dst + ((l * H + h) * ntot + off) * d, sp, seq, l, h, n, 0, n, d);
}

/* Scalar probes used by the generator's own tests. */
double syn_probe_log(double x) { return syn_log(x); }
double syn_probe_cos_turns(double w) { return syn_cos_turns(w); }
double syn_probe_normal(uint64_t key, uint64_t m) { return syn_normal(key, m); }
uint16_t syn_probe_to_bf16(double x) { return syn_to_bf16(x); }
uint64_t syn_probe_perm(uint64_t i, uint64_t n, uint64_t key) { return syn_perm(i, n, key); }
uint64_t syn_probe_at(uint64_t s, uint64_t n) { return syn_at(s, n); }
