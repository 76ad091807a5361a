/* sanitize_driver.c -- drives the C oracle and the host code of the C-ABI
 * library under AddressSanitizer and UndefinedBehaviorSanitizer (test
 * support; built by tests/test_sanitizers.py).
 *
 * OR build (oracle only): every orc_* function on small inputs, including
 * ragged and degenerate shapes.
 * API build (oracle + libmcmoe host code): additionally the C-ABI calls that
 * run on the host without a GPU -- the size queries, every validation path
 * that returns before a launch, the pruning-threshold helper, the PMQ
 * significance and the Eq. 4 allocation.
 * Exit status 0 when every call returned as expected; the sanitizers abort
 * with a report on any memory or undefined-behaviour error. */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

/* the oracle's C entry points (oracle/mc_oracle.c) */
double orc_f16_to_double(uint16_t h);
double orc_bf16_to_double(uint16_t h);
int orc_quantize_group(const float *w, int G, int bits, uint16_t *s_out, uint16_t *z_out, uint8_t *q_out);
int orc_quantize_matrix(const float *W, int R, int K, int G, int bits, uint8_t *q, uint16_t *s, uint16_t *z);
double orc_dequant(uint16_t s16, uint16_t z16, int q);
void orc_dequant_matrix_f16(const uint8_t *q, const uint16_t *s, const uint16_t *z, int R, int K, int G,
                            uint16_t *out);
int orc_layout_pack(const uint8_t *q, int R, int K, int bits, uint32_t *words);
int orc_layout_unpack(const uint32_t *words, int R, int K, int bits, uint8_t *q);
int orc_layout_pack_sz(const uint16_t *s, const uint16_t *z, int R, int K, int G, uint32_t *sz);
int orc_layout_unpack_sz(const uint32_t *sz, int R, int K, int G, uint16_t *s, uint16_t *z);
int orc_route(const float *logits, const uint8_t *important, int T, int E, int k, double tau, float delta32,
              int32_t *topk_idx, double *topk_w, uint8_t *kept, int32_t *counts, int32_t *offsets,
              int32_t *pair_token, int32_t *pair_rank, double *pair_w, int32_t *pair_pos, int32_t *n_pruned);
int orc_expert_forward(const double *X, int nt, int d, int ffn, int G, const uint8_t *qg, const uint16_t *sg,
                       const uint16_t *zg, const uint8_t *qu, const uint16_t *su, const uint16_t *zu,
                       const uint8_t *qd, const uint16_t *sd, const uint16_t *zd, const int32_t *rows,
                       int nrows, double *H, double *Y);
int orc_token_importance(const uint16_t *attn, int H, int L, const uint16_t *x, int d, int n, double *I,
                         uint8_t *mask);
double orc_median_ratio(const float *logits, int T, int E);

#ifdef WITH_API
#include "../../include/mc_moe.h"
#endif

static int failures = 0;
#define EXPECT(c)                                                        \
  do {                                                                   \
    if (!(c)) {                                                          \
      fprintf(stderr, "%s:%d: expectation failed: %s\n", __FILE__, __LINE__, #c); \
      ++failures;                                                        \
    }                                                                    \
  } while (0)

static uint64_t rng = 88172645463325252ull;
static double urand(void) {     /* xorshift64*, uniform in [0, 1) */
  rng ^= rng >> 12;
  rng ^= rng << 25;
  rng ^= rng >> 27;
  return (double)((rng * 2685821657736338717ull) >> 11) / 9007199254740992.0;
}
static float nrand(void) {      /* Box-Muller */
  double u = urand() + 1e-12, v = urand();
  return (float)(sqrt(-2.0 * log(u)) * cos(6.283185307179586 * v));
}

static void oracle_calls(void) {
  for (int bits = 1; bits <= 3; ++bits) {
    const int R = 48, K = 256, G = 32, ng = K / G;
    float *W = malloc(sizeof(float) * R * K);
    for (int i = 0; i < R * K; ++i) W[i] = 0.02f * nrand();
    for (int i = 0; i < G; ++i) W[i] = 0.25f;              /* a constant group */
    uint8_t *q = malloc(R * K), *q2 = malloc(R * K);
    uint16_t *s = malloc(2 * R * ng), *z = malloc(2 * R * ng), *s2 = malloc(2 * R * ng), *z2 = malloc(2 * R * ng);
    uint16_t *deq = malloc(2 * R * K);
    EXPECT(orc_quantize_matrix(W, R, K, G, bits, q, s, z) == 0);
    orc_dequant_matrix_f16(q, s, z, R, K, G, deq);
    const int nw = R * K / 32 * bits;
    uint32_t *words = malloc(4 * nw), *sz = malloc(4 * R * ng);
    EXPECT(orc_layout_pack(q, R, K, bits, words) == 0);
    EXPECT(orc_layout_unpack(words, R, K, bits, q2) == 0);
    EXPECT(memcmp(q, q2, R * K) == 0);
    EXPECT(orc_layout_pack_sz(s, z, R, K, G, sz) == 0);
    EXPECT(orc_layout_unpack_sz(sz, R, K, G, s2, z2) == 0);
    EXPECT(memcmp(s, s2, 2 * R * ng) == 0 && memcmp(z, z2, 2 * R * ng) == 0);
    uint16_t s1, z1;
    uint8_t q1[32];
    EXPECT(orc_quantize_group(W, G, bits, &s1, &z1, q1) == 0);
    EXPECT(orc_quantize_group(W, G, 4, &s1, &z1, q1) != 0);    /* rejected width */
    EXPECT(isfinite(orc_dequant(s1, z1, 1)));
    free(W); free(q); free(q2); free(s); free(z); free(s2); free(z2); free(deq); free(words); free(sz);
  }
  EXPECT(orc_f16_to_double(0x3c00) == 1.0 && orc_bf16_to_double(0x3f80) == 1.0);

  /* routing: k = 1, 2 and 8 on ragged token counts, with and without a mask */
  const int Es[3] = {4, 8, 64}, ks[3] = {1, 2, 8}, Ts[3] = {1, 7, 33};
  for (int c = 0; c < 3; ++c) {
    const int T = Ts[c], E = Es[c], k = ks[c], P = T * k;
    float *lg = malloc(sizeof(float) * T * E);
    uint8_t *imp = malloc(T), *kept = malloc(P);
    for (int i = 0; i < T * E; ++i) lg[i] = nrand();
    for (int t = 0; t < T; ++t) imp[t] = (t % 5) == 0;
    int32_t *idx = malloc(4 * P), *counts = malloc(4 * E), *offs = malloc(4 * (E + 1)), *ptok = malloc(4 * P),
            *prank = malloc(4 * P), *ppos = malloc(4 * P), npr;
    double *tw = malloc(8 * P), *pw = malloc(8 * P);
    EXPECT(orc_route(lg, c == 1 ? NULL : imp, T, E, k, 0.3, 0.8472979f, idx, tw, kept, counts, offs, ptok, prank,
                     pw, ppos, &npr) == 0);
    EXPECT(offs[E] == P - npr);
    EXPECT(orc_route(lg, imp, T, E, E + 1, 0.3, 0.8472979f, idx, tw, kept, counts, offs, ptok, prank, pw, ppos,
                     &npr) != 0);
    if (E >= 2) EXPECT(orc_median_ratio(lg, T, E) > 0.0);
    free(lg); free(imp); free(kept); free(idx); free(counts); free(offs); free(ptok); free(prank); free(ppos);
    free(tw); free(pw);
  }

  /* one SwiGLU expert on a few tokens, all rows and a row subset */
  {
    const int nt = 3, d = 128, ffn = 256, G = 64;
    double *X = malloc(8 * nt * d), *H = malloc(8 * nt * ffn), *Y = malloc(8 * nt * d);
    for (int i = 0; i < nt * d; ++i) X[i] = nrand();
    uint8_t *qg = calloc(ffn * d, 1), *qu = calloc(ffn * d, 1), *qd = calloc(ffn * d, 1);
    uint16_t *sgz = malloc(2 * ffn * d / G);
    for (int i = 0; i < ffn * d / G; ++i) sgz[i] = 0x2000;   /* small scales; zero = the same bits */
    for (int i = 0; i < ffn * d; ++i) { qg[i] = i % 4; qu[i] = (i / 3) % 4; qd[i] = (i / 7) % 4; }
    EXPECT(orc_expert_forward(X, nt, d, ffn, G, qg, sgz, sgz, qu, sgz, sgz, qd, sgz, sgz, NULL, d, H, Y) == 0);
    const int32_t rows[3] = {0, 5, d - 1};
    EXPECT(orc_expert_forward(X, nt, d, ffn, G, qg, sgz, sgz, qu, sgz, sgz, qd, sgz, sgz, rows, 3, H, Y) == 0);
    EXPECT(orc_expert_forward(X, nt, d + 1, ffn, G, qg, sgz, sgz, qu, sgz, sgz, qd, sgz, sgz, NULL, d, H, Y) != 0);
    free(X); free(H); free(Y); free(qg); free(qu); free(qd); free(sgz);
  }

  /* token importance over a small causal map */
  {
    const int Hh = 2, L = 37, d = 16;
    uint16_t *attn = malloc(2 * Hh * L * L), *x = malloc(2 * L * d);
    for (int i = 0; i < Hh * L * L; ++i) attn[i] = 0x3c00 + (i % 7);
    for (int i = 0; i < L * d; ++i) x[i] = 0x3f80 + (i % 11);
    double *I = malloc(8 * L);
    uint8_t *mask = malloc(L);
    EXPECT(orc_token_importance(attn, Hh, L, x, d, 3, I, mask) == 0);
    EXPECT(orc_token_importance(attn, Hh, L, x, d, L + 1, I, mask) != 0);
    free(attn); free(x); free(I); free(mask);
  }
}

#ifdef WITH_API
static void api_calls(void) {
  const int bits8[8] = {3, 3, 3, 2, 2, 2, 2, 3};
  size_t wb = 0, szb = 0, ws = 0;
  EXPECT(mc_pack_sizes(8, 4096, 14336, bits8, 128, &wb, &szb) == MC_OK && wb == 440401920u);
  const int badbits[2] = {0, 4};
  EXPECT(mc_pack_sizes(2, 256, 512, badbits, 32, &wb, &szb) == MC_EINVAL);
  EXPECT(mc_pack_sizes(8, 4096, 14336, bits8, 48, &wb, &szb) != MC_OK);
  EXPECT(mc_pack_sizes(300, 256, 512, bits8, 32, &wb, &szb) == MC_EINVAL);
  EXPECT(mc_forward_workspace(32, 8, 2, 4096, 14336, &ws) == MC_OK && ws > 0);
  EXPECT(mc_forward_workspace(4096, 8, 2, 4096, 14336, &ws) == MC_OK && ws > 0);
  EXPECT(mc_forward_workspace(70000, 8, 2, 4096, 14336, &ws) == MC_EUNSUPPORTED);
  EXPECT(mc_forward_workspace(32, 8, 9, 4096, 14336, &ws) == MC_EINVAL);
  EXPECT(mc_stack_workspace(64, 8, 2, 4096, 14336, &ws) == MC_OK);
  EXPECT(mc_importance_workspace(32, 4096, &ws) == MC_OK);
  EXPECT(mc_gptq_workspace(14336, 4096, &ws) == MC_OK);
  EXPECT(strlen(mc_last_error()) < 512);

  /* validation paths that return before any launch */
  mc_layer L;
  memset(&L, 0, sizeof(L));
  L.E = 8; L.d = 4096; L.ffn = 14336; L.group = 128; L.bits_host = bits8;
  EXPECT(mc_pack(NULL, NULL, NULL, &L, NULL) == MC_EINVAL);
  mc_routing r;
  memset(&r, 0, sizeof(r));
  r.T = 32; r.E = 8; r.k = 2;
  EXPECT(mc_route_and_prune(NULL, NULL, 0.3f, &r, NULL) == MC_EINVAL);
  EXPECT(mc_moe_forward(NULL, &r, &L, NULL, NULL, 0, NULL) == MC_EINVAL);
  EXPECT(mc_moe_forward_noalloc(NULL, &r, &L, NULL, NULL) == MC_EINVAL);
  EXPECT(mc_timing_read("no_such_kernel", NULL, NULL) == MC_EINVAL);

  /* host helpers */
  const int T = 257, E = 8;
  float *lg = malloc(sizeof(float) * T * E);
  for (int i = 0; i < T * E; ++i) lg[i] = nrand();
  double mu = 0, tau = 0, phi[8], w[8], eps[8 * 3], obj = 0;
  EXPECT(mc_odp_threshold(lg, T, E, &mu, &tau) == MC_OK && mu > 0 && tau > 0 && tau < 0.5);
  EXPECT(mc_odp_threshold(lg, 0, E, &mu, &tau) == MC_EINVAL);
  EXPECT(mc_pmq_significance(lg, T, E, 2, phi, w) == MC_OK);
  for (int i = 0; i < 3 * E; ++i) eps[i] = 1.0 / (1 + i % 3) + 0.01 * (i / 3);
  int bits[8];
  EXPECT(mc_pmq_allocate(phi, w, eps, E, 1.0, 1.0, 2.0, 20, bits, &obj) == MC_OK);
  int tot = 0;
  for (int e = 0; e < E; ++e) tot += bits[e];
  EXPECT(tot == 20);
  EXPECT(mc_pmq_allocate(phi, w, eps, E, 1.0, 1.0, 2.0, 40, bits, &obj) == MC_EINVAL);
  free(lg);
}
#endif

int main(void) {
  oracle_calls();
#ifdef WITH_API
  api_calls();
#endif
  if (failures) {
    fprintf(stderr, "%d expectation(s) failed\n", failures);
    return 1;
  }
  printf("sanitized run ok\n");
  return 0;
}
