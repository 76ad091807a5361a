/*
 * mc_oracle.c -- plain, slow CPU reference of the MC expert path.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product library calls, links or
 * loads this file; only the tests, the smoke check and the CPU-baseline leg
 * of the benchmark use it.  It shares no code, header or table with the HIP
 * kernels.  Floating point is done in fp64 (weights, activations and sums);
 * where the method's definition itself fixes an fp32 or fp16 operation
 * (the quantizer's scale and zero, the k = 2 pruning test) that operation is
 * written out in that precision.  Build: gcc -O2 -ffp-contract=off -fopenmp.
 *
 * Sections followed (Mixture Compressor for MoE LLMs, ICLR 2025):
 *   Sec. 3.1 "Quantization technique"  -- uniform asymmetric group quantizer;
 *   Sec. 3.1 Eq. 1                     -- MoE layer output over the top-k;
 *   Sec. 3.3.1 Eq. 5                   -- weight-only expert pruning;
 *   Sec. 3.3.2                         -- protected (important) tokens keep
 *                                         all their experts;
 *   Sec. 3.3.2 Eq. 6                   -- token importance, protected set;
 *   Sec. 3.3.1                         -- threshold as the median of w1/w0.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

/* ------------------------------------------------------------------------ */
/* IEEE half / bfloat16 conversions, from the format definitions.           */
/* ------------------------------------------------------------------------ */

double orc_f16_to_double(uint16_t h) {
  int sign = (h >> 15) & 1;
  int ex = (h >> 10) & 0x1f;
  int man = h & 0x3ff;
  double v;
  if (ex == 0)
    v = ldexp((double)man, -24);                /* subnormal: man * 2^-24 */
  else if (ex == 31)
    v = man ? NAN : INFINITY;
  else
    v = ldexp((double)(man + 1024), ex - 25);   /* (1 + man/1024) * 2^(ex-15) */
  return sign ? -v : v;
}

/* Round v to the nearest fp16 value, ties to even.  saturate != 0 clamps the
 * result to +-65504 instead of producing an infinity. */
static uint16_t f16_round(double v, int saturate) {
  uint16_t sign = signbit(v) ? 0x8000 : 0;
  double a = fabs(v);
  if (isnan(v)) return 0x7e00;
  if (isinf(a)) return saturate ? (uint16_t)(sign | 0x7bff) : (uint16_t)(sign | 0x7c00);
  if (a == 0.0) return sign;
  int e2;
  frexp(a, &e2);                 /* a = m * 2^e2, m in [0.5, 1) => a in [2^(e2-1), 2^e2) */
  int e = e2 - 1;                /* a in [2^e, 2^(e+1)) */
  if (e < -14) e = -14;          /* below the normal range the quantum is 2^-24 */
  double quantum = ldexp(1.0, e - 10);
  double r = rint(a / quantum) * quantum;   /* a / quantum is exact; rint ties to even */
  if (r > 65504.0) return saturate ? (uint16_t)(sign | 0x7bff) : (uint16_t)(sign | 0x7c00);
  if (r < ldexp(1.0, -14)) {     /* subnormal (or rounded up to the smallest normal) */
    int man = (int)(r / ldexp(1.0, -24));
    return (uint16_t)(sign | man);
  }
  int re2;
  double m = frexp(r, &re2);     /* r = m * 2^re2 */
  int ex = re2 - 1 + 15;
  int man = (int)(ldexp(m, 11)) - 1024;
  return (uint16_t)(sign | (ex << 10) | man);
}

uint16_t orc_f16_from_double(double v) { return f16_round(v, 0); }
uint16_t orc_f16_from_double_sat(double v) { return f16_round(v, 1); }

double orc_bf16_to_double(uint16_t h) {
  uint32_t bits = (uint32_t)h << 16;
  float f;
  memcpy(&f, &bits, 4);
  return (double)f;
}

/* Round v to the nearest bfloat16 (8 significant bits, fp32 exponent range),
 * ties to even; overflow gives an infinity. */
uint16_t orc_bf16_from_double(double v) {
  uint16_t sign = signbit(v) ? 0x8000 : 0;
  double a = fabs(v);
  if (isnan(v)) return 0x7fc0;
  if (a == 0.0) return sign;
  if (isinf(a)) return (uint16_t)(sign | 0x7f80);
  int e2;
  frexp(a, &e2);
  int e = e2 - 1;
  if (e < -126) e = -126;
  double quantum = ldexp(1.0, e - 7);
  double r = rint(a / quantum) * quantum;
  if (r >= ldexp(1.0, 128)) return (uint16_t)(sign | 0x7f80);
  float f = (float)r;            /* r has <= 8 significant bits: exact in fp32 */
  uint32_t bits;
  memcpy(&bits, &f, 4);
  return (uint16_t)(sign | (bits >> 16));
}

/* ------------------------------------------------------------------------ */
/* Sec. 3.1: uniform asymmetric quantizer of one group.                      */
/* ------------------------------------------------------------------------ */

/* The integer grid is [0, 2^b - 1].  Scale and zero are fp16 values made by
 * the fp32 operations below; each code is the grid point whose dequantized
 * level s*(j - z) is nearest to w (ties to the even j), found by comparing w
 * with the exact midpoints s*(j + 1/2 - z) in fp64 (j + 1/2 - z needs at most
 * 41 bits and the product with the 11-bit s at most 52, so no rounding). */
int orc_quantize_group(const float *w, int G, int bits, uint16_t *s_out,
                       uint16_t *z_out, uint8_t *q_out) {
  if (bits < 1 || bits > 3 || G <= 0) return 1;
  int L = (1 << bits) - 1;
  float mn = w[0], mx = w[0];
  for (int i = 1; i < G; i++) {
    if (w[i] < mn) mn = w[i];
    if (w[i] > mx) mx = w[i];
  }
  float range = mx - mn;                       /* fp32 subtraction */
  float s32 = range / (float)L;                /* fp32 division, correctly rounded */
  uint16_t s16 = orc_f16_from_double_sat((double)s32);
  if ((s16 & 0x7fff) == 0) s16 = 0x3c00;       /* scale 0 -> 1.0 */
  double s = orc_f16_to_double(s16);
  float z32 = -mn / (float)s;                  /* fp32 division */
  uint16_t z16 = orc_f16_from_double_sat((double)z32);
  if (z16 == 0x8000) z16 = 0;                  /* -0 -> +0 */
  double z = orc_f16_to_double(z16);
  for (int i = 0; i < G; i++) {
    double wi = (double)w[i];
    int below = 0;                              /* midpoints strictly below w */
    for (int j = 0; j < L; j++) {
      double mid = s * (((double)j + 0.5) - z);
      if (mid < wi) below++;
    }
    int q = below;
    if (below < L) {
      double mid = s * (((double)below + 0.5) - z);
      if (mid == wi && (below & 1)) q = below + 1;   /* tie: take the even code */
    }
    q_out[i] = (uint8_t)q;
  }
  *s_out = s16;
  *z_out = z16;
  return 0;
}

/* Row-major W[R][K], groups of G along K.  q: [R][K]; s, z: [R][K/G]. */
int orc_quantize_matrix(const float *W, int R, int K, int G, int bits,
                        uint8_t *q, uint16_t *s, uint16_t *z) {
  if (R <= 0 || K <= 0 || G <= 0 || K % G) return 1;
  int ng = K / G;
  int err = 0;
#pragma omp parallel for schedule(static) reduction(| : err)
  for (int r = 0; r < R; r++)
    for (int g = 0; g < ng; g++)
      err |= orc_quantize_group(W + (size_t)r * K + (size_t)g * G, G, bits,
                                &s[(size_t)r * ng + g], &z[(size_t)r * ng + g],
                                q + (size_t)r * K + (size_t)g * G);
  return err;
}

/* Exact dequantized value s*(q - z): q - z and the product are exact in fp64. */
double orc_dequant(uint16_t s16, uint16_t z16, int q) {
  return orc_f16_to_double(s16) * ((double)q - orc_f16_to_double(z16));
}

/* fp16 export of a matrix: one round-to-nearest-even of the exact value. */
void orc_dequant_matrix_f16(const uint8_t *q, const uint16_t *s, const uint16_t *z,
                            int R, int K, int G, uint16_t *out) {
  int ng = K / G;
#pragma omp parallel for schedule(static)
  for (int r = 0; r < R; r++)
    for (int k = 0; k < K; k++) {
      size_t gi = (size_t)r * ng + k / G;
      out[(size_t)r * K + k] = orc_f16_from_double(orc_dequant(s[gi], z[gi], q[(size_t)r * K + k]));
    }
}

/* ------------------------------------------------------------------------ */
/* Packed layout (normative description in the library header), written     */
/* element by element from the index function.                              */
/* ------------------------------------------------------------------------ */

/* Locate the bits of code (n, k): *word = word index, positions of its b bits
 * in pos[0..b-1] (bit p of the code goes to (word + wofs[p], pos[p])). */
static void layout_locate(int n, int k, int K, int bits, size_t *word, int wofs[3], int pos[3]) {
  int tile_row = n / 16, tile_col = k / 128;
  int kk = k % 128;
  int u = kk / 32, kq = (kk % 32) / 8, j = kk % 8;
  int lane = (n % 16) + 16 * kq;
  int i = 4 * u + j / 2;
  int h = j % 2;
  *word = (((size_t)tile_row * (size_t)(K / 128) + (size_t)tile_col) * 64 + (size_t)lane) * (size_t)bits;
  if (bits == 1) {
    wofs[0] = 0; pos[0] = 16 * h + i;
  } else if (bits == 2) {
    for (int p = 0; p < 2; p++) { wofs[p] = i / 8; pos[p] = 16 * h + 2 * (i % 8) + p; }
  } else {
    if (i < 15) {
      for (int p = 0; p < 3; p++) { wofs[p] = i / 5; pos[p] = 16 * h + 3 * (i % 5) + p; }
    } else {
      for (int p = 0; p < 3; p++) { wofs[p] = p; pos[p] = 16 * h + 15; }
    }
  }
}

int orc_layout_pack(const uint8_t *q, int R, int K, int bits, uint32_t *words) {
  if (R % 16 || K % 128 || bits < 1 || bits > 3) return 1;
  size_t nwords = (size_t)R * K * bits / 32;
  memset(words, 0, nwords * 4);
  for (int n = 0; n < R; n++)
    for (int k = 0; k < K; k++) {
      size_t w; int wofs[3], pos[3];
      layout_locate(n, k, K, bits, &w, wofs, pos);
      int code = q[(size_t)n * K + k];
      for (int p = 0; p < bits; p++)
        if ((code >> p) & 1) words[w + wofs[p]] |= (uint32_t)1 << pos[p];
    }
  return 0;
}

int orc_layout_unpack(const uint32_t *words, int R, int K, int bits, uint8_t *q) {
  if (R % 16 || K % 128 || bits < 1 || bits > 3) return 1;
  for (int n = 0; n < R; n++)
    for (int k = 0; k < K; k++) {
      size_t w; int wofs[3], pos[3];
      layout_locate(n, k, K, bits, &w, wofs, pos);
      int code = 0;
      for (int p = 0; p < bits; p++) code |= (int)((words[w + wofs[p]] >> pos[p]) & 1u) << p;
      q[(size_t)n * K + k] = (uint8_t)code;
    }
  return 0;
}

/* Scale/zero word of (row n, group g): index ((n/16)*(K/G) + g)*16 + n%16. */
int orc_layout_pack_sz(const uint16_t *s, const uint16_t *z, int R, int K, int G, uint32_t *sz) {
  if (R % 16 || K % G) return 1;
  int ng = K / G;
  for (int n = 0; n < R; n++)
    for (int g = 0; g < ng; g++) {
      size_t idx = ((size_t)(n / 16) * ng + g) * 16 + n % 16;
      sz[idx] = (uint32_t)s[(size_t)n * ng + g] | ((uint32_t)z[(size_t)n * ng + g] << 16);
    }
  return 0;
}

int orc_layout_unpack_sz(const uint32_t *sz, int R, int K, int G, uint16_t *s, uint16_t *z) {
  if (R % 16 || K % G) return 1;
  int ng = K / G;
  for (int n = 0; n < R; n++)
    for (int g = 0; g < ng; g++) {
      size_t idx = ((size_t)(n / 16) * ng + g) * 16 + n % 16;
      s[(size_t)n * ng + g] = (uint16_t)(sz[idx] & 0xffffu);
      z[(size_t)n * ng + g] = (uint16_t)(sz[idx] >> 16);
    }
  return 0;
}

/* ------------------------------------------------------------------------ */
/* Eq. 1 routing, Eq. 5 pruning and token protection (Sec. 3.3).             */
/* ------------------------------------------------------------------------ */

/* Experts sorted by logit, largest first; equal logits by lower index.
 * Float comparison treats -0 and +0 as equal. */
static int rank_before(const float *l, int a, int b) {
  if (l[a] > l[b]) return 1;
  if (l[a] < l[b]) return 0;
  return a < b;
}

/* tau: threshold on the top-k-normalised weight.  delta32: fp32 threshold on
 * the logit gap used for k = 2 (the caller passes fp32(ln((1-tau)/tau)),
 * +inf for tau = 0).  topk_w / pair_w are fp64 here. */
int orc_route(const float *logits, const uint8_t *important, int T, int E, int k,
              double tau, float delta32, int32_t *topk_idx, double *topk_w,
              uint8_t *kept, int32_t *counts, int32_t *offsets, int32_t *pair_token,
              int32_t *pair_rank, double *pair_w, int32_t *pair_pos, int32_t *n_pruned) {
  if (T <= 0 || E <= 0 || k <= 0 || k > E) return 1;
  int pruned = 0;
  int *order = (int *)malloc(sizeof(int) * E);
  for (int t = 0; t < T; t++) {
    const float *l = logits + (size_t)t * E;
    /* selection sort on the ranking rule: obviously correct, O(E^2) */
    for (int i = 0; i < E; i++) order[i] = i;
    for (int i = 0; i < k; i++) {
      int best = i;
      for (int j = i + 1; j < E; j++)
        if (rank_before(l, order[j], order[best])) best = j;
      int tmp = order[i]; order[i] = order[best]; order[best] = tmp;
    }
    double ex[8], sum_all = 0.0;
    for (int r = 0; r < k; r++) {
      topk_idx[(size_t)t * k + r] = order[r];
      ex[r] = exp((double)l[order[r]] - (double)l[order[0]]);
      sum_all += ex[r];
    }
    int prot = important ? (important[t] != 0) : 0;
    uint8_t keep[8];
    keep[0] = 1;
    for (int r = 1; r < k; r++) {
      int drop;
      if (prot) {
        drop = 0;
      } else if (k == 2) {
        float gap = l[order[0]] - l[order[1]];      /* fp32 subtraction */
        drop = gap > delta32;
      } else {
        drop = ex[r] < tau * sum_all;               /* p_r < tau, in fp64 */
      }
      keep[r] = (uint8_t)!drop;
      pruned += drop;
    }
    double sum_kept = 0.0;
    for (int r = 0; r < k; r++) if (keep[r]) sum_kept += ex[r];
    for (int r = 0; r < k; r++) {
      kept[(size_t)t * k + r] = keep[r];
      topk_w[(size_t)t * k + r] = keep[r] ? ex[r] / sum_kept : 0.0;
      pair_pos[(size_t)t * k + r] = -1;
    }
  }
  free(order);
  int pos = 0;
  for (int e = 0; e < E; e++) {
    offsets[e] = pos;
    for (int t = 0; t < T; t++)
      for (int r = 0; r < k; r++)
        if (topk_idx[(size_t)t * k + r] == e && kept[(size_t)t * k + r]) {
          pair_token[pos] = t;
          pair_rank[pos] = r;
          pair_w[pos] = topk_w[(size_t)t * k + r];
          pair_pos[(size_t)t * k + r] = pos;
          pos++;
        }
    counts[e] = pos - offsets[e];
  }
  offsets[E] = pos;
  *n_pruned = pruned;
  return 0;
}

/* ------------------------------------------------------------------------ */
/* Expert FFN (SwiGLU) and Eq. 1 combination on exact dequantized weights.   */
/* ------------------------------------------------------------------------ */

static double silu(double a) { return a / (1.0 + exp(-a)); }

/* One expert on nt token vectors X[nt][d] (fp64).  Codes row-major per
 * matrix; scale/zero [R][K/G] per matrix.  H[nt][ffn] receives
 * silu(Wg x) * (Wu x); Y[nt][nrows] receives (Wd h) at the listed output rows
 * (rows == NULL: all d rows). */
int orc_expert_forward(const double *X, int nt, int d, int ffn, int G,
                       const uint8_t *qg, const uint16_t *sg, const uint16_t *zg,
                       const uint8_t *qu, const uint16_t *su, const uint16_t *zu,
                       const uint8_t *qd, const uint16_t *sd, const uint16_t *zd,
                       const int32_t *rows, int nrows, double *H, double *Y) {
  if (d % G || ffn % G) return 1;
  int ngd = d / G, ngf = ffn / G;
#pragma omp parallel for schedule(static)
  for (int n = 0; n < ffn; n++) {
    double *wg = (double *)malloc(sizeof(double) * d);
    double *wu = (double *)malloc(sizeof(double) * d);
    for (int c = 0; c < d; c++) {
      size_t gi = (size_t)n * ngd + c / G;
      wg[c] = orc_dequant(sg[gi], zg[gi], qg[(size_t)n * d + c]);
      wu[c] = orc_dequant(su[gi], zu[gi], qu[(size_t)n * d + c]);
    }
    for (int t = 0; t < nt; t++) {
      double a = 0.0, b = 0.0;
      for (int c = 0; c < d; c++) {
        a += wg[c] * X[(size_t)t * d + c];
        b += wu[c] * X[(size_t)t * d + c];
      }
      H[(size_t)t * ffn + n] = silu(a) * b;
    }
    free(wg);
    free(wu);
  }
  int nr = rows ? nrows : d;
#pragma omp parallel for schedule(static)
  for (int ri = 0; ri < nr; ri++) {
    int i = rows ? rows[ri] : ri;
    double *wd = (double *)malloc(sizeof(double) * ffn);
    for (int c = 0; c < ffn; c++) {
      size_t gi = (size_t)i * ngf + c / G;
      wd[c] = orc_dequant(sd[gi], zd[gi], qd[(size_t)i * ffn + c]);
    }
    for (int t = 0; t < nt; t++) {
      double acc = 0.0;
      for (int c = 0; c < ffn; c++) acc += wd[c] * H[(size_t)t * ffn + c];
      Y[(size_t)t * nr + ri] = acc;
    }
    free(wd);
  }
  return 0;
}

/* ------------------------------------------------------------------------ */
/* Token importance (Sec. 3.3.2, Eq. 6), the protected set, and the pruning */
/* threshold as a calibration median (Sec. 3.3.1).                          */
/* ------------------------------------------------------------------------ */

/* attn: [H][L][L] bf16 bits, attn[h][i][j] = attention probability of query i
 * on key j (causal: only j <= i is read); x: [L][d] bf16 bits (the tokens).
 * With 0-based j the key is seen by the queries i = j..L-1, L - j of them:
 *   I_j = ||x_j||_1 * (1/H) * sum_h sum_{i=j}^{L-1} attn[h][i][j] / (L - j)
 * in fp64.  mask: the n largest I_j, equal values ordered by lower index
 * (repeated selection of the best remaining token). */
int orc_token_importance(const uint16_t *attn, int H, int L, const uint16_t *x, int d, int n,
                         double *I, uint8_t *mask) {
  if (H <= 0 || L <= 0 || d <= 0 || n < 0 || n > L) return 1;
  for (int j = 0; j < L; j++) {
    double col = 0.0;
    for (int h = 0; h < H; h++)
      for (int i = j; i < L; i++) col += orc_bf16_to_double(attn[((size_t)h * L + i) * L + j]);
    double norm = 0.0;
    for (int c = 0; c < d; c++) norm += fabs(orc_bf16_to_double(x[(size_t)j * d + c]));
    I[j] = norm * (col / H) / (double)(L - j);
    mask[j] = 0;
  }
  for (int s = 0; s < n; s++) {
    int best = -1;
    for (int j = 0; j < L; j++)
      if (!mask[j] && (best < 0 || I[j] > I[best])) best = j;
    mask[best] = 1;
  }
  return 0;
}

static int cmp_double(const void *a, const void *b) {
  const double x = *(const double *)a, y = *(const double *)b;
  return x < y ? -1 : (x > y ? 1 : 0);
}

/* mu = the median over tokens of w_1 / w_0 = exp(l_1 - l_0) of the top-2
 * experts (ranking rule of orc_route); for an even count the mean of the two
 * middle values.  Returns mu, or -1 on bad arguments. */
double orc_median_ratio(const float *logits, int T, int E) {
  if (T <= 0 || E < 2) return -1.0;
  double *r = (double *)malloc(sizeof(double) * T);
  for (int t = 0; t < T; t++) {
    const float *l = logits + (size_t)t * E;
    int a = 0;
    for (int e = 1; e < E; e++) if (rank_before(l, e, a)) a = e;
    int b = a == 0 ? 1 : 0;
    for (int e = 0; e < E; e++) if (e != a && rank_before(l, e, b)) b = e;
    r[t] = exp((double)l[b] - (double)l[a]);
  }
  qsort(r, T, sizeof(double), cmp_double);
  const double mu = (T & 1) ? r[T / 2] : 0.5 * (r[T / 2 - 1] + r[T / 2]);
  free(r);
  return mu;
}
