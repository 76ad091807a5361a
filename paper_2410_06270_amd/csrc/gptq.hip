// gptq.hip -- the GPTQ quantizer the paper applies to every expert (Sec. 3.1:
// Hessian H = 2 X^T X of the layer-wise squared error, columns quantized in
// order with each column's error compensated on the columns after it), on
// the packed format of the Sec. 3.1 group quantizer.  All arithmetic fp64.
//
// Three steps, each its own entry point:
//   hessian   H (+)= 2 X^T X from bf16 calibration inputs X [N][K];
//   factor    dead inputs (H_kk = 0 -> H_kk = 1), damping H += damp * mean(diag
//             H) * I, and U, the upper Cholesky factor of H^-1 (H^-1 = U^T U);
//   quantize  for k = 0 .. K-1: at a group start the Sec. 3.1 scale/zero of
//             the fp32 rounding of the group's current values; q_k = nearest
//             level of fp32(w_k); e_k = (w_k - s (q_k - z)) / U_kk; w_j -= e_k
//             U_kj for j > k.  Codes and scale/zero go straight into the
//             layer's packed storage.
//
// U without forming H^-1: with J the index reversal, J H J = L L^T (lower
// Cholesky) gives H = V V^T with V = J L J upper triangular, so H^-1 =
// V^-T V^-1 and U = V^-1 = J L^-1 J.  The factor step therefore runs one
// blocked Cholesky and one recursive triangular inverse on the reversed matrix.
//
// Kernels: a tiled fp64 GEMM with arbitrary (also negative) strides carries
// the bulk of every step (Hessian, Cholesky trailing updates, the inverse's
// corner blocks, GPTQ's deferred updates); the sequential parts run one
// wavefront per row (64 x 64 triangular solves with readlane broadcasts, and
// the GPTQ column loop over 128-column blocks with the block of U in LDS).
#include "mc_internal.hpp"

namespace mc {

constexpr int kGemmTile = 64;
constexpr int kGemmK = 16;
constexpr int kNb = 64;            // Cholesky / inverse block
constexpr int kQb = 128;           // GPTQ column block
constexpr int kQRows = 16;         // rows (wavefronts) per GPTQ workgroup

__device__ __forceinline__ double load_f64(const double* p) { return *p; }
__device__ __forceinline__ double load_f64(const uint16_t* p) {
  return (double)__uint_as_float((uint32_t)*p << 16);
}

// C[m][n] += alpha * sum_k A(m, k) B(k, n), A(m, k) = A[m*sam + k*sak],
// B(k, n) = B[k*sbk + n*sbn]; 64 x 64 tiles, 4 x 4 outputs per thread.
// LOWER: tiles strictly above the diagonal are skipped.
// SEQ: C[m][n] -= A(m, k) B(k, n) one k after the other, each product and
// each subtraction rounded (alpha ignored): the order and roundings of
// applying GPTQ's per-column updates one column at a time.
template <typename TA, typename TB, bool LOWER, bool SEQ>
__global__ void __launch_bounds__(256) gemm_f64_kernel(int M, int N, int Kc, double alpha, const TA* __restrict__ A,
                                                       long long sam, long long sak, const TB* __restrict__ B,
                                                       long long sbk, long long sbn, double* __restrict__ C,
                                                       long long ldc) {
  const int tm = blockIdx.y, tn = blockIdx.x;
  if (LOWER && tn > tm) return;
  __shared__ double As[kGemmK][kGemmTile + 1];
  __shared__ double Bs[kGemmK][kGemmTile + 1];
  const int tid = threadIdx.x, tx = tid & 15, ty = tid >> 4;
  const int m0 = tm * kGemmTile, n0 = tn * kGemmTile;
  const bool a_kfast = sak == 1, b_nfast = sbn == 1;
  double acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int m = m0 + ty + 16 * i, n = n0 + tx + 16 * j;
      acc[i][j] = (SEQ && m < M && n < N) ? C[(long long)m * ldc + n] : 0.0;
    }

  for (int k0 = 0; k0 < Kc; k0 += kGemmK) {
#pragma unroll
    for (int p = 0; p < 4; ++p) {
      const int e = tid + 256 * p;
      const int am = a_kfast ? e >> 4 : e & 63, ak = a_kfast ? e & 15 : e >> 6;
      const int gm = m0 + am, gk = k0 + ak;
      As[ak][am] = (gm < M && gk < Kc) ? load_f64(A + (long long)gm * sam + (long long)gk * sak) : 0.0;
      const int bn = b_nfast ? e & 63 : e >> 4, bk = b_nfast ? e >> 6 : e & 15;
      const int gn = n0 + bn, gk2 = k0 + bk;
      Bs[bk][bn] = (gn < N && gk2 < Kc) ? load_f64(B + (long long)gk2 * sbk + (long long)gn * sbn) : 0.0;
    }
    __syncthreads();
#pragma unroll 4
    for (int kk = 0; kk < kGemmK; ++kk) {
      double a[4], b[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) a[i] = As[kk][ty + 16 * i];
#pragma unroll
      for (int j = 0; j < 4; ++j) b[j] = Bs[kk][tx + 16 * j];
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j)
          acc[i][j] = SEQ ? __dsub_rn(acc[i][j], __dmul_rn(a[i], b[j])) : __fma_rn(a[i], b[j], acc[i][j]);
    }
    __syncthreads();
  }
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int m = m0 + ty + 16 * i, n = n0 + tx + 16 * j;
      if (m < M && n < N) C[(long long)m * ldc + n] = SEQ ? acc[i][j] : C[(long long)m * ldc + n] + alpha * acc[i][j];
    }
}

template <typename TA, typename TB, bool SEQ = false>
static void gemm(int M, int N, int Kc, double alpha, const TA* A, long long sam, long long sak, const TB* B,
                 long long sbk, long long sbn, double* C, long long ldc, bool lower, hipStream_t st) {
  if (M <= 0 || N <= 0 || Kc <= 0) return;
  const dim3 grid((N + kGemmTile - 1) / kGemmTile, (M + kGemmTile - 1) / kGemmTile);
  if (lower)
    hipLaunchKernelGGL((gemm_f64_kernel<TA, TB, true, SEQ>), grid, dim3(256), 0, st, M, N, Kc, alpha, A, sam, sak, B,
                       sbk, sbn, C, ldc);
  else
    hipLaunchKernelGGL((gemm_f64_kernel<TA, TB, false, SEQ>), grid, dim3(256), 0, st, M, N, Kc, alpha, A, sam, sak,
                       B, sbk, sbn, C, ldc);
}

__global__ void __launch_bounds__(256) fill_f64_kernel(double* __restrict__ p, long long rows, int cols, long long ld) {
  const long long n = rows * cols;
  for (long long i = (long long)blockIdx.x * 256 + threadIdx.x; i < n; i += (long long)gridDim.x * 256)
    p[(i / cols) * ld + i % cols] = 0.0;
}

static void zero2d(double* p, long long rows, int cols, long long ld, hipStream_t st) {
  const long long n = rows * cols;
  if (n <= 0) return;
  const long long blocks = (n + 255) / 256;
  hipLaunchKernelGGL(fill_f64_kernel, dim3((unsigned)(blocks < 8192 ? blocks : 8192)), dim3(256), 0, st, p, rows,
                     cols, ld);
}

// ---------------------------------------------------------------- factor --
// mean of the diagonal with dead entries counted as 1 (fixed order), times damp.
__global__ void __launch_bounds__(1024) gptq_diag_kernel(const double* __restrict__ H, int K, double damp,
                                                         uint8_t* __restrict__ dead, double* __restrict__ aux) {
  __shared__ double red[16];
  double s = 0.0;
  for (int k = threadIdx.x; k < K; k += 1024) {
    const double h = H[(size_t)k * K + k];
    dead[k] = h == 0.0 ? 1 : 0;
    s += h == 0.0 ? 1.0 : h;
  }
  for (int off = 32; off > 0; off >>= 1) s += __shfl_xor(s, off);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = s;
  __syncthreads();
  if (threadIdx.x == 0) {
    double t = 0.0;
    for (int w = 0; w < 16; ++w) t += red[w];
    aux[0] = damp * (t / K);
  }
}

// A[i][j] = H[K-1-i][K-1-j], dead diagonal entries 1, plus the damping.
__global__ void __launch_bounds__(256) gptq_reverse_kernel(const double* __restrict__ H, int K,
                                                           const double* __restrict__ aux, double* __restrict__ A) {
  const long long n = (long long)K * K;
  const double add = aux[0];
  for (long long idx = (long long)blockIdx.x * 256 + threadIdx.x; idx < n; idx += (long long)gridDim.x * 256) {
    const int i = (int)(idx / K), j = (int)(idx % K);
    double h = H[(size_t)(K - 1 - i) * K + (K - 1 - j)];
    if (i == j) h = (h == 0.0 ? 1.0 : h) + add;
    A[idx] = h;
  }
}

// In-place Cholesky of the 64 x 64 diagonal block kb (lower triangle).
__global__ void __launch_bounds__(256) chol_diag_kernel(double* __restrict__ A, int K, int kb) {
  __shared__ double a[kNb][kNb + 1];
  double* blk = A + (size_t)kb * kNb * K + (size_t)kb * kNb;
  const int tid = threadIdx.x;
  for (int idx = tid; idx < kNb * kNb; idx += 256) a[idx >> 6][idx & 63] = blk[(size_t)(idx >> 6) * K + (idx & 63)];
  __syncthreads();
  for (int j = 0; j < kNb; ++j) {
    if (tid == 0) a[j][j] = sqrt(a[j][j]);
    __syncthreads();
    if (tid > j && tid < kNb) a[tid][j] = a[tid][j] / a[j][j];
    __syncthreads();
    for (int idx = tid; idx < kNb * kNb; idx += 256) {
      const int i = idx >> 6, c = idx & 63;
      if (c > j && i >= c) a[i][c] -= a[i][j] * a[c][j];
    }
    __syncthreads();
  }
  for (int idx = tid; idx < kNb * kNb; idx += 256) {
    const int i = idx >> 6, c = idx & 63;
    if (i >= c) blk[(size_t)i * K + c] = a[i][c];
  }
}

// Panel below block kb: each row x of A[r][kb*64 .. +64] solves x L_kk^T = a.
// One wavefront per row; lane j holds column j.
__global__ void __launch_bounds__(256) chol_panel_kernel(double* __restrict__ A, int K, int kb) {
  __shared__ double Lt[kNb][kNb];      // Lt[m][j] = L_kk[j][m]
  const double* blk = A + (size_t)kb * kNb * K + (size_t)kb * kNb;
  for (int idx = threadIdx.x; idx < kNb * kNb; idx += 256) {
    const int j = idx >> 6, m = idx & 63;
    Lt[m][j] = j >= m ? blk[(size_t)j * K + m] : 0.0;
  }
  __syncthreads();
  const int row = (kb + 1) * kNb + blockIdx.x * 4 + (int)(threadIdx.x >> 6);
  if (row >= K) return;
  const int l = threadIdx.x & 63;
  double* a = A + (size_t)row * K + (size_t)kb * kNb;
  double r = a[l], x = 0.0;
  for (int m = 0; m < kNb; ++m) {
    const double xm = readlane_f64(r, m) / Lt[m][m];
    if (l == m) x = xm;
    if (l > m) r -= xm * Lt[m][l];
  }
  a[l] = x;
}

// Mi[ib][ib] = inverse of the lower 64 x 64 block L_ii (zeros above its
// diagonal).  16 wavefronts, 4 columns each; lane i holds row i.
__global__ void __launch_bounds__(1024) tri_inv_diag_kernel(const double* __restrict__ A, int K, int ib,
                                                            double* __restrict__ Mi) {
  __shared__ double Lt[kNb][kNb];      // Lt[m][i] = L_ii[i][m]
  const double* blk = A + (size_t)ib * kNb * K + (size_t)ib * kNb;
  for (int idx = threadIdx.x; idx < kNb * kNb; idx += 1024) {
    const int i = idx >> 6, m = idx & 63;
    Lt[m][i] = i >= m ? blk[(size_t)i * K + m] : 0.0;
  }
  __syncthreads();
  const int l = threadIdx.x & 63, w = (int)(threadIdx.x >> 6);
  double* out = Mi + (size_t)ib * kNb * K + (size_t)ib * kNb;
  for (int t = 0; t < 4; ++t) {
    const int c = 4 * w + t;
    double r = l == c ? 1.0 : 0.0, y = 0.0;
    for (int m = c; m < kNb; ++m) {
      const double ym = readlane_f64(r, m) / Lt[m][m];
      if (l == m) y = ym;
      if (l > m) r -= Lt[m][l] * ym;
    }
    out[(size_t)l * K + c] = l >= c ? y : 0.0;
  }
}

// U[i][j] = Mi[K-1-i][K-1-j] on and above the diagonal, 0 below.
__global__ void __launch_bounds__(256) gptq_unreverse_kernel(const double* __restrict__ Mi, int K,
                                                             double* __restrict__ U) {
  const long long n = (long long)K * K;
  for (long long idx = (long long)blockIdx.x * 256 + threadIdx.x; idx < n; idx += (long long)gridDim.x * 256) {
    const int i = (int)(idx / K), j = (int)(idx % K);
    U[idx] = j >= i ? Mi[(size_t)(K - 1 - i) * K + (K - 1 - j)] : 0.0;
  }
}

static unsigned grid_for(long long n) {
  const long long b = (n + 255) / 256;
  return (unsigned)(b < 16384 ? b : 16384);
}

// Rows/columns of the first half of a recursive split of n (a multiple of 64).
static int split_half(int n) { return ((n / kNb) / 2) * kNb; }

// Workspace of the factor: the reversed matrix and its Cholesky factor (in
// place), the inverse, the inverse's scratch product (at most the first split's
// (n - n1) x n1 block) and one scalar.
size_t gptq_factor_bytes(int K) {
  const int n1 = split_half(K);
  return 2 * (size_t)K * K * sizeof(double) + (size_t)(K - n1) * (size_t)(n1 > 0 ? n1 : 1) * sizeof(double) + 256;
}

// Mi[off..off+n)^2 = inverse of the lower-triangular L[off..off+n)^2 (both
// row-major with leading dimension K; Mi's strictly upper part in the range
// is zero on entry and stays zero).  With L = [[A, 0], [B, C]]:
// L^-1 = [[A^-1, 0], [-C^-1 B A^-1, C^-1]], the two halves recursively, the
// corner by two GEMMs through the scratch X; 64 x 64 blocks by wavefront
// substitution.
static void tri_inverse(const double* L, double* Mi, double* X, int K, int off, int n, hipStream_t st) {
  if (n == kNb) {
    hipLaunchKernelGGL(tri_inv_diag_kernel, dim3(1), dim3(1024), 0, st, L, K, off / kNb, Mi);
    return;
  }
  const int n1 = split_half(n), n2 = n - n1;
  tri_inverse(L, Mi, X, K, off, n1, st);
  tri_inverse(L, Mi, X, K, off + n1, n2, st);
  const double* B = L + (size_t)(off + n1) * K + off;             // n2 x n1
  const double* Ainv = Mi + (size_t)off * K + off;                // n1 x n1
  const double* Cinv = Mi + (size_t)(off + n1) * K + off + n1;    // n2 x n2
  zero2d(X, n2, n1, n1, st);
  gemm<double, double>(n2, n1, n1, 1.0, B, K, 1, Ainv, K, 1, X, n1, false, st);          // X = B A^-1
  gemm<double, double>(n2, n1, n2, -1.0, Cinv, K, 1, X, n1, 1, Mi + (size_t)(off + n1) * K + off, K, false, st);
}

hipError_t launch_gptq_hessian(const uint16_t* x, int N, int K, double* H, bool accumulate, hipStream_t st) {
  timing_begin(st, kSiteGptqHessian);
  if (!accumulate) zero2d(H, K, K, K, st);
  // H(m, n) += 2 sum_t X[t][m] X[t][n]
  gemm<uint16_t, uint16_t>(K, K, N, 2.0, x, 1, K, x, K, 1, H, K, false, st);
  timing_end(st, kSiteGptqHessian);
  return hipGetLastError();
}

hipError_t launch_gptq_factor(const double* H, int K, double damp, double* U, uint8_t* dead, void* ws,
                              hipStream_t st) {
  double* A = static_cast<double*>(ws);
  double* Mi = A + (size_t)K * K;
  double* X = Mi + (size_t)K * K;
  const int n1 = split_half(K);
  double* aux = X + (size_t)(K - n1) * (size_t)(n1 > 0 ? n1 : 1);
  const int nb = K / kNb;
  timing_begin(st, kSiteGptqFactor);
  hipLaunchKernelGGL(gptq_diag_kernel, dim3(1), dim3(1024), 0, st, H, K, damp, dead, aux);
  hipLaunchKernelGGL(gptq_reverse_kernel, dim3(grid_for((long long)K * K)), dim3(256), 0, st, H, K, aux, A);
  zero2d(Mi, K, K, K, st);
  for (int kb = 0; kb < nb; ++kb) {
    hipLaunchKernelGGL(chol_diag_kernel, dim3(1), dim3(256), 0, st, A, K, kb);
    const int rows = K - (kb + 1) * kNb;
    if (rows > 0) {
      hipLaunchKernelGGL(chol_panel_kernel, dim3((rows + 3) / 4), dim3(256), 0, st, A, K, kb);
      const double* p = A + (size_t)(kb + 1) * kNb * K + (size_t)kb * kNb;
      gemm<double, double>(rows, rows, kNb, -1.0, p, K, 1, p, 1, K,
                           A + (size_t)(kb + 1) * kNb * K + (size_t)(kb + 1) * kNb, K, true, st);
    }
  }
  tri_inverse(A, Mi, X, K, 0, K, st);
  hipLaunchKernelGGL(gptq_unreverse_kernel, dim3(grid_for((long long)K * K)), dim3(256), 0, st, Mi, K, U);
  timing_end(st, kSiteGptqFactor);
  return hipGetLastError();
}

// -------------------------------------------------------------- quantize --
size_t gptq_quantize_bytes(int R, int K) {
  const size_t ww = (size_t)R * K * sizeof(double);
  const size_t er = (size_t)R * kQb * sizeof(double);
  return ww + er + (((size_t)R * K + 255) / 256) * 256;
}

__global__ void __launch_bounds__(256) gptq_prep_kernel(const float* __restrict__ W, const uint8_t* __restrict__ dead,
                                                        int R, int K, double* __restrict__ Ww,
                                                        double* __restrict__ loss) {
  const long long n = (long long)R * K;
  for (long long idx = (long long)blockIdx.x * 256 + threadIdx.x; idx < n; idx += (long long)gridDim.x * 256)
    Ww[idx] = dead[idx % K] ? 0.0 : (double)W[idx];
  if (loss)
    for (long long r = (long long)blockIdx.x * 256 + threadIdx.x; r < R; r += (long long)gridDim.x * 256) loss[r] = 0.0;
}

// One 128-column block [b0, b0 + 128) for 16 rows: one wavefront per row,
// lane l holds columns b0 + l and b0 + 64 + l; the block of U sits in LDS.
// Writes the codes, the block's errors e_k (for the deferred update of the
// columns after the block), the scale/zero words and the loss.
__global__ void __launch_bounds__(1024) gptq_block_kernel(double* __restrict__ Ww, const double* __restrict__ U,
                                                          int R, int K, int b0, int bits, int G,
                                                          uint8_t* __restrict__ q, double* __restrict__ Er,
                                                          uint32_t* __restrict__ sz, double* __restrict__ loss) {
  __shared__ double Ub[kQb][kQb];
  for (int idx = threadIdx.x; idx < kQb * kQb; idx += 1024) {
    const int k = idx >> 7, j = idx & 127;
    Ub[k][j] = j >= k ? U[(size_t)(b0 + k) * K + b0 + j] : 0.0;
  }
  __syncthreads();
  const int row = blockIdx.x * kQRows + (int)(threadIdx.x >> 6);
  if (row >= R) return;
  const int l = threadIdx.x & 63;
  const int Lc = (1 << bits) - 1, ng = K / G;
  double* w = Ww + (size_t)row * K + b0;
  double v0 = w[l], v1 = w[64 + l];
  uint32_t c0 = 0, c1 = 0;
  double e0 = 0.0, e1 = 0.0, s = 1.0, z = 0.0, lsum = 0.0;
  for (int k = 0; k < kQb; ++k) {
    if (k % G == 0) {
      const float f0 = (float)v0, f1 = (float)v1;
      const bool in0 = l >= k && l < k + G, in1 = 64 + l >= k && 64 + l < k + G;
      float mn = in0 ? f0 : __builtin_inff(), mx = in0 ? f0 : -__builtin_inff();
      if (in1) {
        mn = fminf(mn, f1);
        mx = fmaxf(mx, f1);
      }
      for (int off = 1; off < 64; off <<= 1) {
        mn = fminf(mn, __shfl_xor(mn, off));
        mx = fmaxf(mx, __shfl_xor(mx, off));
      }
      const uint32_t word = group_sz_word(mn, mx, bits);
      s = (double)half_bits_to_float(word & 0xffffu);
      z = (double)half_bits_to_float(word >> 16);
      if (l == 0) {
        const int g = (b0 + k) / G;
        sz[((size_t)(row / 16) * ng + g) * 16 + (row % 16)] = word;
      }
    }
    const double wk = readlane_f64(k < 64 ? v0 : v1, k & 63);
    const int code = nearest_code((float)wk, s, z, Lc);
    const double err = (wk - s * ((double)code - z)) / Ub[k][k];
    lsum += err * err / 2.0;
    if (l == (k & 63)) {
      if (k < 64) {
        c0 = (uint32_t)code;
        e0 = err;
      } else {
        c1 = (uint32_t)code;
        e1 = err;
      }
    }
    if (l > k) v0 = __dsub_rn(v0, __dmul_rn(err, Ub[k][l]));
    if (64 + l > k) v1 = __dsub_rn(v1, __dmul_rn(err, Ub[k][64 + l]));
  }
  uint8_t* qr = q + (size_t)row * K + b0;
  qr[l] = (uint8_t)c0;
  qr[64 + l] = (uint8_t)c1;
  Er[(size_t)row * kQb + l] = e0;
  Er[(size_t)row * kQb + 64 + l] = e1;
  if (l == 0 && loss) loss[row] += lsum;
}

// Codes [R][K] -> the packed words of one matrix (same layout as the pack
// kernel): one thread per (16 x 128 tile, lane), the width a compile-time
// constant so that every code lands at a fixed bit position.
template <int B>
__global__ void __launch_bounds__(256) pack_codes_u8_kernel(const uint8_t* __restrict__ q, int R, int K,
                                                            uint32_t* __restrict__ words) {
  const long long tid = (long long)blockIdx.x * 256 + threadIdx.x;
  if (tid >= (long long)R * K / 32) return;
  const int lane = (int)(tid & 63);
  const long long tile = tid >> 6;
  const int tiles_per_row = K / kTileCols;
  const int trow = (int)(tile / tiles_per_row), tcol = (int)(tile % tiles_per_row);
  const int n = trow * kTileRows + (lane & 15), kq = lane >> 4;
  uint32_t w[3] = {0u, 0u, 0u};
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    const int k0 = tcol * kTileCols + 32 * u + 8 * kq;
    const uint2 v = *reinterpret_cast<const uint2*>(q + (size_t)n * K + k0);
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const uint32_t code = ((j < 4 ? v.x : v.y) >> (8 * (j & 3))) & 0xffu;
      place_code(w, code, 4 * u + (j >> 1), j & 1, B);
    }
  }
  uint32_t* dst = words + ((size_t)tile * 64 + lane) * B;
#pragma unroll
  for (int p = 0; p < B; ++p) dst[p] = w[p];
}

hipError_t launch_gptq_quantize(const float* W, const double* U, const uint8_t* dead, int R, int K, int bits, int G,
                                uint32_t* words, uint32_t* sz, double* loss, void* ws, hipStream_t st) {
  double* Ww = static_cast<double*>(ws);
  double* Er = Ww + (size_t)R * K;
  uint8_t* q = reinterpret_cast<uint8_t*>(Er + (size_t)R * kQb);
  timing_begin(st, kSiteGptqQuantize);
  hipLaunchKernelGGL(gptq_prep_kernel, dim3(grid_for((long long)R * K)), dim3(256), 0, st, W, dead, R, K, Ww, loss);
  for (int b0 = 0; b0 < K; b0 += kQb) {
    hipLaunchKernelGGL(gptq_block_kernel, dim3((R + kQRows - 1) / kQRows), dim3(1024), 0, st, Ww, U, R, K, b0, bits,
                       G, q, Er, sz, loss);
    const int rest = K - b0 - kQb;
    if (rest > 0)   // w[:, b0+128:] -= E_block U[b0:b0+128, b0+128:], column by column
      gemm<double, double, true>(R, rest, kQb, -1.0, Er, kQb, 1, U + (size_t)b0 * K + b0 + kQb, K, 1, Ww + b0 + kQb, K,
                           false, st);
  }
  const dim3 pgrid((unsigned)(((long long)R * K / 32 + 255) / 256));
  if (bits == 1)
    hipLaunchKernelGGL(pack_codes_u8_kernel<1>, pgrid, dim3(256), 0, st, q, R, K, words);
  else if (bits == 2)
    hipLaunchKernelGGL(pack_codes_u8_kernel<2>, pgrid, dim3(256), 0, st, q, R, K, words);
  else
    hipLaunchKernelGGL(pack_codes_u8_kernel<3>, pgrid, dim3(256), 0, st, q, R, K, words);
  timing_end(st, kSiteGptqQuantize);
  return hipGetLastError();
}

}  // namespace mc
