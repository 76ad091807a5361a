// pmq.hip -- the reconstruction error of Sec. 3.2.2 (the unnumbered equation
// before Eq. 4) that feeds the bit-width programme of Eq. 4, measured layer
// by layer on calibration tokens:
//   eps[e][b] = || F(theta) - F(theta[e -> Q(e, b)]) ||_F,
// F the MoE layer's output (Eq. 1) over the calibration batch, theta the fp32
// weights, Q(e, b) expert e quantized at b bits by the min-max RTN quantizer
// of mc_pack.  Quantizing expert e changes only the terms of the tokens that
// keep e, so the difference is, per token t keeping e with weight w_t,
//   w_t * (E_e^(b)(x_t) - E_e(x_t)),
// and eps[e][b]^2 is the sum of their squared norms.  E_e^(b)(x_t) comes from
// the packed forward's own expert kernels (every expert packed at b bits, the
// per-pair outputs before the weighted combine); E_e(x_t) from the dense fp32
// kernels below (fp32 weights, fp32 arithmetic, h = silu(g) * u kept in fp32).
// Offline code: plain tiled fp32 GEMMs, not tuned.
#include "forward_engine.hpp"
#include "mc_internal.hpp"

namespace mc {

namespace {

constexpr int kDnTile = 64;   // pairs and output rows per workgroup
constexpr int kDnK = 32;      // reduction step staged in LDS

// out[pos][n] for the kept pairs pos of expert e = blockIdx.z (its CSR range,
// 64 per workgroup along x) and rows n of the 64-row tile blockIdx.y:
//   gate/up: A = x[token(pos)] (bf16), out = silu(A.Wa[e][n]) * (A.Wb[e][n]), K = d;
//   down:    A = hin[pos] (fp32),       out = A.Wa[e][n],                     K = ffn.
// Weights fp32 [E][N][K] row-major; each thread holds a 4 x 4 block of the
// 64 x 64 tile and sums over K in column order.
template <bool GATEUP>
__global__ void __launch_bounds__(256) dense_expert_kernel(const float* __restrict__ Wa, const float* __restrict__ Wb,
                                                           const uint16_t* __restrict__ x,
                                                           const float* __restrict__ hin,
                                                           const int32_t* __restrict__ offsets,
                                                           const int32_t* __restrict__ pair_token, int T, int P,
                                                           int N, int K, float* __restrict__ out) {
  __shared__ float As[kDnK][kDnTile + 4];
  __shared__ float Ba[kDnK][kDnTile + 4];
  __shared__ float Bb[kDnK][kDnTile + 4];
  const int e = blockIdx.z;
  int ebase, ecount;
  expert_range_offsets(offsets, e, P, ebase, ecount);
  const int m0 = blockIdx.x * kDnTile, n0 = blockIdx.y * kDnTile;
  if (m0 >= ecount) return;
  const int tid = threadIdx.x, tx = tid & 15, ty = tid >> 4;
  const float* wa = Wa + ((size_t)e * N + n0) * K;
  const float* wb = GATEUP ? Wb + ((size_t)e * N + n0) * K : nullptr;
  float ca[4][4] = {}, cb[4][4] = {};
  for (int k0 = 0; k0 < K; k0 += kDnK) {
#pragma unroll
    for (int i = 0; i < kDnTile * kDnK / 256; ++i) {
      const int idx = tid + 256 * i, r = idx / kDnK, c = idx % kDnK;
      const int m = m0 + r;
      float v = 0.0f;
      if (m < ecount) {
        const int pos = ebase + m;
        if constexpr (GATEUP)
          v = bf16_bits_to_float(x[(size_t)clamp_token(pair_token[pos], T) * K + k0 + c]);
        else
          v = hin[(size_t)pos * K + k0 + c];
      }
      As[c][r] = v;
      Ba[c][r] = wa[(size_t)r * K + k0 + c];
      if constexpr (GATEUP) Bb[c][r] = wb[(size_t)r * K + k0 + c];
    }
    __syncthreads();
#pragma unroll 4
    for (int kk = 0; kk < kDnK; ++kk) {
      float a[4], b[4], bb[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        a[i] = As[kk][ty * 4 + i];
        b[i] = Ba[kk][tx * 4 + i];
        if constexpr (GATEUP) bb[i] = Bb[kk][tx * 4 + i];
      }
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          ca[i][j] = fmaf(a[i], b[j], ca[i][j]);
          if constexpr (GATEUP) cb[i][j] = fmaf(a[i], bb[j], cb[i][j]);
        }
    }
    __syncthreads();
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int m = m0 + ty * 4 + i;
    if (m >= ecount) continue;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const float v = GATEUP ? silu(ca[i][j]) * cb[i][j] : ca[i][j];
      out[(size_t)(ebase + m) * N + n0 + tx * 4 + j] = v;
    }
  }
}

// eps[e][b-1] = sqrt(sum over e's kept pairs pos and rows m of
// (w_pos * (sum_s partial[s][pos][m] - dense[pos][m]))^2), one workgroup per
// expert, fp64 sums in a fixed order (strided per thread, then a tree).
__global__ void __launch_bounds__(256) pmq_error_kernel(const float* __restrict__ partial, size_t part_stride,
                                                        int nsplit, const float* __restrict__ dense,
                                                        const int32_t* __restrict__ offsets,
                                                        const float* __restrict__ pair_w, int P, int d, int b,
                                                        double* __restrict__ eps) {
  __shared__ double red[256];
  const int e = blockIdx.x, t = threadIdx.x;
  int ebase, ecount;
  expert_range_offsets(offsets, e, P, ebase, ecount);
  const long long n = (long long)ecount * d;
  double acc = 0.0;
  for (long long i = t; i < n; i += blockDim.x) {
    const int pos = ebase + (int)(i / d), m = (int)(i % d);
    float q = 0.0f;
    for (int s = 0; s < nsplit; ++s) q += partial[(size_t)s * part_stride + (size_t)pos * d + m];
    const double diff = ((double)q - (double)dense[(size_t)pos * d + m]) * (double)pair_w[pos];
    acc += diff * diff;
  }
  red[t] = acc;
  __syncthreads();
  for (int off = 128; off > 0; off >>= 1) {
    if (t < off) red[t] += red[t + off];
    __syncthreads();
  }
  if (t == 0) eps[e * 3 + (b - 1)] = sqrt(red[0]);
}

}  // namespace

hipError_t launch_dense_expert(const float* wg, const float* wu, const float* wd, int E, int d, int ffn,
                               const uint16_t* x, const mc_routing& r, float* h, float* y, hipStream_t stream) {
  const int P = r.T * r.k;
  const int mt = (P + kDnTile - 1) / kDnTile;
  hipLaunchKernelGGL(dense_expert_kernel<true>, dim3(mt, ffn / kDnTile, E), dim3(256), 0, stream, wg, wu, x,
                     nullptr, r.offsets, r.pair_token, r.T, P, ffn, d, h);
  hipError_t err = hipGetLastError();
  if (err != hipSuccess) return err;
  hipLaunchKernelGGL(dense_expert_kernel<false>, dim3(mt, d / kDnTile, E), dim3(256), 0, stream, wd, nullptr,
                     nullptr, h, r.offsets, r.pair_token, r.T, P, d, ffn, y);
  return hipGetLastError();
}

hipError_t launch_pmq_error(const float* partial, size_t part_stride, int nsplit, const float* dense,
                            const mc_routing& r, int d, int b, double* eps, hipStream_t stream) {
  hipLaunchKernelGGL(pmq_error_kernel, dim3(r.E), dim3(256), 0, stream, partial, part_stride, nsplit, dense,
                     r.offsets, r.pair_w, r.T * r.k, d, b, eps);
  return hipGetLastError();
}

}  // namespace mc
