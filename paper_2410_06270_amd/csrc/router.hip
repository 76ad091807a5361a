// router.hip -- the router's linear layer ahead of routing (Eq. 1: the gate
// scores G(x) are the top-k of x W_r^T).
//
//   logits[t][e] = sum_k x[t][k] * w[e][k],   x [T][d], w [E][d] bf16.
//
// Every product of two bf16 values is exact in fp64 (8-bit significands, and
// the fp64 exponent range holds every product); the d products are summed in
// fp64 and the sum is rounded once to fp32.  The result is faithful: it lies
// between the fp32 roundings of S - g and S + g, S the exact sum and
// g = (d - 1) 2^-53 sum |x_k w_k| the fp64 summation bound (which holds for
// any order of the additions), so it is the correctly rounded value unless S
// lies within g of an fp32 rounding boundary.
//
// With 16 or more experts the sums run on fp64 MFMAs (16x16x4): a workgroup
// of WAVES waves computes a tile of 16 tokens x 16 experts, each wave over a
// 1/WAVES share of the d axis.  Lane l of a wave loads 16-byte pieces (8
// bf16) of token row l % 16 and of expert row l % 16; the four lane groups
// take four consecutive pieces, and the 8 MFMAs of a step take element j of
// every lane's pieces, so that a step covers 32 columns; loads are issued four
// steps ahead of their MFMAs.  The waves' partial tiles are added through LDS
// in wave order (deterministic).  Batches of at least 512 tokens take this
// path (WAVES = 4).
//
// Otherwise (fewer experts: an MFMA tile would be half empty at 8; or a
// small batch, where a few tiles leave the GPU idle) one workgroup
// of 256 threads computes NT tokens x 8 experts with fp64 fmas: each thread
// takes 16-byte pieces of the d axis, strided by 256 pieces, keeps NT * 8 fp64
// accumulators, and the partial sums are reduced through LDS and a short
// shuffle tree in a fixed order.
#include "mc_internal.hpp"

namespace mc {

typedef double f64x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ double bf16_lo(uint32_t w) { return (double)__uint_as_float(w << 16); }
__device__ __forceinline__ double bf16_hi(uint32_t w) { return (double)__uint_as_float(w & 0xffff0000u); }

constexpr int kRtThreads = 256;
constexpr int kRtExperts = 8;

template <int NT>
__global__ void __launch_bounds__(kRtThreads) router_valu_kernel(const uint16_t* __restrict__ x,
                                                            const uint16_t* __restrict__ w, int T, int d,
                                                            int E, float* __restrict__ logits) {
  constexpr int NO = NT * kRtExperts;            // outputs of the workgroup
  constexpr int PER = kRtThreads / NO;           // threads that finish one output
  constexpr int SPAN = kRtThreads / PER;         // partials each of them adds first
  static_assert(kRtThreads % NO == 0 && (PER & (PER - 1)) == 0, "output split");
  __shared__ double red[NO][kRtThreads];

  const int tid = threadIdx.x;
  const int t0 = blockIdx.x * NT;
  const int e0 = blockIdx.y * kRtExperts;
  const int pieces = d >> 3;

  double acc[NT][kRtExperts];
#pragma unroll
  for (int i = 0; i < NT; ++i)
#pragma unroll
    for (int j = 0; j < kRtExperts; ++j) acc[i][j] = 0.0;

  for (int p = tid; p < pieces; p += kRtThreads) {
    u32x4 xv[NT], wv[kRtExperts];
#pragma unroll
    for (int i = 0; i < NT; ++i) {
      const int t = t0 + i;
      xv[i] = t < T ? *reinterpret_cast<const u32x4*>(x + (size_t)t * d + 8 * p) : u32x4{0u, 0u, 0u, 0u};
    }
#pragma unroll
    for (int j = 0; j < kRtExperts; ++j) {
      const int e = e0 + j;
      wv[j] = e < E ? *reinterpret_cast<const u32x4*>(w + (size_t)e * d + 8 * p) : u32x4{0u, 0u, 0u, 0u};
    }
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      double xl[NT], xh[NT];
#pragma unroll
      for (int i = 0; i < NT; ++i) {
        xl[i] = bf16_lo(xv[i][c]);
        xh[i] = bf16_hi(xv[i][c]);
      }
#pragma unroll
      for (int j = 0; j < kRtExperts; ++j) {
        const double wl = bf16_lo(wv[j][c]), wh = bf16_hi(wv[j][c]);
#pragma unroll
        for (int i = 0; i < NT; ++i) acc[i][j] = __fma_rn(xh[i], wh, __fma_rn(xl[i], wl, acc[i][j]));
      }
    }
  }

#pragma unroll
  for (int i = 0; i < NT; ++i)
#pragma unroll
    for (int j = 0; j < kRtExperts; ++j) red[i * kRtExperts + j][tid] = acc[i][j];
  __syncthreads();

  const int o = tid / PER, part = tid % PER;
  double s = 0.0;
  for (int q = 0; q < SPAN; ++q) s += red[o][part * SPAN + q];
#pragma unroll
  for (int m = PER >> 1; m > 0; m >>= 1) s += __shfl_xor(s, m, PER);
  const int t = t0 + o / kRtExperts, e = e0 + o % kRtExperts;
  if (part == 0 && t < T && e < E) logits[(size_t)t * E + e] = (float)s;
}

// The MFMA tiles pay off on large grids only (measured, 64 experts, d = 2048:
// 43.8 -> 19.0 us at 2048 tokens, 6.2 -> 10.4 us at 16 tokens).
constexpr int kRtMfmaMinT = 512;

template <int WAVES>
__global__ void __launch_bounds__(64 * WAVES) router_mfma_kernel(const uint16_t* __restrict__ x,
                                                               const uint16_t* __restrict__ w, int T, int d,
                                                               int E, float* __restrict__ logits) {
  __shared__ double red[WAVES - 1][4][64];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int row = lane & 15, g = lane >> 4;
  const int t = blockIdx.x * 16 + row, e = blockIdx.y * 16 + row;
  const bool tv = t < T, ev = e < E;
  const u32x4* xr = reinterpret_cast<const u32x4*>(x + (size_t)(tv ? t : 0) * d);
  const u32x4* wr = reinterpret_cast<const u32x4*>(w + (size_t)(ev ? e : 0) * d);
  // pieces of 8 columns: wave `wave` takes [p0, p1), a multiple of 4 long
  const int pieces = d >> 3;
  const int per = ((pieces + WAVES - 1) / WAVES + 3) & ~3;
  const int p0 = wave * per;
  const int p1 = (p0 + per) < pieces ? (p0 + per) : pieces;

  f64x4 acc = {0.0, 0.0, 0.0, 0.0};
  for (int pb = p0; pb < p1; pb += 16) {          // uniform trip count over the wave
    u32x4 xv[4], wv[4];
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      const int p = pb + 4 * s + g;
      const bool ok = p < p1;
      xv[s] = (ok && tv) ? xr[p] : u32x4{0u, 0u, 0u, 0u};
      wv[s] = (ok && ev) ? wr[p] : u32x4{0u, 0u, 0u, 0u};
    }
#pragma unroll
    for (int s = 0; s < 4; ++s)
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        acc = __builtin_amdgcn_mfma_f64_16x16x4f64(bf16_lo(xv[s][c]), bf16_lo(wv[s][c]), acc, 0, 0, 0);
        acc = __builtin_amdgcn_mfma_f64_16x16x4f64(bf16_hi(xv[s][c]), bf16_hi(wv[s][c]), acc, 0, 0, 0);
      }
  }
  // D layout of the fp64 16x16x4 MFMA: register i of lane l holds column
  // l % 16 (expert) of row 4 i + l / 16 (token)
  if (wave > 0)
#pragma unroll
    for (int i = 0; i < 4; ++i) red[wave - 1][i][lane] = acc[i];
  __syncthreads();
  if (wave != 0) return;
  const int eo = blockIdx.y * 16 + row;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    double s = acc[i];
#pragma unroll
    for (int v = 0; v < WAVES - 1; ++v) s += red[v][i][lane];
    const int to = blockIdx.x * 16 + 4 * i + g;
    if (to < T && eo < E) logits[(size_t)to * E + eo] = (float)s;
  }
}

hipError_t launch_router(const uint16_t* x, const uint16_t* w, int T, int d, int E, float* logits,
                         hipStream_t stream) {
  timing_begin(stream, kSiteRouter);
  if (E >= 16 && T >= kRtMfmaMinT) {
    hipLaunchKernelGGL(router_mfma_kernel<4>, dim3((T + 15) / 16, (E + 15) / 16), dim3(256), 0, stream, x, w, T,
                       d, E, logits);
  } else {
    const int eb = (E + kRtExperts - 1) / kRtExperts;
    if (T <= 256) {
      hipLaunchKernelGGL(router_valu_kernel<1>, dim3(T, eb), dim3(kRtThreads), 0, stream, x, w, T, d, E, logits);
    } else {
      hipLaunchKernelGGL(router_valu_kernel<4>, dim3((T + 3) / 4, eb), dim3(kRtThreads), 0, stream, x, w, T, d, E,
                         logits);
    }
  }
  timing_end(stream, kSiteRouter);
  return hipGetLastError();
}

}  // namespace mc
