// router.hip -- the router's linear layer ahead of routing (Eq. 1: the gate
// scores G(x) are the top-k of x W_r^T).
//
//   logits[t][e] = sum_k x[t][k] * w[e][k],   x [T][d], w [E][d] bf16.
//
// Every product of two bf16 values is exact in fp64 (8-bit significands, and
// the fp64 exponent range holds every product); the d products are summed in
// fp64 and the sum is rounded once to fp32.  The result is faithful: it lies
// between the fp32 roundings of S - g and S + g, S the exact sum and
// g = (d - 1) 2^-53 sum |x_k w_k| the fp64 summation bound, so it is the
// correctly rounded value unless S lies within g of an fp32 rounding boundary.
//
// One workgroup of 256 threads computes NT tokens x 8 experts: each thread
// takes 16-byte pieces (8 bf16) of the d axis, strided by 256 pieces, keeps
// NT * 8 fp64 accumulators, and the partial sums are reduced through LDS in a
// fixed order (deterministic).  Memory-bound on x for the top-2-of-8 router
// (HBM reads x once; w, 8 x d bf16, stays in L2); for 64 experts the fp64
// multiply-adds set the time.
#include "mc_internal.hpp"

namespace mc {

constexpr int kRtThreads = 256;
constexpr int kRtExperts = 8;

__device__ __forceinline__ double bf16_lo(uint32_t w) { return (double)__uint_as_float(w << 16); }
__device__ __forceinline__ double bf16_hi(uint32_t w) { return (double)__uint_as_float(w & 0xffff0000u); }

template <int NT>
__global__ void __launch_bounds__(kRtThreads) router_kernel(const uint16_t* __restrict__ x,
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

hipError_t launch_router(const uint16_t* x, const uint16_t* w, int T, int d, int E, float* logits,
                         hipStream_t stream) {
  const int eb = (E + kRtExperts - 1) / kRtExperts;
  timing_begin(stream, kSiteRouter);
  if (T <= 256) {
    hipLaunchKernelGGL(router_kernel<1>, dim3(T, eb), dim3(kRtThreads), 0, stream, x, w, T, d, E, logits);
  } else {
    hipLaunchKernelGGL(router_kernel<4>, dim3((T + 3) / 4, eb), dim3(kRtThreads), 0, stream, x, w, T, d, E,
                       logits);
  }
  timing_end(stream, kSiteRouter);
  return hipGetLastError();
}

}  // namespace mc
