// forward.hip -- routing-weighted combination and the forward launcher
// (decode GEMVs: decode.hpp, prefill GEMMs: prefill.hpp, one file per group
// size each).
#include "decode.hpp"

namespace mc {

// ---------------------------------------------------------------- combine --
// y[t][i..i+3] = bf16(res[t][i..i+3] + sum over kept ranks r, in rank order,
// of w_r * sum over splits s, in order, of partial[s][pos(t, r)][i..i+3]);
// res is the bf16 residual input (none when null).  NSPLIT = 0: the number
// of splits is the run-time `nsplit` (more than 8).
template <int NSPLIT>
__device__ __forceinline__ f32x4 combine4(const float* __restrict__ partial, size_t part_stride,
                                          const int32_t* __restrict__ pair_pos, const float* __restrict__ topk_w,
                                          int k, int d, int P, const uint16_t* __restrict__ res, int t, int i,
                                          int nsplit = NSPLIT) {
  f32x4 acc = {0.0f, 0.0f, 0.0f, 0.0f};
  if (res) {
    const uint2 rv = *reinterpret_cast<const uint2*>(res + (size_t)t * d + i);
    acc[0] = bf16_bits_to_float(rv.x & 0xffffu);
    acc[1] = bf16_bits_to_float(rv.x >> 16);
    acc[2] = bf16_bits_to_float(rv.y & 0xffffu);
    acc[3] = bf16_bits_to_float(rv.y >> 16);
  }
  // every rank's list position and weight are loaded first, then the rows
  // of RB ranks at a time (absent ranks read row 0, in bounds, and are
  // dropped), so that the rows' loads do not wait on one another; the sums
  // still run in rank order
  int pos[MC_MAX_TOPK];
  float wr[MC_MAX_TOPK];
#pragma unroll
  for (int r = 0; r < MC_MAX_TOPK; ++r) {
    pos[r] = r < k ? checked_pos(pair_pos[(size_t)t * k + r], P) : -1;
    wr[r] = r < k ? topk_w[(size_t)t * k + r] : 0.0f;
  }
  if constexpr (NSPLIT == 0) {
#pragma unroll
    for (int r = 0; r < MC_MAX_TOPK; ++r) {
      if (pos[r] < 0) continue;
      const float* row = partial + (size_t)pos[r] * d + i;
      f32x4 sum = *reinterpret_cast<const f32x4*>(row);
      for (int s = 1; s < nsplit; ++s) sum += *reinterpret_cast<const f32x4*>(row + s * part_stride);
#pragma unroll
      for (int c = 0; c < 4; ++c) acc[c] = fmaf(wr[r], sum[c], acc[c]);
    }
  } else {
    constexpr int RB = NSPLIT <= 4 ? 4 : 2;   // ranks in flight (RB * NSPLIT rows of 16 bytes)
#pragma unroll
    for (int r0 = 0; r0 < MC_MAX_TOPK; r0 += RB) {
      if (r0 >= k) break;
      f32x4 v[RB][NSPLIT];
#pragma unroll
      for (int j = 0; j < RB; ++j) {
        const float* row = partial + (size_t)(pos[r0 + j] >= 0 ? pos[r0 + j] : 0) * d + i;
#pragma unroll
        for (int s = 0; s < NSPLIT; ++s) v[j][s] = *reinterpret_cast<const f32x4*>(row + s * part_stride);
      }
#pragma unroll
      for (int j = 0; j < RB; ++j) {
        if (pos[r0 + j] < 0) continue;
        f32x4 sum = v[j][0];
#pragma unroll
        for (int s = 1; s < NSPLIT; ++s) sum += v[j][s];
#pragma unroll
        for (int c = 0; c < 4; ++c) acc[c] = fmaf(wr[r0 + j], sum[c], acc[c]);
      }
    }
  }
  return acc;
}

__device__ __forceinline__ uint2 bf16x4(const f32x4& a) {
  return make_uint2((uint32_t)float_to_bf16(a[0]) | ((uint32_t)float_to_bf16(a[1]) << 16),
                    (uint32_t)float_to_bf16(a[2]) | ((uint32_t)float_to_bf16(a[3]) << 16));
}

template <int NSPLIT>
__global__ void __launch_bounds__(256) combine_kernel(const float* __restrict__ partial,
                                                      size_t part_stride,
                                                      const int32_t* __restrict__ pair_pos,
                                                      const float* __restrict__ topk_w, int k, int d,
                                                      int P, const uint16_t* __restrict__ res,
                                                      uint16_t* __restrict__ y, int nsplit) {
  const int t = blockIdx.y;
  const int i = 4 * (blockIdx.x * blockDim.x + threadIdx.x);
  if (i >= d) return;
  *reinterpret_cast<uint2*>(y + (size_t)t * d + i) =
      bf16x4(combine4<NSPLIT>(partial, part_stride, pair_pos, topk_w, k, d, P, res, t, i, nsplit));
}

// ---------------------------------------------------------------- rmsnorm --
// xn[t][i] = bf16(h[t][i] / sqrt(mean_j h[t][j]^2 + eps)): the sum of squares
// in fp64 in a fixed order (lane partials, wave butterfly, waves in order),
// the quotient in fp64, rounded once.  One workgroup per token.
constexpr int kNormThreads = 1024;

__global__ void __launch_bounds__(kNormThreads) rmsnorm_kernel(const uint16_t* __restrict__ h, int d,
                                                               double eps, uint16_t* __restrict__ xn) {
  __shared__ double part[kNormThreads / 64];
  const size_t base = (size_t)blockIdx.x * d;
  double ss = 0.0;
  for (int i = 4 * threadIdx.x; i < d; i += 4 * kNormThreads) {
    const uint2 v = *reinterpret_cast<const uint2*>(h + base + i);
    const double a = bf16_bits_to_float(v.x & 0xffffu), b = bf16_bits_to_float(v.x >> 16);
    const double c = bf16_bits_to_float(v.y & 0xffffu), e = bf16_bits_to_float(v.y >> 16);
    ss += a * a;
    ss += b * b;
    ss += c * c;
    ss += e * e;
  }
  for (int off = 1; off < 64; off <<= 1) ss += __shfl_xor(ss, off);
  if ((threadIdx.x & 63) == 0) part[threadIdx.x >> 6] = ss;
  __syncthreads();
  double tot = 0.0;
  for (int w = 0; w < kNormThreads / 64; ++w) tot += part[w];
  const double r = 1.0 / sqrt(tot / d + eps);
  for (int i = 4 * threadIdx.x; i < d; i += 4 * kNormThreads) {
    const uint2 v = *reinterpret_cast<const uint2*>(h + base + i);
    const uint32_t lo = (uint32_t)double_to_bf16_rne(bf16_bits_to_float(v.x & 0xffffu) * r) |
                        ((uint32_t)double_to_bf16_rne(bf16_bits_to_float(v.x >> 16) * r) << 16);
    const uint32_t hi = (uint32_t)double_to_bf16_rne(bf16_bits_to_float(v.y & 0xffffu) * r) |
                        ((uint32_t)double_to_bf16_rne(bf16_bits_to_float(v.y >> 16) * r) << 16);
    *reinterpret_cast<uint2*>(xn + base + i) = make_uint2(lo, hi);
  }
}

// The combine of a stack layer that also forms the next layer's input: one
// workgroup per token writes y[t] as combine_kernel does and xn[t] =
// RMSNorm(y[t]) as rmsnorm_kernel would from y -- each thread takes the same
// columns in the same order as there, so the sum of squares, its reduction
// and every rounding are those of the two separate launches.
template <int NSPLIT>
__global__ void __launch_bounds__(kNormThreads) combine_norm_kernel(
    const float* __restrict__ partial, size_t part_stride, const int32_t* __restrict__ pair_pos,
    const float* __restrict__ topk_w, int k, int d, int P, const uint16_t* __restrict__ res,
    uint16_t* __restrict__ y, double eps, uint16_t* __restrict__ xn, int nsplit) {
  __shared__ double part[kNormThreads / 64];
  const int t = blockIdx.x;
  const size_t base = (size_t)t * d;
  double ss = 0.0;
  for (int i = 4 * threadIdx.x; i < d; i += 4 * kNormThreads) {
    const uint2 v = bf16x4(combine4<NSPLIT>(partial, part_stride, pair_pos, topk_w, k, d, P, res, t, i, nsplit));
    *reinterpret_cast<uint2*>(y + base + i) = v;
    const double a = bf16_bits_to_float(v.x & 0xffffu), b = bf16_bits_to_float(v.x >> 16);
    const double c = bf16_bits_to_float(v.y & 0xffffu), e = bf16_bits_to_float(v.y >> 16);
    ss += a * a;
    ss += b * b;
    ss += c * c;
    ss += e * e;
  }
  for (int off = 1; off < 64; off <<= 1) ss += __shfl_xor(ss, off);
  if ((threadIdx.x & 63) == 0) part[threadIdx.x >> 6] = ss;
  __syncthreads();
  double tot = 0.0;
  for (int w = 0; w < kNormThreads / 64; ++w) tot += part[w];
  const double r = 1.0 / sqrt(tot / d + eps);
  for (int i = 4 * threadIdx.x; i < d; i += 4 * kNormThreads) {
    const uint2 v = *reinterpret_cast<const uint2*>(y + base + i);   // this thread's own stores
    const uint32_t lo = (uint32_t)double_to_bf16_rne(bf16_bits_to_float(v.x & 0xffffu) * r) |
                        ((uint32_t)double_to_bf16_rne(bf16_bits_to_float(v.x >> 16) * r) << 16);
    const uint32_t hi = (uint32_t)double_to_bf16_rne(bf16_bits_to_float(v.y & 0xffffu) * r) |
                        ((uint32_t)double_to_bf16_rne(bf16_bits_to_float(v.y >> 16) * r) << 16);
    *reinterpret_cast<uint2*>(xn + base + i) = make_uint2(lo, hi);
  }
}

hipError_t launch_rmsnorm(const uint16_t* h, int T, int d, double eps, uint16_t* xn, hipStream_t stream) {
  timing_begin(stream, kSiteRmsNorm);
  hipLaunchKernelGGL(rmsnorm_kernel, dim3(T), dim3(kNormThreads), 0, stream, h, d, eps, xn);
  timing_end(stream, kSiteRmsNorm);
  return hipGetLastError();
}


// --------------------------------------------------------------- launchers --

// Splits of the decode GEMVs' reductions: as few as let one item's
// activations (16 rows of 128-column chunks) fit the LDS slab -- one for the
// gate/up reduction over d up to 4352, four for Mixtral's ffn = 14336 (28
// chunks each).  The slab capacity does not depend on the group size.
static_assert(decode_slab_chunks(1) == decode_slab_chunks(4), "slab capacity independent of G");
static int decode_splits(int K, int* c_per) {
  const int nt = K / kTileCols, cap = decode_slab_chunks(1);
  const int S = (nt + cap - 1) / cap;
  if (c_per) *c_per = (nt + S - 1) / S;
  return S;
}

// Splits of the down reduction: the decode GEMV's, or the prefill GEMM's.
int forward_nsplit(int T, int E, int k, int d, int ffn) {
  if (T > kDecodeMaxT) return prefill_layout(T, E, k, d, ffn).nsplit;
  return decode_splits(ffn, nullptr);
}

// Splits of the decode gate/up reduction over d (1 up to d = 4352).
int forward_ksplit(int T, int E, int k, int d, int ffn) {
  (void)T; (void)E; (void)k; (void)ffn;
  return decode_splits(d, nullptr);
}

// Compute units of the current device (one decode workgroup each).
static int device_cus() {
  static int cached[64] = {0};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) dev = 0;
  if (cached[dev] == 0) {
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0) n = 256;
    cached[dev] = n;
  }
  return cached[dev];
}

// Workspace: h (fp16) | gate/up partials (when split) | down partials, each
// part rounded up to 256 bytes.
static size_t round256(size_t b) { return ((b + 255) / 256) * 256; }

size_t forward_workspace_bytes(int T, int E, int k, int d, int ffn) {
  if (T > kDecodeMaxT) return prefill_layout(T, E, k, d, ffn).total;
  const size_t P = (size_t)T * k;
  const int ks = forward_ksplit(T, E, k, d, ffn);
  const size_t h = round256(P * ffn * sizeof(uint16_t));
  const size_t gu = ks > 1 ? round256((size_t)ks * 2 * P * ffn * sizeof(float)) : 0;
  const size_t part = (size_t)forward_nsplit(T, E, k, d, ffn) * P * d * sizeof(float);
  return h + gu + part;
}

size_t routing_set_bytes(int T, int E, int k) {
  const size_t P = (size_t)T * k;
  return 6 * round256(P * 4) + round256(P) + round256((size_t)E * 4) + round256(((size_t)E + 1) * 4) + 256;
}

mc_routing routing_set(void* base, int T, int E, int k) {
  const size_t P = (size_t)T * k;
  char* p = static_cast<char*>(base);
  auto take = [&](size_t bytes) {
    void* q = p;
    p += round256(bytes);
    return q;
  };
  mc_routing r;
  r.T = T;
  r.E = E;
  r.k = k;
  r.topk_idx = static_cast<int32_t*>(take(P * 4));
  r.topk_w = static_cast<float*>(take(P * 4));
  r.kept = static_cast<uint8_t*>(take(P));
  r.counts = static_cast<int32_t*>(take((size_t)E * 4));
  r.offsets = static_cast<int32_t*>(take(((size_t)E + 1) * 4));
  r.pair_token = static_cast<int32_t*>(take(P * 4));
  r.pair_rank = static_cast<int32_t*>(take(P * 4));
  r.pair_w = static_cast<float*>(take(P * 4));
  r.pair_pos = static_cast<int32_t*>(take(P * 4));
  r.n_pruned = static_cast<int32_t*>(take(4));
  return r;
}

size_t stack_workspace_bytes(int T, int E, int k, int d, int ffn) {
  const size_t routes = route_batch_fits(T, E) ? (size_t)kRouteBatch * routing_set_bytes(T, E, k) : 0;
  return round256((size_t)T * d * sizeof(uint16_t)) + routes + forward_workspace_bytes(T, E, k, d, ffn);
}

static hipError_t launch_combine(const float* partial, size_t part_stride, int nsplit,
                                 const mc_routing& r, int d, const uint16_t* res, uint16_t* y,
                                 uint16_t* xn_next, hipStream_t stream) {
  timing_begin(stream, kSiteCombine);
  const dim3 cgrid((d / 4 + 255) / 256, r.T);
#define MC_COMBINE(S)                                                                              \
  if (xn_next)                                                                                     \
    hipLaunchKernelGGL(combine_norm_kernel<S>, dim3(r.T), dim3(kNormThreads), 0, stream, partial,  \
                       part_stride, r.pair_pos, r.topk_w, r.k, d, r.T * r.k, res, y, kRmsNormEps,   \
                       xn_next, nsplit);                                                           \
  else                                                                                             \
    hipLaunchKernelGGL(combine_kernel<S>, cgrid, dim3(256), 0, stream, partial, part_stride,       \
                       r.pair_pos, r.topk_w, r.k, d, r.T * r.k, res, y, nsplit)
  switch (nsplit) {
    case 1: MC_COMBINE(1); break;
    case 2: MC_COMBINE(2); break;
    case 3: MC_COMBINE(3); break;
    case 4: MC_COMBINE(4); break;
    case 5: MC_COMBINE(5); break;
    case 6: MC_COMBINE(6); break;
    case 7: MC_COMBINE(7); break;
    case 8: MC_COMBINE(8); break;
    default: MC_COMBINE(0); break;
  }
#undef MC_COMBINE
  timing_end(stream, kSiteCombine);
  return hipGetLastError();
}

hipError_t launch_expert_partials(const uint16_t* x, const LayerArgs& L, const mc_routing& r, void* ws,
                                  float** partial_out, size_t* part_stride_out, int* nsplit_out,
                                  hipStream_t stream) {
  const int T = r.T, k = r.k;
  if (T > kDecodeMaxT) return launch_prefill(x, L, r, ws, partial_out, part_stride_out, nsplit_out, stream);
  const size_t P = (size_t)T * k;
  DecodeArgs a;
  a.x = x;
  a.counts = r.counts;
  a.offsets = r.offsets;
  a.pair_token = r.pair_token;
  a.T = T;
  a.P = (int)P;
  a.nwg = device_cus();
  int c_gu = 0, c_dn = 0;
  const int s_gu = decode_splits(L.d, &c_gu);
  const int nsplit = decode_splits(L.ffn, &c_dn);
  uint16_t* h = static_cast<uint16_t*>(ws);
  char* p = static_cast<char*>(ws) + round256(P * L.ffn * sizeof(uint16_t));
  float* gu_part = reinterpret_cast<float*>(p);
  if (s_gu > 1) p += round256((size_t)s_gu * 2 * P * L.ffn * sizeof(float));
  float* partial = reinterpret_cast<float*>(p);
  const size_t part_stride = P * L.d;
  *partial_out = partial;
  *part_stride_out = part_stride;
  *nsplit_out = nsplit;

  a.h = nullptr;
  a.gu_in = nullptr;
  a.h_out = h;
  a.gu_out = gu_part;
  a.partial = nullptr;
  a.part_stride = 0;
  a.S = s_gu;
  a.c_per = c_gu;
  a.gu_split = 1;
  hipError_t err;
  timing_begin(stream, kSiteGateUp);
  if (L.G == 128) err = launch_decode<1, true>(L, a, stream);
  else if (L.G == 64) err = launch_decode<2, true>(L, a, stream);
  else err = launch_decode<4, true>(L, a, stream);
  timing_end(stream, kSiteGateUp);
  if (err != hipSuccess) return err;

  a.h = h;
  a.gu_in = gu_part;
  a.h_out = nullptr;
  a.gu_out = nullptr;
  a.partial = partial;
  a.part_stride = part_stride;
  a.S = nsplit;
  a.c_per = c_dn;
  a.gu_split = s_gu;
  timing_begin(stream, kSiteDown);
  if (L.G == 128) err = launch_decode<1, false>(L, a, stream);
  else if (L.G == 64) err = launch_decode<2, false>(L, a, stream);
  else err = launch_decode<4, false>(L, a, stream);
  timing_end(stream, kSiteDown);
  return err;
}

hipError_t launch_forward(const uint16_t* x, const LayerArgs& L, const mc_routing& r, uint16_t* y,
                          void* ws, const uint16_t* residual, hipStream_t stream, const RouteArgs* route,
                          uint16_t* xn_next) {
  if (route) {
    const hipError_t err = launch_route(route->logits, route->important, route->delta32, route->tau, r, stream);
    if (err != hipSuccess) return err;
  }
  float* partial = nullptr;
  size_t part_stride = 0;
  int nsplit = 1;
  const hipError_t err = launch_expert_partials(x, L, r, ws, &partial, &part_stride, &nsplit, stream);
  if (err != hipSuccess) return err;
  return launch_combine(partial, part_stride, nsplit, r, L.d, residual, y, xn_next, stream);
}

}  // namespace mc
