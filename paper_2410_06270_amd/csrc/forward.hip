// forward.hip -- routing-weighted combination and the forward launcher
// (gate/up and down kernels: fwd_kernels.hpp, one file per group size).
#include "forward_engine.hpp"

namespace mc {

// ---------------------------------------------------------------- combine --
// y[t][i..i+3] = bf16(res[t][i..i+3] + sum over kept ranks r, in rank order,
// of w_r * sum over splits s, in order, of partial[s][pos(t, r)][i..i+3]);
// res is the bf16 residual input (none when null).
template <int NSPLIT>
__device__ __forceinline__ f32x4 combine4(const float* __restrict__ partial, size_t part_stride,
                                          const int32_t* __restrict__ pair_pos, const float* __restrict__ topk_w,
                                          int k, int d, int P, const uint16_t* __restrict__ res, int t, int i) {
  f32x4 acc = {0.0f, 0.0f, 0.0f, 0.0f};
  if (res) {
    const uint2 rv = *reinterpret_cast<const uint2*>(res + (size_t)t * d + i);
    acc[0] = bf16_bits_to_float(rv.x & 0xffffu);
    acc[1] = bf16_bits_to_float(rv.x >> 16);
    acc[2] = bf16_bits_to_float(rv.y & 0xffffu);
    acc[3] = bf16_bits_to_float(rv.y >> 16);
  }
  for (int r = 0; r < k; ++r) {
    const int pos = pair_pos[(size_t)t * k + r];
    if (pos < 0 || pos >= P) continue;
    const float w = topk_w[(size_t)t * k + r];
    f32x4 v[NSPLIT];
#pragma unroll
    for (int s = 0; s < NSPLIT; ++s)
      v[s] = *reinterpret_cast<const f32x4*>(partial + s * part_stride + (size_t)pos * d + i);
    f32x4 sum = v[0];
#pragma unroll
    for (int s = 1; s < NSPLIT; ++s) sum += v[s];
#pragma unroll
    for (int c = 0; c < 4; ++c) acc[c] = fmaf(w, sum[c], acc[c]);
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
                                                      uint16_t* __restrict__ y) {
  const int t = blockIdx.y;
  const int i = 4 * (blockIdx.x * blockDim.x + threadIdx.x);
  if (i >= d) return;
  *reinterpret_cast<uint2*>(y + (size_t)t * d + i) =
      bf16x4(combine4<NSPLIT>(partial, part_stride, pair_pos, topk_w, k, d, P, res, t, i));
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
    uint16_t* __restrict__ y, double eps, uint16_t* __restrict__ xn) {
  __shared__ double part[kNormThreads / 64];
  const int t = blockIdx.x;
  const size_t base = (size_t)t * d;
  double ss = 0.0;
  for (int i = 4 * threadIdx.x; i < d; i += 4 * kNormThreads) {
    const uint2 v = bf16x4(combine4<NSPLIT>(partial, part_stride, pair_pos, topk_w, k, d, P, res, t, i));
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

// Split of the down projection's reduction so that small batches still give
// enough workgroups: about 1024 while the batch has fewer than 24 kept-pair
// slots, 512 beyond, where the fp32 partials (splits x T*k x d x 4 bytes,
// written here and read by the combine) cost more than the parallelism gains
// (8-expert layer: down 47.9 -> 45.1 us at T = 32, 2.6 to 3.7 us less from
// T = 12 to 64, 1.6 us more at T = 8).  Active experts are estimated as for
// the gate/up split.  The prefill GEMMs choose their own split.
int forward_nsplit(int T, int E, int k, int d, int ffn) {
  if (T > kDecodeMaxT) return prefill_layout(T, E, k, d, ffn).nsplit;
  const int tiles = (d + 255) / 256;
  int active = (T * k) < E ? (T * k) : E;
  if (E > 8) active = (active + 1) / 2;
  const int target = T * k >= 24 ? 512 : 1024;
  int s = (target + tiles * active - 1) / (tiles * active);
  const int maxs = (ffn / kTileCols) / 4;
  if (s > maxs) s = maxs;
  if (s > kMaxNsplit) s = kMaxNsplit;
  if (s < 1) s = 1;
  return s;
}

// Split of the gate/up reduction (over d) when the active experts give fewer
// than two workgroups per CU (batches of a few tokens); each split covers at
// least two 128-column chunks.  With many experts the estimate of the active
// ones is half of min(T*k, E): routers are skewed (on the OLMoE-shaped layer
// 16 tokens x top-8 touch about 23 of 64 experts), and sizing for all of them
// left the gate/up launch at under one workgroup per CU (measured there: gate/up
// 25.9 -> 17.7 us, step 53.0 -> 49.0 us at T = 16).
int forward_ksplit(int T, int E, int k, int d, int ffn) {
  if (T > 16) return 1;
  int active = (T * k) < E ? (T * k) : E;
  if (E > 8) active = (active + 1) / 2;
  const int wgs = (ffn / (16 * kWavesPerWg)) * active;
  int s = (512 + wgs - 1) / wgs;
  const int maxs = (d / kTileCols) / 2;
  if (s > maxs) s = maxs;
  if (s > kMaxKsplit) s = kMaxKsplit;
  if (s < 1) s = 1;
  return s;
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

size_t stack_workspace_bytes(int T, int E, int k, int d, int ffn) {
  return round256((size_t)T * d * sizeof(uint16_t)) + forward_workspace_bytes(T, E, k, d, ffn);
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
                       xn_next);                                                                   \
  else                                                                                             \
    hipLaunchKernelGGL(combine_kernel<S>, cgrid, dim3(256), 0, stream, partial, part_stride,       \
                       r.pair_pos, r.topk_w, r.k, d, r.T * r.k, res, y)
  switch (nsplit) {
    case 1: MC_COMBINE(1); break;
    case 2: MC_COMBINE(2); break;
    case 3: MC_COMBINE(3); break;
    case 4: MC_COMBINE(4); break;
    case 5: MC_COMBINE(5); break;
    case 6: MC_COMBINE(6); break;
    case 7: MC_COMBINE(7); break;
    default: MC_COMBINE(8); break;
  }
#undef MC_COMBINE
  timing_end(stream, kSiteCombine);
  return hipGetLastError();
}

hipError_t launch_forward(const uint16_t* x, const LayerArgs& L, const mc_routing& r, uint16_t* y,
                          void* ws, const uint16_t* residual, hipStream_t stream, const RouteArgs* route,
                          uint16_t* xn_next) {
  const int T = r.T, k = r.k;
  if (route) {
    const hipError_t err = launch_route(route->logits, route->important, route->delta32, route->tau, r, stream);
    if (err != hipSuccess) return err;
  }
  if (T > kDecodeMaxT) {
    float* partial = nullptr;
    size_t part_stride = 0;
    int nsplit = 1;
    const hipError_t err = launch_prefill(x, L, r, ws, &partial, &part_stride, &nsplit, stream);
    if (err != hipSuccess) return err;
    return launch_combine(partial, part_stride, nsplit, r, L.d, residual, y, xn_next, stream);
  }
  const size_t P = (size_t)T * k;
  Hidden hid;
  hid.P = (int)P;
  hid.T = T;
  hid.h = static_cast<uint16_t*>(ws);
  char* p = static_cast<char*>(ws) + round256(P * L.ffn * sizeof(uint16_t));
  hid.ksplit = forward_ksplit(T, r.E, k, L.d, L.ffn);
  hid.gu_part = reinterpret_cast<float*>(p);
  if (hid.ksplit > 1) p += round256((size_t)hid.ksplit * 2 * P * L.ffn * sizeof(float));
  float* partial = reinterpret_cast<float*>(p);
  const size_t part_stride = P * L.d;
  const int nsplit = forward_nsplit(T, r.E, k, L.d, L.ffn);
  // A workgroup holds at most min(T, 16*ntmax) of an expert's tokens; an
  // expert with more gets a workgroup per 32 of them (measured faster at 48
  // and 64 tokens than one workgroup of up to 64 at half the occupancy).
  const int ntmax = T <= 16 ? 1 : 2;
  const int xs_bytes = kXsBytes;
  hipError_t err;
  timing_begin(stream, kSiteGateUp);
  if (L.G == 128) err = launch_gateup<1>(x, L, r, hid, ntmax, xs_bytes, stream);
  else if (L.G == 64) err = launch_gateup<2>(x, L, r, hid, ntmax, xs_bytes, stream);
  else err = launch_gateup<4>(x, L, r, hid, ntmax, xs_bytes, stream);
  timing_end(stream, kSiteGateUp);
  if (err != hipSuccess) return err;
  timing_begin(stream, kSiteDown);
  if (L.G == 128) err = launch_down<1>(hid, L, r, nsplit, partial, part_stride, ntmax, xs_bytes, stream);
  else if (L.G == 64) err = launch_down<2>(hid, L, r, nsplit, partial, part_stride, ntmax, xs_bytes, stream);
  else err = launch_down<4>(hid, L, r, nsplit, partial, part_stride, ntmax, xs_bytes, stream);
  timing_end(stream, kSiteDown);
  if (err != hipSuccess) return err;
  return launch_combine(partial, part_stride, nsplit, r, L.d, residual, y, xn_next, stream);
}

}  // namespace mc
