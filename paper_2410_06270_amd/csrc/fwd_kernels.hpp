// fwd_kernels.hpp -- the gate/up and down kernels of the expert forward and
// their launchers, templated on groups per 128-column chunk (GPC = 128/G) and
// on the largest number of 16-token blocks a launch can see (NTMAX).  Each
// gateup_g*.hip / down_g*.hip translation unit instantiates one GPC.
#pragma once

#include "forward_engine.hpp"

namespace mc {

// Per-width dispatch: the expert's width is uniform in a workgroup.
template <int GPC, int PLANES, int NTMAX, typename RowFn>
__device__ __forceinline__ void run_expert(int bits, const Streams& sp, int c_begin, int c_end,
                                           RowFn rowsrc, size_t plane_stride, int nt, int G,
                                           uint16_t* xs, float* sxs, int xs_elems,
                                           f32x4 (&tot)[2][NTMAX]) {
  if (bits == 1)
    run_width<1, GPC, PLANES, NTMAX>(sp, c_begin, c_end, rowsrc, plane_stride, nt, G, xs, sxs, xs_elems, tot);
  else if (bits == 2)
    run_width<2, GPC, PLANES, NTMAX>(sp, c_begin, c_end, rowsrc, plane_stride, nt, G, xs, sxs, xs_elems, tot);
  else
    run_width<3, GPC, PLANES, NTMAX>(sp, c_begin, c_end, rowsrc, plane_stride, nt, G, xs, sxs, xs_elems, tot);
}

// Buffer resources of one stream: row block rb of matrix m of expert e,
// chunks [c_begin, c_end) (words) and their groups (scale/zero).
__device__ __forceinline__ void stream_rsrc(const LayerArgs& L, int e, int m, int rb, int K,
                                            int c_begin, int c_end, rsrc_t& w, rsrc_t& s) {
  const int b = L.cum_bits[e + 1] - L.cum_bits[e];
  const int ntiles = K / kTileCols, ng = K / L.G, gpc = kTileCols / L.G;
  const uint32_t* wbase = L.words + layer_word_offset(L, e, m) +
                          ((size_t)rb * ntiles + c_begin) * 64 * b;
  const uint32_t* sbase = L.sz + layer_sz_offset(L, e, m) + ((size_t)rb * ng + (size_t)c_begin * gpc) * 16;
  w = make_rsrc(wbase, (uint32_t)(c_end - c_begin) * 64u * b * 4u);
  s = make_rsrc(sbase, (uint32_t)(c_end - c_begin) * gpc * 64u);
}

// ---------------------------------------------------------------- gate/up --
// Workgroup: expert e, 64 rows (4 waves x 16) of gate and up, up to
// 16*NTMAX of the expert's tokens.  Writes h = silu(gate x) * (up x)
// as bf16 hi/lo planes.
// Up to 32 tokens per workgroup the kernels are held to 128 registers so that
// four workgroups (16 waves) share a CU.
template <int GPC, int NTMAX>
__global__ void __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(NTMAX <= 2 ? 4 : 2)))
gateup_kernel(const uint16_t* __restrict__ x, LayerArgs L,
                                                     const int32_t* __restrict__ counts,
                                                     const int32_t* __restrict__ offsets,
                                                     const int32_t* __restrict__ pair_token,
                                                     uint16_t* __restrict__ h_hi,
                                                     uint16_t* __restrict__ h_lo, int xs_bytes) {
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
  __shared__ int toks[16 * NTMAX];
  uint16_t* xs = reinterpret_cast<uint16_t*>(smem);
  float* sxs = reinterpret_cast<float*>(smem + xs_bytes);
  const int e = blockIdx.y;
  const int t0 = blockIdx.z * 16 * NTMAX;
  const int ce = counts[e];
  if (t0 >= ce) return;
  const int nt = (ce - t0) < 16 * NTMAX ? (ce - t0) : 16 * NTMAX;
  const int pbase = offsets[e] + t0;
  for (int i = threadIdx.x; i < nt; i += blockDim.x) toks[i] = pair_token[pbase + i];
  const int lane = threadIdx.x & 63, wave = wave_id();
  const int K = L.d, G = L.G, ntiles = K / kTileCols;
  const int b = L.cum_bits[e + 1] - L.cum_bits[e];
  const int rb = blockIdx.x * 4 + wave;
  Streams sp;
  for (int m = 0; m < 2; ++m) stream_rsrc(L, e, m, rb, K, 0, ntiles, sp.w[m], sp.s[m]);
  sp.lane_w = (uint32_t)lane * b * 4u;
  sp.lane_s = (uint32_t)(lane & 15) * 4u;
  f32x4 tot[2][NTMAX];
#pragma unroll
  for (int st = 0; st < 2; ++st)
#pragma unroll
    for (int tb = 0; tb < NTMAX; ++tb)
#pragma unroll
      for (int i = 0; i < 4; ++i) tot[st][tb][i] = 0.0f;
  auto rowsrc = [&](int m) { return x + (size_t)toks[m] * K; };
  run_expert<GPC, 1, NTMAX>(b, sp, 0, ntiles, rowsrc, 0, nt, G, xs, sxs, xs_bytes / 2, tot);
  const int n = rb * 16 + (lane & 15);
#pragma unroll
  for (int tb = 0; tb < NTMAX; ++tb) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int m = tb * 16 + 4 * (lane >> 4) + i;
      if (m < nt) {
        const float h = silu(tot[0][tb][i]) * tot[1][tb][i];
        const uint16_t hi = float_to_bf16(h);
        const uint16_t lo = float_to_bf16(h - bf16_bits_to_float(hi));
        const size_t o = (size_t)(pbase + m) * L.ffn + n;
        h_hi[o] = hi;
        h_lo[o] = lo;
      }
    }
  }
}

// ------------------------------------------------------------------- down --
// Workgroup: expert e, 128 output rows (4 waves x 2 row blocks), one split of
// the ffn reduction, up to 16*NTMAX of the expert's pairs -> fp32 partials.
template <int GPC, int NTMAX>
__global__ void __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(NTMAX <= 2 ? 4 : 2)))
down_kernel(const uint16_t* __restrict__ h_hi,
                                                   size_t plane_stride, LayerArgs L,
                                                   const int32_t* __restrict__ counts,
                                                   const int32_t* __restrict__ offsets, int nsplit,
                                                   float* __restrict__ partial, size_t part_stride,
                                                   int xs_bytes) {
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
  uint16_t* xs = reinterpret_cast<uint16_t*>(smem);
  float* sxs = reinterpret_cast<float*>(smem + xs_bytes);
  const int e = blockIdx.y;
  const int chunk = blockIdx.z / nsplit, split = blockIdx.z - chunk * nsplit;
  const int t0 = chunk * 16 * NTMAX;
  const int ce = counts[e];
  if (t0 >= ce) return;
  const int nt = (ce - t0) < 16 * NTMAX ? (ce - t0) : 16 * NTMAX;
  const int pbase = offsets[e] + t0;
  const int lane = threadIdx.x & 63, wave = wave_id();
  const int K = L.ffn, G = L.G, ntiles = K / kTileCols;
  const int b = L.cum_bits[e + 1] - L.cum_bits[e];
  const int per = (ntiles + nsplit - 1) / nsplit;
  const int c_begin = split * per;
  const int c_end = (c_begin + per) < ntiles ? (c_begin + per) : ntiles;
  const int rb0 = blockIdx.x * 8 + wave * 2;
  f32x4 tot[2][NTMAX];
#pragma unroll
  for (int st = 0; st < 2; ++st)
#pragma unroll
    for (int tb = 0; tb < NTMAX; ++tb)
#pragma unroll
      for (int i = 0; i < 4; ++i) tot[st][tb][i] = 0.0f;
  if (c_begin < c_end) {
    Streams sp;
    for (int j = 0; j < 2; ++j) stream_rsrc(L, e, 2, rb0 + j, K, c_begin, c_end, sp.w[j], sp.s[j]);
    sp.lane_w = (uint32_t)lane * b * 4u;
    sp.lane_s = (uint32_t)(lane & 15) * 4u;
    auto rowsrc = [&](int m) { return h_hi + (size_t)(pbase + m) * K; };
    run_expert<GPC, 2, NTMAX>(b, sp, c_begin, c_end, rowsrc, plane_stride, nt, G, xs, sxs,
                              xs_bytes / 2, tot);
  }
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    const int n = (rb0 + j) * 16 + (lane & 15);
#pragma unroll
    for (int tb = 0; tb < NTMAX; ++tb) {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int m = tb * 16 + 4 * (lane >> 4) + i;
        if (m < nt)
          partial[(size_t)split * part_stride + (size_t)(pbase + m) * L.d + n] = tot[j][tb][i];
      }
    }
  }
}

// --------------------------------------------------------------- launchers --

template <typename K>
static hipError_t allow_lds(K kernel, int bytes) {
  return hipFuncSetAttribute(reinterpret_cast<const void*>(kernel),
                             hipFuncAttributeMaxDynamicSharedMemorySize, bytes);
}

template <int GPC, int NTMAX>
static hipError_t launch_gateup_nt(const uint16_t* x, const LayerArgs& L, const mc_routing& r,
                                   uint16_t* h_hi, uint16_t* h_lo, int xs_bytes,
                                   hipStream_t stream) {
  static bool attr = false;
  if (!attr) {
    hipError_t e = allow_lds(&gateup_kernel<GPC, NTMAX>, kXsBytesLarge + kSxBytes);
    if (e != hipSuccess) return e;
    attr = true;
  }
  const int chunks = (r.T + 16 * NTMAX - 1) / (16 * NTMAX);
  hipLaunchKernelGGL((gateup_kernel<GPC, NTMAX>), dim3(L.ffn / 64, L.E, chunks), dim3(256),
                     xs_bytes + kSxBytes, stream, x, L, r.counts, r.offsets, r.pair_token, h_hi,
                     h_lo, xs_bytes);
  return hipGetLastError();
}

template <int GPC, int NTMAX>
static hipError_t launch_down_nt(const uint16_t* h_hi, size_t plane_stride, const LayerArgs& L,
                                 const mc_routing& r, int nsplit, float* partial,
                                 size_t part_stride, int xs_bytes, hipStream_t stream) {
  static bool attr = false;
  if (!attr) {
    hipError_t e = allow_lds(&down_kernel<GPC, NTMAX>, kXsBytesLarge + kSxBytes);
    if (e != hipSuccess) return e;
    attr = true;
  }
  const int chunks = (r.T + 16 * NTMAX - 1) / (16 * NTMAX);
  hipLaunchKernelGGL((down_kernel<GPC, NTMAX>), dim3(L.d / 128, L.E, chunks * nsplit), dim3(256),
                     xs_bytes + kSxBytes, stream, h_hi, plane_stride, L, r.counts, r.offsets,
                     nsplit, partial, part_stride, xs_bytes);
  return hipGetLastError();
}

template <int GPC>
hipError_t launch_gateup(const uint16_t* x, const LayerArgs& L, const mc_routing& r,
                         uint16_t* h_hi, uint16_t* h_lo, int ntmax, int xs_bytes,
                         hipStream_t stream) {
  if (ntmax == 1) return launch_gateup_nt<GPC, 1>(x, L, r, h_hi, h_lo, xs_bytes, stream);
  if (ntmax == 2) return launch_gateup_nt<GPC, 2>(x, L, r, h_hi, h_lo, xs_bytes, stream);
  return launch_gateup_nt<GPC, 4>(x, L, r, h_hi, h_lo, xs_bytes, stream);
}

template <int GPC>
hipError_t launch_down(const uint16_t* h_hi, size_t plane_stride, const LayerArgs& L,
                       const mc_routing& r, int nsplit, float* partial, size_t part_stride,
                       int ntmax, int xs_bytes, hipStream_t stream) {
  if (ntmax == 1)
    return launch_down_nt<GPC, 1>(h_hi, plane_stride, L, r, nsplit, partial, part_stride, xs_bytes, stream);
  if (ntmax == 2)
    return launch_down_nt<GPC, 2>(h_hi, plane_stride, L, r, nsplit, partial, part_stride, xs_bytes, stream);
  return launch_down_nt<GPC, 4>(h_hi, plane_stride, L, r, nsplit, partial, part_stride, xs_bytes, stream);
}

}  // namespace mc
