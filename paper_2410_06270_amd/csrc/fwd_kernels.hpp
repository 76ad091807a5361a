// fwd_kernels.hpp -- the gate/up and down kernels of the expert forward and
// their launchers, templated on groups per 128-column chunk (GPC = 128/G) and
// on the largest number of 16-token blocks a launch can see (NTMAX).  Each
// gateup_g*.hip / down_g*.hip translation unit instantiates one GPC.
#pragma once

#include "forward_engine.hpp"

namespace mc {

// Per-width dispatch: the expert's width is uniform in a workgroup.
template <int GPC, int NTMAX, bool F16, typename StageFn>
__device__ __forceinline__ void run_expert(int bits, const Streams& sp, int c_begin, int c_end,
                                           StageFn stage, int nt, int G, uint16_t* xs, float* sxs,
                                           int xs_elems, f32x4 (&tot)[2][NTMAX]) {
  if (bits == 1)
    run_width<1, GPC, NTMAX, F16>(sp, c_begin, c_end, stage, nt, G, xs, sxs, xs_elems, tot);
  else if (bits == 2)
    run_width<2, GPC, NTMAX, F16>(sp, c_begin, c_end, stage, nt, G, xs, sxs, xs_elems, tot);
  else
    run_width<3, GPC, NTMAX, F16>(sp, c_begin, c_end, stage, nt, G, xs, sxs, xs_elems, tot);
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

__device__ __forceinline__ void zero_tot(f32x4* t, int n) {
  for (int i = 0; i < n; ++i) t[i] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
}

// ---------------------------------------------------------------- gate/up --
// Workgroup: expert e, 16*WAVES rows (one 16-row block per wave) of gate
// and up, up to 16*NTMAX of the expert's tokens, one of ksplit ranges of the
// d reduction.  ksplit == 1 writes h = fp16(silu(gate x) * (up x));
// ksplit > 1 writes the fp32 partial sums of gate and up, which the down
// kernel adds up (in split order) before the SiLU.
// The kernels are held to 128 registers so that two workgroups (16 waves)
// share a CU.
template <int GPC, int NTMAX, int WAVES>
__global__ void __launch_bounds__(64 * WAVES)
__attribute__((amdgpu_waves_per_eu(4))) gateup_kernel(
    const uint16_t* __restrict__ x, LayerArgs L, const int32_t* __restrict__ counts,
    const int32_t* __restrict__ offsets, const int32_t* __restrict__ pair_token, Hidden hid,
    int xs_bytes) {
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
  __shared__ int toks[16 * NTMAX];
  uint16_t* xs = reinterpret_cast<uint16_t*>(smem);
  float* sxs = reinterpret_cast<float*>(smem + xs_bytes);
  const int e = blockIdx.y;
  const int chunk = blockIdx.z / hid.ksplit, split = blockIdx.z - chunk * hid.ksplit;
  const int t0 = chunk * 16 * NTMAX;
  int ebase, ce;
  expert_range(counts, offsets, e, hid.P, ebase, ce);
  if (t0 >= ce) return;
  const int nt = (ce - t0) < 16 * NTMAX ? (ce - t0) : 16 * NTMAX;
  const int pbase = ebase + t0;
  for (int i = threadIdx.x; i < nt; i += blockDim.x) toks[i] = clamp_token(pair_token[pbase + i], hid.T);
  const int lane = threadIdx.x & 63, wave = wave_id();
  const int K = L.d, G = L.G, ntiles = K / kTileCols;
  const int per = (ntiles + hid.ksplit - 1) / hid.ksplit;
  const int c_begin = split * per;
  const int c_end = (c_begin + per) < ntiles ? (c_begin + per) : ntiles;
  const int b = L.cum_bits[e + 1] - L.cum_bits[e];
  const int rb = blockIdx.x * WAVES + wave;
  f32x4 tot[2][NTMAX];
  zero_tot(&tot[0][0], 2 * NTMAX);
  if (c_begin < c_end) {
    Streams sp;
    for (int m = 0; m < 2; ++m) stream_rsrc(L, e, m, rb, K, c_begin, c_end, sp.w[m], sp.s[m]);
    sp.lane_w = (uint32_t)lane * b * 4u;
    sp.lane_s = (uint32_t)(lane & 15) * 4u;
    auto stage = [&](uint16_t* xs_, float* sxs_, int rows, int ks, int kw, int RS) {
      stage_rows<false, true>(
          xs_, sxs_, [&](int m) { return x + (size_t)toks[m] * K; },
          [](int, int) { return 0.0f; }, nt, rows, ks, kw, RS, G);
    };
    run_expert<GPC, NTMAX, false>(b, sp, c_begin, c_end, stage, nt, G, xs, sxs, xs_bytes / 2, tot);
  }
  const int n = rb * 16 + (lane & 15);
  const size_t P = hid.P;
  if (hid.ksplit == 1) {
#pragma unroll
    for (int tb = 0; tb < NTMAX; ++tb) {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int m = tb * 16 + 4 * (lane >> 4) + i;
        if (m < nt)
          hid.h[(size_t)(pbase + m) * L.ffn + n] = float_to_half_sat(silu(tot[0][tb][i]) * tot[1][tb][i]);
      }
    }
  } else {
    float* part = hid.gu_part + (size_t)split * 2 * P * L.ffn;
#pragma unroll
    for (int tb = 0; tb < NTMAX; ++tb) {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int m = tb * 16 + 4 * (lane >> 4) + i;
        if (m < nt) {
          const size_t o = (size_t)(pbase + m) * L.ffn + n;
          part[o] = tot[0][tb][i];
          part[P * L.ffn + o] = tot[1][tb][i];
        }
      }
    }
  }
}

// ------------------------------------------------------------------- down --
// Workgroup: expert e, 32*WAVES output rows (two 16-row blocks per
// wave), one split of the ffn reduction, up to 16*NTMAX of the expert's pairs
// -> fp32 partials.  When d is not a multiple of the workgroup's rows, the
// surplus waves of the last workgroup repeat the last row blocks (identical
// values written twice) so that every wave takes part in the staging barriers.
template <int GPC, int NTMAX, int WAVES>
__global__ void __launch_bounds__(64 * WAVES)
__attribute__((amdgpu_waves_per_eu(4))) down_kernel(
    Hidden hid, LayerArgs L, const int32_t* __restrict__ counts,
    const int32_t* __restrict__ offsets, int nsplit, float* __restrict__ partial,
    size_t part_stride, int xs_bytes) {
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
  uint16_t* xs = reinterpret_cast<uint16_t*>(smem);
  float* sxs = reinterpret_cast<float*>(smem + xs_bytes);
  const int e = blockIdx.y;
  const int chunk = blockIdx.z / nsplit, split = blockIdx.z - chunk * nsplit;
  const int t0 = chunk * 16 * NTMAX;
  int ebase, ce;
  expert_range(counts, offsets, e, hid.P, ebase, ce);
  if (t0 >= ce) return;
  const int nt = (ce - t0) < 16 * NTMAX ? (ce - t0) : 16 * NTMAX;
  const int pbase = ebase + t0;
  const int lane = threadIdx.x & 63, wave = wave_id();
  const int K = L.ffn, G = L.G, ntiles = K / kTileCols;
  const int b = L.cum_bits[e + 1] - L.cum_bits[e];
  const int per = (ntiles + nsplit - 1) / nsplit;
  const int c_begin = split * per;
  const int c_end = (c_begin + per) < ntiles ? (c_begin + per) : ntiles;
  const int last_rb = L.d / kTileRows - 2;
  const int rb_want = (blockIdx.x * WAVES + wave) * 2;
  const int rb0 = rb_want < last_rb ? rb_want : last_rb;
  f32x4 tot[2][NTMAX];
  zero_tot(&tot[0][0], 2 * NTMAX);
  if (c_begin < c_end) {
    Streams sp;
    for (int j = 0; j < 2; ++j) stream_rsrc(L, e, 2, rb0 + j, K, c_begin, c_end, sp.w[j], sp.s[j]);
    sp.lane_w = (uint32_t)lane * b * 4u;
    sp.lane_s = (uint32_t)(lane & 15) * 4u;
    if (hid.ksplit == 1) {
      auto stage = [&](uint16_t* xs_, float* sxs_, int rows, int ks, int kw, int RS) {
        stage_rows<true, true>(
            xs_, sxs_, [&](int m) { return hid.h + (size_t)(pbase + m) * K; },
            [](int, int) { return 0.0f; }, nt, rows, ks, kw, RS, G);
      };
      run_expert<GPC, NTMAX, true>(b, sp, c_begin, c_end, stage, nt, G, xs, sxs, xs_bytes / 2, tot);
    } else {
      // h from the gate/up partial sums (added in split order), rounded to
      // fp16 as the ksplit == 1 gate/up epilogue would have formed it
      const size_t P = hid.P;
      auto piece = [&](int m, int k) {
        const size_t o = (size_t)(pbase + m) * K + k;
        f32x4 g0 = {0.f, 0.f, 0.f, 0.f}, g1 = g0, u0 = g0, u1 = g0;
        for (int s = 0; s < hid.ksplit; ++s) {
          const float* part = hid.gu_part + (size_t)s * 2 * P * K + o;
          g0 += *reinterpret_cast<const f32x4*>(part);
          g1 += *reinterpret_cast<const f32x4*>(part + 4);
          u0 += *reinterpret_cast<const f32x4*>(part + P * K);
          u1 += *reinterpret_cast<const f32x4*>(part + P * K + 4);
        }
        u32x4 v;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const float ha = silu(j < 2 ? g0[2 * j] : g1[2 * j - 4]) * (j < 2 ? u0[2 * j] : u1[2 * j - 4]);
          const float hb = silu(j < 2 ? g0[2 * j + 1] : g1[2 * j - 3]) *
                           (j < 2 ? u0[2 * j + 1] : u1[2 * j - 3]);
          v[j] = (uint32_t)float_to_half_sat(ha) | ((uint32_t)float_to_half_sat(hb) << 16);
        }
        return v;
      };
      auto stage = [&](uint16_t* xs_, float* sxs_, int rows, int ks, int kw, int RS) {
        stage_pieces<true>(xs_, sxs_, piece, nt, rows, ks, kw, RS, G);
      };
      run_expert<GPC, NTMAX, true>(b, sp, c_begin, c_end, stage, nt, G, xs, sxs, xs_bytes / 2, tot);
    }
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

template <int GPC, int NTMAX, int WAVES>
static hipError_t launch_gateup_nt(const uint16_t* x, const LayerArgs& L, const mc_routing& r,
                                   const Hidden& h, int xs_bytes, hipStream_t stream) {
  // set once per instantiation (thread-safe static initialisation); the slab
  // size of an instantiation is fixed
  static const hipError_t attr = allow_lds(&gateup_kernel<GPC, NTMAX, WAVES>, xs_bytes + kSxBytes + 512);
  if (attr != hipSuccess) return attr;
  const int chunks = (r.T + 16 * NTMAX - 1) / (16 * NTMAX);
  hipLaunchKernelGGL((gateup_kernel<GPC, NTMAX, WAVES>),
                     dim3(L.ffn / (16 * WAVES), L.E, chunks * h.ksplit),
                     dim3(64 * WAVES), xs_bytes + kSxBytes, stream, x, L, r.counts,
                     r.offsets, r.pair_token, h, xs_bytes);
  return hipGetLastError();
}

template <int GPC, int NTMAX, int WAVES>
static hipError_t launch_down_nt(const Hidden& h, const LayerArgs& L, const mc_routing& r,
                                 int nsplit, float* partial, size_t part_stride, int xs_bytes,
                                 hipStream_t stream) {
  // set once per instantiation (thread-safe static initialisation); the slab
  // size of an instantiation is fixed
  static const hipError_t attr = allow_lds(&down_kernel<GPC, NTMAX, WAVES>, xs_bytes + kSxBytes + 512);
  if (attr != hipSuccess) return attr;
  const int chunks = (r.T + 16 * NTMAX - 1) / (16 * NTMAX);
  const int rows_per_wg = 32 * WAVES;
  hipLaunchKernelGGL((down_kernel<GPC, NTMAX, WAVES>),
                     dim3((L.d + rows_per_wg - 1) / rows_per_wg, L.E, chunks * nsplit),
                     dim3(64 * WAVES), xs_bytes + kSxBytes, stream, h, L, r.counts,
                     r.offsets, nsplit, partial, part_stride, xs_bytes);
  return hipGetLastError();
}

template <int GPC>
hipError_t launch_gateup(const uint16_t* x, const LayerArgs& L, const mc_routing& r,
                         const Hidden& h, int ntmax, int xs_bytes, hipStream_t stream) {
  if (ntmax == 1) return launch_gateup_nt<GPC, 1, kWavesPerWg>(x, L, r, h, xs_bytes, stream);
  if (L.ffn % (16 * kGuWaves32) == 0 && h.ksplit == 1)
    return launch_gateup_nt<GPC, 2, kGuWaves32>(x, L, r, h, kGuXsBytes32, stream);
  return launch_gateup_nt<GPC, 2, kWavesPerWg>(x, L, r, h, xs_bytes, stream);
}

// As for gate/up: 32-token blocks take one 16-wave workgroup per CU (512
// output rows) with the larger h slab (measured: down 42.9 -> 39.7 us at
// T = 32, 58.6 -> 52.7 us at T = 64; slower for 16-token blocks).
template <int GPC>
hipError_t launch_down(const Hidden& h, const LayerArgs& L, const mc_routing& r, int nsplit,
                       float* partial, size_t part_stride, int ntmax, int xs_bytes,
                       hipStream_t stream) {
  if (ntmax == 1)
    return launch_down_nt<GPC, 1, kWavesPerWg>(h, L, r, nsplit, partial, part_stride, xs_bytes, stream);
  return launch_down_nt<GPC, 2, kGuWaves32>(h, L, r, nsplit, partial, part_stride, kGuXsBytes32, stream);
}

}  // namespace mc
