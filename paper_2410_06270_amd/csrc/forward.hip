// forward.hip -- Eq. 1 over packed SwiGLU experts (dequantization in registers).
//
// y_t = sum over kept ranks r of w_r * E_{e_r}(x_t),
// E_e(x) = W_down (silu(W_gate x) * (W_up x)), weights s*(q - z) per group.
//
// The codes go straight into bf16 MFMA operands as 128 + q (exact), so the
// dequantized weight is never rounded: for each group g of G inputs
//   sum_k s (q_k - z) x_k = s * (acc_g - (128 + z) * sum_k x_k),
// acc_g = sum_k (128 + q_k) x_k from the MFMA; the group sums of x are formed
// once per workgroup in LDS.  The hidden vector h is kept as two bf16 planes
// (h = hi + lo, ~16 significant bits) for the down projection.
//
// Kernels (all on the caller's stream, no host synchronisation; experts with
// no kept token exit at once because the counts are read on the device):
//   gateup_kernel  grid (ffn/64, E, chunks): 4 waves x 16 rows of gate and up,
//                  tokens of one expert (<= 16*NTB per chunk) -> h planes;
//   down_kernel    grid (d/64, E, chunks*S): split-K over ffn -> fp32 partials;
//   combine_kernel grid (d/256, T): y = bf16(sum_r w_r sum_s partial), fixed
//                  order, so the result is deterministic.
#include "mc_internal.hpp"

namespace mc {

constexpr uint32_t kMagic2 = 0x43004300u;     // bf16 128.0 in both halves
constexpr int kXsBytes = 40 * 1024;           // activation slab (LDS)
constexpr int kSxBytes = 8 * 1024;            // group sums of the slab (LDS)
constexpr int kRowPad = 8;                    // bf16 elements of padding per slab row

struct SlabShape {
  int KS;   // slab width (multiple of max(128, G))
  int RS;   // LDS row stride in bf16 elements
};

__device__ __forceinline__ SlabShape slab_shape(int K, int G, int nt, int planes, int ntb) {
  const int unit = G > kTileCols ? G : kTileCols;
  int ks = (kXsBytes / (2 * planes * nt)) - kRowPad;
  const int ks_sx = (kSxBytes / (4 * 16 * ntb)) * G;
  ks = ks < ks_sx ? ks : ks_sx;
  ks = (ks / unit) * unit;
  if (ks < unit) ks = unit;
  if (ks > K) ks = K;
  return {ks, ks + kRowPad};
}

__device__ __forceinline__ float silu(float a) { return a / (1.0f + expf(-a)); }

__device__ __forceinline__ bf16x8 load_a(const uint16_t* p, bool valid) {
  u32x4 v = {0u, 0u, 0u, 0u};
  if (valid) v = *reinterpret_cast<const u32x4*>(p);
  return __builtin_bit_cast(bf16x8, v);
}

template <int BITS>
__device__ __forceinline__ bf16x8 b_operand(const uint32_t* w, int u) {
  u32x4 v;
  v[0] = extract_pair<BITS>(w, 4 * u + 0, kMagic2);
  v[1] = extract_pair<BITS>(w, 4 * u + 1, kMagic2);
  v[2] = extract_pair<BITS>(w, 4 * u + 2, kMagic2);
  v[3] = extract_pair<BITS>(w, 4 * u + 3, kMagic2);
  return __builtin_bit_cast(bf16x8, v);
}

// Stage rows of activations [nt][kw] (plane 0, and plane 1 when PLANES == 2)
// into LDS and form their group sums.  rowptr(m) gives the source row start.
template <int PLANES, typename RowFn>
__device__ __forceinline__ void stage_slab(uint16_t* xs, float* sxs, RowFn rowptr, int nt, int ntb,
                                           int ks, int kw, int RS, int G, size_t plane_stride) {
  const int pieces = kw / 8;   // 16-byte pieces per row
  for (int idx = threadIdx.x; idx < PLANES * nt * pieces; idx += blockDim.x) {
    const int pl = idx / (nt * pieces);
    const int rest = idx - pl * nt * pieces;
    const int m = rest / pieces, p = rest - m * pieces;
    const uint16_t* src = rowptr(m) + pl * plane_stride + ks + 8 * p;
    *reinterpret_cast<u32x4*>(xs + (size_t)(pl * nt + m) * RS + 8 * p) =
        *reinterpret_cast<const u32x4*>(src);
  }
  __syncthreads();
  const int ngs = kw / G, rows = 16 * ntb;
  for (int idx = threadIdx.x; idx < ngs * rows; idx += blockDim.x) {
    const int gl = idx / rows, m = idx - gl * rows;
    float s = 0.0f;
    if (m < nt) {
      for (int pl = 0; pl < PLANES; ++pl) {
        const uint16_t* r = xs + (size_t)(pl * nt + m) * RS + gl * G;
        for (int j = 0; j < G; ++j) s += bf16_bits_to_float(r[j]);
      }
    }
    sxs[gl * rows + m] = s;
  }
  __syncthreads();
}

// Group epilogue: tot += s * (acc - (128 + z) * sum_x); acc = 0.
__device__ __forceinline__ void group_end(f32x4& acc, f32x4& tot, uint32_t szw, const float* sx4p) {
  const float s = half_bits_to_float(szw & 0xffffu);
  const float c = 128.0f + half_bits_to_float(szw >> 16);
  const f32x4 sx = *reinterpret_cast<const f32x4*>(sx4p);
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const float t = fmaf(-c, sx[i], acc[i]);
    tot[i] = fmaf(s, t, tot[i]);
    acc[i] = 0.0f;
  }
}

// ---------------------------------------------------------------- gate/up --

template <int BITS, int NTB>
__device__ void gateup_body(const uint16_t* __restrict__ x, const LayerArgs& L, int e, int nt,
                            int pbase, const int* toks, uint16_t* __restrict__ h_hi,
                            uint16_t* __restrict__ h_lo, uint16_t* xs, float* sxs) {
  const int K = L.d, G = L.G, ng = K / G;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int rb = blockIdx.x * 4 + wave;
  const int ntiles = K / kTileCols;
  const int ntb = (nt + 15) / 16;
  const size_t wofs = ((size_t)rb * ntiles * 64 + lane) * BITS;
  const uint32_t* wg = L.words + layer_word_offset(L, e, 0) + wofs;
  const uint32_t* wu = L.words + layer_word_offset(L, e, 1) + wofs;
  const uint32_t* szg = L.sz + layer_sz_offset(L, e, 0) + (size_t)rb * ng * 16 + (lane & 15);
  const uint32_t* szu = L.sz + layer_sz_offset(L, e, 1) + (size_t)rb * ng * 16 + (lane & 15);
  const SlabShape sh = slab_shape(K, G, nt, 1, ntb);
  const int rows = 16 * ntb;

  f32x4 accg[NTB], accu[NTB], totg[NTB], totu[NTB];
#pragma unroll
  for (int tb = 0; tb < NTB; ++tb)
    for (int i = 0; i < 4; ++i) accg[tb][i] = accu[tb][i] = totg[tb][i] = totu[tb][i] = 0.0f;

  auto rowptr = [&](int m) { return x + (size_t)toks[m] * K; };
  for (int ks = 0; ks < K; ks += sh.KS) {
    const int kw = (K - ks) < sh.KS ? (K - ks) : sh.KS;
    __syncthreads();
    stage_slab<1>(xs, sxs, rowptr, nt, ntb, ks, kw, sh.RS, G, 0);
    const int nch = kw / kTileCols;
    for (int c = 0; c < nch; ++c) {
      const size_t kc = (size_t)(ks / kTileCols + c);
      uint32_t gw[BITS], uw[BITS];
#pragma unroll
      for (int p = 0; p < BITS; ++p) {
        gw[p] = wg[kc * 64 * BITS + p];
        uw[p] = wu[kc * 64 * BITS + p];
      }
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const bf16x8 bg = b_operand<BITS>(gw, u);
        const bf16x8 bu = b_operand<BITS>(uw, u);
        const int kk = c * kTileCols + 32 * u + 8 * (lane >> 4);
#pragma unroll
        for (int tb = 0; tb < NTB; ++tb) {
          if (tb < ntb) {
            const int m = tb * 16 + (lane & 15);
            const bf16x8 a = load_a(xs + (size_t)m * sh.RS + kk, m < nt);
            accg[tb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, bg, accg[tb], 0, 0, 0);
            accu[tb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, bu, accu[tb], 0, 0, 0);
          }
        }
        const int kend = ks + c * kTileCols + 32 * (u + 1);
        if (kend % G == 0) {
          const int g = kend / G - 1, gl = g - ks / G;
          const uint32_t sg = szg[(size_t)g * 16], su = szu[(size_t)g * 16];
#pragma unroll
          for (int tb = 0; tb < NTB; ++tb) {
            if (tb < ntb) {
              const float* sxp = sxs + gl * rows + tb * 16 + 4 * (lane >> 4);
              group_end(accg[tb], totg[tb], sg, sxp);
              group_end(accu[tb], totu[tb], su, sxp);
            }
          }
        }
      }
    }
  }
  const int n = rb * 16 + (lane & 15);
#pragma unroll
  for (int tb = 0; tb < NTB; ++tb) {
    for (int i = 0; i < 4; ++i) {
      const int m = tb * 16 + 4 * (lane >> 4) + i;
      if (tb < ntb && m < nt) {
        const float h = silu(totg[tb][i]) * totu[tb][i];
        const uint16_t hi = float_to_bf16(h);
        const uint16_t lo = float_to_bf16(h - bf16_bits_to_float(hi));
        const size_t o = (size_t)(pbase + m) * L.ffn + n;
        h_hi[o] = hi;
        h_lo[o] = lo;
      }
    }
  }
}

template <int NTB>
__global__ void __launch_bounds__(256) gateup_kernel(const uint16_t* __restrict__ x, LayerArgs L,
                                                     const int32_t* __restrict__ counts,
                                                     const int32_t* __restrict__ offsets,
                                                     const int32_t* __restrict__ pair_token,
                                                     uint16_t* __restrict__ h_hi,
                                                     uint16_t* __restrict__ h_lo) {
  __shared__ __attribute__((aligned(16))) uint16_t xs[kXsBytes / 2];
  __shared__ __attribute__((aligned(16))) float sxs[kSxBytes / 4];
  __shared__ int toks[16 * NTB];
  const int e = blockIdx.y;
  const int t0 = blockIdx.z * 16 * NTB;
  const int ce = counts[e];
  if (t0 >= ce) return;
  const int nt = (ce - t0) < 16 * NTB ? (ce - t0) : 16 * NTB;
  const int pbase = offsets[e] + t0;
  for (int i = threadIdx.x; i < nt; i += blockDim.x) toks[i] = pair_token[pbase + i];
  const int b = L.cum_bits[e + 1] - L.cum_bits[e];
  if (b == 1) gateup_body<1, NTB>(x, L, e, nt, pbase, toks, h_hi, h_lo, xs, sxs);
  else if (b == 2) gateup_body<2, NTB>(x, L, e, nt, pbase, toks, h_hi, h_lo, xs, sxs);
  else gateup_body<3, NTB>(x, L, e, nt, pbase, toks, h_hi, h_lo, xs, sxs);
}

// ------------------------------------------------------------------- down --

template <int BITS, int NTB>
__device__ void down_body(const uint16_t* __restrict__ h_hi, size_t plane_stride, const LayerArgs& L,
                          int e, int nt, int pbase, int split, int nsplit, float* __restrict__ partial,
                          size_t part_stride, uint16_t* xs, float* sxs) {
  const int K = L.ffn, G = L.G, ng = K / G;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int rb = blockIdx.x * 4 + wave;
  const int ntiles = K / kTileCols;
  const int ntb = (nt + 15) / 16;
  const int per = (ntiles + nsplit - 1) / nsplit;             // chunks per split (G <= 128)
  const int c_begin = split * per;
  const int c_end = (c_begin + per) < ntiles ? (c_begin + per) : ntiles;
  const size_t wofs = ((size_t)rb * ntiles * 64 + lane) * BITS;
  const uint32_t* wd = L.words + layer_word_offset(L, e, 2) + wofs;
  const uint32_t* szd = L.sz + layer_sz_offset(L, e, 2) + (size_t)rb * ng * 16 + (lane & 15);
  const SlabShape sh = slab_shape(K, G, nt, 2, ntb);
  const int rows = 16 * ntb;

  f32x4 acc[NTB], tot[NTB];
#pragma unroll
  for (int tb = 0; tb < NTB; ++tb)
    for (int i = 0; i < 4; ++i) acc[tb][i] = tot[tb][i] = 0.0f;

  auto rowptr = [&](int m) { return h_hi + (size_t)(pbase + m) * K; };
  const int kbeg = c_begin * kTileCols, kstop = c_end * kTileCols;
  for (int ks = kbeg; ks < kstop; ks += sh.KS) {
    const int kw = (kstop - ks) < sh.KS ? (kstop - ks) : sh.KS;
    __syncthreads();
    stage_slab<2>(xs, sxs, rowptr, nt, ntb, ks, kw, sh.RS, G, plane_stride);
    const int nch = kw / kTileCols;
    for (int c = 0; c < nch; ++c) {
      const size_t kc = (size_t)(ks / kTileCols + c);
      uint32_t dw[BITS];
#pragma unroll
      for (int p = 0; p < BITS; ++p) dw[p] = wd[kc * 64 * BITS + p];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const bf16x8 bd = b_operand<BITS>(dw, u);
        const int kk = c * kTileCols + 32 * u + 8 * (lane >> 4);
#pragma unroll
        for (int tb = 0; tb < NTB; ++tb) {
          if (tb < ntb) {
            const int m = tb * 16 + (lane & 15);
            const bf16x8 ahi = load_a(xs + (size_t)m * sh.RS + kk, m < nt);
            const bf16x8 alo = load_a(xs + (size_t)(nt + m) * sh.RS + kk, m < nt);
            acc[tb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ahi, bd, acc[tb], 0, 0, 0);
            acc[tb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(alo, bd, acc[tb], 0, 0, 0);
          }
        }
        const int kend = ks + c * kTileCols + 32 * (u + 1);
        if (kend % G == 0) {
          const int g = kend / G - 1, gl = (kend - ks) / G - 1;
          const uint32_t sw = szd[(size_t)g * 16];
#pragma unroll
          for (int tb = 0; tb < NTB; ++tb)
            if (tb < ntb) group_end(acc[tb], tot[tb], sw, sxs + gl * rows + tb * 16 + 4 * (lane >> 4));
        }
      }
    }
  }
  const int n = rb * 16 + (lane & 15);
#pragma unroll
  for (int tb = 0; tb < NTB; ++tb) {
    for (int i = 0; i < 4; ++i) {
      const int m = tb * 16 + 4 * (lane >> 4) + i;
      if (tb < ntb && m < nt) partial[(size_t)split * part_stride + (size_t)(pbase + m) * L.d + n] = tot[tb][i];
    }
  }
}

template <int NTB>
__global__ void __launch_bounds__(256) down_kernel(const uint16_t* __restrict__ h_hi,
                                                   size_t plane_stride, LayerArgs L,
                                                   const int32_t* __restrict__ counts,
                                                   const int32_t* __restrict__ offsets, int nsplit,
                                                   float* __restrict__ partial, size_t part_stride) {
  __shared__ __attribute__((aligned(16))) uint16_t xs[kXsBytes / 2];
  __shared__ __attribute__((aligned(16))) float sxs[kSxBytes / 4];
  const int e = blockIdx.y;
  const int chunk = blockIdx.z / nsplit, split = blockIdx.z - chunk * nsplit;
  const int t0 = chunk * 16 * NTB;
  const int ce = counts[e];
  if (t0 >= ce) return;
  const int nt = (ce - t0) < 16 * NTB ? (ce - t0) : 16 * NTB;
  const int pbase = offsets[e] + t0;
  const int b = L.cum_bits[e + 1] - L.cum_bits[e];
  if (b == 1) down_body<1, NTB>(h_hi, plane_stride, L, e, nt, pbase, split, nsplit, partial, part_stride, xs, sxs);
  else if (b == 2) down_body<2, NTB>(h_hi, plane_stride, L, e, nt, pbase, split, nsplit, partial, part_stride, xs, sxs);
  else down_body<3, NTB>(h_hi, plane_stride, L, e, nt, pbase, split, nsplit, partial, part_stride, xs, sxs);
}

// ---------------------------------------------------------------- combine --

__global__ void __launch_bounds__(256) combine_kernel(const float* __restrict__ partial,
                                                      size_t part_stride, int nsplit,
                                                      const int32_t* __restrict__ pair_pos,
                                                      const float* __restrict__ topk_w, int k, int d,
                                                      uint16_t* __restrict__ y) {
  const int t = blockIdx.y;
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= d) return;
  float acc = 0.0f;
  for (int r = 0; r < k; ++r) {
    const int pos = pair_pos[(size_t)t * k + r];
    if (pos < 0) continue;
    float v = 0.0f;
    for (int s = 0; s < nsplit; ++s) v += partial[(size_t)s * part_stride + (size_t)pos * d + i];
    acc = fmaf(topk_w[(size_t)t * k + r], v, acc);
  }
  y[(size_t)t * d + i] = float_to_bf16(acc);
}

// --------------------------------------------------------------- launchers --

// Split of the down projection's reduction so that small batches still give
// about 1024 workgroups; one split for prefill-sized batches.
int forward_nsplit(int T, int E, int k, int d, int ffn) {
  const int tiles = d / 64;
  const int active = (T * k) < E ? (T * k) : E;
  int s = (1024 + tiles * active - 1) / (tiles * active);
  const int maxs = (ffn / kTileCols) / 2;
  if (T > kDecodeMaxT) s = 1;
  if (s > maxs) s = maxs;
  if (s > 8) s = 8;
  if (s < 1) s = 1;
  return s;
}

size_t forward_workspace_bytes(int T, int E, int k, int d, int ffn) {
  const size_t P = (size_t)T * k;
  const size_t h = 2 * P * ffn * sizeof(uint16_t);
  const size_t part = (size_t)forward_nsplit(T, E, k, d, ffn) * P * d * sizeof(float);
  return ((h + 255) / 256) * 256 + part;
}

hipError_t launch_forward(const uint16_t* x, const LayerArgs& L, const mc_routing& r, uint16_t* y,
                          void* ws, hipStream_t stream) {
  const int T = r.T, k = r.k;
  const size_t P = (size_t)T * k;
  uint16_t* h_hi = static_cast<uint16_t*>(ws);
  const size_t plane = P * L.ffn;
  uint16_t* h_lo = h_hi + plane;
  (void)h_lo;
  const size_t hbytes = ((2 * plane * sizeof(uint16_t) + 255) / 256) * 256;
  float* partial = reinterpret_cast<float*>(static_cast<char*>(ws) + hbytes);
  const size_t part_stride = P * L.d;
  const int nsplit = forward_nsplit(T, r.E, k, L.d, L.ffn);
  int ntb = T <= 16 ? 1 : (T <= 32 ? 2 : 4);
  const int tpc = 16 * ntb;                     // tokens per chunk
  const int chunks = (T + tpc - 1) / tpc;
  const dim3 block(256);
  const dim3 g1(L.ffn / 64, L.E, chunks);
  const dim3 g2(L.d / 64, L.E, chunks * nsplit);
#define MC_FWD(NTB)                                                                              \
  hipLaunchKernelGGL((gateup_kernel<NTB>), g1, block, 0, stream, x, L, r.counts, r.offsets,      \
                     r.pair_token, h_hi, h_hi + plane);                                          \
  hipLaunchKernelGGL((down_kernel<NTB>), g2, block, 0, stream, h_hi, plane, L, r.counts,         \
                     r.offsets, nsplit, partial, part_stride);
  if (ntb == 1) { MC_FWD(1) } else if (ntb == 2) { MC_FWD(2) } else { MC_FWD(4) }
#undef MC_FWD
  hipError_t err = hipGetLastError();
  if (err != hipSuccess) return err;
  hipLaunchKernelGGL(combine_kernel, dim3((L.d + 255) / 256, T), block, 0, stream, partial,
                     part_stride, nsplit, r.pair_pos, r.topk_w, k, L.d, y);
  return hipGetLastError();
}

}  // namespace mc
