// prefill.hpp -- grouped GEMMs of the expert forward (Eq. 1) for batches in
// which each active expert sees many tokens: per expert e, with X_e its kept
// tokens (the CSR list of the routing step),
//   H_e = silu(X_e W_gate^T) * (X_e W_up^T)        (gate/up kernel)
//   Y_e = H_e W_down^T                              (down kernel, fp32 partials)
// and y_t = sum_r w_r Y[pos(t, r)] by the combine kernel of the decode path.
//
// The weights are never rounded.  As in the decode kernels, the codes enter
// the MFMA as exact integers offset by a power of two (magic), and the scale
// and zero of each group are applied to the fp32 group sum:
//   sum_{k in g} x_k s (q_k - z) = s * (acc_g - (magic + z) * S_g),
//   acc_g = sum_k x_k (magic + q_k) (MFMA),  S_g = sum_{k in g} x_k,
// so per group of G columns each output costs two fp32 fmas.
//  * gate/up: x stays bf16 (exact), codes are bf16 128 + q,
//    v_mfma_f32_32x32x16_bf16;
//  * down: h is rounded once to fp16 (the only rounding on the path besides
//    fp32 accumulation), codes are fp16 1024 + q, v_mfma_f32_32x32x16_f16.
// Activations are held in a fragment layout: a fragment is 32 rows x 16
// columns (1 KB), stored in the order the MFMA A operand takes it (lane l:
// row l%32, columns 8*(l/32) .. +8); a wave stages a fragment into LDS with one
// direct-to-LDS 16-byte load per lane and reads it back with one
// conflict-free ds_read_b128.  Beside each operand lie its sums over every 32
// columns, [fragment row][32 rows][K/32], from which the group sums S_g are
// formed while staging.  Rows of each expert start at a fragment boundary;
// padding rows are zero.
//
// Workgroup: 8 waves (two per SIMD), WTOK token groups x (8/WTOK) row groups;
// a wave computes 64 tokens x 2 streams of 32 weight rows (gate/up: the same
// 32 ffn rows of gate and of up; down: 64 consecutive d rows), keeping the
// group accumulators and the running fp32 totals in registers.  The
// reduction runs in 128-column chunks, double-buffered in LDS.
#pragma once

#include "forward_engine.hpp"

namespace mc {

typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x8e __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr int kPfFragRows = 32;                    // rows of a fragment (MFMA M)
constexpr int kPfFragBytes = 1024;                 // 32 rows x 16 16-bit values
constexpr int kPfWaves = 8;
constexpr int kPfWaveTiles = 2;                    // fragment rows per wave (64 tokens)
constexpr int kPfWtok = 4;                         // token groups per workgroup
constexpr uint32_t kMagicF16 = 0x64006400u;        // fp16 1024.0 in both halves

template <int WTOK>
struct PfShape {
  static constexpr int kWrow = kPfWaves / WTOK;                  // row groups
  static constexpr int kTiles = WTOK * kPfWaveTiles;             // fragment rows per workgroup
  static constexpr int kTokens = kTiles * kPfFragRows;           // tokens per m-tile
  static constexpr int kFragBytes = kTiles * 8 * kPfFragBytes;   // A fragments of one chunk
  static constexpr int kSBytes = kTiles * kPfFragRows * 4 * 4;   // group sums, <= 4 groups
  static constexpr int kStageBytes = kFragBytes + kSBytes;
  static constexpr int kLdsBytes = 2 * kStageBytes;
  static constexpr int kRowsGateUp = kWrow * 32;                 // ffn rows per gate/up workgroup
  static constexpr int kRowsDown = kWrow * 64;                   // d rows per down workgroup
  static_assert(kLdsBytes <= kLdsPerCu, "prefill stages fit the LDS of a CU");
  static_assert(kTokens <= kPfWaves * 64, "one staging thread per token row");
};
using PfCfg = PfShape<kPfWtok>;

// Expert-to-tile tables written by the set-up kernel into the workspace.
struct PrefillTables {
  int32_t* ftile_base;   // [E+1] first fragment row of each expert
  int32_t* ftile_e;      // [f_max] expert of each fragment row
  int32_t* mt_e;         // [mt_max] expert of each m-tile
  int32_t* mt_j;         // [mt_max] m-tile index within its expert
  int32_t* mt_count;     // [1] m-tiles in use
  int f_max, mt_max;
};

struct PrefillGemm {
  const uint16_t* a;     // fragment-tiled operand, K columns (bf16 x or fp16 h)
  const float* asum;     // [fragment row][32][K/32] sums of the operand over 32 columns
  int K;                 // reduction length: d (gate/up) or ffn (down)
  int n_tiles;           // workgroup row tiles of the weight matrix
  int c_per_split;       // 128-column chunks per split of the reduction
  int nsplit;
  uint16_t* h;           // gate/up output: fragment-tiled fp16 h [.][ffn]
  float* hsum;           // gate/up output: [fragment row][32][ffn/32] sums of the rounded h
  float* partial;        // down output: [nsplit][P][d] fp32
  size_t part_stride;
};

// Byte offset of element (row r, column c) of fragment row f in a tiled
// operand with K columns; an element is 2 bytes.
__host__ __device__ __forceinline__ size_t frag_offset(int f, int r, int c, int K) {
  return ((((size_t)f * (K / 16) + c / 16) * 64 + r + 32 * ((c % 16) / 8)) * 8 + (c % 8)) * 2;
}

// One weight stream: 32 rows of one matrix, this lane's row (lane%32) and two
// 64-column pieces per chunk (packed lanes n%16 + 16*(l/32) and +32).
struct PfStream {
  rsrc_t w, s;
  uint32_t off_w0, off_w1;   // byte offsets of the two pieces in chunk 0
  uint32_t off_s;            // byte offset of the first scale/zero word in chunk 0
};

__device__ __forceinline__ PfStream pf_stream(const LayerArgs& L, int e, int m, int row0, int K,
                                              int bits, int lane) {
  PfStream st;
  const int ntiles = K / kTileCols, ng = K / L.G;
  const int r = row0 + (lane & 31);
  const int rb = r >> 4, n16 = r & 15, hh = lane >> 5;
  const int R = (m == 2) ? L.d : L.ffn;
  const uint32_t* wbase = L.words + layer_word_offset(L, e, m);
  const uint32_t* sbase = L.sz + layer_sz_offset(L, e, m);
  st.w = make_rsrc(wbase, (uint32_t)((size_t)R * K / 32 * bits * 4));
  st.s = make_rsrc(sbase, (uint32_t)((size_t)R * ng * 4));
  const uint32_t row_w = (uint32_t)rb * ntiles * 64u;
  st.off_w0 = (row_w + (uint32_t)(n16 + 16 * hh)) * bits * 4u;
  st.off_w1 = (row_w + (uint32_t)(n16 + 16 * (2 + hh))) * bits * 4u;
  st.off_s = ((uint32_t)rb * ng * 16u + (uint32_t)n16) * 4u;
  return st;
}

template <int BITS, int GPC>
__device__ __forceinline__ void pf_load(uint32_t (&w)[2][BITS], uint32_t (&s)[GPC], const PfStream& st,
                                        int c) {
  const uint32_t cw = (uint32_t)c * 64u * BITS * 4u;
  load_words<BITS>(w[0], st.w, st.off_w0 + cw);
  load_words<BITS>(w[1], st.w, st.off_w1 + cw);
#pragma unroll
  for (int q = 0; q < GPC; ++q)
    s[q] = __builtin_amdgcn_raw_buffer_load_b32(st.s, st.off_s + ((uint32_t)c * GPC + q) * 64u, 0, 0);
}

// B operand of MFMA step u of one 64-column piece: 8 codes as magic + q.
template <int BITS>
__device__ __forceinline__ u32x4 pf_codes(const uint32_t (&w)[BITS], int u, uint32_t magic) {
  return u32x4{extract_pair<BITS>(w, 4 * u + 0, magic), extract_pair<BITS>(w, 4 * u + 1, magic),
               extract_pair<BITS>(w, 4 * u + 2, magic), extract_pair<BITS>(w, 4 * u + 3, magic)};
}

template <bool BF16>
__device__ __forceinline__ f32x16 pf_mfma(u32x4 a, u32x4 b, f32x16 c) {
  if constexpr (BF16)
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8e, a),
                                                   __builtin_bit_cast(bf16x8e, b), c, 0, 0, 0);
  else
    return __builtin_amdgcn_mfma_f32_32x32x16_f16(__builtin_bit_cast(f16x8, a),
                                                  __builtin_bit_cast(f16x8, b), c, 0, 0, 0);
}

// Stage chunk c: the A fragments of the m-tile's nmt fragment rows go
// straight to LDS; the 32-column sums of its rows are loaded (one row per
// thread) and written as group sums by pf_store_sums once they have arrived.
__device__ __forceinline__ void pf_stage_frags(unsigned char* stage, const PrefillGemm& g, int f0, int nmt,
                                               int c, int wave, int lane) {
  const int ksteps = g.K / 16;
  for (int q = wave; q < nmt * 8; q += kPfWaves) {
    const int mt = q >> 3, v = q & 7;
    const unsigned char* src = reinterpret_cast<const unsigned char*>(g.a) +
                               ((size_t)(f0 + mt) * ksteps + (size_t)c * 8 + v) * kPfFragBytes + lane * 16;
    __builtin_amdgcn_global_load_lds((const __attribute__((address_space(1))) void*)src,
                                     (__attribute__((address_space(3))) void*)(stage + q * kPfFragBytes),
                                     16, 0, 0);
  }
}

template <int WTOK>
__device__ __forceinline__ f32x4 pf_load_sums(const PrefillGemm& g, int f0, int nmt, int c) {
  using S = PfShape<WTOK>;
  const int r = threadIdx.x;
  f32x4 v = {0.f, 0.f, 0.f, 0.f};
  if (r < S::kTokens && (r >> 5) < nmt)
    v = *reinterpret_cast<const f32x4*>(g.asum + ((size_t)(f0 + (r >> 5)) * 32 + (r & 31)) * (g.K / 32) + 4 * c);
  return v;
}

// Group sums of the chunk: S[q][row], q < GPC groups of 128/GPC columns.
template <int GPC, int WTOK>
__device__ __forceinline__ void pf_store_sums(unsigned char* stage, f32x4 p) {
  using S = PfShape<WTOK>;
  const int r = threadIdx.x;
  if (r >= S::kTokens) return;
  float* s = reinterpret_cast<float*>(stage + S::kFragBytes);
  if constexpr (GPC == 1) {
    s[r] = (p[0] + p[1]) + (p[2] + p[3]);
  } else if constexpr (GPC == 2) {
    s[r] = p[0] + p[1];
    s[S::kTokens + r] = p[2] + p[3];
  } else {
#pragma unroll
    for (int q = 0; q < 4; ++q) s[q * S::kTokens + r] = p[q];
  }
}

template <int BITS, int GPC, bool BF16, int WTOK>
__device__ __forceinline__ void pf_loop(const PfStream (&sp)[2], const PrefillGemm& g, int f0, int nmt,
                                        int tg, bool active, int c_begin, int c_end,
                                        unsigned char* smem, int wave, int lane,
                                        f32x16 (&tot)[kPfWaveTiles][2]) {
  using S = PfShape<WTOK>;
  constexpr uint32_t magic = BF16 ? kMagic2 : kMagicF16;
  const float mval = BF16 ? 128.0f : 1024.0f;
  constexpr int KV = 8 / GPC;   // MFMA steps per group
  uint32_t w[2][2][BITS], s[2][GPC];
  f32x4 part = {0.f, 0.f, 0.f, 0.f};
  if (c_begin < c_end) {
    pf_stage_frags(smem, g, f0, nmt, c_begin, wave, lane);
    pf_store_sums<GPC, WTOK>(smem, pf_load_sums<WTOK>(g, f0, nmt, c_begin));
#pragma unroll
    for (int j = 0; j < 2; ++j) pf_load<BITS, GPC>(w[j], s[j], sp[j], c_begin);
  }
  for (int c = c_begin; c < c_end; ++c) {
    unsigned char* cur = smem + ((c - c_begin) & 1) * S::kStageBytes;
    unsigned char* nxt = smem + (((c - c_begin) & 1) ^ 1) * S::kStageBytes;
    __builtin_amdgcn_s_waitcnt(0x0F70);   // vmcnt(0): this chunk's fragments have landed
    __syncthreads();
    uint32_t wc[2][2][BITS], sc[2][GPC];
#pragma unroll
    for (int j = 0; j < 2; ++j) {
#pragma unroll
      for (int p = 0; p < 2; ++p)
#pragma unroll
        for (int b = 0; b < BITS; ++b) wc[j][p][b] = w[j][p][b];
#pragma unroll
      for (int q = 0; q < GPC; ++q) sc[j][q] = s[j][q];
    }
    const bool more = c + 1 < c_end;
    if (more) {
      pf_stage_frags(nxt, g, f0, nmt, c + 1, wave, lane);
      part = pf_load_sums<WTOK>(g, f0, nmt, c + 1);
#pragma unroll
      for (int j = 0; j < 2; ++j) pf_load<BITS, GPC>(w[j], s[j], sp[j], c + 1);
    }
    if (active) {
      const unsigned char* arow = cur + (2 * tg * 8) * kPfFragBytes + lane * 16;
      const float* ssum = reinterpret_cast<const float*>(cur + S::kFragBytes);
#pragma unroll
      for (int q = 0; q < GPC; ++q) {
        f32x16 acc[kPfWaveTiles][2];
#pragma unroll
        for (int vv = 0; vv < KV; ++vv) {
          const int v = q * KV + vv;
          u32x4 a[kPfWaveTiles];
#pragma unroll
          for (int t = 0; t < kPfWaveTiles; ++t)
            a[t] = *reinterpret_cast<const u32x4*>(arow + (t * 8 + v) * kPfFragBytes);
          const u32x4 b0 = pf_codes<BITS>(wc[0][v & 1], v >> 1, magic);
          const u32x4 b1 = pf_codes<BITS>(wc[1][v & 1], v >> 1, magic);
#pragma unroll
          for (int t = 0; t < kPfWaveTiles; ++t) {
            const f32x16 z = {};
            acc[t][0] = pf_mfma<BF16>(a[t], b0, vv == 0 ? z : acc[t][0]);
            acc[t][1] = pf_mfma<BF16>(a[t], b1, vv == 0 ? z : acc[t][1]);
          }
        }
        // tot += s * (acc - (magic + z) * S_g), per lane: its row's s and z
        float sj[2], cj[2];
#pragma unroll
        for (int j = 0; j < 2; ++j) {
          sj[j] = half_bits_to_float(sc[j][q] & 0xffffu);
          cj[j] = mval + half_bits_to_float(sc[j][q] >> 16);
        }
#pragma unroll
        for (int t = 0; t < kPfWaveTiles; ++t) {
          const float* sr = ssum + q * S::kTokens + (2 * tg + t) * 32 + 4 * (lane >> 5);
          f32x4 sx[4];
#pragma unroll
          for (int k4 = 0; k4 < 4; ++k4) sx[k4] = *reinterpret_cast<const f32x4*>(sr + 8 * k4);
#pragma unroll
          for (int j = 0; j < 2; ++j)
#pragma unroll
            for (int i = 0; i < 16; ++i) {
              const float u = fmaf(-cj[j], sx[i >> 2][i & 3], acc[t][j][i]);
              tot[t][j][i] = fmaf(sj[j], u, tot[t][j][i]);
            }
        }
      }
    }
    if (more) pf_store_sums<GPC, WTOK>(nxt, part);
  }
}

// Grid: mt_max * n_tiles * nsplit workgroups (m-tile major); workgroups past
// the m-tiles in use exit at once.
template <int GPC, bool GATEUP>
__global__ void __launch_bounds__(64 * kPfWaves) __attribute__((amdgpu_waves_per_eu(2, 2)))
prefill_kernel(LayerArgs L, const int32_t* __restrict__ offsets, PrefillTables tb, PrefillGemm g) {
  using S = PfCfg;
  extern __shared__ __attribute__((aligned(1024))) unsigned char smem[];
  const int per_mt = g.n_tiles * g.nsplit;
  const int mt = blockIdx.x / per_mt;
  if (mt >= *tb.mt_count) return;
  const int rest = blockIdx.x - mt * per_mt;
  const int split = rest / g.n_tiles, nt = rest - split * g.n_tiles;
  const int e = tb.mt_e[mt], j = tb.mt_j[mt];
  const int f0 = tb.ftile_base[e] + S::kTiles * j;
  const int nf = tb.ftile_base[e + 1] - f0;
  const int nmt = nf < S::kTiles ? nf : S::kTiles;
  const int lane = threadIdx.x & 63, wave = wave_id();
  const int tg = wave / S::kWrow, rg = wave - tg * S::kWrow;
  const bool active = 2 * tg < nmt;
  const int ntiles = g.K / kTileCols;
  const int c_begin = split * g.c_per_split;
  const int c_end = (c_begin + g.c_per_split) < ntiles ? (c_begin + g.c_per_split) : ntiles;
  const int bits = L.cum_bits[e + 1] - L.cum_bits[e];

  int row[2];
  PfStream sp[2];
  if (GATEUP) {
    row[0] = row[1] = nt * S::kRowsGateUp + 32 * rg;
    sp[0] = pf_stream(L, e, 0, row[0], g.K, bits, lane);
    sp[1] = pf_stream(L, e, 1, row[1], g.K, bits, lane);
  } else {
    int r0 = nt * S::kRowsDown + 64 * rg;
    if (r0 + 64 > L.d) r0 = L.d - 64;   // surplus waves of the last tile repeat the last rows
    row[0] = r0;
    row[1] = r0 + 32;
    sp[0] = pf_stream(L, e, 2, row[0], g.K, bits, lane);
    sp[1] = pf_stream(L, e, 2, row[1], g.K, bits, lane);
  }

  f32x16 tot[kPfWaveTiles][2];
#pragma unroll
  for (int t = 0; t < kPfWaveTiles; ++t)
#pragma unroll
    for (int s = 0; s < 2; ++s)
#pragma unroll
      for (int i = 0; i < 16; ++i) tot[t][s][i] = 0.0f;

  if (bits == 1)
    pf_loop<1, GPC, GATEUP, kPfWtok>(sp, g, f0, nmt, tg, active, c_begin, c_end, smem, wave, lane, tot);
  else if (bits == 2)
    pf_loop<2, GPC, GATEUP, kPfWtok>(sp, g, f0, nmt, tg, active, c_begin, c_end, smem, wave, lane, tot);
  else
    pf_loop<3, GPC, GATEUP, kPfWtok>(sp, g, f0, nmt, tg, active, c_begin, c_end, smem, wave, lane, tot);
  if (!active) return;

  // D layout: lane holds column n = lane%32 (weight row) and, for i < 16,
  // row m = 8*(i/4) + 4*(lane/32) + i%4 (token) of each 32x32 tile.
  const int n = lane & 31;
  if (GATEUP) {
    const int col = row[0] + n;
    unsigned char* hb = reinterpret_cast<unsigned char*>(g.h);
#pragma unroll
    for (int t = 0; t < kPfWaveTiles; ++t) {
      const int f = f0 + 2 * tg + t;
      if (2 * tg + t < nmt) {
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          const int m = 8 * (i >> 2) + 4 * (lane >> 5) + (i & 3);
          const uint16_t h16 = float_to_half_sat(silu(tot[t][0][i]) * tot[t][1][i]);
          *reinterpret_cast<uint16_t*>(hb + frag_offset(f, m, col, L.ffn)) = h16;
          // sum of the rounded h over this wave's 32 columns (the lanes of one half), fixed order
          float v = half_bits_to_float(h16);
#pragma unroll
          for (int off = 1; off < 32; off <<= 1) v += __shfl_xor(v, off);
          if (n == 0) g.hsum[((size_t)f * 32 + m) * (L.ffn / 32) + row[0] / 32] = v;
        }
      }
    }
  } else {
    const int pbase = offsets[e] + S::kTokens * j;
    const int pend = offsets[e + 1];
    float* out = g.partial + (size_t)split * g.part_stride;
#pragma unroll
    for (int t = 0; t < kPfWaveTiles; ++t) {
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const int m = 8 * (i >> 2) + 4 * (lane >> 5) + (i & 3);
        const int pos = pbase + (2 * tg + t) * 32 + m;
        if (pos < pend) {
#pragma unroll
          for (int s = 0; s < 2; ++s) out[(size_t)pos * L.d + row[s] + n] = tot[t][s][i];
        }
      }
    }
  }
}

template <int GPC>
hipError_t launch_prefill_gemm(const LayerArgs& L, const int32_t* offsets, const PrefillTables& tb,
                               const PrefillGemm& g, bool gateup, hipStream_t stream) {
  static bool attr[2] = {false, false};
  const void* fn = gateup ? reinterpret_cast<const void*>(&prefill_kernel<GPC, true>)
                          : reinterpret_cast<const void*>(&prefill_kernel<GPC, false>);
  if (!attr[gateup]) {
    const hipError_t e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, PfCfg::kLdsBytes);
    if (e != hipSuccess) return e;
    attr[gateup] = true;
  }
  const dim3 grid(tb.mt_max * g.n_tiles * g.nsplit);
  if (gateup)
    hipLaunchKernelGGL((prefill_kernel<GPC, true>), grid, dim3(64 * kPfWaves), PfCfg::kLdsBytes, stream, L,
                       offsets, tb, g);
  else
    hipLaunchKernelGGL((prefill_kernel<GPC, false>), grid, dim3(64 * kPfWaves), PfCfg::kLdsBytes, stream, L,
                       offsets, tb, g);
  return hipGetLastError();
}

}  // namespace mc
