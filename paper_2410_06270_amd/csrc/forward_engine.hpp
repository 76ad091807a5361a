// forward_engine.hpp -- Eq. 1 over packed SwiGLU experts (dequantization in
// registers): the pieces the bandwidth-bound GEMVs (decode.hpp) are built of.
//
// y_t = sum over kept ranks r of w_r * E_{e_r}(x_t),
// E_e(x) = W_down (silu(W_gate x) * (W_up x)), weights s*(q - z) per group.
//
// The codes go straight into 16-bit MFMA operands as the exact value
// 1 + q * 2^-b (the code in the top b mantissa bits of 1.0; bf16 against the
// bf16 activations x for gate and up, fp16 against the fp16 hidden vector h
// for down), so the dequantized weight is never rounded: for each group g of
// G inputs a_k, with S = sum_k a_k,
//   sum_k s (q_k - z) a_k = (s * 2^b) * (acc_g - (1 + z * 2^-b) * S),
// acc_g = sum_k (1 + q_k 2^-b) a_k from the MFMA.  The accumulators stay near
// the size of the activation sums, so fp32 accumulation loses little.  The
// group sums of the activations (of the fp16 values, for h) are formed while
// they are staged into LDS.
#pragma once

#include "mc_internal.hpp"

namespace mc {

constexpr int kRowPad = 8;                    // elements of padding per slab row
constexpr int kLdsPerCu = 160 * 1024;
// Chunks (16 rows x 128 columns of codes) kept in flight per weight stream:
// fewer where the scale/zero words of a chunk take many registers.
__host__ __device__ constexpr int prefetch_depth(int ntb, int gpc) {
  return (ntb >= 3 || gpc >= 4) ? 2 : 4;
}

// silu(a) = a / (1 + e^-a) from the hardware base-2 exponential and
// reciprocal (each within about 1 ulp): a few ulp of fp32, far below the fp16
// rounding that follows it.  Large |a| saturate correctly (e^-a = inf gives
// -0, e^-a = 0 gives a).
__device__ __forceinline__ float silu(float a) {
  return a * __builtin_amdgcn_rcpf(1.0f + __builtin_amdgcn_exp2f(-a * 1.4426950408889634f));
}

// Operand format of the activations: bf16 (x) or fp16 (h).  Codes of b bits
// sit in the top b bits of the mantissa of 1.0 (bit kPos<b> upwards).
template <bool F16>
struct Fmt {
  static constexpr uint32_t kMagic2 = F16 ? 0x3c003c00u : 0x3f803f80u;   // 1.0 in both halves
  template <int BITS>
  static constexpr int kPos = (F16 ? 10 : 7) - BITS;
};

template <bool F16>
__device__ __forceinline__ f32x4 mfma16(u32x4 a, u32x4 b, f32x4 c) {
  if constexpr (F16)
    return __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(f16x8, a),
                                                  __builtin_bit_cast(f16x8, b), c, 0, 0, 0);
  else
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                   __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}

// A constant the compiler keeps in a VGPR: with the mask in an SGPR it lets
// (w >> f) & mask | magic issue as one v_and_or_b32 (gfx9 VOP3 encodings take
// no literal constants).
__device__ __forceinline__ uint32_t vgpr_constant(uint32_t c) {
  uint32_t v;
  asm volatile("v_mov_b32 %0, %1" : "=v"(v) : "i"(c));
  return v;
}

template <int BITS, bool F16>
__device__ __forceinline__ u32x4 b_operand(const uint32_t* w, int u, uint32_t magic) {
  constexpr int POS = Fmt<F16>::template kPos<BITS>;
  u32x4 v;
  v[0] = code_pair<BITS, POS>(w, 4 * u + 0, magic);
  v[1] = code_pair<BITS, POS>(w, 4 * u + 1, magic);
  v[2] = code_pair<BITS, POS>(w, 4 * u + 2, magic);
  v[3] = code_pair<BITS, POS>(w, 4 * u + 3, magic);
  return v;
}

// Sum of the eight 16-bit values of a piece, in element order.
template <bool F16>
__device__ __forceinline__ float sum8(u32x4 v) {
  float s = 0.0f;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    if constexpr (F16) {
      s += half_bits_to_float(v[i] & 0xffffu);
      s += half_bits_to_float(v[i] >> 16);
    } else {
      s += __uint_as_float(v[i] << 16);
      s += __uint_as_float(v[i] & 0xffff0000u);
    }
  }
  return s;
}

// Group epilogue: tot += s 2^b * (acc - (1 + z 2^-b) * sum_a) (both scalings
// by powers of two are exact).  The next group's first MFMA starts from zero.
template <int BITS>
__device__ __forceinline__ void group_end(const f32x4& acc, f32x4& tot, uint32_t szw, const float* sx4p) {
  const float s = half_bits_to_float(szw & 0xffffu) * (float)(1 << BITS);
  const float c = fmaf(half_bits_to_float(szw >> 16), 1.0f / (float)(1 << BITS), 1.0f);
  const f32x4 sx = *reinterpret_cast<const f32x4*>(sx4p);
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const float t = fmaf(-c, sx[i], acc[i]);
    tot[i] = fmaf(s, t, tot[i]);
  }
}

// Weight streams read through buffer resources: a wave-uniform chunk offset
// and one lane-offset VGPR, with the hardware's range check.
typedef __amdgpu_buffer_rsrc_t rsrc_t;
constexpr int kRsrcWord3 = 0x00020000;   // raw 32-bit buffer (gfx9 family)

__device__ __forceinline__ rsrc_t make_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes, kRsrcWord3);
}

template <int BITS>
__device__ __forceinline__ void load_words(uint32_t (&w)[BITS], rsrc_t r, uint32_t off) {
  if constexpr (BITS == 1) {
    w[0] = __builtin_amdgcn_raw_buffer_load_b32(r, off, 0, 0);
  } else if constexpr (BITS == 2) {
    const auto v = __builtin_amdgcn_raw_buffer_load_b64(r, off, 0, 0);
    w[0] = v[0];
    w[1] = v[1];
  } else {
    const auto v = __builtin_amdgcn_raw_buffer_load_b96(r, off, 0, 0);
    w[0] = v[0];
    w[1] = v[1];
    w[2] = v[2];
  }
}

// As load_words, with a VGPR offset (the lane's) and an SGPR offset (wave-uniform).
template <int BITS>
__device__ __forceinline__ void load_words_so(uint32_t (&w)[BITS], rsrc_t r, uint32_t voff, uint32_t soff) {
  if constexpr (BITS == 1) {
    w[0] = __builtin_amdgcn_raw_buffer_load_b32(r, voff, soff, 0);
  } else if constexpr (BITS == 2) {
    const auto v = __builtin_amdgcn_raw_buffer_load_b64(r, voff, soff, 0);
    w[0] = v[0];
    w[1] = v[1];
  } else {
    const auto v = __builtin_amdgcn_raw_buffer_load_b96(r, voff, soff, 0);
    w[0] = v[0];
    w[1] = v[1];
    w[2] = v[2];
  }
}

// ------------------------------------------------------------------ slabs --
// A slab holds columns [ks, ks + kw) of the nt token rows (row stride RS =
// slab width + kRowPad elements; a zero row follows for padding tokens) and
// the sums of each group of G columns, sxs[group][rows].

// Rows that are plain copies of global memory (x; h when the gate/up reduction
// was not split), row m starting at row_src(m), in two halves so that other
// loads can be issued between them:
//  * stage_rows_issue: direct-to-LDS 16-byte loads, 64 consecutive pieces of
//    a row per wave instruction, so every wave has all its loads in flight at
//    once;
//  * stage_rows_sums, once the caller has waited for those loads: each wave
//    forms the group sums of its own row segments (a segment is 512 columns,
//    a whole number of groups; the G/8 lanes of a group add in a fixed
//    butterfly order), then the workgroup's barrier.
// The waves w of the nwaves that stage this slab (a workgroup may stage
// several slabs at once) take its segments in turn.
template <typename RowFn>
__device__ __forceinline__ void stage_rows_issue(uint16_t* xs, RowFn row_src, int nt, int ks, int kw, int RS,
                                                 int wave, int nwaves) {
  const int lane = threadIdx.x & 63;
  const int pieces = kw >> 3;
  const int segs = (pieces + 63) >> 6;
  const int nseg = nt * segs;
  for (int s = wave; s < nseg; s += nwaves) {
    const int m = s / segs, sg = s - m * segs;
    const int p = sg * 64 + lane;
    if (p < pieces) lds_dma16(row_src(m) + ks + 8 * p, xs + (size_t)m * RS + sg * 512);
  }
}

// Sum over aligned groups of GP = 4, 8 or 16 lanes by a butterfly of DPP
// lane moves (register moves, no LDS round trips): partners at distance 1
// and 2 (quad permutations), then the other quad of each 8 (half-row mirror),
// then the other 8 of each 16 (row mirror).  After every step all lanes of a
// block hold the same bits (own + partner, and fp32 addition commutes), so
// the result is that of the xor butterfly with distances 1, 2, 4, 8.
template <int GP>
__device__ __forceinline__ float lane_group_sum(float v) {
  static_assert(GP == 4 || GP == 8 || GP == 16, "DPP rows hold 16 lanes");
  v += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0xb1, 0xf, 0xf, false));    // [1,0,3,2]
  v += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x4e, 0xf, 0xf, false));    // [2,3,0,1]
  if constexpr (GP >= 8)
    v += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x141, 0xf, 0xf, false));  // half mirror
  if constexpr (GP >= 16)
    v += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x140, 0xf, 0xf, false));  // mirror
  return v;
}

// GP = G/8: the lanes of a group (each lane holds 8 columns).
template <bool F16, int GP>
__device__ __forceinline__ void stage_rows_sums(const uint16_t* xs, float* sxs, int nt, int rows, int kw, int RS,
                                                int wave, int nwaves) {
  const int lane = threadIdx.x & 63;
  const int pieces = kw >> 3;
  const int segs = (pieces + 63) >> 6;
  const int nseg = nt * segs;
  for (int s = wave; s < nseg; s += nwaves) {
    const int m = s / segs, sg = s - m * segs;
    const int p = sg * 64 + lane;
    float sum = 0.0f;
    if (p < pieces) sum = sum8<F16>(*reinterpret_cast<const u32x4*>(xs + (size_t)m * RS + 8 * p));
    sum = lane_group_sum<GP>(sum);
    if (p < pieces && (p % GP) == 0) sxs[(p / GP) * rows + m] = sum;
  }
  __syncthreads();
}

// Rows computed piece by piece (8 columns, 16 bytes) by src(m, k); the group
// sums are those of the computed values.  Waves as for stage_rows.
template <bool F16, int GP, typename PieceFn>
__device__ __forceinline__ void stage_pieces(uint16_t* xs, float* sxs, PieceFn src, int nt, int rows,
                                             int ks, int kw, int RS, int wave, int nwaves) {
  const int lane = threadIdx.x & 63;
  const int pieces = kw >> 3;
  const int total = nt * pieces;
  for (int base = wave * 64; base < total; base += nwaves * 64) {
    const int idx = base + lane;
    const bool valid = idx < total;
    int m = 0, p = 0;
    float sum = 0.0f;
    if (valid) {
      m = idx / pieces;
      p = idx - m * pieces;
      const u32x4 v = src(m, ks + 8 * p);
      *reinterpret_cast<u32x4*>(xs + (size_t)m * RS + 8 * p) = v;
      sum = sum8<F16>(v);
    }
    sum = lane_group_sum<GP>(sum);
    if (valid && (p % GP) == 0) sxs[(p / GP) * rows + m] = sum;
  }
  __syncthreads();
}

template <int BITS, int NT, int GPC, bool F16>
__device__ __forceinline__ void compute_chunk(const uint32_t (&w)[2][BITS],
                                              const uint32_t (&s)[2][GPC], f32x4 (&acc)[2][NT],
                                              f32x4 (&tot)[2][NT], const uint16_t* const (&arow)[NT],
                                              const float* sxs, int lc, int lane, uint32_t magic) {
  constexpr int SPG = 4 / GPC;   // MFMA steps per quantization group
  constexpr int rows = 16 * NT;
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    const u32x4 b0 = b_operand<BITS, F16>(w[0], u, magic);
    const u32x4 b1 = b_operand<BITS, F16>(w[1], u, magic);
    const int kk = lc * kTileCols + 32 * u;
    const bool first = u % SPG == 0;     // first MFMA step of a group
    const f32x4 zero = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
    for (int tb = 0; tb < NT; ++tb) {
      const u32x4 a = *reinterpret_cast<const u32x4*>(arow[tb] + kk);
      acc[0][tb] = mfma16<F16>(a, b0, first ? zero : acc[0][tb]);
      acc[1][tb] = mfma16<F16>(a, b1, first ? zero : acc[1][tb]);
    }
    if ((u + 1) % SPG == 0) {
      const int q = (u + 1) / SPG - 1;
      const int gl = lc * GPC + q;
#pragma unroll
      for (int tb = 0; tb < NT; ++tb) {
        const float* sxp = sxs + gl * rows + tb * 16 + 4 * (lane >> 4);
        group_end<BITS>(acc[0][tb], tot[0][tb], s[0][q], sxp);
        group_end<BITS>(acc[1][tb], tot[1][tb], s[1][q], sxp);
      }
    }
    // steps stay in order: hoisting the B operands of later steps ahead of
    // their MFMAs runs the 32-token kernels out of registers (spills)
    __builtin_amdgcn_sched_barrier(0);
  }
}

}  // namespace mc
