// mc_device.hpp -- device-side helpers shared by the gfx950 kernels of the
// MC expert path: number formats, the packed-code layout and launch-argument
// structs.  Internal to the library.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/mc_moe.h"

namespace mc {

typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8;
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float f32x4;
typedef __attribute__((__vector_size__(4 * sizeof(uint32_t)))) uint32_t u32x4;

constexpr int kTileRows = 16;    // rows of one packed tile (MFMA N)
constexpr int kTileCols = 128;   // reduction columns of one packed tile (4 MFMA K-steps)
constexpr int kWave = 64;

// Index of the calling wavefront in its workgroup, as a wave-uniform (scalar) value.
__device__ __forceinline__ int wave_id() { return __builtin_amdgcn_readfirstlane(threadIdx.x >> 6); }

// ---------------------------------------------------------------- formats --

__device__ __forceinline__ float half_bits_to_float(uint32_t h) {
  _Float16 v;
  uint16_t b = (uint16_t)h;
  __builtin_memcpy(&v, &b, 2);
  return (float)v;
}

// Round to nearest even fp16; saturate to +-65504 instead of infinity.
__device__ __forceinline__ uint16_t float_to_half_sat(float f) {
  _Float16 v = (_Float16)f;
  uint16_t b;
  __builtin_memcpy(&b, &v, 2);
  if ((b & 0x7fffu) == 0x7c00u) b = (uint16_t)((b & 0x8000u) | 0x7bffu);
  return b;
}

__device__ __forceinline__ float bf16_bits_to_float(uint32_t h) {
  return __uint_as_float(h << 16);
}

// Round to nearest even bfloat16 (finite inputs).
__device__ __forceinline__ uint16_t float_to_bf16(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7fffu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

// fp16 bits of the single round-to-nearest-even rounding of a double.
// Rounds to fp32 with round-to-odd first (24 >= 11 + 2 bits, so the second
// rounding cannot create a double-rounding error: Boldo & Melquiond,
// "Emulation of FMA and correctly rounded sums: proved algorithms using
// rounding to odd", IEEE TC 2008), then to fp16 with round-to-nearest-even.
__device__ __forceinline__ uint16_t double_to_half_rne(double v) {
  float f = (float)v;
  if ((double)f != v) {
    uint32_t b = __float_as_uint(f);
    if (fabs((double)f) > fabs(v)) b -= 1u;   // step the magnitude toward zero
    b |= 1u;                                  // sticky odd bit
    f = __uint_as_float(b);
  }
  _Float16 h = (_Float16)f;
  uint16_t r;
  __builtin_memcpy(&r, &h, 2);
  return r;
}

// bfloat16 bits of the single round-to-nearest-even rounding of a double
// (finite): round to fp32 with round-to-odd first (24 >= 8 + 2 bits, so the
// second rounding is correct, by the same argument as double_to_half_rne).
__device__ __forceinline__ uint16_t double_to_bf16_rne(double v) {
  float f = (float)v;
  if ((double)f != v) {
    uint32_t b = __float_as_uint(f);
    if (fabs((double)f) > fabs(v)) b -= 1u;
    b |= 1u;
    f = __uint_as_float(b);
  }
  return float_to_bf16(f);
}

// ------------------------------------------------------- memory helpers --

// s_waitcnt vmcnt(n) (expcnt and lgkmcnt left alone).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

// Direct-to-LDS 16-byte load: lane l reads 16 bytes at src (its own address)
// and the wave writes them to dst + 16*l (dst is wave-uniform).  Counted by
// vmcnt; lanes outside EXEC neither read nor write.
__device__ __forceinline__ void lds_dma16(const void* src, void* dst) {
  __builtin_amdgcn_global_load_lds((const __attribute__((address_space(1))) void*)src,
                                   (__attribute__((address_space(3))) void*)dst, 16, 0, 0);
}

// ------------------------------------------------------------------ layout --
// Lane l of a 16x128 tile holds, for MFMA step u (32 columns) and register v
// (0..3), the codes of columns 32u + 8*(l/16) + 2v (low half) and +1 (high
// half) of row l%16: "pair" i = 4u + v.  extract_pair returns that pair as
// two 16-bit lanes holding the code in bits 0..2 with `magic` OR-ed in
// (0x4300 = bf16 128.0: the lane then holds the bf16 value 128 + code).

template <int BITS>
__device__ __forceinline__ uint32_t extract_pair(const uint32_t* w, int i, uint32_t magic2) {
  if constexpr (BITS == 1) {
    return ((w[0] >> i) & 0x00010001u) | magic2;
  } else if constexpr (BITS == 2) {
    return ((w[i >> 3] >> (2 * (i & 7))) & 0x00030003u) | magic2;
  } else {
    if (i < 15) {
      const int wi = i / 5, f = i - 5 * wi;
      return ((w[wi] >> (3 * f)) & 0x00070007u) | magic2;
    }
    return ((w[0] >> 15) & 0x00010001u) | ((w[1] >> 14) & 0x00020002u) |
           ((w[2] >> 13) & 0x00040004u) | magic2;
  }
}

// MFMA operand pair with the codes at the top of the mantissa: each 16-bit
// half is magic2's half (1.0) with code q in bits POS .. POS+BITS-1, i.e. the
// value 1 + q * 2^-BITS when POS + BITS is the format's mantissa width.  The
// products of a group then sum to S + 2^-BITS * sum(q * a) with S = sum(a), so
// the fp32 accumulators stay near the size of the activations.
template <int BITS, int POS>
__device__ __forceinline__ uint32_t code_pair(const uint32_t* w, int i, uint32_t magic2) {
  constexpr uint32_t kMask = (((1u << BITS) - 1u) << POS) * 0x00010001u;
  // moves bit `src` of each half to bit POS (one shift once i is a constant)
  auto mv = [](uint32_t x, int src) -> uint32_t { return src >= POS ? x >> (src - POS) : x << (POS - src); };
  if constexpr (BITS == 1) {
    return (mv(w[0], i) & kMask) | magic2;
  } else if constexpr (BITS == 2) {
    return (mv(w[i >> 3], 2 * (i & 7)) & kMask) | magic2;
  } else {
    if (i < 15) {
      const int wi = i / 5, f = i - 5 * wi;
      return (mv(w[wi], 3 * f) & kMask) | magic2;
    }
    constexpr uint32_t b0 = 0x00010001u << POS;
    return (mv(w[0], 15) & b0) | (mv(w[1], 14) & (b0 << 1)) | (mv(w[2], 13) & (b0 << 2)) | magic2;
  }
}

// Code of pair i, half h (for the export kernels).
template <int BITS>
__device__ __forceinline__ int extract_code(const uint32_t* w, int i, int h) {
  return (int)((extract_pair<BITS>(w, i, 0u) >> (16 * h)) & 7u);
}

// --------------------------------------------------------------- arguments --

// Lane `src`'s value of v, as a wave-uniform value (src must be uniform).
__device__ __forceinline__ double readlane_f64(double v, int src) {
  const unsigned long long b = __double_as_longlong(v);
  const uint32_t lo = __builtin_amdgcn_readlane((uint32_t)b, src);
  const uint32_t hi = __builtin_amdgcn_readlane((uint32_t)(b >> 32), src);
  return __longlong_as_double(((long long)hi << 32) | lo);
}

// ------------------------------------------------------------- quantizer --
// Sec. 3.1 group parameters from the group's fp32 min and max, as one
// scale/zero word (s16 low, z16 high), L = 2^b - 1:
//   s = fp16(fp32(max - min) / L) (1.0 if it rounds to zero), z = fp16(-min / s).
__device__ __forceinline__ uint32_t group_sz_word(float mn, float mx, int b) {
  const float Lf = (float)((1 << b) - 1);
  const float s32 = (mx - mn) / Lf;                 // IEEE fp32 division
  uint16_t s16 = float_to_half_sat(s32);
  if ((s16 & 0x7fffu) == 0) s16 = 0x3c00;           // scale 0 -> 1.0
  const float z32 = -mn / half_bits_to_float(s16);
  uint16_t z16 = float_to_half_sat(z32);
  if (z16 == 0x8000u) z16 = 0;                      // -0 -> +0
  return (uint32_t)s16 | ((uint32_t)z16 << 16);
}

// Code of w under scale s and zero z (fp16 values widened): the number of
// level midpoints s*(j + 1/2 - z) below w, moved to the even neighbour when w
// sits exactly on a midpoint.  Each midpoint is exact in fp64 (j + 1/2 - z
// needs <= 41 bits, times the 11-bit s <= 52).
__device__ __forceinline__ int nearest_code(float w, double s, double z, int L) {
  const double wd = (double)w;
  int below = 0;
  for (int j = 0; j < L; ++j) below += (s * (((double)j + 0.5) - z) < wd) ? 1 : 0;
  if (below < L && (below & 1) && s * (((double)below + 0.5) - z) == wd) ++below;
  return below;
}

// Places one code into a lane's b packed words: code pair i (0..15) of the
// lane's 32 codes, half h (0: first, 1: second of the pair).
__device__ __forceinline__ void place_code(uint32_t (&w)[3], uint32_t code, int i, int h, int b) {
  if (b == 1) {
    w[0] |= code << (16 * h + i);
  } else if (b == 2) {
    w[i >> 3] |= code << (16 * h + 2 * (i & 7));
  } else if (i < 15) {
    w[i / 5] |= code << (16 * h + 3 * (i % 5));
  } else {
    for (int p = 0; p < 3; ++p) w[p] |= ((code >> p) & 1u) << (16 * h + 15);
  }
}

struct LayerArgs {
  const uint32_t* words;
  const uint32_t* sz;
  int E, d, ffn, G;
  uint16_t cum_bits[MC_MAX_EXPERTS + 1];   // prefix sums of the expert widths
  uint32_t sign_mask[MC_MAX_EXPERTS / 32]; // bit e: expert e is sign-binarized (1 bit)
};

__device__ __forceinline__ bool expert_is_sign(const LayerArgs& L, int e) {
  return (L.sign_mask[e >> 5] >> (e & 31)) & 1u;
}

// Word offset of matrix m (0 gate, 1 up, 2 down) of expert e.
__device__ __forceinline__ size_t layer_word_offset(const LayerArgs& L, int e, int m) {
  const size_t per_bit = (size_t)L.d * (size_t)L.ffn / 32;
  const int b = L.cum_bits[e + 1] - L.cum_bits[e];
  return (3 * (size_t)L.cum_bits[e] + (size_t)m * b) * per_bit;
}

__device__ __forceinline__ size_t layer_sz_offset(const LayerArgs& L, int e, int m) {
  return (3 * (size_t)e + m) * ((size_t)L.d * (size_t)L.ffn / L.G);
}

// ------------------------------------------------ routing-derived indices --
// Every index the forward kernels derive from the routing buffers goes
// through these helpers, so that inconsistent routing (a caller's garbage,
// or buffers a routing call never filled) gives wrong values but never an
// access outside a buffer.  They are host-callable too: a CPU audit feeds
// them garbage and checks every derived index against its buffer.

// Kept-pair range [begin, begin + count) of expert e from the routing counts
// and offsets, or an empty range when they are inconsistent with P = T*k
// kept-pair slots, so that no index derived from them leaves its buffer.
__host__ __device__ __forceinline__ void expert_range(const int32_t* counts, const int32_t* offsets, int e, int P,
                                                      int& begin, int& count) {
  int c = counts[e], b = offsets[e];
  if (c < 0 || b < 0 || c > P || b > P - c) c = b = 0;
  begin = b;
  count = c;
}

// The same range from the offsets alone (count = offsets[e+1] - offsets[e]).
__host__ __device__ __forceinline__ void expert_range_offsets(const int32_t* offsets, int e, int P, int& begin,
                                                              int& count) {
  int b = offsets[e], c = offsets[e + 1] - b;
  if (c < 0 || b < 0 || c > P || b > P - c) c = b = 0;
  begin = b;
  count = c;
}

// A token index from the routing lists, clamped into [0, T).
__host__ __device__ __forceinline__ int clamp_token(int t, int T) { return t < 0 ? 0 : (t >= T ? T - 1 : t); }

// Pairs [pbase, pbase + nt) of block j (blocks of `block` pairs) of an expert
// whose kept pairs are [begin, begin + count): nt <= 0 when the block is empty.
__host__ __device__ __forceinline__ void pair_block(int begin, int count, int j, int block, int& pbase, int& nt) {
  pbase = begin + block * j;
  nt = (count - block * j) < block ? (count - block * j) : block;
}

// A kept-pair position of the per-token table (pair_pos), or -1 when it is
// outside [0, P) (the combine then skips that rank).
__host__ __device__ __forceinline__ int checked_pos(int pos, int P) { return (pos < 0 || pos >= P) ? -1 : pos; }

// An expert's count as the prefill set-up takes it: counts outside [0, P] are 0.
__host__ __device__ __forceinline__ int checked_count(int c, int P) { return (c < 0 || c > P) ? 0 : c; }

}  // namespace mc
