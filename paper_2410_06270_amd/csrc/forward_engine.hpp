// forward_engine.hpp -- Eq. 1 over packed SwiGLU experts (dequantization in registers).
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
// they are staged.
//
// Kernels (all on the caller's stream, no host synchronisation; experts with
// no kept token exit at once because the counts are read on the device):
//   gateup_kernel  grid (ffn/128, E, chunks x d-splits): 8 waves x 16 rows of
//                  gate and up, up to 16*NTMAX (<= 32) tokens of one expert per chunk
//                  -> h (fp16), or fp32 gate/up partials when d is split;
//   down_kernel    grid (d/256, E, chunks*S): 8 waves x 32 rows, split-K over
//                  ffn -> fp32 partials;
//   combine_kernel grid (d/1024, T): y = bf16(sum_r w_r sum_s partial), fixed
//                  order, so the result is deterministic.
#pragma once

#include "mc_internal.hpp"

namespace mc {

constexpr int kRowPad = 8;                    // elements of padding per slab row
constexpr int kSxBytes = 4 * 1024;            // group sums of the staged slab (LDS)

constexpr int kWavesPerWg = 8;                // workgroups of 512 threads share one slab
constexpr int kMaxNsplit = 8;                 // largest split of the down reduction
constexpr int kMaxKsplit = 2;                 // largest split of the gate/up reduction
// LDS for the staged activation slab.  A workgroup holds at most 32 tokens
// of one expert (an expert with more gets one workgroup per 32 of its
// tokens); the kernels are held to 128 registers (four waves per SIMD) and
// two workgroups of 75.5 KB share a CU.
constexpr int kXsBytes = 75 * 1024 + 512;
constexpr int kLdsPerCu = 160 * 1024;
static_assert(2 * (kXsBytes + 4 * 1024 + 32 * 4) <= kLdsPerCu, "two workgroups per CU");
// The kernels of 32-token blocks run one workgroup of 16 waves per CU
// instead (the same 16 waves): the gate/up slab then takes all of d = 4096
// for up to 16 tokens and half of it for 32, against two and four slabs in
// 75.5 KB, the down slab a whole ffn split, and each slab change drains the
// weight ring.
constexpr int kGuWaves32 = 16;
constexpr int kGuXsBytes32 = 146 * 1024;
static_assert(kGuXsBytes32 + 4 * 1024 + 32 * 4 + 512 <= kLdsPerCu, "one 16-wave gate/up workgroup per CU");
// Chunks (16 rows x 128 columns of codes) kept in flight per stream.  The slab
// is a multiple of this many chunks, so it is smaller where the slab rows are
// many (token blocks) or the registers few (groups per chunk).
__host__ __device__ constexpr int prefetch_depth(int ntb, int gpc) {
  return (ntb >= 3 || gpc >= 4) ? 2 : 4;
}
// Smallest slab (one ring of chunks) of the worst case of each token-block
// count must fit its LDS budget: (tokens + zero row) x (columns + pad) x 2 bytes.
constexpr int slab_floor_bytes(int ntb) {
  return (16 * ntb + 1) * (prefetch_depth(ntb, 1) * kTileCols + kRowPad) * 2;
}
static_assert(slab_floor_bytes(1) <= kXsBytes, "LDS budget (<= 16 tokens)");
static_assert(slab_floor_bytes(2) <= kXsBytes, "LDS budget (<= 32 tokens)");
static_assert(slab_floor_bytes(2) <= kGuXsBytes32, "LDS budget (<= 32 tokens, 16 waves)");
// Group sums: 16*ntb rows x (slab / G) groups x 4 bytes; the slab is capped by
// kSxBytes, which must allow at least one ring of chunks at G = 32.
static_assert((kSxBytes / (4 * 32)) * 32 >= 4 * kTileCols, "group-sum budget (32 tokens)");

__device__ __forceinline__ float silu(float a) { return a / (1.0f + expf(-a)); }

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

// Two weight streams per wave (gate and up rows of one block, or two row
// blocks of down) share every activation fragment.  Each stream reads through
// a buffer resource that covers exactly its chunks [c_begin, c_end): the chunk
// offset is wave-uniform and the lane offset is one VGPR.
typedef __amdgpu_buffer_rsrc_t rsrc_t;
constexpr int kRsrcWord3 = 0x00020000;   // raw 32-bit buffer (gfx9 family)

__device__ __forceinline__ rsrc_t make_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes, kRsrcWord3);
}

struct Streams {
  rsrc_t w[2];        // packed words of chunks [c_begin, c_end) of the stream's row block
  rsrc_t s[2];        // scale/zero words of the same groups
  uint32_t lane_w;    // byte offset of this lane's words inside a chunk
  uint32_t lane_s;    // byte offset of this lane's scale/zero word inside a group
};

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

// Loads chunk min(cc, last) (relative to c_begin) so that the ring refill is
// unconditional (no control flow around the in-flight registers); refills
// past the end re-read the last chunk and are never consumed.
template <int BITS, int GPC>
__device__ __forceinline__ void load_chunk(uint32_t (&w)[2][BITS], uint32_t (&s)[2][GPC],
                                           const Streams& st, int cc, int last) {
  const uint32_t c = (uint32_t)(cc < last ? cc : last);
  const uint32_t ow = st.lane_w + c * (64u * BITS * 4u);
#pragma unroll
  for (int j = 0; j < 2; ++j) load_words<BITS>(w[j], st.w[j], ow);
#pragma unroll
  for (int q = 0; q < GPC; ++q) {
    const uint32_t os = st.lane_s + (c * GPC + q) * 64u;
#pragma unroll
    for (int j = 0; j < 2; ++j) s[j][q] = __builtin_amdgcn_raw_buffer_load_b32(st.s[j], os, 0, 0);
  }
}

// ------------------------------------------------------------------ slabs --
// A slab holds columns [ks, ks + kw) of the nt token rows (row stride RS =
// slab width + kRowPad elements; a zero row follows for padding tokens) and
// the sums of each group of G columns, sxs[group][rows].

// Rows that are plain copies of global memory (x; h when the gate/up reduction
// was not split), row m starting at row_src(m): direct-to-LDS 16-byte loads,
// 64 consecutive pieces of a row per wave instruction, so every wave has all
// its loads in flight at once.  With SUMS each wave then forms the group sums
// of its own row segments (a segment is 512 columns, a whole number of groups;
// the G/8 lanes of a group add in a fixed butterfly order); otherwise the sums
// are read from sum_src(m, g) for the slab's groups g.
template <bool F16, bool SUMS, typename RowFn, typename SumFn>
__device__ __forceinline__ void stage_rows(uint16_t* xs, float* sxs, RowFn row_src, SumFn sum_src,
                                           int nt, int rows, int ks, int kw, int RS, int G) {
  const int lane = threadIdx.x & 63, wave = wave_id(), nwaves = blockDim.x >> 6;
  const int pieces = kw >> 3;
  const int segs = (pieces + 63) >> 6;
  const int nseg = nt * segs;
  for (int s = wave; s < nseg; s += nwaves) {
    const int m = s / segs, sg = s - m * segs;
    const int p = sg * 64 + lane;
    if (p < pieces) lds_dma16(row_src(m) + ks + 8 * p, xs + (size_t)m * RS + sg * 512);
  }
  if constexpr (!SUMS) {
    const int ngs = kw / G;
    for (int i = threadIdx.x; i < nt * ngs; i += blockDim.x) {
      const int m = i / ngs, g = i - m * ngs;
      sxs[g * rows + m] = sum_src(m, g);
    }
  }
  wait_vmcnt<0>();
  asm volatile("" ::: "memory");
  if constexpr (SUMS) {
    const int gp = G >> 3;
    for (int s = wave; s < nseg; s += nwaves) {
      const int m = s / segs, sg = s - m * segs;
      const int p = sg * 64 + lane;
      float sum = 0.0f;
      if (p < pieces) sum = sum8<F16>(*reinterpret_cast<const u32x4*>(xs + (size_t)m * RS + 8 * p));
      for (int off = 1; off < gp; off <<= 1) sum += __shfl_xor(sum, off);
      if (p < pieces && (p % gp) == 0) sxs[(p / gp) * rows + m] = sum;
    }
  }
  __syncthreads();
}

// Rows computed piece by piece (8 columns, 16 bytes) by src(m, k); the group
// sums are those of the computed values.
template <bool F16, typename PieceFn>
__device__ __forceinline__ void stage_pieces(uint16_t* xs, float* sxs, PieceFn src, int nt, int rows,
                                             int ks, int kw, int RS, int G) {
  const int lane = threadIdx.x & 63;
  const int pieces = kw >> 3;
  const int total = nt * pieces;
  const int gp = G >> 3;
  for (int base = wave_id() * 64; base < total; base += blockDim.x) {
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
    for (int off = 1; off < gp; off <<= 1) sum += __shfl_xor(sum, off);
    if (valid && (p % gp) == 0) sxs[(p / gp) * rows + m] = sum;
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

// Stream chunks [c_begin, c_end) of two weight streams against the staged
// activations of nt (<= 16*NT) tokens; a ring of D chunks of packed words and
// scale/zero words stays in flight in registers across chunk and slab
// boundaries.  stage(xs, sxs, rows, ks, kw, RS) fills a slab.
template <int BITS, int NT, int GPC, bool F16, typename StageFn>
__device__ __forceinline__ void stream_pair(const Streams& sp, int c_begin, int c_end,
                                            StageFn stage, int nt, int G,
                                            uint16_t* xs, float* sxs, int xs_elems,
                                            f32x4 (&tot)[2][NT]) {
  constexpr int D = prefetch_depth(NT, GPC);
  constexpr int rows = 16 * NT;
  const int lane = threadIdx.x & 63;
  int ks = xs_elems / (nt + 1) - kRowPad;   // + one zero row for padding tokens
  const int ks_sx = (kSxBytes / (4 * rows)) * G;
  ks = ks < ks_sx ? ks : ks_sx;
  const int unit = D * kTileCols;
  ks = (ks / unit) * unit;
  if (ks < unit) ks = unit;               // the host's LDS budget makes this fit
  const int slab_chunks = ks / kTileCols;
  const int RS = ks + kRowPad;
  const int last = c_end - c_begin - 1;     // ring chunk indices are relative to c_begin

  f32x4 acc[2][NT];
#pragma unroll
  for (int st = 0; st < 2; ++st)
#pragma unroll
    for (int tb = 0; tb < NT; ++tb)
#pragma unroll
      for (int i = 0; i < 4; ++i) acc[st][tb][i] = 0.0f;

  uint32_t wr[D][2][BITS];
  uint32_t sr[D][2][GPC];
#pragma unroll
  for (int j = 0; j < D; ++j) load_chunk<BITS, GPC>(wr[j], sr[j], sp, j, last);

  // zero row after the staged rows; lanes of tokens >= nt read it
  uint16_t* zrow = xs + (size_t)nt * RS;
  for (int i = threadIdx.x; i < RS / 8; i += blockDim.x)
    *reinterpret_cast<u32x4*>(zrow + 8 * i) = u32x4{0u, 0u, 0u, 0u};
  const uint16_t* arow[NT];
#pragma unroll
  for (int tb = 0; tb < NT; ++tb) {
    const int m = tb * 16 + (lane & 15);
    arow[tb] = (m < nt ? xs + (size_t)m * RS : zrow) + 8 * (lane >> 4);
  }
  const uint32_t magic = vgpr_constant(Fmt<F16>::kMagic2);

  for (int c0 = c_begin; c0 < c_end; c0 += slab_chunks) {
    const int c1 = (c0 + slab_chunks) < c_end ? (c0 + slab_chunks) : c_end;
    __syncthreads();
    stage(xs, sxs, rows, c0 * kTileCols, (c1 - c0) * kTileCols, RS);
    int c = c0;
    for (; c + D <= c1; c += D) {
#pragma unroll
      for (int j = 0; j < D; ++j) {
        compute_chunk<BITS, NT, GPC, F16>(wr[j], sr[j], acc, tot, arow, sxs, c + j - c0, lane, magic);
        load_chunk<BITS, GPC>(wr[j], sr[j], sp, c + j + D - c_begin, last);
        // the refill issues here, not later: left to itself the scheduler
        // sinks all refills of the unrolled ring to the end of the loop body,
        // behind a wait for every load in flight, which drains the ring
        __builtin_amdgcn_sched_barrier(0);
      }
    }
#pragma unroll
    for (int j = 0; j < D; ++j) {        // remainder of the last slab
      if (c + j < c1)
        compute_chunk<BITS, NT, GPC, F16>(wr[j], sr[j], acc, tot, arow, sxs, c + j - c0, lane, magic);
    }
  }
}

// Runs the streams for one expert width with the number of 16-token blocks
// fixed at compile time (no token-block branches inside the loop).  NTMAX is
// the largest block count a launch can see; tot[st][tb] for blocks beyond the
// workgroup's count are left as they were.
template <int BITS, int GPC, int NTMAX, bool F16, typename StageFn>
__device__ __forceinline__ void run_width(const Streams& sp, int c_begin, int c_end, StageFn stage,
                                          int nt, int G, uint16_t* xs, float* sxs, int xs_elems,
                                          f32x4 (&tot)[2][NTMAX]) {
  const int ntb = (nt + 15) >> 4;
  if (NTMAX == 1 || ntb == 1) {
    f32x4 t[2][1];
    t[0][0] = tot[0][0];
    t[1][0] = tot[1][0];
    stream_pair<BITS, 1, GPC, F16>(sp, c_begin, c_end, stage, nt, G, xs, sxs, xs_elems, t);
    tot[0][0] = t[0][0];
    tot[1][0] = t[1][0];
  } else if (NTMAX == 2 || ntb == 2) {
    constexpr int N = NTMAX < 2 ? NTMAX : 2;
    f32x4 t[2][N];
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int b = 0; b < N; ++b) t[j][b] = tot[j][b];
    stream_pair<BITS, N, GPC, F16>(sp, c_begin, c_end, stage, nt, G, xs, sxs, xs_elems, t);
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int b = 0; b < N; ++b) tot[j][b] = t[j][b];
  } else {
    stream_pair<BITS, NTMAX, GPC, F16>(sp, c_begin, c_end, stage, nt, G, xs, sxs, xs_elems, tot);
  }
}

// Launchers (one translation unit per kernel and group size).
// Hidden activations between the two kernels: h = fp16(silu(gate) * up), or
// (small batches, gate/up split over d) fp32 partial sums of gate and up per
// split.
struct Hidden {
  uint16_t* h;           // [P][ffn] fp16
  float* gu_part;        // [ksplit][2][P][ffn] when ksplit > 1
  int P;                 // T * k
  int T;
  int ksplit;
};

template <int GPC>
hipError_t launch_gateup(const uint16_t* x, const LayerArgs& L, const mc_routing& r,
                         const Hidden& h, int ntmax, int xs_bytes, hipStream_t stream);
template <int GPC>
hipError_t launch_down(const Hidden& h, const LayerArgs& L, const mc_routing& r, int nsplit,
                       float* partial, size_t part_stride, int ntmax, int xs_bytes,
                       hipStream_t stream);

}  // namespace mc
