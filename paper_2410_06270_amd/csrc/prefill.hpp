// prefill.hpp -- grouped GEMMs of the expert forward (Eq. 1) for batches in
// which each active expert sees many tokens: per expert e, with X_e its kept
// tokens (the CSR list of the routing step),
//   H_e = silu(X_e W_gate^T) * (X_e W_up^T)        (gate/up kernel)
//   Y_e = H_e W_down^T                              (down kernel, fp32 partials)
// and y_t = sum_r w_r Y[pos(t, r)] by the combine kernel of the decode path.
//
// The weights are never rounded.  As in the decode kernels, the codes enter
// the MFMA as the exact values 1 + q 2^-b (code in the top b mantissa bits of
// 1.0), and the scale and zero of each group are applied to the fp32 group sum:
//   sum_{k in g} x_k s (q_k - z) = s 2^b * acc_g - s 2^b (1 + z 2^-b) * S_g,
//   acc_g = sum_k x_k (1 + q_k 2^-b) (MFMA),  S_g = sum_{k in g} x_k.
// The first term costs one fp32 fma per output and group; the second, summed
// over the groups, is a product of the token-by-group sums S_g and the
// group-by-row coefficients, taken in fp32 on v_mfma_f32_32x32x2_f32 (two
// groups per MFMA) into the same totals.
//  * gate/up: x stays bf16 (exact), codes in bf16, v_mfma_f32_32x32x16_bf16;
//  * down: h is rounded once to fp16 (the only rounding on the path besides
//    fp32 accumulation), codes in fp16, v_mfma_f32_32x32x16_f16.
// Activations are held in a fragment layout: a fragment is 32 rows x 16
// columns (1 KB), stored in the order the MFMA A operand takes it (lane l:
// row l%32, columns 8*(l/32) .. +8); a wave stages a fragment into LDS with one
// direct-to-LDS 16-byte load per lane and reads it back with one
// conflict-free ds_read_b128.  Beside each operand lie its sums over every 32
// columns, [fragment row][32 rows][K/32], from which the group sums S_g are
// formed while staging.  Rows of each expert start at a fragment boundary;
// padding rows are zero.
//
// Workgroup: 8 waves (two per SIMD) on one m-tile of 128 tokens (four
// fragment rows); each wave computes all 128 tokens against one stream of 32
// weight rows (gate/up: waves 2r and 2r+1 take the same 32 ffn rows of gate
// and of up; down: 32 consecutive d rows), so that the codes a wave unpacks
// for one MFMA step feed four MFMAs.  The group accumulators and the running
// fp32 totals stay in registers; the reduction runs in 128-column chunks,
// staged through a ring of four LDS slots.
#pragma once

#include "forward_engine.hpp"

namespace mc {

typedef __bf16 bf16x8e __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr int kPfFragRows = 32;                    // rows of a fragment (MFMA M)
constexpr int kPfFragBytes = 1024;                 // 32 rows x 16 16-bit values
constexpr int kPfWaves = 8;
constexpr int kPfSlots = 4;                        // LDS ring: chunks c-1 .. c+2

struct PfCfg {
  static constexpr int kTiles = 4;                               // fragment rows per m-tile
  static constexpr int kTokens = kTiles * kPfFragRows;           // tokens per m-tile
  static constexpr int kFragBytes = kTiles * 8 * kPfFragBytes;   // A fragments of one chunk
  static constexpr int kSumBytes = 2048;                         // group sums: kTiles x <= 4 groups x 32 rows
  static constexpr int kStageBytes = kFragBytes + kSumBytes;
  static constexpr int kLdsBytes = kPfSlots * kStageBytes;
  static constexpr int kRowsGateUp = kPfWaves / 2 * 32;          // ffn rows per gate/up workgroup
  static constexpr int kRowsDown = kPfWaves * 32;                // d rows per down workgroup
  // every wave issues the same number of staging loads per chunk (counted waits)
  static constexpr int kFragLoadsPerWave = kTiles * 8 / kPfWaves;
  static_assert(kTiles * 8 % kPfWaves == 0, "fragments spread evenly over the waves");
  static_assert(kTiles * 4 * 32 * 4 <= kSumBytes, "group sums of a chunk");
  static_assert(kLdsBytes <= kLdsPerCu, "prefill stages fit the LDS of a CU");
  static_assert(kRowsGateUp % 128 == 0, "a gate/up workgroup covers whole groups of h columns");
  static_assert(kPfWaves * 2 * 16 * 64 * 4 + kTiles * 8 * kPfFragBytes <= kLdsBytes,
                "the exchanged totals and the h tile fit the ring");
};

// Expert-to-tile tables, written into the workspace by workgroup 0 of the
// preparation launch (prefill_prep_kernel).
struct PrefillTables {
  int32_t* ftile_base;   // [E+1] first fragment row of each expert
  int32_t* mt_e;         // [mt_max] expert of each m-tile
  int32_t* mt_j;         // [mt_max] m-tile index within its expert
  int32_t* mt_count;     // [1] m-tiles in use
  int f_max, mt_max;
  int T, P;              // tokens and kept-pair slots (T*k) of the routing
};

struct PrefillGemm {
  const uint16_t* a;     // fragment-tiled operand, K columns (bf16 x or fp16 h)
  const float* asum;     // [fragment row][K/G][32] sums of the operand over each group
  int K;                 // reduction length: d (gate/up) or ffn (down)
  int n_tiles;           // workgroup row tiles of the weight matrix
  int c_per_split;       // 128-column chunks per split of the reduction
  int nsplit;
  uint16_t* h;           // gate/up output: fragment-tiled fp16 h [.][ffn]
  float* hsum;           // gate/up output: [fragment row][ffn/G][32] group sums of the rounded h
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

// B operand of MFMA step u of one 64-column piece: 8 codes as 1 + q 2^-b.
template <int BITS, bool BF16>
__device__ __forceinline__ u32x4 pf_codes(const uint32_t (&w)[BITS], int u, uint32_t magic) {
  constexpr int POS = Fmt<!BF16>::template kPos<BITS>;
  return u32x4{code_pair<BITS, POS>(w, 4 * u + 0, magic), code_pair<BITS, POS>(w, 4 * u + 1, magic),
               code_pair<BITS, POS>(w, 4 * u + 2, magic), code_pair<BITS, POS>(w, 4 * u + 3, magic)};
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

// Stage chunk c straight into LDS: the A fragments of the kTiles fragment rows
// (rows past the m-tile's end read the padding rows of the buffer; their sums
// are dropped) and the group sums [tile][GPC][32].  Each wave issues
// kFragLoadsPerWave + 1 loads; the sums are split in two 1 KB halves, and
// waves loading the same half write identical bytes.
template <int GPC>
__device__ __forceinline__ void pf_stage(unsigned char* stage, const PrefillGemm& g, int f0, int c, int wave,
                                         int lane) {
  using S = PfCfg;
  const int ksteps = g.K / 16, ng = g.K * GPC / kTileCols;
#pragma unroll
  for (int i = 0; i < S::kFragLoadsPerWave; ++i) {
    const int q = wave + kPfWaves * i;
    const int mt = q >> 3, v = q & 7;
    lds_dma16(reinterpret_cast<const unsigned char*>(g.a) +
                  ((size_t)(f0 + mt) * ksteps + (size_t)c * 8 + v) * kPfFragBytes + lane * 16,
              stage + q * kPfFragBytes);
  }
  const int half = wave & 1;
  const int p = half * 64 + lane;                 // 16-byte piece of the sums area
  int t = p / (GPC * 8), rest = p - t * GPC * 8;
  if (t >= S::kTiles) { t = 0; rest = 0; }         // past the sums: any valid address
  const int q = rest >> 3, r4 = (rest & 7) * 4;
  lds_dma16(g.asum + ((size_t)(f0 + t) * ng + (size_t)c * GPC + q) * 32 + r4,
            stage + S::kFragBytes + half * 1024);
}

// Group epilogue: tot += s 2^b * acc_g (the scale of this lane's row, word
// sw).  The zero-point part of the group's term, -(s 2^b (1 + z 2^-b)) * S_g,
// goes to the correction (PfZero).
template <int BITS, int NT>
__device__ __forceinline__ void pf_epilogue(const f32x16 (&acc)[PfCfg::kTiles], uint32_t sw,
                                            f32x16 (&tot)[PfCfg::kTiles]) {
  const float sj = half_bits_to_float(sw & 0xffffu) * (float)(1 << BITS);
#pragma unroll
  for (int t = 0; t < NT; ++t)
#pragma unroll
    for (int i = 0; i < 16; ++i) tot[t][i] = fmaf(sj, acc[t][i], tot[t][i]);
}

// The zero-point correction, sum over groups g of -(s_g 2^b (1 + z_g 2^-b))
// * S_g (S_g the group sum of a token row), as a product [tokens x groups] .
// [groups x weight rows] on v_mfma_f32_32x32x2_f32, two groups per MFMA: the
// lanes of half h hold group g of each pair with g % 2 == h (A: S_g of token
// lane % 32 per fragment row; B: the coefficient of weight row lane % 32).
// Groups are numbered from the first of the loop's range; take() records one
// group's operands from the stage and its scale/zero word, and after each
// odd-numbered group the pair's MFMAs (one per live fragment row, NT) add
// into tot.
template <int NT>
struct PfZero {
  float a[PfCfg::kTiles];
  float b;
  template <int BITS, int GPC>
  __device__ __forceinline__ void take(const unsigned char* stage, int q, uint32_t sw, int rel, int lane,
                                       f32x16 (&tot)[PfCfg::kTiles]) {
    const bool mine = (rel & 1) == (lane >> 5);
    const float* ssum = reinterpret_cast<const float*>(stage + PfCfg::kFragBytes);
    const float sj = half_bits_to_float(sw & 0xffffu) * (float)(1 << BITS);
    const float cj = fmaf(half_bits_to_float(sw >> 16), 1.0f / (float)(1 << BITS), 1.0f);
#pragma unroll
    for (int t = 0; t < NT; ++t) {
      const float v = ssum[(t * GPC + q) * 32 + (lane & 31)];
      a[t] = mine ? v : a[t];
    }
    b = mine ? -(sj * cj) : b;
    if (rel & 1) flush(tot);
  }
  __device__ __forceinline__ void flush(f32x16 (&tot)[PfCfg::kTiles]) {
#pragma unroll
    for (int t = 0; t < NT; ++t) tot[t] = __builtin_amdgcn_mfma_f32_32x32x2f32(a[t], b, tot[t], 0, 0, 0);
  }
  // an odd number of groups leaves half a pair: its other half is zero
  __device__ __forceinline__ void finish(int ngroups, int lane, f32x16 (&tot)[PfCfg::kTiles]) {
    if (ngroups & 1) {
      if (lane >> 5) {
#pragma unroll
        for (int t = 0; t < NT; ++t) a[t] = 0.0f;
        b = 0.0f;
      }
      flush(tot);
    }
  }
};

// MFMAs of group q of the chunk in `stage` with the words `w`: per step the
// eight codes of this lane's row feed the MFMAs of the NT fragment rows that
// hold the expert's tokens (the m-tile's others are padding: skipped).  The
// A fragments of step v+1 are read while the MFMAs of step v run.
template <int BITS, int GPC, bool BF16, int NT>
__device__ __forceinline__ void pf_group(const unsigned char* stage, const uint32_t (&w)[2][BITS], int q, int lane,
                                         uint32_t magic, f32x16 (&acc)[PfCfg::kTiles]) {
  constexpr int KV = 8 / GPC;   // MFMA steps per group
  const unsigned char* arow = stage + lane * 16;
  u32x4 a[2][PfCfg::kTiles];
#pragma unroll
  for (int t = 0; t < NT; ++t) a[0][t] = *reinterpret_cast<const u32x4*>(arow + (t * 8 + q * KV) * kPfFragBytes);
#pragma unroll
  for (int vv = 0; vv < KV; ++vv) {
    const int v = q * KV + vv;
    if (vv + 1 < KV) {
#pragma unroll
      for (int t = 0; t < NT; ++t)
        a[(vv + 1) & 1][t] = *reinterpret_cast<const u32x4*>(arow + (t * 8 + v + 1) * kPfFragBytes);
    }
    const u32x4 b = pf_codes<BITS, BF16>(w[v & 1], v >> 1, magic);
#pragma unroll
    for (int t = 0; t < NT; ++t) {
      const f32x16 z = {};
      acc[t] = pf_mfma<BF16>(a[vv & 1][t], b, vv == 0 ? z : acc[t]);
    }
    // one step per scheduling region: left free, the scheduler ran each
    // fragment row's eight dependent MFMAs back to back, each behind its own
    // LDS read, instead of the four independent MFMAs of a step
    asm volatile("" ::: "memory");
    __builtin_amdgcn_sched_barrier(0);
  }
}

template <int BITS, int GPC, bool BF16, int NT>
__device__ __forceinline__ void pf_chunk_body(const unsigned char* __restrict__ cur,
                                              unsigned char* __restrict__ next, const PfStream& sp,
                                              const PrefillGemm& g, int f0, bool late, bool first, int c, int last,
                                              int rel0, int wave, int lane, const uint32_t (&w)[2][BITS],
                                              const uint32_t (&s)[GPC], uint32_t (&nw)[2][BITS],
                                              uint32_t (&ns)[GPC], uint32_t& ps, uint32_t magic, PfZero<NT>& zc,
                                              f32x16 (&acc)[PfCfg::kTiles], f32x16 (&tot)[PfCfg::kTiles]) {
  if (late && !first) pf_epilogue<BITS, NT>(acc, ps, tot);
  pf_load<BITS, GPC>(nw, ns, sp, c + 1 < last ? c + 1 : last);
  __builtin_amdgcn_sched_barrier(0);   // the words go out before the stage (counted waits)
  pf_stage<GPC>(next, g, f0, c + 2 < last ? c + 2 : last, wave, lane);
#pragma unroll
  for (int q = 0; q < GPC; ++q) {
    pf_group<BITS, GPC, BF16, NT>(cur, w, q, lane, magic, acc);
    if (q < GPC - 1 || !late) pf_epilogue<BITS, NT>(acc, s[q], tot);
    else ps = s[q];
    zc.template take<BITS, GPC>(cur, q, s[q], rel0 + q, lane, tot);
  }
}

// One chunk.  Wait for its stage, issue the words of chunk c+1 into `nw`/`ns`
// and stage c+2 (chunk indices clamped to the last one, so that every wave has
// the same loads in flight everywhere: at the top of a chunk only stage c+1
// may still be outstanding behind the words of c), then the MFMAs and group
// epilogues.  The two waves of a SIMD run half a phase apart: a "late" wave
// does the epilogue of the previous chunk's last group first (its acc, its
// scale word `ps` and its stage, kept by the fourth LDS slot) and defers its
// own last group's epilogue, so that one wave's epilogue overlaps the other's
// MFMAs.
template <int BITS, int GPC, bool BF16, int NT>
__device__ __forceinline__ void pf_chunk(const PfStream& sp, const PrefillGemm& g, int f0, bool late, bool first,
                                         int c, int last, int rel0, int slot, unsigned char* smem, int wave,
                                         int lane, const uint32_t (&w)[2][BITS], const uint32_t (&s)[GPC],
                                         uint32_t (&nw)[2][BITS], uint32_t (&ns)[GPC], uint32_t& ps, uint32_t magic,
                                         PfZero<NT>& zc, f32x16 (&acc)[PfCfg::kTiles], f32x16 (&tot)[PfCfg::kTiles]) {
  using S = PfCfg;
  // Stage c has landed in LDS once at most the loads issued after it (stage
  // c+1) are outstanding; the plain barrier then publishes it (a fenced
  // __syncthreads would also wait for stage c+1, which is still in flight).
  wait_vmcnt<S::kFragLoadsPerWave + 1>();
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
  const int slot2 = slot + 2 >= kPfSlots ? slot + 2 - kPfSlots : slot + 2;
  pf_chunk_body<BITS, GPC, BF16, NT>(smem + slot * S::kStageBytes, smem + slot2 * S::kStageBytes, sp, g, f0, late,
                                 first, c, last, rel0, wave, lane, w, s, nw, ns, ps, magic, zc, acc, tot);
}

// Chunks [c_begin, c_end) of the reduction, two per iteration so that the
// two register sets of weight words alternate without copies.
template <int BITS, int GPC, bool BF16, int NT>
__device__ __forceinline__ void pf_loop(const PfStream& sp, const PrefillGemm& g, int f0, bool late, int c_begin,
                                        int c_end, unsigned char* smem, int wave, int lane,
                                        f32x16 (&tot)[PfCfg::kTiles]) {
  using S = PfCfg;
  if (c_begin >= c_end) return;
  const uint32_t magic = vgpr_constant(Fmt<!BF16>::kMagic2);
  const int last = c_end - 1;
  uint32_t wa[2][BITS], sa[GPC], wb[2][BITS], sb[GPC], ps = 0u;
  f32x16 acc[S::kTiles];
  pf_load<BITS, GPC>(wa, sa, sp, c_begin);
  pf_stage<GPC>(smem, g, f0, c_begin, wave, lane);
  pf_stage<GPC>(smem + S::kStageBytes, g, f0, c_begin + 1 < last ? c_begin + 1 : last, wave, lane);
  PfZero<NT> zc{};
  int slot = 0;
  for (int it = 0, c = c_begin; c < c_end; ++it, c += 2) {
    const int rel0 = it * 2 * GPC;   // even: the parity of a group's number is known per call site
    pf_chunk<BITS, GPC, BF16, NT>(sp, g, f0, late, c == c_begin, c, last, rel0, slot, smem, wave, lane, wa, sa, wb, sb,
                              ps, magic, zc, acc, tot);
    slot = slot + 1 == kPfSlots ? 0 : slot + 1;
    if (c + 1 < c_end)
      pf_chunk<BITS, GPC, BF16, NT>(sp, g, f0, late, false, c + 1, last, rel0 + GPC, slot, smem, wave, lane, wb, sb, wa,
                                sa, ps, magic, zc, acc, tot);
    slot = slot + 1 == kPfSlots ? 0 : slot + 1;
  }
  if (late) pf_epilogue<BITS, NT>(acc, ps, tot);   // the late waves' deferred last epilogue
  zc.finish((c_end - c_begin) * GPC, lane, tot);
  wait_vmcnt<0>();   // the clamped re-reads of the last chunks land before LDS is reused
}

template <int GPC, bool BF16, int NT>
__device__ __forceinline__ void pf_loop_bits(int bits, const PfStream& sp, const PrefillGemm& g, int f0, bool late,
                                             int c_begin, int c_end, unsigned char* smem, int wave, int lane,
                                             f32x16 (&tot)[PfCfg::kTiles]) {
  if (bits == 1)
    pf_loop<1, GPC, BF16, NT>(sp, g, f0, late, c_begin, c_end, smem, wave, lane, tot);
  else if (bits == 2)
    pf_loop<2, GPC, BF16, NT>(sp, g, f0, late, c_begin, c_end, smem, wave, lane, tot);
  else
    pf_loop<3, GPC, BF16, NT>(sp, g, f0, late, c_begin, c_end, smem, wave, lane, tot);
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
  const int nmt = nf < S::kTiles ? nf : S::kTiles;   // fragment rows of this m-tile that hold the expert's rows
  const int lane = threadIdx.x & 63, wave = wave_id();
  const bool late = wave >= kPfWaves / 2;   // shares a SIMD with wave - 4: runs half a phase later
  const int ntiles = g.K / kTileCols;
  const int c_begin = split * g.c_per_split;
  const int c_end = (c_begin + g.c_per_split) < ntiles ? (c_begin + g.c_per_split) : ntiles;
  const int bits = L.cum_bits[e + 1] - L.cum_bits[e];

  // This wave's 32 weight rows.  ffn and d are multiples of 128, so a block of
  // 32 rows lies wholly inside or outside its matrix; the surplus waves of
  // the last down tile read the matrix's last rows (in bounds) and write nothing.
  const int rb = GATEUP ? wave >> 1 : wave;
  int row = nt * (GATEUP ? S::kRowsGateUp : S::kRowsDown) + 32 * rb;
  const bool row_valid = row < (GATEUP ? L.ffn : L.d);
  if (!row_valid) row = (GATEUP ? L.ffn : L.d) - 32;
  const PfStream sp = pf_stream(L, e, GATEUP ? (wave & 1) : 2, row, g.K, bits, lane);

  f32x16 tot[S::kTiles];
#pragma unroll
  for (int t = 0; t < S::kTiles; ++t)
#pragma unroll
    for (int i = 0; i < 16; ++i) tot[t][i] = 0.0f;

  // the MFMAs cover the fragment rows that hold the expert's tokens: one,
  // two, or all four (three run as four; their fourth row is padding)
  if (nmt == 1)
    pf_loop_bits<GPC, GATEUP, 1>(bits, sp, g, f0, late, c_begin, c_end, smem, wave, lane, tot);
  else if (nmt == 2)
    pf_loop_bits<GPC, GATEUP, 2>(bits, sp, g, f0, late, c_begin, c_end, smem, wave, lane, tot);
  else
    pf_loop_bits<GPC, GATEUP, S::kTiles>(bits, sp, g, f0, late, c_begin, c_end, smem, wave, lane, tot);

  // D layout: lane holds column n = lane%32 (weight row) and, for i < 16,
  // row m = 8*(i/4) + 4*(lane/32) + i%4 (token) of each 32x32 tile.
  const int n = lane & 31;
  if (GATEUP) {
    // The gate and up waves of the same rows (waves 2r, 2r+1) share the h
    // pass: each hands the other the half of its totals the other needs
    // (gate: fragment rows 2 and 3, up: 0 and 1) through LDS, and forms
    // h = silu(gate) * up rounded to fp16 for its own half, into an LDS copy
    // of the workgroup's h tile laid out as in global memory (per fragment
    // row 8 KB: its 128 columns are 8 consecutive 1 KB fragments); all
    // threads then store the tile with 16-byte writes, and the group sums of
    // the rounded h are read back from it, each in column order.
    __syncthreads();                       // the ring is free
    float* xch = reinterpret_cast<float*>(smem);                               // [wave][2 rows][i][64 lanes]
    unsigned char* ht = smem + kPfWaves * 2 * 16 * 64 * 4;                     // [t][8 fragments]
    const bool upw = wave & 1;
    static_assert(S::kTiles == 4, "the h pass splits four fragment rows in halves");
#pragma unroll
    for (int tt = 0; tt < 2; ++tt)
#pragma unroll
      for (int i = 0; i < 16; ++i) xch[((wave * 2 + tt) * 16 + i) * 64 + lane] = upw ? tot[tt][i] : tot[tt + 2][i];
    __syncthreads();
    {
      const int c = 32 * rb + n;           // column within the workgroup's 128
      const int partner = wave ^ 1;
#pragma unroll
      for (int tt = 0; tt < 2; ++tt) {
        const int t = upw ? tt + 2 : tt;   // the fragment row this wave forms
        if (t < nmt) {
#pragma unroll
          for (int i = 0; i < 16; ++i) {
            const int m = 8 * (i >> 2) + 4 * (lane >> 5) + (i & 3);
            const float other = xch[((partner * 2 + tt) * 16 + i) * 64 + lane];
            const float mine = upw ? tot[tt + 2][i] : tot[tt][i];
            const float gv = upw ? other : mine, uv = upw ? mine : other;
            *reinterpret_cast<uint16_t*>(ht + (size_t)t * 8 * kPfFragBytes + frag_offset(0, m, c, 128)) =
                float_to_half_sat(silu(gv) * uv);
          }
        }
      }
    }
    __syncthreads();
    unsigned char* hb = reinterpret_cast<unsigned char*>(g.h);
    for (int idx = threadIdx.x; idx < nmt * 8 * kPfFragBytes / 16; idx += blockDim.x) {
      const int t = idx / (8 * kPfFragBytes / 16), p = idx - t * (8 * kPfFragBytes / 16);
      *reinterpret_cast<u32x4*>(hb + frag_offset(f0 + t, 0, nt * S::kRowsGateUp, L.ffn) + 16 * p) =
          *reinterpret_cast<const u32x4*>(ht + (size_t)t * 8 * kPfFragBytes + 16 * p);
    }
    const int ngw = S::kRowsGateUp / L.G;           // groups in this workgroup
    for (int idx = threadIdx.x; idx < nmt * 32 * ngw; idx += blockDim.x) {
      const int r = idx % (nmt * 32), q = idx / (nmt * 32);
      const int t = r >> 5, m = r & 31;
      float v = 0.0f;
      for (int c0 = q * L.G; c0 < (q + 1) * L.G; c0 += 8) {
        const u32x4 h8 = *reinterpret_cast<const u32x4*>(ht + (size_t)t * 8 * kPfFragBytes + frag_offset(0, m, c0, 128));
#pragma unroll
        for (int w = 0; w < 4; ++w) {
          v += half_bits_to_float(h8[w] & 0xffffu);
          v += half_bits_to_float(h8[w] >> 16);
        }
      }
      g.hsum[((size_t)(f0 + t) * (L.ffn / L.G) + (nt * S::kRowsGateUp) / L.G + q) * 32 + m] = v;
    }
  } else {
    if (!row_valid) return;
    int ebase, ecount;
    expert_range_offsets(offsets, e, tb.P, ebase, ecount);
    const int pbase = ebase + S::kTokens * j;
    const int pend = ebase + ecount;
    float* out = g.partial + (size_t)split * g.part_stride;
#pragma unroll
    for (int t = 0; t < S::kTiles; ++t) {
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const int m = 8 * (i >> 2) + 4 * (lane >> 5) + (i & 3);
        const int pos = pbase + t * 32 + m;
        if (pos < pend) out[(size_t)pos * L.d + row + n] = tot[t][i];
      }
    }
  }
}

template <int GPC>
hipError_t launch_prefill_gemm(const LayerArgs& L, const int32_t* offsets, const PrefillTables& tb,
                               const PrefillGemm& g, bool gateup, hipStream_t stream) {
  // set once per kernel (thread-safe static initialisation)
  static const hipError_t attr_gu = hipFuncSetAttribute(reinterpret_cast<const void*>(&prefill_kernel<GPC, true>),
                                                        hipFuncAttributeMaxDynamicSharedMemorySize, PfCfg::kLdsBytes);
  static const hipError_t attr_dn = hipFuncSetAttribute(reinterpret_cast<const void*>(&prefill_kernel<GPC, false>),
                                                        hipFuncAttributeMaxDynamicSharedMemorySize, PfCfg::kLdsBytes);
  if (attr_gu != hipSuccess) return attr_gu;
  if (attr_dn != hipSuccess) return attr_dn;
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
