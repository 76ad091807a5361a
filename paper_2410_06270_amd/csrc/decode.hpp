// decode.hpp -- the expert GEMVs of small batches (Eq. 1), bandwidth-bound:
//   gate/up: h = fp16(silu(W_gate x) * (W_up x)) per kept (token, expert) pair,
//   down:    fp32 partial sums of W_down h per split of the ffn reduction,
// codes dequantized in registers as in forward_engine.hpp (the exact value
// 1 + q 2^-b enters the MFMA, scale and zero are applied per group in fp32).
//
// Work decomposition.  A work item is (expert e, block of up to 16 of its
// kept pairs, split s of the reduction): a GEMV over R row units (gate/up:
// 16 ffn rows of gate and the same rows of up; down: two 16-row blocks of d)
// and C 128-column chunks.  The grid has one workgroup per compute unit; the
// chunks of all items (a chunk: 16 rows x 128 columns of both streams) are
// laid end to end and each workgroup takes an equal share of them, rounded to
// whole row units, so every CU does the same work whatever the number of
// touched experts and their widths.  The share is counted in chunks, not
// bytes: a chunk costs the same register work (code extraction, MFMAs, group
// epilogues) at every width, and measured per-wave chunk rates were equal for
// 2- and 3-bit experts, so equal chunk counts finish together (equal byte
// counts gave the 2-bit workgroups 45 % more chunks).  Inside a workgroup the 16
// waves split the share's (row unit, chunk) sequence into 16 equal
// contiguous ranges; a row unit whose chunks fall to several waves is summed
// in LDS, in wave order, by the wave that holds its last chunk (fixed order:
// the result does not depend on timing).  Each workgroup reads the routing
// counts and computes its share itself (no planning launch).
//
// The activations of an item (x for gate/up; h, or the gate/up partials, for
// down) are staged once into an LDS slab covering the item's whole reduction
// range.  Copied rows (x, or h) go out as direct-to-LDS loads ahead of each
// wave's weight ring, and the wave waits only for them (a counted wait that
// leaves the ring in flight): the loop starts as soon as the slab has landed,
// while the ring is still arriving, and the weight stream never stops for the
// staging.
#pragma once

#include "forward_engine.hpp"

namespace mc {

constexpr int kDecTok = 16;                   // pairs of a work item (MFMA M)
static_assert(kDecodeMaxT * MC_MAX_TOPK <= 512, "the decode pair list fits its LDS copy");
constexpr int kDecWaves = 16;                 // waves of a workgroup (one workgroup per CU), at most
constexpr int kDecSlabBytes = 146 * 1024;     // activation slab (x or h rows)
constexpr int kDecSumBytes = 9 * 1024;        // group sums of the slab
static_assert(kDecSlabBytes + kDecSumBytes + 128 <= kLdsPerCu, "decode LDS");
static_assert(kDecWaves * 64 * 8 * 4 <= kDecSlabBytes, "the tails fit in the slab");

// Chunks of the reduction an item's slab can hold: (16 tokens + a zero row)
// rows of (chunks*128 + pad) 16-bit values, and their group sums.
__host__ __device__ constexpr int decode_slab_chunks(int gpc) {
  return ((kDecSlabBytes / 2) / (kDecTok + 1) - kRowPad) / kTileCols < kDecSumBytes / (4 * kDecTok * gpc)
             ? ((kDecSlabBytes / 2) / (kDecTok + 1) - kRowPad) / kTileCols
             : kDecSumBytes / (4 * kDecTok * gpc);
}

struct DecodeArgs {
  const uint16_t* x;          // gate/up input: bf16 [T][d]
  const uint16_t* h;          // down input: fp16 [P][ffn] (gu_split == 1)
  const float* gu_in;         // down input: gate/up partials [gu_split][2][P][ffn] (gu_split > 1)
  uint16_t* h_out;            // gate/up output when S == 1
  float* gu_out;              // gate/up output when S > 1: [S][2][P][ffn]
  float* partial;             // down output: [S][P][d]
  size_t part_stride;         // P * d
  const int32_t* counts;
  const int32_t* offsets;
  const int32_t* pair_token;
  int T, P;                   // tokens, kept-pair slots (T*k)
  int S;                      // splits of this GEMV's reduction
  int c_per;                  // chunks per split (the last split may be shorter)
  int gu_split;               // down: splits of the gate/up reduction (1: read h)
  int nwg;                    // workgroups in the grid
};

// -------------------------------------------------------------- the plan --
// Items are laid out expert by expert, pair block j, then split s; item
// (e, j, s) holds R row units of C_s chunks.  A workgroup owns the row units
// whose first chunk lies in [lo, hi) of the layer's chunks, lo = total * wg /
// nwg.  Chunk counts fit 32 bits: at most (T*k/16 + E) items of d*ffn/2048
// chunks, d*ffn <= 2^31.

// Inclusive prefix sum over the 64 lanes with DPP row shifts and row
// broadcasts (register moves, no LDS round trips).
__device__ __forceinline__ uint32_t wave_incl_scan32(uint32_t v) {
  v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x111, 0xf, 0xf, false);   // row_shr:1
  v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x112, 0xf, 0xf, false);   // row_shr:2
  v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x114, 0xf, 0xf, false);   // row_shr:4
  v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x118, 0xf, 0xf, false);   // row_shr:8
  v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x142, 0xa, 0xf, false);   // row_bcast:15, rows 1, 3
  v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x143, 0xc, 0xf, false);   // row_bcast:31, rows 2, 3
  return v;
}

// One expert per lane: its kept-pair range, width, first code-word unit and
// its chunk count over all its items (0 if it has no kept pair).
struct DecLane {
  int eb, ec, b;
  uint32_t cb;          // cum_bits[e]: the expert's codes start at 3 * cb * d * ffn / 32 words
  uint32_t we;
};

__device__ __forceinline__ DecLane expert_lane(const LayerArgs& L, const DecodeArgs& a, int e, uint32_t per_block) {
  DecLane x;
  x.eb = x.ec = x.b = 0;
  x.cb = 0;
  x.we = 0;
  if (e < L.E) {
    expert_range(a.counts, a.offsets, e, a.P, x.eb, x.ec);
    x.cb = L.cum_bits[e];
    x.b = L.cum_bits[e + 1] - (int)x.cb;
    x.we = (uint32_t)((x.ec + kDecTok - 1) / kDecTok) * per_block;
  }
  return x;
}

struct DecPiece {
  int e, b, s, C, u0, u1, pbase, nt;
  uint32_t cb;
  uint32_t next;        // chunk position after the piece's item
  // set when the pieces are grouped (plan_round): pieces of one batch run
  // at the same time on waves [w0, w1), each with its own slab
  int batch, w0, w1, slab_off, sum_off;
};

// ceil(x / y) for y > 0, 0 for x <= 0.
__device__ __forceinline__ int ceil_div_pos(int x, int y) { return x <= 0 ? 0 : (x + y - 1) / y; }

// The piece that begins at chunk position pos if it lies in the experts of
// x (lanes e0 + lane, whose items start at chunk position base): the item
// containing pos and the row units of it whose first chunk lies in [lo, hi).
// Returns false when pos is not in these experts.
__device__ __forceinline__ bool piece_in(const DecodeArgs& a, const DecLane& x, int e0, uint32_t base, int R,
                                         int ntiles, uint32_t lo, uint32_t hi, uint32_t pos, uint32_t incl,
                                         DecPiece& p) {
  const uint32_t ebase = base + incl - x.we;
  const unsigned long long mask = __ballot(x.we > 0 && ebase <= pos && pos < ebase + x.we);
  if (!mask) return false;
  const int l = __builtin_ctzll(mask);
  const uint32_t per_block = (uint32_t)R * ntiles;
  const uint32_t xb = __builtin_amdgcn_readlane(ebase, l);
  const int eb = __builtin_amdgcn_readlane(x.eb, l);
  const int ec = __builtin_amdgcn_readlane(x.ec, l);
  p.e = e0 + l;
  p.b = __builtin_amdgcn_readlane(x.b, l);
  p.cb = __builtin_amdgcn_readlane(x.cb, l);
  const uint32_t off = pos - xb;                     // chunk position inside the expert
  const int j = (int)(off / per_block);               // pair block
  const uint32_t rest = off - (uint32_t)j * per_block;
  int s = (int)(rest / ((uint32_t)R * a.c_per));      // split
  if (s >= a.S) s = a.S - 1;
  const int c0 = s * a.c_per;
  const int C = (ntiles - c0) < a.c_per ? (ntiles - c0) : a.c_per;
  const uint32_t ib = xb + (uint32_t)j * per_block + (uint32_t)R * c0;   // item base
  const int u0 = ceil_div_pos((int)lo - (int)ib, C);
  const int u1 = ceil_div_pos((int)hi - (int)ib, C);
  p.u0 = u0 < R ? u0 : R;
  p.u1 = u1 < R ? u1 : R;
  p.s = s;
  p.C = C;
  pair_block(eb, ec, j, kDecTok, p.pbase, p.nt);
  p.next = ib + (uint32_t)C * R;
  return true;
}

// The piece at pos, reading the routing counts again (pieces after the
// first; they are rare: a share crosses at most a few items).
__device__ __forceinline__ DecPiece find_piece(const LayerArgs& L, const DecodeArgs& a, int R, int ntiles,
                                               uint32_t lo, uint32_t hi, uint32_t pos) {
  DecPiece p;
  p.u0 = p.u1 = 0;
  p.next = hi;
  const int lane = threadIdx.x & 63;
  uint32_t base = 0;
  for (int e0 = 0; e0 < L.E; e0 += 64) {
    const DecLane x = expert_lane(L, a, e0 + lane, (uint32_t)R * ntiles);
    const uint32_t incl = wave_incl_scan32(x.we);
    if (piece_in(a, x, e0, base, R, ntiles, lo, hi, pos, incl, p)) return p;
    base += __builtin_amdgcn_readlane(incl, 63);
  }
  return p;
}

// ------------------------------------------------------------- streaming --

// Position in a wave's chunk range: row unit u, chunk c of the item's range,
// and the byte offsets of the chunk (relative to the streams' bases).
struct DecCursor {
  int u, c;
  uint32_t wo, so;
};

struct DecGeom {
  rsrc_t w, s;                // buffer resources over the expert's matrices (gate and up, or down)
  uint32_t bw[2], bs[2];      // byte offsets of (unit 0, chunk 0) of each stream
  uint32_t uw, us;            // byte strides of one row unit (codes, scale/zero)
  uint32_t cw, cs;            // byte strides of one chunk (codes, scale/zero)
  uint32_t lane_w, lane_s;    // this lane's offsets inside a chunk
  int C;                      // chunks per row unit
};

// Advances the cursor by one chunk when adv (wave-uniform) holds; written
// with selects, not branches, so that the unrolled ring stays one basic
// block (a branch there made the compiler drain the ring at the loop's back
// edge).
__device__ __forceinline__ void cursor_next(DecCursor& k, const DecGeom& g, bool adv = true) {
  const bool wrap = k.c + 1 == g.C;
  const int c = wrap ? 0 : k.c + 1;
  const uint32_t dw = wrap ? g.uw - (uint32_t)(g.C - 1) * g.cw : g.cw;
  const uint32_t ds = wrap ? g.us - (uint32_t)(g.C - 1) * g.cs : g.cs;
  k.u = adv ? k.u + (wrap ? 1 : 0) : k.u;
  k.c = adv ? c : k.c;
  k.wo = adv ? k.wo + dw : k.wo;
  k.so = adv ? k.so + ds : k.so;
}

// The lane's offset is the load's VGPR offset; the wave-uniform chunk offset
// goes into the SGPR offset field, so a refill costs no vector adds.
template <int BITS, int GPC>
__device__ __forceinline__ void dec_load(uint32_t (&w)[2][BITS], uint32_t (&s)[2][GPC], const DecGeom& g,
                                         const DecCursor& k) {
#pragma unroll
  for (int j = 0; j < 2; ++j) load_words_so<BITS>(w[j], g.w, g.lane_w, g.bw[j] + k.wo);
#pragma unroll
  for (int q = 0; q < GPC; ++q)
#pragma unroll
    for (int j = 0; j < 2; ++j)
      s[j][q] = __builtin_amdgcn_raw_buffer_load_b32(g.s, g.lane_s, g.bs[j] + k.so + q * 64u, 0);
}

__device__ __forceinline__ void zero2(f32x4 (&t)[2]) {
  t[0] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
  t[1] = t[0];
}

__device__ __forceinline__ void set_progress_priority(int quarter) {
  if (quarter <= 0) __builtin_amdgcn_s_setprio(3);
  else if (quarter == 1) __builtin_amdgcn_s_setprio(2);
  else if (quarter == 2) __builtin_amdgcn_s_setprio(1);
  else __builtin_amdgcn_s_setprio(0);
}

// Start of part w of a piece of N chunks in groups of D: the nw parts (one
// per wave working on the piece) are equal contiguous ranges of whole groups.
__device__ __forceinline__ int dec_part_start(int N, int D, int w, int nw) {
  return D * (int)(((uint32_t)(N / D) * (uint32_t)w) / (uint32_t)nw);   // N/D * 16 fits 32 bits
}

// Streams this wave's part of the piece (row units [u0, u1), C chunks each;
// D divides C) against the slab that stage_early() and stage_late() fill
// (before and after the first D chunks of the weight ring are issued), writes
// every row unit it completes with emit(u, t), and reduces the row units
// split over several waves.  Vector
// memory stores happen only between row units (outside the unrolled ring), so
// the compiler's load counting keeps the ring in flight.
template <int BITS, int GPC, bool F16, int D, typename EarlyFn, typename LateFn, typename EmitFn>
__device__ __forceinline__ void decode_run(const DecGeom& g, int u0, int u1, int C, int w0, int w1,
                                           const uint16_t* arow, const float* sxs, float* tails,
                                           EarlyFn stage_early, LateFn stage_late, EmitFn emit) {
  const int lane = threadIdx.x & 63, wave = wave_id();
  const int nw = w1 - w0, wl = wave - w0;       // this piece's waves, this wave among them
  const int N = (u1 - u0) * C;
  const int qa = dec_part_start(N, D, wl, nw), qb = dec_part_start(N, D, wl + 1, nw);
  DecCursor pc;                 // prefetch cursor: stops at the part's last chunk
  pc.u = u0 + qa / C;
  pc.c = qa - (pc.u - u0) * C;
  pc.wo = (uint32_t)pc.u * g.uw + (uint32_t)pc.c * g.cw;
  pc.so = (uint32_t)pc.u * g.us + (uint32_t)pc.c * g.cs;
  int pleft = qb - qa - 1;
  uint32_t wr[D][2][BITS];
  uint32_t sr[D][2][GPC];
  stage_early();
  if (qa < qb) {
#pragma unroll
    for (int j = 0; j < D; ++j) {
      dec_load<BITS, GPC>(wr[j], sr[j], g, pc);
      cursor_next(pc, g, pleft > 0);
      pleft = pleft > 0 ? pleft - 1 : 0;
    }
    // the staging copies, issued before the ring, have landed once at most
    // the ring's loads (2 + 2 GPC instructions a chunk) are outstanding
    wait_vmcnt<D * (2 + 2 * GPC)>();
  } else {
    wait_vmcnt<0>();
  }
  asm volatile("" ::: "memory");
  stage_late();

  f32x4 acc[2][1], tot[2][1], head[2];
  zero2(head);
  tot[0][0] = head[0];
  tot[1][0] = head[0];
  acc[0][0] = head[0];
  acc[1][0] = head[0];
  const uint16_t* ar[1] = {arow};
  const uint32_t magic = vgpr_constant(Fmt<F16>::kMagic2);
  bool has_head = false;
  int u = u0 + qa / C, c = qa - (u - u0) * C;
  bool started = (c == 0);      // the current row unit begins inside this part
  const int t1 = qa + (qb - qa) / 4, t2 = qa + (qb - qa) / 2, t3 = qb - (qb - qa) / 4;   // quarters
  for (int q = qa; q < qb;) {
    const int ce = (C - c) < (qb - q) ? C : c + (qb - q);   // end of this unit's share of the part
    q += ce - c;
    for (; c < ce; c += D) {
      // fair issue among the waves of a SIMD: the arbiter favours older
      // waves, which then finish their (equal) ranges long before the
      // youngest; a wave's priority drops with each quarter of its range done
      const int at = q - (ce - c);             // position of chunk c
      set_progress_priority((at >= t1) + (at >= t2) + (at >= t3));
#pragma unroll
      for (int j = 0; j < D; ++j) {
        compute_chunk<BITS, 1, GPC, F16>(wr[j], sr[j], acc, tot, ar, sxs, c + j, lane, magic);
        dec_load<BITS, GPC>(wr[j], sr[j], g, pc);
        cursor_next(pc, g, pleft > 0);
        pleft = pleft > 0 ? pleft - 1 : 0;
        // the refill issues here, not later: left to itself the scheduler
        // sinks the ring's refills to the end of the loop body
        __builtin_amdgcn_sched_barrier(0);
      }
    }
    if (c == C) {               // the row unit is complete in this part
      const f32x4 t[2] = {tot[0][0], tot[1][0]};
      if (started) {
        emit(u, t);
      } else {
        head[0] = t[0];
        head[1] = t[1];
        has_head = true;
      }
      tot[0][0] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
      tot[1][0] = tot[0][0];
      started = true;
      ++u;
      c = 0;
    }
  }
  wait_vmcnt<0>();   // the ring's last (never consumed) refills
  __builtin_amdgcn_s_setprio(0);

  // row units split over several waves: every wave but the last of a unit
  // leaves its part (its tail) in LDS; the wave holding the unit's last
  // chunk adds them in wave order to its own part (its head)
  const bool has_tail = qa < qb && c != 0;
  __syncthreads();                 // the slab is no longer read
  if (has_tail) {
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int i = 0; i < 4; ++i) tails[((wave * 2 + j) * 4 + i) * 64 + lane] = tot[j][0][i];
  }
  __syncthreads();
  if (has_head) {
    const int ua = u0 + qa / C;                    // the unit this wave's part starts in
    const int first = (ua - u0) * C;               // its first chunk
    int wf = 0;                                    // the part holding that chunk
    for (int w2 = 1; w2 < nw; ++w2)
      if (dec_part_start(N, D, w2, nw) <= first) wf = w2;
    f32x4 t[2];
    zero2(t);
    for (int w2 = wf; w2 < wl; ++w2) {
      // empty parts (pieces of fewer groups than waves) hold nothing
      if (dec_part_start(N, D, w2, nw) == dec_part_start(N, D, w2 + 1, nw)) continue;
      const int wg = w0 + w2;                      // the workgroup's wave of part w2
#pragma unroll
      for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int i = 0; i < 4; ++i) t[j][i] += tails[((wg * 2 + j) * 4 + i) * 64 + lane];
    }
    t[0] += head[0];
    t[1] += head[1];
    emit(ua, t);
  }
}

// One piece for an expert of width BITS: the streams' geometry, the staging
// of its activations and the writing of its outputs, then decode_run.
template <int BITS, int GPC, bool GATEUP>
__device__ __forceinline__ void decode_piece(const LayerArgs& L, const DecodeArgs& a, unsigned char* smem,
                                             const int32_t* s_tok, const DecPiece& p) {
  const int e = p.e, s = p.s, C = p.C, u0 = p.u0, u1 = p.u1, pbase = p.pbase, nt = p.nt;
  constexpr bool F16 = !GATEUP;
  const int lane = threadIdx.x & 63;
  const int K = GATEUP ? L.d : L.ffn;
  const int ntiles = K / kTileCols, ng = ntiles * GPC;
  const int c0 = s * a.c_per;
  uint16_t* xs = reinterpret_cast<uint16_t*>(smem + p.slab_off);
  float* sxs = reinterpret_cast<float*>(smem + kDecSlabBytes + p.sum_off);
  float* tails = reinterpret_cast<float*>(smem);
  const int nw = p.w1 - p.w0, wl = wave_id() - p.w0;   // the waves staging and streaming this piece

  // geometry of the two streams
  DecGeom g;
  g.C = C;
  g.cw = 64u * BITS * 4u;
  g.cs = (uint32_t)GPC * 64u;
  g.lane_w = (uint32_t)lane * BITS * 4u;
  g.lane_s = (uint32_t)(lane & 15) * 4u;
  const uint32_t rb_per_unit = GATEUP ? 1u : 2u;
  g.uw = rb_per_unit * (uint32_t)ntiles * g.cw;
  g.us = rb_per_unit * (uint32_t)ng * 64u;
  // gate and up of an expert are adjacent in memory (codes and scale/zero
  // words alike): one resource covers both streams
  const uint32_t mat_w = (uint32_t)((size_t)L.d * L.ffn / 32 * BITS * 4);   // bytes of one matrix's codes
  const uint32_t mat_s = (uint32_t)((size_t)L.d * L.ffn * GPC / 32);       // ... and scale/zero words (G = 128/GPC)
  // the expert's matrices: codes at 3 * cum_bits[e] (+ 2 * b for down) bit
  // planes of d*ffn/32 words, scale/zero words at (3e (+ 2)) * d*ffn/G
  const size_t plane = (size_t)L.d * L.ffn / 32;
  const size_t wofs = (3 * (size_t)p.cb + (GATEUP ? 0 : 2 * BITS)) * plane;
  const size_t sofs = (3 * (size_t)e + (GATEUP ? 0 : 2)) * ((size_t)L.d * L.ffn * GPC / 128);
  g.w = make_rsrc(L.words + wofs, (GATEUP ? 2u : 1u) * mat_w);
  g.s = make_rsrc(L.sz + sofs, (GATEUP ? 2u : 1u) * mat_s);
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    // gate/up: stream j is matrix j; down: stream j takes row block 2u + j
    const uint32_t rb = GATEUP ? 0u : (uint32_t)j;
    g.bw[j] = (GATEUP ? (uint32_t)j * mat_w : 0u) + (rb * (uint32_t)ntiles + (uint32_t)c0) * g.cw;
    g.bs[j] = (GATEUP ? (uint32_t)j * mat_s : 0u) + (rb * (uint32_t)ng + (uint32_t)c0 * GPC) * 64u;
  }

  // the activation slab: rows pbase .. pbase+nt-1, chunks [c0, c0+C)
  const int kw = C * kTileCols;
  const int RS = kw + kRowPad;
  uint16_t* zrow = xs + (size_t)nt * RS;
  // Staging in two parts around the weight ring's first loads: the copies
  // of x (or h) go out as direct-to-LDS loads before the ring (stage_early),
  // so that they land first and the loop can start while the ring is still
  // arriving; their sums, or the h rows formed from the gate/up partials,
  // follow the ring (stage_late).
  const bool copy_rows = GATEUP || a.gu_split == 1;
  auto stage_early = [&]() {
    for (int i = wl * 64 + lane; i < RS / 8; i += nw * 64)
      *reinterpret_cast<u32x4*>(zrow + 8 * i) = u32x4{0u, 0u, 0u, 0u};
    if (GATEUP) {
      // lane m < nt holds the token of pair pbase + m (from the workgroup's
      // LDS copy of the pair list), so the row of each staged segment is a
      // register read, not a dependent global load per segment
      const int tok = (lane < nt) ? clamp_token(s_tok[pbase + lane], a.T) : 0;
      stage_rows_issue(
          xs, [&](int m) { return a.x + (size_t)__builtin_amdgcn_readlane(tok, m) * K; }, nt, c0 * kTileCols, kw,
          RS, wl, nw);
    } else if (a.gu_split == 1) {
      stage_rows_issue(xs, [&](int m) { return a.h + (size_t)(pbase + m) * K; }, nt, c0 * kTileCols, kw, RS, wl,
                       nw);
    }
  };
  auto stage_late = [&]() {
    if (copy_rows) {
      stage_rows_sums<F16, 16 / GPC>(xs, sxs, nt, kDecTok, kw, RS, wl, nw);
    } else {
      // h from the gate/up partial sums (added in split order), rounded to
      // fp16 as an unsplit gate/up epilogue forms it
      const size_t P = a.P;
      auto piece = [&](int m, int k) {
        const size_t o = (size_t)(pbase + m) * K + k;
        f32x4 g0 = {0.f, 0.f, 0.f, 0.f}, g1 = g0, v0 = g0, v1 = g0;
        for (int sp = 0; sp < a.gu_split; ++sp) {
          const float* part = a.gu_in + (size_t)sp * 2 * P * K + o;
          g0 += *reinterpret_cast<const f32x4*>(part);
          g1 += *reinterpret_cast<const f32x4*>(part + 4);
          v0 += *reinterpret_cast<const f32x4*>(part + P * K);
          v1 += *reinterpret_cast<const f32x4*>(part + P * K + 4);
        }
        u32x4 v;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const float ha = silu(q < 2 ? g0[2 * q] : g1[2 * q - 4]) * (q < 2 ? v0[2 * q] : v1[2 * q - 4]);
          const float hb = silu(q < 2 ? g0[2 * q + 1] : g1[2 * q - 3]) * (q < 2 ? v0[2 * q + 1] : v1[2 * q - 3]);
          v[q] = (uint32_t)float_to_half_sat(ha) | ((uint32_t)float_to_half_sat(hb) << 16);
        }
        return v;
      };
      stage_pieces<true, 16 / GPC>(xs, sxs, piece, nt, kDecTok, c0 * kTileCols, kw, RS, wl, nw);
    }
  };

  // outputs of a complete row unit
  auto emit = [&](int u, const f32x4 (&t)[2]) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int m = 4 * (lane >> 4) + i;
      if (m >= nt) continue;
      if (GATEUP) {
        const int n = u * 16 + (lane & 15);
        if (a.S == 1) {
          a.h_out[(size_t)(pbase + m) * L.ffn + n] = float_to_half_sat(silu(t[0][i]) * t[1][i]);
        } else {
          const size_t o = ((size_t)s * 2 * a.P + pbase + m) * L.ffn + n;
          a.gu_out[o] = t[0][i];
          a.gu_out[o + (size_t)a.P * L.ffn] = t[1][i];
        }
      } else {
#pragma unroll
        for (int j = 0; j < 2; ++j)
          a.partial[(size_t)s * a.part_stride + (size_t)(pbase + m) * L.d + (2 * u + j) * 16 + (lane & 15)] =
              t[j][i];
      }
    }
  };

  const uint16_t* arow = ((lane & 15) < nt ? xs + (size_t)(lane & 15) * RS : zrow) + 8 * (lane >> 4);
  // ring depth: the deepest that divides C, so that ring slot j always holds
  // chunk c + j of a unit and the unrolled loop needs no remainder.  The
  // waves' parts are whole groups of D chunks, so a small piece (a few groups
  // per wave) is shared out unevenly: there the shallower ring halves the
  // grain (measured on the OLMoE-shaped layer, 92 chunks a workgroup at 16
  // tokens: gate/up 20.4 -> 18.9 us), and below two groups of two chunks a
  // wave the one-chunk ring (down there, 46 chunks a workgroup: 14.6 ->
  // 13.9 us).  With 8 waves or fewer the shallow ring keeps too few bytes in
  // flight, so it takes a smaller piece to pay.
  constexpr int DM = prefetch_depth(1, GPC);
  const int nchunks = (u1 - u0) * C, nwp = p.w1 - p.w0;
  const bool deep = DM == 2 || nchunks >= (nwp > 8 ? 4 : 3) * DM * nwp;
  if (C % DM == 0 && deep)
    decode_run<BITS, GPC, F16, DM>(g, u0, u1, C, p.w0, p.w1, arow, sxs, tails, stage_early, stage_late, emit);
  else if (C % 2 == 0 && nchunks >= 2 * 2 * nwp)
    decode_run<BITS, GPC, F16, 2>(g, u0, u1, C, p.w0, p.w1, arow, sxs, tails, stage_early, stage_late, emit);
  else
    decode_run<BITS, GPC, F16, 1>(g, u0, u1, C, p.w0, p.w1, arow, sxs, tails, stage_early, stage_late, emit);
}

constexpr int kDecMaxPieces = 8;   // pieces planned per round (a share crosses few items)

struct DecPlan {
  DecPiece piece[kDecMaxPieces];
  int n;                 // pieces of this round
  int nbatch;            // batches of pieces that run at the same time
  int more;              // another round follows
  uint32_t pos;          // where the next round starts
};
// dynamic (slab, sums) and static (plan, pair list) LDS of the decode kernel
static_assert(kDecSlabBytes + kDecSumBytes + sizeof(DecPlan) + sizeof(int32_t) * kDecodeMaxT * MC_MAX_TOPK <=
                  kLdsPerCu,
              "decode LDS");

// Pieces [b0, b1) of the plan run together: every piece gets one wave, the
// other waves are shared out in proportion to the pieces' chunks.
template <int NW>
__device__ __forceinline__ void share_waves(DecPlan& plan, int b0, int b1) {
  const int nb = b1 - b0;
  uint32_t tot = 0;
  for (int i = b0; i < b1; ++i) tot += (uint32_t)(plan.piece[i].u1 - plan.piece[i].u0) * plan.piece[i].C;
  uint32_t cum = 0;
  for (int i = b0; i < b1; ++i) {
    DecPiece& p = plan.piece[i];
    p.w0 = (i - b0) + (int)(((unsigned long long)(NW - nb) * cum) / tot);
    cum += (uint32_t)(p.u1 - p.u0) * p.C;
    p.w1 = (i - b0) + 1 + (int)(((unsigned long long)(NW - nb) * cum) / tot);
  }
}

// Plans pieces from pos on (wave 0): up to kDecMaxPieces of them, the first
// from the cached lanes x0 when pos == lo; then groups consecutive pieces
// whose slabs fit the LDS together into batches.
template <int GPC, int NW>
__device__ __forceinline__ void plan_round(const LayerArgs& L, const DecodeArgs& a, const DecLane* x0,
                                           uint32_t incl0, int R, int ntiles, uint32_t lo, uint32_t hi,
                                           uint32_t pos, DecPlan& plan) {
  const int lane = threadIdx.x & 63;
  int n = 0;
  while (pos < hi && n < kDecMaxPieces) {
    DecPiece p;
    if (!(x0 && pos == lo && piece_in(a, *x0, 0, 0, R, ntiles, lo, hi, pos, incl0, p)))
      p = find_piece(L, a, R, ntiles, lo, hi, pos);
    pos = p.next > pos ? p.next : hi;    // always advances
    if (p.u0 >= p.u1) continue;
    if (lane == 0) plan.piece[n] = p;
    ++n;
  }
  if (lane == 0) {
    int b0 = 0, batch = 0, used_slab = 0, used_sum = 0;
    for (int i = 0; i < n; ++i) {
      DecPiece& p = plan.piece[i];
      const int slab = (((p.nt + 1) * (p.C * kTileCols + kRowPad) * 2) + 15) & ~15;
      const int sum = kDecTok * p.C * GPC * 4;
      if (i > b0 && (used_slab + slab > kDecSlabBytes || used_sum + sum > kDecSumBytes || i - b0 >= NW)) {
        share_waves<NW>(plan, b0, i);
        b0 = i;
        ++batch;
        used_slab = used_sum = 0;
      }
      p.batch = batch;
      p.slab_off = used_slab;
      p.sum_off = used_sum;
      used_slab += slab;
      used_sum += sum;
    }
    if (n > 0) share_waves<NW>(plan, b0, n);
    plan.n = n;
    plan.nbatch = n > 0 ? batch + 1 : 0;
    plan.more = pos < hi;
    plan.pos = pos;
  }
}

template <int GPC, bool GATEUP, int NW>
__global__ void __launch_bounds__(64 * NW) __attribute__((amdgpu_waves_per_eu(NW / 4)))
decode_kernel(LayerArgs L, DecodeArgs a) {
  static_assert(NW >= 2 && NW <= kDecWaves, "waves of the decode workgroup");
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
  // the workgroup's pieces, planned by wave 0 (the other waves would only
  // repeat the same scalar work on their SIMDs)
  __shared__ DecPlan plan;
  // gate/up: the batch's pair list (token of each kept-pair slot), copied by
  // the other waves while wave 0 plans, so that staging needs no global load
  // round trip before its copies go out
  __shared__ int32_t s_tok[GATEUP ? kDecodeMaxT * MC_MAX_TOPK : 1];
  const int lane = threadIdx.x & 63, wave = wave_id();
  const int K = GATEUP ? L.d : L.ffn;
  const int ntiles = K / kTileCols;
  const int R = GATEUP ? L.ffn / 16 : L.d / 32;
  const uint32_t per_block = (uint32_t)R * ntiles;
  uint32_t lo = 0, hi = 0;     // wave 0's: this workgroup's share of the chunks
  if (wave == 0) {
    // one round of loads: the first 64 experts (every expert of most layers)
    const DecLane x0 = expert_lane(L, a, lane, per_block);
    const uint32_t incl0 = wave_incl_scan32(x0.we);
    uint32_t total = __builtin_amdgcn_readlane(incl0, 63);
    for (int e0 = 64; e0 < L.E; e0 += 64)
      total += __builtin_amdgcn_readlane(wave_incl_scan32(expert_lane(L, a, e0 + lane, per_block).we), 63);
    // lo = total * wg / nwg in 32-bit arithmetic
    const uint32_t q = total / (uint32_t)a.nwg, rm = total % (uint32_t)a.nwg;
    lo = q * blockIdx.x + (rm * blockIdx.x) / a.nwg;
    hi = q * (blockIdx.x + 1) + (rm * (blockIdx.x + 1)) / a.nwg;
    plan_round<GPC, NW>(L, a, &x0, incl0, R, ntiles, lo, hi, lo, plan);
  } else if (GATEUP) {
    for (int i = (wave - 1) * 64 + lane; i < a.P; i += (NW - 1) * 64) s_tok[i] = a.pair_token[i];
  }
  __syncthreads();
  for (;;) {
    const int n = plan.n, nbatch = plan.nbatch, more = plan.more;
    for (int bt = 0; bt < nbatch; ++bt) {
      if (bt > 0) __syncthreads();   // the previous batch's LDS reads are done
      // this wave's piece of the batch (the batch's pieces share out all waves)
      int mine = 0;
      for (int i = 0; i < n; ++i)
        if (plan.piece[i].batch == bt && plan.piece[i].w0 <= wave && wave < plan.piece[i].w1) mine = i;
      const DecPiece p = plan.piece[mine];
      if (p.b == 1)
        decode_piece<1, GPC, GATEUP>(L, a, smem, s_tok, p);
      else if (p.b == 2)
        decode_piece<2, GPC, GATEUP>(L, a, smem, s_tok, p);
      else
        decode_piece<3, GPC, GATEUP>(L, a, smem, s_tok, p);
    }
    if (!more) break;
    __syncthreads();                 // every wave has read the plan and left the slab
    if (wave == 0) plan_round<GPC, NW>(L, a, nullptr, 0, R, ntiles, lo, hi, plan.pos, plan);
    __syncthreads();
  }
}

// Waves of the decode workgroup.  Small batches, whose items hold one or two
// tokens, run best with 8 (each wave streams twice the chunks and the
// per-piece set-up, staging and tail reduction are shared by fewer waves);
// larger ones with 16, whose staging and reductions of the fuller slabs go
// faster on more waves.  Measured on the Mixtral- and OLMoE-shaped layers:
// 8 waves win for gate/up up to 8 tokens, for down up to 4.
inline int decode_waves(bool gateup, int T) { return T <= (gateup ? 8 : 4) ? 8 : 16; }

template <int GPC, bool GATEUP, int NW>
hipError_t launch_decode_nw(const LayerArgs& L, const DecodeArgs& a, hipStream_t stream) {
  constexpr int lds = kDecSlabBytes + kDecSumBytes;
  // set once per instantiation (thread-safe static initialisation)
  static const hipError_t attr = hipFuncSetAttribute(
      reinterpret_cast<const void*>(&decode_kernel<GPC, GATEUP, NW>), hipFuncAttributeMaxDynamicSharedMemorySize, lds);
  if (attr != hipSuccess) return attr;
  hipLaunchKernelGGL((decode_kernel<GPC, GATEUP, NW>), dim3(a.nwg), dim3(64 * NW), lds, stream, L, a);
  return hipGetLastError();
}

template <int GPC, bool GATEUP>
hipError_t launch_decode(const LayerArgs& L, const DecodeArgs& a, hipStream_t stream) {
  return decode_waves(GATEUP, a.T) == 8 ? launch_decode_nw<GPC, GATEUP, 8>(L, a, stream)
                                        : launch_decode_nw<GPC, GATEUP, 16>(L, a, stream);
}

}  // namespace mc
