// route_device.hpp -- the per-token selection of Eq. 1 / Eq. 5 / Sec. 3.3.2
// and the small-batch list builder of the routing kernels.
#pragma once

#include "mc_internal.hpp"

namespace mc {

// Order-preserving integer image of a float, with -0 mapped onto +0.
__device__ __forceinline__ uint32_t ordered_bits(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) == 0) u = 0;
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// Lane segments of the selection: a wave selects 64 / S tokens at once, one
// per segment of S lanes, S the smallest power of two >= E (at most 64; with
// more than 64 experts lane q holds experts q, q+64, ...).
__host__ __device__ constexpr int sel_segment(int E) { return E <= 1 ? 1 : E <= 64 ? 1 << (32 - __builtin_clz(E - 1)) : 64; }

// Per-wave LDS scratch of the selection: the segments' keys (segment g at
// [g*S, g*S + E)), and per segment its k selected (expert, logit) pairs in
// rank order and their exp terms (segment g at [g*k, g*k + k); 64/S segments
// of k <= S entries).
struct SelScratch {
  unsigned long long* key;   // [max(64, E)]
  int* sel_e;                // [64]
  float* sel_l;              // [64]
  double* ex;                // [64]
};
constexpr int kSelScratchBytes = MC_MAX_EXPERTS * 8 + 64 * (4 + 4 + 8);

__device__ __forceinline__ SelScratch sel_scratch(unsigned char* base) {
  SelScratch s;
  s.key = reinterpret_cast<unsigned long long*>(base);
  s.ex = reinterpret_cast<double*>(base + MC_MAX_EXPERTS * 8);
  s.sel_e = reinterpret_cast<int*>(base + MC_MAX_EXPERTS * 8 + 64 * 8);
  s.sel_l = reinterpret_cast<float*>(base + MC_MAX_EXPERTS * 8 + 64 * 12);
  return s;
}

// The lane's share of token t's inputs (t >= T: none): the logits of experts
// q, q+S, ... (q the lane within its segment of S lanes) and the protection
// flag (important NULL: unprotected).
struct SelInput {
  float lv[4];
  int prot;
};

__device__ __forceinline__ SelInput sel_load(const float* __restrict__ logits, const uint8_t* __restrict__ important,
                                             int t, int T, int E, int S) {
  const int q = (threadIdx.x & 63) & (S - 1);
  const bool tv = t < T;
  SelInput in;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int e = q + S * j;
    in.lv[j] = (tv && e < E) ? logits[(size_t)t * E + e] : 0.0f;
  }
  in.prot = (tv && important != nullptr) ? (int)important[t] : 0;
  return in;
}

// Selects and prunes token t (one segment of S lanes of the wave; every lane
// of the wave calls it, each segment with its own token; t >= T: nothing is
// written).  The lanes hold the logits as distinct 64-bit keys (ordered logit
// bits, then the complement of the expert index, so larger key = earlier
// rank); the keys go to the segment's LDS scratch and each key's rank is the
// number of larger keys of the segment.  The rank-r pair goes to slot r,
// lane r < k of the segment takes it; the softmax sums run over the ranks in
// order (fp64).  Lane r < k writes rank r's outputs (when `publish`); when
// s_ent/s_w are given it also records them in LDS (expert, or 0xffff if
// pruned).
static __device__ void select_token(const SelInput& in, int t, int T, int E, int S, int k, float delta32,
                                    double tau, int32_t* __restrict__ topk_idx, float* __restrict__ topk_w,
                                    uint8_t* __restrict__ kept, int32_t* __restrict__ pair_pos, bool publish,
                                    uint16_t* s_ent, float* s_w, const SelScratch& sc) {
  const int lane = threadIdx.x & 63;
  const int q = lane & (S - 1), seg = lane >> __builtin_ctz((unsigned)S);
  const int kb = seg * S, sb = seg * k;   // the segment's keys and selection slots
  const float* lv = in.lv;
  const int prot_flag = in.prot;
  unsigned long long key[4];
  int rank[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int e = q + S * j;
    key[j] = (e < E) ? (((unsigned long long)ordered_bits(lv[j]) << 32) | (unsigned)(0xffff - e)) : 0ull;
    rank[j] = 0;
    if (e < E) sc.key[kb + e] = key[j];
  }
  __builtin_amdgcn_wave_barrier();
  const int nj = (E + S - 1) / S;                    // keys per lane (wave-uniform)
  int e2 = 0;
  if (nj == 1) {
    // one key per lane (E <= 64): sixteen broadcast reads in flight per wait
    int r0 = 0;
    for (; e2 + 16 <= E; e2 += 16) {
      unsigned long long o[16];
#pragma unroll
      for (int u = 0; u < 16; ++u) o[u] = sc.key[kb + e2 + u];
#pragma unroll
      for (int u = 0; u < 16; ++u) r0 += o[u] > key[0] ? 1 : 0;
    }
    for (; e2 + 4 <= E; e2 += 4) {
      unsigned long long o[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) o[u] = sc.key[kb + e2 + u];
#pragma unroll
      for (int u = 0; u < 4; ++u) r0 += o[u] > key[0] ? 1 : 0;
    }
    for (; e2 < E; ++e2) r0 += sc.key[kb + e2] > key[0] ? 1 : 0;
    rank[0] = r0;
  }
  for (; e2 + 4 <= E; e2 += 4) {
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const unsigned long long o = sc.key[kb + e2 + u];
#pragma unroll
      for (int j = 0; j < 4; ++j)
        if (j < nj) rank[j] += o > key[j] ? 1 : 0;
    }
  }
  for (; e2 < E; ++e2) {
    const unsigned long long o = sc.key[kb + e2];
#pragma unroll
    for (int j = 0; j < 4; ++j)
      if (j < nj) rank[j] += o > key[j] ? 1 : 0;
  }
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int e = q + S * j;
    if (e < E && rank[j] < k) {
      sc.sel_e[sb + rank[j]] = e;
      sc.sel_l[sb + rank[j]] = lv[j];
    }
  }
  __builtin_amdgcn_wave_barrier();
  const bool mine = q < k;
  const int my_e = mine ? sc.sel_e[sb + q] : 0;
  const float my_l = mine ? sc.sel_l[sb + q] : 0.0f;
  const float l0 = sc.sel_l[sb];
  const float l1 = k < 2 ? l0 : sc.sel_l[sb + 1];
  const bool prot = prot_flag != 0;
  const double ex = mine ? exp((double)my_l - (double)l0) : 0.0;
  if (mine) sc.ex[sb + q] = ex;
  __builtin_amdgcn_wave_barrier();
  double sum_all = 0.0;
  for (int r = 0; r < k; ++r) sum_all += sc.ex[sb + r];
  bool keep = mine;
  if (mine && q > 0 && !prot) {
    if (k == 2) {
      const float gap = l0 - l1;
      keep = !(gap > delta32);
    } else {
      keep = !(ex < tau * sum_all);
    }
  }
  const unsigned long long kbits = __ballot(keep) >> kb;   // this segment's ranks from bit 0
  double sum_kept = 0.0;
  for (int r = 0; r < k; ++r)
    if ((kbits >> r) & 1ull) sum_kept += sc.ex[sb + r];
  if (mine && t < T) {
    const size_t o = (size_t)t * k + q;
    const float w = keep ? (float)(ex / sum_kept) : 0.0f;
    if (publish) {
      topk_idx[o] = my_e;
      kept[o] = keep ? 1 : 0;
      topk_w[o] = w;
      if (!keep) pair_pos[o] = -1;
    }
    if (s_ent) {
      s_ent[o] = keep ? (uint16_t)my_e : (uint16_t)0xffff;
      s_w[o] = w;
    }
  }
  __builtin_amdgcn_wave_barrier();   // the scratch is free for the wave's next tokens
}

// Exclusive scan of cnt[0..E) into base[] and offsets[0..E] (one wave: each
// lane owns 4 consecutive experts); with `publish`, also the global counts
// and the number of pruned pairs.
// base needs E + 1 entries; offsets, counts and n_pruned are written only
// with `publish`.
static __device__ void scan_counts(int T, int E, int k, const int* cnt, int* base, int32_t* counts,
                                   int32_t* offsets, int32_t* n_pruned, bool publish = true) {
  const int lane = threadIdx.x & 63;
  int c[4], local = 0;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int e = 4 * lane + j;
    c[j] = e < E ? cnt[e] : 0;
    local += c[j];
  }
  int incl = local;
  for (int off = 1; off < 64; off <<= 1) {
    const int v = __shfl_up(incl, off);
    if (lane >= off) incl += v;
  }
  int run = incl - local;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int e = 4 * lane + j;
    if (e < E) {
      base[e] = run;
      if (publish) {
        offsets[e] = run;
        counts[e] = c[j];
      }
    }
    run += c[j];
  }
  if (lane == 63) {
    base[E] = incl;
    if (publish) {
      offsets[E] = incl;
      *n_pruned = T * k - incl;
    }
  }
}

// Routing scratch of a small batch (T <= kRouteFusedMaxT) in LDS.
struct RouteLds {
  uint16_t* ent;             // [T*k] kept expert of (t, r), 0xffff when pruned
  float* w;                  // [T*k] combine weight of (t, r)
  int* cnt;                  // [E]
  int* base;                 // [E+1] list start of each expert (exclusive scan)
  unsigned long long* bal;   // [E] tokens (bit t) routed to each expert
};

// Lists of a small batch from the selections in LDS (one wavefront, lane t =
// token t): every kept pair ORs its token's bit into its expert's mask (LDS
// atomics; an OR does not depend on the order), the masks give the counts,
// the counts' scan the list starts, and each kept pair goes to its expert's
// start plus the number of earlier tokens with that expert -- lists in token
// order.  With `publish` the routing outputs go to memory.
static __device__ void small_batch_lists(int T, int E, int k, const RouteLds& s, bool publish, int32_t* counts,
                                         int32_t* offsets, int32_t* pair_token, int32_t* pair_rank, float* pair_w,
                                         int32_t* pair_pos, int32_t* n_pruned) {
  const int lane = threadIdx.x & 63;
  const bool act = lane < T;
  int my_e[MC_MAX_TOPK];
#pragma unroll
  for (int r = 0; r < MC_MAX_TOPK; ++r) my_e[r] = (act && r < k) ? s.ent[lane * k + r] : 0xffff;
  for (int e = lane; e < E; e += 64) s.bal[e] = 0ull;
  __builtin_amdgcn_wave_barrier();
#pragma unroll
  for (int r = 0; r < MC_MAX_TOPK; ++r)
    if (my_e[r] != 0xffff) atomicOr(&s.bal[my_e[r]], 1ull << lane);
  __builtin_amdgcn_wave_barrier();
  for (int e = lane; e < E; e += 64) s.cnt[e] = __popcll(s.bal[e]);
  __builtin_amdgcn_wave_barrier();
  scan_counts(T, E, k, s.cnt, s.base, counts, offsets, n_pruned, publish);
  if (!publish) return;
  __builtin_amdgcn_wave_barrier();
  const unsigned long long below = (1ull << lane) - 1ull;
#pragma unroll
  for (int r = 0; r < MC_MAX_TOPK; ++r) {
    const int e = my_e[r];
    if (e != 0xffff) {
      const int pos = s.base[e] + __popcll(s.bal[e] & below);
      pair_token[pos] = lane;
      pair_rank[pos] = r;
      pair_w[pos] = s.w[lane * k + r];
      pair_pos[lane * k + r] = pos;
    }
  }
}

}  // namespace mc
