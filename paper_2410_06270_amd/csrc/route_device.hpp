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

// Selects and prunes token t (one wavefront).  Lanes hold the logits (lane l
// has experts l, l+64, ...) as distinct 64-bit keys (ordered logit bits, then
// the complement of the expert index, so larger key = earlier rank); each
// key's rank is the number of larger keys, counted against every key
// broadcast in turn (no cross-lane reductions).  Lane r < k then takes rank r
// and evaluates it; the softmax sums run over the ranks in order.  Lane r < k
// writes rank r's outputs (when `publish`); when s_ent/s_w are given it also
// records them in LDS (expert, or 0xffff if pruned).  l: the token's E logits
// and prot_src: its protection flag (NULL: unprotected), in memory or LDS.
static __device__ void select_token(const float* l, const uint8_t* prot_src, int t, int E, int k, float delta32,
                                    double tau, int32_t* __restrict__ topk_idx, float* __restrict__ topk_w,
                                    uint8_t* __restrict__ kept, int32_t* __restrict__ pair_pos, bool publish,
                                    uint16_t* s_ent, float* s_w) {
  const int lane = threadIdx.x & 63;
  const int nj = (E + 63) >> 6;                      // logits per lane (wave-uniform)
  float lv[4];
  unsigned long long key[4];
  int rank[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int e = lane + 64 * j;
    lv[j] = (e < E) ? l[e] : 0.0f;
  }
  // the protection flag is loaded beside the logits (one memory round trip)
  const int prot_flag = prot_src != nullptr ? (int)*prot_src : 0;
  asm volatile("" ::"v"(lv[0]), "v"(lv[1]), "v"(lv[2]), "v"(lv[3]), "v"(prot_flag));
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int e = lane + 64 * j;
    key[j] = (e < E) ? (((unsigned long long)ordered_bits(lv[j]) << 32) | (unsigned)(0xffff - e)) : 0ull;
    rank[j] = 0;
  }
  for (int sj = 0; sj < nj; ++sj) {
    const int n = (E - 64 * sj) < 64 ? (E - 64 * sj) : 64;
    const unsigned long long ks = sj == 0 ? key[0] : sj == 1 ? key[1] : sj == 2 ? key[2] : key[3];
    const uint32_t khs = (uint32_t)(ks >> 32), kls = (uint32_t)ks;
    int src = 0;
    for (; src + 4 <= n; src += 4) {
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const unsigned long long o =
            ((unsigned long long)__builtin_amdgcn_readlane(khs, src + u) << 32) |
            __builtin_amdgcn_readlane(kls, src + u);
#pragma unroll
        for (int j = 0; j < 4; ++j)
          if (j < nj) rank[j] += o > key[j] ? 1 : 0;
      }
    }
    for (; src < n; ++src) {
      const unsigned long long o =
          ((unsigned long long)__builtin_amdgcn_readlane(khs, src) << 32) | __builtin_amdgcn_readlane(kls, src);
#pragma unroll
      for (int j = 0; j < 4; ++j)
        if (j < nj) rank[j] += o > key[j] ? 1 : 0;
    }
  }
  const bool prot = prot_flag != 0;
  int my_e = 0;
  float my_l = 0.0f;
  float l0 = 0.0f, l1 = 0.0f;
  for (int r = 0; r < k; ++r) {
    int e = 0;
    float le = 0.0f;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      if (j < nj) {
        const unsigned long long b = __ballot(rank[j] == r);
        if (b) {
          const int src = __ffsll((long long)b) - 1;
          e = 64 * j + src;
          le = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(uint32_t, lv[j]), src));
        }
      }
    }
    if (r == 0) l0 = le;
    if (r == 1) l1 = le;
    if (lane == r) {
      my_e = e;
      my_l = le;
    }
  }
  if (k < 2) l1 = l0;
  const bool mine = lane < k;
  const double ex = mine ? exp((double)my_l - (double)l0) : 0.0;
  double sum_all = 0.0;
  for (int r = 0; r < k; ++r) sum_all += readlane_f64(ex, r);
  bool keep = mine;
  if (mine && lane > 0 && !prot) {
    if (k == 2) {
      const float gap = l0 - l1;
      keep = !(gap > delta32);
    } else {
      keep = !(ex < tau * sum_all);
    }
  }
  const unsigned long long kb = __ballot(keep);
  double sum_kept = 0.0;
  for (int r = 0; r < k; ++r)
    if ((kb >> r) & 1ull) sum_kept += readlane_f64(ex, r);
  if (mine) {
    const size_t o = (size_t)t * k + lane;
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
// token t): every token's mask of kept experts, one ballot per selected expert
// (the tokens that chose it), the counts' scan, then each kept pair at its
// expert's offset plus the number of earlier tokens with that expert -- lists
// in token order, no atomics.  With `publish` the routing outputs go to memory.
static __device__ void small_batch_lists(int T, int E, int k, const RouteLds& s, bool publish, int32_t* counts,
                                         int32_t* offsets, int32_t* pair_token, int32_t* pair_rank, float* pair_w,
                                         int32_t* pair_pos, int32_t* n_pruned) {
  const int lane = threadIdx.x & 63;
  const bool act = lane < T;
  int my_e[MC_MAX_TOPK];
  unsigned long long m[MC_MAX_EXPERTS / 64] = {0ull, 0ull, 0ull, 0ull};
#pragma unroll
  for (int r = 0; r < MC_MAX_TOPK; ++r) {
    my_e[r] = 0xffff;
    if (act && r < k) {
      const int e = s.ent[lane * k + r];
      my_e[r] = e;
      if (e != 0xffff) {
        const unsigned long long bit = 1ull << (e & 63);
#pragma unroll
        for (int j = 0; j < MC_MAX_EXPERTS / 64; ++j) m[j] |= (e >> 6) == j ? bit : 0ull;
      }
    }
  }
  for (int e = lane; e < E; e += 64) {
    s.cnt[e] = 0;
    s.bal[e] = 0ull;
  }
#pragma unroll
  for (int j = 0; j < MC_MAX_EXPERTS / 64; ++j) {
    if (64 * j >= E) break;
    // experts of this 64-block that some token selected (OR over the lanes)
    unsigned long long any = m[j];
    for (int off = 1; off < 64; off <<= 1) {
      const uint32_t lo = __shfl_xor((uint32_t)any, off), hi = __shfl_xor((uint32_t)(any >> 32), off);
      any |= ((unsigned long long)hi << 32) | lo;
    }
    any = ((unsigned long long)__builtin_amdgcn_readfirstlane((uint32_t)(any >> 32)) << 32) |
          __builtin_amdgcn_readfirstlane((uint32_t)any);
    while (any) {
      const int i = __ffsll((long long)any) - 1;
      any &= any - 1ull;
      const unsigned long long b = __ballot((m[j] >> i) & 1ull);
      if (lane == 0) {
        s.cnt[64 * j + i] = __popcll(b);
        s.bal[64 * j + i] = b;
      }
    }
  }
  scan_counts(T, E, k, s.cnt, s.base, counts, offsets, n_pruned, publish);
  if (!publish) return;
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
