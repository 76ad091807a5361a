// route.hip -- top-k routing with Online Dynamic Pruning and token protection.
//
// Eq. 1: each token is sent to its top-k experts (largest logits; equal logits
// ordered by lower expert index), weighted by the softmax over the selected k.
// Eq. 5 (k = 2): the secondary expert is dropped when w1/w0 < mu, decided here
// as fp32(l0 - l1) > delta with delta = fp32(ln((1 - tau)/tau)), tau = mu/(1+mu);
// for k > 2 rank r >= 1 is dropped when its normalised weight is below tau
// (fp64).  Sec. 3.3.2: a protected token keeps every selected expert.  The
// kept weights are renormalised over the kept ranks.
//
// Selection (one wavefront per token): lanes hold the logits, every key's
// rank is counted against all keys broadcast in turn, lane r then evaluates
// rank r; the softmax sums add the ranks in order.
// Lists: per-expert token lists in ascending token order, built with ballots
// and popcount prefixes (list positions never depend on timing, so the lists
// are deterministic).  Small batches run both phases in one launch with
// everything kept in LDS; larger ones scatter by token blocks, each block
// counting the selections of all tokens (expert totals) and of the tokens
// before it (its start in each list).
#include "mc_internal.hpp"

namespace mc {

constexpr int kCsrThreads = 1024;
constexpr int kListBlocks = 64;     // at most this many token blocks scatter the lists
constexpr int kListMaxBlockT = 1024;
static_assert(kListBlocks * kListMaxBlockT >= MC_MAX_TOKENS, "list blocks cover every token");

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
// writes rank r's outputs; when s_ent/s_w are given it also records them in
// LDS (expert, or 0xffff if pruned).
__device__ void select_token(const float* __restrict__ logits, const uint8_t* __restrict__ important,
                             int t, int E, int k, float delta32, double tau,
                             int32_t* __restrict__ topk_idx, float* __restrict__ topk_w,
                             uint8_t* __restrict__ kept, int32_t* __restrict__ pair_pos,
                             uint16_t* s_ent, float* s_w) {
  const int lane = threadIdx.x & 63;
  const float* l = logits + (size_t)t * E;
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
  const int prot_flag = important != nullptr ? (int)important[t] : 0;
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
    topk_idx[o] = my_e;
    kept[o] = keep ? 1 : 0;
    topk_w[o] = w;
    if (!keep) pair_pos[o] = -1;
    if (s_ent) {
      s_ent[o] = keep ? (uint16_t)my_e : (uint16_t)0xffff;
      s_w[o] = w;
    }
  }
}

// Exclusive scan of cnt[0..E) into base[] and offsets[0..E] (one wave: each
// lane owns 4 consecutive experts); with `publish`, also the global counts
// and the number of pruned pairs.
__device__ void scan_counts(int T, int E, int k, const int* cnt, int* base, int32_t* counts, int32_t* offsets,
                            int32_t* n_pruned, bool publish = true) {
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
      offsets[e] = run;
      if (publish) counts[e] = c[j];
    }
    run += c[j];
  }
  if (lane == 63) {
    offsets[E] = incl;
    if (publish) *n_pruned = T * k - incl;
  }
}

// One pass over the tokens [c0, c0+nc) of expert e held in ent (LDS, indexed
// from token c0): counts (pass 0) or writes the list entries from run (pass 1).
__device__ __forceinline__ int list_pass(int pass, int e, int run, int c0, int nc, int k,
                                         const uint16_t* ent, const float* w_src, bool w_in_lds,
                                         const float* __restrict__ topk_w,
                                         int32_t* __restrict__ pair_token,
                                         int32_t* __restrict__ pair_rank, float* __restrict__ pair_w,
                                         int32_t* __restrict__ pair_pos) {
  const int lane = threadIdx.x & 63;
  for (int t0 = 0; t0 < nc; t0 += 64) {
    const int tl = t0 + lane;
    int rr = -1;
    if (tl < nc)
      for (int r = 0; r < k; ++r)
        if (ent[tl * k + r] == e) rr = r;
    const unsigned long long m = __ballot(rr >= 0);
    if (pass == 1 && rr >= 0) {
      const int pos = run + __popcll(m & ((1ull << lane) - 1ull));
      const int t = c0 + tl;
      pair_token[pos] = t;
      pair_rank[pos] = rr;
      pair_w[pos] = w_in_lds ? w_src[tl * k + rr] : topk_w[(size_t)t * k + rr];
      pair_pos[(size_t)t * k + rr] = pos;
    }
    run += __popcll(m);
  }
  return run;
}

__global__ void __launch_bounds__(256) route_select_kernel(const float* __restrict__ logits,
                                                           const uint8_t* __restrict__ important,
                                                           int T, int E, int k, float delta32,
                                                           double tau, int32_t* topk_idx,
                                                           float* topk_w, uint8_t* kept,
                                                           int32_t* pair_pos) {
  const int t = blockIdx.x * (blockDim.x >> 6) + wave_id();
  if (t >= T) return;
  select_token(logits, important, t, E, k, delta32, tau, topk_idx, topk_w, kept, pair_pos,
               nullptr, nullptr);
}

// Tokens per list block: a multiple of 64, at most kListBlocks blocks.
static int list_block_tokens(int T) {
  int bt = (T + kListBlocks - 1) / kListBlocks;
  bt = ((bt + 63) / 64) * 64;
  return bt < 64 ? 64 : bt;
}

// Lists for any T: workgroup b takes tokens [b*BT, (b+1)*BT).  Its histograms
// (LDS atomics; the counts, not their order, depend on them) give every
// expert's total and its entries before the block; block 0 publishes the
// counts and offsets.  The block's entries then go out in token order.
__global__ void __launch_bounds__(kCsrThreads) route_scatter_kernel(
    int T, int E, int k, int BT, const int32_t* __restrict__ topk_idx, const uint8_t* __restrict__ kept,
    const float* __restrict__ topk_w, int32_t* counts, int32_t* offsets, int32_t* pair_token,
    int32_t* pair_rank, float* pair_w, int32_t* pair_pos, int32_t* n_pruned) {
  __shared__ uint16_t ent[kListMaxBlockT * MC_MAX_TOPK];
  __shared__ int tot[MC_MAX_EXPERTS], pre[MC_MAX_EXPERTS], base[MC_MAX_EXPERTS];
  __shared__ int32_t offs[MC_MAX_EXPERTS + 1];
  const int tid = threadIdx.x, wave = wave_id(), nwaves = blockDim.x >> 6;
  const int t0 = blockIdx.x * BT;
  const int nc = (T - t0) < BT ? (T - t0) : BT;
  for (int e = tid; e < E; e += blockDim.x) tot[e] = pre[e] = 0;
  __syncthreads();
  const int n = T * k, n0 = t0 * k;
  for (int i = tid; i < n; i += blockDim.x) {
    if (kept[i]) {
      const int e = topk_idx[i];
      atomicAdd(&tot[e], 1);
      if (i < n0) atomicAdd(&pre[e], 1);
    }
  }
  for (int i = tid; i < nc * k; i += blockDim.x) {
    const size_t o = (size_t)n0 + i;
    ent[i] = kept[o] ? (uint16_t)topk_idx[o] : (uint16_t)0xffff;
  }
  __syncthreads();
  if (wave == 0) scan_counts(T, E, k, tot, base, counts, offs, n_pruned, blockIdx.x == 0);
  __syncthreads();
  if (blockIdx.x == 0)
    for (int e = tid; e <= E; e += blockDim.x) offsets[e] = offs[e];
  for (int e = wave; e < E; e += nwaves)
    list_pass(1, e, base[e] + pre[e], t0, nc, k, ent, nullptr, false, topk_w, pair_token, pair_rank,
              pair_w, pair_pos);
}

// Small batches (T <= kRouteFusedMaxT = 64): one launch.  The waves select
// tokens in parallel (the selection kept in LDS); then wave 0, one lane per
// token, forms each token's mask of kept experts, counts every expert's
// tokens with one ballot per expert (the ballots kept in LDS), scans the
// counts, and writes each kept pair at its expert's offset plus the number of
// earlier tokens with that expert -- lists in token order, no atomics.
__global__ void __launch_bounds__(kCsrThreads) route_fused_kernel(
    const float* __restrict__ logits, const uint8_t* __restrict__ important, int T, int E, int k,
    float delta32, double tau, int32_t* topk_idx, float* topk_w, uint8_t* kept, int32_t* counts,
    int32_t* offsets, int32_t* pair_token, int32_t* pair_rank, float* pair_w, int32_t* pair_pos,
    int32_t* n_pruned) {
  static_assert(kRouteFusedMaxT <= 64, "one lane per token");
  __shared__ uint16_t ent[kRouteFusedMaxT * MC_MAX_TOPK];
  __shared__ float wsel[kRouteFusedMaxT * MC_MAX_TOPK];
  __shared__ int cnt[MC_MAX_EXPERTS];
  __shared__ int base[MC_MAX_EXPERTS];
  __shared__ unsigned long long bal[MC_MAX_EXPERTS];
  const int wave = wave_id(), nwaves = blockDim.x >> 6, lane = threadIdx.x & 63;
  for (int t = wave; t < T; t += nwaves)
    select_token(logits, important, t, E, k, delta32, tau, topk_idx, topk_w, kept, pair_pos, ent,
                 wsel);
  __syncthreads();
  if (wave != 0) return;
  const bool act = lane < T;
  int my_e[MC_MAX_TOPK];
  unsigned long long m[MC_MAX_EXPERTS / 64] = {0ull, 0ull, 0ull, 0ull};
#pragma unroll
  for (int r = 0; r < MC_MAX_TOPK; ++r) {
    my_e[r] = 0xffff;
    if (act && r < k) {
      const int e = ent[lane * k + r];
      my_e[r] = e;
      if (e != 0xffff) {
        const unsigned long long bit = 1ull << (e & 63);
#pragma unroll
        for (int j = 0; j < MC_MAX_EXPERTS / 64; ++j) m[j] |= (e >> 6) == j ? bit : 0ull;
      }
    }
  }
  for (int e = lane; e < E; e += 64) cnt[e] = 0;
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
        cnt[64 * j + i] = __popcll(b);
        bal[64 * j + i] = b;
      }
    }
  }
  scan_counts(T, E, k, cnt, base, counts, offsets, n_pruned);
  const unsigned long long below = (1ull << lane) - 1ull;
#pragma unroll
  for (int r = 0; r < MC_MAX_TOPK; ++r) {
    const int e = my_e[r];
    if (e != 0xffff) {
      const int pos = base[e] + __popcll(bal[e] & below);
      pair_token[pos] = lane;
      pair_rank[pos] = r;
      pair_w[pos] = wsel[lane * k + r];
      pair_pos[lane * k + r] = pos;
    }
  }
}

hipError_t launch_route(const float* logits, const uint8_t* important, float delta32, double tau,
                        const mc_routing& r, hipStream_t stream) {
  if (r.T <= kRouteFusedMaxT) {
    timing_begin(stream, kSiteRouteFused);
    hipLaunchKernelGGL(route_fused_kernel, dim3(1), dim3(kCsrThreads), 0, stream, logits,
                       important, r.T, r.E, r.k, delta32, tau, r.topk_idx, r.topk_w, r.kept,
                       r.counts, r.offsets, r.pair_token, r.pair_rank, r.pair_w, r.pair_pos,
                       r.n_pruned);
    timing_end(stream, kSiteRouteFused);
    return hipGetLastError();
  }
  timing_begin(stream, kSiteRouteSelect);
  hipLaunchKernelGGL(route_select_kernel, dim3((r.T + 3) / 4), dim3(256), 0, stream, logits,
                     important, r.T, r.E, r.k, delta32, tau, r.topk_idx, r.topk_w, r.kept,
                     r.pair_pos);
  timing_end(stream, kSiteRouteSelect);
  hipError_t err = hipGetLastError();
  if (err != hipSuccess) return err;
  timing_begin(stream, kSiteRouteLists);
  const int bt = list_block_tokens(r.T);
  hipLaunchKernelGGL(route_scatter_kernel, dim3((r.T + bt - 1) / bt), dim3(kCsrThreads), 0, stream, r.T, r.E,
                     r.k, bt, r.topk_idx, r.kept, r.topk_w, r.counts, r.offsets, r.pair_token, r.pair_rank,
                     r.pair_w, r.pair_pos, r.n_pruned);
  timing_end(stream, kSiteRouteLists);
  return hipGetLastError();
}

}  // namespace mc
