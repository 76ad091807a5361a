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
// Selection (one segment of S lanes per token, S the power of two covering
// the experts, 64/S tokens per wavefront): lanes hold the logits, every key's
// rank is counted against the segment's keys in turn, lane r then evaluates
// rank r; the softmax sums add the ranks in order.
// Lists: per-expert token lists in ascending token order, built with ballots
// and popcount prefixes (list positions never depend on timing, so the lists
// are deterministic).  Small batches run both phases in one launch with
// everything kept in LDS; larger ones scatter by token blocks, each block
// counting the selections of all tokens (expert totals) and of the tokens
// before it (its start in each list).
#include "route_device.hpp"

namespace mc {

constexpr int kCsrThreads = 1024;
constexpr int kListBlocks = 64;     // at most this many token blocks scatter the lists
constexpr int kListMaxBlockT = 1024;
static_assert(kListBlocks * kListMaxBlockT >= MC_MAX_TOKENS, "list blocks cover every token");

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
                                                           int T, int E, int S, int k, float delta32,
                                                           double tau, int32_t* topk_idx,
                                                           float* topk_w, uint8_t* kept,
                                                           int32_t* pair_pos) {
  __shared__ __attribute__((aligned(16))) unsigned char scratch[4][kSelScratchBytes];
  const int lane = threadIdx.x & 63, ns = 64 / S;
  const int t0 = (blockIdx.x * (blockDim.x >> 6) + wave_id()) * ns;
  if (t0 >= T) return;
  const int t = t0 + lane / S;
  const SelInput in = sel_load(logits, important, t, T, E, S);
  select_token(in, t, T, E, S, k, delta32, tau, topk_idx, topk_w, kept, pair_pos, true, nullptr, nullptr,
               sel_scratch(scratch[wave_id()]));
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
  __shared__ int tot[MC_MAX_EXPERTS], pre[MC_MAX_EXPERTS], base[MC_MAX_EXPERTS + 1];
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

// Small batches run in one launch: at most kRouteFusedMaxT tokens (a lane per
// token in the lists) that one round of the workgroup's 16 waves selects
// (64/S tokens a wave; measured: 64 experts, 16 tokens: 8.6 us against 11.0
// in two launches).  With more than 64 experts a lane ranks several keys and
// a selection is slower: there T * E <= 512 (as measured at 64 experts before
// the ranks were batched: 32 tokens took 20 us against 11.5 in two launches).
// Larger batches spread the selections over many CUs.
__host__ __device__ constexpr bool route_fused_fits(int T, int E) {
  return T <= kRouteFusedMaxT && (E <= 64 ? T <= (kCsrThreads / 64) * (64 / sel_segment(E)) : T * E <= 512);
}

// The small-batch routing of one batch (a workgroup): the waves select the
// tokens side by side (the selections kept in LDS), then wave 0 builds the
// lists (small_batch_lists).
__device__ __forceinline__ void route_fused_body(const float* __restrict__ logits,
                                                 const uint8_t* __restrict__ important, int T, int E, int k,
                                                 float delta32, double tau, const RouteBufs& o) {
  static_assert(kRouteFusedMaxT <= 64, "one lane per token");
  __shared__ uint16_t ent[kRouteFusedMaxT * MC_MAX_TOPK];
  __shared__ float wsel[kRouteFusedMaxT * MC_MAX_TOPK];
  __shared__ int cnt[MC_MAX_EXPERTS];
  __shared__ int base[MC_MAX_EXPERTS + 1];
  __shared__ unsigned long long bal[MC_MAX_EXPERTS];
  __shared__ __attribute__((aligned(16))) unsigned char scratch[kCsrThreads / 64][kSelScratchBytes];
  const int wave = wave_id(), nwaves = blockDim.x >> 6;
  const SelScratch sc = sel_scratch(scratch[wave]);
  const int S = sel_segment(E), ns = 64 / S;
  // a wave selects ns tokens at once; route_fused_fits makes one round of
  // the 16 waves enough
  for (int t0 = wave * ns; t0 < T; t0 += nwaves * ns) {
    const int t = t0 + (threadIdx.x & 63) / S;
    const SelInput in = sel_load(logits, important, t, T, E, S);
    select_token(in, t, T, E, S, k, delta32, tau, o.topk_idx, o.topk_w, o.kept, o.pair_pos, true, ent, wsel,
                 sc);
  }
  __syncthreads();
  if (wave != 0) return;
  const RouteLds s{ent, wsel, cnt, base, bal};
  small_batch_lists(T, E, k, s, true, o.counts, o.offsets, o.pair_token, o.pair_rank, o.pair_w, o.pair_pos,
                    o.n_pruned);
}

__global__ void __launch_bounds__(kCsrThreads) route_fused_kernel(
    const float* __restrict__ logits, const uint8_t* __restrict__ important, int T, int E, int k,
    float delta32, double tau, RouteBufs o) {
  route_fused_body(logits, important, T, E, k, delta32, tau, o);
}

// Several batches of the same shape at once, one workgroup each: batch b's
// logits at logits + b*T*E, its flags at important + b*T (the layers of a
// stack, whose routing depends only on their own logits).
__global__ void __launch_bounds__(kCsrThreads) route_fused_batch_kernel(
    const float* __restrict__ logits, const uint8_t* __restrict__ important, int T, int E, int k,
    float delta32, double tau, RouteBatch o) {
  const size_t b = blockIdx.x;
  route_fused_body(logits + b * T * E, important ? important + b * T : nullptr, T, E, k, delta32, tau,
                   o.r[b]);
}

static RouteBufs route_bufs(const mc_routing& r) {
  return RouteBufs{r.topk_idx, r.topk_w, r.kept, r.counts, r.offsets, r.pair_token, r.pair_rank, r.pair_w,
                   r.pair_pos, r.n_pruned};
}

bool route_batch_fits(int T, int E) { return route_fused_fits(T, E); }

hipError_t launch_route_batch(const float* logits, const uint8_t* important, float delta32, double tau,
                              const mc_routing* rs, int nb, hipStream_t stream) {
  if (nb < 1 || nb > kRouteBatch || !route_fused_fits(rs[0].T, rs[0].E)) return hipErrorInvalidValue;
  RouteBatch o;
  for (int b = 0; b < nb; ++b) o.r[b] = route_bufs(rs[b]);
  timing_begin(stream, kSiteRouteFused);
  hipLaunchKernelGGL(route_fused_batch_kernel, dim3(nb), dim3(kCsrThreads), 0, stream, logits, important,
                     rs[0].T, rs[0].E, rs[0].k, delta32, tau, o);
  timing_end(stream, kSiteRouteFused);
  return hipGetLastError();
}

hipError_t launch_route(const float* logits, const uint8_t* important, float delta32, double tau,
                        const mc_routing& r, hipStream_t stream) {
  if (route_fused_fits(r.T, r.E)) {
    timing_begin(stream, kSiteRouteFused);
    hipLaunchKernelGGL(route_fused_kernel, dim3(1), dim3(kCsrThreads), 0, stream, logits,
                       important, r.T, r.E, r.k, delta32, tau, route_bufs(r));
    timing_end(stream, kSiteRouteFused);
    return hipGetLastError();
  }
  timing_begin(stream, kSiteRouteSelect);
  const int S = sel_segment(r.E), per_wg = 4 * (64 / S);   // tokens per workgroup
  hipLaunchKernelGGL(route_select_kernel, dim3((r.T + per_wg - 1) / per_wg), dim3(256), 0, stream, logits,
                     important, r.T, r.E, S, r.k, delta32, tau, r.topk_idx, r.topk_w, r.kept, r.pair_pos);
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
