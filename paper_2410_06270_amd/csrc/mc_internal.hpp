// mc_internal.hpp -- launchers shared between the kernel files and the C-ABI.
#pragma once

#include "mc_device.hpp"

namespace mc {

constexpr int kRouteFusedMaxT = 64;    // up to this many tokens routing may run in one launch
constexpr int kDecodeMaxT = 64;        // up to this many tokens one workgroup holds all of an expert's tokens

enum TimingSite {
  kSitePackSz, kSitePackCodes, kSiteExport, kSiteRouteFused, kSiteRouteSelect, kSiteRouteLists,
  kSiteGateUp, kSiteDown, kSiteCombine, kSitePrefillPrep, kSiteImpColsum, kSiteImpFinish, kSiteImpSelect,
  kSiteRmsNorm, kSiteRouter, kSiteGptqHessian, kSiteGptqFactor, kSiteGptqQuantize,
  kNumSites
};
void timing_begin(hipStream_t stream, int site);
void timing_end(hipStream_t stream, int site);
int timing_site(const char* name);
hipError_t timing_read(int site, double* total_ms, int* launches);
void timing_enable(int on);

// any_sign: some expert of L.sign_mask is sign-binarized.
hipError_t launch_pack(const float* wg, const float* wu, const float* wd, const LayerArgs& L,
                       uint32_t* words, uint32_t* sz, bool any_sign, hipStream_t stream);
hipError_t launch_export(const uint32_t* words, const uint32_t* sz, int bits, int R, int K, int G,
                         bool dequant, void* out, hipStream_t stream);
hipError_t launch_route(const float* logits, const uint8_t* important, float delta32, double tau,
                        const mc_routing& r, hipStream_t stream);
// The device buffers of one routing result (those of mc_routing).
struct RouteBufs {
  int32_t* topk_idx;
  float* topk_w;
  uint8_t* kept;
  int32_t *counts, *offsets, *pair_token, *pair_rank;
  float* pair_w;
  int32_t *pair_pos, *n_pruned;
};
constexpr int kRouteBatch = 8;          // batches routed by one launch_route_batch
struct RouteBatch {
  RouteBufs r[kRouteBatch];
};
// Whether launch_route_batch takes batches of T tokens over E experts (the
// one-workgroup routing of small batches).
bool route_batch_fits(int T, int E);
// Routes nb <= kRouteBatch batches of the same shape (rs[b].T, E, k equal) in
// one launch: batch b's logits at logits + b*T*E, its flags at important +
// b*T (or none), its results into rs[b] as launch_route writes them.
hipError_t launch_route_batch(const float* logits, const uint8_t* important, float delta32, double tau,
                              const mc_routing* rs, int nb, hipStream_t stream);
// Bytes of one set of routing buffers for T tokens (each buffer 256-aligned),
// and the set laid out at base.
size_t routing_set_bytes(int T, int E, int k);
mc_routing routing_set(void* base, int T, int E, int k);
int forward_nsplit(int T, int E, int k, int d, int ffn);
int forward_ksplit(int T, int E, int k, int d, int ffn);
size_t forward_workspace_bytes(int T, int E, int k, int d, int ffn);
// Workspace of the prefill path (byte offsets): expert tile tables, the
// fragment-tiled copies of the routed x rows (bf16) and of h (fp16) with their
// 32-column sums, and the fp32 down partials [nsplit][T*k][d].
struct PrefillLayout {
  size_t tables, x, xsum, h, hsum, part, total;
  int f_max, mt_max, nsplit;
};
PrefillLayout prefill_layout(int T, int E, int k, int d, int ffn);
hipError_t launch_prefill(const uint16_t* x, const LayerArgs& L, const mc_routing& r, void* ws,
                          float** partial, size_t* part_stride, int* nsplit, hipStream_t stream);
// Routing inputs of a forward call that routes its batch first (the outputs
// go to the mc_routing buffers as mc_route_and_prune writes them).
struct RouteArgs {
  const float* logits;       // [T][E]
  const uint8_t* important;  // [T] or null
  float delta32;             // fp32 logit-gap threshold (k = 2)
  double tau;                // normalised-weight threshold (k > 2)
};
// The expert outputs of every kept pair, unweighted and split over the
// reduction: partial[s][pos][0..d) for s < nsplit, pos the pair's CSR
// position (the forward's workspace holds them; launch_forward combines them).
hipError_t launch_expert_partials(const uint16_t* x, const LayerArgs& L, const mc_routing& r, void* ws,
                                  float** partial, size_t* part_stride, int* nsplit, hipStream_t stream);
// The reconstruction error of Sec. 3.2.2 (pmq.hip): the dense fp32 expert
// outputs of every kept pair (h [P][ffn], y [P][d], fp32 weights [E][N][K]),
// and eps[e][b-1] from the packed forward's per-pair partials against them.
hipError_t launch_dense_expert(const float* wg, const float* wu, const float* wd, int E, int d, int ffn,
                               const uint16_t* x, const mc_routing& r, float* h, float* y, hipStream_t stream);
hipError_t launch_pmq_error(const float* partial, size_t part_stride, int nsplit, const float* dense,
                            const mc_routing& r, int d, int b, double* eps, hipStream_t stream);
// residual (may be null): y = bf16(residual + sum_r w_r E_{e_r}(x)).
// route (may be null): route the batch first (the routing kernels).
// xn_next (may be null): also write RMSNorm(y) there, the next stack layer's
// input (the combine forms it; the bytes of a separate rmsnorm launch).
hipError_t launch_forward(const uint16_t* x, const LayerArgs& L, const mc_routing& r, uint16_t* y,
                          void* ws, const uint16_t* residual, hipStream_t stream,
                          const RouteArgs* route = nullptr,
                          uint16_t* xn_next = nullptr);
// Stack of layers: xn = RMSNorm(h) (fp64, one bf16 rounding) before each layer.
constexpr double kRmsNormEps = 1e-5;
hipError_t launch_rmsnorm(const uint16_t* h, int T, int d, double eps, uint16_t* xn, hipStream_t stream);
// xn [T][d], the routing sets of kRouteBatch layers when route_batch_fits,
// and the forward workspace.
size_t stack_workspace_bytes(int T, int E, int k, int d, int ffn);
// logits [T][E] fp32 = x [T][d] . w [E][d]^T (bf16), fp64 sums rounded once.
hipError_t launch_router(const uint16_t* x, const uint16_t* w, int T, int d, int E, float* logits,
                         hipStream_t stream);
// GPTQ (fp64): H (+)= 2 X^T X; the factor U (upper Cholesky of the damped
// H^-1) with the dead-input mask; in-order quantization into one matrix's
// packed words and scale/zero words.
size_t gptq_factor_bytes(int K);
size_t gptq_quantize_bytes(int R, int K);
hipError_t launch_gptq_hessian(const uint16_t* x, int N, int K, double* H, bool accumulate, hipStream_t st);
hipError_t launch_gptq_factor(const double* H, int K, double damp, double* U, uint8_t* dead, void* ws,
                              hipStream_t st);
hipError_t launch_gptq_quantize(const float* W, const double* U, const uint8_t* dead, int R, int K, int bits, int G,
                                uint32_t* words, uint32_t* sz, double* loss, void* ws, hipStream_t st);
size_t importance_workspace_bytes(int H, int L);
hipError_t launch_importance(const uint16_t* attn, int H, int L, const uint16_t* x, int d, float rho,
                             float* importance, uint8_t* mask, void* ws, hipStream_t stream);

}  // namespace mc
