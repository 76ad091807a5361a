/*
 * mc_moe.h -- C-ABI of the Mixture Compressor (MC) MoE expert path on gfx950.
 *
 * The paper (Mixture Compressor for MoE LLMs, ICLR 2025) stores every expert
 * at its own 1-, 2- or 3-bit width (Sec. 3.2, Eq. 4 chooses the widths) with
 * asymmetric, group-wise uniform quantization (Sec. 3.1), and at inference
 * prunes a token's low-weight experts unless the token is marked important
 * (Sec. 3.3, Eq. 5 and the token-protection rule).  This library runs that
 * inference path:
 *
 *   mc_pack            fp32 expert weights -> packed codes + fp16 scale/zero
 *   mc_gptq_*          GPTQ quantization of one matrix into the packed layer
 *   mc_router_logits   the router's linear layer: x -> router logits
 *   mc_route_and_prune router logits -> top-k, Eq. 5 pruning, protection,
 *                      per-expert token lists (CSR)
 *   mc_moe_forward     Eq. 1 over the packed SwiGLU experts
 *   mc_moe_route_forward  routing and Eq. 1 in one call
 *   mc_moe_stack_forward  a stack of MoE layers with residual connections
 *   mc_token_importance   Eq. 6 token importance -> the protected set
 *   mc_odp_threshold, mc_pmq_significance, mc_pmq_allocate
 *                      host helpers: the pruning threshold, expert
 *                      significance and the Eq. 4 width allocation
 *   mc_pmq_error_workspace, mc_pmq_expert_error
 *                      the per-expert, per-width reconstruction error the
 *                      Eq. 4 allocation takes, on the device
 *
 * Conventions for every call
 *   - Pointers are DEVICE pointers unless the comment says "host".
 *   - Every call that takes `stream` (a hipStream_t; NULL = legacy default
 *     stream) is asynchronous: it enqueues kernels and returns.
 *   - The library never allocates device memory.  The caller owns every
 *     buffer; sizes come from mc_pack_sizes / mc_forward_workspace.
 *   - Arguments are validated on the host before anything is enqueued.  On any
 *     status other than MC_OK nothing was enqueued (MC_EHIP: a launch failed;
 *     earlier launches of the same call may have been enqueued) and
 *     mc_last_error() describes the problem.
 *   - Shape limits: 1 <= E <= 256 experts, 1 <= k <= min(E, 8), d and ffn
 *     multiples of 128 with d*ffn <= 2^31, group size G one of 32, 64, 128
 *     (other multiples of 32 give MC_EUNSUPPORTED).
 *
 * Packed layout (normative; used by every kernel).  A matrix with R output
 * rows and K input columns (row-major W[R][K], the reduction runs over K) at
 * b bits is cut into tiles of 16 rows x 128 columns.  Column k of row n lives
 * in tile (n/16, k/128) at lane l = (n%16) + 16*kq, with kk = k%128,
 * u = kk/32, kq = (kk%32)/8, j = kk%8, pair i = 4u + j/2 and half
 * h = j%2 (0: bits 0..15, 1: bits 16..31).  Each lane owns b consecutive
 * 32-bit words starting at word ((tile_row*(K/128) + tile_col)*64 + l)*b:
 *   b = 1: bit 16h + i of word 0;
 *   b = 2: bits 16h + 2(i%8) .. +1 of word i/8;
 *   b = 3: i < 15: bits 16h + 3(i%5) .. +2 of word i/5;
 *          i = 15: bit p of the code sits at bit 16h + 15 of word p.
 * Scale and zero of group g of row n form one 32-bit word (fp16 scale in
 * bits 0..15, fp16 zero in bits 16..31) at index ((n/16)*(K/G) + g)*16 + n%16.
 * A layer holds, expert after expert, the gate [ffn][d], up [ffn][d] and
 * down [d][ffn] matrices in that order, each with its expert's width; the
 * scale/zero words follow the same order.
 */
#ifndef MC_MOE_H
#define MC_MOE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define MC_MAX_EXPERTS 256
#define MC_MAX_TOPK 8
#define MC_MAX_TOKENS 65536   /* tokens per routing call (MC_EUNSUPPORTED above) */

typedef enum mc_status {
  MC_OK = 0,
  MC_EINVAL = 1,        /* bad argument (shape, null pointer, bit-width, threshold) */
  MC_ENOSPACE = 2,      /* a caller buffer is smaller than required */
  MC_EHIP = 3,          /* the HIP runtime reported an error */
  MC_EUNSUPPORTED = 4   /* valid in principle, not supported by this build */
} mc_status;

/* Descriptor of one packed MoE layer; it only references caller memory. */
typedef struct mc_layer {
  int E;                 /* number of experts */
  int d;                 /* hidden size (input of gate/up, output of down) */
  int ffn;               /* expert intermediate size */
  int group;             /* quantization group size G along the input dim */
  const int *bits_host;  /* host [E]; expert e is stored at bits_host[e] in {1,2,3} */
  void *words;           /* device; packed codes, words_bytes long */
  uint32_t *sz;          /* device; scale/zero words, sz_bytes long */
  size_t words_bytes;
  size_t sz_bytes;
} mc_layer;

/* Bytes needed for the packed codes and the scale/zero words of a layer.
 * codes: sum over experts of 3*d*ffn*bits/8;  scale/zero: 3*E*d*ffn/G*4.
 * Pure host computation.  Errors: MC_EINVAL on a shape or width outside the
 * limits above or a null pointer. */
mc_status mc_pack_sizes(int E, int d, int ffn, const int *bits_host, int group,
                        size_t *words_bytes, size_t *sz_bytes);

/* Quantize and pack all experts of a layer (Sec. 3.1: uniform asymmetric
 * group-wise quantizer; the widths come from the PMQ allocation of Eq. 4).
 * For each group of G consecutive inputs of one row, with L = 2^b - 1:
 *   s = fp16(fp32(fp32(max - min) / L)), replaced by 1 if it rounds to 0;
 *   z = fp16(fp32(-min / s)), a -0 zero is stored as +0;
 *   code q = the j in [0, L] whose level s*(j - z) is nearest to w, ties to
 *   even j (decided exactly);
 * fp16() is round-to-nearest-even, saturating to +-65504.
 * w_gate, w_up: [E][ffn][d] fp32; w_down: [E][d][ffn] fp32; all weights must
 * be finite.  L->words / L->sz receive the layout described above.
 * Errors: MC_EINVAL (shape/width/null), MC_ENOSPACE (L->words_bytes or
 * L->sz_bytes smaller than mc_pack_sizes), MC_EHIP. */
mc_status mc_pack(const float *w_gate, const float *w_up, const float *w_down,
                  const mc_layer *L, void *stream);

/* Quantization method per expert for mc_pack_methods. */
#define MC_QUANT_RTN 0    /* the min-max round-to-nearest quantizer of mc_pack */
#define MC_QUANT_SIGN 1   /* 1-bit sign binarization (appendix A.2, Eq. 7-9) */

/* mc_pack with a method per expert (method_host: host [E], NULL = all RTN).
 * MC_QUANT_SIGN (1-bit experts only): code = 1 where w >= 0, else 0 (sign(0)
 * = +1), and every group of each of the expert's matrices stores
 *   s = fp16(2 * ||W||_1 / (rows * cols)),  z = 1/2,
 * so the dequantized weight s*(code - z) is +-||W||_1 / (rows * cols): the
 * binarized matrix times its scale (Eq. 7-9), and the forward computes
 * s * (sum of x where code = 1 - sum of x where code = 0), Eq. 10.  ||W||_1
 * is summed in fp64 (fixed order) and rounded once; 2*mean|W| above 65504
 * saturates.  The layout is that of mc_pack; every other call is unchanged.
 * Errors: as mc_pack, plus MC_EINVAL for an unknown method or a sign method
 * on an expert wider than 1 bit. */
mc_status mc_pack_methods(const float *w_gate, const float *w_up, const float *w_down,
                          const mc_layer *L, const int *method_host, void *stream);

/* Test surface: write the dequantized matrix `mat` (0 gate, 1 up, 2 down) of
 * expert e as row-major fp16 [R][K]; each value is the round-to-nearest-even
 * fp16 of the exact product s*(q - z) (one rounding).  out must hold R*K
 * halves.  Errors: MC_EINVAL, MC_EHIP. */
mc_status mc_dequant_export(const mc_layer *L, int e, int mat, uint16_t *out,
                            void *stream);

/* Test surface: write the integer codes of matrix `mat` of expert e as
 * row-major uint8 [R][K].  Errors: MC_EINVAL, MC_EHIP. */
mc_status mc_codes_export(const mc_layer *L, int e, int mat, uint8_t *out,
                          void *stream);

/* Routing result, device-resident; the host ints give its shape. */
typedef struct mc_routing {
  int T, E, k;           /* host: tokens, experts, experts per token */
  int32_t *topk_idx;     /* [T][k] rank r's expert: logits in descending order,
                            equal logits ordered by lower expert index */
  float *topk_w;         /* [T][k] combine weight of rank r after pruning
                            (softmax over the kept ranks), 0 when dropped */
  uint8_t *kept;         /* [T][k] 1 when (t, r) is computed, 0 when pruned */
  int32_t *counts;       /* [E] kept pairs per expert */
  int32_t *offsets;      /* [E+1] exclusive scan of counts */
  int32_t *pair_token;   /* [T*k]; entries offsets[e]..offsets[e+1]-1 list the
                            tokens routed to e in ascending order */
  int32_t *pair_rank;    /* [T*k] the rank r of each listed pair */
  float *pair_w;         /* [T*k] its combine weight */
  int32_t *pair_pos;     /* [T][k] list position of (t, r), -1 when pruned */
  int32_t *n_pruned;     /* [1] number of pruned pairs */
} mc_routing;

/* GPTQ, the quantizer the paper applies to the experts (Sec. 3.1: Hessian
 * H = 2 X^T X of the layer-wise squared error ||W X^T - Q X^T||^2, columns
 * quantized in order, each column's error compensated on the columns after
 * it), producing the same packed format as mc_pack.  Offline; all arithmetic
 * fp64; deterministic.  For a matrix W [R][K] (R outputs, K inputs) with
 * calibration inputs X [N][K]:
 *
 *   mc_gptq_hessian   H = 2 X^T X (accumulate = 0) or H += 2 X^T X
 *                     (accumulate != 0, for calibration sets in pieces).
 *                     x_bf16: [N][K] bf16; H: [K][K] fp64 (8-byte aligned).
 *   mc_gptq_factor    inputs with H_kk = 0 are dead (dead[k] = 1; H_kk taken
 *                     as 1), H += damp * mean(diag H) * I (GPTQ uses damp =
 *                     0.01), and U [K][K] fp64 = the upper-triangular
 *                     Cholesky factor of H^-1 (H^-1 = U^T U; zeros below the
 *                     diagonal).  H is read only.  H must be symmetric
 *                     positive semi-definite with damp > 0, or positive
 *                     definite; otherwise U holds NaNs.
 *   mc_gptq_quantize  quantizes matrix `mat` (0 gate [ffn][d], 1 up [ffn][d],
 *                     2 down [d][ffn]) of expert e of L at the expert's width
 *                     and L's group size, writing its codes and scale/zero
 *                     words into L (the other matrices are untouched):
 *                     dead inputs get weight 0; for k = 0 .. K-1, at a group
 *                     start s and z are the Sec. 3.1 parameters (as mc_pack)
 *                     of the fp32 rounding of the group's current values;
 *                     q_k = nearest level of fp32(w_k); e_k = (w_k - s(q_k -
 *                     z)) / U_kk; w_j -= e_k U_kj for j > k, applied one
 *                     column after the other.  W: [R][K] fp32; loss (may be
 *                     NULL): [R] fp64, sum_k e_k^2 / 2 per row.
 *
 * K (the input width) must be a multiple of 128, at most MC_GPTQ_MAX_K.
 * Workspace: mc_gptq_workspace(R, K) bytes (about 2.25 K^2 doubles for the
 * factor, R K (8 + 1) + 1024 R bytes for the quantizer), 8-byte aligned.
 * Errors: MC_EINVAL (shape, NULL or misaligned pointer, damp < 0 or not
 * finite), MC_ENOSPACE (workspace or layer buffers), MC_EHIP. */
#define MC_GPTQ_MAX_K 32768
mc_status mc_gptq_workspace(int R, int K, size_t *bytes);
mc_status mc_gptq_hessian(const uint16_t *x_bf16, int N, int K, double *H, int accumulate, void *stream);
mc_status mc_gptq_factor(const double *H, int K, double damp, double *U, uint8_t *dead, void *workspace,
                         size_t ws_bytes, void *stream);
mc_status mc_gptq_quantize(const mc_layer *L, int e, int mat, const float *W, const double *U,
                           const uint8_t *dead, double *loss, void *workspace, size_t ws_bytes, void *stream);

/* Router logits, the scores whose top-k Eq. 1 takes:
 *   logits[t][e] = sum_k x[t][k] * w_router[e][k]
 * x: [T][d] bf16 (the MoE layer input), w_router: [E][d] bf16, both 16-byte
 * aligned; logits: [T][E] fp32.  Every product is exact in fp64, the d
 * products are summed in fp64 and the sum is rounded once to fp32, so each
 * logit lies between the fp32 roundings of S - g and S + g, with S the exact
 * sum and g = (d - 1) 2^-53 sum_k |x_k w_k|: the correctly rounded value
 * except when S is that close to an fp32 rounding boundary.  Deterministic.
 * Limits: 1 <= T <= MC_MAX_TOKENS, 1 <= E <= 256, d a positive multiple of 8.
 * Errors: MC_EINVAL (shape, NULL or misaligned pointer), MC_EUNSUPPORTED
 * (T above MC_MAX_TOKENS), MC_EHIP. */
mc_status mc_router_logits(const uint16_t *x_bf16, const uint16_t *w_router_bf16, int T, int d, int E,
                           float *logits, void *stream);

/* Top-k routing with Online Dynamic Pruning (Eq. 1, Eq. 5, token protection).
 * logits: [T][E] fp32, finite.  important: [T] uint8, nonzero = protected
 * (may be NULL: no token protected).  threshold tau in [0, 1] acts on the
 * top-k-normalised weight p_r = exp(l_r - l_0) / sum_{i<k} exp(l_i - l_0):
 * for an unprotected token, rank r >= 1 is dropped when p_r < tau; rank 0 is
 * never dropped; tau = 0 disables pruning.  For k = 2 this is Eq. 5 with
 * mu = tau / (1 - tau) and is decided as fp32(l_0 - l_1) > delta, delta the
 * fp32 rounding of ln((1 - tau) / tau); for k > 2 it is evaluated in fp64.
 * Errors: MC_EINVAL (shape, null pointer, tau outside [0, 1]), MC_EHIP. */
mc_status mc_route_and_prune(const float *logits, const uint8_t *important,
                             float threshold, const mc_routing *r, void *stream);

/* Workspace bytes mc_moe_forward needs for T tokens. Errors: MC_EINVAL. */
mc_status mc_forward_workspace(int T, int E, int k, int d, int ffn, size_t *bytes);

/* Eq. 1 over the kept pairs: y_t = sum_r w_r * E_{e_r}(x_t) with
 * E_e(x) = W_down (silu(W_gate x) * (W_up x)) on the exact dequantized
 * weights s*(q - z).  x: [T][d] bf16; y: [T][d] bf16 (round to nearest even
 * of the fp32 result).  r must come from mc_route_and_prune on the same
 * stream (or be complete).  workspace: ws_bytes >= mc_forward_workspace.
 * Errors: MC_EINVAL (shape mismatch, null pointer), MC_ENOSPACE, MC_EHIP. */
mc_status mc_moe_forward(const uint16_t *x_bf16, const mc_routing *r,
                         const mc_layer *L, uint16_t *y_bf16, void *workspace,
                         size_t ws_bytes, void *stream);

/* mc_moe_forward for callers that cannot allocate device memory (code under
 * HIP graph capture, tight serving loops, harnesses that forbid hipMalloc):
 * the same kernels and results, with the workspace taken from a device
 * array the library holds on every GPU it runs on (MC_NOALLOC_SCRATCH_BYTES,
 * kept until the process ends).  Nothing is allocated by the call.  The
 * array is shared by all such calls on a GPU and keeps the last call's
 * contents (the forward writes every workspace byte it reads, nothing needs
 * clearing): calls that overlap on one GPU (other streams, other threads)
 * race and must be serialised by the caller.  Errors: as mc_moe_forward;
 * MC_ENOSPACE when mc_forward_workspace(T, ...) exceeds the array (decode
 * batches of up to 64 tokens of the Mixtral-shaped layer fit). */
#define MC_NOALLOC_SCRATCH_BYTES (32u << 20)
mc_status mc_moe_forward_noalloc(const uint16_t *x_bf16, const mc_routing *r,
                                 const mc_layer *L, uint16_t *y_bf16, void *stream);

/* mc_route_and_prune followed by mc_moe_forward in one call (the routing
 * kernels, then the expert kernels, on `stream`), with the same results:
 * the routing buffers of r as mc_route_and_prune writes them, y as
 * mc_moe_forward writes it.  Arguments and errors: those of the two calls
 * (workspace: mc_forward_workspace). */
mc_status mc_moe_route_forward(const uint16_t *x_bf16, const float *logits, const uint8_t *important,
                               float threshold, const mc_routing *r, const mc_layer *L, uint16_t *y_bf16,
                               void *workspace, size_t ws_bytes, void *stream);

/* Workspace bytes mc_moe_stack_forward needs: the normalised layer input
 * (T*d bf16, rounded up to 256 bytes); for batches that route in one
 * workgroup (T <= 64 and T <= 16*64/S, S the least power of two >= E, up to
 * 64 experts; T*E <= 512 above) the routing buffers of 8 layers, which are
 * then routed together (each buffer rounded up to 256 bytes); and
 * mc_forward_workspace.  Errors: MC_EINVAL. */
mc_status mc_stack_workspace(int T, int E, int k, int d, int ffn, size_t *bytes);

/* A stack of n_layers MoE layers joined by residual connections: the expert
 * half of Mixtral-style decoder blocks, each with its pre-MoE RMSNorm (unit
 * gain, eps = 1e-5); attention is not part of this library.
 *   h_0 = x;  for l = 0 .. n_layers-1:
 *     xn_l    = bf16(h_l / sqrt(mean_j h_l[j]^2 + 1e-5))   (per token; the
 *               sum of squares and the quotient in fp64, one rounding),
 *     route layer l's logits (as mc_route_and_prune, same threshold),
 *     h_{l+1} = bf16(h_l + sum_r w_r * E_{e_r}(xn_l))   (Eq. 1 + residual,
 *               the sum in fp32, one round-to-nearest-even);
 *   y = h_{n_layers}.
 * layers: HOST array [n_layers] of descriptors sharing E, d, ffn and group
 * (each layer has its own widths and buffers).  logits: [n_layers][T][E]
 * fp32; important: [n_layers][T] uint8 or NULL.  r: routing buffers for T
 * tokens (k taken from it), reused by every layer; after the call it holds
 * the last layer's routing.  x, y, tmp: [T][d] bf16, three distinct,
 * non-overlapping buffers (tmp holds every other layer's output; it may be
 * NULL when n_layers == 1).  workspace: ws_bytes >= mc_stack_workspace(T, E,
 * k, d, ffn), reused by every layer.  Everything runs in order on `stream`.
 * Errors: MC_EINVAL (shape mismatch between layers, null or overlapping
 * buffers, tau outside [0, 1]), MC_ENOSPACE, MC_EHIP. */
mc_status mc_moe_stack_forward(const uint16_t *x_bf16, int n_layers, const mc_layer *layers,
                               const float *logits, const uint8_t *important, float threshold,
                               const mc_routing *r, uint16_t *y_bf16, uint16_t *tmp_bf16,
                               void *workspace, size_t ws_bytes, void *stream);

/* Workspace bytes mc_token_importance needs for H heads and L tokens: fp32
 * partial sums, 512 B per 128x128 tile of the lower triangle and slice of
 * heads (about 2 MB up to 8192 tokens, 67 MB at 65,536), plus 12 B per token.
 * Errors: MC_EINVAL, MC_EUNSUPPORTED (L above MC_MAX_TOKENS). */
mc_status mc_importance_workspace(int H, int L, size_t *bytes);

/* Token importance (Sec. 3.3.2, Eq. 6) and the protected set for
 * mc_route_and_prune.  attn: [H][L][L] bf16 causal attention probabilities
 * (>= 0), attn[h][i][j] = weight of query i on key j; only j <= i is read.
 * x: [L][d] bf16 token vectors (the MoE layer input).  With 0-based j:
 *   I_j = ||x_j||_1 * (1/H) * sum_h sum_{i=j}^{L-1} attn[h][i][j] / (L - j),
 * the mean attention key j receives from the L - j queries that see it,
 * averaged over heads; fp32 sums in a fixed order.  important[j] = 1 for the
 * floor(rho*L + 1/2) largest I_j (equal values: lower j first), 0 otherwise;
 * the paper protects 2 % (rho = 0.02).  importance ([L] fp32) may be NULL.
 * workspace: ws_bytes >= mc_importance_workspace(H, L).  Async on `stream`.
 * Errors: MC_EINVAL (shape, rho outside [0, 1], NULL pointer), MC_ENOSPACE,
 * MC_EUNSUPPORTED (L above MC_MAX_TOKENS), MC_EHIP. */
mc_status mc_token_importance(const uint16_t *attn_bf16, int H, int L, const uint16_t *x_bf16, int d,
                              float rho, float *importance, uint8_t *important, void *workspace,
                              size_t ws_bytes, void *stream);

/* Pruning threshold from calibration router logits (Sec. 3.3.1: mu is the
 * median of w_1/w_0 over calibration tokens).  logits_host: [T][E] fp32 in
 * HOST memory, finite.  w_1/w_0 = exp(l_1 - l_0) of the two largest logits
 * (equal logits: lower expert index first); *mu = their median (mean of the
 * two middle values for even T); *tau = mu / (1 + mu), the threshold
 * mc_route_and_prune takes (identical decision at k = 2).  Offline helper,
 * pure host computation.  Errors: MC_EINVAL. */
mc_status mc_odp_threshold(const float *logits_host, int T, int E, double *mu, double *tau);

/* Offline PMQ allocation (Sec. 3.2), pure host computation.
 * Expert significance (Sec. 3.2.1) from calibration router logits
 * logits_host [T][E] fp32 (HOST memory, finite): each token's top-k experts
 * by (logit descending, expert index ascending) with routing weights the
 * softmax over the selected k (fp64);  phi[e] = (tokens that select e) / T,
 * w[e] = (sum of e's routing weights) / T  (host [E] each; sum phi = k,
 * sum w = 1).  Errors: MC_EINVAL. */
mc_status mc_pmq_significance(const float *logits_host, int T, int E, int k, double *phi, double *w);

/* Expert widths by the integer program of Eq. 4: b_e in {1, 2, 3} minimising
 *   sum_e phi_e^alpha * w_e^beta * eps[e][b_e - 1]^gamma
 * subject to sum_e b_e = total_bits (E * target average), at least one expert
 * at 3 bits and at least one at 2.  phi, w: host [E] (>= 0); eps: host [E][3]
 * reconstruction errors at 1, 2, 3 bits (>= 0; Eq. 3 measures them as the
 * F-norm of the output change when only that expert is quantized).  The paper
 * fixes gamma = 2 and finds alpha, beta in {1, 1.5, 2} equivalent.  Solved
 * exactly (dynamic programme over experts); the objective of an allocation is
 * its terms summed in expert order in fp64, and among allocations with equal
 * objective the lexicographically smallest width vector is returned.
 * bits: host [E] output; objective (may be NULL): the minimum.
 * Errors: MC_EINVAL (E < 2, total_bits outside [E + 3, 3E - 1], negative or
 * non-finite inputs, alpha or beta < 0, gamma <= 0). */
mc_status mc_pmq_allocate(const double *phi, const double *w, const double *eps, int E, double alpha,
                          double beta, double gamma, int total_bits, int *bits, double *objective);

/* The reconstruction error that Eq. 4 takes (Sec. 3.2.2, the equation
 * before Eq. 4), measured on one MoE layer and a calibration batch:
 *   eps[e][b-1] = || F(theta) - F(theta[e -> Q(e, b)]) ||_F,   b = 1, 2, 3,
 * F the layer output of Eq. 1 over the batch's T tokens (routing r, the
 * weights theta: w_gate, w_up [E][ffn][d], w_down [E][d][ffn], fp32, DEVICE),
 * Q(e, b) expert e alone quantized at b bits by mc_pack's min-max RTN
 * quantizer (group size `group`).  Since only the tokens that keep e change,
 * eps[e][b-1]^2 = sum over e's kept pairs of ||w_r (E_e^(b)(x_t) - E_e(x_t))||^2:
 * E_e(x_t) from fp32 weights in fp32 arithmetic (h = silu(g) * u unrounded),
 * E_e^(b)(x_t) from the packed forward's own kernels.  x_bf16 [T][d] DEVICE;
 * r: the batch's routing from mc_route_and_prune (the paper measures the
 * unpruned model: threshold 0); eps_host: HOST [E][3] output.  Workspace
 * (DEVICE) of mc_pmq_error_workspace bytes: the layer packed at each width in
 * turn, the forward's buffers and the dense outputs.  Offline call: it waits
 * for the stream before returning.  Errors: MC_EINVAL (shapes as mc_pack and
 * mc_moe_forward, NULL pointers, routing of another E), MC_ENOSPACE (short
 * workspace), MC_EUNSUPPORTED, MC_EHIP. */
mc_status mc_pmq_error_workspace(int T, int E, int k, int d, int ffn, int group, size_t *bytes);
mc_status mc_pmq_expert_error(const float *w_gate, const float *w_up, const float *w_down, int E, int d,
                              int ffn, int group, const uint16_t *x_bf16, const mc_routing *r,
                              double *eps_host, void *workspace, size_t ws_bytes, void *stream);

/* Instrumentation.  mc_timing_enable(1) clears the record and brackets every
 * kernel launch made afterwards by two HIP events on the launch stream;
 * mc_timing_enable(0) stops recording.  mc_timing_read waits for the recorded
 * events of one kernel and returns the summed duration in ms and the number
 * of launches.  Kernel names: pack_scale_zero, pack_codes, export,
 * route_fused, route_select, route_lists, prefill_prep, gateup, down, combine,
 * importance_colsum, importance_finish, importance_select, rmsnorm, router,
 * gptq_hessian, gptq_factor, gptq_quantize (each a whole call).
 * Errors: MC_EINVAL (unknown name, NULL pointer), MC_EHIP. */
mc_status mc_timing_enable(int on);
mc_status mc_timing_read(const char *kernel, double *total_ms, int *launches);

/* Message for the last non-OK status returned on this thread. */
const char *mc_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* MC_MOE_H */
