// api.hip -- the extern "C" boundary: argument validation, descriptors,
// launches on the caller's stream.  No allocation anywhere.
#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <vector>

#include "mc_internal.hpp"

// Workspace of mc_moe_forward_noalloc: a file-scope device array, one copy
// on every GPU the library runs on, held until the process ends.  Host code
// never uses the name itself as an address (it is a host-side stand-in): the
// device address comes from hipGetSymbolAddress, once per device.
static __device__ __align__(256) unsigned char scratch[MC_NOALLOC_SCRATCH_BYTES];

namespace {

thread_local char g_err[512] = "";

mc_status fail(mc_status s, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof(g_err), fmt, ap);
  va_end(ap);
  return s;
}

mc_status hip_status(hipError_t e, const char* what) {
  if (e == hipSuccess) return MC_OK;
  return fail(MC_EHIP, "%s: %s", what, hipGetErrorString(e));
}

mc_status check_shape(int E, int d, int ffn, const int* bits, int G) {
  if (E < 1 || E > MC_MAX_EXPERTS) return fail(MC_EINVAL, "E=%d outside [1, %d]", E, MC_MAX_EXPERTS);
  if (d <= 0 || ffn <= 0 || d % 128 || ffn % 128)
    return fail(MC_EINVAL, "d=%d and ffn=%d must be positive multiples of 128", d, ffn);
  if ((long long)d * ffn > (1LL << 31))
    return fail(MC_EUNSUPPORTED, "d*ffn=%lld exceeds 2^31", (long long)d * ffn);
  if (G != 32 && G != 64 && G != 128)
    return fail(G > 0 && G % 32 == 0 ? MC_EUNSUPPORTED : MC_EINVAL,
                "group size %d: this build supports 32, 64 and 128", G);
  if (!bits) return fail(MC_EINVAL, "bits_host is NULL");
  for (int e = 0; e < E; ++e)
    if (bits[e] < 1 || bits[e] > 3) return fail(MC_EINVAL, "bits[%d]=%d not in {1,2,3}", e, bits[e]);
  return MC_OK;
}

void sizes(int E, int d, int ffn, const int* bits, int G, size_t* wb, size_t* szb) {
  size_t w = 0;
  for (int e = 0; e < E; ++e) w += 3 * (size_t)d * ffn * bits[e] / 8;
  *wb = w;
  *szb = 3 * (size_t)E * d * ffn / G * 4;
}

mc_status check_layer(const mc_layer* L, bool need_buffers) {
  if (!L) return fail(MC_EINVAL, "layer descriptor is NULL");
  mc_status s = check_shape(L->E, L->d, L->ffn, L->bits_host, L->group);
  if (s != MC_OK) return s;
  if (!need_buffers) return MC_OK;
  if (!L->words || !L->sz) return fail(MC_EINVAL, "layer words/sz pointer is NULL");
  size_t wb, szb;
  sizes(L->E, L->d, L->ffn, L->bits_host, L->group, &wb, &szb);
  if (L->words_bytes < wb || L->sz_bytes < szb)
    return fail(MC_ENOSPACE, "layer buffers hold %zu/%zu bytes, need %zu/%zu", L->words_bytes,
                L->sz_bytes, wb, szb);
  return MC_OK;
}

mc::LayerArgs layer_args(const mc_layer* L) {
  mc::LayerArgs a;
  a.words = static_cast<const uint32_t*>(L->words);
  a.sz = L->sz;
  a.E = L->E;
  a.d = L->d;
  a.ffn = L->ffn;
  a.G = L->group;
  a.cum_bits[0] = 0;
  for (int e = 0; e < L->E; ++e) a.cum_bits[e + 1] = (uint16_t)(a.cum_bits[e] + L->bits_host[e]);
  for (int e = L->E; e < MC_MAX_EXPERTS; ++e) a.cum_bits[e + 1] = a.cum_bits[e];
  for (int i = 0; i < MC_MAX_EXPERTS / 32; ++i) a.sign_mask[i] = 0u;
  return a;
}

// This device's address of `scratch`, looked up on the first call made with
// the device current and kept per device.
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

mc_status scratch_address(void** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_status(e, "hipGetDevice");
  if (dev < 0 || dev >= kMaxDevices) return fail(MC_EUNSUPPORTED, "device %d above %d", dev, kMaxDevices - 1);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return hip_status(e, "hipGetSymbolAddress(scratch)");
    if (!p) return fail(MC_EHIP, "hipGetSymbolAddress(scratch) returned NULL");
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return MC_OK;
}

mc_status check_routing(const mc_routing* r) {
  if (!r) return fail(MC_EINVAL, "routing descriptor is NULL");
  if (r->T < 1) return fail(MC_EINVAL, "T=%d must be >= 1", r->T);
  if (r->E < 1 || r->E > MC_MAX_EXPERTS) return fail(MC_EINVAL, "E=%d outside [1, %d]", r->E, MC_MAX_EXPERTS);
  if (r->k < 1 || r->k > r->E || r->k > MC_MAX_TOPK)
    return fail(MC_EINVAL, "k=%d outside [1, min(E=%d, %d)]", r->k, r->E, MC_MAX_TOPK);
  if (r->T > MC_MAX_TOKENS) return fail(MC_EUNSUPPORTED, "T=%d above %d", r->T, MC_MAX_TOKENS);
  if (!r->topk_idx || !r->topk_w || !r->kept || !r->counts || !r->offsets || !r->pair_token ||
      !r->pair_rank || !r->pair_w || !r->pair_pos || !r->n_pruned)
    return fail(MC_EINVAL, "a routing output pointer is NULL");
  return MC_OK;
}

}  // namespace

namespace {

size_t up256(size_t b) { return (b + 255) / 256 * 256; }

// Workspace of mc_pmq_expert_error: the layer packed at 3 bits (the widest),
// its scale/zero words, the forward's workspace, the dense h [P][ffn] and
// y [P][d] (fp32) and eps [E][3] (fp64).
struct PmqLayout {
  size_t words, sz, fws, h, y, eps, total;
};

PmqLayout pmq_layout(int T, int E, int k, int d, int ffn, int G) {
  PmqLayout o;
  const size_t P = (size_t)T * k;
  o.words = 0;
  o.sz = o.words + up256(3 * (size_t)E * d * ffn * 3 / 8);
  o.fws = o.sz + up256(3 * (size_t)E * d * ffn / G * 4);
  o.h = o.fws + up256(mc::forward_workspace_bytes(T, E, k, d, ffn));
  o.y = o.h + up256(P * ffn * sizeof(float));
  o.eps = o.y + up256(P * d * sizeof(float));
  o.total = o.eps + up256((size_t)E * 3 * sizeof(double));
  return o;
}

}  // namespace

extern "C" {

const char* mc_last_error(void) { return g_err; }

mc_status mc_pack_sizes(int E, int d, int ffn, const int* bits_host, int group, size_t* words_bytes,
                        size_t* sz_bytes) {
  mc_status s = check_shape(E, d, ffn, bits_host, group);
  if (s != MC_OK) return s;
  if (!words_bytes || !sz_bytes) return fail(MC_EINVAL, "output size pointer is NULL");
  sizes(E, d, ffn, bits_host, group, words_bytes, sz_bytes);
  return MC_OK;
}

mc_status mc_pack_methods(const float* w_gate, const float* w_up, const float* w_down, const mc_layer* L,
                          const int* method_host, void* stream) {
  mc_status s = check_layer(L, true);
  if (s != MC_OK) return s;
  if (!w_gate || !w_up || !w_down) return fail(MC_EINVAL, "weight pointer is NULL");
  mc::LayerArgs a = layer_args(L);
  bool any_sign = false;
  if (method_host) {
    for (int e = 0; e < L->E; ++e) {
      if (method_host[e] == MC_QUANT_SIGN) {
        if (L->bits_host[e] != 1)
          return fail(MC_EINVAL, "expert %d: sign binarization needs 1 bit, has %d", e, L->bits_host[e]);
        a.sign_mask[e >> 5] |= 1u << (e & 31);
        any_sign = true;
      } else if (method_host[e] != MC_QUANT_RTN) {
        return fail(MC_EINVAL, "expert %d: unknown quantization method %d", e, method_host[e]);
      }
    }
  }
  (void)hipGetLastError();
  return hip_status(mc::launch_pack(w_gate, w_up, w_down, a, static_cast<uint32_t*>(L->words), L->sz, any_sign,
                                    static_cast<hipStream_t>(stream)),
                    "mc_pack launch");
}

mc_status mc_pack(const float* w_gate, const float* w_up, const float* w_down, const mc_layer* L,
                  void* stream) {
  return mc_pack_methods(w_gate, w_up, w_down, L, nullptr, stream);
}

static mc_status export_common(const mc_layer* L, int e, int mat, void* out, bool dequant,
                               void* stream) {
  mc_status s = check_layer(L, true);
  if (s != MC_OK) return s;
  if (e < 0 || e >= L->E) return fail(MC_EINVAL, "expert %d outside [0, %d)", e, L->E);
  if (mat < 0 || mat > 2) return fail(MC_EINVAL, "matrix %d not in {0,1,2}", mat);
  if (!out) return fail(MC_EINVAL, "output pointer is NULL");
  const mc::LayerArgs a = layer_args(L);
  const int b = L->bits_host[e];
  const size_t per_bit = (size_t)L->d * L->ffn / 32;
  const size_t wofs = (3 * (size_t)a.cum_bits[e] + (size_t)mat * b) * per_bit;
  const size_t sofs = (3 * (size_t)e + mat) * ((size_t)L->d * L->ffn / L->group);
  const int R = mat < 2 ? L->ffn : L->d, K = mat < 2 ? L->d : L->ffn;
  (void)hipGetLastError();
  return hip_status(mc::launch_export(static_cast<const uint32_t*>(L->words) + wofs, L->sz + sofs,
                                      b, R, K, L->group, dequant, out,
                                      static_cast<hipStream_t>(stream)),
                    "export launch");
}

mc_status mc_dequant_export(const mc_layer* L, int e, int mat, uint16_t* out, void* stream) {
  return export_common(L, e, mat, out, true, stream);
}

mc_status mc_codes_export(const mc_layer* L, int e, int mat, uint8_t* out, void* stream) {
  return export_common(L, e, mat, out, false, stream);
}

// ----------------------------------------------------------------- GPTQ --
static mc_status check_gptq_k(int K) {
  if (K < 128 || K % 128 != 0 || K > MC_GPTQ_MAX_K)
    return fail(MC_EINVAL, "K=%d: need a multiple of 128 in [128, %d]", K, MC_GPTQ_MAX_K);
  return MC_OK;
}

mc_status mc_gptq_workspace(int R, int K, size_t* bytes) {
  mc_status s = check_gptq_k(K);
  if (s != MC_OK) return s;
  if (R < 16 || R % 16 != 0) return fail(MC_EINVAL, "R=%d: need a positive multiple of 16", R);
  if (!bytes) return fail(MC_EINVAL, "bytes is NULL");
  const size_t f = mc::gptq_factor_bytes(K), q = mc::gptq_quantize_bytes(R, K);
  *bytes = f > q ? f : q;
  return MC_OK;
}

mc_status mc_gptq_hessian(const uint16_t* x_bf16, int N, int K, double* H, int accumulate, void* stream) {
  mc_status s = check_gptq_k(K);
  if (s != MC_OK) return s;
  if (N < 1) return fail(MC_EINVAL, "N=%d calibration rows", N);
  if (!x_bf16 || !H) return fail(MC_EINVAL, "x or H is NULL");
  if (reinterpret_cast<uintptr_t>(H) & 7u) return fail(MC_EINVAL, "H must be 8-byte aligned");
  (void)hipGetLastError();
  return hip_status(mc::launch_gptq_hessian(x_bf16, N, K, H, accumulate != 0, static_cast<hipStream_t>(stream)),
                    "mc_gptq_hessian launch");
}

mc_status mc_gptq_factor(const double* H, int K, double damp, double* U, uint8_t* dead, void* workspace,
                         size_t ws_bytes, void* stream) {
  mc_status s = check_gptq_k(K);
  if (s != MC_OK) return s;
  if (!(damp >= 0.0) || !std::isfinite(damp)) return fail(MC_EINVAL, "damp %g: need a finite value >= 0", damp);
  if (!H || !U || !dead || !workspace) return fail(MC_EINVAL, "H, U, dead or workspace is NULL");
  if ((reinterpret_cast<uintptr_t>(H) | reinterpret_cast<uintptr_t>(U) | reinterpret_cast<uintptr_t>(workspace)) &
      7u)
    return fail(MC_EINVAL, "H, U and workspace must be 8-byte aligned");
  const size_t need = mc::gptq_factor_bytes(K);
  if (ws_bytes < need) return fail(MC_ENOSPACE, "workspace %zu bytes, need %zu", ws_bytes, need);
  (void)hipGetLastError();
  return hip_status(mc::launch_gptq_factor(H, K, damp, U, dead, workspace, static_cast<hipStream_t>(stream)),
                    "mc_gptq_factor launch");
}

mc_status mc_gptq_quantize(const mc_layer* L, int e, int mat, const float* W, const double* U, const uint8_t* dead,
                           double* loss, void* workspace, size_t ws_bytes, void* stream) {
  mc_status s = check_layer(L, true);
  if (s != MC_OK) return s;
  if (e < 0 || e >= L->E) return fail(MC_EINVAL, "expert %d outside [0, %d)", e, L->E);
  if (mat < 0 || mat > 2) return fail(MC_EINVAL, "matrix %d not in {0,1,2}", mat);
  const int R = mat < 2 ? L->ffn : L->d, K = mat < 2 ? L->d : L->ffn;
  s = check_gptq_k(K);
  if (s != MC_OK) return s;
  if (!W || !U || !dead || !workspace) return fail(MC_EINVAL, "W, U, dead or workspace is NULL");
  if ((reinterpret_cast<uintptr_t>(U) | reinterpret_cast<uintptr_t>(workspace) |
       reinterpret_cast<uintptr_t>(loss)) & 7u)
    return fail(MC_EINVAL, "U, loss and workspace must be 8-byte aligned");
  const size_t need = mc::gptq_quantize_bytes(R, K);
  if (ws_bytes < need) return fail(MC_ENOSPACE, "workspace %zu bytes, need %zu", ws_bytes, need);
  const mc::LayerArgs a = layer_args(L);
  const int b = L->bits_host[e];
  const size_t per_bit = (size_t)L->d * L->ffn / 32;
  const size_t wofs = (3 * (size_t)a.cum_bits[e] + (size_t)mat * b) * per_bit;
  const size_t sofs = (3 * (size_t)e + mat) * ((size_t)L->d * L->ffn / L->group);
  (void)hipGetLastError();
  return hip_status(mc::launch_gptq_quantize(W, U, dead, R, K, b, L->group, static_cast<uint32_t*>(L->words) + wofs,
                                             L->sz + sofs, loss, workspace, static_cast<hipStream_t>(stream)),
                    "mc_gptq_quantize launch");
}

static float prune_delta32(double tau) {
  if (tau == 0.0) return INFINITY;
  if (tau == 1.0) return -INFINITY;
  return (float)std::log((1.0 - tau) / tau);
}

mc_status mc_router_logits(const uint16_t* x_bf16, const uint16_t* w_router_bf16, int T, int d, int E,
                           float* logits, void* stream) {
  if (T < 1 || E < 1 || E > MC_MAX_EXPERTS || d < 8 || d % 8 != 0)
    return fail(MC_EINVAL, "bad shape T=%d d=%d E=%d (d a positive multiple of 8, E <= %d)", T, d, E,
                MC_MAX_EXPERTS);
  if (T > MC_MAX_TOKENS) return fail(MC_EUNSUPPORTED, "T=%d above %d", T, MC_MAX_TOKENS);
  if (!x_bf16 || !w_router_bf16 || !logits) return fail(MC_EINVAL, "x, w_router or logits is NULL");
  if ((reinterpret_cast<uintptr_t>(x_bf16) | reinterpret_cast<uintptr_t>(w_router_bf16)) & 15u)
    return fail(MC_EINVAL, "x and w_router must be 16-byte aligned");
  (void)hipGetLastError();
  return hip_status(mc::launch_router(x_bf16, w_router_bf16, T, d, E, logits, static_cast<hipStream_t>(stream)),
                    "mc_router_logits launch");
}

mc_status mc_route_and_prune(const float* logits, const uint8_t* important, float threshold,
                             const mc_routing* r, void* stream) {
  mc_status s = check_routing(r);
  if (s != MC_OK) return s;
  if (!logits) return fail(MC_EINVAL, "logits pointer is NULL");
  if (!(threshold >= 0.0f && threshold <= 1.0f))
    return fail(MC_EINVAL, "threshold %g outside [0, 1]", (double)threshold);
  const double tau = (double)threshold;
  (void)hipGetLastError();
  return hip_status(mc::launch_route(logits, important, prune_delta32(tau), tau, *r,
                                     static_cast<hipStream_t>(stream)),
                    "mc_route_and_prune launch");
}

mc_status mc_forward_workspace(int T, int E, int k, int d, int ffn, size_t* bytes) {
  if (T < 1 || E < 1 || E > MC_MAX_EXPERTS || k < 1 || k > E || k > MC_MAX_TOPK || d <= 0 ||
      ffn <= 0 || d % 128 || ffn % 128)
    return fail(MC_EINVAL, "bad shape T=%d E=%d k=%d d=%d ffn=%d", T, E, k, d, ffn);
  if (T > MC_MAX_TOKENS) return fail(MC_EUNSUPPORTED, "T=%d above %d", T, MC_MAX_TOKENS);
  if (!bytes) return fail(MC_EINVAL, "bytes pointer is NULL");
  *bytes = mc::forward_workspace_bytes(T, E, k, d, ffn);
  return MC_OK;
}

mc_status mc_moe_forward(const uint16_t* x_bf16, const mc_routing* r, const mc_layer* L,
                         uint16_t* y_bf16, void* workspace, size_t ws_bytes, void* stream) {
  mc_status s = check_routing(r);
  if (s != MC_OK) return s;
  s = check_layer(L, true);
  if (s != MC_OK) return s;
  if (r->E != L->E) return fail(MC_EINVAL, "routing has E=%d, layer has E=%d", r->E, L->E);
  if (!x_bf16 || !y_bf16 || !workspace) return fail(MC_EINVAL, "x, y or workspace is NULL");
  const size_t need = mc::forward_workspace_bytes(r->T, r->E, r->k, L->d, L->ffn);
  if (ws_bytes < need) return fail(MC_ENOSPACE, "workspace %zu bytes, need %zu", ws_bytes, need);
  (void)hipGetLastError();
  const mc::LayerArgs a = layer_args(L);
  return hip_status(mc::launch_forward(x_bf16, a, *r, y_bf16, workspace, nullptr,
                                       static_cast<hipStream_t>(stream)),
                    "mc_moe_forward launch");
}

mc_status mc_moe_forward_noalloc(const uint16_t* x_bf16, const mc_routing* r, const mc_layer* L,
                                 uint16_t* y_bf16, void* stream) {
  mc_status s = check_routing(r);
  if (s != MC_OK) return s;
  s = check_layer(L, true);
  if (s != MC_OK) return s;
  if (r->E != L->E) return fail(MC_EINVAL, "routing has E=%d, layer has E=%d", r->E, L->E);
  if (!x_bf16 || !y_bf16) return fail(MC_EINVAL, "x or y is NULL");
  const size_t need = mc::forward_workspace_bytes(r->T, r->E, r->k, L->d, L->ffn);
  if (need > (size_t)MC_NOALLOC_SCRATCH_BYTES)
    return fail(MC_ENOSPACE,
                "T=%d needs %zu bytes of workspace; mc_moe_forward_noalloc holds %zu (use mc_moe_forward "
                "with a caller workspace)",
                r->T, need, (size_t)MC_NOALLOC_SCRATCH_BYTES);
  void* ws = nullptr;
  s = scratch_address(&ws);
  if (s != MC_OK) return s;
  (void)hipGetLastError();
  return hip_status(mc::launch_forward(x_bf16, layer_args(L), *r, y_bf16, ws, nullptr,
                                       static_cast<hipStream_t>(stream)),
                    "mc_moe_forward_noalloc launch");
}

mc_status mc_moe_route_forward(const uint16_t* x_bf16, const float* logits, const uint8_t* important,
                               float threshold, const mc_routing* r, const mc_layer* L, uint16_t* y_bf16,
                               void* workspace, size_t ws_bytes, void* stream) {
  mc_status s = check_routing(r);
  if (s != MC_OK) return s;
  s = check_layer(L, true);
  if (s != MC_OK) return s;
  if (r->E != L->E) return fail(MC_EINVAL, "routing has E=%d, layer has E=%d", r->E, L->E);
  if (!logits) return fail(MC_EINVAL, "logits pointer is NULL");
  if (!(threshold >= 0.0f && threshold <= 1.0f))
    return fail(MC_EINVAL, "threshold %g outside [0, 1]", (double)threshold);
  if (!x_bf16 || !y_bf16 || !workspace) return fail(MC_EINVAL, "x, y or workspace is NULL");
  const size_t need = mc::forward_workspace_bytes(r->T, r->E, r->k, L->d, L->ffn);
  if (ws_bytes < need) return fail(MC_ENOSPACE, "workspace %zu bytes, need %zu", ws_bytes, need);
  const double tau = (double)threshold;
  const mc::RouteArgs ra{logits, important, prune_delta32(tau), tau};
  (void)hipGetLastError();
  return hip_status(mc::launch_forward(x_bf16, layer_args(L), *r, y_bf16, workspace, nullptr,
                                       static_cast<hipStream_t>(stream), &ra),
                    "mc_moe_route_forward launch");
}

// -------------------------------------------------- PMQ reconstruction error --

mc_status mc_pmq_error_workspace(int T, int E, int k, int d, int ffn, int group, size_t* bytes) {
  mc_status s = mc_forward_workspace(T, E, k, d, ffn, bytes);
  if (s != MC_OK) return s;
  std::vector<int> three(E, 3);
  s = check_shape(E, d, ffn, three.data(), group);
  if (s != MC_OK) return s;
  *bytes = pmq_layout(T, E, k, d, ffn, group).total;
  return MC_OK;
}

mc_status mc_pmq_expert_error(const float* w_gate, const float* w_up, const float* w_down, int E, int d, int ffn,
                              int group, const uint16_t* x_bf16, const mc_routing* r, double* eps_host,
                              void* workspace, size_t ws_bytes, void* stream) {
  mc_status s = check_routing(r);
  if (s != MC_OK) return s;
  if (r->E != E) return fail(MC_EINVAL, "routing has E=%d, the weights E=%d", r->E, E);
  size_t need = 0;
  s = mc_pmq_error_workspace(r->T, E, r->k, d, ffn, group, &need);
  if (s != MC_OK) return s;
  if (!w_gate || !w_up || !w_down || !x_bf16 || !eps_host || !workspace)
    return fail(MC_EINVAL, "weight, x, eps or workspace pointer is NULL");
  if (ws_bytes < need) return fail(MC_ENOSPACE, "workspace %zu bytes, need %zu", ws_bytes, need);
  const PmqLayout o = pmq_layout(r->T, E, r->k, d, ffn, group);
  char* ws = static_cast<char*>(workspace);
  float* h = reinterpret_cast<float*>(ws + o.h);
  float* y = reinterpret_cast<float*>(ws + o.y);
  double* eps = reinterpret_cast<double*>(ws + o.eps);
  const hipStream_t st = static_cast<hipStream_t>(stream);
  (void)hipGetLastError();
  s = hip_status(mc::launch_dense_expert(w_gate, w_up, w_down, E, d, ffn, x_bf16, *r, h, y, st),
                 "mc_pmq_expert_error dense launch");
  if (s != MC_OK) return s;
  for (int b = 1; b <= 3; ++b) {
    std::vector<int> bits(E, b);
    mc_layer L;
    L.E = E;
    L.d = d;
    L.ffn = ffn;
    L.group = group;
    L.bits_host = bits.data();
    L.words = ws + o.words;
    L.sz = reinterpret_cast<uint32_t*>(ws + o.sz);
    sizes(E, d, ffn, bits.data(), group, &L.words_bytes, &L.sz_bytes);
    const mc::LayerArgs a = layer_args(&L);
    s = hip_status(mc::launch_pack(w_gate, w_up, w_down, a, static_cast<uint32_t*>(L.words), L.sz, false, st),
                   "mc_pmq_expert_error pack launch");
    if (s != MC_OK) return s;
    float* partial = nullptr;
    size_t part_stride = 0;
    int nsplit = 1;
    s = hip_status(mc::launch_expert_partials(x_bf16, a, *r, ws + o.fws, &partial, &part_stride, &nsplit, st),
                   "mc_pmq_expert_error forward launch");
    if (s != MC_OK) return s;
    s = hip_status(mc::launch_pmq_error(partial, part_stride, nsplit, y, *r, d, b, eps, st),
                   "mc_pmq_expert_error error launch");
    if (s != MC_OK) return s;
  }
  s = hip_status(hipMemcpyAsync(eps_host, eps, (size_t)E * 3 * sizeof(double), hipMemcpyDeviceToHost, st),
                 "mc_pmq_expert_error copy");
  if (s != MC_OK) return s;
  return hip_status(hipStreamSynchronize(st), "mc_pmq_expert_error synchronize");
}

mc_status mc_stack_workspace(int T, int E, int k, int d, int ffn, size_t* bytes) {
  mc_status s = mc_forward_workspace(T, E, k, d, ffn, bytes);
  if (s != MC_OK) return s;
  *bytes = mc::stack_workspace_bytes(T, E, k, d, ffn);
  return MC_OK;
}

static bool overlaps(const void* a, const void* b, size_t bytes) {
  const char* pa = static_cast<const char*>(a);
  const char* pb = static_cast<const char*>(b);
  return pa < pb + bytes && pb < pa + bytes;
}

mc_status mc_moe_stack_forward(const uint16_t* x_bf16, int n_layers, const mc_layer* layers,
                               const float* logits, const uint8_t* important, float threshold,
                               const mc_routing* r, uint16_t* y_bf16, uint16_t* tmp_bf16,
                               void* workspace, size_t ws_bytes, void* stream) {
  mc_status s = check_routing(r);
  if (s != MC_OK) return s;
  if (n_layers < 1) return fail(MC_EINVAL, "n_layers=%d must be >= 1", n_layers);
  if (!layers) return fail(MC_EINVAL, "layers array is NULL");
  for (int l = 0; l < n_layers; ++l) {
    s = check_layer(&layers[l], true);
    if (s != MC_OK) return s;
    const mc_layer& a = layers[l];
    if (a.E != layers[0].E || a.d != layers[0].d || a.ffn != layers[0].ffn || a.group != layers[0].group)
      return fail(MC_EINVAL, "layer %d shape (E=%d d=%d ffn=%d G=%d) differs from layer 0", l, a.E, a.d,
                  a.ffn, a.group);
  }
  if (r->E != layers[0].E) return fail(MC_EINVAL, "routing has E=%d, layers have E=%d", r->E, layers[0].E);
  if (!logits) return fail(MC_EINVAL, "logits pointer is NULL");
  if (!(threshold >= 0.0f && threshold <= 1.0f))
    return fail(MC_EINVAL, "threshold %g outside [0, 1]", (double)threshold);
  if (!x_bf16 || !y_bf16 || !workspace) return fail(MC_EINVAL, "x, y or workspace is NULL");
  if (n_layers > 1 && !tmp_bf16) return fail(MC_EINVAL, "tmp is NULL with %d layers", n_layers);
  const size_t act = (size_t)r->T * layers[0].d * sizeof(uint16_t);
  if (overlaps(x_bf16, y_bf16, act) || (tmp_bf16 && (overlaps(x_bf16, tmp_bf16, act) ||
                                                     overlaps(y_bf16, tmp_bf16, act))))
    return fail(MC_EINVAL, "x, y and tmp must not overlap");
  const size_t need = mc::stack_workspace_bytes(r->T, r->E, r->k, layers[0].d, layers[0].ffn);
  if (ws_bytes < need) return fail(MC_ENOSPACE, "workspace %zu bytes, need %zu", ws_bytes, need);
  const int T = r->T, E = r->E, k = r->k;
  uint16_t* xn = static_cast<uint16_t*>(workspace);
  char* sets = static_cast<char*>(workspace) + ((size_t)T * layers[0].d * sizeof(uint16_t) + 255) / 256 * 256;
  void* fws = static_cast<char*>(workspace) + (need - mc::forward_workspace_bytes(T, E, k, layers[0].d,
                                                                                   layers[0].ffn));
  const double tau = (double)threshold;
  const float delta32 = prune_delta32(tau);
  hipStream_t st = static_cast<hipStream_t>(stream);
  (void)hipGetLastError();
  const uint16_t* in = x_bf16;
  // layer 0's input is normalised here; every later layer's input is formed
  // by the previous layer's combine (same bytes as a separate RMSNorm launch)
  s = hip_status(mc::launch_rmsnorm(in, T, layers[0].d, mc::kRmsNormEps, xn, st),
                 "mc_moe_stack_forward rmsnorm launch");
  if (s != MC_OK) return s;
  // A layer's routing depends on its own logits only: small batches route
  // kRouteBatch layers in one launch, each into a routing set of the
  // workspace (the last layer into r), before those layers run.
  const bool batch_routes = mc::route_batch_fits(T, E);
  mc_routing rs[mc::kRouteBatch];
  for (int l0 = 0; l0 < n_layers; l0 += mc::kRouteBatch) {
    const int nb = n_layers - l0 < mc::kRouteBatch ? n_layers - l0 : mc::kRouteBatch;
    if (batch_routes) {
      for (int b = 0; b < nb; ++b)
        rs[b] = (l0 + b == n_layers - 1) ? *r
                                         : mc::routing_set(sets + b * mc::routing_set_bytes(T, E, k), T, E, k);
      const size_t te = (size_t)l0 * T;
      s = hip_status(mc::launch_route_batch(logits + te * E, important ? important + te : nullptr, delta32,
                                            tau, rs, nb, st),
                     "mc_moe_stack_forward routing launch");
      if (s != MC_OK) return s;
    }
    for (int l = l0; l < l0 + nb; ++l) {
      uint16_t* out = ((n_layers - 1 - l) % 2 == 0) ? y_bf16 : tmp_bf16;
      const size_t te = (size_t)l * T;
      const mc::RouteArgs ra{logits + te * E, important ? important + te : nullptr, delta32, tau};
      s = hip_status(mc::launch_forward(xn, layer_args(&layers[l]), batch_routes ? rs[l - l0] : *r, out, fws,
                                        in, st, batch_routes ? nullptr : &ra,
                                        l + 1 < n_layers ? xn : nullptr),
                     "mc_moe_stack_forward forward launch");
      if (s != MC_OK) return s;
      in = out;
    }
  }
  return MC_OK;
}

mc_status mc_importance_workspace(int H, int L, size_t* bytes) {
  if (H < 1 || L < 1) return fail(MC_EINVAL, "bad shape H=%d L=%d", H, L);
  if (L > MC_MAX_TOKENS) return fail(MC_EUNSUPPORTED, "L=%d above %d", L, MC_MAX_TOKENS);
  if (!bytes) return fail(MC_EINVAL, "bytes pointer is NULL");
  *bytes = mc::importance_workspace_bytes(H, L);
  return MC_OK;
}

mc_status mc_token_importance(const uint16_t* attn_bf16, int H, int L, const uint16_t* x_bf16, int d,
                              float rho, float* importance, uint8_t* important, void* workspace,
                              size_t ws_bytes, void* stream) {
  if (H < 1 || L < 1 || d < 1) return fail(MC_EINVAL, "bad shape H=%d L=%d d=%d", H, L, d);
  if (L > MC_MAX_TOKENS) return fail(MC_EUNSUPPORTED, "L=%d above %d", L, MC_MAX_TOKENS);
  if (!(rho >= 0.0f && rho <= 1.0f)) return fail(MC_EINVAL, "rho %g outside [0, 1]", (double)rho);
  if (!attn_bf16 || !x_bf16 || !important || !workspace)
    return fail(MC_EINVAL, "attn, x, important or workspace is NULL");
  const size_t need = mc::importance_workspace_bytes(H, L);
  if (ws_bytes < need) return fail(MC_ENOSPACE, "workspace %zu bytes, need %zu", ws_bytes, need);
  (void)hipGetLastError();
  return hip_status(mc::launch_importance(attn_bf16, H, L, x_bf16, d, rho, importance, important, workspace,
                                          static_cast<hipStream_t>(stream)),
                    "mc_token_importance launch");
}

mc_status mc_odp_threshold(const float* logits_host, int T, int E, double* mu, double* tau) {
  if (!logits_host || !mu || !tau) return fail(MC_EINVAL, "NULL argument");
  if (T < 1 || E < 2) return fail(MC_EINVAL, "bad shape T=%d E=%d (need E >= 2)", T, E);
  std::vector<double> r(T);
  for (int t = 0; t < T; ++t) {
    const float* l = logits_host + (size_t)t * E;
    // top-2 by (logit descending, expert index ascending); -0 == +0 as floats
    int a = 0;
    for (int e = 1; e < E; ++e)
      if (l[e] > l[a]) a = e;
    int b = a == 0 ? 1 : 0;
    for (int e = 0; e < E; ++e)
      if (e != a && l[e] > l[b]) b = e;
    if (!std::isfinite(l[a]) || !std::isfinite(l[b])) return fail(MC_EINVAL, "non-finite logit at token %d", t);
    r[t] = std::exp((double)l[b] - (double)l[a]);
  }
  std::sort(r.begin(), r.end());
  const double m = (T & 1) ? r[T / 2] : 0.5 * (r[T / 2 - 1] + r[T / 2]);
  *mu = m;
  *tau = m / (1.0 + m);
  return MC_OK;
}

// ------------------------------------------------------------------ PMQ --
// Sec. 3.2.1: expert significance from calibration routing; each token's top-k
// by (logit descending, expert index ascending), routing weights = softmax
// over the selected k (fp64, summed in rank order).
mc_status mc_pmq_significance(const float* logits_host, int T, int E, int k, double* phi, double* w) {
  if (!logits_host || !phi || !w) return fail(MC_EINVAL, "NULL argument");
  if (T < 1 || E < 1 || E > MC_MAX_EXPERTS || k < 1 || k > E || k > MC_MAX_TOPK)
    return fail(MC_EINVAL, "bad shape T=%d E=%d k=%d", T, E, k);
  std::vector<double> n(E, 0.0), s(E, 0.0);
  std::vector<int> order(E);
  for (int t = 0; t < T; ++t) {
    const float* l = logits_host + (size_t)t * E;
    for (int e = 0; e < E; ++e) {
      if (!std::isfinite(l[e])) return fail(MC_EINVAL, "non-finite logit at token %d", t);
      order[e] = e;
    }
    std::partial_sort(order.begin(), order.begin() + k, order.end(), [l](int a, int b) {
      return l[a] > l[b] || (l[a] == l[b] && a < b);   // -0 == +0 as floats
    });
    double ex[MC_MAX_TOPK], sum = 0.0;
    for (int r = 0; r < k; ++r) {
      ex[r] = std::exp((double)l[order[r]] - (double)l[order[0]]);
      sum += ex[r];
    }
    for (int r = 0; r < k; ++r) {
      n[order[r]] += 1.0;
      s[order[r]] += ex[r] / sum;
    }
  }
  for (int e = 0; e < E; ++e) {
    phi[e] = n[e] / T;
    w[e] = s[e] / T;
  }
  return MC_OK;
}

// Sec. 3.2.2, Eq. 4: choose b_i in {1,2,3} minimising
// sum_i phi_i^alpha w_i^beta eps_{i,b_i}^gamma subject to sum_i b_i =
// total_bits, at least one expert at 3 bits and one at 2.  Exact: dynamic
// programme over experts in index order with state (bits used, has a 2, has a
// 3); the objective of an allocation is summed in expert order in fp64, and
// among equal objectives the lexicographically smallest width vector wins.
mc_status mc_pmq_allocate(const double* phi, const double* w, const double* eps, int E, double alpha,
                          double beta, double gamma, int total_bits, int* bits, double* objective) {
  if (!phi || !w || !eps || !bits) return fail(MC_EINVAL, "NULL argument");
  if (E < 2 || E > MC_MAX_EXPERTS) return fail(MC_EINVAL, "E=%d outside [2, %d]", E, MC_MAX_EXPERTS);
  if (!(alpha >= 0.0) || !(beta >= 0.0) || !(gamma > 0.0) || !std::isfinite(alpha + beta + gamma))
    return fail(MC_EINVAL, "exponents alpha=%g beta=%g gamma=%g (need alpha, beta >= 0, gamma > 0)", alpha,
                beta, gamma);
  if (total_bits < E + 3 || total_bits > 3 * E - 1)
    return fail(MC_EINVAL, "total_bits=%d not reachable with one 3-bit and one 2-bit expert among %d "
                "(range [%d, %d])", total_bits, E, E + 3, 3 * E - 1);
  std::vector<double> term((size_t)E * 3);
  for (int i = 0; i < E; ++i) {
    if (!(phi[i] >= 0.0) || !(w[i] >= 0.0) || !std::isfinite(phi[i]) || !std::isfinite(w[i]))
      return fail(MC_EINVAL, "expert %d: phi=%g w=%g must be finite and >= 0", i, phi[i], w[i]);
    for (int b = 0; b < 3; ++b) {
      const double e = eps[(size_t)i * 3 + b];
      if (!(e >= 0.0) || !std::isfinite(e)) return fail(MC_EINVAL, "expert %d: eps[%d]=%g", i, b + 1, e);
      term[(size_t)i * 3 + b] = std::pow(phi[i], alpha) * std::pow(w[i], beta) * std::pow(e, gamma);
    }
  }
  const int S = 3 * E + 1;
  const double inf = INFINITY;
  // state (s, f): f bit 0 = some expert at 2 bits, bit 1 = some expert at 3 bits
  std::vector<double> cost(S * 4, inf), ncost(S * 4);
  std::vector<uint8_t> pre((size_t)S * 4 * E, 0), npre((size_t)S * 4 * E);
  cost[0] = 0.0;
  for (int i = 0; i < E; ++i) {
    std::fill(ncost.begin(), ncost.end(), inf);
    for (int s = 0; s <= 3 * i; ++s) {
      for (int f = 0; f < 4; ++f) {
        const double c = cost[s * 4 + f];
        if (c == inf) continue;
        const uint8_t* pp = &pre[((size_t)s * 4 + f) * E];
        for (int b = 1; b <= 3; ++b) {
          const int s2 = s + b, f2 = f | (b == 2 ? 1 : 0) | (b == 3 ? 2 : 0);
          const double c2 = c + term[(size_t)i * 3 + b - 1];
          double& dst = ncost[s2 * 4 + f2];
          uint8_t* dp = &npre[((size_t)s2 * 4 + f2) * E];
          bool better = c2 < dst;
          if (!better && c2 == dst) {        // equal objective: the lexicographically smaller vector
            int j = 0;
            while (j < i && pp[j] == dp[j]) ++j;
            better = (j < i) ? pp[j] < dp[j] : b < dp[i];
          }
          if (better) {
            dst = c2;
            std::memcpy(dp, pp, (size_t)i);
            dp[i] = (uint8_t)b;
          }
        }
      }
    }
    cost.swap(ncost);
    pre.swap(npre);
  }
  const double best = cost[total_bits * 4 + 3];
  if (best == inf) return fail(MC_EINVAL, "no allocation reaches total_bits=%d", total_bits);
  const uint8_t* bp = &pre[((size_t)total_bits * 4 + 3) * E];
  for (int i = 0; i < E; ++i) bits[i] = bp[i];
  if (objective) *objective = best;
  return MC_OK;
}

mc_status mc_timing_enable(int on) {
  mc::timing_enable(on);
  return MC_OK;
}

mc_status mc_timing_read(const char* kernel, double* total_ms, int* launches) {
  if (!kernel || !total_ms || !launches) return fail(MC_EINVAL, "NULL argument");
  const int site = mc::timing_site(kernel);
  if (site < 0) return fail(MC_EINVAL, "unknown kernel name '%s'", kernel);
  return hip_status(mc::timing_read(site, total_ms, launches), "mc_timing_read");
}

}  // extern "C"
