// timing.hip -- optional per-kernel timing with HIP events on the launch stream.
// Disabled by default; when enabled every kernel launch of the library is
// bracketed by two events recorded on the caller's stream.
#include <atomic>
#include <cstring>
#include <mutex>
#include <vector>

#include "mc_internal.hpp"

namespace mc {
namespace {

const char* const kSiteNames[kNumSites] = {
    "pack_scale_zero", "pack_codes", "export", "route_fused", "route_select",
    "route_lists",     "gateup",     "down",   "combine", "prefill_prep",
    "importance_colsum", "importance_finish", "importance_select", "rmsnorm", "router", "gptq_hessian", "gptq_factor", "gptq_quantize"};

struct Pair {
  hipEvent_t start, stop;
};

std::atomic<int> g_enabled{0};
std::mutex g_mu;
std::vector<Pair> g_done[kNumSites];
hipEvent_t g_open[kNumSites];
std::vector<hipEvent_t> g_pool;

hipEvent_t get_event() {
  if (!g_pool.empty()) {
    hipEvent_t e = g_pool.back();
    g_pool.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  // timing only: no system-scope fence when an event completes (the default
  // one writes back and invalidates the caches between the bracketed kernels)
  if (hipEventCreateWithFlags(&e, hipEventDisableSystemFence) != hipSuccess) return nullptr;
  return e;
}

void recycle_all() {
  for (int s = 0; s < kNumSites; ++s) {
    for (auto& p : g_done[s]) {
      g_pool.push_back(p.start);
      g_pool.push_back(p.stop);
    }
    g_done[s].clear();
  }
}

}  // namespace

void timing_begin(hipStream_t stream, int site) {
  if (!g_enabled.load(std::memory_order_relaxed)) return;
  std::lock_guard<std::mutex> lk(g_mu);
  hipEvent_t e = get_event();
  if (e && hipEventRecord(e, stream) == hipSuccess) g_open[site] = e;
  else g_open[site] = nullptr;
}

void timing_end(hipStream_t stream, int site) {
  if (!g_enabled.load(std::memory_order_relaxed)) return;
  std::lock_guard<std::mutex> lk(g_mu);
  if (!g_open[site]) return;
  hipEvent_t e = get_event();
  if (e && hipEventRecord(e, stream) == hipSuccess) g_done[site].push_back({g_open[site], e});
  g_open[site] = nullptr;
}

int timing_site(const char* name) {
  for (int s = 0; s < kNumSites; ++s)
    if (std::strcmp(name, kSiteNames[s]) == 0) return s;
  return -1;
}

hipError_t timing_read(int site, double* total_ms, int* launches) {
  std::lock_guard<std::mutex> lk(g_mu);
  double sum = 0.0;
  for (auto& p : g_done[site]) {
    hipError_t err = hipEventSynchronize(p.stop);
    if (err != hipSuccess) return err;
    float ms = 0.0f;
    err = hipEventElapsedTime(&ms, p.start, p.stop);
    if (err != hipSuccess) return err;
    sum += ms;
  }
  *total_ms = sum;
  *launches = (int)g_done[site].size();
  return hipSuccess;
}

void timing_enable(int on) {
  std::lock_guard<std::mutex> lk(g_mu);
  recycle_all();
  g_enabled.store(on ? 1 : 0);
}

}  // namespace mc
