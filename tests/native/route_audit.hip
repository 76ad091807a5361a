// route_audit.hip -- host-side audit of the routing-derived indices of the
// forward kernels (test support, not part of the library).
//
// The kernels derive every index into their buffers from the routing
// buffers (counts, offsets, pair_token, pair_pos) through the helpers of
// mc_device.hpp: expert_range, expert_range_offsets, pair_block,
// clamp_token, checked_pos, checked_count.  This file compiles those helpers
// for the host and walks, for arbitrary (garbage) routing buffers, every
// index the kernels form from them, in the kernels' own loop structure:
//   decode GEMVs  (decode.hpp)   pair blocks of 16 per expert: pair_token
//                                reads, x rows, h / partial writes;
//   combine       (forward.hip)  per (token, rank): partial reads;
//   prefill       (prefill.hip)  set-up tables, gather reads and writes,
//                                the down GEMM's partial writes.
// Returns the number of indices outside their buffers (0 expected).  With
// raw != 0 the helpers' range checks are bypassed (raw counts, offsets,
// tokens and positions): the test uses that to show its garbage inputs do
// reach past the buffers, so that a zero count means the checks held.
#include "../../paper_2410_06270_amd/csrc/prefill.hpp"   // PfCfg; includes mc_device.hpp

#include <vector>

using namespace mc;

namespace {

long long g_bad = 0;
inline void check(long long idx, long long size) {
  if (idx < 0 || idx >= size) ++g_bad;
}

}  // namespace

// Tokens per prefill m-tile (the workspace capacities depend on it).
extern "C" int route_audit_mt_tokens() { return PfCfg::kTokens; }

extern "C" long long route_audit(int T, int E, int k, int d, int ffn, const int32_t* counts,
                                 const int32_t* offsets, const int32_t* pair_token, const int32_t* pair_pos,
                                 int f_max, int mt_max, int raw) {
  g_bad = 0;
  const int P = T * k;
  auto range = [&](int e, int& b, int& c) {
    if (raw) { b = offsets[e]; c = counts[e]; } else expert_range(counts, offsets, e, P, b, c);
  };
  auto range_off = [&](int e, int& b, int& c) {
    if (raw) { b = offsets[e]; c = offsets[e + 1] - offsets[e]; } else expert_range_offsets(offsets, e, P, b, c);
  };
  auto tok = [&](int t) { return raw ? t : clamp_token(t, T); };
  auto cpos = [&](int q) { return raw ? q : checked_pos(q, P); };
  auto ccount = [&](int c) { return raw ? (c < 0 ? 0 : c) : checked_count(c, P); };
  // decode GEMVs: every expert's pair blocks (the plan covers exactly these)
  for (int e = 0; e < E; ++e) {
    int eb, ec;
    range(e, eb, ec);
    if (raw && ec > 4 * P) ec = 4 * P;                        // keep the raw walk short
    for (int j = 0; 16 * j < ec; ++j) {
      int pbase, nt;
      pair_block(eb, ec, j, 16, pbase, nt);
      for (int m = 0; m < nt; ++m) {
        check(pbase + m, P);                                  // pair_token read
        if (pbase + m < 0 || pbase + m >= P) continue;
        const int t = tok(pair_token[pbase + m]);
        check((long long)t * d, (long long)T * d);            // x row
        check((long long)(pbase + m) * ffn + ffn - 1, (long long)P * ffn);   // h row written / read
        check((long long)(pbase + m) * d + d - 1, (long long)P * d);         // partial row written
      }
    }
  }
  // combine: per (token, rank)
  for (int t = 0; t < T; ++t)
    for (int r = 0; r < k; ++r) {
      const int pos = cpos(pair_pos[t * k + r]);
      if (raw || pos >= 0) check((long long)pos * d + d - 1, (long long)P * d);
    }
  // prefill set-up: fragment rows of 32 and m-tiles of PfCfg::kTokens per
  // expert, the tables left empty when they would not fit their capacity
  std::vector<int> ftile_base(E + 1, 0), ftile_e(f_max > 0 ? f_max : 1, -1);
  int nf_tot = 0, nm_tot = 0;
  for (int e = 0; e < E; ++e) {
    const int c = ccount(counts[e]);
    nf_tot += (c + 31) / 32;
    nm_tot += (c + PfCfg::kTokens - 1) / PfCfg::kTokens;
  }
  if (nf_tot <= f_max && nm_tot <= mt_max) {
    int fb = 0;
    for (int e = 0; e < E; ++e) {
      const int c = ccount(counts[e]);
      ftile_base[e] = fb;
      for (int i = 0; i < (c + 31) / 32; ++i) {
        check(fb + i, f_max);
        ftile_e[fb + i] = e;
      }
      fb += (c + 31) / 32;
    }
    ftile_base[E] = fb;
  }
  // gather: fragment rows f < ftile_base[E]
  for (int f = 0; f < ftile_base[E]; ++f) {
    const int e = ftile_e[f];
    check(e, E);
    if (e < 0 || e >= E) continue;
    int ebase, ecount;
    range_off(e, ebase, ecount);
    const int pos0 = ebase + (f - ftile_base[e]) * 32;
    for (int m = 0; m < 32; ++m) {
      const int pos = pos0 + m;
      if (pos < ebase + ecount) {
        check(pos, P);                                        // pair_token read
        if (pos >= 0 && pos < P) check((long long)tok(pair_token[pos]) * d, (long long)T * d);
      }
    }
    check(f, f_max);                                          // the tiled copy written
  }
  // prefill GEMMs: m-tiles of PfCfg::kTokens pairs of each expert, the
  // staged fragment rows and the down GEMM's partial writes
  for (int e = 0; e < E; ++e) {
    if (!(nf_tot <= f_max && nm_tot <= mt_max)) break;
    const int c = ccount(counts[e]);
    int ebase, ecount;
    range_off(e, ebase, ecount);
    for (int j = 0; PfCfg::kTokens * j < c; ++j) {
      // staged fragment rows (kTiles padding rows past f_max)
      check(ftile_base[e] + PfCfg::kTiles * j + PfCfg::kTiles - 1, f_max + PfCfg::kTiles);
      for (int m = 0; m < PfCfg::kTokens; ++m) {
        const int pos = ebase + PfCfg::kTokens * j + m;
        if (pos < ebase + ecount) check((long long)pos * d + d - 1, (long long)P * d);
      }
    }
  }
  return g_bad;
}
