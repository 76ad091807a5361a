// prefill.hip -- preparation of the prefill grouped GEMMs (expert tile tables
// and the bf16 fragment-tiled copy of the routed token rows, in one launch)
// and their launcher.  The GEMM kernels are in prefill.hpp, one file per
// group size.
#include "prefill.hpp"

namespace mc {

extern template hipError_t launch_prefill_gemm<1>(const LayerArgs&, const int32_t*, const PrefillTables&,
                                                  const PrefillGemm&, bool, hipStream_t);
extern template hipError_t launch_prefill_gemm<2>(const LayerArgs&, const int32_t*, const PrefillTables&,
                                                  const PrefillGemm&, bool, hipStream_t);
extern template hipError_t launch_prefill_gemm<4>(const LayerArgs&, const int32_t*, const PrefillTables&,
                                                  const PrefillGemm&, bool, hipStream_t);

// The prefill's preparation, one workgroup per fragment row f (f_max of
// them).  Every workgroup first scans the expert counts itself (thread e:
// fragment rows ceil(M_e/32) and m-tiles of PfCfg::kTokens tokens; wave
// prefix sums), which gives the expert that f belongs to; workgroup 0 also
// writes the tables the GEMMs read.  Counts outside [0, P] are taken as 0,
// and tables that would not fit their capacity are left empty (no m-tiles,
// no fragment rows), so inconsistent routing cannot make any later access
// leave its buffer.
// Then f's 32 routed rows of x (zero past the expert's count) are copied
// into the fragment layout (bf16, unchanged), with the sum of each group of G
// columns of each row in fp32.  Column blocks of 512:
// each wave reads whole rows of the block (64 lanes x 16 consecutive bytes)
// into a row-major LDS tile and forms the group sums of its pieces (the GP =
// G/8 lanes of a group add with the DPP butterfly of the decode slabs); then
// the workgroup writes the block's fragments (contiguous in the fragment
// layout) from the tile with consecutive 16-byte stores.
constexpr int kGatherThreads = 256;
constexpr int kGatherCols = 512;                     // columns of a block: 8 per lane
constexpr int kGatherStride = kGatherCols + 8;       // LDS row stride (elements): rows start on different banks

template <int GP>
__global__ void __launch_bounds__(kGatherThreads) prefill_prep_kernel(const uint16_t* __restrict__ x, int d, int E,
                                                                      const int32_t* __restrict__ counts,
                                                                      const int32_t* __restrict__ offsets,
                                                                      const int32_t* __restrict__ pair_token,
                                                                      PrefillTables tb, uint16_t* __restrict__ xt,
                                                                      float* __restrict__ xsum) {
  static_assert(kPfFragRows * kGatherStride * 2 <= 64 * 1024, "gather tile");
  static_assert(kGatherThreads >= MC_MAX_EXPERTS, "a thread per expert");
  constexpr int kWaves = kGatherThreads / 64;
  __shared__ __attribute__((aligned(16))) uint16_t tile[kPfFragRows * kGatherStride];
  __shared__ int wf[kWaves], wm[kWaves], s_e, s_fb;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int f = blockIdx.x;

  // tables: exclusive prefix sums of the experts' fragment rows and m-tiles
  const int c = tid < E ? checked_count(counts[tid], tb.P) : 0;
  const int nf = (c + kPfFragRows - 1) / kPfFragRows;
  const int nm = (c + PfCfg::kTokens - 1) / PfCfg::kTokens;
  int sf = nf, sm = nm;
  for (int off = 1; off < 64; off <<= 1) {
    const int a = __shfl_up(sf, off), b = __shfl_up(sm, off);
    if (lane >= off) {
      sf += a;
      sm += b;
    }
  }
  if (lane == 63) {
    wf[wave] = sf;
    wm[wave] = sm;
  }
  __syncthreads();
  int tf = 0, tm = 0, fb = sf - nf, mb = sm - nm;
  for (int w = 0; w < kWaves; ++w) {
    if (w < wave) {
      fb += wf[w];
      mb += wm[w];
    }
    tf += wf[w];
    tm += wm[w];
  }
  const bool fits = tf <= tb.f_max && tm <= tb.mt_max;
  if (f == 0) {
    if (!fits) {
      for (int i = tid; i <= E; i += kGatherThreads) tb.ftile_base[i] = 0;
      if (tid == 0) *tb.mt_count = 0;
    } else {
      if (tid < E) {
        tb.ftile_base[tid] = fb;
        for (int i = 0; i < nm; ++i) {
          tb.mt_e[mb + i] = tid;
          tb.mt_j[mb + i] = i;
        }
      }
      if (tid == 0) {
        tb.ftile_base[E] = tf;
        *tb.mt_count = tm;
      }
    }
  }
  if (!fits || f >= tf) return;   // workgroup-uniform
  if (tid < E && fb <= f && f < fb + nf) {   // exactly one expert holds f
    s_e = tid;
    s_fb = fb;
  }
  __syncthreads();
  const int e = s_e;
  int ebase, ecount;
  expert_range_offsets(offsets, e, tb.P, ebase, ecount);
  const int pos0 = ebase + (f - s_fb) * kPfFragRows;
  const int pend = ebase + ecount;
  constexpr int kRowsPerWave = kPfFragRows / (kGatherThreads / 64);
  // this wave's rows: m = wave + 4 j; token rows (or none: zero rows)
  const uint16_t* src[kRowsPerWave];
#pragma unroll
  for (int j = 0; j < kRowsPerWave; ++j) {
    const int pos = pos0 + wave + 4 * j;
    src[j] = pos < pend ? x + (size_t)clamp_token(pair_token[pos], tb.T) * d : nullptr;
  }
  const int ng = d / (8 * GP);
  unsigned char* out = reinterpret_cast<unsigned char*>(xt) + frag_offset(f, 0, 0, d);
  for (int c0 = 0; c0 < d; c0 += kGatherCols) {
    const int w = (d - c0) < kGatherCols ? (d - c0) : kGatherCols;   // a multiple of 128
    const bool on = 8 * lane < w;
    u32x4 v[kRowsPerWave];
#pragma unroll
    for (int j = 0; j < kRowsPerWave; ++j) {
      v[j] = u32x4{0u, 0u, 0u, 0u};
      if (on && src[j]) v[j] = *reinterpret_cast<const u32x4*>(src[j] + c0 + 8 * lane);
    }
    if (c0 > 0) __syncthreads();   // the previous block's tile has been written out
#pragma unroll
    for (int j = 0; j < kRowsPerWave; ++j) {
      const int m = wave + 4 * j;
      if (on) *reinterpret_cast<u32x4*>(tile + m * kGatherStride + 8 * lane) = v[j];
      const float sum = lane_group_sum<GP>(sum8<false>(v[j]));
      if (on && lane % GP == 0) xsum[((size_t)f * ng + (c0 + 8 * lane) / (8 * GP)) * 32 + m] = sum;
    }
    __syncthreads();
    // fragment fi of the block, piece mm: row mm % 32, columns 16 fi + 8 (mm / 32)
    const int pieces = (w / 16) * 64;
    for (int p = threadIdx.x; p < pieces; p += kGatherThreads) {
      const int fi = p >> 6, mm = p & 63;
      *reinterpret_cast<u32x4*>(out + ((size_t)(c0 / 16 + fi) * 64 + mm) * 16) =
          *reinterpret_cast<const u32x4*>(tile + (mm & 31) * kGatherStride + 16 * fi + 8 * (mm >> 5));
    }
  }
}

static size_t round256(size_t b) { return ((b + 255) / 256) * 256; }

PrefillLayout prefill_layout(int T, int E, int k, int d, int ffn) {
  PrefillLayout pl;
  const size_t P = (size_t)T * k;
  pl.f_max = (int)((P + (size_t)(kPfFragRows - 1) * E) / kPfFragRows);
  pl.mt_max = (int)((P + (size_t)(PfCfg::kTokens - 1) * E) / PfCfg::kTokens);
  const int nt_down = (d + PfCfg::kRowsDown - 1) / PfCfg::kRowsDown;
  // Split the down GEMM's reduction so that its workgroups fill the 256 CUs
  // in whole rounds: pick s minimising rounds(s) / s (the time of one round
  // shrinks as 1/s), the smallest on ties; at least 8 chunks per split.
  const long long wgs = (long long)pl.mt_max * nt_down;
  int maxs = (ffn / kTileCols) / 8;
  if (maxs > 4) maxs = 4;
  int s = 1;
  for (int c = 2; c <= maxs; ++c)
    if ((double)((wgs * c + 255) / 256) / c < (double)((wgs * s + 255) / 256) / s - 1e-9) s = c;
  pl.nsplit = s;
  // the GEMMs stage whole m-tiles: kTiles - 1 padding fragment rows past the last one
  const size_t rows = (size_t)(pl.f_max + PfCfg::kTiles) * kPfFragRows;
  pl.tables = 0;
  const size_t tab = (size_t)(E + 1 + 2 * pl.mt_max + 1) * sizeof(int32_t);
  pl.x = round256(tab);
  pl.xsum = pl.x + round256(rows * d * sizeof(uint16_t));
  pl.h = pl.xsum + round256(rows * (d / 32) * sizeof(float));   // G >= 32
  pl.hsum = pl.h + round256(rows * ffn * sizeof(uint16_t));
  pl.part = pl.hsum + round256(rows * (ffn / 32) * sizeof(float));
  pl.total = pl.part + (size_t)pl.nsplit * P * d * sizeof(float);
  return pl;
}

hipError_t launch_prefill(const uint16_t* x, const LayerArgs& L, const mc_routing& r, void* ws,
                          float** partial, size_t* part_stride, int* nsplit, hipStream_t stream) {
  const PrefillLayout pl = prefill_layout(r.T, r.E, r.k, L.d, L.ffn);
  char* base = static_cast<char*>(ws);
  PrefillTables tb;
  int32_t* t = reinterpret_cast<int32_t*>(base + pl.tables);
  tb.ftile_base = t;
  tb.mt_e = t + (r.E + 1);
  tb.mt_j = tb.mt_e + pl.mt_max;
  tb.mt_count = tb.mt_j + pl.mt_max;
  tb.f_max = pl.f_max;
  tb.mt_max = pl.mt_max;
  tb.T = r.T;
  tb.P = r.T * r.k;
  uint16_t* xt = reinterpret_cast<uint16_t*>(base + pl.x);
  float* xsum = reinterpret_cast<float*>(base + pl.xsum);
  uint16_t* ht = reinterpret_cast<uint16_t*>(base + pl.h);
  float* hsum = reinterpret_cast<float*>(base + pl.hsum);
  *partial = reinterpret_cast<float*>(base + pl.part);
  *part_stride = (size_t)r.T * r.k * L.d;
  *nsplit = pl.nsplit;

  timing_begin(stream, kSitePrefillPrep);
  if (L.G == 128)
    hipLaunchKernelGGL(prefill_prep_kernel<16>, dim3(pl.f_max), dim3(kGatherThreads), 0, stream, x, L.d, r.E,
                       r.counts, r.offsets, r.pair_token, tb, xt, xsum);
  else if (L.G == 64)
    hipLaunchKernelGGL(prefill_prep_kernel<8>, dim3(pl.f_max), dim3(kGatherThreads), 0, stream, x, L.d, r.E,
                       r.counts, r.offsets, r.pair_token, tb, xt, xsum);
  else
    hipLaunchKernelGGL(prefill_prep_kernel<4>, dim3(pl.f_max), dim3(kGatherThreads), 0, stream, x, L.d, r.E,
                       r.counts, r.offsets, r.pair_token, tb, xt, xsum);
  timing_end(stream, kSitePrefillPrep);
  hipError_t err = hipGetLastError();
  if (err != hipSuccess) return err;

  PrefillGemm gu;
  gu.a = xt;
  gu.asum = xsum;
  gu.K = L.d;
  gu.n_tiles = L.ffn / PfCfg::kRowsGateUp;
  gu.c_per_split = L.d / kTileCols;
  gu.nsplit = 1;
  gu.h = ht;
  gu.hsum = hsum;
  gu.partial = nullptr;
  gu.part_stride = 0;
  timing_begin(stream, kSiteGateUp);
  if (L.G == 128) err = launch_prefill_gemm<1>(L, r.offsets, tb, gu, true, stream);
  else if (L.G == 64) err = launch_prefill_gemm<2>(L, r.offsets, tb, gu, true, stream);
  else err = launch_prefill_gemm<4>(L, r.offsets, tb, gu, true, stream);
  timing_end(stream, kSiteGateUp);
  if (err != hipSuccess) return err;

  PrefillGemm dn;
  const int ntk = L.ffn / kTileCols;
  dn.a = ht;
  dn.asum = hsum;
  dn.K = L.ffn;
  dn.n_tiles = (L.d + PfCfg::kRowsDown - 1) / PfCfg::kRowsDown;
  dn.c_per_split = (ntk + pl.nsplit - 1) / pl.nsplit;
  dn.nsplit = pl.nsplit;
  dn.h = nullptr;
  dn.hsum = nullptr;
  dn.partial = *partial;
  dn.part_stride = *part_stride;
  timing_begin(stream, kSiteDown);
  if (L.G == 128) err = launch_prefill_gemm<1>(L, r.offsets, tb, dn, false, stream);
  else if (L.G == 64) err = launch_prefill_gemm<2>(L, r.offsets, tb, dn, false, stream);
  else err = launch_prefill_gemm<4>(L, r.offsets, tb, dn, false, stream);
  timing_end(stream, kSiteDown);
  return err;
}

}  // namespace mc
