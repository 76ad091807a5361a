// importance.hip -- token importance (Sec. 3.3.2, Eq. 6) and the protected
// set that route_and_prune takes.
//
// From causal attention probabilities A[h][i][j] (query i, key j <= i) and
// the token vectors x_j, with 0-based j:
//   I_j = ||x_j||_1 * (1/H) * sum_h sum_{i=j}^{L-1} A[h][i][j] / (L - j),
// the mean attention key j receives from the L - j queries that see it,
// averaged over heads and weighted by the token's l1 norm.  The protected set
// is the n = floor(rho*L + 1/2) largest I_j, equal values ordered by lower
// index.  All sums are fp32 in a fixed order (deterministic).
//
// Kernels:
//   importance_colsum_kernel  one workgroup per 128x128 tile of the lower
//     triangle (query tile >= key tile) and slice of heads: per-key partial
//     sums; plus workgroups of 16 tokens for the l1 norms;
//   importance_finish_kernel  one wave per key: its partials, the norm,
//     I_j, and the selection key (I_j bits << 32 | ~j: larger key = larger
//     I_j, then lower j);
//   importance_select_kernel  one workgroup: radix selection of the n-th
//     largest key (up to 8 passes of 8 bits), then the mask.
// The attention map is read once, in 256-byte row pieces per wave (HBM-bound).
#include "mc_internal.hpp"

namespace mc {

constexpr int kImpTile = 128;
constexpr int kImpThreads = 256;
constexpr int kImpSelectThreads = 1024;

__host__ __device__ static inline int imp_tiles(int L) { return (L + kImpTile - 1) / kImpTile; }

// Heads are split over blockIdx.y so that a launch has about 4096 workgroups
// (a 4096-token map has only 528 tile pairs): hs head slices of hpw heads.
static int imp_pairs(int L) {
  const int nt = imp_tiles(L);
  return nt * (nt + 1) / 2;
}

static void imp_head_split(int H, int L, int& hs, int& hpw) {
  const int want = (4096 + imp_pairs(L) - 1) / imp_pairs(L);
  hs = want < H ? want : H;
  hpw = (H + hs - 1) / hs;
  hs = (H + hpw - 1) / hpw;
}

static size_t imp_partial_bytes(int H, int L) {
  int hs, hpw;
  imp_head_split(H, L, hs, hpw);
  return (((size_t)imp_pairs(L) * hs * kImpTile * sizeof(float) + 255) / 256) * 256;
}

static size_t imp_norm_bytes(int L) { return (((size_t)L * sizeof(float) + 255) / 256) * 256; }

// Workspace: partial sums | l1 norms | selection keys.
size_t importance_workspace_bytes(int H, int L) {
  return imp_partial_bytes(H, L) + imp_norm_bytes(L) + (size_t)L * sizeof(uint64_t);
}

// Pair index p -> (query tile, key tile), ordered by key tile then query tile.
__device__ __forceinline__ void imp_pair(int p, int nt, int& tq, int& tk) {
  int tkk = 0, base = 0;
  while (p >= base + (nt - tkk)) {
    base += nt - tkk;
    ++tkk;
  }
  tk = tkk;
  tq = tkk + (p - base);
}

__device__ __forceinline__ size_t imp_pair_base(int tk, int nt) {
  return (size_t)tk * nt - (size_t)tk * (tk - 1) / 2;   // sum_{t < tk} (nt - t)
}

__device__ __forceinline__ void imp_add8(float (&acc)[8], const u32x4& v) {
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    acc[2 * q] += bf16_bits_to_float(v[q] & 0xffffu);
    acc[2 * q + 1] += bf16_bits_to_float(v[q] >> 16);
  }
}

// Adds the 8 keys j0..j0+7 of one row whose index exceeds j0 by di; keys
// above the diagonal (j > i, i.e. c > di) are skipped.
__device__ __forceinline__ void imp_add8_causal(float (&acc)[8], const u32x4& v, int di) {
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    acc[2 * q] += 2 * q <= di ? bf16_bits_to_float(v[q] & 0xffffu) : 0.0f;
    acc[2 * q + 1] += 2 * q + 1 <= di ? bf16_bits_to_float(v[q] >> 16) : 0.0f;
  }
}

// One head's 8 rows (already loaded) into the column sums; DIAG masks j > i.
template <bool DIAG>
__device__ __forceinline__ void imp_add_rows(float (&acc)[8], const u32x4* v, int di0) {
#pragma unroll
  for (int k = 0; k < 8; ++k) {
    if (DIAG)
      imp_add8_causal(acc, v[k], di0 + 16 * k);
    else
      imp_add8(acc, v[k]);
  }
}

// Full tiles with VEC (L a multiple of 8, 16-byte aligned map): per head, the
// thread's 8 rows as 16-byte loads, all issued before any is used (with 4+
// waves per SIMD that keeps enough bytes in flight to stream HBM).
// di0 = first row - j0.
template <bool DIAG>
__device__ __forceinline__ void imp_full_tile(float (&acc)[8], const uint16_t* p, size_t hstride, size_t rstride,
                                              int nh, int di0) {
  for (int h = 0; h < nh; ++h, p += hstride) {
    u32x4 v[8];
#pragma unroll
    for (int k = 0; k < 8; ++k) v[k] = *reinterpret_cast<const u32x4*>(p + k * rstride);
    imp_add_rows<DIAG>(acc, v, di0);
  }
}

__device__ __forceinline__ float imp_abs_sum8(const u32x4& v) {
  float s = 0.0f;
#pragma unroll
  for (int q = 0; q < 4; ++q) s += fabsf(bf16_bits_to_float(v[q] & 0xffffu)) + fabsf(bf16_bits_to_float(v[q] >> 16));
  return s;
}

// l1 norms of kNormTokens tokens, one wave per token at a time; XVEC = 16-byte
// loads (d a multiple of 8, x 16-byte aligned), 8 in flight per lane.
constexpr int kNormTokens = 16;

__device__ void imp_norms(const uint16_t* __restrict__ x, int L, int d, bool xvec, int blk,
                          float* __restrict__ norms) {
  const int lane = threadIdx.x & 63, nw = kImpThreads / 64;
  for (int j = blk * kNormTokens + wave_id(); j < min(L, (blk + 1) * kNormTokens); j += nw) {
    const uint16_t* xr = x + (size_t)j * d;
    float n1 = 0.0f;
    if (xvec) {
      int c = 8 * lane;
      for (; c + 7 * 512 < d; c += 8 * 512) {
        u32x4 v[8];
#pragma unroll
        for (int k = 0; k < 8; ++k) v[k] = *reinterpret_cast<const u32x4*>(xr + c + 512 * k);
#pragma unroll
        for (int k = 0; k < 8; ++k) n1 += imp_abs_sum8(v[k]);
      }
      for (; c < d; c += 512) n1 += imp_abs_sum8(*reinterpret_cast<const u32x4*>(xr + c));
    } else {
      for (int c = lane; c < d; c += 64) n1 += fabsf(bf16_bits_to_float(xr[c]));
    }
    for (int off = 32; off >= 1; off >>= 1) n1 += __shfl_xor(n1, off);
    if (lane == 0) norms[j] = n1;
  }
}

// Tile pair `pair` and head slice `slice`.  Thread (column group cg of 8 keys,
// row phase r of 16): rows i = r, r+16, ... of the query tile, keys
// 8cg..8cg+7 of the key tile.  Full tiles take imp_full_tile (the diagonal one
// masking j > i after the load); ragged tiles and maps without VEC check every
// element against i >= j and the map's edge.
template <bool VEC>
__device__ void imp_colsum_tile(const uint16_t* __restrict__ attn, int H, int L, int hpw, int pair, int slice,
                                float* __restrict__ out) {
  __shared__ float red[16][kImpTile + 4];
  const int nt = imp_tiles(L);
  int tq, tk;
  imp_pair(pair, nt, tq, tk);
  const int h0 = slice * hpw, h1 = min(H, h0 + hpw);
  const int cg = threadIdx.x & 15, r = threadIdx.x >> 4;
  const int j0 = tk * kImpTile + 8 * cg;
  float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
  const size_t hstride = (size_t)L * L, rstride = (size_t)16 * L;
  if (VEC && (tq + 1) * kImpTile <= L) {
    const int i0 = tq * kImpTile + r;
    const uint16_t* p = attn + (size_t)h0 * hstride + (size_t)i0 * L + j0;
    if (tq > tk)
      imp_full_tile<false>(acc, p, hstride, rstride, h1 - h0, 0);
    else
      imp_full_tile<true>(acc, p, hstride, rstride, h1 - h0, i0 - j0);
  } else {
    for (int h = h0; h < h1; ++h) {
      const uint16_t* ah = attn + (size_t)h * hstride;
      for (int ii = r; ii < kImpTile; ii += 16) {
        const int i = tq * kImpTile + ii;
        if (i >= L) break;
        const uint16_t* row = ah + (size_t)i * L + j0;
        if (VEC && j0 + 7 < L && j0 + 7 <= i) {
          imp_add8(acc, *reinterpret_cast<const u32x4*>(row));
        } else {
#pragma unroll
          for (int c = 0; c < 8; ++c)
            if (j0 + c < L && j0 + c <= i) acc[c] += bf16_bits_to_float(row[c]);
        }
      }
    }
  }
#pragma unroll
  for (int c = 0; c < 8; ++c) red[r][8 * cg + c] = acc[c];
  __syncthreads();
  if (threadIdx.x < kImpTile) {
    float s = 0.0f;
    for (int q = 0; q < 16; ++q) s += red[q][threadIdx.x];   // row phases in order
    out[threadIdx.x] = s;
  }
}

// One launch, two kinds of workgroup: the first n_norm blocks compute the l1
// norms (dispatched first, they overlap the attention stream), the rest one
// (head slice, tile pair) each, slice-major, writing partial[block][128].
template <bool VEC>
__global__ void __launch_bounds__(kImpThreads) importance_colsum_kernel(const uint16_t* __restrict__ attn, int H,
                                                                        int L, int hpw, int n_norm,
                                                                        const uint16_t* __restrict__ x, int d,
                                                                        bool xvec, float* __restrict__ norms,
                                                                        float* __restrict__ partial) {
  const int b = blockIdx.x;
  if (b < n_norm) {
    imp_norms(x, L, d, xvec, b, norms);
    return;
  }
  const int t = b - n_norm, pairs = imp_tiles(L) * (imp_tiles(L) + 1) / 2;
  imp_colsum_tile<VEC>(attn, H, L, hpw, t % pairs, t / pairs, partial + (size_t)t * kImpTile);
}

// One wave per key j (4 per workgroup): the key's partial sums over its query
// tiles and head slices (lane-strided, butterfly-reduced; fixed order, so
// deterministic), then I_j and its selection key.
__global__ void __launch_bounds__(kImpThreads) importance_finish_kernel(const float* __restrict__ partial, int H,
                                                                        int L, int hs,
                                                                        const float* __restrict__ norms,
                                                                        float* __restrict__ importance,
                                                                        uint64_t* __restrict__ keys) {
  const int lane = threadIdx.x & 63;
  const int j = blockIdx.x * (kImpThreads / 64) + wave_id();
  if (j >= L) return;
  const int nt = imp_tiles(L), tk = j / kImpTile, jj = j % kImpTile, cnt = nt - tk;
  const size_t pairs = (size_t)nt * (nt + 1) / 2;
  const float* pj = partial + imp_pair_base(tk, nt) * kImpTile + jj;
  float cs = 0.0f;
#pragma unroll 4
  for (int t = lane; t < hs * cnt; t += 64)   // (head slice, query tile)
    cs += pj[((size_t)(t / cnt) * pairs + t % cnt) * kImpTile];
  for (int off = 32; off >= 1; off >>= 1) cs += __shfl_xor(cs, off);
  if (lane == 0) {
    const float I = norms[j] * (cs / (float)H) / (float)(L - j);
    if (importance) importance[j] = I;
    // I >= 0: its bits order like the value; ~j puts lower indices first
    keys[j] = ((uint64_t)__float_as_uint(I) << 32) | (uint64_t)(0xffffffffu - (uint32_t)j);
  }
}

// Radix selection over L distinct keys, most significant byte first: each pass
// histograms the keys that share the prefix chosen so far, and wave 0 finds
// the bin holding the n-th largest (a scan over 4 bins per lane, descending).
// Once the chosen bin is taken whole, every key whose prefix is at least the
// chosen one is selected and the search stops (at the last byte it always is,
// keys being distinct).  Then mask_j = [key_j >> shift >= prefix >> shift].
// The first kSelCached keys per thread stay in registers across passes; in a
// wave, the lanes whose bin equals the first active lane's add with one atomic
// (early passes put most keys in one or two bins).
constexpr int kSelCached = 4;

__device__ __forceinline__ void imp_hist_add(int* hist, bool valid, int bin) {
  const uint64_t act = __ballot(valid);
  if (act == 0) return;
  const int first = __ffsll((unsigned long long)act) - 1;
  const int b0 = __shfl(bin, first);
  const uint64_t same = __ballot(valid && bin == b0);
  const int lane = threadIdx.x & 63;
  if (lane == first) atomicAdd(&hist[b0], __popcll(same));
  else if (valid && bin != b0) atomicAdd(&hist[bin], 1);
}

__global__ void __launch_bounds__(kImpSelectThreads) importance_select_kernel(const uint64_t* __restrict__ keys,
                                                                              int L, int n,
                                                                              uint8_t* __restrict__ mask) {
  __shared__ int hist[256];
  __shared__ uint64_t s_prefix;
  __shared__ int s_need, s_shift;
  if (n == 0) {
    for (int j = threadIdx.x; j < L; j += blockDim.x) mask[j] = 0;
    return;
  }
  uint64_t kc[kSelCached];
#pragma unroll
  for (int q = 0; q < kSelCached; ++q) {
    const int j = threadIdx.x + q * kImpSelectThreads;
    kc[q] = j < L ? keys[j] : 0ull;
  }
  if (threadIdx.x == 0) {
    s_prefix = 0;
    s_need = n;
    s_shift = 64;
  }
  for (int pass = 7; pass >= 0; --pass) {
    const int shift = 8 * pass;
    const uint64_t hi_mask = pass == 7 ? 0ull : (~0ull << (shift + 8));
    for (int b = threadIdx.x; b < 256; b += blockDim.x) hist[b] = 0;
    __syncthreads();
    const uint64_t prefix = s_prefix;
#pragma unroll
    for (int q = 0; q < kSelCached; ++q) {
      const int j = threadIdx.x + q * kImpSelectThreads;
      imp_hist_add(hist, j < L && (kc[q] & hi_mask) == prefix, (int)((kc[q] >> shift) & 0xff));
    }
    for (int j = threadIdx.x + kSelCached * kImpSelectThreads; j < L; j += kImpSelectThreads) {
      const uint64_t k = keys[j];
      if ((k & hi_mask) == prefix) atomicAdd(&hist[(k >> shift) & 0xff], 1);
    }
    __syncthreads();
    if (threadIdx.x < 64) {
      const int lane = threadIdx.x;
      int c[4], t = 0;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        c[q] = hist[255 - 4 * lane - q];
        t += c[q];
      }
      int inc = t;
      for (int off = 1; off < 64; off <<= 1) {
        const int v = __shfl_up(inc, off);
        if (lane >= off) inc += v;
      }
      const int before = inc - t, need = s_need;
      if (before < need && need <= inc) {   // exactly one lane
        int r = need - before, q = 0;
        while (q < 3 && r > c[q]) r -= c[q++];
        s_prefix = prefix | ((uint64_t)(255 - 4 * lane - q) << shift);
        s_need = r;
        if (r == c[q]) s_shift = shift;
      }
    }
    __syncthreads();
    if (s_shift == shift) break;
  }
  const int sh = s_shift;
  const uint64_t cut = s_prefix >> sh;
#pragma unroll
  for (int q = 0; q < kSelCached; ++q) {
    const int j = threadIdx.x + q * kImpSelectThreads;
    if (j < L) mask[j] = (kc[q] >> sh) >= cut ? 1 : 0;
  }
  for (int j = threadIdx.x + kSelCached * kImpSelectThreads; j < L; j += kImpSelectThreads)
    mask[j] = (keys[j] >> sh) >= cut ? 1 : 0;
}

hipError_t launch_importance(const uint16_t* attn, int H, int L, const uint16_t* x, int d, float rho,
                             float* importance, uint8_t* mask, void* ws, hipStream_t stream) {
  int hs, hpw;
  imp_head_split(H, L, hs, hpw);
  char* w = static_cast<char*>(ws);
  float* partial = reinterpret_cast<float*>(w);
  float* norms = reinterpret_cast<float*>(w + imp_partial_bytes(H, L));
  uint64_t* keys = reinterpret_cast<uint64_t*>(w + imp_partial_bytes(H, L) + imp_norm_bytes(L));
  const bool vec = (L % 8) == 0 && (reinterpret_cast<uintptr_t>(attn) % 16) == 0;
  const bool xvec = (d % 8) == 0 && (reinterpret_cast<uintptr_t>(x) % 16) == 0;
  const int n_norm = (L + kNormTokens - 1) / kNormTokens;
  const dim3 cgrid(n_norm + imp_pairs(L) * hs);
  timing_begin(stream, kSiteImpColsum);
  if (vec)
    hipLaunchKernelGGL((importance_colsum_kernel<true>), cgrid, dim3(kImpThreads), 0, stream, attn, H, L, hpw,
                       n_norm, x, d, xvec, norms, partial);
  else
    hipLaunchKernelGGL((importance_colsum_kernel<false>), cgrid, dim3(kImpThreads), 0, stream, attn, H, L, hpw,
                       n_norm, x, d, xvec, norms, partial);
  timing_end(stream, kSiteImpColsum);
  hipError_t err = hipGetLastError();
  if (err != hipSuccess) return err;
  timing_begin(stream, kSiteImpFinish);
  hipLaunchKernelGGL(importance_finish_kernel, dim3((L + kImpThreads / 64 - 1) / (kImpThreads / 64)),
                     dim3(kImpThreads), 0, stream, partial, H, L, hs, norms, importance, keys);
  timing_end(stream, kSiteImpFinish);
  timing_begin(stream, kSiteImpSelect);
  const int n = (int)floor((double)rho * L + 0.5);
  hipLaunchKernelGGL(importance_select_kernel, dim3(1), dim3(kImpSelectThreads), 0, stream, keys, L, n, mask);
  timing_end(stream, kSiteImpSelect);
  return hipGetLastError();
}

}  // namespace mc
