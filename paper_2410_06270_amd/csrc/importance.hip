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
//     triangle (query tile >= key tile), all heads: per-key partial sums;
//   importance_finish_kernel  one workgroup per key tile: partials added in
//     query-tile order, l1 norms, I_j, and the selection key
//     (I_j bits << 32 | ~j: larger key = larger I_j, then lower j);
//   importance_select_kernel  one workgroup: radix selection of the n-th
//     largest key (8 passes of 8 bits), then the mask.
// The attention map is read once, in 256-byte row pieces per wave (HBM-bound).
#include "mc_internal.hpp"

namespace mc {

constexpr int kImpTile = 128;
constexpr int kImpThreads = 256;
constexpr int kImpSelectThreads = 1024;

__host__ __device__ static inline int imp_tiles(int L) { return (L + kImpTile - 1) / kImpTile; }

size_t importance_workspace_bytes(int H, int L) {
  (void)H;
  const size_t nt = (size_t)imp_tiles(L);
  const size_t pairs = nt * (nt + 1) / 2;
  return ((pairs * kImpTile * sizeof(float) + 255) / 256) * 256 + (size_t)L * sizeof(uint64_t);
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

// Thread (column group cg of 8 keys, row phase r of 16): rows i = r, r+16, ...
// of the query tile, keys 8cg..8cg+7 of the key tile; VEC = 16-byte loads
// (L a multiple of 8).
template <bool VEC>
__global__ void __launch_bounds__(kImpThreads) importance_colsum_kernel(const uint16_t* __restrict__ attn, int H,
                                                                        int L, float* __restrict__ partial) {
  __shared__ float red[16][kImpTile + 4];
  const int nt = imp_tiles(L);
  int tq, tk;
  imp_pair(blockIdx.x, nt, tq, tk);
  const int cg = threadIdx.x & 15, r = threadIdx.x >> 4;
  const int j0 = tk * kImpTile + 8 * cg;
  float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
  for (int h = 0; h < H; ++h) {
    const uint16_t* ah = attn + (size_t)h * L * L;
    for (int ii = r; ii < kImpTile; ii += 16) {
      const int i = tq * kImpTile + ii;
      if (i >= L) break;
      const uint16_t* row = ah + (size_t)i * L + j0;
      if (VEC && j0 + 7 < L && j0 + 7 <= i) {
        const u32x4 v = *reinterpret_cast<const u32x4*>(row);
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          acc[2 * q] += bf16_bits_to_float(v[q] & 0xffffu);
          acc[2 * q + 1] += bf16_bits_to_float(v[q] >> 16);
        }
      } else {
#pragma unroll
        for (int c = 0; c < 8; ++c)
          if (j0 + c < L && j0 + c <= i) acc[c] += bf16_bits_to_float(row[c]);
      }
    }
  }
#pragma unroll
  for (int c = 0; c < 8; ++c) red[r][8 * cg + c] = acc[c];
  __syncthreads();
  if (threadIdx.x < kImpTile) {
    float s = 0.0f;
    for (int q = 0; q < 16; ++q) s += red[q][threadIdx.x];   // row phases in order
    partial[(size_t)blockIdx.x * kImpTile + threadIdx.x] = s;
  }
}

// One workgroup per key tile: 4 waves x 32 keys.
__global__ void __launch_bounds__(kImpThreads) importance_finish_kernel(const float* __restrict__ partial, int H,
                                                                        int L, const uint16_t* __restrict__ x,
                                                                        int d, float* __restrict__ importance,
                                                                        uint64_t* __restrict__ keys) {
  __shared__ float colsum[kImpTile];
  const int nt = imp_tiles(L), tk = blockIdx.x;
  const size_t base = imp_pair_base(tk, nt);
  if (threadIdx.x < kImpTile) {
    float s = 0.0f;
    for (int tq = tk; tq < nt; ++tq) s += partial[(base + (tq - tk)) * kImpTile + threadIdx.x];
    colsum[threadIdx.x] = s;
  }
  __syncthreads();
  const int lane = threadIdx.x & 63, wave = wave_id();
  for (int jj = wave; jj < kImpTile; jj += kImpThreads / 64) {
    const int j = tk * kImpTile + jj;
    if (j >= L) break;
    float n1 = 0.0f;
    for (int c = lane; c < d; c += 64) n1 += fabsf(bf16_bits_to_float(x[(size_t)j * d + c]));
    for (int off = 32; off >= 1; off >>= 1) n1 += __shfl_xor(n1, off);
    if (lane == 0) {
      const float I = n1 * (colsum[jj] / (float)H) / (float)(L - j);
      if (importance) importance[j] = I;
      // I >= 0: its bits order like the value; ~j puts lower indices first
      keys[j] = ((uint64_t)__float_as_uint(I) << 32) | (uint64_t)(0xffffffffu - (uint32_t)j);
    }
  }
}

// Radix selection of the n-th largest of L distinct keys, then the mask.
__global__ void __launch_bounds__(kImpSelectThreads) importance_select_kernel(const uint64_t* __restrict__ keys,
                                                                              int L, int n,
                                                                              uint8_t* __restrict__ mask) {
  __shared__ int hist[256];
  __shared__ uint64_t s_prefix;
  __shared__ int s_need;
  if (n == 0) {
    for (int j = threadIdx.x; j < L; j += blockDim.x) mask[j] = 0;
    return;
  }
  if (threadIdx.x == 0) {
    s_prefix = 0;
    s_need = n;
  }
  __syncthreads();
  for (int pass = 7; pass >= 0; --pass) {
    const int shift = 8 * pass;
    const uint64_t hi_mask = pass == 7 ? 0ull : (~0ull << (shift + 8));
    for (int b = threadIdx.x; b < 256; b += blockDim.x) hist[b] = 0;
    __syncthreads();
    const uint64_t prefix = s_prefix;
    for (int j = threadIdx.x; j < L; j += blockDim.x) {
      const uint64_t k = keys[j];
      if ((k & hi_mask) == prefix) atomicAdd(&hist[(k >> shift) & 0xff], 1);
    }
    __syncthreads();
    if (threadIdx.x == 0) {
      int need = s_need, b = 255;
      for (; b > 0; --b) {            // largest bin first
        if (hist[b] >= need) break;
        need -= hist[b];
      }
      s_prefix = prefix | ((uint64_t)b << shift);
      s_need = need;
    }
    __syncthreads();
  }
  const uint64_t kth = s_prefix;       // the n-th largest key (keys are distinct)
  for (int j = threadIdx.x; j < L; j += blockDim.x) mask[j] = keys[j] >= kth ? 1 : 0;
}

hipError_t launch_importance(const uint16_t* attn, int H, int L, const uint16_t* x, int d, float rho,
                             float* importance, uint8_t* mask, void* ws, hipStream_t stream) {
  const int nt = imp_tiles(L);
  const int pairs = nt * (nt + 1) / 2;
  float* partial = static_cast<float*>(ws);
  uint64_t* keys = reinterpret_cast<uint64_t*>(static_cast<char*>(ws) +
                                               (((size_t)pairs * kImpTile * sizeof(float) + 255) / 256) * 256);
  const bool vec = (L % 8) == 0 && (reinterpret_cast<uintptr_t>(attn) % 16) == 0;
  timing_begin(stream, kSiteImpColsum);
  if (vec)
    hipLaunchKernelGGL((importance_colsum_kernel<true>), dim3(pairs), dim3(kImpThreads), 0, stream, attn, H, L,
                       partial);
  else
    hipLaunchKernelGGL((importance_colsum_kernel<false>), dim3(pairs), dim3(kImpThreads), 0, stream, attn, H, L,
                       partial);
  timing_end(stream, kSiteImpColsum);
  hipError_t err = hipGetLastError();
  if (err != hipSuccess) return err;
  timing_begin(stream, kSiteImpSelect);
  hipLaunchKernelGGL(importance_finish_kernel, dim3(nt), dim3(kImpThreads), 0, stream, partial, H, L, x, d,
                     importance, keys);
  const int n = (int)floor((double)rho * L + 0.5);
  hipLaunchKernelGGL(importance_select_kernel, dim3(1), dim3(kImpSelectThreads), 0, stream, keys, L, n, mask);
  timing_end(stream, kSiteImpSelect);
  return hipGetLastError();
}

}  // namespace mc
