// pack.hip -- quantize + pack kernels and the dequant/code export kernels.
//
// Quantizer (paper Sec. 3.1: uniform asymmetric, group-wise, values mapped onto
// the integer grid 0..2^b-1; widths 1/2/3 from the PMQ allocation of Eq. 4).
// Per group of G inputs of one row, L = 2^b - 1:
//   s = fp16(fp32(max - min) / L) (1.0 if it rounds to zero), z = fp16(-min / s),
//   code = nearest level s*(j - z), ties to the even j, decided exactly in fp64.
// Sign binarization (appendix A.2, Eq. 7-9; 1-bit experts that ask for it):
// code = 1 where w >= 0, else 0, and every group of the matrix gets
// s = fp16(2 * ||W||_1 / (rows * cols)), z = 1/2, so that s*(code - z) =
// +-||W||_1 / (rows * cols) -- the binarized weight times its scale, in the same
// packed format (the kernels' product is then Eq. 10's add/subtract form).
#include "mc_internal.hpp"

namespace mc {

// ------------------------------------------------------------ scale / zero --
// One group per `lpg` consecutive lanes (lpg = min(64, G/4)); every lane
// reduces float4 pieces, then the group's lanes combine with butterflies.
__global__ void __launch_bounds__(256) pack_sz_kernel(const float* __restrict__ wg,
                                                      const float* __restrict__ wu,
                                                      const float* __restrict__ wd,
                                                      LayerArgs L, uint32_t* __restrict__ sz_out,
                                                      long long total_groups) {
  const int G = L.G;
  const int lpg = G / 4 < 64 ? G / 4 : 64;          // lanes per group (power of two)
  const int per_lane = G / 4 / lpg;                  // float4 pieces per lane
  const int lane = threadIdx.x & 63;
  const long long wave = ((long long)blockIdx.x * blockDim.x + threadIdx.x) >> 6;
  const long long grp = wave * (64 / lpg) + lane / lpg;
  const int sub = lane % lpg;
  const bool valid = grp < total_groups;
  const long long gpm = (long long)L.d * L.ffn / G;  // groups per matrix
  const long long gg = valid ? grp : 0;
  const int em = (int)(gg / gpm);
  const int e = em / 3, m = em % 3;
  const long long gi = gg % gpm;
  const int K = (m < 2) ? L.d : L.ffn;
  const int ng = K / G;
  const int row = (int)(gi / ng), g = (int)(gi % ng);
  const float* W = (m == 0) ? wg : (m == 1) ? wu : wd;
  const float* src = W + (size_t)e * L.d * L.ffn + (size_t)row * K + (size_t)g * G;

  float mn = __builtin_inff(), mx = -__builtin_inff();
  if (valid) {
    for (int p = 0; p < per_lane; ++p) {
      const float4 v = reinterpret_cast<const float4*>(src)[sub + p * lpg];
      mn = fminf(mn, fminf(fminf(v.x, v.y), fminf(v.z, v.w)));
      mx = fmaxf(mx, fmaxf(fmaxf(v.x, v.y), fmaxf(v.z, v.w)));
    }
  }
  for (int off = 1; off < lpg; off <<= 1) {
    mn = fminf(mn, __shfl_xor(mn, off));
    mx = fmaxf(mx, __shfl_xor(mx, off));
  }
  if (!valid || sub != 0) return;
  const int b = L.cum_bits[e + 1] - L.cum_bits[e];
  const size_t idx = layer_sz_offset(L, e, m) + ((size_t)(row / 16) * ng + g) * 16 + (row % 16);
  sz_out[idx] = group_sz_word(mn, mx, b);
}

// ------------------------------------------------------------------- codes --
// One thread per (matrix, tile, lane): 32 codes -> b words.

__global__ void __launch_bounds__(256) pack_codes_kernel(const float* __restrict__ wg,
                                                         const float* __restrict__ wu,
                                                         const float* __restrict__ wd,
                                                         LayerArgs L,
                                                         const uint32_t* __restrict__ sz,
                                                         uint32_t* __restrict__ words_out,
                                                         long long total_lanes) {
  const long long tid = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  if (tid >= total_lanes) return;
  const long long lpm = (long long)L.d * L.ffn / 32;   // lanes per matrix
  const int em = (int)(tid / lpm);
  const int e = em / 3, m = em % 3;
  const long long rest = tid % lpm;
  const int lane = (int)(rest & 63);
  const long long tile = rest >> 6;
  const int K = (m < 2) ? L.d : L.ffn;
  const int tiles_per_row = K / kTileCols;
  const int trow = (int)(tile / tiles_per_row), tcol = (int)(tile % tiles_per_row);
  const int n = trow * kTileRows + (lane & 15);
  const int kq = lane >> 4;
  const int G = L.G, ng = K / G;
  const int b = L.cum_bits[e + 1] - L.cum_bits[e];
  const int Lc = (1 << b) - 1;
  const bool sign = expert_is_sign(L, e);
  const float* W = (m == 0) ? wg : (m == 1) ? wu : wd;
  const float* row = W + (size_t)e * L.d * L.ffn + (size_t)n * K;
  const uint32_t* szm = sz + layer_sz_offset(L, e, m);

  uint32_t w[3] = {0u, 0u, 0u};
  for (int u = 0; u < 4; ++u) {
    const int k0 = tcol * kTileCols + 32 * u + 8 * kq;
    const int g = k0 / G;
    const uint32_t szw = szm[((size_t)(n / 16) * ng + g) * 16 + (n % 16)];
    const double s = (double)half_bits_to_float(szw & 0xffffu);
    const double z = (double)half_bits_to_float(szw >> 16);
    const float4 a = reinterpret_cast<const float4*>(row + k0)[0];
    const float4 c = reinterpret_cast<const float4*>(row + k0)[1];
    const float v[8] = {a.x, a.y, a.z, a.w, c.x, c.y, c.z, c.w};
    for (int j = 0; j < 8; ++j) {
      const uint32_t code = sign ? (v[j] >= 0.0f ? 1u : 0u) : (uint32_t)nearest_code(v[j], s, z, Lc);
      place_code(w, code, 4 * u + (j >> 1), j & 1, b);
    }
  }
  uint32_t* dst = words_out + layer_word_offset(L, e, m) + ((size_t)tile * 64 + lane) * b;
  for (int p = 0; p < b; ++p) dst[p] = w[p];
}

// ------------------------------------------------------- sign binarization --
// ||W||_1 of every sign-binarized matrix: kSignParts partial sums in fp64 per
// matrix (each over a contiguous slice, fixed order inside the block), kept
// in the matrix's own scale/zero words (overwritten by the finish kernel).
constexpr int kSignThreads = 256;

__host__ __device__ inline int sign_parts(long long groups_per_matrix) {
  // partials (8 bytes = 2 words each) fit in the matrix's scale/zero words
  const long long cap = groups_per_matrix / 2;
  return (int)(cap < 1 ? 1 : (cap < 1024 ? cap : 1024));
}

__device__ __forceinline__ double block_sum_f64(double v, double* red) {
  for (int off = 1; off < 64; off <<= 1) v += __shfl_xor(v, off);
  __syncthreads();
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = v;
  __syncthreads();
  double t = 0.0;
  for (int w = 0; w < kSignThreads / 64; ++w) t += red[w];
  return t;
}

// grid (parts, 3E matrices); matrices of other experts exit at once.
__global__ void __launch_bounds__(kSignThreads) sign_l1_kernel(const float* __restrict__ wg,
                                                               const float* __restrict__ wu,
                                                               const float* __restrict__ wd, LayerArgs L,
                                                               uint32_t* __restrict__ sz) {
  __shared__ double red[kSignThreads / 64];
  const int e = blockIdx.y / 3, m = blockIdx.y % 3;
  if (!expert_is_sign(L, e)) return;
  const long long n4 = (long long)L.d * L.ffn / 4;                    // float4 pieces
  const long long gpm = (long long)L.d * L.ffn / L.G;
  const int parts = sign_parts(gpm);
  const int part = blockIdx.x;
  if (part >= parts) return;
  const long long per = (n4 + parts - 1) / parts;
  const long long b0 = part * per, b1 = (b0 + per) < n4 ? (b0 + per) : n4;
  const float* W = ((m == 0) ? wg : (m == 1) ? wu : wd) + (size_t)e * L.d * L.ffn;
  double acc = 0.0;
  for (long long i = b0 + threadIdx.x; i < b1; i += kSignThreads) {
    const float4 v = reinterpret_cast<const float4*>(W)[i];
    acc += (double)fabsf(v.x) + (double)fabsf(v.y) + (double)fabsf(v.z) + (double)fabsf(v.w);
  }
  const double t = block_sum_f64(acc, red);
  if (threadIdx.x == 0) {             // two 32-bit words (the buffer is only 4-byte aligned)
    const unsigned long long b = __double_as_longlong(t);
    uint32_t* dst = sz + layer_sz_offset(L, e, m) + 2 * (size_t)part;
    dst[0] = (uint32_t)b;
    dst[1] = (uint32_t)(b >> 32);
  }
}

// One workgroup per matrix of a binarized expert: adds the partials in order,
// then writes the scale/zero word of every group.
__global__ void __launch_bounds__(kSignThreads) sign_finish_kernel(LayerArgs L, uint32_t* __restrict__ sz) {
  __shared__ double red[kSignThreads / 64];
  const int e = blockIdx.x / 3, m = blockIdx.x % 3;
  if (!expert_is_sign(L, e)) return;
  const long long gpm = (long long)L.d * L.ffn / L.G;
  const int parts = sign_parts(gpm);
  uint32_t* dst = sz + layer_sz_offset(L, e, m);
  double acc = 0.0;
  const int per = (parts + kSignThreads - 1) / kSignThreads;
  for (int i = threadIdx.x * per; i < (threadIdx.x + 1) * per && i < parts; ++i)
    acc += __longlong_as_double((long long)(((unsigned long long)dst[2 * i + 1] << 32) | dst[2 * i]));
  const double l1 = block_sum_f64(acc, red);             // every partial read before any write
  double s2 = 2.0 * (l1 / ((double)L.d * (double)L.ffn));
  if (s2 > 65504.0) s2 = 65504.0;
  const uint32_t word = (uint32_t)double_to_half_rne(s2) | (0x3800u << 16);   // z = 1/2
  __syncthreads();
  for (long long i = threadIdx.x; i < gpm; i += kSignThreads) dst[i] = word;
}

// ------------------------------------------------------------------ export --
// One thread per tile lane of one matrix: writes its 32 values.
template <int BITS, bool DEQUANT>
__global__ void __launch_bounds__(256) export_kernel(const uint32_t* __restrict__ words,
                                                    const uint32_t* __restrict__ sz, int R, int K,
                                                    int G, void* __restrict__ out) {
  const long long tid = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  const long long lanes = (long long)R * K / 32;
  if (tid >= lanes) return;
  const int lane = (int)(tid & 63);
  const long long tile = tid >> 6;
  const int tiles_per_row = K / kTileCols;
  const int trow = (int)(tile / tiles_per_row), tcol = (int)(tile % tiles_per_row);
  const int n = trow * kTileRows + (lane & 15);
  const int kq = lane >> 4;
  const int ng = K / G;
  uint32_t w[3] = {0u, 0u, 0u};
  const uint32_t* src = words + ((size_t)tile * 64 + lane) * BITS;
  for (int p = 0; p < BITS; ++p) w[p] = src[p];
  for (int u = 0; u < 4; ++u) {
    const int k0 = tcol * kTileCols + 32 * u + 8 * kq;
    const uint32_t szw = sz[((size_t)(n / 16) * ng + k0 / G) * 16 + (n % 16)];
    const double s = (double)half_bits_to_float(szw & 0xffffu);
    const double z = (double)half_bits_to_float(szw >> 16);
    for (int j = 0; j < 8; ++j) {
      const int code = extract_code<BITS>(w, 4 * u + (j >> 1), j & 1);
      const size_t o = (size_t)n * K + k0 + j;
      if constexpr (DEQUANT) {
        // s*(q - z): q - z needs <= 41 bits, the product <= 52: exact in fp64.
        static_cast<uint16_t*>(out)[o] = double_to_half_rne(s * ((double)code - z));
      } else {
        static_cast<uint8_t*>(out)[o] = (uint8_t)code;
      }
    }
  }
}

// ---------------------------------------------------------------- launchers --

hipError_t launch_pack(const float* wg, const float* wu, const float* wd, const LayerArgs& L,
                       uint32_t* words, uint32_t* sz, bool any_sign, hipStream_t stream) {
  const long long groups = 3LL * L.E * L.d * L.ffn / L.G;
  const int lpg = L.G / 4 < 64 ? L.G / 4 : 64;
  const long long waves = (groups + (64 / lpg) - 1) / (64 / lpg);
  const long long blocks_sz = (waves * 64 + 255) / 256;
  timing_begin(stream, kSitePackSz);
  hipLaunchKernelGGL(pack_sz_kernel, dim3((unsigned)blocks_sz), dim3(256), 0, stream, wg, wu, wd,
                     L, sz, groups);
  if (any_sign) {
    const int parts = sign_parts((long long)L.d * L.ffn / L.G);
    hipLaunchKernelGGL(sign_l1_kernel, dim3(parts, 3 * L.E), dim3(kSignThreads), 0, stream, wg, wu, wd, L, sz);
    hipLaunchKernelGGL(sign_finish_kernel, dim3(3 * L.E), dim3(kSignThreads), 0, stream, L, sz);
  }
  timing_end(stream, kSitePackSz);
  hipError_t err = hipGetLastError();
  if (err != hipSuccess) return err;
  const long long lanes = 3LL * L.E * L.d * L.ffn / 32;
  timing_begin(stream, kSitePackCodes);
  hipLaunchKernelGGL(pack_codes_kernel, dim3((unsigned)((lanes + 255) / 256)), dim3(256), 0, stream,
                     wg, wu, wd, L, sz, words, lanes);
  timing_end(stream, kSitePackCodes);
  return hipGetLastError();
}

hipError_t launch_export(const uint32_t* words, const uint32_t* sz, int bits, int R, int K, int G,
                         bool dequant, void* out, hipStream_t stream) {
  const long long lanes = (long long)R * K / 32;
  const dim3 grid((unsigned)((lanes + 255) / 256)), block(256);
#define MC_EXPORT_CASE(B)                                                                     \
  if (bits == B) {                                                                            \
    if (dequant)                                                                              \
      hipLaunchKernelGGL((export_kernel<B, true>), grid, block, 0, stream, words, sz, R, K, G, \
                         out);                                                                \
    else                                                                                      \
      hipLaunchKernelGGL((export_kernel<B, false>), grid, block, 0, stream, words, sz, R, K,  \
                         G, out);                                                             \
  }
  timing_begin(stream, kSiteExport);
  MC_EXPORT_CASE(1)
  MC_EXPORT_CASE(2)
  MC_EXPORT_CASE(3)
  timing_end(stream, kSiteExport);
#undef MC_EXPORT_CASE
  return hipGetLastError();
}

}  // namespace mc
