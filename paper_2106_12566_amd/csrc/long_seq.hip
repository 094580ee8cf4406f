// Sequences longer than one transform block (n > 2^kMaxLog2N, attention
// only).  The Toeplitz matrix C of Eqs. (12)-(13) is taken in blocks of
// nbk = 2^kMaxLog2N positions: block (I, J) maps the keys of block J to the
// queries of block I and is itself Toeplitz, with entries c_{j - i + (J - I) nbk},
// i.e. the bias window b[(J - I) nbk - (nbk - 1) .. (J - I) nbk + (nbk - 1)].  The
// numerators and denominator of Eq. (10) of query block I are the sums over J
// of the blockwise products, all J in one run of the convolution kernel (one
// partial result per J, summed by the combine kernel).  These are the helpers
// around those runs: block copies of phi, the bias windows, the certification
// weights summed over J, and the scattering of the block results.  In a translation unit of their own so
// that the convolution kernel's code generation does not change with them.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>

#include "common.hpp"
#include "launch.hpp"

namespace krpe {

// dst[bh][r][i] = src[bh][r][K nbk + i] for r < R, i < nbk (rows of length Ntot).
__global__ void k_block_rows(const float* __restrict__ src, float* __restrict__ dst, int R, int nbk, int Ntot,
                             int K, long long total) {
  const long long e = static_cast<long long>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (e >= total) return;
  const long long i = e % nbk, row = e / nbk;  // row = bh * R + r
  dst[e] = src[row * Ntot + static_cast<long long>(K) * nbk + i];
}

// Bias windows of query block I against every key block J < nb:
// out[J][h][s] = b_t with t = s - (nbk - 1) + (J - I) nbk for s < 2 nbk - 1,
// -inf where t is outside (-n, n) (such offsets pair no real query with a
// real key).
__global__ void k_bias_window(const float* __restrict__ b, float* __restrict__ out, int H, int n, int nbk, int I,
                              long long total) {
  const long long e = static_cast<long long>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (e >= total) return;
  const long long len = 2LL * nbk - 1, w = e / len, s = e - w * len;
  const long long J = w / H, h = w % H;
  const long long t = s - (nbk - 1) + (J - I) * nbk;
  out[e] = (t > -n && t < n) ? b[h * (2LL * n - 1) + t + n - 1] : -INFINITY;
}

// Certification weights of query block I summed over the key blocks J: the
// FFT error of block (I, J) scales with ||h_IJ||_2 (hnorm[J H + h].y) times
// the channel norms of key block J (wbJ[J]), so
// wbI[bh][l] = sum_J ||h_IJ|| wbJ[J][bh][l] for l < M, and wbI[bh][M] (the
// largest column scale) is the maximum over J.
__global__ void k_wb_accum(float2* __restrict__ wbI, const float2* __restrict__ wbJ, const float2* __restrict__ hnorm,
                           int BH, int H, int M, int nb) {
  const long long e = static_cast<long long>(blockIdx.x) * blockDim.x + threadIdx.x;
  const long long per = static_cast<long long>(BH) * (M + 1);
  if (e >= per) return;
  const int bh = static_cast<int>(e / (M + 1)), l = static_cast<int>(e % (M + 1));
  float2 acc = make_float2(0.f, 0.f);
  for (int J = 0; J < nb; ++J) {
    const float2 w = wbJ[J * per + e];
    if (l < M) {
      const float hn = hnorm[J * H + bh % H].y;
      acc = make_float2(fmaf(w.x, hn, acc.x), fmaf(w.y, hn, acc.y));
    } else {
      acc.x = fmaxf(acc.x, w.x);
    }
  }
  wbI[e] = acc;
}

// full[bh][K nbk / 64 + t] = blk[bh][t], t < tiles_b: the queued rows of block K
// in the whole sequence's row masks.
__global__ void k_merge_mask(const unsigned long long* __restrict__ blk, unsigned long long* __restrict__ full,
                             int BH, int tiles_b, int tiles_full, int K, int nbk) {
  const long long e = static_cast<long long>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (e >= static_cast<long long>(BH) * tiles_b) return;
  const int bh = static_cast<int>(e / tiles_b), t = static_cast<int>(e % tiles_b);
  full[static_cast<size_t>(bh) * tiles_full + static_cast<size_t>(K) * (nbk / 64) + t] = blk[e];
}

// z[bh][K nbk + i][c] = zb[bh][i][c] for i < lenK.
__global__ void k_scatter_rows(const float* __restrict__ zb, float* __restrict__ z, int n, int nbk, int d, int K,
                               int lenK, long long total) {
  const long long e = static_cast<long long>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (e >= total) return;
  const long long c = e % d, i = (e / d) % lenK, bh = e / (static_cast<long long>(d) * lenK);
  z[(bh * n + static_cast<long long>(K) * nbk + i) * d + c] = zb[e];
}

// ones[h] = (1, 1): a unit "spectrum norm" for the combine kernel, whose
// weights then already carry the per-block norms.
__global__ void k_unit_hnorm(float2* __restrict__ hn, int H) {
  const int e = blockIdx.x * blockDim.x + threadIdx.x;
  if (e < H) hn[e] = make_float2(1.f, 1.f);
}

namespace {
unsigned grid_of(long long total) { return static_cast<unsigned>((total + 255) / 256); }
}  // namespace

hipError_t launch_block_rows(const float* src, float* dst, int BH, int R, int nbk, int Ntot, int K, hipStream_t st) {
  const long long total = static_cast<long long>(BH) * R * nbk;
  hipLaunchKernelGGL(k_block_rows, dim3(grid_of(total)), dim3(256), 0, st, src, dst, R, nbk, Ntot, K, total);
  return hipGetLastError();
}

hipError_t launch_bias_window(const float* b, float* out, int H, int n, int nbk, int nb, int I, hipStream_t st) {
  const long long total = static_cast<long long>(nb) * H * (2LL * nbk - 1);
  hipLaunchKernelGGL(k_bias_window, dim3(grid_of(total)), dim3(256), 0, st, b, out, H, n, nbk, I, total);
  return hipGetLastError();
}

hipError_t launch_wb_accum(float2* wbI, const float2* wbJ, const float2* hnorm, int BH, int H, int M, int nb,
                           hipStream_t st) {
  const long long total = static_cast<long long>(BH) * (M + 1);
  hipLaunchKernelGGL(k_wb_accum, dim3(grid_of(total)), dim3(256), 0, st, wbI, wbJ, hnorm, BH, H, M, nb);
  return hipGetLastError();
}

hipError_t launch_merge_mask(const unsigned long long* blk, unsigned long long* full, int BH, int tiles_b,
                             int tiles_full, int K, int nbk, hipStream_t st) {
  const long long total = static_cast<long long>(BH) * tiles_b;
  hipLaunchKernelGGL(k_merge_mask, dim3(grid_of(total)), dim3(256), 0, st, blk, full, BH, tiles_b, tiles_full, K,
                     nbk);
  return hipGetLastError();
}

hipError_t launch_scatter_rows(const float* zb, float* z, int BH, int n, int nbk, int d, int K, int lenK,
                               hipStream_t st) {
  const long long total = static_cast<long long>(BH) * lenK * d;
  hipLaunchKernelGGL(k_scatter_rows, dim3(grid_of(total)), dim3(256), 0, st, zb, z, n, nbk, d, K, lenK, total);
  return hipGetLastError();
}

hipError_t launch_unit_hnorm(float2* hn, int H, hipStream_t st) {
  hipLaunchKernelGGL(k_unit_hnorm, dim3(grid_of(H)), dim3(256), 0, st, hn, H);
  return hipGetLastError();
}

}  // namespace krpe
