// HIP kernels (gfx950) of the forward pass of kernelized attention with RPE.
//
//   z_i = phi(q_i) sum_j c_{j-i} phi(k_j)^T v_j / phi(q_i) sum_j c_{j-i} phi(k_j)^T
//                                                           (Section 3.2, Eq. (10))
//
// following the steps of Algorithm 1 (c = exp(b); A1 = phi(K)^T V and
// A2 = phi(K)^T; the two Toeplitz products; the final ratio):
//
//  k_twiddles        W_{2N}^k = exp(-i pi k / N), k < 2N, computed in fp64.
//  k_spectrum        spectrum of the circulant embedding of c (length 2N),
//                    split into its even and odd bins, pre-scaled by 1/(2N).
//  k_feature_map     phi(q), phi(k) by Eq. (5): an fp32 MFMA contraction over
//                    the head dimension with exp(. - ||x||^2/2)/sqrt(m) fused
//                    into the epilogue.
//  k_conv_contract   the hot loop: channel formation (A1, A2 of Eq. (11)), the
//                    FFT product with C (Eqs. (12)-(13)) and the contraction
//                    with phi(q), all in registers/LDS of one work-group.
//  k_combine         the ratio of Eq. (10), plus a per-row rounding-error bound.
//  k_fixup           exact evaluation of Eq. (10) for rows the bound rejects.
//
// The Toeplitz product alone (krpe_toeplitz_conv) runs k_conv_contract with
// phi(q) = phi(k) = a row of ones and the channels as the value columns.
//
// The Toeplitz product of a length-n signal a is the first n outputs of the
// circular convolution of length L = 2N (N = next power of two >= n) of the
// zero-padded a with the kernel h, where h[s] = c_{-s} for 0 <= s < n,
// h[L - s] = c_s for 0 < s < n and 0 elsewhere.  With w = exp(-i pi / N), the
// even and odd bins of the length-2N transform are the length-N transforms of
// a and of a_j w^j, so
//
//   y_i = 1/(2N) [ IDFT_N(He * DFT_N(a))_i + w^{-i} IDFT_N(Ho * DFT_N(a w^j))_i ]
//
// with He = DFT_N(h[s] + h[s+N]) and Ho = DFT_N((h[s] - h[s+N]) w^s).  Each
// half is an independent length-N problem, so a work-group only ever holds N
// complex values (128 KiB of LDS at n = 16384); the two halves run in separate
// work-groups whose results are summed by k_combine.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>
#include <type_traits>

#include "common.hpp"
#include "conv.hpp"
#include "launch.hpp"

namespace krpe {

// ------------------------------------------------------------ twiddles --
__global__ void k_twiddles(float2* __restrict__ tw, int log2n) {
  const int N = 1 << log2n;
  const int k = blockIdx.x * blockDim.x + threadIdx.x;
  if (k < 2 * N) {
    double s, c;
    sincospi(-static_cast<double>(k) / static_cast<double>(N), &s, &c);
    tw[k] = make_float2(static_cast<float>(c), static_cast<float>(s));
  }
}

// Entries past W_{2N} of the extended twiddle table of Conf<L2> (C::TWC):
//   [M, 2M):        per-thread first-pass twiddles of the convolution units,
//                   entry M + (r R + i) T + tau = W_{2N}^{tau (r + S i)}
//   [2M, TABLE):    W_{L_p}^k, k < L_p, for the passes p >= 1 (Fft::twc_offset)
// with M = 2N, computed in double and rounded.
template <int L2>
__global__ void k_twiddles_ext(float2* __restrict__ tw) {
  using C = Conf<L2>;
  using F = typename C::F;
  constexpr int M = F::M_TAB;
  const int e = M + blockIdx.x * blockDim.x + threadIdx.x;
  if (e >= F::TABLE) return;
  long long num;
  long long den;
  if (e < 2 * M) {
    const int q = e - M, tau = q % F::T, i = (q / F::T) % F::R, r = q / (F::T * F::R);
    num = (static_cast<long long>(tau) * (r + C::S * i)) % M;
    den = M;
  } else {
    int p = 1;
    while (p + 1 < F::P && e >= F::twc_offset(p + 1)) ++p;
    num = e - F::twc_offset(p);
    den = F::N >> (F::LR * p);
  }
  double sn, cs;
  sincospi(-2.0 * static_cast<double>(num) / static_cast<double>(den), &sn, &cs);
  tw[e] = make_float2(static_cast<float>(cs), static_cast<float>(sn));
}

// ------------------------------------------------------------ spectrum --
// c_{-s} embedded circularly in length 2N (see the header comment).
__device__ __forceinline__ float circ_kernel(const float* __restrict__ bh, int s, int n, int N) {
  if (s < n) return expf(bh[n - 1 - s]);
  if (s > 2 * N - n) return expf(bh[2 * N - s + n - 1]);
  return 0.f;
}

// One transform per (head, residue class r < S): the bins k = S k' + r of the
// length-2N transform of h are DFT_{LT}(g_r) with
//   g_r[j] = W_{2N}^{r j} sum_{p < S} h[j + p LT] W_S^{p r},   j < LT = 2N / S.
// Hs[h][r][.] holds them, scaled by 1/(2N), in register order (below).  Also,
// when requested: hnorm[h] = (||h||_1, ||h||_2).
template <int L2>
__global__ __launch_bounds__(Conf<L2>::THREADS) void k_spectrum(const float* __restrict__ b,
                                                                 const float2* __restrict__ tw,
                                                                 float2* __restrict__ Hs,
                                                                 float2* __restrict__ hnorm, int H, int n) {
  using C = Conf<L2>;
  using F = typename C::F;
  constexpr int S = C::S;
  __shared__ float2 lds[C::LDS_SLOTS];
  __shared__ float red[C::WAVES];
  // With one unit per work-group the unit index is wave-uniform: say so, so
  // that per-unit pointers live in scalar registers.
  const int g = C::G == 1 ? 0 : threadIdx.x / F::T, tau = C::G == 1 ? threadIdx.x : threadIdx.x % F::T;
  const int units = S * H;
  int unit = blockIdx.x * C::G + g;
  const bool active = unit < units;
  if (!active) unit = units - 1;
  const int h = unit / S, r = unit % S;
  const float* bh = b + static_cast<size_t>(h) * (2 * n - 1);
  float2 x[F::R];
  float s1 = 0.f, s2 = 0.f;
#pragma unroll
  for (int i = 0; i < F::R; ++i) {
    const int j = tau + F::T * i;
    float2 acc = make_float2(0.f, 0.f);
#pragma unroll
    for (int p = 0; p < S; ++p) {
      const float hv = circ_kernel(bh, j + p * F::N, n, C::N);
      s1 += hv;
      s2 = fmaf(hv, hv, s2);
      acc = cadd(acc, rot_dyn<S, false>(make_float2(hv, 0.f), p * r));
    }
    x[i] = r == 0 ? acc : cmul(acc, tw[r * j]);
  }
  if (hnorm) {
    s1 = unit_reduce<F::T>(s1, red, OpAdd());
    s2 = unit_reduce<F::T>(s2, red, OpAdd());
    if (active && r == 0 && tau == 0) hnorm[h] = make_float2(s1, sqrtf(s2));
  }
  F::forward(x, lds + g * (F::P > 1 ? F::LDS : 0), tw, tau);
  if (active) {
    // Stored in the order the forward transform leaves the bins in registers:
    // element i * T + tau is register i of thread tau (frequency
    // F::frequency_of(F::spectrum_pos(tau, i))).
    const float scale = 1.0f / static_cast<float>(2 * C::N);
    float2* out = Hs + static_cast<size_t>(unit) * F::N;
#pragma unroll
    for (int i = 0; i < F::R; ++i) out[i * F::T + tau] = make_float2(x[i].x * scale, x[i].y * scale);
  }
}

// --------------------------------------------------------- feature map --
typedef float floatx16 __attribute__((ext_vector_type(16)));

// Feature maps of the projections s = x W^T (Sec. 2): PRF, Eq. (5),
// phi_l = exp(s_l - ||x||^2/2) / sqrt(m) (m features); TRF, the trigonometric
// map, phi_l = exp(||x||^2/2) sin(s_l) / sqrt(m) and phi_{m+l} = exp(||x||^2/2)
// cos(s_l) / sqrt(m) (2m signed features).  Up to two sources (q and k) in
// one launch.  Tile: 64 positions x 64 projections per work-group, four waves
// of 32 x 32 v_mfma_f32_32x32x2f32 tiles; K (= d) staged through LDS in chunks
// of 32.  FEATURE_MAJOR writes phi[bh][l][i] for i < ld (zeros for
// n <= i < ld; lanes run along positions), otherwise phi[bh][i][l] (lanes run
// along features): stores stay coalesced either way because the operand
// roles are swapped.  M = m (PRF) or 2m (TRF) is the row length of phi.
template <typename TX, bool FEATURE_MAJOR>
__global__ __launch_bounds__(256) void k_feature_map(const TX* __restrict__ x0, const TX* __restrict__ x1,
                                                     const float* __restrict__ W, float* __restrict__ phi0,
                                                     float* __restrict__ phi1, int H, int n, int ld, int d,
                                                     int m, float inv_sqrt_m, int tiles_n, int tiles_m,
                                                     int BH, unsigned* __restrict__ fix_counts, int nprf,
                                                     int trf) {
  // Clear the exact-evaluation queue counters (fix_counts[0..BH]) for k_combine.
  if (fix_counts && threadIdx.x == 0 && blockIdx.x <= static_cast<unsigned>(BH)) fix_counts[blockIdx.x] = 0u;
  __shared__ float xs[64][33];
  __shared__ float wsm[64][33];
  __shared__ float half_sq[64];
  __shared__ float row_scale[64];
  __shared__ float trf_amp[64];
  int bid = blockIdx.x;
  const int tn = bid % tiles_n;
  bid /= tiles_n;
  const int tm = bid % tiles_m;
  bid /= tiles_m;
  const int bh = bid % BH;
  const int src = bid / BH;
  const TX* __restrict__ x = src == 0 ? x0 : x1;
  float* __restrict__ phi = src == 0 ? phi0 : phi1;
  const int h = bh % H;
  const int i0 = tn * 64, l0 = tm * 64;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wi = (wave & 1) * 32, wl = (wave >> 1) * 32;
  const TX* __restrict__ xb = x + static_cast<size_t>(bh) * n * d;
  const float* __restrict__ Wh = W + static_cast<size_t>(h) * m * d;

  floatx16 acc;
#pragma unroll
  for (int v = 0; v < 16; ++v) acc[v] = 0.f;
  float sq = 0.f;
  for (int k0 = 0; k0 < d; k0 += 32) {
    for (int e = threadIdx.x; e < 64 * 32; e += 256) {
      const int r = e >> 5, c = e & 31;
      const int i = i0 + r, l = l0 + r, k = k0 + c;
      xs[r][c] = (i < n && k < d) ? to_f32(xb[static_cast<size_t>(i) * d + k]) : 0.f;
      wsm[r][c] = (l < m && k < d) ? Wh[static_cast<size_t>(l) * d + k] : 0.f;
    }
    __syncthreads();
    if (threadIdx.x < 64) {
#pragma unroll
      for (int c = 0; c < 32; ++c) sq = fmaf(xs[threadIdx.x][c], xs[threadIdx.x][c], sq);
    }
#pragma unroll
    for (int kk = 0; kk < 32; kk += 2) {
      const int kq = kk + (lane >> 5);
      const float xa = xs[wi + (lane & 31)][kq];
      const float wb = wsm[wl + (lane & 31)][kq];
      if constexpr (FEATURE_MAJOR)
        acc = __builtin_amdgcn_mfma_f32_32x32x2f32(wb, xa, acc, 0, 0, 0);
      else
        acc = __builtin_amdgcn_mfma_f32_32x32x2f32(xa, wb, acc, 0, 0, 0);
    }
    __syncthreads();
  }
  if (threadIdx.x < 64) {
    // phi of x / ||x|| when normalising (Algorithm 1, first step): the
    // projections scale by 1 / ||x|| and ||x||^2 / 2 becomes 1/2 (a zero row
    // stays zero)
    const bool nz = sq > 0.f;
    half_sq[threadIdx.x] = nprf ? (nz ? 0.5f : 0.f) : 0.5f * sq;
    row_scale[threadIdx.x] = nprf ? (nz ? rsqrtf(sq) : 0.f) : 1.f;
    trf_amp[threadIdx.x] = expf(half_sq[threadIdx.x]) * inv_sqrt_m;
  }
  __syncthreads();
  const int n_store = FEATURE_MAJOR ? ld : n;
  const int M = trf ? 2 * m : m;
#pragma unroll
  for (int v = 0; v < 16; ++v) {
    // 32x32 MFMA result layout: lane holds column lane%32, rows 8(v/4) + 4(lane/32) + v%4
    const int row = 8 * (v >> 2) + 4 * (lane >> 5) + (v & 3);
    const int col = lane & 31;
    const int li = FEATURE_MAJOR ? wl + row : wl + col;  // feature within tile
    const int ii = FEATURE_MAJOR ? wi + col : wi + row;  // position within tile
    const int l = l0 + li, i = i0 + ii;
    if (i < n_store && l < m) {
      if (trf) {
        float sv = 0.f, cv = 0.f;
        if (i < n) {
          sincosf(acc[v] * row_scale[ii], &sv, &cv);
          sv *= trf_amp[ii];
          cv *= trf_amp[ii];
        }
        if constexpr (FEATURE_MAJOR) {
          phi[(static_cast<size_t>(bh) * M + l) * ld + i] = sv;
          phi[(static_cast<size_t>(bh) * M + m + l) * ld + i] = cv;
        } else {
          phi[(static_cast<size_t>(bh) * n + i) * M + l] = sv;
          phi[(static_cast<size_t>(bh) * n + i) * M + m + l] = cv;
        }
      } else {
        const float val = i < n ? expf(fmaf(acc[v], row_scale[ii], -half_sq[ii])) * inv_sqrt_m : 0.f;
        if constexpr (FEATURE_MAJOR)
          phi[(static_cast<size_t>(bh) * M + l) * ld + i] = val;
        else
          phi[(static_cast<size_t>(bh) * n + i) * M + l] = val;
      }
    }
  }
}

// k_feature_map for d = 64 with the operands loaded straight into registers.
// d = 64.  Work-group: 256 positions of one (source, batch-head) and every
// feature, eight waves of 32 positions each.  The x rows are read once with
// coalesced 16-byte loads (consecutive threads, consecutive addresses),
// staged through LDS (rows padded to 68 floats: the 16-byte reads of 16
// lanes then fall in distinct banks) and kept in registers; W then streams
// through the same LDS buffer 128 features at a time (70 KiB of LDS: two
// work-groups, 16 waves per CU).  The MFMA sums over k in any order both
// operands agree on: half-wave h supplies k = 32 h + s at step s.  Same
// outputs and epilogue as k_feature_map.
constexpr int kFm64Pos = 256;
constexpr int kFmThreads = 2 * kFm64Pos;  // 8 waves of 32 positions
constexpr int kFm64Stride = 68;

template <typename TX>
__device__ __forceinline__ void stage_rows64(const TX* __restrict__ src, int rows_ok, float* __restrict__ dst,
                                             int nrows) {
  // nrows x 64 values -> dst[row][kFm64Stride], zero past rows_ok
  if constexpr (std::is_same<TX, float>::value) {
    for (int e = threadIdx.x; e < nrows * 16; e += kFmThreads) {
      const int row = e >> 4, c4 = e & 15;
      const float4 v = row < rows_ok ? reinterpret_cast<const float4*>(src)[e] : make_float4(0.f, 0.f, 0.f, 0.f);
      *reinterpret_cast<float4*>(dst + row * kFm64Stride + 4 * c4) = v;
    }
  } else {
    for (int e = threadIdx.x; e < nrows * 8; e += kFmThreads) {
      const int row = e >> 3, c8 = e & 7;
      const uint4 v = row < rows_ok ? reinterpret_cast<const uint4*>(src)[e] : make_uint4(0u, 0u, 0u, 0u);
      const unsigned w[4] = {v.x, v.y, v.z, v.w};
      float* o = dst + row * kFm64Stride + 8 * c8;
      *reinterpret_cast<float4*>(o) = make_float4(__uint_as_float(w[0] << 16), __uint_as_float(w[0] & 0xffff0000u),
                                                  __uint_as_float(w[1] << 16), __uint_as_float(w[1] & 0xffff0000u));
      *reinterpret_cast<float4*>(o + 4) =
          make_float4(__uint_as_float(w[2] << 16), __uint_as_float(w[2] & 0xffff0000u), __uint_as_float(w[3] << 16),
                      __uint_as_float(w[3] & 0xffff0000u));
    }
  }
}

// 32 values k = 32 h .. 32 h + 31 of LDS row `row` (8 x 16-byte reads)
__device__ __forceinline__ void lds_half_row64(const float* __restrict__ rows, int row, int h, float (&r)[32]) {
  const float4* p = reinterpret_cast<const float4*>(rows + row * kFm64Stride + 32 * h);
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    const float4 v = p[j];
    r[4 * j] = v.x;
    r[4 * j + 1] = v.y;
    r[4 * j + 2] = v.z;
    r[4 * j + 3] = v.w;
  }
}

template <typename TX, bool FEATURE_MAJOR>
__global__ __launch_bounds__(512) __attribute__((amdgpu_waves_per_eu(FEATURE_MAJOR ? 4 : 1))) void k_feature_map64(const TX* __restrict__ x0, const TX* __restrict__ x1,
                                                       const float* __restrict__ W, float* __restrict__ phi0,
                                                       float* __restrict__ phi1, int H, int n, int ld, int m,
                                                       float inv_sqrt_m, int tiles_n, int BH,
                                                       unsigned* __restrict__ fix_counts, int nprf, int trf) {
  constexpr int D = 64;
  __shared__ __align__(16) float xs[kFm64Pos * kFm64Stride];  // x tile, then W 128 features at a time
  float* const ws = xs;
  // Clear the exact-evaluation queue counters (fix_counts[0..BH]) for k_combine.
  if (fix_counts && threadIdx.x == 0)
    for (int b = blockIdx.x; b <= BH; b += gridDim.x) fix_counts[b] = 0u;
  int bid = blockIdx.x;
  const int tn = bid % tiles_n;
  bid /= tiles_n;
  const int bh = bid % BH;
  const int src = bid / BH;
  const TX* __restrict__ x = src == 0 ? x0 : x1;
  float* __restrict__ phi = src == 0 ? phi0 : phi1;
  const int h = bh % H;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int half = lane >> 5, c = lane & 31;
  const int p0 = tn * kFm64Pos;
  const int i0 = p0 + 32 * wave;  // this wave's 32 positions
  const int rows_ok = min(kFm64Pos, n - p0);
  stage_rows64(x + (static_cast<size_t>(bh) * n + p0) * D, rows_ok, xs, kFm64Pos);
  __syncthreads();
  float xr[32];
  lds_half_row64(xs, 32 * wave + c, half, xr);
  float sq = 0.f;
#pragma unroll
  for (int s2 = 0; s2 < 32; ++s2) sq = fmaf(xr[s2], xr[s2], sq);
  sq += __shfl_xor(sq, 32);  // ||x||^2 of position i0 + c
  const int n_store = FEATURE_MAJOR ? ld : n;
  const int M = trf ? 2 * m : m;
  // Whole tiles of the PRF map in the feature-major layout: position i0 + c
  // of this lane; phi = 2^(a s log2(e) + e0) with e0 = -h log2(e) - log2(sqrt(m))
  // (s, h: the row scale and ||x||^2 / 2 of the epilogue below), stored
  // through a buffer resource over this (source, batch-head)'s rows: the
  // lane's offset in a VGPR, the feature's in an SGPR.
  constexpr float kLog2e = 1.44269504088896341f;
  const bool nzl = sq > 0.f;
  const float hs_l = nprf ? (nzl ? 0.5f : 0.f) : 0.5f * sq;
  const float rs_l = (nprf ? (nzl ? rsqrtf(sq) : 0.f) : 1.f) * kLog2e;
  const float e0_l = fmaf(-hs_l, kLog2e, __log2f(inv_sqrt_m));
  const bool pos_ok = i0 + c < n;  // positions n .. ld - 1 are zeros
  const __amdgpu_buffer_rsrc_t out_rsrc = __builtin_amdgcn_make_buffer_rsrc(
      phi + static_cast<size_t>(bh) * M * ld, 0, FEATURE_MAJOR ? M * ld * 4 : 0, 0x00020000);
  const uint32_t out_voff = static_cast<uint32_t>(4 * half * ld + i0 + c) * 4u;
  for (int l0 = 0; l0 < m; l0 += 64) {
    if (l0 % 128 == 0) {
      __syncthreads();  // x rows / the previous W features consumed
      stage_rows64(W + (static_cast<size_t>(h) * m + l0) * D, min(128, m - l0), ws, 128);
      __syncthreads();
    }
    floatx16 acc[2];
#pragma unroll
    for (int t = 0; t < 2; ++t) {
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[t][v] = 0.f;
      float wr[32];
      lds_half_row64(ws, (l0 % 128) + 32 * t + c, half, wr);
#pragma unroll
      for (int s2 = 0; s2 < 32; ++s2) {
        if constexpr (FEATURE_MAJOR)
          acc[t] = __builtin_amdgcn_mfma_f32_32x32x2f32(wr[s2], xr[s2], acc[t], 0, 0, 0);
        else
          acc[t] = __builtin_amdgcn_mfma_f32_32x32x2f32(xr[s2], wr[s2], acc[t], 0, 0, 0);
      }
    }
    if (FEATURE_MAJOR && !trf && i0 + 32 <= n_store && l0 + 64 <= m) {  // uniform
#pragma unroll
      for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          // feature l0 + 32 t + 8 (v / 4) + 4 (lane / 32) + v % 4 of position i0 + c
          const float val = pos_ok ? __builtin_amdgcn_exp2f(fmaf(acc[t][v], rs_l, e0_l)) : 0.f;
          const uint32_t soff = static_cast<uint32_t>((l0 + 32 * t + 8 * (v >> 2) + (v & 3)) * ld) * 4u;
          __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(val), out_rsrc, out_voff, soff, 0);
        }
      continue;
    }
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        // 32x32 MFMA result layout: lane holds column lane%32, rows 8(v/4) + 4(lane/32) + v%4
        const int row = 8 * (v >> 2) + 4 * half + (v & 3);
        const int li = FEATURE_MAJOR ? row : c;  // feature within the 32-feature tile t
        const int ii = FEATURE_MAJOR ? c : row;  // position within the wave's 32
        // ||x||^2 of position i0 + ii lives in lanes ii and ii + 32
        const float sqi = FEATURE_MAJOR ? sq : __shfl(sq, ii);
        const bool nz = sqi > 0.f;
        // phi of x / ||x|| when normalising (Algorithm 1, first step): the
        // projections scale by 1 / ||x|| and ||x||^2 / 2 becomes 1/2 (a zero
        // row stays zero)
        const float half_sq = nprf ? (nz ? 0.5f : 0.f) : 0.5f * sqi;
        const float row_scale = nprf ? (nz ? rsqrtf(sqi) : 0.f) : 1.f;
        const int l = l0 + 32 * t + li, i = i0 + ii;
        if (i < n_store && l < m) {
          if (trf) {
            float sv = 0.f, cv = 0.f;
            if (i < n) {
              const float amp = expf(half_sq) * inv_sqrt_m;
              sincosf(acc[t][v] * row_scale, &sv, &cv);
              sv *= amp;
              cv *= amp;
            }
            if constexpr (FEATURE_MAJOR) {
              phi[(static_cast<size_t>(bh) * M + l) * ld + i] = sv;
              phi[(static_cast<size_t>(bh) * M + m + l) * ld + i] = cv;
            } else {
              phi[(static_cast<size_t>(bh) * n + i) * M + l] = sv;
              phi[(static_cast<size_t>(bh) * n + i) * M + m + l] = cv;
            }
          } else {
            const float val = i < n ? expf(fmaf(acc[t][v], row_scale, -half_sq)) * inv_sqrt_m : 0.f;
            if constexpr (FEATURE_MAJOR)
              phi[(static_cast<size_t>(bh) * M + l) * ld + i] = val;
            else
              phi[(static_cast<size_t>(bh) * n + i) * M + l] = val;
          }
        }
      }
  }
}

// The elu + 1 map of the linear transformer the paper compares with (Sec. 2):
// phi_l(x) = x_l + 1 for x_l > 0, exp(x_l) otherwise, d features, no
// projections (of x / ||x|| when normalising; a zero row stays zero before
// the map).  Block: 64 positions of one (source, batch-head), x staged through
// LDS; same output layouts and queue-counter duty as k_feature_map.
template <typename TX, bool FEATURE_MAJOR>
__global__ __launch_bounds__(256) void k_feature_elu(const TX* __restrict__ x0, const TX* __restrict__ x1,
                                                     float* __restrict__ phi0, float* __restrict__ phi1, int n,
                                                     int ld, int d, int tiles_n, int BH,
                                                     unsigned* __restrict__ fix_counts, int nprf) {
  if (fix_counts && threadIdx.x == 0 && blockIdx.x <= static_cast<unsigned>(BH)) fix_counts[blockIdx.x] = 0u;
  __shared__ float xs[64][kMaxD + 1];
  __shared__ float scale[64];
  int bid = blockIdx.x;
  const int tn = bid % tiles_n;
  bid /= tiles_n;
  const int bh = bid % BH, src = bid / BH;
  const TX* __restrict__ xb = (src == 0 ? x0 : x1) + static_cast<size_t>(bh) * n * d;
  float* __restrict__ phi = src == 0 ? phi0 : phi1;
  const int i0 = tn * 64;
  for (int e = threadIdx.x; e < 64 * d; e += 256) {
    const int r = e / d, c = e - r * d;
    xs[r][c] = i0 + r < n ? to_f32(xb[static_cast<size_t>(i0 + r) * d + c]) : 0.f;
  }
  __syncthreads();
  if (threadIdx.x < 64) {
    float sq = 0.f;
    for (int c = 0; c < d; ++c) sq = fmaf(xs[threadIdx.x][c], xs[threadIdx.x][c], sq);
    scale[threadIdx.x] = nprf ? (sq > 0.f ? rsqrtf(sq) : 0.f) : 1.f;
  }
  __syncthreads();
  const int rows = FEATURE_MAJOR ? ld : n;
  for (int e = threadIdx.x; e < 64 * d; e += 256) {
    // feature-major: lanes along positions; position-major: lanes along features
    const int r = FEATURE_MAJOR ? (e & 63) : e / d, l = FEATURE_MAJOR ? (e >> 6) : e - (e / d) * d;
    const int i = i0 + r;
    if (i >= rows) continue;
    float val = 0.f;
    if (i < n) {
      const float t = xs[r][l] * scale[r];
      val = t > 0.f ? t + 1.f : expf(t);
    }
    if constexpr (FEATURE_MAJOR)
      phi[(static_cast<size_t>(bh) * d + l) * ld + i] = val;
    else
      phi[(static_cast<size_t>(bh) * n + i) * d + l] = val;
  }
}

// ------------------------------------------------------------ v prep --
// The value columns v'(pos, c) = v[bh * bh_stride + pos * sp + c * sc]
// (c < ncols; column ncols is all ones when with_ones: the denominator's
// channel A2 of Eq. (11)), scaled per column by
// s_c = max_pos |v'(pos, c)| and packed as column pairs:
//   vsc[bh][p][pos] = (v'(pos, 2p) / s_2p, v'(pos, 2p+1) / s_2p+1)  for pos < n,
//   0 for n <= pos < N;  colmax[bh][c] = s_c.
// Two passes, both reading v along its contiguous index (columns when
// sc == 1, positions otherwise): k_vmax takes per-chunk column maxima of
// 256 positions x 64 columns, k_vscale reduces them and writes 64 positions x
// 32 pairs per block through an LDS transpose.
constexpr int kVmaxChunk = 256;

template <typename TV>
__global__ __launch_bounds__(256) void k_vmax(const TV* __restrict__ v, long long sp, long long sc,
                                              long long bh_stride, int ncols, int n, int nchunk, int cgroups,
                                              float* __restrict__ pmax) {
  __shared__ unsigned cm[64];
  int bid = blockIdx.x;
  const int cg = bid % cgroups;
  bid /= cgroups;
  const int ch = bid % nchunk, bh = bid / nchunk;
  const TV* __restrict__ vb = v + bh * bh_stride;
  const int tid = threadIdx.x;
  const int c0 = cg * 64, nc = min(64, ncols - c0);
  const int pos0 = ch * kVmaxChunk, np = min(kVmaxChunk, n - pos0);
  if (tid < 64) cm[tid] = 0u;
  __syncthreads();
  if (sc == 1) {
    // rows contiguous in the columns: thread (tid & 63) keeps its column's
    // maximum over rows tid >> 6, + 4, ... in a register (loads coalesced
    // along the row), then one LDS maximum per thread
    const int c = tid & 63;
    float mx = 0.f;
    if (c < nc) {
#pragma unroll 8
      for (int r = tid >> 6; r < np; r += 4) mx = fmaxf(mx, fabsf(to_f32(vb[(pos0 + r) * sp + c0 + c])));
    }
    if (c < nc) atomicMax(&cm[c], __float_as_uint(mx));  // mx >= 0: bit patterns order like the values
  } else {
    // columns strided: wave w takes columns w, w + 4, ..., its lanes the
    // positions lane, lane + 64, ... (loads coalesced along the column), and
    // reduces across the wave
    const int wave = tid >> 6, lane = tid & 63;
    for (int c = wave; c < nc; c += 4) {
      float mx = 0.f;
      for (int r = lane; r < np; r += 64) mx = fmaxf(mx, fabsf(to_f32(vb[(pos0 + r) * sp + (c0 + c) * sc])));
#pragma unroll
      for (int off = 32; off > 0; off >>= 1) mx = fmaxf(mx, __shfl_xor(mx, off));
      if (lane == 0) cm[c] = __float_as_uint(mx);
    }
  }
  __syncthreads();
  if (tid < nc) pmax[(static_cast<size_t>(bh) * nchunk + ch) * ncols + c0 + tid] = __uint_as_float(cm[tid]);
}

template <typename TV>
__global__ __launch_bounds__(256) void k_vscale(const TV* __restrict__ v, long long sp, long long sc,
                                                long long bh_stride, int ncols, int with_ones, int n, int N,
                                                int nchunk, int cgroups, const float* __restrict__ pmax,
                                                float* __restrict__ colmax, float2* __restrict__ vsc) {
  __shared__ float tile[64][65];  // [column][position]
  __shared__ float scale[64];
  int bid = blockIdx.x;
  const int cg = bid % cgroups;
  bid /= cgroups;
  const int ptiles = (N + 63) / 64;
  const int pt = bid % ptiles, bh = bid / ptiles;
  const int cols = ncols + with_ones, pairs = (cols + 1) / 2;
  const TV* __restrict__ vb = v + bh * bh_stride;
  const int tid = threadIdx.x;
  const int c0 = cg * 64, nc = min(64, cols - c0);
  const int pos0 = pt * 64;
  if (tid < nc) {
    const int c = c0 + tid;
    float sv = 1.f;  // the ones column
    if (c < ncols) {
      sv = 0.f;
      const float* __restrict__ pm = pmax + static_cast<size_t>(bh) * nchunk * ncols + c;
      int ch = 0;
      for (; ch + 4 <= nchunk; ch += 4)
        sv = fmaxf(fmaxf(sv, fmaxf(pm[ch * ncols], pm[(ch + 1) * ncols])),
                   fmaxf(pm[(ch + 2) * ncols], pm[(ch + 3) * ncols]));
      for (; ch < nchunk; ++ch) sv = fmaxf(sv, pm[ch * ncols]);
    }
    if (pt == 0) colmax[static_cast<size_t>(bh) * cols + c] = sv;
    scale[tid] = sv > 0.f ? sv : 1.f;
  }
  const int np = max(0, min(64, n - pos0));
  const int nv = max(0, min(nc, ncols - c0));  // value columns of this group
  if (sc == 1) {
    // thread (tid & 63) reads its column along rows tid >> 6, + 4, ...
    const int c = tid & 63;
    if (c < nv) {
#pragma unroll
      for (int r = tid >> 6; r < 64; r += 4)
        if (r < np) tile[c][r] = to_f32(vb[(pos0 + r) * sp + c0 + c]);
    }
  } else {
    // columns strided: thread (tid & 63) reads position tid & 63 of columns
    // tid >> 6, + 4, ... (coalesced along the column)
    const int r = tid & 63;
    if (r < np)
      for (int c = tid >> 6; c < nv; c += 4) tile[c][r] = to_f32(vb[(pos0 + r) * sp + (c0 + c) * sc]);
  }
  __syncthreads();
  const int npairs = (nc + 1) / 2;
  for (int e = tid; e < npairs * 64; e += 256) {
    const int pl = e >> 6, r = e & 63;
    const int ca = 2 * pl, cb = 2 * pl + 1;
    float a = 0.f, b2 = 0.f;
    if (r < np) {
      a = ca < nv ? tile[ca][r] / scale[ca] : (ca < nc ? 1.f : 0.f);
      b2 = cb < nv ? tile[cb][r] / scale[cb] : (cb < nc ? 1.f : 0.f);
    }
    if (pos0 + r < N) vsc[(static_cast<size_t>(bh) * pairs + c0 / 2 + pl) * N + pos0 + r] = make_float2(a, b2);
  }
}

// The same two passes for rows of v contiguous in the columns (sc == 1) with
// ncols, the row stride and the base 4-element aligned: every thread reads
// 4-column quads (16 bytes in fp32, 8 in bf16), quad t % 16 of rows t / 16,
// + 16, ...; rows past a chunk or past n read a valid row instead (the max
// is unchanged, the scaled values of positions >= n are written as zeros).
// Grids (column group, chunk or 64-position tile, batch-head).
template <typename TV>
__device__ __forceinline__ float4 load_quad(const TV* __restrict__ p) {
  if constexpr (sizeof(TV) == 4) {
    return *reinterpret_cast<const float4*>(p);
  } else {
    const uint2 u = *reinterpret_cast<const uint2*>(p);
    return make_float4(__uint_as_float(u.x << 16), __uint_as_float(u.x & 0xffff0000u), __uint_as_float(u.y << 16),
                       __uint_as_float(u.y & 0xffff0000u));
  }
}

template <typename TV>
__global__ __launch_bounds__(256) void k_vmax_q(const TV* __restrict__ v, int sp, long long bh_stride, int ncols,
                                                int n, int nchunk, float* __restrict__ pmax) {
  __shared__ float wm[4][64];
  const int cg = blockIdx.x, ch = blockIdx.y, bh = blockIdx.z;
  const int tid = threadIdx.x, q = tid & 15, r0 = tid >> 4, lane = tid & 63, wave = tid >> 6;
  const int c0 = cg * 64, nq = min(16, (ncols - c0) / 4);
  const int pos0 = ch * kVmaxChunk, np = min(kVmaxChunk, n - pos0);
  // the chunk's first row (uniform), then 32-bit offsets; all loads before any use
  const TV* __restrict__ vb = v + bh * bh_stride + static_cast<long long>(pos0) * sp + c0;
  const int qo = 4 * min(q, nq - 1);
  constexpr int J = kVmaxChunk / 16;
  float4 x[J];
#pragma unroll
  for (int j = 0; j < J; ++j) x[j] = load_quad(vb + (min(r0 + 16 * j, np - 1) * sp + qo));
  float m0 = 0.f, m1 = 0.f, m2 = 0.f, m3 = 0.f;
#pragma unroll
  for (int j = 0; j < J; ++j) {
    m0 = fmaxf(m0, fabsf(x[j].x));
    m1 = fmaxf(m1, fabsf(x[j].y));
    m2 = fmaxf(m2, fabsf(x[j].z));
    m3 = fmaxf(m3, fabsf(x[j].w));
  }
  // lanes q, q + 16, q + 32, q + 48 of a wave hold the same quad
#pragma unroll
  for (int off = 16; off < 64; off <<= 1) {
    m0 = fmaxf(m0, __shfl_xor(m0, off));
    m1 = fmaxf(m1, __shfl_xor(m1, off));
    m2 = fmaxf(m2, __shfl_xor(m2, off));
    m3 = fmaxf(m3, __shfl_xor(m3, off));
  }
  if (lane < 16) {
    wm[wave][4 * lane] = m0;
    wm[wave][4 * lane + 1] = m1;
    wm[wave][4 * lane + 2] = m2;
    wm[wave][4 * lane + 3] = m3;
  }
  __syncthreads();
  if (tid < 4 * nq)
    pmax[(static_cast<size_t>(bh) * nchunk + ch) * ncols + c0 + tid] =
        fmaxf(fmaxf(wm[0][tid], wm[1][tid]), fmaxf(wm[2][tid], wm[3][tid]));
}

// Group cg holds columns [64 cg, 64 cg + 64) of v' (the ones column too when
// it falls there); when ncols is a multiple of 64 the ones column's pair
// (1, 0) is written by the last group.
template <typename TV>
__global__ __launch_bounds__(256) void k_vscale_q(const TV* __restrict__ v, int sp, long long bh_stride,
                                                  int ncols, int with_ones, int n, int N, int nchunk,
                                                  const float* __restrict__ pmax, float* __restrict__ colmax,
                                                  float2* __restrict__ vsc) {
  __shared__ float tile[64][65];  // [column][position]
  __shared__ float scale[64];
  const int cg = blockIdx.x, pt = blockIdx.y, bh = blockIdx.z;
  const int cols = ncols + with_ones, pairs = (cols + 1) / 2;
  const int tid = threadIdx.x;
  const int c0 = cg * 64, nv = min(64, ncols - c0), nc = min(64, cols - c0);
  const bool extra = with_ones && cg == static_cast<int>(gridDim.x) - 1 && ncols - c0 == 64;
  const int pos0 = pt * 64;
  const int np = max(0, min(64, n - pos0));
  // this tile's quads first (their latency overlaps the scale reduction)
  const int q = tid & 15, r0 = tid >> 4;
  float4 x[4];
  const TV* __restrict__ vb = v + bh * bh_stride + c0;
  const int qo = 4 * min(q, nv / 4 - 1);
#pragma unroll
  for (int j = 0; j < 4; ++j) x[j] = load_quad(vb + (min(pos0 + r0 + 16 * j, n - 1) * sp + qo));
  if (tid < nc) {
    const int c = c0 + tid;
    float sv = 1.f;  // the ones column
    if (c < ncols) {
      sv = 0.f;
      const float* __restrict__ pm = pmax + static_cast<size_t>(bh) * nchunk * ncols + c;
      int ch = 0;
      for (; ch + 4 <= nchunk; ch += 4)
        sv = fmaxf(fmaxf(sv, fmaxf(pm[ch * ncols], pm[(ch + 1) * ncols])),
                   fmaxf(pm[(ch + 2) * ncols], pm[(ch + 3) * ncols]));
      for (; ch < nchunk; ++ch) sv = fmaxf(sv, pm[ch * ncols]);
    }
    if (pt == 0) colmax[static_cast<size_t>(bh) * cols + c] = sv;
    scale[tid] = sv > 0.f ? sv : 1.f;
  }
  if (extra && pt == 0 && tid == 0) colmax[static_cast<size_t>(bh) * cols + ncols] = 1.f;
  if (q < nv / 4) {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int r = r0 + 16 * j;
      tile[4 * q][r] = x[j].x;
      tile[4 * q + 1][r] = x[j].y;
      tile[4 * q + 2][r] = x[j].z;
      tile[4 * q + 3][r] = x[j].w;
    }
  }
  __syncthreads();
  const int npairs = (nc + 1) / 2 + (extra ? 1 : 0);
  const int ones = ncols - c0;  // the ones column, group-relative (may lie past this group)
  for (int e = tid; e < npairs * 64; e += 256) {
    const int pl = e >> 6, r = e & 63;
    const int ca = 2 * pl, cb = 2 * pl + 1;
    float a = 0.f, b2 = 0.f;
    if (r < np) {
      a = ca < nv ? tile[ca][r] / scale[ca] : (with_ones && ca == ones ? 1.f : 0.f);
      b2 = cb < nv ? tile[cb][r] / scale[cb] : (with_ones && cb == ones ? 1.f : 0.f);
    }
    if (pos0 + r < N) vsc[(static_cast<size_t>(bh) * pairs + c0 / 2 + pl) * N + pos0 + r] = make_float2(a, b2);
  }
}

// ------------------------------------------------------- channel norms --
// X2[bh][ks][l][p] = sum over positions of slice ks of phi_l(k_j)^2 |vsc_p(j)|^2
// = ||x_{l,p}||^2 restricted to the slice, x_{l,p} the packed signal the
// convolution kernel transforms for feature l and column pair p.  Block
// (bh, l-tile of 64, slice ks), positions staged through LDS 64 at a time, the
// product phi^2 |vsc|^2 over positions on the matrix cores: wave w takes the
// 32 features 32 (w & 1) .. and the 32-pair tiles w >> 1, (w >> 1) + 2.
constexpr int kMaxPairs = (kMaxD + 2) / 2;
constexpr int kGramPT = (kMaxPairs + 31) / 32;  // 32-pair tiles
constexpr int kGramL = 128;                      // features per work-group (eight waves of 32 x 32-pair tiles)

__global__ __launch_bounds__(512) void k_gram(const float* __restrict__ phik, const float2* __restrict__ vsc,
                                              float* __restrict__ X2, int m, int N, int pairs, int ltiles,
                                              int ksplit) {
  __shared__ float4 A4[64][kGramL / 4 + 1];  // phi^2, [position][feature quad]
  __shared__ float Bq[64][kMaxPairs | 1];  // |vsc|^2, [position][pair]
  int bid = blockIdx.x;
  const int ks = bid % ksplit;
  bid /= ksplit;
  const int lt = bid % ltiles, bh = bid / ltiles;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int ft = wave & 3, pt0 = wave >> 2, lr = lane & 31, lk = lane >> 5;
  const int l0 = lt * kGramL;
  const float* __restrict__ pk = phik + static_cast<size_t>(bh) * m * N;
  const float2* __restrict__ vb = vsc + static_cast<size_t>(bh) * pairs * N;
  const int slice = N / ksplit, pos_begin = ks * slice, pos_end = pos_begin + slice;
  constexpr int AS = 4 * (kGramL / 4 + 1);  // floats per position row of A4
  const float* __restrict__ Af = reinterpret_cast<const float*>(&A4[0][0]);  // [position][AS]: feature f at f
  floatx16 acc[2];
  float vs[2] = {0.f, 0.f};
#pragma unroll
  for (int t = 0; t < 2; ++t)
#pragma unroll
    for (int e = 0; e < 16; ++e) acc[t][e] = 0.f;
  // The next chunk's values are loaded into registers while the current
  // chunk is multiplied out of LDS (thread tid holds positions tid & 63 of
  // feature quads tid >> 6 + 8 e and of pairs tid >> 6 + 8 e).
  constexpr int kGramPB = (kMaxPairs + 7) / 8;
  float na[4][4];
  float2 nb[kGramPB];
  const int xl = tid & 63, ql = tid >> 6;
  auto fetch = [&](int p0) {
#pragma unroll
    for (int e = 0; e < 4; ++e)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int l = l0 + 4 * (ql + 8 * e) + j;
        na[e][j] = (l < m && p0 + xl < pos_end) ? pk[static_cast<size_t>(l) * N + p0 + xl] : 0.f;
      }
#pragma unroll
    for (int e = 0; e < kGramPB; ++e) {
      const int p = ql + 8 * e;
      nb[e] = (p < pairs && p0 + xl < pos_end) ? vb[static_cast<size_t>(p) * N + p0 + xl] : make_float2(0.f, 0.f);
    }
  };
  if (pos_begin < pos_end) fetch(pos_begin);
  for (int p0 = pos_begin; p0 < pos_end; p0 += 64) {
    __syncthreads();
#pragma unroll
    for (int e = 0; e < 4; ++e)
      A4[xl][ql + 8 * e] = make_float4(na[e][0] * na[e][0], na[e][1] * na[e][1], na[e][2] * na[e][2],
                                       na[e][3] * na[e][3]);
#pragma unroll
    for (int e = 0; e < kGramPB; ++e) {
      const int p = ql + 8 * e;
      if (p < pairs) Bq[xl][p] = nb[e].x * nb[e].x + nb[e].y * nb[e].y;
    }
    __syncthreads();
    if (p0 + 64 < pos_end) fetch(p0 + 64);
    // A[feature][position] = phi^2, B[position][pair] = |vsc|^2, 2 positions per step
#pragma unroll
    for (int t = 0; t < 2; ++t) {
      const int p0 = 32 * (pt0 + 2 * t), p = p0 + lr;
      if (pt0 + 2 * t < kGramPT && p0 + 1 == pairs) {
        // a tile with one pair (the last, e.g. the ones column's): lane sums
        // its feature 32 ft + lr over the positions of its half, on the VALU
#pragma unroll 8
        for (int s2 = 0; s2 < 32; ++s2) {
          const int x = 2 * s2 + lk;
          vs[t] = fmaf(Af[x * AS + 32 * ft + lr], Bq[x][p0], vs[t]);
        }
      } else if (pt0 + 2 * t < kGramPT && p0 < pairs) {
#pragma unroll 8
        for (int s2 = 0; s2 < 32; ++s2) {
          const int x = 2 * s2 + lk;
          const float a = Af[x * AS + 32 * ft + lr];
          const float bq = p < pairs ? Bq[x][p] : 0.f;
          acc[t] = __builtin_amdgcn_mfma_f32_32x32x2f32(a, bq, acc[t], 0, 0, 0);
        }
      }
    }
  }
  // result tile t: lane holds pair 32 (pt0 + 2 t) + lr, features 32 ft + row(e)
  float* __restrict__ out = X2 + (static_cast<size_t>(bh) * ksplit + ks) * m * pairs;
#pragma unroll
  for (int t = 0; t < 2; ++t) {
    const int p0 = 32 * (pt0 + 2 * t), p = p0 + lr;
    if (pt0 + 2 * t < kGramPT && p0 + 1 == pairs) {
      const float v = vs[t] + __shfl_xor(vs[t], 32);  // both halves of the positions
      const int l = l0 + 32 * ft + lr;
      if (lk == 0 && l < m) out[static_cast<size_t>(l) * pairs + p0] = v;
    } else if (pt0 + 2 * t < kGramPT && p < pairs) {
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int l = l0 + 32 * ft + 8 * (e >> 2) + 4 * lk + (e & 3);
        if (l < m) out[static_cast<size_t>(l) * pairs + p] = acc[t][e];
      }
    }
  }
}

// Bound weights of k_combine, per (bh, feature l):
//   Wb[bh][l] = (A_l, D_l),  A_l = max_{c < d} s_c ||x_{l,c/2}||,  D_l = ||x_{l,d/2}||
// (column d is the all-ones column of the denominator, scale 1), and
//   Wb[bh][m] = (max_{c < d} s_c, 0).
__global__ __launch_bounds__(256) void k_bound_weights(const float* __restrict__ X2, const float* __restrict__ colmax,
                                                       float2* __restrict__ Wb, int BH, int m, int d, int pairs,
                                                       int ksplit) {
  // one wave per (bh, l): lane p (p < pairs, two rounds of 64) sums its
  // slices, the wave reduces the maxima
  const long long e = static_cast<long long>(blockIdx.x) * 4 + (threadIdx.x >> 6);
  if (e >= static_cast<long long>(BH) * (m + 1)) return;  // uniform per wave
  const int lane = threadIdx.x & 63;
  const int bh = static_cast<int>(e / (m + 1)), l = static_cast<int>(e % (m + 1));
  const float* __restrict__ s = colmax + static_cast<size_t>(bh) * (d + 1);
  float A = 0.f, D = 0.f;
  if (l == m) {
    for (int c = lane; c < d; c += 64) A = fmaxf(A, s[c]);
  } else {
    for (int p = lane; p < pairs; p += 64) {
      float x2 = 0.f;
      for (int ks = 0; ks < ksplit; ++ks) x2 += X2[((static_cast<size_t>(bh) * ksplit + ks) * m + l) * pairs + p];
      const float nrm = sqrtf(x2);
      const int c0 = 2 * p, c1 = 2 * p + 1;
      if (c0 < d) A = fmaxf(A, nrm * s[c0]);
      if (c1 < d) A = fmaxf(A, nrm * s[c1]);
      if (c0 == d || c1 == d) D = nrm;
    }
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) {
    A = fmaxf(A, __shfl_xor(A, off));
    D = fmaxf(D, __shfl_xor(D, off));  // one lane holds D, the others 0
  }
  if (lane == 0) Wb[e] = make_float2(A, D);
}

// -------------------------------------------------------------- combine --
// z[bh][i][c] = sum_s P_s[c][i] / sum_s P_s[d][i],  P = part[bh], s < nsplit,
// and the certification of each row.  With K = kGamma u log2(L) ||h||_2 / sqrt(L)
// the error model of common.hpp bounds the rounding error of numerator c by
// K s_c sum_l phi_l(q_i) ||x_{l,c/2}||_2 <= K sum_l phi_l(q_i) A_l (+ a part
// relative to the value itself) and that of the denominator by
// K sum_l phi_l(q_i) D_l (weights of k_bound_weights).  A row whose normwise
// relative bound exceeds kTau is queued for k_fixup.  Block: 64 rows of one
// (batch, head); dynamic LDS holds the (d + 1) x 64 tile of sums and the
// m + 1 weights.
template <int NS>
__global__ __launch_bounds__(256) void k_combine(const float* __restrict__ part, const float* __restrict__ phiq,
                                                 const float2* __restrict__ Wb, const float2* __restrict__ hnorm,
                                                 float* __restrict__ z, float* __restrict__ den_out,
                                                 unsigned* __restrict__ fix,
                                                 unsigned long long* __restrict__ fixmask, int BH, int H, int n, int N,
                                                 int log2N, int d, int m, int nsplit, int tiles_n) {
  extern __shared__ float dyn[];
  const int cols = d + 1;
  float* tile = dyn;                                                  // [cols][65]
  float2* wl = reinterpret_cast<float2*>(dyn + ((cols * 65 + 1) & ~1));  // [m + 1]
  __shared__ float2 bsum[4][64];
  __shared__ float zpart[4][64];
  __shared__ float rden[64];
  const int bh = blockIdx.x / tiles_n, i0 = (blockIdx.x % tiles_n) * 64;
  const int h = bh % H;
  const int tid = threadIdx.x, li = tid & 63, qg = tid >> 6;
  const float* __restrict__ p0 = part + static_cast<size_t>(bh) * nsplit * cols * n;
  if constexpr (NS > 0) {
    // NS partials per value, four values per thread at a time: 4 NS loads in
    // flight before any is used, each value summed in split order
    const size_t step = static_cast<size_t>(cols) * n;
    for (int e0 = tid; e0 < cols * 64; e0 += 4 * 256) {
      float a[4][NS];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int e = e0 + 256 * u, c = min(e >> 6, cols - 1), pos = min(i0 + (e & 63), n - 1);
        const float* __restrict__ pc = p0 + static_cast<size_t>(c) * n + pos;
#pragma unroll
        for (int sp = 0; sp < NS; ++sp) a[u][sp] = pc[sp * step];
      }
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int e = e0 + 256 * u;
        if (e < cols * 64) {
          float t = a[u][0];
#pragma unroll
          for (int sp = 1; sp < NS; ++sp) t += a[u][sp];
          tile[(e >> 6) * 65 + (e & 63)] = i0 + (e & 63) < n ? t : 1.f;
        }
      }
    }
  } else {
    for (int e = tid; e < cols * 64; e += 256) {
      const int c = e >> 6, i = e & 63;
      const int pos = i0 + i;
      float t = 1.f;
      if (pos < n) {
        // the partials' loads issued together, summed in split order
        const float* __restrict__ pc = p0 + static_cast<size_t>(c) * n + pos;
        const size_t step = static_cast<size_t>(cols) * n;
        t = pc[0];
        int sp = 1;
        for (; sp + 3 <= nsplit; sp += 3) {
          const float a1 = pc[sp * step], a2 = pc[(sp + 1) * step], a3 = pc[(sp + 2) * step];
          t = ((t + a1) + a2) + a3;
        }
        for (; sp < nsplit; ++sp) t += pc[sp * step];
      }
      tile[c * 65 + i] = t;
    }
  }
  for (int l = tid; l <= m; l += 256) wl[l] = Wb[static_cast<size_t>(bh) * (m + 1) + l];
  __syncthreads();
  // bound sums (features qg, qg + 4, ...) and the largest numerator magnitude
  // (columns qg, qg + 4, ...) of row li
  {
    const int pos = i0 + li;
    float bA = 0.f, bD = 0.f;
    if (pos < n) {
      const float* __restrict__ pq = phiq + static_cast<size_t>(bh) * m * N + pos;
#pragma unroll 8
      for (int l = qg; l < m; l += 4) {
        const float f = fabsf(pq[static_cast<size_t>(l) * N]);  // signed features (TRF)
        const float2 w = wl[l];
        bA = fmaf(f, w.x, bA);
        bD = fmaf(f, w.y, bD);
      }
    }
    float zm = 0.f;
    for (int c = qg; c < d; c += 4) zm = fmaxf(zm, fabsf(tile[c * 65 + li]));
    bsum[qg][li] = make_float2(bA, bD);
    zpart[qg][li] = zm;
  }
  __syncthreads();
  if (tid < 64) {
    const int i = tid, pos = i0 + i;
    const float den = tile[d * 65 + i];
    const float inv = 1.0f / den;
    rden[i] = inv;
    if (den_out && pos < n) den_out[static_cast<size_t>(bh) * n + pos] = den;
    bool flag = false;
    if (pos < n) {
      const float L = static_cast<float>(2 << log2N);
      const float lg = static_cast<float>(log2N + 1);
      const float K = kGamma * kUnitRoundoff * lg * hnorm[h].y * rsqrtf(L);
      float bA = 0.f, bD = 0.f, num = 0.f;
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        bA += bsum[g][i].x;
        bD += bsum[g][i].y;
        num = fmaxf(num, zpart[g][i]);
      }
      const float zm = num * fabsf(inv);  // max_c |z_c|
      const float vmax = wl[m].x;
      const float err = K * bA + zm * (K * bD);
      const float scale = fmaxf(zm, 1e-6f * vmax);
      const float rel_floor = 2.f * kGamma * kUnitRoundoff * lg;
      const bool ok = isfinite(den) && den != 0.f && isfinite(zm) && err <= (kTau - rel_floor) * scale * fabsf(den);
      flag = !ok;
    }
    // One wave holds the tile's 64 rows: its uncertified rows as one mask
    // word, counted per head (fix[0..BH)) and in total (fix[BH]).
    const unsigned long long mask = __ballot(flag);
    if (threadIdx.x == 0) {
      fixmask[static_cast<size_t>(bh) * tiles_n + blockIdx.x % tiles_n] = mask;
      if (mask != 0ull) {
        const unsigned nflag = static_cast<unsigned>(__popcll(mask));
        atomicAdd(&fix[bh], nflag);
        atomicAdd(&fix[BH], nflag);
      }
    }
  }
  __syncthreads();
  float* __restrict__ zb = z + static_cast<size_t>(bh) * n * d;
  for (int e = tid; e < 64 * d; e += 256) {
    const int i = e / d, c = e - i * d;
    const int pos = i0 + i;
    if (pos < n) zb[static_cast<size_t>(pos) * d + c] = tile[c * 65 + i] * rden[i];
  }
}

// Exact rows: Eq. (10) evaluated directly for the rows queued per head (the
// rows the FFT route cannot certify, or every row on the direct route), in
// groups of 32 rows taken in row order.  A group's keys run in chunks of 128;
// when a head has fewer groups than work-group slots, k_fix_plan cuts each
// group's chunks into parts of about equal size (work items), else an item is
// a whole group.  Wave w of the work-group takes the 32 keys jc + 32 w of
// every chunk of the item:
//   S^T = phi(k_keys) phi(q_rows)^T   32 keys x 32 rows, fp32 MFMA over the m features
//   P   = S^T * c_{j-i}               c = exp(b) from a table per head; 0 for keys >= n
//   Z  += P^T [v, ...]                fp32 MFMA, whose A operand is exactly the
//                                     layout S^T leaves in the registers (no LDS)
// and the denominator as the sum of P over the keys.  Per 32 keys the fp32
// sums are added into fp64 totals; the four waves' totals are added in wave
// order at the end, so results are bitwise deterministic.  Keys outside a
// row's finite-b range contribute exact zeros, and chunks outside the
// group's range are skipped.  A group in one part writes its rows; parts go
// to fixpart and k_fixup_combine adds them in part order.
constexpr int kFixRows = 32;
constexpr int kFixKeys = 128;
constexpr int kFixL = 32;  // features staged per step
constexpr int kFixMaxTiles = (1 << kMaxLongLog2N) / 64;
constexpr int kFixMaxGroups = (1 << kMaxLongLog2N) / kFixRows;
// smallest part (chunks) worth a work item of its own
constexpr int kFixMinPart = 16;

// The exact-row plan (workspace, int32), for BH heads of n rows and `slots`
// work-group slots per head:
//   items [BH][slots] int4   {group, first chunk, end chunk, parts of the group}
//   hdr   [BH] int2          {work items, 1 if the items table is used}
//   rows  [BH][n]            queued rows of the head in row order
//   gfirst [BH][n / 32 + 1]  first item of each group, then the item count
struct FixPlan {
  int4* items;
  int2* hdr;
  int* rows;
  int* gfirst;
  int n, slots, gstride;
  __host__ __device__ FixPlan(int* base, int BH, int n_, int slots_)
      : n(n_), slots(slots_), gstride((n_ + kFixRows - 1) / kFixRows + 1) {
    items = reinterpret_cast<int4*>(base);
    hdr = reinterpret_cast<int2*>(base + static_cast<size_t>(BH) * slots * 4);
    rows = base + static_cast<size_t>(BH) * slots * 4 + static_cast<size_t>(BH) * 2;
    gfirst = rows + static_cast<size_t>(BH) * n;
  }
  __host__ __device__ static size_t bytes(int BH, int n, int slots) {
    return (static_cast<size_t>(BH) * slots * 4 + static_cast<size_t>(BH) * 2 + static_cast<size_t>(BH) * n +
            static_cast<size_t>(BH) * ((n + kFixRows - 1) / kFixRows + 1)) * sizeof(int);
  }
};

// Block-wide exclusive scan of one value per thread over the 256 threads of
// the work-group; *total receives the sum.  wtot: 4 words of LDS.  Contains
// two barriers (every thread must call it).
__device__ __forceinline__ unsigned block_excl_scan(unsigned v, unsigned* wtot, unsigned* total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  unsigned x = v;  // inclusive scan over the wave
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const unsigned y = __shfl_up(x, off);
    if (lane >= off) x += y;
  }
  if (lane == 63) wtot[wave] = x;
  __syncthreads();
  unsigned base = 0, all = 0;
#pragma unroll
  for (int w = 0; w < 4; ++w) {
    if (w < wave) base += wtot[w];
    all += wtot[w];
  }
  __syncthreads();  // wtot free again
  *total = all;
  return base + x - v;
}

// Exclusive prefix counts of the set bits of the row-mask words w[0, nw):
// pre[t] = number of queued rows in words < t, pre[nw] = all of them
// (nw <= kFixMaxTiles); thread tid counts words 4 tid .. 4 tid + 3.  Every
// thread of the work-group must call it; ends with a barrier.
__device__ __forceinline__ void fix_mask_prefix(const unsigned long long* w, unsigned* pre, unsigned* wtot, int nw) {
  constexpr int P = kFixMaxTiles / 256;
  const int tid = threadIdx.x;
  unsigned c[P], sum = 0;
#pragma unroll
  for (int j = 0; j < P; ++j) {
    const int t = P * tid + j;
    c[j] = t < nw ? static_cast<unsigned>(__popcll(w[t])) : 0u;
    sum += c[j];
  }
  unsigned total;
  unsigned acc = block_excl_scan(sum, wtot, &total);
#pragma unroll
  for (int j = 0; j < P; ++j) {
    if (P * tid + j < nw) pre[P * tid + j] = acc;
    acc += c[j];
  }
  if (tid == 0) pre[nw] = total;
  __syncthreads();
}

// Row of the queued row of rank `rank` (< pre[nw]) from the masks and their
// prefix counts in LDS: the last word with pre <= rank holds it.
__device__ __forceinline__ int fix_row_of_rank(unsigned rank, const unsigned long long* w, const unsigned* pre,
                                               int nw) {
  int lo = 0, hi = nw;
  while (hi - lo > 1) {
    const int mid = (lo + hi) >> 1;
    if (pre[mid] <= rank) lo = mid; else hi = mid;
  }
  unsigned long long x = w[lo];
  for (unsigned c = pre[lo]; c < rank; ++c) x &= x - 1ull;
  return lo * 64 + __ffsll(static_cast<long long>(x)) - 1;
}

// The plan of one head per work-group.  Its queued rows are listed in row
// order.  With G groups of 32 rows and G < slots, each group's span of key
// chunks (from its first and last row and the finite-b range of the head) is
// cut into ceil(chunks / P) parts of about equal size, P the smallest part
// size (at least kFixMinPart) that fits every part of the head into the
// slots: sum_g ceil(c_g / P) <= U / P + G <= slots for P >= U / (slots - G),
// U the head's chunks.  A head with G >= slots runs its groups whole.
__global__ __launch_bounds__(256) void k_fix_plan(const unsigned* __restrict__ fix,
                                                  const unsigned long long* __restrict__ fixmask,
                                                  const int2* __restrict__ brange, int* __restrict__ plan, int BH,
                                                  int H, int n, int slots) {
  __shared__ unsigned long long smask[kFixMaxTiles];
  __shared__ unsigned spre[kFixMaxTiles + 1];
  __shared__ int gch[kFixMaxGroups], gc0[kFixMaxGroups];
  __shared__ unsigned swtot[4];
  const FixPlan P(plan, BH, n, slots);
  const int bh = blockIdx.x, tid = threadIdx.x;
  const unsigned count = fix[bh];
  const int tiles_n = (n + 63) / 64;
  for (int t = tid; t < tiles_n; t += 256) smask[t] = fixmask[static_cast<size_t>(bh) * tiles_n + t];
  __syncthreads();
  fix_mask_prefix(smask, spre, swtot, tiles_n);
  int* __restrict__ rows = P.rows + static_cast<size_t>(bh) * n;
  for (int t = tid; t < tiles_n; t += 256) {
    unsigned long long x = smask[t];
    unsigned r = spre[t];
    while (x) {
      rows[r++] = t * 64 + __ffsll(static_cast<long long>(x)) - 1;
      x &= x - 1ull;
    }
  }
  const int G = static_cast<int>((count + kFixRows - 1) / kFixRows);
  const int2 br = brange[bh % H];
  unsigned u = 0;
  for (int g = tid; g < G; g += 256) {
    const int first = fix_row_of_rank(static_cast<unsigned>(kFixRows * g), smask, spre, tiles_n);
    const int last = fix_row_of_rank(min(static_cast<unsigned>(kFixRows * g + kFixRows - 1), count - 1u), smask,
                                     spre, tiles_n);
    const int jlo = max(0, first + br.x - (n - 1)), jhi = min(n - 1, last + br.y - (n - 1));
    const int c0 = jlo / kFixKeys, nch = jhi >= jlo ? jhi / kFixKeys - c0 + 1 : 0;
    gch[g] = nch;
    gc0[g] = c0;
    u += static_cast<unsigned>(nch);
  }
  unsigned U;
  block_excl_scan(u, swtot, &U);  // (also the barrier after gch, gc0)
  if (G >= slots || G == 0) {
    if (tid == 0) P.hdr[bh] = make_int2(G, 0);
    return;
  }
  const int part = max(kFixMinPart, static_cast<int>((U + (slots - G) - 1) / static_cast<unsigned>(slots - G)));
  constexpr int GPT = kFixMaxGroups / 256;  // consecutive groups per thread
  int np[GPT];
  unsigned s = 0;
#pragma unroll
  for (int j = 0; j < GPT; ++j) {
    const int g = GPT * tid + j;
    np[j] = g < G ? max(1, (gch[g] + part - 1) / part) : 0;
    s += static_cast<unsigned>(np[j]);
  }
  unsigned total;
  unsigned acc = block_excl_scan(s, swtot, &total);
  int* __restrict__ gfirst = P.gfirst + static_cast<size_t>(bh) * P.gstride;
  int4* __restrict__ items = P.items + static_cast<size_t>(bh) * slots;
#pragma unroll
  for (int j = 0; j < GPT; ++j) {
    const int g = GPT * tid + j;
    if (g < G) {
      gfirst[g] = static_cast<int>(acc);
      const int c0 = gc0[g], nch = gch[g];
      for (int p = 0; p < np[j]; ++p)
        items[acc + p] = make_int4(g, c0 + nch * p / np[j], c0 + nch * (p + 1) / np[j], np[j]);
    }
    acc += static_cast<unsigned>(np[j]);
  }
  if (tid == 0) {
    gfirst[G] = static_cast<int>(total);
    P.hdr[bh] = make_int2(static_cast<int>(total), 1);
  }
}

// Range [lo, hi] of s = t + n - 1 where b_t is finite, per head (lo > hi if
// none), and the table cexp[h][s] = exp(b[h][s]) (c_t of Eq. (6)).
__global__ __launch_bounds__(256) void k_brange(const float* __restrict__ b, int2* __restrict__ brange,
                                                float* __restrict__ cexp, int n) {
  __shared__ int smin, smax;
  const float* __restrict__ bh = b + static_cast<size_t>(blockIdx.x) * (2 * n - 1);
  float* __restrict__ ch = cexp + static_cast<size_t>(blockIdx.x) * (2 * n - 1);
  if (threadIdx.x == 0) {
    smin = 2 * n;
    smax = -1;
  }
  __syncthreads();
  int lo = 2 * n, hi = -1;
#pragma unroll 8
  for (int sidx = threadIdx.x; sidx < 2 * n - 1; sidx += 256) {
    const float bv = bh[sidx];
    ch[sidx] = expf(bv);
    if (bv != -INFINITY) {
      lo = min(lo, sidx);
      hi = max(hi, sidx);
    }
  }
  atomicMin(&smin, lo);
  atomicMax(&smax, hi);
  __syncthreads();
  if (threadIdx.x == 0) brange[blockIdx.x] = make_int2(smin, smax);
}

template <typename TV, bool MTAIL>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(2))) void k_fixup(
    const float* __restrict__ phiq, const float* __restrict__ phik, const TV* __restrict__ vv,
    const float* __restrict__ cexp, float* __restrict__ z, float* __restrict__ den_out,
    const unsigned* __restrict__ fix, const int* __restrict__ plan, double* __restrict__ fixpart,
    const int2* __restrict__ brange, int BH, int H, int n, int ld, int d, int m, int slots) {
  extern __shared__ __align__(16) float sq[];  // phi(q) of the group's rows, [l][32], l < m rounded up to 64
  __shared__ double red[2][16][64];            // another wave's totals (two column tiles)
  __shared__ double rden[4][kFixRows];
  __shared__ int srows[kFixRows];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int lr = lane & 31, lh = lane >> 5;
  // Grid (head, batch, slot), slots counted down along z: the work-groups
  // holding a head's first items (the only ones with work when a head has
  // fewer items than slots) are dispatched before the empty ones, which
  // return at once.  (No division: the indices, and the buffer descriptors
  // built from them, stay in SGPRs; a descriptor the compiler cannot keep
  // there costs a loop around every load.)
  const int h = blockIdx.x, bh = blockIdx.y * H + h, kslot = slots - 1 - static_cast<int>(blockIdx.z);
  const FixPlan P(const_cast<int*>(plan), BH, n, slots);
  const int2 hdr = P.hdr[bh];
  const int items = hdr.x;
  const bool split = hdr.y != 0;
  // no item for this slot (its first one, slots - 1 - kslot, is the smallest)
  if (slots - 1 - kslot >= items) return;  // uniform per work-group
  const unsigned count = fix[bh];
  const int2 br = brange[h];
  const float* __restrict__ ch = cexp + static_cast<size_t>(h) * (2 * n - 1);
  const float* __restrict__ pq = phiq + static_cast<size_t>(bh) * m * ld;
  const float* __restrict__ pk = phik + static_cast<size_t>(bh) * m * ld;
  const TV* __restrict__ vh = vv + static_cast<size_t>(bh) * n * d;
  const BufRd bk(pk, static_cast<uint32_t>(m) * ld * 4u), bv(vh, static_cast<uint32_t>(n) * d * sizeof(TV));
  const BufRd bc(ch, static_cast<uint32_t>(2 * n - 1) * 4u);
  const BufRd bq(pq, static_cast<uint32_t>(m) * ld * 4u);
  // features in steps of 2 kFixL (phi(k) operands ping-pong between two
  // register sets); the operands of features m .. mr - 1 are zeros
  const int mr = (m + 2 * kFixL - 1) & ~(2 * kFixL - 1);
  const int tiles = (d + 31) / 32;
  const int* __restrict__ hrows = P.rows + static_cast<size_t>(bh) * n;

  // Items in serpentine order: round i takes the items of [i slots, (i + 1) slots)
  // counted down for even i and up for odd i: the last (under a causal mask
  // the widest) groups start first, and every work-group's total is about
  // the same.
  auto item_at = [&](int round) { return (round & 1) ? round * slots + kslot : (round + 1) * slots - 1 - kslot; };
  // {group, first chunk, end chunk, parts} (the chunks of a whole group below)
  auto describe = [&](int item) {
    return split ? P.items[static_cast<size_t>(bh) * slots + item] : make_int4(item, 0, 0, 1);
  };
  auto row_of = [&](int grp) {
    const unsigned rank = static_cast<unsigned>(grp * kFixRows + tid);
    return tid < kFixRows && rank < count ? hrows[rank] : -1;
  };
  // the item's descriptor and (lanes < 32) row, loaded during the previous item
  int4 cur = describe(item_at(0));
  int crow = row_of(cur.x);
  for (int round = 0; round * slots < items; ++round) {
    const int item = item_at(round);
    if (item >= items) continue;  // uniform per work-group
    const int nparts = cur.w;
    int cb = cur.y, ce = cur.z;
    __syncthreads();  // previous item's srows / sq / red consumed
    if (tid < kFixRows) srows[tid] = crow;
    __syncthreads();
    if (const int next = item_at(round + 1); (round + 1) * slots < items && next < items) {
      cur = describe(next);
      crow = row_of(cur.x);
    }
    int first = n, last = -1;
    for (int r = 0; r < kFixRows; ++r) {
      const int i = srows[r];
      if (i >= 0) {
        first = min(first, i);
        last = max(last, i);
      }
    }
    if (!split) {  // the group's whole span of key chunks
      const int jlo = max(0, first + br.x - (n - 1)), jhi = min(n - 1, last + br.y - (n - 1));
      cb = jlo / kFixKeys;
      ce = jhi >= jlo ? jhi / kFixKeys + 1 : cb;
    }
    {
      // thread tid stages feature rows tid / 32 + 8 k of row srows[tid % 32];
      // the rows m .. mr - 1 are zero
      const int r = tid & (kFixRows - 1), i = srows[r], l1 = tid >> 5;
      const uint32_t voff = static_cast<uint32_t>(l1 * ld + max(i, 0)) * 4u;
#pragma unroll 8
      for (int l = l1; l < m; l += 256 / kFixRows) {
        const float x = bq.f32(voff, static_cast<uint32_t>((l - l1) * ld) * 4u);
        sq[l * kFixRows + r] = i >= 0 ? x : 0.f;
      }
      for (int l = m + l1; l < mr; l += 256 / kFixRows) sq[l * kFixRows + r] = 0.f;
    }
    const int myrow = srows[lr];  // the query row of this lane in S^T and P
    __syncthreads();              // sq staged

    // column tiles of [v]: two per pass (the S^T products are recomputed for
    // a second pass when d > 64)
    for (int t0 = 0; t0 < tiles; t0 += 2) {
      double zt[2][16];
      double dsum = 0.0;
#pragma unroll
      for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int e = 0; e < 16; ++e) zt[t][e] = 0.0;
      // phi(k) operands of one 32-feature step: A[key jc + lr][feature l0 + 2 q + lh],
      // two sets: a step multiplies one while the other is loaded.  Keys past
      // n read key n - 1 (masked in P).  The buffer range check covers the
      // lane (VGPR) offset only: when m is not a multiple of 64 (MTAIL) the
      // feature offset goes into the lane offset too, so the rows past m read
      // zero.
      float ka[kFixL / 2], kc[kFixL / 2];
      auto load_k = [&](float (&dst)[kFixL / 2], int jc, int l0) {
        uint32_t voff = static_cast<uint32_t>(lh * ld + min(jc + lr, n - 1)) * 4u;
        if constexpr (MTAIL) {
          // (opaque: the 16 sums are formed per step, not kept live across steps)
          voff += static_cast<uint32_t>(l0 * ld) * 4u;
          asm volatile("" : "+v"(voff));
        }
#pragma unroll
        for (int q = 0; q < kFixL / 2; ++q) {
          const uint32_t fo = static_cast<uint32_t>((MTAIL ? 2 * q : l0 + 2 * q) * ld) * 4u;
          dst[q] = MTAIL ? bk.f32(voff + fo, 0u) : bk.f32(voff, fo);
        }
      };
      auto s_step = [&](const float (&kk)[kFixL / 2], int l0, floatx16& acc) {
#pragma unroll
        for (int q = 0; q < kFixL / 2; ++q) {
          const float qb = sq[(l0 + 2 * q + lh) * kFixRows + lr];
          acc = __builtin_amdgcn_mfma_f32_32x32x2f32(kk[q], qb, acc, 0, 0, 0);
        }
      };
      int jc = cb * kFixKeys + 32 * wave;
      if (jc < ce * kFixKeys) load_k(ka, jc, 0);
      for (; jc < ce * kFixKeys; jc += kFixKeys) {
        // value rows of these 32 keys, in the key order of the P V steps:
        // step e uses key jc + 8 (e / 4) + 4 lh + e % 4 on lane half lh
        // (columns >= d are masked).  In the last block of a sequence whose
        // length is not a multiple of 32 the row offset goes into the
        // range-checked lane offset: rows past n read zero.
        const bool full = jc + 32 <= n;  // uniform
        float vb[2][16];
        auto load_v = [&](auto tail) {
#pragma unroll
          for (int t = 0; t < 2; ++t) {
            const int col = (t0 + t) * 32 + lr;
            const uint32_t voff = static_cast<uint32_t>((jc + 4 * lh) * d + min(col, d - 1)) * sizeof(TV);
#pragma unroll
            for (int e = 0; e < 16; ++e) {
              const uint32_t eoff = static_cast<uint32_t>((8 * (e >> 2) + (e & 3)) * d) * sizeof(TV);
              const uint32_t vo = decltype(tail)::value ? voff + eoff : voff;
              const uint32_t so = decltype(tail)::value ? 0u : eoff;
              float x;
              if constexpr (sizeof(TV) == 2) {
                x = to_f32(bv.u16(vo, so));
              } else {
                x = bv.f32(vo, so);
              }
              vb[t][e] = col < d ? x : 0.f;
            }
          }
        };
        if (full) {
          load_v(std::false_type{});
        } else {
          load_v(std::true_type{});
        }
        // ---- S^T[key][row] over the m features
        floatx16 sacc;
#pragma unroll
        for (int e = 0; e < 16; ++e) sacc[e] = 0.f;
        for (int l0 = 0; l0 < mr; l0 += 2 * kFixL) {
          load_k(kc, jc, l0 + kFixL);
          s_step(ka, l0, sacc);
          if (l0 + 2 * kFixL < mr) {
            load_k(ka, jc, l0 + 2 * kFixL);
          } else if (jc + kFixKeys < ce * kFixKeys) {
            load_k(ka, jc + kFixKeys, 0);  // the next key block's first step
          }
          s_step(kc, l0 + kFixL, sacc);
        }
        // ---- P = S^T c_{j-i}: lane holds keys jc + 8 (e / 4) + 4 lh + e % 4 of row myrow
        // (index key - row + n - 1 lies in [0, 2n - 2] for keys < n; a lane
        // without a row reads row 0's entries, masked below; past n as for v)
        float pv[16];
        float ds = 0.f;
        const uint32_t coff = static_cast<uint32_t>(jc + 4 * lh - max(myrow, 0) + n - 1) * 4u;
        float cv[16];
        if (full) {
#pragma unroll
          for (int e = 0; e < 16; ++e) cv[e] = bc.f32(coff, static_cast<uint32_t>(8 * (e >> 2) + (e & 3)) * 4u);
        } else {
#pragma unroll
          for (int e = 0; e < 16; ++e) cv[e] = bc.f32(coff + static_cast<uint32_t>(8 * (e >> 2) + (e & 3)) * 4u, 0u);
        }
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const int key = jc + 8 * (e >> 2) + 4 * lh + (e & 3);
          pv[e] = (myrow >= 0 && key < n) ? sacc[e] * cv[e] : 0.f;
          ds += pv[e];
        }
        dsum += static_cast<double>(ds);
        // ---- Z[row][col] += sum_key P[row][key] v[key][col]
#pragma unroll
        for (int t = 0; t < 2; ++t) {
          if (t0 + t < tiles) {
            floatx16 zc;
#pragma unroll
            for (int e = 0; e < 16; ++e) zc[e] = 0.f;
#pragma unroll
            for (int e = 0; e < 16; ++e) zc = __builtin_amdgcn_mfma_f32_32x32x2f32(pv[e], vb[t][e], zc, 0, 0, 0);
#pragma unroll
            for (int e = 0; e < 16; ++e) zt[t][e] += static_cast<double>(zc[e]);
          }
        }
      }
      // ---- the four waves' totals, added in wave order
      dsum += __shfl_xor(dsum, 32);  // the other half-wave's keys of row lr
      if (t0 == 0 && lh == 0) rden[wave][lr] = dsum;
      for (int w = 1; w < 4; ++w) {
        __syncthreads();
        if (wave == w) {
#pragma unroll
          for (int t = 0; t < 2; ++t)
#pragma unroll
            for (int e = 0; e < 16; ++e) red[t][e][lane] = zt[t][e];
        }
        __syncthreads();
        if (wave == 0) {
#pragma unroll
          for (int t = 0; t < 2; ++t)
#pragma unroll
            for (int e = 0; e < 16; ++e) zt[t][e] += red[t][e][lane];
        }
      }
      __syncthreads();
      // wave 0 holds the totals: row 8 (e / 4) + 4 lh + e % 4, column (t0 + t) 32 + lr
      if (wave == 0) {
        double* __restrict__ out =
            nparts == 1 ? nullptr : fixpart + (static_cast<size_t>(bh) * slots + item) * kFixRows * (d + 1);
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const int row = 8 * (e >> 2) + 4 * lh + (e & 3);
          const int i = srows[row];
          const double den = ((rden[0][row] + rden[1][row]) + rden[2][row]) + rden[3][row];
#pragma unroll
          for (int t = 0; t < 2; ++t) {
            const int col = (t0 + t) * 32 + lr;
            if (i < 0 || t0 + t >= tiles || col >= d) continue;
            if (nparts == 1) {
              z[(static_cast<size_t>(bh) * n + i) * d + col] = static_cast<float>(zt[t][e] / den);
            } else {
              out[row * (d + 1) + col] = zt[t][e];
            }
          }
          if (t0 == 0 && lr == 0) {
            if (nparts == 1) {
              if (den_out && i >= 0) den_out[static_cast<size_t>(bh) * n + i] = static_cast<float>(den);
            } else {
              out[row * (d + 1) + d] = den;
            }
          }
        }
      }
    }
  }
}

// Sums the parts of every group k_fixup split (in part order, so the result
// is deterministic) and writes the rows.  Work-group (bh, slot) takes groups
// slot, slot + slots, ...
__global__ __launch_bounds__(256) void k_fixup_combine(const unsigned* __restrict__ fix, const int* __restrict__ plan,
                                                       const double* __restrict__ fixpart, float* __restrict__ z,
                                                       float* __restrict__ den_out, int BH, int n, int d, int slots) {
  __shared__ int srows[kFixRows];
  const int bh = blockIdx.x % BH, kslot = blockIdx.x / BH;
  const FixPlan P(const_cast<int*>(plan), BH, n, slots);
  const int2 hdr = P.hdr[bh];
  const unsigned count = fix[bh];
  const int ngroups = static_cast<int>((count + kFixRows - 1) / kFixRows);
  if (hdr.y == 0 || kslot >= ngroups) return;
  const int tid = threadIdx.x;
  const int* __restrict__ gfirst = P.gfirst + static_cast<size_t>(bh) * P.gstride;
  for (int grp = kslot; grp < ngroups; grp += slots) {
    const int first = gfirst[grp], nparts = gfirst[grp + 1] - first;
    if (nparts == 1) continue;  // written by k_fixup
    __syncthreads();
    if (tid < kFixRows) {
      const unsigned rank = static_cast<unsigned>(grp * kFixRows + tid);
      srows[tid] = rank < count ? P.rows[static_cast<size_t>(bh) * n + rank] : -1;
    }
    __syncthreads();
    const double* __restrict__ base = fixpart + (static_cast<size_t>(bh) * slots + first) * kFixRows * (d + 1);
    for (int e = tid; e < kFixRows * d; e += 256) {
      const int row = e / d, c = e % d;
      const int i = srows[row];
      if (i < 0) continue;
      double num = 0.0, den = 0.0;
      for (int p = 0; p < nparts; ++p) {
        const double* part = base + static_cast<size_t>(p) * kFixRows * (d + 1) + row * (d + 1);
        num += part[c];
        den += part[d];
      }
      z[(static_cast<size_t>(bh) * n + i) * d + c] = static_cast<float>(num / den);
      if (den_out && c == 0) den_out[static_cast<size_t>(bh) * n + i] = static_cast<float>(den);
    }
  }
}

// Direct route with at most 128 features: every row of every head, one wave
// per 32 query rows.  A work-group holds 128 consecutive rows of one
// (batch, head), each wave its own 32 (phi(q) of them staged in LDS), and
// each wave walks every key block of 32 in its rows' finite-b range with the
// products of k_fixup:
//   S^T = phi(k_keys) phi(q_rows)^T, P = S^T * c_{j-i}, Z += P^T [v, ...]
// (fp32 MFMA; per 32 keys the fp32 sums added into fp64 totals, blocks in
// key order), then writes its rows.  No wave shares a row, so there is no
// reduction across waves and no plan.  Work-groups take the row tiles from
// the last one down: under a causal mask the last rows see the most keys.
constexpr int kDirRows = 4 * kFixRows;  // rows per work-group

template <bool MTAIL>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(2))) void k_direct_rows(
    const float* __restrict__ phiq, const float* __restrict__ phik, const float* __restrict__ vv,
    const float* __restrict__ cexp, float* __restrict__ z, float* __restrict__ den_out,
    const int2* __restrict__ brange, int H, int n, int ld, int d, int m) {
  extern __shared__ __align__(16) float sqw[];  // [wave][l][32], l < m rounded up to 64
  __shared__ double wden[4][kFixRows];
  // (the wave index read from the first lane: the compiler then knows it,
  // and every row and key bound derived from it, to be wave-uniform, so the
  // key-block loop runs on scalar registers and branches)
  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int lr = lane & 31, lh = lane >> 5;
  const int ntile = (n + kDirRows - 1) / kDirRows;
  const int tile = ntile - 1 - static_cast<int>(blockIdx.x);
  const int h = blockIdx.z, bh = blockIdx.y * H + h;  // grid (row tile, batch, head): no division
  const int row0 = tile * kDirRows + kFixRows * wave;
  const int mr = (m + 2 * kFixL - 1) & ~(2 * kFixL - 1);
  float* __restrict__ sq = sqw + wave * mr * kFixRows;
  const float* __restrict__ pq = phiq + static_cast<size_t>(bh) * m * ld;
  const float* __restrict__ pk = phik + static_cast<size_t>(bh) * m * ld;
  const float* __restrict__ vh = vv + static_cast<size_t>(bh) * n * d;
  const float* __restrict__ ch = cexp + static_cast<size_t>(h) * (2 * n - 1);
  const BufRd bk(pk, static_cast<uint32_t>(m) * ld * 4u), bv(vh, static_cast<uint32_t>(n) * d * 4u);
  const BufRd bc(ch, static_cast<uint32_t>(2 * n - 1) * 4u), bq(pq, static_cast<uint32_t>(m) * ld * 4u);
  // this wave's rows' phi(q): lane stages feature rows lane / 32 + 2 k of row
  // row0 + lane % 32 (zero past m and past n)
  {
    const int r = lr, i = row0 + r, l1 = lh;
    const uint32_t voff = static_cast<uint32_t>(l1 * ld + min(i, n - 1)) * 4u;
#pragma unroll 8
    for (int l = l1; l < m; l += 2) {
      const float x = bq.f32(voff, static_cast<uint32_t>((l - l1) * ld) * 4u);
      sq[l * kFixRows + r] = i < n ? x : 0.f;
    }
    for (int l = m + l1; l < mr; l += 2) sq[l * kFixRows + r] = 0.f;
  }
  __syncthreads();  // (each wave reads only its own rows; one barrier orders the stores)
  if (row0 >= n) return;  // uniform per wave; no barrier follows
  const int myrow = row0 + lr < n ? row0 + lr : -1;
  const int last = min(row0 + kFixRows, n) - 1;
  const int2 br = brange[h];
  const int jlo = max(0, row0 + br.x - (n - 1)), jhi = min(n - 1, last + br.y - (n - 1));
  const int tiles = (d + 31) / 32;
  for (int t0 = 0; t0 < tiles; t0 += 2) {
    double zt[2][16];
    double dsum = 0.0;
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
      for (int e = 0; e < 16; ++e) zt[t][e] = 0.0;
    // phi(k) operands as in k_fixup: A[key jc + lr][feature l0 + 2 q + lh], two
    // register sets over 32-feature steps; keys past n read key n - 1 (masked
    // in P); with MTAIL the feature offset is range-checked (zeros past m)
    float ka[kFixL / 2], kc[kFixL / 2];
    auto load_k = [&](float (&dst)[kFixL / 2], int jc, int l0) {
      uint32_t voff = static_cast<uint32_t>(lh * ld + min(jc + lr, n - 1)) * 4u;
      if constexpr (MTAIL) {
        voff += static_cast<uint32_t>(l0 * ld) * 4u;
        asm volatile("" : "+v"(voff));
      }
#pragma unroll
      for (int q = 0; q < kFixL / 2; ++q) {
        const uint32_t fo = static_cast<uint32_t>((MTAIL ? 2 * q : l0 + 2 * q) * ld) * 4u;
        dst[q] = MTAIL ? bk.f32(voff + fo, 0u) : bk.f32(voff, fo);
      }
    };
    auto s_step = [&](const float (&kk)[kFixL / 2], int l0, floatx16& acc) {
#pragma unroll
      for (int q = 0; q < kFixL / 2; ++q) {
        const float qb = sq[(l0 + 2 * q + lh) * kFixRows + lr];
        acc = __builtin_amdgcn_mfma_f32_32x32x2f32(kk[q], qb, acc, 0, 0, 0);
      }
    };
    const int jend = jhi >= jlo ? jhi + 1 : 0;
    int jc = jlo & ~31;
    if (jc < jend) load_k(ka, jc, 0);
    for (; jc < jend; jc += 32) {
      const bool full = jc + 32 <= n;  // uniform
      float vb[2][16];
      auto load_v = [&](auto tail) {
#pragma unroll
        for (int t = 0; t < 2; ++t) {
          const int col = (t0 + t) * 32 + lr;
          const uint32_t voff = static_cast<uint32_t>((jc + 4 * lh) * d + min(col, d - 1)) * 4u;
#pragma unroll
          for (int e = 0; e < 16; ++e) {
            const uint32_t eoff = static_cast<uint32_t>((8 * (e >> 2) + (e & 3)) * d) * 4u;
            // (a column past d reads column d - 1: it feeds only columns of Z
            // that are not stored)
            vb[t][e] = decltype(tail)::value ? bv.f32(voff + eoff, 0u) : bv.f32(voff, eoff);
          }
        }
      };
      if (full) {
        load_v(std::false_type{});
      } else {
        load_v(std::true_type{});
      }
      // the c-table entries of these keys (P below), loaded ahead of the S
      // product so that their latency passes under it
      const uint32_t coff = static_cast<uint32_t>(jc + 4 * lh - max(myrow, 0) + n - 1) * 4u;
      float cv[16];
      if (full) {
#pragma unroll
        for (int e = 0; e < 16; ++e) cv[e] = bc.f32(coff, static_cast<uint32_t>(8 * (e >> 2) + (e & 3)) * 4u);
      } else {
#pragma unroll
        for (int e = 0; e < 16; ++e) cv[e] = bc.f32(coff + static_cast<uint32_t>(8 * (e >> 2) + (e & 3)) * 4u, 0u);
      }
      floatx16 sacc;
#pragma unroll
      for (int e = 0; e < 16; ++e) sacc[e] = 0.f;
      for (int l0 = 0; l0 < mr; l0 += 2 * kFixL) {
        load_k(kc, jc, l0 + kFixL);
        s_step(ka, l0, sacc);
        if (l0 + 2 * kFixL < mr) {
          load_k(ka, jc, l0 + 2 * kFixL);
        } else if (jc + 32 < jend) {
          load_k(ka, jc + 32, 0);  // the next key block's first step
        }
        s_step(kc, l0 + kFixL, sacc);
      }
      // P = S^T c_{j-i}, lane: keys jc + 8 (e / 4) + 4 lh + e % 4 of row myrow.
      // A lane without a row (past n) has S = 0 (its phi(q) is staged as
      // zeros) and its P, sums and totals are never stored, so only keys
      // past n, in the last block, are masked: there v reads zero but the
      // denominator would take them.
      float pv[16];
      float ds = 0.f;
      if (full) {
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          pv[e] = sacc[e] * cv[e];
          ds += pv[e];
        }
      } else {
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const int key = jc + 8 * (e >> 2) + 4 * lh + (e & 3);
          pv[e] = key < n ? sacc[e] * cv[e] : 0.f;
          ds += pv[e];
        }
      }
      dsum += static_cast<double>(ds);
#pragma unroll
      for (int t = 0; t < 2; ++t) {
        if (t0 + t < tiles) {
          floatx16 zc;
#pragma unroll
          for (int e = 0; e < 16; ++e) zc[e] = 0.f;
#pragma unroll
          for (int e = 0; e < 16; ++e) zc = __builtin_amdgcn_mfma_f32_32x32x2f32(pv[e], vb[t][e], zc, 0, 0, 0);
#pragma unroll
          for (int e = 0; e < 16; ++e) zt[t][e] += static_cast<double>(zc[e]);
        }
      }
    }
    // row lr's denominator: this half-wave's keys plus the other half's
    dsum += __shfl_xor(dsum, 32);
    if (lh == 0) wden[wave][lr] = dsum;
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    // lane holds rows 8 (e / 4) + 4 lh + e % 4, column (t0 + t) 32 + lr
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      const int row = 8 * (e >> 2) + 4 * lh + (e & 3), i = row0 + row;
      const double den = wden[wave][row];
#pragma unroll
      for (int t = 0; t < 2; ++t) {
        const int col = (t0 + t) * 32 + lr;
        if (i < n && t0 + t < tiles && col < d)
          z[(static_cast<size_t>(bh) * n + i) * d + col] = static_cast<float>(zt[t][e] / den);
      }
      if (t0 == 0 && lr == 0 && den_out && i < n) den_out[static_cast<size_t>(bh) * n + i] = static_cast<float>(den);
    }
    __builtin_amdgcn_wave_barrier();  // wden read before the next pass writes it
  }
}

// Direct (quadratic) route: every row of every head queued for k_fixup, which
// then evaluates Eq. (10) as S = phi(Q) phi(K)^T o C and S [v, 1] on MFMA.
// fixmask[bh][t] holds the bits of the rows < n of tile t; fix[bh] = n,
// fix[BH] = BH n.
__global__ void k_mark_all(unsigned* __restrict__ fix, unsigned long long* __restrict__ fixmask, int BH, int n,
                           int tiles_n) {
  const long long e = static_cast<long long>(blockIdx.x) * blockDim.x + threadIdx.x;
  const long long words = static_cast<long long>(BH) * tiles_n;
  if (e < words) {
    const int t = static_cast<int>(e % tiles_n);
    const int rows = min(64, n - 64 * t);
    fixmask[e] = rows >= 64 ? ~0ull : ((1ull << rows) - 1ull);
  }
  if (e < BH) fix[e] = static_cast<unsigned>(n);
  if (e == BH) fix[BH] = static_cast<unsigned>(BH) * static_cast<unsigned>(n);
}

// dst[e] = bf16 src[e] widened to fp32 (exact), so that the direct route's
// value loads are 4-byte and coalesced like the fp32 ones.
__global__ void k_widen_bf16(const uint16_t* __restrict__ src, float* __restrict__ dst, long long count) {
  const long long e = static_cast<long long>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (e < count) dst[e] = to_f32(src[e]);
}

// ------------------------------------------------------ Toeplitz helpers --
// ones[pos] = 1 for pos < n, 0 below N: the broadcast "feature" with which the
// convolution kernel computes plain Toeplitz products (m = 1, phi = 1).
__global__ void k_ones(float* __restrict__ ones, int n, int N) {
  const int pos = blockIdx.x * blockDim.x + threadIdx.x;
  if (pos < N) ones[pos] = pos < n ? 1.f : 0.f;
}

// y[bh][c][i] = sum_s part[bh][s][c][i]
__global__ void k_sum_splits(const float* __restrict__ part, float* __restrict__ y, int C, int n, int ldy,
                             int nsplit, long long total) {
  const long long e = static_cast<long long>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (e >= total) return;
  const long long per = static_cast<long long>(C) * n;
  const long long bh = e / per, r = e % per;
  const long long row = bh * C + r / n, i = r % n;  // output row (bh, c) and position
  // independent loads in flight (sums in split order, as a plain loop)
  const float* __restrict__ p = part + bh * nsplit * per + r;
  float s = 0.f;
  int sp = 0;
  for (; sp + 4 <= nsplit; sp += 4) {
    const float a0 = p[sp * per], a1 = p[(sp + 1) * per], a2 = p[(sp + 2) * per], a3 = p[(sp + 3) * per];
    s = (((s + a0) + a1) + a2) + a3;
  }
  for (; sp < nsplit; ++sp) s += p[sp * per];
  y[row * ldy + i] = s;
}

// ============================================================= backward ==
// Gradients of L = <G, z> through Eq. (10) with the feature map of Eq. (5), W
// fixed.  With A = C o (Phi_q Phi_k^T) (C_ij = c_{j-i}), den = A 1 and
// z = (A v) / den, the gradient of L with respect to [numerator, denominator]
// of row i is Gh_i = [G_i / den_i, -(G_i . z_i) / den_i], and with
// V' = [v, 1] (Eq. (11)'s channels):
//   dv      = A^T Gh[:, :d]:   dv_j      = sum_l phi_l(k_j) (C^T (phi_l(q) o Gh_c))_j
//   dPhi_q  = (Gh V'^T o C) Phi_k:  dphi_l(q_i) = sum_c Gh_ic (C (V'_c o phi_l(k)))_i
//   dPhi_k  = (Gh V'^T o C)^T Phi_q:  dphi_l(k_j) = sum_c V'_jc (C^T (Gh_c o phi_l(q)))_j
// Each is the product the forward convolution kernel computes,
// sum_f f_f o C (a_f o col), with the roles of features and columns
// assigned as written (C^T is the Toeplitz matrix of the reversed b).

// Gh and V' feature-major ([bh][c][pos], c <= d, zero for n <= pos < N), from
// G, the forward's z and den, and v.  Block: 64 positions of one (batch, head).
template <typename TV>
__global__ __launch_bounds__(256) void k_bwd_prep(const float* __restrict__ G, const float* __restrict__ z,
                                                  const float* __restrict__ den, const TV* __restrict__ v,
                                                  float* __restrict__ Gh, float* __restrict__ Vh, int n, int N,
                                                  int d, int tiles) {
  __shared__ float gs[64][kMaxD + 1];
  __shared__ float rden[64], dden[64];
  const int bh = blockIdx.x / tiles, i0 = (blockIdx.x % tiles) * 64;
  const int tid = threadIdx.x;
  const float* __restrict__ Gb = G + static_cast<size_t>(bh) * n * d;
  const float* __restrict__ zb = z + static_cast<size_t>(bh) * n * d;
  const TV* __restrict__ vb = v + static_cast<size_t>(bh) * n * d;
  for (int e = tid; e < 64 * d; e += 256) {
    const int r = e / d, c = e - r * d, pos = i0 + r;
    gs[r][c] = pos < n ? Gb[static_cast<size_t>(pos) * d + c] : 0.f;
  }
  __syncthreads();
  if (tid < 64) {
    const int pos = i0 + tid;
    float dot = 0.f, inv = 0.f;
    if (pos < n) {
      inv = 1.0f / den[static_cast<size_t>(bh) * n + pos];
      for (int c = 0; c < d; ++c) dot = fmaf(gs[tid][c], zb[static_cast<size_t>(pos) * d + c], dot);
    }
    rden[tid] = inv;
    dden[tid] = -dot * inv;
  }
  __syncthreads();
  for (int e = tid; e < (d + 1) * 64; e += 256) {
    const int c = e >> 6, r = e & 63, pos = i0 + r;
    if (pos >= N) continue;
    float gv = 0.f, vv = 0.f;
    if (pos < n) {
      gv = c < d ? gs[r][c] * rden[r] : dden[r];
      vv = c < d ? to_f32(vb[static_cast<size_t>(pos) * d + c]) : 1.f;
    }
    const size_t o = (static_cast<size_t>(bh) * (d + 1) + c) * N + pos;
    Gh[o] = gv;
    Vh[o] = vv;
  }
}

// brev[h][s] = b[h][2n - 2 - s]: the bias of the transposed Toeplitz matrix.
__global__ void k_reverse_bias(const float* __restrict__ b, float* __restrict__ brev, int n, int H) {
  const long long e = static_cast<long long>(blockIdx.x) * blockDim.x + threadIdx.x;
  const long long len = 2LL * n - 1;
  if (e >= len * H) return;
  const long long h = e / len, s = e - h * len;
  brev[e] = b[h * len + (len - 1 - s)];
}

// dv[bh][i][c] = sum_s part[bh][s][c][i] for c < d: the class splits of the
// convolution kernel's output summed and transposed.  Block: 64 positions.
__global__ __launch_bounds__(256) void k_bwd_dv(const float* __restrict__ part, float* __restrict__ dv, int n,
                                                int d, int cols, int nsplit, int tiles) {
  __shared__ float t[64][kMaxD + 1];
  const int bh = blockIdx.x / tiles, i0 = (blockIdx.x % tiles) * 64;
  for (int e = threadIdx.x; e < d * 64; e += 256) {
    const int c = e >> 6, r = e & 63, pos = i0 + r;
    float acc = 0.f;
    if (pos < n)
      for (int sp = 0; sp < nsplit; ++sp) acc += part[((static_cast<size_t>(bh) * nsplit + sp) * cols + c) * n + pos];
    t[r][c] = acc;
  }
  __syncthreads();
  for (int e = threadIdx.x; e < d * 64; e += 256) {
    const int r = e / d, c = e - r * d, pos = i0 + r;
    if (pos < n) dv[(static_cast<size_t>(bh) * n + pos) * d + c] = t[r][c];
  }
}

// Feature-map backward for Eq. (5): d phi_l / dx = phi_l (w_l - x), so
//   dx = sum_l P_l w_l - x sum_l P_l,   P_l = dphi_l phi_l,
// and with row normalisation (x = u / |u|, Algorithm 1) du = (dx - x (x . dx)) / |u|
// (0 for a zero row).  dphi is summed over the nsplit class splits of the
// convolution kernel's output part[bh][s][l][i]; phi is feature-major [bh][l][N].
// Block: 64 positions of one (batch, head); wave w accumulates the columns
// a = w, w + 4, ...; features staged through LDS 32 at a time.
template <typename TX>
__global__ __launch_bounds__(256) void k_feature_bwd(const TX* __restrict__ x, const float* __restrict__ W,
                                                     const float* __restrict__ phi, const float* __restrict__ part,
                                                     float* __restrict__ dx, int H, int n, int N, int d, int m,
                                                     int nsplit, int nprf, int tiles) {
  constexpr int KC = 32, ACC = kMaxD / 4;
  __shared__ float Ps[KC][64];
  __shared__ float Ws[KC][kMaxD];
  __shared__ float red[4][64];
  const int bh = blockIdx.x / tiles, i0 = (blockIdx.x % tiles) * 64, h = bh % H;
  const int tid = threadIdx.x, r = tid & 63, w = tid >> 6;
  const int i = i0 + r;
  // wave w owns the cpw contiguous columns w cpw .. (cpw a multiple of 4, so
  // the weights are read as float4, one LDS read per four products)
  const int cpw = ((d + 3) / 4 + 3) / 4 * 4, cbase = w * cpw;
  float acc[ACC];
#pragma unroll
  for (int j = 0; j < ACC; ++j) acc[j] = 0.f;
  float rs = 0.f;
  for (int l0 = 0; l0 < m; l0 += KC) {
    __syncthreads();
    for (int e = tid; e < KC * 64; e += 256) {
      const int lq = e >> 6, rr = e & 63, l = l0 + lq, pos = i0 + rr;
      float p = 0.f;
      if (l < m && pos < n) {
        float dp = 0.f;
        for (int sp = 0; sp < nsplit; ++sp) dp += part[((static_cast<size_t>(bh) * nsplit + sp) * m + l) * n + pos];
        p = dp * phi[(static_cast<size_t>(bh) * m + l) * N + pos];
      }
      Ps[lq][rr] = p;
    }
    // columns past d (up to the waves' 4 cpw) zero: they meet the
    // discarded accumulators only, which must stay finite
    for (int e = tid; e < KC * 4 * cpw; e += 256) {
      const int lq = e / (4 * cpw), a = e - lq * (4 * cpw), l = l0 + lq;
      Ws[lq][a] = (l < m && a < d) ? W[(static_cast<size_t>(h) * m + l) * d + a] : 0.f;
    }
    __syncthreads();
    for (int lq = 0; lq < KC; ++lq) {
      const float p = Ps[lq][r];
      rs += p;
#pragma unroll
      for (int q = 0; q < ACC / 4; ++q) {
        if (4 * q < cpw) {
          const float4 wv = *reinterpret_cast<const float4*>(&Ws[lq][cbase + 4 * q]);
          acc[4 * q] = fmaf(p, wv.x, acc[4 * q]);
          acc[4 * q + 1] = fmaf(p, wv.y, acc[4 * q + 1]);
          acc[4 * q + 2] = fmaf(p, wv.z, acc[4 * q + 2]);
          acc[4 * q + 3] = fmaf(p, wv.w, acc[4 * q + 3]);
        }
      }
    }
  }
  // x of the row (normalised when asked) and its norm
  float xa[ACC];
  float sq = 0.f;
#pragma unroll
  for (int j = 0; j < ACC; ++j) {
    const int a = cbase + j;
    xa[j] = (j < cpw && a < d && i < n) ? to_f32(x[(static_cast<size_t>(bh) * n + i) * d + a]) : 0.f;
    sq = fmaf(xa[j], xa[j], sq);
  }
  red[w][r] = sq;
  __syncthreads();
  sq = red[0][r] + red[1][r] + red[2][r] + red[3][r];
  const float scale = nprf ? (sq > 0.f ? rsqrtf(sq) : 0.f) : 1.f;
  float dot = 0.f;
#pragma unroll
  for (int j = 0; j < ACC; ++j) {
    xa[j] *= scale;                   // the x phi was taken of
    acc[j] = acc[j] - xa[j] * rs;     // dL/dx
    dot = fmaf(xa[j], acc[j], dot);
  }
  if (nprf) {
    __syncthreads();
    red[w][r] = dot;
    __syncthreads();
    dot = red[0][r] + red[1][r] + red[2][r] + red[3][r];
#pragma unroll
    for (int j = 0; j < ACC; ++j) acc[j] = (acc[j] - xa[j] * dot) * scale;
  }
  if (i < n) {
#pragma unroll
    for (int j = 0; j < ACC; ++j) {
      const int a = cbase + j;
      if (j < cpw && a < d) dx[(static_cast<size_t>(bh) * n + i) * d + a] = acc[j];
    }
  }
}

// ============================================================ launchers ==
namespace {

template <int L2>
hipError_t spectrum_l2(const float* b, const float2* tw, float2* Hs, float2* hnorm, int H, int n, hipStream_t st) {
  using C = Conf<L2>;
  const int blocks = (C::S * H + C::G - 1) / C::G;
  hipLaunchKernelGGL(k_spectrum<L2>, dim3(blocks), dim3(C::THREADS), 0, st, b, tw, Hs, hnorm, H, n);
  return hipGetLastError();
}

template <int L2>
hipError_t conv_l2(const float* phiq, const float* phik, long long phi_bh_stride, const float2* vsc,
                   const float* colmax, const float2* Hs, const float2* hnorm, const float2* tw, float* part, int BH,
                   int H, int n, int cols, int m, int nkb, int fsplit, hipStream_t st) {
  if constexpr (L2 == kMaxLog2N) {
    return conv_launch_top(phiq, phik, phi_bh_stride, vsc, colmax, Hs, hnorm, tw, part, BH, H, n, cols, m, nkb,
                           fsplit, st);
  } else {
    return conv_launch<L2>(phiq, phik, phi_bh_stride, vsc, colmax, Hs, hnorm, tw, part, BH, H, n, cols, m, nkb,
                           fsplit, st);
  }
}

// Run-time dispatch on log2 N over the compiled lengths 2^0 .. 2^kMaxLog2N.
template <template <int> class Fn, int L2 = 0, typename... Args>
hipError_t dispatch(int l2, Args... args) {
  if constexpr (L2 > kMaxLog2N) {
    return hipErrorInvalidValue;
  } else {
    if (l2 == L2) return Fn<L2>::run(args...);
    return dispatch<Fn, L2 + 1>(l2, args...);
  }
}
template <int L2>
struct SpectrumFn {
  template <typename... A>
  static hipError_t run(A... a) { return spectrum_l2<L2>(a...); }
};
template <int L2>
struct ConvFn {
  template <typename... A>
  static hipError_t run(A... a) { return conv_l2<L2>(a...); }
};
template <int L2>
struct TwExtFn {
  static hipError_t run(float2* tw, int extra, hipStream_t st) {
    hipLaunchKernelGGL(k_twiddles_ext<L2>, dim3((extra + 255) / 256), dim3(256), 0, st, tw);
    return hipGetLastError();
  }
};
template <int L2>
struct TableFn {
  static hipError_t run(int* out) {
    *out = Conf<L2>::TWC ? Conf<L2>::F::TABLE : 2 * Conf<L2>::N;
    return hipSuccess;
  }
};
template <int L2>
struct SplitFn {
  static hipError_t run(int* out) {
    *out = Conf<L2>::HSPLIT;
    return hipSuccess;
  }
};

}  // namespace

int twiddle_slots(int l2) {
  int t = 2 << l2;
  (void)dispatch<TableFn>(l2, &t);
  return t;
}

int conv_splits(int l2) {
  int s = 2;
  (void)dispatch<SplitFn>(l2, &s);
  return s;
}

int gram_splits(int BH, int m, int N) {
  // enough blocks to fill the GPU, slices of at least 1024 positions
  const int ltiles = (m + kGramL - 1) / kGramL;
  int ks = 1;
  while (ks < 16 && static_cast<long long>(BH) * ltiles * ks < 1024 && N / (2 * ks) >= 1024) ks *= 2;
  return ks;
}

hipError_t launch_twiddles(float2* tw, int l2, hipStream_t st) {
  const int count = 2 << l2;
  hipLaunchKernelGGL(k_twiddles, dim3((count + 255) / 256), dim3(256), 0, st, tw, l2);
  if (hipError_t e = hipGetLastError(); e != hipSuccess) return e;
  const int extra = twiddle_slots(l2) - count;
  if (extra > 0) {
    if (hipError_t e = dispatch<TwExtFn>(l2, tw, extra, st); e != hipSuccess) return e;
  }
  return hipGetLastError();
}

hipError_t launch_spectrum(int l2, const float* b, const float2* tw, float2* Hs, float2* hnorm, int H, int n,
                           hipStream_t st) {
  return dispatch<SpectrumFn>(l2, b, tw, Hs, hnorm, H, n, st);
}

hipError_t launch_feature_map(bool bf16, const void* x0, const void* x1, const float* W, float* phi0, float* phi1,
                              int nsrc, bool feature_major, int ld, int BH, int H, int n, int d, int m,
                              unsigned* fix_counts, bool nprf, int kind, hipStream_t st) {
  const int rows = feature_major ? ld : n;
  const int tiles_n = (rows + 63) / 64;
  const dim3 block(256);
  if (kind == kFeatElu) {
    const dim3 grid(static_cast<unsigned>(static_cast<long long>(tiles_n) * BH * nsrc));
    const int np = nprf ? 1 : 0;
    if (bf16) {
      const uint16_t* a = static_cast<const uint16_t*>(x0);
      const uint16_t* c = static_cast<const uint16_t*>(x1);
      if (feature_major)
        hipLaunchKernelGGL((k_feature_elu<uint16_t, true>), grid, block, 0, st, a, c, phi0, phi1, n, ld, d, tiles_n,
                           BH, fix_counts, np);
      else
        hipLaunchKernelGGL((k_feature_elu<uint16_t, false>), grid, block, 0, st, a, c, phi0, phi1, n, ld, d, tiles_n,
                           BH, fix_counts, np);
    } else {
      const float* a = static_cast<const float*>(x0);
      const float* c = static_cast<const float*>(x1);
      if (feature_major)
        hipLaunchKernelGGL((k_feature_elu<float, true>), grid, block, 0, st, a, c, phi0, phi1, n, ld, d, tiles_n, BH,
                           fix_counts, np);
      else
        hipLaunchKernelGGL((k_feature_elu<float, false>), grid, block, 0, st, a, c, phi0, phi1, n, ld, d, tiles_n,
                           BH, fix_counts, np);
    }
    return hipGetLastError();
  }
  const int tiles_m = (m + 63) / 64;
  const long long blocks = static_cast<long long>(tiles_n) * tiles_m * BH * nsrc;
  const float inv_sqrt_m = static_cast<float>(1.0 / std::sqrt(static_cast<double>(m)));
  const dim3 grid(static_cast<unsigned>(blocks));
  const int np = nprf ? 1 : 0, trf = kind == kFeatTrf ? 1 : 0;
  if (d == 64) {
    // 256 positions and every feature per work-group
    const int tiles_fm = (rows + kFm64Pos - 1) / kFm64Pos;
    const dim3 grid(static_cast<unsigned>(static_cast<long long>(tiles_fm) * BH * nsrc));
    const int tiles_n = tiles_fm;
    const dim3 block(kFmThreads);
    if (bf16) {
      const uint16_t* a = static_cast<const uint16_t*>(x0);
      const uint16_t* c = static_cast<const uint16_t*>(x1);
      if (feature_major)
        hipLaunchKernelGGL((k_feature_map64<uint16_t, true>), grid, block, 0, st, a, c, W, phi0, phi1, H, n, ld, m,
                           inv_sqrt_m, tiles_n, BH, fix_counts, np, trf);
      else
        hipLaunchKernelGGL((k_feature_map64<uint16_t, false>), grid, block, 0, st, a, c, W, phi0, phi1, H, n, ld, m,
                           inv_sqrt_m, tiles_n, BH, fix_counts, np, trf);
    } else {
      const float* a = static_cast<const float*>(x0);
      const float* c = static_cast<const float*>(x1);
      if (feature_major)
        hipLaunchKernelGGL((k_feature_map64<float, true>), grid, block, 0, st, a, c, W, phi0, phi1, H, n, ld, m,
                           inv_sqrt_m, tiles_n, BH, fix_counts, np, trf);
      else
        hipLaunchKernelGGL((k_feature_map64<float, false>), grid, block, 0, st, a, c, W, phi0, phi1, H, n, ld, m,
                           inv_sqrt_m, tiles_n, BH, fix_counts, np, trf);
    }
    return hipGetLastError();
  }
  if (bf16) {
    const uint16_t* a = static_cast<const uint16_t*>(x0);
    const uint16_t* c = static_cast<const uint16_t*>(x1);
    if (feature_major)
      hipLaunchKernelGGL((k_feature_map<uint16_t, true>), grid, block, 0, st, a, c, W, phi0, phi1, H, n, ld, d, m,
                         inv_sqrt_m, tiles_n, tiles_m, BH, fix_counts, np, trf);
    else
      hipLaunchKernelGGL((k_feature_map<uint16_t, false>), grid, block, 0, st, a, c, W, phi0, phi1, H, n, ld, d,
                         m, inv_sqrt_m, tiles_n, tiles_m, BH, fix_counts, np, trf);
  } else {
    const float* a = static_cast<const float*>(x0);
    const float* c = static_cast<const float*>(x1);
    if (feature_major)
      hipLaunchKernelGGL((k_feature_map<float, true>), grid, block, 0, st, a, c, W, phi0, phi1, H, n, ld, d, m,
                         inv_sqrt_m, tiles_n, tiles_m, BH, fix_counts, np, trf);
    else
      hipLaunchKernelGGL((k_feature_map<float, false>), grid, block, 0, st, a, c, W, phi0, phi1, H, n, ld, d, m,
                         inv_sqrt_m, tiles_n, tiles_m, BH, fix_counts, np, trf);
  }
  return hipGetLastError();
}

hipError_t launch_vprep(bool bf16, const void* v, long long sp, long long sc, long long bh_stride, int ncols,
                        bool with_ones, int BH, int n, int N, float* pmax, float* colmax, float2* vsc,
                        hipStream_t st) {
  const int cols = ncols + (with_ones ? 1 : 0);
  const int nchunk = vmax_chunks(n);
  const int vgroups = (ncols + 63) / 64, sgroups = (cols + 63) / 64;
  const dim3 block(256);
  const size_t esz = bf16 ? 2 : 4;
  if (sc == 1 && ncols > 0 && ncols % 4 == 0 && sp % 4 == 0 && bh_stride % 4 == 0 &&
      reinterpret_cast<uintptr_t>(v) % (4 * esz) == 0 && static_cast<long long>(n) * sp < (1ll << 31)) {
    const int spi = static_cast<int>(sp);
    const dim3 gmax(static_cast<unsigned>(vgroups), static_cast<unsigned>(nchunk), static_cast<unsigned>(BH));
    const dim3 gscale(static_cast<unsigned>(vgroups), static_cast<unsigned>((N + 63) / 64), static_cast<unsigned>(BH));
    if (bf16) {
      const uint16_t* vv = static_cast<const uint16_t*>(v);
      hipLaunchKernelGGL(k_vmax_q<uint16_t>, gmax, block, 0, st, vv, spi, bh_stride, ncols, n, nchunk, pmax);
      hipLaunchKernelGGL(k_vscale_q<uint16_t>, gscale, block, 0, st, vv, spi, bh_stride, ncols, with_ones ? 1 : 0, n,
                         N, nchunk, pmax, colmax, vsc);
    } else {
      const float* vv = static_cast<const float*>(v);
      hipLaunchKernelGGL(k_vmax_q<float>, gmax, block, 0, st, vv, spi, bh_stride, ncols, n, nchunk, pmax);
      hipLaunchKernelGGL(k_vscale_q<float>, gscale, block, 0, st, vv, spi, bh_stride, ncols, with_ones ? 1 : 0, n, N,
                         nchunk, pmax, colmax, vsc);
    }
    return hipGetLastError();
  }
  const dim3 grid_max(static_cast<unsigned>(static_cast<long long>(BH) * nchunk * vgroups));
  const dim3 grid_scale(static_cast<unsigned>(static_cast<long long>(BH) * ((N + 63) / 64) * sgroups));
  if (bf16) {
    const uint16_t* vv = static_cast<const uint16_t*>(v);
    if (ncols > 0)
      hipLaunchKernelGGL(k_vmax<uint16_t>, grid_max, block, 0, st, vv, sp, sc, bh_stride, ncols, n, nchunk, vgroups,
                         pmax);
    hipLaunchKernelGGL(k_vscale<uint16_t>, grid_scale, block, 0, st, vv, sp, sc, bh_stride, ncols,
                       with_ones ? 1 : 0, n, N, nchunk, sgroups, pmax, colmax, vsc);
  } else {
    const float* vv = static_cast<const float*>(v);
    if (ncols > 0)
      hipLaunchKernelGGL(k_vmax<float>, grid_max, block, 0, st, vv, sp, sc, bh_stride, ncols, n, nchunk, vgroups,
                         pmax);
    hipLaunchKernelGGL(k_vscale<float>, grid_scale, block, 0, st, vv, sp, sc, bh_stride, ncols, with_ones ? 1 : 0, n,
                       N, nchunk, sgroups, pmax, colmax, vsc);
  }
  return hipGetLastError();
}

int vmax_chunks(int n) { return (n + kVmaxChunk - 1) / kVmaxChunk; }

hipError_t launch_conv(int l2, const float* phiq, const float* phik, long long phi_bh_stride, const float2* vsc,
                       const float* colmax, const float2* Hs, const float2* tw, float* part, int BH, int H, int n,
                       int cols, int m, hipStream_t st) {
  return dispatch<ConvFn>(l2, phiq, phik, phi_bh_stride, vsc, colmax, Hs, static_cast<const float2*>(nullptr), tw,
                          part, BH, H, n, cols, m, 1, 1, st);
}

hipError_t launch_conv_split(int l2, const float* phiq, const float* phik, long long phi_bh_stride,
                             const float2* vsc, const float* colmax, const float2* Hs, const float2* hnorm,
                             const float2* tw, float* part, int BH, int H, int n, int cols, int m, int nkb,
                             int fsplit, hipStream_t st) {
  return dispatch<ConvFn>(l2, phiq, phik, phi_bh_stride, vsc, colmax, Hs, hnorm, tw, part, BH, H, n, cols, m, nkb,
                          fsplit, st);
}

int conv_units(int l2, int BH, int cols) {
  int hsplit = 2;
  (void)dispatch<SplitFn>(l2, &hsplit);
  return BH * hsplit * ((cols + 1) / 2);
}

hipError_t launch_gram(const float* phik, const float2* vsc, float* X2, int BH, int m, int N, int pairs,
                       int ksplit, hipStream_t st) {
  const int ltiles = (m + kGramL - 1) / kGramL;
  const long long blocks = static_cast<long long>(BH) * ltiles * ksplit;
  hipLaunchKernelGGL(k_gram, dim3(static_cast<unsigned>(blocks)), dim3(512), 0, st, phik, vsc, X2, m, N, pairs,
                     ltiles, ksplit);
  return hipGetLastError();
}

hipError_t launch_bound_weights(const float* X2, const float* colmax, float2* Wb, int BH, int m, int d,
                                int ksplit, hipStream_t st) {
  const long long total = static_cast<long long>(BH) * (m + 1);  // one wave each
  hipLaunchKernelGGL(k_bound_weights, dim3(static_cast<unsigned>((total + 3) / 4)), dim3(256), 0, st, X2, colmax,
                     Wb, BH, m, d, (d + 2) / 2, ksplit);
  return hipGetLastError();
}

hipError_t launch_combine(const float* part, const float* phiq, const float2* Wb, const float2* hnorm, float* z,
                          float* den_out, unsigned* fix, unsigned long long* fixmask, int BH, int H, int n, int l2,
                          int d, int m, int nsplit, hipStream_t st) {
  const int tiles_n = (n + 63) / 64;
  const size_t lds = (static_cast<size_t>((d + 1) * 65 + 1) & ~static_cast<size_t>(1)) * sizeof(float) +
                     static_cast<size_t>(m + 1) * sizeof(float2);
  const dim3 grid(static_cast<unsigned>(static_cast<long long>(BH) * tiles_n));
  auto go = [&](auto kernel) {
    hipLaunchKernelGGL(kernel, grid, dim3(256), lds, st, part, phiq, Wb, hnorm, z, den_out, fix, fixmask, BH, H, n,
                       1 << l2, l2, d, m, nsplit, tiles_n);
  };
  switch (nsplit) {
    case 2: go(k_combine<2>); break;
    case 4: go(k_combine<4>); break;
    case 8: go(k_combine<8>); break;
    default: go(k_combine<0>); break;
  }
  return hipGetLastError();
}

int fix_slots(int BH) {
  const int s = 4096 / (BH > 0 ? BH : 1);
  return s < 32 ? 32 : (s > 512 ? 512 : s);
}

size_t fix_plan_bytes(int BH, int n) { return FixPlan::bytes(BH, n, fix_slots(BH)); }

hipError_t launch_fixup(const float* phiq, const float* phik, const void* v, bool bf16, const float* b, float* z,
                        float* den_out, const unsigned* fix, const unsigned long long* fixmask, int* plan,
                        double* fixpart, int2* brange, float* cexp, int BH, int H, int n, int ld, int d, int m,
                        hipStream_t st) {
  const int slots = fix_slots(BH);
  hipLaunchKernelGGL(k_brange, dim3(static_cast<unsigned>(H)), dim3(256), 0, st, b, brange, cexp, n);
  if (hipError_t e = hipGetLastError(); e != hipSuccess) return e;
  hipLaunchKernelGGL(k_fix_plan, dim3(static_cast<unsigned>(BH)), dim3(256), 0, st, fix, fixmask, brange, plan, BH, H,
                     n, slots);
  if (hipError_t e = hipGetLastError(); e != hipSuccess) return e;
  const long long blocks = static_cast<long long>(BH) * slots;
  const size_t lds = static_cast<size_t>((m + 2 * kFixL - 1) & ~(2 * kFixL - 1)) * kFixRows * sizeof(float);
  if (lds > 64 * 1024) {
    // phi(q) of a group exceeds the default dynamic LDS limit for m > 512
    static const hipError_t once = [] {
      const int bytes = static_cast<int>(kMaxM * kFixRows * sizeof(float));
      const void* fns[] = {reinterpret_cast<const void*>(&k_fixup<float, false>),
                           reinterpret_cast<const void*>(&k_fixup<float, true>),
                           reinterpret_cast<const void*>(&k_fixup<uint16_t, false>),
                           reinterpret_cast<const void*>(&k_fixup<uint16_t, true>)};
      for (const void* f : fns)
        if (hipError_t e = hipFuncSetAttribute(f, hipFuncAttributeMaxDynamicSharedMemorySize, bytes); e != hipSuccess)
          return e;
      return hipSuccess;
    }();
    if (once != hipSuccess) return once;
  }
  const bool mtail = m % (2 * kFixL) != 0;
  const dim3 grid(static_cast<unsigned>(H), static_cast<unsigned>(BH / H), static_cast<unsigned>(slots));
  auto go = [&](auto kernel, const auto* vt) {
    hipLaunchKernelGGL(kernel, grid, dim3(256), lds, st, phiq, phik, vt, cexp, z, den_out, fix, plan, fixpart, brange,
                       BH, H, n, ld, d, m, slots);
  };
  if (bf16) {
    const auto* vt = static_cast<const uint16_t*>(v);
    if (mtail) go(k_fixup<uint16_t, true>, vt); else go(k_fixup<uint16_t, false>, vt);
  } else {
    const auto* vt = static_cast<const float*>(v);
    if (mtail) go(k_fixup<float, true>, vt); else go(k_fixup<float, false>, vt);
  }
  if (hipError_t e = hipGetLastError(); e != hipSuccess) return e;
  hipLaunchKernelGGL(k_fixup_combine, dim3(static_cast<unsigned>(blocks)), dim3(256), 0, st, fix, plan, fixpart, z,
                     den_out, BH, n, d, slots);
  return hipGetLastError();
}

hipError_t launch_direct_rows(const float* phiq, const float* phik, const float* v, const float* b, float* z,
                              float* den_out, int2* brange, float* cexp, int BH, int H, int n, int ld, int d, int m,
                              hipStream_t st) {
  hipLaunchKernelGGL(k_brange, dim3(static_cast<unsigned>(H)), dim3(256), 0, st, b, brange, cexp, n);
  if (hipError_t e = hipGetLastError(); e != hipSuccess) return e;
  const int mr = (m + 2 * kFixL - 1) & ~(2 * kFixL - 1);
  const size_t lds = static_cast<size_t>(4) * mr * kFixRows * sizeof(float);
  const dim3 grid(static_cast<unsigned>((n + kDirRows - 1) / kDirRows), static_cast<unsigned>(BH / H),
                  static_cast<unsigned>(H));
  if (m % (2 * kFixL) != 0)
    hipLaunchKernelGGL(k_direct_rows<true>, grid, dim3(256), lds, st, phiq, phik, v, cexp, z, den_out, brange, H, n, ld,
                       d, m);
  else
    hipLaunchKernelGGL(k_direct_rows<false>, grid, dim3(256), lds, st, phiq, phik, v, cexp, z, den_out, brange, H, n,
                       ld, d, m);
  return hipGetLastError();
}

hipError_t launch_bwd_prep(bool bf16, const float* G, const float* z, const float* den, const void* v, float* Gh,
                           float* Vh, int BH, int n, int N, int d, hipStream_t st) {
  const int tiles = (N + 63) / 64;
  const dim3 grid(static_cast<unsigned>(static_cast<long long>(BH) * tiles)), block(256);
  if (bf16)
    hipLaunchKernelGGL(k_bwd_prep<uint16_t>, grid, block, 0, st, G, z, den, static_cast<const uint16_t*>(v), Gh, Vh,
                       n, N, d, tiles);
  else
    hipLaunchKernelGGL(k_bwd_prep<float>, grid, block, 0, st, G, z, den, static_cast<const float*>(v), Gh, Vh, n, N,
                       d, tiles);
  return hipGetLastError();
}

hipError_t launch_reverse_bias(const float* b, float* brev, int n, int H, hipStream_t st) {
  const long long total = (2LL * n - 1) * H;
  hipLaunchKernelGGL(k_reverse_bias, dim3(static_cast<unsigned>((total + 255) / 256)), dim3(256), 0, st, b, brev, n,
                     H);
  return hipGetLastError();
}

hipError_t launch_bwd_dv(const float* part, float* dv, int BH, int n, int d, int cols, int nsplit, hipStream_t st) {
  const int tiles = (n + 63) / 64;
  hipLaunchKernelGGL(k_bwd_dv, dim3(static_cast<unsigned>(static_cast<long long>(BH) * tiles)), dim3(256), 0, st,
                     part, dv, n, d, cols, nsplit, tiles);
  return hipGetLastError();
}

hipError_t launch_feature_bwd(bool bf16, const void* x, const float* W, const float* phi, const float* part,
                              float* dx, int BH, int H, int n, int N, int d, int m, int nsplit, bool nprf,
                              hipStream_t st) {
  const int tiles = (n + 63) / 64;
  const dim3 grid(static_cast<unsigned>(static_cast<long long>(BH) * tiles)), block(256);
  if (bf16)
    hipLaunchKernelGGL(k_feature_bwd<uint16_t>, grid, block, 0, st, static_cast<const uint16_t*>(x), W, phi, part,
                       dx, H, n, N, d, m, nsplit, nprf ? 1 : 0, tiles);
  else
    hipLaunchKernelGGL(k_feature_bwd<float>, grid, block, 0, st, static_cast<const float*>(x), W, phi, part, dx, H,
                       n, N, d, m, nsplit, nprf ? 1 : 0, tiles);
  return hipGetLastError();
}

hipError_t launch_widen_bf16(const void* src, float* dst, long long count, hipStream_t st) {
  hipLaunchKernelGGL(k_widen_bf16, dim3(static_cast<unsigned>((count + 255) / 256)), dim3(256), 0, st,
                     static_cast<const uint16_t*>(src), dst, count);
  return hipGetLastError();
}

hipError_t launch_mark_all(unsigned* fix, unsigned long long* fixmask, int BH, int n, hipStream_t st) {
  const int tiles_n = (n + 63) / 64;
  const long long total = static_cast<long long>(BH) * tiles_n > BH + 1 ? static_cast<long long>(BH) * tiles_n : BH + 1;
  hipLaunchKernelGGL(k_mark_all, dim3(static_cast<unsigned>((total + 255) / 256)), dim3(256), 0, st, fix, fixmask, BH,
                     n, tiles_n);
  return hipGetLastError();
}

hipError_t launch_ones(float* ones, int n, int N, hipStream_t st) {
  hipLaunchKernelGGL(k_ones, dim3((N + 255) / 256), dim3(256), 0, st, ones, n, N);
  return hipGetLastError();
}

hipError_t launch_sum_splits(const float* part, float* y, int BH, int C, int n, int ldy, int nsplit,
                             hipStream_t st) {
  const long long total = static_cast<long long>(BH) * C * n;
  hipLaunchKernelGGL(k_sum_splits, dim3(static_cast<unsigned>((total + 255) / 256)), dim3(256), 0, st, part, y, C,
                     n, ldy, nsplit, total);
  return hipGetLastError();
}

}  // namespace krpe
