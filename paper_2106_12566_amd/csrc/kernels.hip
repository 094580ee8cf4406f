// HIP kernels (gfx950) of the forward pass of kernelized attention with RPE.
//
//   z_i = phi(q_i) sum_j c_{j-i} phi(k_j)^T v_j / phi(q_i) sum_j c_{j-i} phi(k_j)^T
//                                                           (Section 3.2, Eq. (7))
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
//  k_conv_contract   the hot loop: channel formation (A1, A2 of Eq. (8)), the
//                    FFT product with C (Eqs. (9)-(10)) and the contraction
//                    with phi(q), all in registers/LDS of one work-group.
//  k_combine         the ratio of Eq. (7), plus a per-row rounding-error bound.
//  k_fixup           exact evaluation of Eq. (7) for rows the bound rejects.
//  k_toeplitz        the Toeplitz product alone (the krpe_toeplitz_conv op).
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

#include "common.hpp"
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

// ------------------------------------------------------------ spectrum --
// c_{-s} embedded circularly in length 2N (see the header comment).
__device__ __forceinline__ float circ_kernel(const float* __restrict__ bh, int s, int n, int N) {
  if (s < n) return expf(bh[n - 1 - s]);
  if (s > 2 * N - n) return expf(bh[2 * N - s + n - 1]);
  return 0.f;
}

// One transform per (head, half).  Hs[h][half][k] in natural frequency order.
// Also, when requested: hnorm[h] = (||h||_1, ||h||_2) and *fix_count = 0.
template <int L2>
__global__ __launch_bounds__(Conf<L2>::THREADS) void k_spectrum(const float* __restrict__ b,
                                                                 const float2* __restrict__ tw,
                                                                 float2* __restrict__ Hs,
                                                                 float2* __restrict__ hnorm,
                                                                 unsigned* __restrict__ fix_count, int H, int n) {
  using C = Conf<L2>;
  using F = typename C::F;
  __shared__ float2 lds[C::LDS_SLOTS];
  __shared__ float red[C::WAVES];
  if (fix_count && blockIdx.x == 0 && threadIdx.x == 0) *fix_count = 0u;
  const int g = threadIdx.x / F::T, tau = threadIdx.x % F::T;
  const int units = 2 * H;
  int unit = blockIdx.x * C::G + g;
  const bool active = unit < units;
  if (!active) unit = units - 1;
  const int h = unit >> 1, half = unit & 1;
  const float* bh = b + static_cast<size_t>(h) * (2 * n - 1);
  float2 x[F::R];
  float s1 = 0.f, s2 = 0.f;
#pragma unroll
  for (int r = 0; r < F::R; ++r) {
    const int s = tau + F::T * r;
    const float lo = circ_kernel(bh, s, n, F::N), hi = circ_kernel(bh, s + F::N, n, F::N);
    s1 += lo + hi;
    s2 = fmaf(lo, lo, fmaf(hi, hi, s2));
    x[r] = half == 0 ? make_float2(lo + hi, 0.f) : make_float2((lo - hi) * tw[s].x, (lo - hi) * tw[s].y);
  }
  if (hnorm) {
    s1 = unit_reduce<F::T>(s1, red, OpAdd());
    s2 = unit_reduce<F::T>(s2, red, OpAdd());
    if (active && half == 0 && tau == 0) hnorm[h] = make_float2(s1, sqrtf(s2));
  }
  F::forward(x, lds + g * (F::P > 1 ? F::LDS : 0), tw, tau);
  if (active) {
    const float scale = 1.0f / static_cast<float>(2 * F::N);
    float2* out = Hs + static_cast<size_t>(unit) * F::N;
#pragma unroll
    for (int i = 0; i < F::R; ++i) {
      const int k = F::frequency_of(F::spectrum_pos(tau, i));
      out[k] = make_float2(x[i].x * scale, x[i].y * scale);
    }
  }
}

// --------------------------------------------------------- feature map --
typedef float floatx16 __attribute__((ext_vector_type(16)));

// phi = exp(x W^T - ||x||^2/2) / sqrt(m) for up to two sources (q and k) in
// one launch.  Tile: 64 positions x 64 features per work-group, four waves of
// 32 x 32 v_mfma_f32_32x32x2f32 tiles; K (= d) staged through LDS in chunks of
// 32.  FEATURE_MAJOR writes phi[bh][l][i] for i < ld (zeros for n <= i < ld;
// lanes run along positions), otherwise phi[bh][i][l] (lanes run along
// features): stores stay coalesced either way because the operand roles are
// swapped.
template <typename TX, bool FEATURE_MAJOR>
__global__ __launch_bounds__(256) void k_feature_map(const TX* __restrict__ x0, const TX* __restrict__ x1,
                                                     const float* __restrict__ W, float* __restrict__ phi0,
                                                     float* __restrict__ phi1, int H, int n, int ld, int d,
                                                     int m, float inv_sqrt_m, int tiles_n, int tiles_m,
                                                     int BH) {
  __shared__ float xs[64][33];
  __shared__ float wsm[64][33];
  __shared__ float half_sq[64];
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
  if (threadIdx.x < 64) half_sq[threadIdx.x] = 0.5f * sq;
  __syncthreads();
  const int n_store = FEATURE_MAJOR ? ld : n;
#pragma unroll
  for (int v = 0; v < 16; ++v) {
    // 32x32 MFMA result layout: lane holds column lane%32, rows 8(v/4) + 4(lane/32) + v%4
    const int row = 8 * (v >> 2) + 4 * (lane >> 5) + (v & 3);
    const int col = lane & 31;
    const int li = FEATURE_MAJOR ? wl + row : wl + col;  // feature within tile
    const int ii = FEATURE_MAJOR ? wi + col : wi + row;  // position within tile
    const int l = l0 + li, i = i0 + ii;
    if (i < n_store && l < m) {
      const float val = i < n ? expf(acc[v] - half_sq[ii]) * inv_sqrt_m : 0.f;
      if constexpr (FEATURE_MAJOR)
        phi[(static_cast<size_t>(bh) * m + l) * ld + i] = val;
      else
        phi[(static_cast<size_t>(bh) * n + i) * m + l] = val;
    }
  }
}

// ---------------------------------------------- convolution + contraction --
// Unit u = ((bh * 2 + half) * pairs + cp), pairs = ceil((d + 1) / 2).  The
// unit owns the two columns c0 = 2 cp and c1 = 2 cp + 1 of v' = [v, 1]
// (column d is the all-ones column of the denominator; c1 > d means none).
// For every feature l the two channels phi_l(k_j) v'_{j,c0} and
// phi_l(k_j) v'_{j,c1} share the envelope phi_l(k), so packing them as the
// real and imaginary parts of one complex signal keeps their magnitudes alike:
// the FFT's rounding error, set by the pair's norm, stays proportional to
// each.  Each column is also scaled by its own max |v| before packing.
//
// Writes, for its spectrum half, the partial numerators / denominator
//   part[bh][half][c][i] = sum_l phi_l(q_i) (C_half a_{l,c})_i,   c in {c0, c1},
// and from half 0 the error-bound weights
//   bnd[bh][cp][i] = sum_l phi_l(q_i) ||x_l||_2   (x_l the packed signal)
// and colmax[bh][c] = max_j |v_{j,c}| for its value columns.
template <typename F, int WAVES, bool HALF1>
__device__ __forceinline__ void conv_loop(const float* __restrict__ pk, const float* __restrict__ pq,
                                          const float2* __restrict__ tw, const float (&v0)[F::R],
                                          const float (&v1)[F::R], const float2 (&Hr)[F::R], float2* lds,
                                          float (*nslot)[WAVES], int tau, int m, float (&acc0)[F::R],
                                          float (&acc1)[F::R], float (&bound)[F::R]) {
  float2 twist[F::R];
  if constexpr (HALF1) {
#pragma unroll
    for (int r = 0; r < F::R; ++r) twist[r] = tw[tau + F::T * r];
  }
  for (int l = 0; l < m; ++l) {
    const float* __restrict__ pkl = pk + static_cast<size_t>(l) * F::N;
    float2 x[F::R];
    float nx = 0.f;
#pragma unroll
    for (int r = 0; r < F::R; ++r) {
      const float a = pkl[tau + F::T * r];
      x[r] = make_float2(a * v0[r], a * v1[r]);
      if constexpr (HALF1) {
        x[r] = cmul(x[r], twist[r]);
      } else {
        nx = fmaf(x[r].x, x[r].x, fmaf(x[r].y, x[r].y, nx));
      }
    }
    if constexpr (!HALF1) {
      nx = wave_unit_reduce<F::T>(nx, OpAdd());
      // Cross-wave part of the reduction rides on the FFT's own barriers:
      // written here, read after the inverse transform; double-buffered on l.
      if constexpr (F::T > 64) {
        if ((threadIdx.x & 63) == 0) nslot[l & 1][threadIdx.x >> 6] = nx;
      }
    }
    F::forward(x, lds, tw, tau);
#pragma unroll
    for (int i = 0; i < F::R; ++i) x[i] = cmul(x[i], Hr[i]);
    F::inverse(x, lds, tw, tau);
    const float* __restrict__ pql = pq + static_cast<size_t>(l) * F::N;
    float xn = 0.f;
    if constexpr (!HALF1) {
      if constexpr (F::T > 64) {
        const int first = (threadIdx.x / F::T) * (F::T / 64);
        nx = nslot[l & 1][first];
#pragma unroll
        for (int w = 1; w < F::T / 64; ++w) nx += nslot[l & 1][first + w];
      }
      xn = sqrtf(nx);
    }
#pragma unroll
    for (int r = 0; r < F::R; ++r) {
      if constexpr (HALF1) x[r] = cmulc(x[r], twist[r]);
      const float f = pql[tau + F::T * r];
      acc0[r] = fmaf(f, x[r].x, acc0[r]);
      acc1[r] = fmaf(f, x[r].y, acc1[r]);
      if constexpr (!HALF1) bound[r] = fmaf(f, xn, bound[r]);
    }
  }
}

template <int L2, typename TV>
__global__ __launch_bounds__(Conf<L2>::THREADS) void k_conv_contract(
    const float* __restrict__ phiq, const float* __restrict__ phik, const TV* __restrict__ v,
    const float2* __restrict__ Hs, const float2* __restrict__ tw, float* __restrict__ part,
    float* __restrict__ bnd, float* __restrict__ colmax, int H, int n, int d, int m, int units) {
  using C = Conf<L2>;
  using F = typename C::F;
  __shared__ float2 lds_all[C::LDS_SLOTS];
  __shared__ float red[C::WAVES];
  __shared__ float nslot[2][C::WAVES];
  const int g = threadIdx.x / F::T, tau = threadIdx.x % F::T;
  const int pairs = (d + 2) / 2;
  int unit = xcd_block(blockIdx.x, gridDim.x) * C::G + g;
  const bool active = unit < units;
  if (!active) unit = units - 1;  // keep the barriers uniform; results discarded
  const int cp = unit % pairs;
  const int rest = unit / pairs;
  const int half = rest & 1, bh = rest >> 1, h = bh % H;
  const int c0 = 2 * cp, c1 = 2 * cp + 1;
  float2* lds = lds_all + g * (F::P > 1 ? F::LDS : 0);

  // Value columns at this thread's positions, and their scales.
  const TV* __restrict__ vb = v + static_cast<size_t>(bh) * n * d;
  float v0[F::R], v1[F::R];
  float mx0 = 0.f, mx1 = 0.f;
#pragma unroll
  for (int r = 0; r < F::R; ++r) {
    const int pos = tau + F::T * r;
    const bool in = pos < n;
    v0[r] = in ? (c0 < d ? to_f32(vb[static_cast<size_t>(pos) * d + c0]) : 1.f) : 0.f;
    v1[r] = in ? (c1 < d ? to_f32(vb[static_cast<size_t>(pos) * d + c1]) : (c1 == d ? 1.f : 0.f)) : 0.f;
    mx0 = fmaxf(mx0, fabsf(v0[r]));
    mx1 = fmaxf(mx1, fabsf(v1[r]));
  }
  mx0 = unit_reduce<F::T>(mx0, red, OpMax());
  mx1 = unit_reduce<F::T>(mx1, red, OpMax());
  const float s0 = mx0 > 0.f ? mx0 : 1.f, s1 = mx1 > 0.f ? mx1 : 1.f;
  const float is0 = 1.f / s0, is1 = 1.f / s1;
#pragma unroll
  for (int r = 0; r < F::R; ++r) {
    v0[r] *= is0;
    v1[r] *= is1;
  }
  if (active && half == 0 && tau == 0) {
    if (c0 < d) colmax[static_cast<size_t>(bh) * d + c0] = mx0;
    if (c1 < d) colmax[static_cast<size_t>(bh) * d + c1] = mx1;
  }

  // Spectrum half in registers, in the order the forward transform leaves it.
  float2 Hr[F::R];
  const float2* __restrict__ Hh = Hs + (static_cast<size_t>(h) * 2 + half) * F::N;
#pragma unroll
  for (int i = 0; i < F::R; ++i) Hr[i] = Hh[F::frequency_of(F::spectrum_pos(tau, i))];

  float acc0[F::R], acc1[F::R], bound[F::R];
#pragma unroll
  for (int r = 0; r < F::R; ++r) acc0[r] = acc1[r] = bound[r] = 0.f;

  const float* __restrict__ pk = phik + static_cast<size_t>(bh) * m * F::N;
  const float* __restrict__ pq = phiq + static_cast<size_t>(bh) * m * F::N;
  if (half)
    conv_loop<F, C::WAVES, true>(pk, pq, tw, v0, v1, Hr, lds, nslot, tau, m, acc0, acc1, bound);
  else
    conv_loop<F, C::WAVES, false>(pk, pq, tw, v0, v1, Hr, lds, nslot, tau, m, acc0, acc1, bound);

  if (active) {
    float* __restrict__ out = part + ((static_cast<size_t>(bh) * 2 + half) * (d + 1) + c0) * n;
    float* __restrict__ bout = bnd + (static_cast<size_t>(bh) * pairs + cp) * n;
#pragma unroll
    for (int r = 0; r < F::R; ++r) {
      const int pos = tau + F::T * r;
      if (pos < n) {
        out[pos] = acc0[r] * s0;
        if (c1 <= d) out[n + pos] = acc1[r] * s1;
        if (half == 0) bout[pos] = bound[r];
      }
    }
  }
}

// -------------------------------------------------------------- combine --
// z[bh][i][c] = (P0[c][i] + P1[c][i]) / (P0[d][i] + P1[d][i]),  P = part[bh],
// and the certification of each row.  With K = kGamma u log2(L) ||h||_2 / sqrt(L),
// the error model of common.hpp bounds the rounding error of numerator c by
// K bnd[p(c)][i] s_c (+ a part relative to the value itself) and that of the
// denominator by K bnd[p(d)][i], p(c) = c / 2 the packed pair of column c.  A
// row whose normwise relative bound exceeds kTau is queued for k_fixup.
__global__ __launch_bounds__(256) void k_combine(const float* __restrict__ part, const float* __restrict__ bnd,
                                                 const float* __restrict__ colmax,
                                                 const float2* __restrict__ hnorm, float* __restrict__ z,
                                                 unsigned* __restrict__ fix_count, unsigned* __restrict__ fix_list,
                                                 int H, int n, int log2N, int d, int tiles_n) {
  __shared__ float tile[kMaxD + 1][65];
  __shared__ float btile[kMaxD / 2 + 1][65];
  __shared__ float scol[kMaxD + 1];
  __shared__ float zmax[64];
  const int bh = blockIdx.x / tiles_n, i0 = (blockIdx.x % tiles_n) * 64;
  const int h = bh % H;
  const int pairs = (d + 2) / 2;
  const float* __restrict__ p0 = part + static_cast<size_t>(bh) * 2 * (d + 1) * n;
  const float* __restrict__ p1 = p0 + static_cast<size_t>(d + 1) * n;
  const float* __restrict__ bb = bnd + static_cast<size_t>(bh) * pairs * n;
  for (int e = threadIdx.x; e < (d + 1) * 64; e += 256) {
    const int c = e >> 6, i = e & 63;
    const int pos = i0 + i;
    tile[c][i] = pos < n ? p0[static_cast<size_t>(c) * n + pos] + p1[static_cast<size_t>(c) * n + pos] : 1.f;
  }
  for (int e = threadIdx.x; e < pairs * 64; e += 256) {
    const int p = e >> 6, i = e & 63;
    const int pos = i0 + i;
    btile[p][i] = pos < n ? bb[static_cast<size_t>(p) * n + pos] : 0.f;
  }
  for (int c = threadIdx.x; c <= d; c += 256) scol[c] = c < d ? colmax[static_cast<size_t>(bh) * d + c] : 1.f;
  __syncthreads();
  if (threadIdx.x < 64) {
    const int i = threadIdx.x;
    float zm = 0.f;
    const float den = tile[d][i];
    for (int c = 0; c < d; ++c) zm = fmaxf(zm, fabsf(tile[c][i] / den));
    zmax[i] = zm;
  }
  __syncthreads();
  float* __restrict__ zb = z + static_cast<size_t>(bh) * n * d;
  for (int e = threadIdx.x; e < 64 * d; e += 256) {
    const int i = e / d, c = e % d;
    const int pos = i0 + i;
    if (pos < n) zb[static_cast<size_t>(pos) * d + c] = tile[c][i] / tile[d][i];
  }
  if (threadIdx.x < 64) {
    const int i = threadIdx.x, pos = i0 + i;
    if (pos < n) {
      const float L = static_cast<float>(2 << log2N);
      const float lg = static_cast<float>(log2N + 1);
      const float K = kGamma * kUnitRoundoff * lg * hnorm[h].y * rsqrtf(L);
      float errN = 0.f, vmax = 0.f;
      for (int c = 0; c < d; ++c) {
        errN = fmaxf(errN, btile[c >> 1][i] * scol[c]);
        vmax = fmaxf(vmax, scol[c]);
      }
      const float den = tile[d][i];
      const float zm = zmax[i];
      const float errD = K * btile[d >> 1][i];
      const float err = K * errN + zm * errD;
      const float scale = fmaxf(zm, 1e-6f * vmax);
      const float rel_floor = 2.f * kGamma * kUnitRoundoff * lg;
      const bool ok = isfinite(den) && den > 0.f && isfinite(zm) && err <= (kTau - rel_floor) * scale * den;
      if (!ok) {
        const unsigned slot = atomicAdd(fix_count, 1u);
        fix_list[slot] = static_cast<unsigned>(bh) * static_cast<unsigned>(n) + static_cast<unsigned>(pos);
      }
    }
  }
}

// ---------------------------------------------------------------- fixup --
// Exact evaluation of Eq. (7) for the rows k_combine could not certify:
//   w_j = c_{j-i} phi(q_i) . phi(k_j)   (skipped where c_{j-i} = 0)
//   z_i = sum_j w_j v_j / sum_j w_j     (accumulated in fp64)
// A fixed grid walks the row list; every work-group exits when it is done.
__global__ __launch_bounds__(256) void k_fixup(const float* __restrict__ phiq, const float* __restrict__ phik,
                                               const void* __restrict__ vraw, int v_bf16,
                                               const float* __restrict__ b, float* __restrict__ z,
                                               const unsigned* __restrict__ fix_count,
                                               const unsigned* __restrict__ fix_list, int H, int n, int ld,
                                               int d, int m) {
  extern __shared__ float smem[];
  float* fq = smem;      // m
  float* w = smem + m;   // n
  __shared__ double red[256];
  __shared__ int jlo_s, jhi_s;
  const unsigned count = *fix_count;
  for (unsigned item = blockIdx.x; item < count; item += gridDim.x) {
    const unsigned row = fix_list[item];
    const int bh = static_cast<int>(row / static_cast<unsigned>(n));
    const int i = static_cast<int>(row % static_cast<unsigned>(n));
    const int h = bh % H;
    const float* __restrict__ pq = phiq + static_cast<size_t>(bh) * m * ld;
    const float* __restrict__ pk = phik + static_cast<size_t>(bh) * m * ld;
    const float* __restrict__ bhv = b + static_cast<size_t>(h) * (2 * n - 1);
    __syncthreads();
    for (int l = threadIdx.x; l < m; l += 256) fq[l] = pq[static_cast<size_t>(l) * ld + i];
    if (threadIdx.x == 0) {
      jlo_s = n;
      jhi_s = -1;
    }
    __syncthreads();
    int lo = n, hi = -1;
    for (int j = threadIdx.x; j < n; j += 256) {
      const float bj = bhv[j - i + n - 1];
      float wj = 0.f;
      if (bj != -INFINITY) {
        float kk = 0.f;
        for (int l = 0; l < m; ++l) kk = fmaf(fq[l], pk[static_cast<size_t>(l) * ld + j], kk);
        wj = expf(bj) * kk;
        lo = min(lo, j);
        hi = max(hi, j);
      }
      w[j] = wj;
    }
    atomicMin(&jlo_s, lo);
    atomicMax(&jhi_s, hi);
    __syncthreads();
    const int jlo = jlo_s, jhi = jhi_s;
    const int cols = d + 1;
    const int groups = 256 / cols;
    const int c = threadIdx.x % cols, grp = threadIdx.x / cols;
    double acc = 0.0;
    if (grp < groups) {
      const size_t vbase = static_cast<size_t>(bh) * n * d;
      for (int j = jlo + grp; j <= jhi; j += groups) {
        const float wj = w[j];
        if (wj == 0.f) continue;
        float vv = 1.f;
        if (c < d) {
          const size_t idx = vbase + static_cast<size_t>(j) * d + c;
          vv = v_bf16 ? to_f32(static_cast<const uint16_t*>(vraw)[idx]) : static_cast<const float*>(vraw)[idx];
        }
        acc += static_cast<double>(wj) * static_cast<double>(vv);
      }
    }
    red[threadIdx.x] = acc;
    __syncthreads();
    // Thread t < cols sums the group partials of its column into slot t; the
    // slots it reads (g * cols + t, g >= 1) are >= cols, so none is overwritten.
    if (threadIdx.x < cols) {
      double s = red[threadIdx.x];
      for (int gg = 1; gg < groups; ++gg) s += red[gg * cols + threadIdx.x];
      red[threadIdx.x] = s;
    }
    __syncthreads();
    if (threadIdx.x < d)
      z[(static_cast<size_t>(bh) * n + i) * d + threadIdx.x] = static_cast<float>(red[threadIdx.x] / red[d]);
  }
}

// ------------------------------------------------------ Toeplitz product --
// Unit u = bh * ceil(C/2) + pair: channels (2 pair, 2 pair + 1) as one complex
// signal, each scaled by its own max |a| so that neither's rounding error is
// set by the other's magnitude; both spectrum halves in turn, summed in
// registers.
template <int L2>
__global__ __launch_bounds__(Conf<L2>::THREADS) void k_toeplitz(const float* __restrict__ a,
                                                                 float* __restrict__ y,
                                                                 const float2* __restrict__ Hs,
                                                                 const float2* __restrict__ tw, int H, int Cch,
                                                                 int n, int units) {
  using Cf = Conf<L2>;
  using F = typename Cf::F;
  __shared__ float2 lds_all[Cf::LDS_SLOTS];
  __shared__ float red[Cf::WAVES];
  const int g = threadIdx.x / F::T, tau = threadIdx.x % F::T;
  int unit = blockIdx.x * Cf::G + g;
  const bool active = unit < units;
  if (!active) unit = units - 1;
  const int pairs = (Cch + 1) / 2;
  const int bh = unit / pairs, pr = unit % pairs, h = bh % H;
  const int c0 = 2 * pr;
  const bool two = c0 + 1 < Cch;
  float2* lds = lds_all + g * (F::P > 1 ? F::LDS : 0);
  const float* __restrict__ a0 = a + (static_cast<size_t>(bh) * Cch + c0) * n;
  float u0[F::R], u1[F::R];
  float mx0 = 0.f, mx1 = 0.f;
#pragma unroll
  for (int r = 0; r < F::R; ++r) {
    const int pos = tau + F::T * r;
    u0[r] = pos < n ? a0[pos] : 0.f;
    u1[r] = (pos < n && two) ? a0[n + pos] : 0.f;
    mx0 = fmaxf(mx0, fabsf(u0[r]));
    mx1 = fmaxf(mx1, fabsf(u1[r]));
  }
  mx0 = unit_reduce<F::T>(mx0, red, OpMax());
  mx1 = unit_reduce<F::T>(mx1, red, OpMax());
  const float s0 = mx0 > 0.f ? mx0 : 1.f, s1 = mx1 > 0.f ? mx1 : 1.f;
  const float is0 = 1.f / s0, is1 = 1.f / s1;
  float2 acc[F::R];
#pragma unroll
  for (int r = 0; r < F::R; ++r) acc[r] = make_float2(0.f, 0.f);
  for (int half = 0; half < 2; ++half) {
    const float2* __restrict__ Hh = Hs + (static_cast<size_t>(h) * 2 + half) * F::N;
    float2 x[F::R];
#pragma unroll
    for (int r = 0; r < F::R; ++r) {
      const int pos = tau + F::T * r;
      x[r] = make_float2(u0[r] * is0, u1[r] * is1);
      if (half) x[r] = cmul(x[r], tw[pos]);
    }
    F::forward(x, lds, tw, tau);
#pragma unroll
    for (int i = 0; i < F::R; ++i) x[i] = cmul(x[i], Hh[F::frequency_of(F::spectrum_pos(tau, i))]);
    F::inverse(x, lds, tw, tau);
#pragma unroll
    for (int r = 0; r < F::R; ++r) {
      const int pos = tau + F::T * r;
      const float2 t = half ? cmulc(x[r], tw[pos]) : x[r];
      acc[r] = cadd(acc[r], t);
    }
  }
  if (active) {
    float* __restrict__ y0 = y + (static_cast<size_t>(bh) * Cch + c0) * n;
#pragma unroll
    for (int r = 0; r < F::R; ++r) {
      const int pos = tau + F::T * r;
      if (pos < n) {
        y0[pos] = acc[r].x * s0;
        if (two) y0[n + pos] = acc[r].y * s1;
      }
    }
  }
}

// ============================================================ launchers ==
namespace {

template <int L2>
hipError_t spectrum_l2(const float* b, const float2* tw, float2* Hs, float2* hnorm, unsigned* fix_count, int H,
                       int n, hipStream_t st) {
  using C = Conf<L2>;
  const int blocks = (2 * H + C::G - 1) / C::G;
  hipLaunchKernelGGL(k_spectrum<L2>, dim3(blocks), dim3(C::THREADS), 0, st, b, tw, Hs, hnorm, fix_count, H, n);
  return hipGetLastError();
}

template <int L2, typename TV>
hipError_t conv_l2(const float* phiq, const float* phik, const TV* v, const float2* Hs, const float2* tw,
                   float* part, float* bnd, float* colmax, int BH, int H, int n, int d, int m, hipStream_t st) {
  using C = Conf<L2>;
  const int units = BH * 2 * ((d + 2) / 2);
  const int blocks = (units + C::G - 1) / C::G;
  hipLaunchKernelGGL((k_conv_contract<L2, TV>), dim3(blocks), dim3(C::THREADS), 0, st, phiq, phik, v, Hs, tw,
                     part, bnd, colmax, H, n, d, m, units);
  return hipGetLastError();
}

template <int L2>
hipError_t toeplitz_l2(const float* a, float* y, const float2* Hs, const float2* tw, int BH, int H, int Cch, int n,
                       hipStream_t st) {
  using C = Conf<L2>;
  const int units = BH * ((Cch + 1) / 2);
  const int blocks = (units + C::G - 1) / C::G;
  hipLaunchKernelGGL(k_toeplitz<L2>, dim3(blocks), dim3(C::THREADS), 0, st, a, y, Hs, tw, H, Cch, n, units);
  return hipGetLastError();
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
struct ConvF32Fn {
  template <typename... A>
  static hipError_t run(A... a) { return conv_l2<L2, float>(a...); }
};
template <int L2>
struct ConvBf16Fn {
  template <typename... A>
  static hipError_t run(A... a) { return conv_l2<L2, uint16_t>(a...); }
};
template <int L2>
struct ToeplitzFn {
  template <typename... A>
  static hipError_t run(A... a) { return toeplitz_l2<L2>(a...); }
};

}  // namespace

hipError_t launch_twiddles(float2* tw, int l2, hipStream_t st) {
  const int count = 2 << l2;
  hipLaunchKernelGGL(k_twiddles, dim3((count + 255) / 256), dim3(256), 0, st, tw, l2);
  return hipGetLastError();
}

hipError_t launch_spectrum(int l2, const float* b, const float2* tw, float2* Hs, float2* hnorm, unsigned* fix_count,
                           int H, int n, hipStream_t st) {
  return dispatch<SpectrumFn>(l2, b, tw, Hs, hnorm, fix_count, H, n, st);
}

hipError_t launch_feature_map(bool bf16, const void* x0, const void* x1, const float* W, float* phi0, float* phi1,
                              int nsrc, bool feature_major, int ld, int BH, int H, int n, int d, int m,
                              hipStream_t st) {
  const int rows = feature_major ? ld : n;
  const int tiles_n = (rows + 63) / 64, tiles_m = (m + 63) / 64;
  const long long blocks = static_cast<long long>(tiles_n) * tiles_m * BH * nsrc;
  const float inv_sqrt_m = static_cast<float>(1.0 / std::sqrt(static_cast<double>(m)));
  const dim3 grid(static_cast<unsigned>(blocks)), block(256);
  if (bf16) {
    const uint16_t* a = static_cast<const uint16_t*>(x0);
    const uint16_t* c = static_cast<const uint16_t*>(x1);
    if (feature_major)
      hipLaunchKernelGGL((k_feature_map<uint16_t, true>), grid, block, 0, st, a, c, W, phi0, phi1, H, n, ld, d, m,
                         inv_sqrt_m, tiles_n, tiles_m, BH);
    else
      hipLaunchKernelGGL((k_feature_map<uint16_t, false>), grid, block, 0, st, a, c, W, phi0, phi1, H, n, ld, d,
                         m, inv_sqrt_m, tiles_n, tiles_m, BH);
  } else {
    const float* a = static_cast<const float*>(x0);
    const float* c = static_cast<const float*>(x1);
    if (feature_major)
      hipLaunchKernelGGL((k_feature_map<float, true>), grid, block, 0, st, a, c, W, phi0, phi1, H, n, ld, d, m,
                         inv_sqrt_m, tiles_n, tiles_m, BH);
    else
      hipLaunchKernelGGL((k_feature_map<float, false>), grid, block, 0, st, a, c, W, phi0, phi1, H, n, ld, d, m,
                         inv_sqrt_m, tiles_n, tiles_m, BH);
  }
  return hipGetLastError();
}

hipError_t launch_conv(int l2, bool bf16, const float* phiq, const float* phik, const void* v, const float2* Hs,
                       const float2* tw, float* part, float* bnd, float* colmax, int BH, int H, int n, int d,
                       int m, hipStream_t st) {
  if (bf16)
    return dispatch<ConvBf16Fn>(l2, phiq, phik, static_cast<const uint16_t*>(v), Hs, tw, part, bnd, colmax, BH, H,
                                n, d, m, st);
  return dispatch<ConvF32Fn>(l2, phiq, phik, static_cast<const float*>(v), Hs, tw, part, bnd, colmax, BH, H, n, d,
                             m, st);
}

hipError_t launch_combine(const float* part, const float* bnd, const float* colmax, const float2* hnorm, float* z,
                          unsigned* fix_count, unsigned* fix_list, int BH, int H, int n, int l2, int d,
                          hipStream_t st) {
  const int tiles_n = (n + 63) / 64;
  hipLaunchKernelGGL(k_combine, dim3(BH * tiles_n), dim3(256), 0, st, part, bnd, colmax, hnorm, z, fix_count,
                     fix_list, H, n, l2, d, tiles_n);
  return hipGetLastError();
}

hipError_t launch_fixup(const float* phiq, const float* phik, const void* v, bool bf16, const float* b, float* z,
                        const unsigned* fix_count, const unsigned* fix_list, int BH, int H, int n, int ld, int d,
                        int m, hipStream_t st) {
  const long long rows = static_cast<long long>(BH) * n;
  const int blocks = static_cast<int>(rows < 1024 ? rows : 1024);
  const size_t lds = (static_cast<size_t>(m) + n) * sizeof(float);
  // Allow the largest dynamic LDS any call can ask for, once per process.
  static const hipError_t attr = hipFuncSetAttribute(
      reinterpret_cast<const void*>(k_fixup), hipFuncAttributeMaxDynamicSharedMemorySize,
      static_cast<int>((static_cast<size_t>(kMaxM) + (1u << kMaxLog2N)) * sizeof(float)));
  if (attr != hipSuccess) return attr;
  hipLaunchKernelGGL(k_fixup, dim3(blocks), dim3(256), lds, st, phiq, phik, v, bf16 ? 1 : 0, b, z, fix_count,
                     fix_list, H, n, ld, d, m);
  return hipGetLastError();
}

hipError_t launch_toeplitz(int l2, const float* a, float* y, const float2* Hs, const float2* tw, int BH, int H,
                           int C, int n, hipStream_t st) {
  return dispatch<ToeplitzFn>(l2, a, y, Hs, tw, BH, H, C, n, st);
}

}  // namespace krpe
