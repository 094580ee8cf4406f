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
// Also, when requested: hnorm[h] = (||h||_1, ||h||_2).
template <int L2>
__global__ __launch_bounds__(Conf<L2>::THREADS) void k_spectrum(const float* __restrict__ b,
                                                                 const float2* __restrict__ tw,
                                                                 float2* __restrict__ Hs,
                                                                 float2* __restrict__ hnorm, int H, int n) {
  using C = Conf<L2>;
  using F = typename C::F;
  __shared__ float2 lds[C::LDS_SLOTS];
  __shared__ float red[C::WAVES];
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
                                                     int BH, unsigned* __restrict__ fix_counts) {
  // Clear the exact-evaluation queue counters (fix_counts[0..BH]) for k_combine.
  if (fix_counts && threadIdx.x == 0 && blockIdx.x <= static_cast<unsigned>(BH)) fix_counts[blockIdx.x] = 0u;
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
// Unit u = ((bh * HSPLIT + hs) * pairs + cp), pairs = ceil((d + 1) / 2).  The
// unit owns the two columns c0 = 2 cp and c1 = 2 cp + 1 of v' = [v, 1]
// (column d is the all-ones column of the denominator; c1 > d means none) and
// the spectrum halves hs*KH .. hs*KH + KH - 1.  For every feature l the two
// channels phi_l(k_j) v'_{j,c0} and phi_l(k_j) v'_{j,c1} share the envelope
// phi_l(k), so packing them as the real and imaginary parts of one complex
// signal keeps their magnitudes alike: the FFT's rounding error, set by the
// pair's norm, stays proportional to each.  Each column is also scaled by its
// own max |v| before packing.
//
// Writes the partial numerators / denominator of Eq. (10) of its halves
//   part[bh][hs][c][i] = sum_l phi_l(q_i) (C_hs a_{l,c})_i,   c in {c0, c1},
// and, from hs = 0, the error-bound weights
//   bnd[bh][cp][i] = sum_l phi_l(q_i) ||x_l||_2   (x_l the packed signal)
// and colmax[bh][c] = max_j |v_{j,c}| for its value columns.
template <typename F, int WAVES, int KH, int HALF0>
__device__ __forceinline__ void conv_loop(const float* __restrict__ pk, const float* __restrict__ pq,
                                          const float2* __restrict__ tw, const float (&v0)[F::R],
                                          const float (&v1)[F::R], const float2 (&Hr)[KH][F::R], float2* lds,
                                          float (*nslot)[WAVES], int tau, int m, float (&acc0)[F::R],
                                          float (&acc1)[F::R], float (&bound)[F::R]) {
  constexpr bool kTwist = HALF0 + KH > 1;   // some half of this unit is the odd one
  constexpr bool kBound = HALF0 == 0;       // one unit per pair accumulates the bound
  float2 twist[F::R];
  if constexpr (kTwist) {
#pragma unroll
    for (int r = 0; r < F::R; ++r) twist[r] = tw[tau + F::T * r];
  }
  float a_next[F::R];
#pragma unroll
  for (int r = 0; r < F::R; ++r) a_next[r] = pk[tau + F::T * r];
  for (int l = 0; l < m; ++l) {
    float a[F::R], f[F::R];
#pragma unroll
    for (int r = 0; r < F::R; ++r) a[r] = a_next[r];
    // Loads for later stay in flight across the transform (the barriers only
    // wait for LDS traffic): phi(q) for this feature, phi(k) for the next.
    const float* __restrict__ pql = pq + static_cast<size_t>(l) * F::N;
#pragma unroll
    for (int r = 0; r < F::R; ++r) f[r] = pql[tau + F::T * r];
    if (l + 1 < m) {
      const float* __restrict__ pkn = pk + static_cast<size_t>(l + 1) * F::N;
#pragma unroll
      for (int r = 0; r < F::R; ++r) a_next[r] = pkn[tau + F::T * r];
    }
    float2 x[KH][F::R];
    float nx = 0.f;
#pragma unroll
    for (int r = 0; r < F::R; ++r) {
      const float2 xb = make_float2(a[r] * v0[r], a[r] * v1[r]);
      if constexpr (kBound) nx = fmaf(xb.x, xb.x, fmaf(xb.y, xb.y, nx));
#pragma unroll
      for (int k = 0; k < KH; ++k) x[k][r] = (HALF0 + k == 1) ? cmul(xb, twist[r]) : xb;
    }
    if constexpr (kBound) {
      nx = wave_unit_reduce<F::T>(nx, OpAdd());
      // Cross-wave part of the reduction rides on the FFT's own barriers:
      // written here, read after the inverse transform; double-buffered on l.
      if constexpr (F::T > 64) {
        if ((threadIdx.x & 63) == 0) nslot[l & 1][threadIdx.x >> 6] = nx;
      }
    }
    F::template forward<KH>(x, lds, tw, tau);
#pragma unroll
    for (int k = 0; k < KH; ++k)
#pragma unroll
      for (int i = 0; i < F::R; ++i) x[k][i] = cmul(x[k][i], Hr[k][i]);
    F::template inverse<KH>(x, lds, tw, tau);
    float xn = 0.f;
    if constexpr (kBound) {
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
      float2 y = (HALF0 == 1) ? cmulc(x[0][r], twist[r]) : x[0][r];
      if constexpr (KH == 2) y = cadd(y, cmulc(x[1][r], twist[r]));
      acc0[r] = fmaf(f[r], y.x, acc0[r]);
      acc1[r] = fmaf(f[r], y.y, acc1[r]);
      if constexpr (kBound) bound[r] = fmaf(f[r], xn, bound[r]);
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
  constexpr int KH = C::KH;
  __shared__ float2 lds_all[C::CONV_LDS_SLOTS];
  __shared__ float red[C::WAVES];
  __shared__ float nslot[2][C::WAVES];
  const int g = threadIdx.x / F::T, tau = threadIdx.x % F::T;
  const int pairs = (d + 2) / 2;
  int unit = xcd_block(blockIdx.x, gridDim.x) * C::G + g;
  const bool active = unit < units;
  if (!active) unit = units - 1;  // keep the barriers uniform; results discarded
  const int cp = unit % pairs;
  const int rest = unit / pairs;
  const int hs = rest % C::HSPLIT, bh = rest / C::HSPLIT, h = bh % H;
  const int c0 = 2 * cp, c1 = 2 * cp + 1;
  float2* lds = lds_all + g * (F::P > 1 ? KH * F::LDS : 0);

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
  if (active && hs == 0 && tau == 0) {
    if (c0 < d) colmax[static_cast<size_t>(bh) * d + c0] = mx0;
    if (c1 < d) colmax[static_cast<size_t>(bh) * d + c1] = mx1;
  }

  // Spectrum halves in registers, in the order the forward transform leaves them.
  float2 Hr[KH][F::R];
#pragma unroll
  for (int k = 0; k < KH; ++k) {
    const float2* __restrict__ Hh = Hs + (static_cast<size_t>(h) * 2 + hs * KH + k) * F::N;
#pragma unroll
    for (int i = 0; i < F::R; ++i) Hr[k][i] = Hh[F::frequency_of(F::spectrum_pos(tau, i))];
  }

  float acc0[F::R], acc1[F::R], bound[F::R];
#pragma unroll
  for (int r = 0; r < F::R; ++r) acc0[r] = acc1[r] = bound[r] = 0.f;

  const float* __restrict__ pk = phik + static_cast<size_t>(bh) * m * F::N;
  const float* __restrict__ pq = phiq + static_cast<size_t>(bh) * m * F::N;
  if constexpr (KH == 2) {
    conv_loop<F, C::WAVES, 2, 0>(pk, pq, tw, v0, v1, Hr, lds, nslot, tau, m, acc0, acc1, bound);
  } else {
    if (hs)
      conv_loop<F, C::WAVES, 1, 1>(pk, pq, tw, v0, v1, Hr, lds, nslot, tau, m, acc0, acc1, bound);
    else
      conv_loop<F, C::WAVES, 1, 0>(pk, pq, tw, v0, v1, Hr, lds, nslot, tau, m, acc0, acc1, bound);
  }

  if (active) {
    float* __restrict__ out = part + ((static_cast<size_t>(bh) * C::HSPLIT + hs) * (d + 1) + c0) * n;
    float* __restrict__ bout = bnd + (static_cast<size_t>(bh) * pairs + cp) * n;
#pragma unroll
    for (int r = 0; r < F::R; ++r) {
      const int pos = tau + F::T * r;
      if (pos < n) {
        out[pos] = acc0[r] * s0;
        if (c1 <= d) out[n + pos] = acc1[r] * s1;
        if (hs == 0) bout[pos] = bound[r];
      }
    }
  }
}

// -------------------------------------------------------------- combine --
// z[bh][i][c] = sum_s P_s[c][i] / sum_s P_s[d][i],  P = part[bh], s < nsplit,
// and the certification of each row.  With K = kGamma u log2(L) ||h||_2 / sqrt(L),
// the error model of common.hpp bounds the rounding error of numerator c by
// K bnd[p(c)][i] s_c (+ a part relative to the value itself) and that of the
// denominator by K bnd[p(d)][i], p(c) = c / 2 the packed pair of column c.  A
// row whose normwise relative bound exceeds kTau is queued for k_fixup.
__global__ __launch_bounds__(256) void k_combine(const float* __restrict__ part, const float* __restrict__ bnd,
                                                 const float* __restrict__ colmax,
                                                 const float2* __restrict__ hnorm, float* __restrict__ z,
                                                 unsigned* __restrict__ fix, int BH, int H, int n, int log2N,
                                                 int d, int nsplit, int tiles_n) {
  __shared__ float tile[kMaxD + 1][65];
  __shared__ float btile[kMaxD / 2 + 1][65];
  __shared__ float scol[kMaxD + 1];
  __shared__ float zmax[64];
  const int bh = blockIdx.x / tiles_n, i0 = (blockIdx.x % tiles_n) * 64;
  const int h = bh % H;
  const int pairs = (d + 2) / 2;
  const float* __restrict__ p0 = part + static_cast<size_t>(bh) * nsplit * (d + 1) * n;
  const float* __restrict__ bb = bnd + static_cast<size_t>(bh) * pairs * n;
  for (int e = threadIdx.x; e < (d + 1) * 64; e += 256) {
    const int c = e >> 6, i = e & 63;
    const int pos = i0 + i;
    float t = 1.f;
    if (pos < n) {
      t = p0[static_cast<size_t>(c) * n + pos];
      for (int sp = 1; sp < nsplit; ++sp) t += p0[(static_cast<size_t>(sp) * (d + 1) + c) * n + pos];
    }
    tile[c][i] = t;
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
    bool flag = false;
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
      flag = !ok;
    }
    // One wave holds the tile's 64 rows: append its uncertified rows, in
    // order, to the head's queue (fix[0..BH) counts, fix[BH] total, then the
    // lists fix[BH + 1 + bh * n + slot]).
    const unsigned long long mask = __ballot(flag);
    if (mask != 0ull) {
      const int nflag = __popcll(mask);
      unsigned base = 0;
      if (threadIdx.x == 0) {
        base = atomicAdd(&fix[bh], static_cast<unsigned>(nflag));
        atomicAdd(&fix[BH], static_cast<unsigned>(nflag));
      }
      base = __shfl(base, 0);
      if (flag) {
        const int rank = __popcll(mask & ((1ull << threadIdx.x) - 1ull));
        fix[BH + 1 + static_cast<size_t>(bh) * n + base + rank] = static_cast<unsigned>(pos);
      }
    }
  }
}

// ---------------------------------------------------------------- fixup --
// Exact evaluation of Eq. (10) for the rows k_combine could not certify.  Work
// group (bh, k) of a fixed grid takes groups k, k + kFixPerHead, ... of 8
// queued rows of head bh:
//   P_rj = c_{j-i_r} phi(q_{i_r}) . phi(k_j)    (only keys with a finite b_{j-i_r})
//   z_r  = sum_j P_rj v_j / sum_j P_rj          (chunk sums in fp32, totals in fp64)
// Keys go in chunks of 1024 aligned to multiples of 1024 (so a row's sums do
// not depend on which rows share its group: the result is deterministic):
// each thread forms P for 4 keys x 8 rows (one load of phi(k) feeds 8 rows),
// then threads split by value column and key subset accumulate P v'.  Rows
// not queued keep the FFT result.  Every work-group exits when its head's
// queue is done.
constexpr int kFixRows = 8;
constexpr int kFixChunk = 1024;
constexpr int kFixPerHead = 32;

__global__ __launch_bounds__(256) void k_fixup(const float* __restrict__ phiq, const float* __restrict__ phik,
                                               const void* __restrict__ vraw, int v_bf16,
                                               const float* __restrict__ b, float* __restrict__ z,
                                               const unsigned* __restrict__ fix, int BH, int H, int n, int ld,
                                               int d, int m) {
  // P chunk, reused after the key loop for the per-thread partial sums of P v'
  __shared__ __align__(16) float sp[kFixRows][kFixChunk];
  static_assert(sizeof(float) * kFixRows * kFixChunk >= sizeof(double) * 256 * kFixRows, "red fits in sp");
  double (*red)[kFixRows] = reinterpret_cast<double (*)[kFixRows]>(&sp[0][0]);
  extern __shared__ __align__(16) float sq_dyn[];  // phi(q) of the group's rows, [l][r], m * 8 floats
  float (*sq)[kFixRows] = reinterpret_cast<float (*)[kFixRows]>(sq_dyn);
  __shared__ int smin, smax;
  const int tid = threadIdx.x;
  const int cols = d + 1;
  const int nsub = 256 / cols;                 // key subsets in the accumulation
  const int col = tid % cols, sub = tid / cols;
  // slot-major order: the first group of every head is dispatched first
  const int bh = blockIdx.x % BH, kslot = blockIdx.x / BH;
  if (bh >= BH) return;
  const unsigned count = fix[bh];
  const unsigned* __restrict__ list = fix + BH + 1 + static_cast<size_t>(bh) * n;
  const int ngroups = static_cast<int>((count + kFixRows - 1) / kFixRows);
  if (kslot >= ngroups) return;                // uniform per work-group
  {
    const int h = bh % H;
    const float* __restrict__ bhv = b + static_cast<size_t>(h) * (2 * n - 1);
    const float* __restrict__ pq = phiq + static_cast<size_t>(bh) * m * ld;
    const float* __restrict__ pk = phik + static_cast<size_t>(bh) * m * ld;
    const size_t vbase = static_cast<size_t>(bh) * n * d;

    // Range of s = t + n - 1 where b_t is finite.
    if (tid == 0) {
      smin = 2 * n;
      smax = -1;
    }
    __syncthreads();
    int lo = 2 * n, hi = -1;
    for (int sidx = tid; sidx < 2 * n - 1; sidx += 256)
      if (bhv[sidx] != -INFINITY) {
        lo = min(lo, sidx);
        hi = max(hi, sidx);
      }
    atomicMin(&smin, lo);
    atomicMax(&smax, hi);
    __syncthreads();
    const int s_lo = smin, s_hi = smax;

    for (int grp = kslot; grp < ngroups; grp += kFixPerHead) {
      int rows[kFixRows];
      int first = n, last = -1;
#pragma unroll
      for (int r = 0; r < kFixRows; ++r) {
        const unsigned slot = static_cast<unsigned>(grp * kFixRows + r);
        rows[r] = slot < count ? static_cast<int>(list[slot]) : -1;
        if (rows[r] >= 0) {
          first = min(first, rows[r]);
          last = max(last, rows[r]);
        }
      }
      const int jlo = max(0, first + s_lo - (n - 1));
      const int jhi = min(n - 1, last + s_hi - (n - 1));

      __syncthreads();
      for (int e2 = tid; e2 < m * kFixRows; e2 += 256) {
        const int l = e2 / kFixRows, r = e2 % kFixRows;
        sq[l][r] = rows[r] >= 0 ? pq[static_cast<size_t>(l) * ld + rows[r]] : 0.f;
      }
      double acc[kFixRows];
#pragma unroll
      for (int r = 0; r < kFixRows; ++r) acc[r] = 0.0;

      for (int jc = (jlo / kFixChunk) * kFixChunk; jc <= jhi; jc += kFixChunk) {
        __syncthreads();  // sq staged / previous chunk's sp consumed
        float kk[kFixRows][4];
#pragma unroll
        for (int r = 0; r < kFixRows; ++r)
#pragma unroll
          for (int q = 0; q < 4; ++q) kk[r][q] = 0.f;
        int jj[4];
#pragma unroll
        for (int q = 0; q < 4; ++q) jj[q] = min(jc + tid + 256 * q, n - 1);
#pragma unroll 8
        for (int l = 0; l < m; ++l) {
          float kv[4];
#pragma unroll
          for (int q = 0; q < 4; ++q) kv[q] = pk[static_cast<size_t>(l) * ld + jj[q]];
          const float4 qa = *reinterpret_cast<const float4*>(&sq[l][0]);
          const float4 qb = *reinterpret_cast<const float4*>(&sq[l][4]);
          const float qr[8] = {qa.x, qa.y, qa.z, qa.w, qb.x, qb.y, qb.z, qb.w};
#pragma unroll
          for (int r = 0; r < kFixRows; ++r)
#pragma unroll
            for (int q = 0; q < 4; ++q) kk[r][q] = fmaf(qr[r], kv[q], kk[r][q]);
        }
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int j = jc + tid + 256 * q;
#pragma unroll
          for (int r = 0; r < kFixRows; ++r) {
            float p = 0.f;
            if (rows[r] >= 0 && j >= jlo && j <= jhi) {
              const float bj = bhv[j - rows[r] + n - 1];
              if (bj != -INFINITY) p = kk[r][q] * expf(bj);
            }
            sp[r][tid + 256 * q] = p;
          }
        }
        __syncthreads();
        if (sub < nsub) {
          float part[kFixRows];
#pragma unroll
          for (int r = 0; r < kFixRows; ++r) part[r] = 0.f;
          const int jend = min(kFixChunk, jhi - jc + 1);
          auto vload = [&](int j) -> float {
            if (col == d) return 1.f;
            const size_t idx = vbase + static_cast<size_t>(jc + j) * d + col;
            return v_bf16 ? to_f32(static_cast<const uint16_t*>(vraw)[idx]) : static_cast<const float*>(vraw)[idx];
          };
          // 8 keys per step so that 8 loads of v are in flight at once
          int j = sub;
          for (; j + 7 * nsub < jend; j += 8 * nsub) {
            float vv[8];
#pragma unroll
            for (int u = 0; u < 8; ++u) vv[u] = vload(j + u * nsub);
#pragma unroll
            for (int u = 0; u < 8; ++u)
#pragma unroll
              for (int r = 0; r < kFixRows; ++r) part[r] = fmaf(sp[r][j + u * nsub], vv[u], part[r]);
          }
          for (; j < jend; j += nsub) {
            const float vv = vload(j);
#pragma unroll
            for (int r = 0; r < kFixRows; ++r) part[r] = fmaf(sp[r][j], vv, part[r]);
          }
#pragma unroll
          for (int r = 0; r < kFixRows; ++r) acc[r] += static_cast<double>(part[r]);
        }
      }
      // sum the key subsets: thread (col, sub) -> red, then thread col < cols adds them up
      __syncthreads();  // red aliases sp
#pragma unroll
      for (int r = 0; r < kFixRows; ++r) red[tid][r] = acc[r];
      __syncthreads();
      if (tid < cols) {
#pragma unroll
        for (int r = 0; r < kFixRows; ++r) {
          double s2 = red[tid][r];
          for (int sb = 1; sb < nsub; ++sb) s2 += red[sb * cols + tid][r];
          acc[r] = s2;
        }
      }
      __syncthreads();
      if (tid < cols) {
#pragma unroll
        for (int r = 0; r < kFixRows; ++r) red[tid][r] = acc[r];
      }
      __syncthreads();
      if (tid < d) {
#pragma unroll
        for (int r = 0; r < kFixRows; ++r)
          if (rows[r] >= 0)
            z[(static_cast<size_t>(bh) * n + rows[r]) * d + tid] = static_cast<float>(red[tid][r] / red[d][r]);
      }
    }
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
hipError_t spectrum_l2(const float* b, const float2* tw, float2* Hs, float2* hnorm, int H, int n, hipStream_t st) {
  using C = Conf<L2>;
  const int blocks = (2 * H + C::G - 1) / C::G;
  hipLaunchKernelGGL(k_spectrum<L2>, dim3(blocks), dim3(C::THREADS), 0, st, b, tw, Hs, hnorm, H, n);
  return hipGetLastError();
}

template <int L2, typename TV>
hipError_t conv_l2(const float* phiq, const float* phik, const TV* v, const float2* Hs, const float2* tw,
                   float* part, float* bnd, float* colmax, int BH, int H, int n, int d, int m, hipStream_t st) {
  using C = Conf<L2>;
  const int units = BH * C::HSPLIT * ((d + 2) / 2);
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

hipError_t launch_spectrum(int l2, const float* b, const float2* tw, float2* Hs, float2* hnorm, int H, int n,
                           hipStream_t st) {
  return dispatch<SpectrumFn>(l2, b, tw, Hs, hnorm, H, n, st);
}

hipError_t launch_feature_map(bool bf16, const void* x0, const void* x1, const float* W, float* phi0, float* phi1,
                              int nsrc, bool feature_major, int ld, int BH, int H, int n, int d, int m,
                              unsigned* fix_counts, hipStream_t st) {
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
                         inv_sqrt_m, tiles_n, tiles_m, BH, fix_counts);
    else
      hipLaunchKernelGGL((k_feature_map<uint16_t, false>), grid, block, 0, st, a, c, W, phi0, phi1, H, n, ld, d,
                         m, inv_sqrt_m, tiles_n, tiles_m, BH, fix_counts);
  } else {
    const float* a = static_cast<const float*>(x0);
    const float* c = static_cast<const float*>(x1);
    if (feature_major)
      hipLaunchKernelGGL((k_feature_map<float, true>), grid, block, 0, st, a, c, W, phi0, phi1, H, n, ld, d, m,
                         inv_sqrt_m, tiles_n, tiles_m, BH, fix_counts);
    else
      hipLaunchKernelGGL((k_feature_map<float, false>), grid, block, 0, st, a, c, W, phi0, phi1, H, n, ld, d, m,
                         inv_sqrt_m, tiles_n, tiles_m, BH, fix_counts);
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

template <int L2>
struct SplitFn {
  static hipError_t run(int* out) {
    *out = Conf<L2>::HSPLIT;
    return hipSuccess;
  }
};

int conv_split(int l2) {
  int s = 2;
  dispatch<SplitFn>(l2, &s);
  return s;
}

hipError_t launch_combine(const float* part, const float* bnd, const float* colmax, const float2* hnorm, float* z,
                          unsigned* fix, int BH, int H, int n, int l2, int d, hipStream_t st) {
  const int tiles_n = (n + 63) / 64;
  hipLaunchKernelGGL(k_combine, dim3(BH * tiles_n), dim3(256), 0, st, part, bnd, colmax, hnorm, z, fix, BH, H, n,
                     l2, d, conv_split(l2), tiles_n);
  return hipGetLastError();
}

hipError_t launch_fixup(const float* phiq, const float* phik, const void* v, bool bf16, const float* b, float* z,
                        const unsigned* fix, int BH, int H, int n, int ld, int d, int m, hipStream_t st) {
  const long long blocks = static_cast<long long>(BH) * kFixPerHead;
  const size_t lds = static_cast<size_t>(m) * kFixRows * sizeof(float);
  hipLaunchKernelGGL(k_fixup, dim3(static_cast<unsigned>(blocks)), dim3(256), lds, st, phiq, phik, v, bf16 ? 1 : 0,
                     b, z, fix, BH, H, n, ld, d, m);
  return hipGetLastError();
}

hipError_t launch_toeplitz(int l2, const float* a, float* y, const float2* Hs, const float2* tw, int BH, int H,
                           int C, int n, hipStream_t st) {
  return dispatch<ToeplitzFn>(l2, a, y, Hs, tw, BH, H, C, n, st);
}

}  // namespace krpe
