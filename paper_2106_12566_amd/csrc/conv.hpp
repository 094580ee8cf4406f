// The convolution kernel of the forward pass (Sec. 3.2, Eqs. (11)-(13) and
// the contraction of Eq. (10)) and its launch, as templates over log2 N.
// Included by kernels.hip, which instantiates the lengths up to 2^13, and by
// conv_top.hip, which instantiates 2^kMaxLog2N in a translation unit of its
// own (compiled with a different instruction-scheduling strategy).
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

#include "common.hpp"

namespace krpe {

// ---------------------------------------------- convolution + contraction --
// Unit u = ((bh * HSPLIT + hs) * pairs + cp).  The unit owns columns
// c0 = 2 cp, c1 = 2 cp + 1 of v' (packed and scaled by k_vprep) and the
// residue classes r = hs*KH .. hs*KH + KH - 1 of the length-2N spectrum.  For
// every feature l the two channels phi_l(k_j) v'_{j,c0} and phi_l(k_j) v'_{j,c1}
// (columns of A1 / A2, Eq. (11)) share the envelope phi_l(k), so packing them
// as the real and imaginary parts of one complex signal keeps their
// magnitudes alike: the FFT's rounding error, set by the pair's norm, stays
// proportional to each.
//
// Residue class r of the circular convolution y = h (*) x of length 2N, with
// x zero from N on, S = 2 FOLD classes and transforms of length LT = N / FOLD:
//   u_r[j]      = W_{2N}^{r j} sum_{p < FOLD} x[j + p LT] W_S^{p r}
//   y[i + q LT] = sum_r W_{2N}^{-r i} W_S^{-q r} IDFT_LT(H_r * DFT_LT(u_r))[i]
// for j, i < LT and q < FOLD (the outputs below N), H_r as in k_spectrum.
//
// Writes the partial numerators / denominator of Eq. (10) of its classes
//   part[bh][hs][c][i] = s_c sum_l phi_l(q_i) (C_hs a_{l,c})_i,   c in {c0, c1}.
// phi rows are [m][N] per (batch, head), phi_bh_stride apart (0 broadcasts one
// set of rows to every head).
//
// The twist W_{2N}^{r j} of class r at position j = tau + T i splits as
// W_{2N}^{r tau} W_{RS}^{r i} (2N = R S T): the second factor is a compile-time constant
// per register, the first is folded into the twiddles of the first pass
// (Fft::forward_w0: w0[s] = W_{2N}^{tau (r + S s)}); the inverse undoes both
// the same way.
template <typename C, int R0>
__device__ __forceinline__ void conv_loop(const float* __restrict__ pk, const float* __restrict__ pq,
                                          const float2* __restrict__ vrow, const float2* __restrict__ tw,
                                          const float2* __restrict__ Hh, float2* lds, int tau, int m,
                                          float (&acc0)[C::FOLD][C::F::R], float (&acc1)[C::FOLD][C::F::R]) {
  using F = typename C::F;
  constexpr int FOLD = C::FOLD, KH = C::KH, S = C::S;
  constexpr bool VREG = C::VREG, PREF = C::PREF, HREG = C::HREG, HOIST = C::HOIST;
  constexpr bool MERGE = F::P > 1;
  // One class per unit with v in registers: the per-register twist factor
  // W_{RS}^{r i} and the fold factors W_S^{p r} of the input are applied to v
  // once, phi_l(k) being real, so the fold is a plain sum of phi v.
  constexpr bool PRETWIST = MERGE && KH == 1 && VREG && R0 != 0;
  // The output twist W_{2N}^{-r i} W_S^{-q r} of a unit with one class does
  // not depend on the feature either: the accumulators hold the untwisted
  // sums of phi_l(q) IDFT(...) and are rotated once after the loop.
  constexpr bool POSTTWIST = MERGE && KH == 1 && R0 != 0;
  constexpr int NP = FOLD * F::N;  // row length of phi and v
  // With C::BUF, phi rows and value pairs are read through buffer resources:
  // the lane's byte offset in a VGPR, the feature's and register's offset in
  // an SGPR (no 64-bit address arithmetic per load).  Otherwise through plain
  // pointers.  With buffer reads the loop loads phi a feature ahead without a
  // branch: on its last iteration feature m, never used, which the range
  // check (it covers the VGPR offset only) does not stop.  That read stays
  // within one phi row past the unit's m rows, and the workspace layouts keep
  // a row of slack after every array the convolution reads as phi rows.
  constexpr bool BUF = C::BUF;
  const BufRd bk(pk, static_cast<uint32_t>(m) * NP * 4u), bq(pq, static_cast<uint32_t>(m) * NP * 4u);
  const BufRd bv(vrow, static_cast<uint32_t>(NP) * 8u);
  auto phi_at = [&](bool kside, int ta, int l, int p, int i) {
    if constexpr (BUF) {
      return (kside ? bk : bq).f32(static_cast<uint32_t>(ta) * 4u,
                                   static_cast<uint32_t>(l * NP + F::T * i + p * F::N) * 4u);
    } else {
      return (kside ? pk : pq)[static_cast<size_t>(l) * NP + ta + F::T * i + p * F::N];
    }
  };
  auto v_at = [&](int ta, int p, int i) {
    if constexpr (BUF) {
      return bv.f64(static_cast<uint32_t>(ta) * 8u, static_cast<uint32_t>(F::T * i + p * F::N) * 8u);
    } else {
      return vrow[ta + F::T * i + p * F::N];
    }
  };
  constexpr bool KS = true, QS = false;
  // Spectrum classes, register order (see k_spectrum): kept in registers when
  // the work-group is small enough, else re-read just before the product.
  float2 Hr[HREG ? KH : 1][F::R];
  if constexpr (HREG) {
#pragma unroll
    for (int k = 0; k < KH; ++k)
#pragma unroll
      for (int i = 0; i < F::R; ++i) Hr[k][i] = Hh[k * F::N + i * F::T + tau];
  }
  float2 vx[VREG ? FOLD : 1][VREG ? F::R : 1];
  if constexpr (VREG) {
#pragma unroll
    for (int p = 0; p < FOLD; ++p)
#pragma unroll
      for (int i = 0; i < F::R; ++i) {
        const float2 vv = v_at(tau, p, i);
        vx[p][i] = PRETWIST ? rot_dyn<S, false>(rot_dyn<F::R * S, false>(vv, R0 * i), p * R0) : vv;
      }
  }
  // Merged first-pass twiddles (MERGE), or the plain twists W_{2N}^{r j}
  // (single-pass transforms), of every class of the unit.
  float2 w0[KH][F::R];
  // With the extended table (C::TWC) the merged twiddles of thread ta are
  // read from the per-thread table, lanes at consecutive entries.
  auto load_w0 = [&](const float2* __restrict__ t, int ta) {
#pragma unroll
    for (int k = 0; k < KH; ++k)
#pragma unroll
      for (int i = 0; i < F::R; ++i)
        w0[k][i] = MERGE ? (C::TWC ? t[F::M_TAB + ((R0 + k) * F::R + i) * F::T + ta] : t[ta * (R0 + k + S * i)])
                         : t[(R0 + k) * (ta + F::T * i)];
  };
  if constexpr (HOIST) load_w0(tw, tau);
  // phi(k) of the next feature is loaded a whole feature ahead so that its
  // latency is hidden behind the transforms: with registers to spare (PREF) at
  // the top of the iteration, else (NEXTK) with this feature's phi(q) after
  // the inverse transform; with C::NEXTQ phi(q) too is loaded a feature
  // ahead.
  constexpr bool NEXTK = VREG && !PREF && BUF;
  constexpr bool NEXTQ = NEXTK && C::NEXTQ;
  constexpr bool AHEAD = PREF || NEXTK;
  float a_next[AHEAD ? FOLD : 1][AHEAD ? F::R : 1];
  float f_next[NEXTQ ? FOLD : 1][NEXTQ ? F::R : 1];
  if constexpr (AHEAD) {
#pragma unroll
    for (int p = 0; p < FOLD; ++p)
#pragma unroll
      for (int i = 0; i < F::R; ++i) a_next[p][i] = phi_at(KS, tau, 0, p, i);
  }
  if constexpr (NEXTQ) {
#pragma unroll
    for (int p = 0; p < FOLD; ++p)
#pragma unroll
      for (int i = 0; i < F::R; ++i) f_next[p][i] = phi_at(QS, tau, 0, p, i);
  }
  for (int l = 0; l < m; ++l) {
    // Large work-groups have too few registers to keep the loop-invariant
    // twiddles: hide the table pointer from loop-invariant code motion so they
    // are re-read (from L1) inside the transforms instead.
    const float2* __restrict__ twl = tw;
    const float2* __restrict__ Hl = Hh;
    int taul = tau;
    if constexpr (!HOIST) {
      asm volatile("" : "+s"(twl));
      asm volatile("" : "+v"(Hl));
      asm volatile("" : "+v"(taul));
      load_w0(twl, taul);
    }
    float a[FOLD][F::R], f[FOLD][F::R];
#pragma unroll
    for (int p = 0; p < FOLD; ++p)
#pragma unroll
      for (int i = 0; i < F::R; ++i)
        a[p][i] = AHEAD ? a_next[AHEAD ? p : 0][AHEAD ? i : 0] : phi_at(KS, taul, l, p, i);
    if constexpr (PREF) {
#pragma unroll
      for (int p = 0; p < FOLD; ++p)
#pragma unroll
        for (int i = 0; i < F::R; ++i) f[p][i] = phi_at(QS, tau, l, p, i);
      if (BUF || l + 1 < m) {  // (see the buffer reads above)
#pragma unroll
        for (int p = 0; p < FOLD; ++p)
#pragma unroll
          for (int i = 0; i < F::R; ++i) a_next[p][i] = phi_at(KS, tau, l + 1, p, i);
      }
    }
    float2 x[KH][F::R];
#pragma unroll
    for (int i = 0; i < F::R; ++i) {
      float2 xb[FOLD];
#pragma unroll
      for (int p = 0; p < FOLD; ++p) {
        const float2 vv = VREG ? vx[VREG ? p : 0][VREG ? i : 0] : v_at(taul, p, i);
        xb[p] = make_float2(a[p][i] * vv.x, a[p][i] * vv.y);
      }
      constexpr_for<KH>([&](auto kc) {
        constexpr int k = decltype(kc)::value, r = R0 + k;
        // fold: u = sum_p xb[p] W_S^{p r} (the factors already in v with PRETWIST)
        float2 u = xb[0];
#pragma unroll
        for (int p = 1; p < FOLD; ++p) u = cadd(u, PRETWIST ? xb[p] : rot_dyn<S, false>(xb[p], p * r));
        if constexpr (r == 0 || PRETWIST) {
          x[k][i] = u;
        } else if constexpr (MERGE) {
          x[k][i] = rot_dyn<F::R * S, false>(u, r * i);
        } else {
          x[k][i] = cmul(u, w0[k][i]);
        }
      });
    }
    if constexpr (MERGE) {
      F::template forward_w0<KH>(x, lds, twl, taul, w0);
    } else {
      F::template forward<KH>(x, lds, twl, taul);
    }
#pragma unroll
    for (int k = 0; k < KH; ++k)
#pragma unroll
      for (int i = 0; i < F::R; ++i)
        x[k][i] = cmul(x[k][i], HREG ? Hr[HREG ? k : 0][i] : Hl[k * F::N + i * F::T + taul]);
    if constexpr (!HOIST) {
      // fresh (opaque) copies: the twiddles are re-read rather than kept live
      // across both transforms
      asm volatile("" : "+s"(twl));
      asm volatile("" : "+v"(taul));
      load_w0(twl, taul);
    }
    if constexpr (MERGE) {
      F::template inverse_w0<KH>(x, lds, twl, taul, w0);
    } else {
      F::template inverse<KH>(x, lds, twl, taul);
    }
    if constexpr (!PREF) {
#pragma unroll
      for (int p = 0; p < FOLD; ++p)
#pragma unroll
        for (int i = 0; i < F::R; ++i) {
          // (the last iteration loads a feature m that is never used: see the
          // buffer reads above)
          if constexpr (NEXTQ) {
            f[p][i] = f_next[NEXTQ ? p : 0][NEXTQ ? i : 0];
            f_next[NEXTQ ? p : 0][NEXTQ ? i : 0] = phi_at(QS, taul, l + 1, p, i);
          } else {
            f[p][i] = phi_at(QS, taul, l, p, i);
          }
          if constexpr (NEXTK) a_next[NEXTK ? p : 0][NEXTK ? i : 0] = phi_at(KS, taul, l + 1, p, i);
        }
    }
#pragma unroll
    for (int i = 0; i < F::R; ++i) {
      float2 yk[KH];
      constexpr_for<KH>([&](auto kc) {
        constexpr int k = decltype(kc)::value, r = R0 + k;
        if constexpr (r == 0 || POSTTWIST) {
          yk[k] = x[k][i];
        } else if constexpr (MERGE) {
          yk[k] = rot_dyn<F::R * S, true>(x[k][i], r * i);
        } else {
          yk[k] = cmulc(x[k][i], w0[k][i]);
        }
      });
#pragma unroll
      for (int q = 0; q < FOLD; ++q) {
        float2 y = make_float2(0.f, 0.f);
#pragma unroll
        for (int k = 0; k < KH; ++k) {
          const float2 t = POSTTWIST ? yk[k] : rot_dyn<S, true>(yk[k], q * (R0 + k));  // W_S^{-q r}
          y = k == 0 ? t : cadd(y, t);
        }
        acc0[q][i] = fmaf(f[q][i], y.x, acc0[q][i]);
        acc1[q][i] = fmaf(f[q][i], y.y, acc1[q][i]);
      }
    }
  }
  if constexpr (POSTTWIST) {
#pragma unroll
    for (int q = 0; q < FOLD; ++q)
#pragma unroll
      for (int i = 0; i < F::R; ++i) {
        const float2 y = rot_dyn<S, true>(rot_dyn<F::R * S, true>(make_float2(acc0[q][i], acc1[q][i]), R0 * i),
                                          q * R0);
        acc0[q][i] = y.x;
        acc1[q][i] = y.y;
      }
  }
}

// Calls conv_loop with the first class of split hs as a compile-time constant.
template <typename C, int HS = 0>
__device__ __forceinline__ void conv_split(int hs, const float* __restrict__ pk, const float* __restrict__ pq,
                                           const float2* __restrict__ vrow, const float2* __restrict__ tw,
                                           const float2* __restrict__ Hh, float2* lds, int tau, int m,
                                           float (&acc0)[C::FOLD][C::F::R], float (&acc1)[C::FOLD][C::F::R]) {
  if constexpr (HS < C::HSPLIT) {
    if (HS + 1 == C::HSPLIT || hs == HS) {
      conv_loop<C, HS * C::KH>(pk, pq, vrow, tw, Hh, lds, tau, m, acc0, acc1);
    } else {
      conv_split<C, HS + 1>(hs, pk, pq, vrow, tw, Hh, lds, tau, m, acc0, acc1);
    }
  }
}

// Work units: (bh, key block J < nkb, feature split fs < fsplit, class split
// hs, column pair cp), unit-major in that order.  Key block J of a launch
// reads phi(k), the column pairs and their scales at batch index J BH + bh
// and the spectrum at J H + h; phi(q) at bh; the feature split takes features
// [fs mf, fs mf + mf) of the m, mf = ceil(m / fsplit).  Unit (bh, J, fs, hs)
// writes its own partial result, split index (J fsplit + fs) HSPLIT + hs of
// row bh, so the nkb fsplit HSPLIT partials of a row sum to the product.
// With nkb = fsplit = 1 this is one (bh, hs) per unit.  When hnorm is given,
// a unit whose spectrum has ||h||_1 = 0 (an all-zero block of C) skips the
// transforms and writes zeros.
template <int L2>
__global__ __launch_bounds__(Conf<L2>::THREADS) __attribute__((amdgpu_waves_per_eu(Conf<L2>::WPE))) void
k_conv_contract(
    const float* __restrict__ phiq, const float* __restrict__ phik, long long phi_bh_stride,
    const float2* __restrict__ vsc, const float* __restrict__ colmax, const float2* __restrict__ Hs,
    const float2* __restrict__ hnorm, const float2* __restrict__ tw, float* __restrict__ part, int BH, int H, int n,
    int cols, int m, int nkb, int fsplit, int units) {
  using C = Conf<L2>;
  using F = typename C::F;
  constexpr int KH = C::KH, FOLD = C::FOLD;
  __shared__ float2 lds_all[C::CONV_LDS_SLOTS];
  // With one unit per work-group the unit index is wave-uniform: say so, so
  // that per-unit pointers live in scalar registers.
  const int g = C::G == 1 ? 0 : threadIdx.x / F::T, tau = C::G == 1 ? threadIdx.x : threadIdx.x % F::T;
  const int pairs = (cols + 1) / 2;
  // Column pairs are padded to a multiple of G, so that the units of one
  // work-group share (bh, J, fs, hs): they run the same class split (same
  // barriers) and the same number of features.
  const int pairs_p = (pairs + C::G - 1) / C::G * C::G;
  const int unit = xcd_block(blockIdx.x, gridDim.x) * C::G + g;
  int cp = unit % pairs_p;
  const int rest = unit / pairs_p;
  const bool active = unit < units && cp < pairs;
  if (cp >= pairs) cp = pairs - 1;  // padding unit: keeps the barriers uniform, results discarded
  const int hs = rest % C::HSPLIT, vb = rest / C::HSPLIT;
  const int fs = vb % fsplit, jb = vb / fsplit;
  const int J = jb % nkb, bh = jb / nkb, h = bh % H;
  const int kb = J * BH + bh, hw = J * H + h;
  const int mf = (m + fsplit - 1) / fsplit, l0 = fs * mf;
  const int mcount = m - l0 < mf ? m - l0 : mf;
  const int c0 = 2 * cp, c1 = 2 * cp + 1;
  float2* lds = lds_all + g * (F::P > 1 ? KH * F::LDS : 0);
  const float2* __restrict__ vrow = vsc + (static_cast<size_t>(kb) * pairs + cp) * C::N;

  const float2* __restrict__ Hh = Hs + (static_cast<size_t>(hw) * C::S + hs * KH) * F::N;
  float acc0[FOLD][F::R], acc1[FOLD][F::R];
#pragma unroll
  for (int q = 0; q < FOLD; ++q)
#pragma unroll
    for (int i = 0; i < F::R; ++i) acc0[q][i] = acc1[q][i] = 0.f;

  const float* __restrict__ pk = phik + kb * phi_bh_stride + static_cast<size_t>(l0) * C::N;
  const float* __restrict__ pq = phiq + bh * phi_bh_stride + static_cast<size_t>(l0) * C::N;
  const bool live = mcount > 0 && (hnorm == nullptr || hnorm[hw].x != 0.f);
  if (live) conv_split<C>(hs, pk, pq, vrow, tw, Hh, lds, tau, mcount, acc0, acc1);

  if (active) {
    const float s0 = colmax[static_cast<size_t>(kb) * cols + c0];
    const float s1 = c1 < cols ? colmax[static_cast<size_t>(kb) * cols + c1] : 0.f;
    float* __restrict__ out = part + ((static_cast<size_t>(vb) * C::HSPLIT + hs) * cols + c0) * n;
#pragma unroll
    for (int q = 0; q < FOLD; ++q)
#pragma unroll
      for (int i = 0; i < F::R; ++i) {
        const int pos = tau + F::T * i + q * F::N;
        if (pos < n) {
          out[pos] = acc0[q][i] * (s0 > 0.f ? s0 : 1.f);
          if (c1 < cols) out[n + pos] = acc1[q][i] * (s1 > 0.f ? s1 : 1.f);
        }
      }
  }
}

// Launch of k_conv_contract<L2> over its work units.
template <int L2>
hipError_t conv_launch(const float* phiq, const float* phik, long long phi_bh_stride, const float2* vsc,
                       const float* colmax, const float2* Hs, const float2* hnorm, const float2* tw, float* part,
                       int BH, int H, int n, int cols, int m, int nkb, int fsplit, hipStream_t st) {
  using C = Conf<L2>;
  const int pairs_p = ((cols + 1) / 2 + C::G - 1) / C::G * C::G;
  const long long units = static_cast<long long>(BH) * nkb * fsplit * C::HSPLIT * pairs_p;
  const long long blocks = units / C::G;
  hipLaunchKernelGGL(k_conv_contract<L2>, dim3(static_cast<unsigned>(blocks)), dim3(C::THREADS), 0, st, phiq, phik,
                     phi_bh_stride, vsc, colmax, Hs, hnorm, tw, part, BH, H, n, cols, m, nkb, fsplit,
                     static_cast<int>(units));
  return hipGetLastError();
}

// The N = 2^kMaxLog2N instance (conv_top.hip).
hipError_t conv_launch_top(const float* phiq, const float* phik, long long phi_bh_stride, const float2* vsc,
                           const float* colmax, const float2* Hs, const float2* hnorm, const float2* tw, float* part,
                           int BH, int H, int n, int cols, int m, int nkb, int fsplit, hipStream_t st);

}  // namespace krpe
