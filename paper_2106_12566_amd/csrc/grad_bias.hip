// Gradient of the relative positional bias b (backward pass): the
// correlation spectra of the channel pairs, their sum per head, its inverse
// per residue class and the gradient per offset.  In a translation unit of
// its own so that the convolution kernel's code generation does not change
// with it.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>

#include "common.hpp"
#include "launch.hpp"

namespace krpe {

// Gradient of b.  dL/dC_ij = (Gh V'^T)_ij (Phi_q Phi_k^T)_ij, so
//   dc_t = sum_l sum_c sum_i (phi_l(q_i) Gh_ic) (phi_l(k_{i+t}) V'_{i+t,c}),
// a cross-correlation of the channels a_lc = phi_l(q) o Gh_c and
// x_lc = phi_l(k) o V'_c summed over (l, c), and db_t = dc_t c_t.  In the
// frequency domain (zero-padded to 2N, so lags |t| < n do not wrap) the sum
// is one spectrum, S = sum_lc conj(A_lc) X_lc.  Two columns are packed as
// one complex signal like the forward's: with P = F(a_l0 + i a_l1),
// Q = F(x_l0 + i x_l1), Re F^-1(conj(P) Q) = corr(a_l0, x_l0) + corr(a_l1, x_l1)
// (the cross terms are imaginary), so a unit accumulates conj(P) Q over its
// features for its residue classes.  Units and transforms as in the
// convolution kernel; the spectra go to spart[bh][pair][r][i * T + tau]
// (register order of class r).
template <typename C, int R0>
__device__ __forceinline__ void corr_loop(const float* __restrict__ pk, const float* __restrict__ pq,
                                          const float2* __restrict__ vp, const float2* __restrict__ gp,
                                          const float2* __restrict__ tw, float2* lds, int tau, int m,
                                          float2 (&acc)[C::KH][C::F::R]) {
  using F = typename C::F;
  constexpr int FOLD = C::FOLD, KH = C::KH, S = C::S;
  constexpr bool MERGE = F::P > 1, REG = C::VREG && FOLD == 1;
  constexpr int NP = FOLD * F::N;
  float2 vx[REG ? FOLD : 1][REG ? F::R : 1], gx[REG ? FOLD : 1][REG ? F::R : 1];
  if constexpr (REG) {
#pragma unroll
    for (int p = 0; p < FOLD; ++p)
#pragma unroll
      for (int i = 0; i < F::R; ++i) {
        vx[p][i] = vp[tau + F::T * i + p * F::N];
        gx[p][i] = gp[tau + F::T * i + p * F::N];
      }
  }
  float2 w0[KH][F::R];
#pragma unroll
  for (int k = 0; k < KH; ++k)
#pragma unroll
    for (int i = 0; i < F::R; ++i)
      w0[k][i] = MERGE ? tw[tau * (R0 + k + S * i)] : tw[(R0 + k) * (tau + F::T * i)];
  // class transform input of a real envelope e times a column pair c
  auto form = [&](const float (&e)[FOLD][F::R], auto colv, float2 (&x)[KH][F::R]) {
#pragma unroll
    for (int i = 0; i < F::R; ++i) {
      float2 xb[FOLD];
#pragma unroll
      for (int p = 0; p < FOLD; ++p) {
        const float2 c = colv(p, i);
        xb[p] = make_float2(e[p][i] * c.x, e[p][i] * c.y);
      }
      constexpr_for<KH>([&](auto kc) {
        constexpr int k = decltype(kc)::value, r = R0 + k;
        float2 u = xb[0];
#pragma unroll
        for (int p = 1; p < FOLD; ++p) u = cadd(u, rot_dyn<S, false>(xb[p], p * r));
        if constexpr (r == 0) {
          x[k][i] = u;
        } else if constexpr (MERGE) {
          x[k][i] = rot_dyn<F::R * S, false>(u, r * i);
        } else {
          x[k][i] = cmul(u, w0[k][i]);
        }
      });
    }
  };
  // The next transform's first pass writes positions that other threads
  // read in this one's last pass: a work-group barrier between transforms.
  auto transform = [&](float2 (&x)[KH][F::R]) {
    if constexpr (MERGE) {
      F::template forward_w0<KH>(x, lds, tw, tau, w0);
    } else {
      F::template forward<KH>(x, lds, tw, tau);
    }
    if constexpr (F::P > 1) __syncthreads();
  };
  for (int l = 0; l < m; ++l) {
    const float* __restrict__ pkl = pk + static_cast<size_t>(l) * NP;
    const float* __restrict__ pql = pq + static_cast<size_t>(l) * NP;
    float a[FOLD][F::R], f[FOLD][F::R];
#pragma unroll
    for (int p = 0; p < FOLD; ++p)
#pragma unroll
      for (int i = 0; i < F::R; ++i) {
        a[p][i] = pkl[tau + F::T * i + p * F::N];
        f[p][i] = pql[tau + F::T * i + p * F::N];
      }
    float2 xq[KH][F::R], xp[KH][F::R];
    form(a, [&](int p, int i) { return REG ? vx[REG ? p : 0][REG ? i : 0] : vp[tau + F::T * i + p * F::N]; }, xq);
    transform(xq);
    form(f, [&](int p, int i) { return REG ? gx[REG ? p : 0][REG ? i : 0] : gp[tau + F::T * i + p * F::N]; }, xp);
    transform(xp);
#pragma unroll
    for (int k = 0; k < KH; ++k)
#pragma unroll
      for (int i = 0; i < F::R; ++i) {
        // acc += conj(P) Q
        acc[k][i].x = fmaf(xp[k][i].x, xq[k][i].x, fmaf(xp[k][i].y, xq[k][i].y, acc[k][i].x));
        acc[k][i].y = fmaf(xp[k][i].x, xq[k][i].y, fmaf(-xp[k][i].y, xq[k][i].x, acc[k][i].y));
      }
  }
}

template <typename C, int HS = 0>
__device__ __forceinline__ void corr_split(int hs, const float* __restrict__ pk, const float* __restrict__ pq,
                                           const float2* __restrict__ vp, const float2* __restrict__ gp,
                                           const float2* __restrict__ tw, float2* lds, int tau, int m,
                                           float2 (&acc)[C::KH][C::F::R]) {
  if constexpr (HS < C::HSPLIT) {
    if (HS + 1 == C::HSPLIT || hs == HS) {
      corr_loop<C, HS * C::KH>(pk, pq, vp, gp, tw, lds, tau, m, acc);
    } else {
      corr_split<C, HS + 1>(hs, pk, pq, vp, gp, tw, lds, tau, m, acc);
    }
  }
}

// phiq/phik: [bh][m][N] (phi_bh_stride apart); V' and Gh packed as column
// pairs vpk/gpk [bh][pairs][N] (float2, unscaled).
// Two waves per SIMD (at most 256 registers, a few spilled) beat one wave
// with everything in registers: 13.2 -> 8.4 ms at n = 4096, 96 heads.
template <int L2>
__global__ __launch_bounds__(Conf<L2>::THREADS) __attribute__((amdgpu_waves_per_eu(Conf<L2>::WPE > 2 ? 2 : Conf<L2>::WPE))) void
k_corr_spectrum(const float* __restrict__ phiq, const float* __restrict__ phik, long long phi_bh_stride,
                const float2* __restrict__ vpk, const float2* __restrict__ gpk, const float2* __restrict__ tw,
                float2* __restrict__ spart, int pairs, int m, int units) {
  using C = Conf<L2>;
  using F = typename C::F;
  constexpr int KH = C::KH;
  __shared__ float2 lds_all[F::P > 1 ? C::G * KH * F::LDS : 1];
  const int g = C::G == 1 ? 0 : threadIdx.x / F::T, tau = C::G == 1 ? threadIdx.x : threadIdx.x % F::T;
  const int pairs_p = (pairs + C::G - 1) / C::G * C::G;
  const int unit = xcd_block(blockIdx.x, gridDim.x) * C::G + g;
  int cp = unit % pairs_p;
  const int rest = unit / pairs_p;
  const bool active = unit < units && cp < pairs;
  if (cp >= pairs) cp = pairs - 1;  // padding unit: keeps the barriers uniform, results discarded
  const int hs = rest % C::HSPLIT, bh = rest / C::HSPLIT;
  float2* lds = lds_all + g * (F::P > 1 ? KH * F::LDS : 0);
  const size_t prow = (static_cast<size_t>(bh) * pairs + cp) * C::N;
  float2 acc[KH][F::R];
#pragma unroll
  for (int k = 0; k < KH; ++k)
#pragma unroll
    for (int i = 0; i < F::R; ++i) acc[k][i] = make_float2(0.f, 0.f);
  corr_split<C>(hs, phik + bh * phi_bh_stride, phiq + bh * phi_bh_stride, vpk + prow, gpk + prow, tw, lds, tau, m,
                acc);
  if (active) {
#pragma unroll
    for (int k = 0; k < KH; ++k) {
      const int r = hs * KH + k;
      float2* __restrict__ out = spart + ((static_cast<size_t>(bh) * pairs + cp) * C::S + r) * F::N;
#pragma unroll
      for (int i = 0; i < F::R; ++i) out[i * F::T + tau] = acc[k][i];
    }
  }
}

// Column pairs of two feature-major arrays [bh][cols][N] as float2 [bh][pairs][N]
// (the second column of an odd last pair is 0).
__global__ void k_pack_pairs(const float* __restrict__ a, float2* __restrict__ out, int cols, int N,
                             long long total) {
  const long long e = static_cast<long long>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (e >= total) return;
  const int pairs = (cols + 1) / 2;
  const long long pos = e % N, t = e / N;
  const int p = static_cast<int>(t % pairs);
  const long long bh = t / pairs;
  const float* __restrict__ base = a + bh * cols * N;
  const int c0 = 2 * p, c1 = 2 * p + 1;
  out[e] = make_float2(base[static_cast<size_t>(c0) * N + pos], c1 < cols ? base[static_cast<size_t>(c1) * N + pos] : 0.f);
}

// S[h][r][e] = sum over the batch and the column pairs of spart[bh][pair][r][e].
__global__ void k_corr_reduce(const float2* __restrict__ spart, float2* __restrict__ Sh, int B, int H, int pairs,
                              int len, long long total) {
  const long long e = static_cast<long long>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (e >= total) return;
  const long long h = e / len, o = e % len;
  float2 s = make_float2(0.f, 0.f);
  for (int beta = 0; beta < B; ++beta)
    for (int p = 0; p < pairs; ++p) {
      const float2 v = spart[((static_cast<size_t>(beta) * H + h) * pairs + p) * len + o];
      s.x += v.x;
      s.y += v.y;
    }
  Sh[e] = s;
}

// y[h][r][j] = IDFT_{2N/S}(S_h class r)[j] in natural order (one unit per (head, class)).
template <int L2>
__global__ __launch_bounds__(Conf<L2>::THREADS) void k_corr_idft(const float2* __restrict__ Sh,
                                                                  const float2* __restrict__ tw,
                                                                  float2* __restrict__ y, int H) {
  using C = Conf<L2>;
  using F = typename C::F;
  __shared__ float2 lds[C::LDS_SLOTS];
  const int g = C::G == 1 ? 0 : threadIdx.x / F::T, tau = C::G == 1 ? threadIdx.x : threadIdx.x % F::T;
  const int units = C::S * H;
  int unit = blockIdx.x * C::G + g;
  const bool active = unit < units;
  if (!active) unit = units - 1;
  const float2* __restrict__ in = Sh + static_cast<size_t>(unit) * F::N;
  float2 x[F::R];
#pragma unroll
  for (int i = 0; i < F::R; ++i) x[i] = in[i * F::T + tau];
  F::inverse(x, lds + g * (F::P > 1 ? F::LDS : 0), tw, tau);
  if (active) {
    float2* __restrict__ out = y + static_cast<size_t>(unit) * F::N;
#pragma unroll
    for (int i = 0; i < F::R; ++i) out[tau + F::T * i] = x[i];
  }
}

// db[h][s] = c_t dc_t, t = s - (n - 1): the correlation at lag J = t mod 2N is
// (1/2N) sum_r Re(W_{2N}^{-r J} y[h][r][J mod L']), L' = 2N / S; 0 where b = -inf.
__global__ void k_db_final(const float2* __restrict__ y, const float2* __restrict__ tw, const float* __restrict__ b,
                           float* __restrict__ db, int n, int N2, int S, long long total) {
  const long long e = static_cast<long long>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (e >= total) return;
  const int len = 2 * n - 1;
  const long long h = e / len;
  const int s = static_cast<int>(e % len), t = s - (n - 1);
  const float bv = b[e];
  if (!(bv > -INFINITY)) {
    db[e] = 0.f;
    return;
  }
  const int J = t >= 0 ? t : N2 + t, LT = N2 / S;
  float acc = 0.f;
  for (int r = 0; r < S; ++r) {
    const float2 v = y[(static_cast<size_t>(h) * S + r) * LT + J % LT];
    const float2 w = tw[(static_cast<long long>(r) * J) % N2];  // W_{2N}^{rJ}; conj below
    acc += v.x * w.x + v.y * w.y;                              // Re(conj(w) v)
  }
  db[e] = acc / static_cast<float>(N2) * expf(bv);
}

namespace {

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
hipError_t db_l2(const float* phiq, const float* phik, long long phi_bh_stride, const float* gh, const float* vh,
                 const float2* tw, float2* gpk, float2* vpk, float2* spart, float2* Sh, float2* ycorr,
                 const float* b, float* db, int B, int H, int n, int cols, int m, hipStream_t st) {
  using C = Conf<L2>;
  const int BH = B * H, pairs = (cols + 1) / 2;
  const long long ptotal = static_cast<long long>(BH) * pairs * C::N;
  const unsigned pblocks = static_cast<unsigned>((ptotal + 255) / 256);
  hipLaunchKernelGGL(k_pack_pairs, dim3(pblocks), dim3(256), 0, st, gh, gpk, cols, C::N, ptotal);
  hipLaunchKernelGGL(k_pack_pairs, dim3(pblocks), dim3(256), 0, st, vh, vpk, cols, C::N, ptotal);
  const int pairs_p = (pairs + C::G - 1) / C::G * C::G;
  const long long units = static_cast<long long>(BH) * C::HSPLIT * pairs_p;
  hipLaunchKernelGGL(k_corr_spectrum<L2>, dim3(static_cast<unsigned>(units / C::G)), dim3(C::THREADS), 0, st, phiq,
                     phik, phi_bh_stride, vpk, gpk, tw, spart, pairs, m, static_cast<int>(units));
  if (hipError_t e = hipGetLastError(); e != hipSuccess) return e;
  const int len = 2 * C::N;  // S classes of 2N / S bins
  const long long rtotal = static_cast<long long>(H) * len;
  hipLaunchKernelGGL(k_corr_reduce, dim3(static_cast<unsigned>((rtotal + 255) / 256)), dim3(256), 0, st, spart, Sh,
                     B, H, pairs, len, rtotal);
  const int iblocks = (C::S * H + C::G - 1) / C::G;
  hipLaunchKernelGGL(k_corr_idft<L2>, dim3(static_cast<unsigned>(iblocks)), dim3(C::THREADS), 0, st, Sh, tw, ycorr,
                     H);
  const long long dtotal = static_cast<long long>(H) * (2 * n - 1);
  hipLaunchKernelGGL(k_db_final, dim3(static_cast<unsigned>((dtotal + 255) / 256)), dim3(256), 0, st, ycorr, tw, b,
                     db, n, 2 * C::N, C::S, dtotal);
  return hipGetLastError();
}

template <int L2>
struct DbFn {
  template <typename... A>
  static hipError_t run(A... a) { return db_l2<L2>(a...); }
};

}  // namespace

hipError_t launch_db(int l2, const float* phiq, const float* phik, long long phi_bh_stride, const float* gh,
                     const float* vh, const float2* tw, float2* gpk, float2* vpk, float2* spart, float2* Sh,
                     float2* ycorr, const float* b, float* db, int B, int H, int n, int cols, int m, hipStream_t st) {
  return dispatch<DbFn>(l2, phiq, phik, phi_bh_stride, gh, vh, tw, gpk, vpk, spart, Sh, ycorr, b, db, B, H, n, cols,
                        m, st);
}

}  // namespace krpe
