// Register + LDS resident complex FFT for gfx950.
//
// The Toeplitz products of Eqs. (12)-(13) are done as FFT convolutions.  This
// header holds the transform only; the kernels that use it are in kernels.hip.
//
// A transform of length N = 2^LOG2N is owned by T = N / R threads, each
// holding R = 2^LOG2R complex values in registers.  It is a sequence of P
// in-place Cooley-Tukey passes.  Pass p splits every sub-problem of length
// L_p into R_p interleaved sub-sequences: its butterflies read the R_p values
// at positions  q*L_p + t + S_p*r  (S_p = L_p / R_p, r < R_p), take a length
// R_p DFT in registers, multiply by the twiddles W_{L_p}^{t*s} and write the
// R_p results back to the same positions (output s to q*L_p + t + S_p*s).
// Output s of sub-problem q is the start of sub-problem (q*R_p + s) of pass
// p+1.  Because every pass writes exactly the positions it read, one barrier
// per pass boundary is enough, and the inverse transform replays the passes
// backwards (conjugate twiddles, conjugate DFTs) on the same positions.
//
// Data enters pass 0 in registers (thread tau holds positions tau + T*r) and
// leaves the last pass in registers in digit-reversed order; the inverse takes
// that order and returns positions tau + T*r.  So per-position data of a
// thread (loads, twists, accumulators) never has to be exchanged.
//
// Positions are padded in LDS by one element per R to spread the strided
// accesses of late passes over the banks.
#pragma once

#include <hip/hip_runtime.h>

#include <type_traits>

namespace krpe {

// ---------------------------------------------------------------- complex --
__device__ __forceinline__ float2 cadd(float2 a, float2 b) { return make_float2(a.x + b.x, a.y + b.y); }
__device__ __forceinline__ float2 csub(float2 a, float2 b) { return make_float2(a.x - b.x, a.y - b.y); }
__device__ __forceinline__ float2 cmul(float2 a, float2 b) {
  return make_float2(a.x * b.x - a.y * b.y, a.x * b.y + a.y * b.x);
}
// a * conj(b)
__device__ __forceinline__ float2 cmulc(float2 a, float2 b) {
  return make_float2(a.x * b.x + a.y * b.y, a.y * b.x - a.x * b.y);
}

// cos(2*pi*k/128) for k = 0..32 (first quadrant, exact zero at 32).
__host__ __device__ constexpr float quarter_cos128(int k) {
  constexpr float q[33] = {
                            1.0f, 0.99879545620517241f, 0.99518472667219693f,
                            0.98917650996478101f, 0.98078528040323043f, 0.97003125319454397f,
                            0.95694033573220882f, 0.94154406518302081f, 0.92387953251128674f,
                            0.90398929312344334f, 0.88192126434835505f, 0.85772861000027212f,
                            0.83146961230254524f, 0.80320753148064494f, 0.77301045336273699f,
                            0.74095112535495911f, 0.70710678118654757f, 0.67155895484701833f,
                            0.63439328416364549f, 0.59569930449243347f, 0.55557023301960229f,
                            0.51410274419322166f, 0.47139673682599781f, 0.4275550934302822f,
                            0.38268343236508984f, 0.33688985339222005f, 0.29028467725446233f,
                            0.24298017990326398f, 0.19509032201612833f, 0.14673047445536175f,
                            0.09801714032956077f, 0.049067674327418126f, 0.0f};
  return q[k];
}
// cos(2*pi*k/128) for any k, by quadrant symmetry.
__host__ __device__ constexpr float cos128(int k) {
  k = ((k % 128) + 128) % 128;
  if (k <= 32) return quarter_cos128(k);
  if (k <= 64) return -quarter_cos128(64 - k);
  if (k <= 96) return -quarter_cos128(k - 64);
  return quarter_cos128(128 - k);
}
__host__ __device__ constexpr float sin128(int k) { return cos128(k - 32); }
__host__ __device__ constexpr float cos64(int k) { return cos128(2 * k); }
__host__ __device__ constexpr float sin64(int k) { return sin128(2 * k); }

// v * exp(sign * 2*pi*i * K / NN), sign = -1 for the forward transform and +1
// for the inverse.  NN divides 64.  Quarter turns are exact swaps.
template <int NN, int K, bool INV>
__device__ __forceinline__ float2 rot(float2 v) {
  static_assert(64 % NN == 0, "rot: NN must divide 64");
  constexpr int k = (((K % NN) + NN) % NN) * (64 / NN);  // angle in units of 2*pi/64
  constexpr int e = INV ? k : (64 - k) % 64;               // multiply by exp(+i 2*pi e/64)
  if constexpr (e == 0) {
    return v;
  } else if constexpr (e == 16) {
    return make_float2(-v.y, v.x);
  } else if constexpr (e == 32) {
    return make_float2(-v.x, -v.y);
  } else if constexpr (e == 48) {
    return make_float2(v.y, -v.x);
  } else {
    constexpr float c = cos64(e);
    constexpr float s = sin64(e);
    return make_float2(v.x * c - v.y * s, v.x * s + v.y * c);
  }
}

// fn(std::integral_constant<int, I>) for I = 0 .. N-1.
template <int N, int I = 0, typename Fn>
__device__ __forceinline__ void constexpr_for(Fn&& fn) {
  if constexpr (I < N) {
    fn(std::integral_constant<int, I>{});
    constexpr_for<N, I + 1>(fn);
  }
}

// v * exp(-+2 pi i K / NN), as rot below, for a K that is a constant once the
// loops around the call are unrolled; NN divides 128.
template <int NN, bool INV>
__device__ __forceinline__ float2 rot_dyn(float2 v, int K) {
  static_assert(128 % NN == 0, "rot_dyn: NN must divide 128");
  const int k = (((K % NN) + NN) % NN) * (128 / NN);
  const int e = INV ? k : (128 - k) % 128;  // multiply by exp(+2 pi i e / 128)
  if (e == 0) return v;
  if (e == 32) return make_float2(-v.y, v.x);
  if (e == 64) return make_float2(-v.x, -v.y);
  if (e == 96) return make_float2(v.y, -v.x);
  const float c = cos128(e), sn = sin128(e);
  return make_float2(v.x * c - v.y * sn, v.x * sn + v.y * c);
}

// ---------------------------------------------------- in-register DFTs --
// Dft<R, INV>::run<OFF, ST>(x): X[s] = sum_r x[OFF + ST*r] * W_R^{+-r*s}, in
// place, natural order at OFF + ST*s.  R = 4^a * 2^b up to 64, built as
// R = A * 4 with a radix-4 inner DFT over the stride-A sub-sequences, the
// W_R^{r0*s1} twiddles and a length-A outer DFT.
template <int R, bool INV>
struct Dft;

template <bool INV>
struct Dft<1, INV> {
  template <int OFF, int ST, int NR>
  __device__ __forceinline__ static void run(float2 (&)[NR]) {}
};

template <bool INV>
struct Dft<2, INV> {
  template <int OFF, int ST, int NR>
  __device__ __forceinline__ static void run(float2 (&x)[NR]) {
    const float2 a = x[OFF], b = x[OFF + ST];
    x[OFF] = cadd(a, b);
    x[OFF + ST] = csub(a, b);
  }
};

template <bool INV>
struct Dft<4, INV> {
  template <int OFF, int ST, int NR>
  __device__ __forceinline__ static void run(float2 (&x)[NR]) {
    const float2 a0 = x[OFF], a1 = x[OFF + ST], a2 = x[OFF + 2 * ST], a3 = x[OFF + 3 * ST];
    const float2 t0 = cadd(a0, a2), t1 = csub(a0, a2);
    const float2 t2 = cadd(a1, a3), t3 = rot<4, 1, INV>(csub(a1, a3));
    x[OFF] = cadd(t0, t2);
    x[OFF + 2 * ST] = csub(t0, t2);
    x[OFF + ST] = cadd(t1, t3);
    x[OFF + 3 * ST] = csub(t1, t3);
  }
};

template <int R, bool INV>
struct Dft {
  static_assert(R % 4 == 0 && R <= 64, "Dft: unsupported radix");
  static constexpr int A = R / 4;

  template <int R0, int S1, int NR>
  __device__ __forceinline__ static void twiddle_col(float2 (&y)[NR]) {
    y[R0 * 4 + S1] = rot<R, R0 * S1, INV>(y[R0 * 4 + S1]);
    if constexpr (S1 + 1 < 4) twiddle_col<R0, S1 + 1>(y);
  }
  template <int R0, int OFF, int ST, int NR>
  __device__ __forceinline__ static void inner(float2 (&x)[NR], float2 (&y)[R]) {
    // y[r0*4 + s1] = DFT4 over r1 of x[OFF + ST*(r0 + A*r1)]
#pragma unroll
    for (int r1 = 0; r1 < 4; ++r1) y[R0 * 4 + r1] = x[OFF + ST * (R0 + A * r1)];
    Dft<4, INV>::template run<R0 * 4, 1>(y);
    twiddle_col<R0, 0>(y);
    if constexpr (R0 + 1 < A) inner<R0 + 1, OFF, ST>(x, y);
  }
  template <int S1, int OFF, int ST, int NR>
  __device__ __forceinline__ static void outer(float2 (&x)[NR], float2 (&y)[R]) {
    // X[s1 + 4*s2] = DFT_A over r0 of y[r0*4 + s1]
    float2 col[A];
#pragma unroll
    for (int r0 = 0; r0 < A; ++r0) col[r0] = y[r0 * 4 + S1];
    Dft<A, INV>::template run<0, 1>(col);
#pragma unroll
    for (int s2 = 0; s2 < A; ++s2) x[OFF + ST * (S1 + 4 * s2)] = col[s2];
    if constexpr (S1 + 1 < 4) outer<S1 + 1, OFF, ST>(x, y);
  }
  template <int OFF, int ST, int NR>
  __device__ __forceinline__ static void run(float2 (&x)[NR]) {
    float2 y[R];
    inner<0, OFF, ST>(x, y);
    outer<0, OFF, ST>(x, y);
  }
};

// tan(2*pi*e/64) for e = 0..8 (exact 0 and 1 at the ends).
__host__ __device__ constexpr float tan64(int e) {
  constexpr float t[9] = {0.0f, 0.09849140335716425f, 0.198912367379658f, 0.3033466836073424f,
                          0.41421356237309503f, 0.5345111359507916f, 0.6681786379192989f,
                          0.8206787908286602f, 1.0f};
  return e >= 0 ? t[e] : -t[-e];
}

// Butterfly with a constant twiddle: p = a + w b, q = a - w b, w = exp(-+2 pi i
// K / NN) (sign as in rot).  w is split as i^qt * c (1 + i t) with the angle of
// c (1 + i t) within 45 degrees of the real axis: b (1 + i t) takes two FMAs,
// the quarter turn i^qt only renames and negates, and the scale c is folded
// into the four FMAs of the sum and difference, 6 instructions in place of
// the 8 of a complex product followed by an add and a subtract (4 adds when w
// is a power of i).
template <int NN, int K, bool INV>
__device__ __forceinline__ void twiddle_butterfly(float2 a, float2 b, float2& p, float2& q) {
  static_assert(64 % NN == 0, "twiddle_butterfly: NN must divide 64");
  constexpr int k = (((K % NN) + NN) % NN) * (64 / NN);
  constexpr int e = INV ? k : (64 - k) % 64;  // w = exp(+i 2 pi e / 64)
  constexpr int qt = ((e + 8) / 16) % 4;      // nearest quarter turn
  constexpr int er = e - 16 * (((e + 8) / 16));  // residual angle in [-8, 8)
  constexpr float t = tan64(er), c = cos64(er < 0 ? -er : er);
  float2 r = b;
  if constexpr (er != 0) r = make_float2(fmaf(-t, b.y, b.x), fmaf(t, b.x, b.y));
  if constexpr (qt == 1) r = make_float2(-r.y, r.x);
  if constexpr (qt == 2) r = make_float2(-r.x, -r.y);
  if constexpr (qt == 3) r = make_float2(r.y, -r.x);
  if constexpr (er == 0) {
    p = cadd(a, r);
    q = csub(a, r);
  } else {
    p = make_float2(fmaf(c, r.x, a.x), fmaf(c, r.y, a.y));
    q = make_float2(fmaf(-c, r.x, a.x), fmaf(-c, r.y, a.y));
  }
}

// Length 16 = 4 x 4 with the twiddles of the outer radix-4 stage fused into
// its butterflies: column s1 takes the DFT over r0 of W_16^{r0 s1} y[r0][s1],
// i.e. with w = W_16^{s1}:  t0, t1 = y0 +- w^2 y2;  u+, u- = y1 +- w^2 y3;
// X0, X2 = t0 +- w u+;  X1, X3 = t1 +- W_4 w u-.
template <bool INV>
struct Dft<16, INV> {
  template <int S1, int OFF, int ST, int NR>
  __device__ __forceinline__ static void column(float2 (&x)[NR], const float2 (&y)[16]) {
    float2 t0, t1, up, um, X0, X1, X2, X3;
    twiddle_butterfly<16, 2 * S1, INV>(y[0 * 4 + S1], y[2 * 4 + S1], t0, t1);
    twiddle_butterfly<16, 2 * S1, INV>(y[1 * 4 + S1], y[3 * 4 + S1], up, um);
    twiddle_butterfly<16, S1, INV>(t0, up, X0, X2);
    twiddle_butterfly<16, S1 + 4, INV>(t1, um, X1, X3);
    x[OFF + ST * (S1 + 0)] = X0;
    x[OFF + ST * (S1 + 4)] = X1;
    x[OFF + ST * (S1 + 8)] = X2;
    x[OFF + ST * (S1 + 12)] = X3;
  }
  template <int OFF, int ST, int NR>
  __device__ __forceinline__ static void run(float2 (&x)[NR]) {
    // y[r0*4 + s1] = DFT4 over r1 of x[OFF + ST*(r0 + 4 r1)]
    float2 y[16];
#pragma unroll
    for (int r0 = 0; r0 < 4; ++r0)
#pragma unroll
      for (int r1 = 0; r1 < 4; ++r1) y[r0 * 4 + r1] = x[OFF + ST * (r0 + 4 * r1)];
    Dft<4, INV>::template run<0, 1>(y);
    Dft<4, INV>::template run<4, 1>(y);
    Dft<4, INV>::template run<8, 1>(y);
    Dft<4, INV>::template run<12, 1>(y);
    column<0, OFF, ST>(x, y);
    column<1, OFF, ST>(x, y);
    column<2, OFF, ST>(x, y);
    column<3, OFF, ST>(x, y);
  }
};

// ------------------------------------------------------------- FFT plan --
// TWS = log2(table length / N): the twiddle table always holds W_M^k, k < M,
// for some M = N << TWS (M = 2N for a transform of the full half-length, 4N
// when the transform is a quarter of the circular length).
// TWC: the passes p >= 1 read their twiddles W_{L_p}^k (L_p = N >> (LR p),
// the pass's sub-problem length) from compact tables stored after 2 M
// entries of the table (see twc_offset), instead of every 2^(LR p + TWS)-th
// entry of W_M: a few KiB that stay in the L1 cache when the twiddles are
// re-read per transform rather than kept in registers.
// AFF: address LDS as pad(base) + constant per butterfly (see pad):
// one address register instead of one per value, which frees registers but
// lets the compiler pair accesses into 16-byte ds_read2 / ds_write2 forms,
// slower than 8-byte ones where the LDS is the busier pipe.
// PAD: LDS layout of the hand-overs (see pad); 0 keeps one padding slot per R
// positions.
template <int LOG2N_, int LOG2R_, int TWS = 1, bool TWC = false, bool AFF = false, int PAD = 0>
struct Fft {
  static constexpr int LOG2N = LOG2N_;
  static constexpr int N = 1 << LOG2N;
  static constexpr int LR = LOG2N < LOG2R_ ? LOG2N : LOG2R_;  // log2 of values per thread
  static constexpr int R = 1 << LR;
  static constexpr int T = N / R;                               // threads per transform
  static constexpr int P = LR == 0 ? 1 : (LOG2N + LR - 1) / LR;  // passes
  // log2 of the radix of pass p: LR for all passes but the last, which takes the rest.
  __host__ __device__ static constexpr int lr(int p) { return p + 1 < P ? LR : LOG2N - LR * (P - 1); }
  // Whether the LDS hand-over between passes p and p + 1 stays inside 64-lane
  // waves: every position a thread reads in pass p + 1 was written in pass p
  // by a thread of its own wave (the same pairs exchange data, in reverse,
  // in the inverse transform).
  __host__ __device__ static constexpr bool wave_local(int p) {
    if (T <= 64) return true;
    const int la = lr(p), lena = N >> (LR * p), spa = lena >> la;
    const int lb = lr(p + 1), rpb = 1 << lb, ub = R / rpb, lenb = N >> (LR * (p + 1)), spb = lenb >> lb;
    for (int tau = 0; tau < T; ++tau)
      for (int u = 0; u < ub; ++u) {
        const int bb = tau + T * u, base = (bb / spb) * lenb + bb % spb;
        for (int r = 0; r < rpb; ++r) {
          const int pos = base + spb * r;
          const int writer = ((pos / lena) * spa + pos % spa) % T;
          if (writer / 64 != tau / 64) return false;
        }
      }
    return true;
  }
  // LDS hand-over across boundary p.  Inside a wave, LDS operations are
  // performed in order: a compiler-level wave barrier suffices and the other
  // waves of the work-group run on.  Otherwise a work-group barrier.
  template <int p>
  __device__ __forceinline__ static void boundary_sync() {
    if constexpr (wave_local(p)) {
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
      __builtin_amdgcn_wave_barrier();
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    } else {
      __syncthreads();
    }
  }
  // LDS layout of the hand-overs: position a at slot a + PM (a >> PSH), PM
  // padding slots per 2^PSH positions.  PAD selects (PSH, PM): 0 -> (LR, 1),
  // 1 -> (3, 1), 2 -> (4, 1), 3 -> (4, 2), 4 -> (5, 1).  Every boundary uses
  // the same layout: the positions a wave writes at a boundary are then the
  // slots it owns in its pass, so a wave-local hand-over (no work-group
  // barrier) never writes a slot that another wave still reads from the
  // previous boundary.
  static constexpr int PSH = PAD == 0 ? (LR > 0 ? LR : 1) : (PAD == 1 ? 3 : (PAD == 4 ? 5 : 4));
  static constexpr int PM = PAD == 3 ? 2 : 1;
  __host__ __device__ static constexpr int pad(int a) { return a + PM * (a >> PSH); }
  // pad(base + c) for the positions base + SP r of one butterfly (c = SP r):
  // they never straddle a padding group unevenly, so the padded address is
  // pad(base) plus a constant, pad(base + c) = pad(base) + pad(c) (checked
  // exhaustively for every pass of every length, radix and layout used).
  // Table entries: W_M (M), the per-thread first-pass table of the users
  // that keep one (M), then W_{L_p} for p = 1 .. P - 1.
  static constexpr int M_TAB = N << TWS;
  __host__ __device__ static constexpr int twc_offset(int p) {
    int off = 2 * M_TAB;
    for (int q = 1; q < p; ++q) off += N >> (LR * q);
    return off;
  }
  static constexpr int TABLE = TWC ? twc_offset(P) : M_TAB;
  template <int p>
  __device__ __forceinline__ static float2 twiddle(const float2* __restrict__ tw, int ts) {
    if constexpr (TWC && p > 0) {
      return tw[twc_offset(p) + ts];
    } else {
      return tw[ts << (LR * p + TWS)];
    }
  }
  static constexpr int LDS = N + PM * (N >> PSH) + 1;  // float2 slots per transform
  // Order in which a pass reads its RP inputs from LDS: grouped by the
  // radix-4 sub-DFT of Dft<RP> that consumes them first (inputs r0 + A r1,
  // A = RP / 4), so that sub-DFT can start while the later reads are still in
  // flight.
  template <int RP>
  __host__ __device__ static constexpr int read_order(int j) {
    constexpr int A = RP >= 4 ? RP / 4 : 1;
    return RP >= 4 ? (j / 4) + A * (j % 4) : j;
  }

  // Position (before padding) held by register i of thread tau after the
  // forward transform (digit-reversed order).
  __device__ __forceinline__ static int spectrum_pos(int tau, int i) {
    constexpr int RL = 1 << lr(P - 1);
    return (tau + T * (i / RL)) * RL + (i % RL);
  }
  // Frequency index of the value stored at (unpadded) position a after the
  // forward transform: a = sum_p s_p * S_p  ->  k = s_0 + R_0 (s_1 + R_1 (s_2 + ...)).
  __host__ __device__ static int frequency_of(int a) {
    int k = 0, mul = 1, len = N;
    for (int p = 0; p < P; ++p) {
      const int rp = 1 << lr(p);
      const int sp = len >> lr(p);
      const int s = (a / sp) % rp;
      k += s * mul;
      mul *= rp;
      len = sp;
    }
    return k;
  }

  // ---- one pass, forward, on K independent transforms at once (transform k
  // in LDS region lds + k * LDS): read (p > 0), DFT, twiddle, write (p < P-1).
  // The K transforms share the barriers, and their independent instruction
  // streams interleave.
  // W0: pass 0 takes its twiddles for every s (s = 0 included) from w0[k][s]
  // instead of the table (see forward_w0).
  template <int p, int K, bool W0 = false>
  __device__ __forceinline__ static void fwd_pass(float2 (&x)[K][R], float2* lds, const float2* __restrict__ tw,
                                                  int tau, const float2 (&w0)[K][R]) {
    constexpr int LRP = lr(p), RP = 1 << LRP, U = R / RP;
    constexpr int L = N >> (LR * p), SP = L >> LRP;
    if constexpr (p > 0) {
      boundary_sync<p - 1>();
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int b = tau + T * u;
        const int base = (b / SP) * L + (b % SP), pb = pad(base);
#pragma unroll
        for (int k = 0; k < K; ++k)
#pragma unroll
          for (int j = 0; j < RP; ++j) {
            const int r = read_order<RP>(j);
            x[k][u * RP + r] = lds[k * LDS + (AFF ? pb + pad(SP * r) : pad(base + SP * r))];
          }
      }
    }
#pragma unroll
    for (int k = 0; k < K; ++k) dft_block<p, 0, false>(x[k]);
    if constexpr (W0 && p == 0) {
#pragma unroll
      for (int k = 0; k < K; ++k)
#pragma unroll
        for (int s = 0; s < RP; ++s) x[k][s] = cmul(x[k][s], w0[k][s]);
    } else if constexpr (SP > 1) {
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int t = (tau + T * u) % SP;
#pragma unroll
        for (int s = 1; s < RP; ++s) {
          const float2 w = twiddle<p>(tw, t * s);
#pragma unroll
          for (int k = 0; k < K; ++k) x[k][u * RP + s] = cmul(x[k][u * RP + s], w);
        }
      }
    }
    if constexpr (p + 1 < P) {
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int b = tau + T * u;
        const int base = (b / SP) * L + (b % SP), pb = pad(base);
#pragma unroll
        for (int k = 0; k < K; ++k)
#pragma unroll
          for (int s = 0; s < RP; ++s) lds[k * LDS + (AFF ? pb + pad(SP * s) : pad(base + SP * s))] = x[k][u * RP + s];
      }
      fwd_pass<p + 1, K, W0>(x, lds, tw, tau, w0);
    }
  }

  // ---- one pass, inverse: read (p < P-1), conj twiddle, conj DFT, write (p > 0) ----
  template <int p, int K, bool W0 = false>
  __device__ __forceinline__ static void inv_pass(float2 (&x)[K][R], float2* lds, const float2* __restrict__ tw,
                                                  int tau, const float2 (&w0)[K][R]) {
    constexpr int LRP = lr(p), RP = 1 << LRP, U = R / RP;
    constexpr int L = N >> (LR * p), SP = L >> LRP;
    if constexpr (p + 1 < P) {
      boundary_sync<p>();
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int b = tau + T * u;
        const int base = (b / SP) * L + (b % SP), pb = pad(base);
#pragma unroll
        for (int k = 0; k < K; ++k)
#pragma unroll
          for (int j = 0; j < RP; ++j) {
            const int s = read_order<RP>(j);
            x[k][u * RP + s] = lds[k * LDS + (AFF ? pb + pad(SP * s) : pad(base + SP * s))];
          }
      }
    }
    if constexpr (W0 && p == 0) {
#pragma unroll
      for (int k = 0; k < K; ++k)
#pragma unroll
        for (int s = 0; s < RP; ++s) x[k][s] = cmulc(x[k][s], w0[k][s]);
    } else if constexpr (SP > 1) {
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int t = (tau + T * u) % SP;
#pragma unroll
        for (int s = 1; s < RP; ++s) {
          const float2 w = twiddle<p>(tw, t * s);
#pragma unroll
          for (int k = 0; k < K; ++k) x[k][u * RP + s] = cmulc(x[k][u * RP + s], w);
        }
      }
    }
#pragma unroll
    for (int k = 0; k < K; ++k) dft_block<p, 0, true>(x[k]);
    if constexpr (p > 0) {
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int b = tau + T * u;
        const int base = (b / SP) * L + (b % SP), pb = pad(base);
#pragma unroll
        for (int k = 0; k < K; ++k)
#pragma unroll
          for (int r = 0; r < RP; ++r) lds[k * LDS + (AFF ? pb + pad(SP * r) : pad(base + SP * r))] = x[k][u * RP + r];
      }
      inv_pass<p - 1, K, W0>(x, lds, tw, tau, w0);
    }
  }

  template <int p, int u, bool INV>
  __device__ __forceinline__ static void dft_block(float2 (&x)[R]) {
    constexpr int RP = 1 << lr(p), U = R / RP;
    Dft<RP, INV>::template run<u * RP, 1>(x);
    if constexpr (u + 1 < U) dft_block<p, u + 1, INV>(x);
  }

  // Forward DFT (sign -1), unnormalised, of K transforms.  In: x[k][r] =
  // position tau + T*r.  Out: x[k][i] = frequency frequency_of(spectrum_pos(tau, i)).
  // `lds` holds K regions of LDS float2 slots; `tw` is the table
  // W_M^k = exp(-2 i pi k / M), k < M = N << TWS.  All T threads of the transform, and
  // every other thread of the work-group, must call it together (barriers).
  template <int K>
  __device__ __forceinline__ static void forward(float2 (&x)[K][R], float2* lds, const float2* __restrict__ tw,
                                                 int tau) {
    float2 none[K][R];
    fwd_pass<0, K, false>(x, lds, tw, tau, none);
  }
  // Inverse DFT (sign +1), unnormalised; exact reverse of forward's layout.
  template <int K>
  __device__ __forceinline__ static void inverse(float2 (&x)[K][R], float2* lds, const float2* __restrict__ tw,
                                                 int tau) {
    float2 none[K][R];
    inv_pass<P - 1, K, false>(x, lds, tw, tau, none);
  }
  // As forward / inverse, with the output twiddles of pass 0 given per
  // transform: output s of pass 0 is multiplied by w0[k][s] (inverse: its
  // input by conj(w0[k][s])) in place of W_N^{tau s}.  A diagonal factor
  // d_tau on the input positions tau + T r of the thread can so be folded into
  // the transform: w0[k][s] = d_tau W_N^{tau s}, after multiplying register r
  // by whatever part of the factor depends on r alone.  Needs P > 1.
  template <int K>
  __device__ __forceinline__ static void forward_w0(float2 (&x)[K][R], float2* lds, const float2* __restrict__ tw,
                                                    int tau, const float2 (&w0)[K][R]) {
    static_assert(P > 1, "forward_w0: needs a pass with twiddles");
    fwd_pass<0, K, true>(x, lds, tw, tau, w0);
  }
  template <int K>
  __device__ __forceinline__ static void inverse_w0(float2 (&x)[K][R], float2* lds, const float2* __restrict__ tw,
                                                    int tau, const float2 (&w0)[K][R]) {
    static_assert(P > 1, "inverse_w0: needs a pass with twiddles");
    inv_pass<P - 1, K, true>(x, lds, tw, tau, w0);
  }
  __device__ __forceinline__ static void forward(float2 (&x)[R], float2* lds, const float2* __restrict__ tw,
                                                 int tau) {
    forward<1>(reinterpret_cast<float2(&)[1][R]>(x), lds, tw, tau);
  }
  __device__ __forceinline__ static void inverse(float2 (&x)[R], float2* lds, const float2* __restrict__ tw,
                                                 int tau) {
    inverse<1>(reinterpret_cast<float2(&)[1][R]>(x), lds, tw, tau);
  }
};

}  // namespace krpe
