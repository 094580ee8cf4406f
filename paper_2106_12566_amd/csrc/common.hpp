// Device-side constants and helpers shared by the kernels.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

#include "fft.hpp"

namespace krpe {

constexpr int kMaxLog2N = 14;  // n <= 16384 (FFT length 2N <= 32768)
// Longer sequences (attention only) run as blocks of 2^kMaxLog2N positions:
// n <= 2^kMaxLongLog2N, the Toeplitz matrix taken block by block.
constexpr int kMaxLongLog2N = 16;
constexpr int kMaxD = 128;
constexpr int kMaxM = 1024;
constexpr int kLog2R = 4;      // 16 complex values per thread

// Feature maps (Sec. 2): PRF of Eq. (5), the trigonometric map TRF (2m signed
// features), elu + 1 (d features, no projections).
constexpr int kFeatPrf = 0;
constexpr int kFeatTrf = 1;
constexpr int kFeatElu = 2;

// Launch shape of the products of length-2N circular convolutions, N = 2^L2.
//
// The 2N frequency bins are split into S = 2 FOLD residue classes
// k = S k' + r; class r is a length L' = 2N / S transform (L' = N / FOLD) of
// the input folded FOLD times (Section 3.2 leaves the FFT open; see the
// convolution kernel for the algebra).  FOLD = 1 up to N = 8192 (the classes
// are the even and odd bins) and 4 at N = 16384: transforms never exceed
// 8192 points (64 KiB of LDS).
//
// A transform is owned by T = L' / R threads (R complex values each); a
// work-group holds G units of T threads (G > 1 only for transforms of fewer
// than 128 threads, filling 256); a unit of the convolution kernel runs KH
// residue classes as interleaved transforms sharing loads, barriers and
// accumulators.
template <int L2>
struct Conf {
  // Classes of the length-2N spectrum: two (one 2N/2-point transform each)
  // up to N = 8192, eight (4096 points each, four folds) at N = 16384.
  static constexpr int FOLD = L2 <= 13 ? 1 : 4;
  static constexpr int S = 2 * FOLD;                  // residue classes
  static constexpr int L2T = L2 <= 13 ? L2 : 12;       // log2 of the transform length
  // 8 values per thread at N = 16384: 512 threads share the 64 positions x
  // 2 columns of accumulators a 256-thread group could not hold
  static constexpr int LOG2R = L2 == 14 ? 3 : kLog2R;
  // Compact per-pass twiddle tables (and the per-thread first-pass table of
  // the convolution) for the lengths whose units cannot keep their twiddles
  // in registers.
  static constexpr bool TWC = L2 == 13;
  // phi rows and value pairs read through buffer resources, with phi(k) (and
  // at N = 4096 phi(q)) loaded a feature ahead: measured faster at N = 2048
  // and 4096 only (slower at 512, 1024 and 16384).
  static constexpr bool BUF = L2 == 11 || L2 == 12;
  // Twiddles come from the W_{2N} table.  Affine LDS addressing where it
  // frees the registers that the loads one feature ahead need, and at
  // N = 16384.  At N = 4096 and 16384 the LDS layout has two padding slots
  // per 16 positions (Fft's PAD): timed one hand-over at a time, it removes
  // the bank conflicts of the cross-wave boundary and is the fastest single
  // layout at every boundary of both transforms.
  static constexpr int PAD = (L2 == 14 || L2 == 12) ? 3 : 0;
  using F = Fft<L2T, LOG2R, 1 + L2 - L2T, TWC, L2 == 14 || BUF, PAD>;
  static constexpr int N = 1 << L2;
  static constexpr int LT = F::N;  // transform length 2N / S
  static constexpr int G = F::T >= 128 ? 1 : 256 / F::T;  // units per work-group
  static constexpr int THREADS = G * F::T;
  static constexpr int WAVES = (THREADS + 63) / 64;
  static constexpr int LDS_SLOTS = F::P > 1 ? G * F::LDS : 1;
  // Two work-groups per CU for the mid-size transforms: one runs while the
  // other waits at a barrier (register budget 256 per thread; 128 for the
  // 512-thread groups of N = 8192, which then re-read their per-position
  // values, spectrum and twiddles from the L1-friendly tables).
  static constexpr int WPE = (L2 >= 9 && L2 <= 12) ? 2 : (L2 == 13 ? 4 : 1);
  static constexpr int KH =
      (WPE == 1 && FOLD <= 2 && F::T <= 256 && F::R <= 16 && 2 * G * F::LDS * 8 <= 144 * 1024) ? 2 : 1;
  static constexpr int HSPLIT = S / KH;  // work units per column pair and head
  static constexpr int CONV_LDS_SLOTS = F::P > 1 ? G * KH * F::LDS : 1;
  // Per-position values (v pairs, prefetched phi), the spectrum and the
  // hoisted twiddles stay in registers for work-groups of <= 256 threads
  // (their 256-register budget holds them); the 512-thread groups of
  // N = 8192 re-read them.  At N = 16384 (512 threads, one group per CU) the
  // FOLD x R value pairs of a thread stay in registers too, pre-rotated by
  // the class and fold twists; phi is not loaded ahead there (PREF).
  static constexpr bool VREG = (THREADS <= 256 && FOLD == 1) || L2 == 14;
  static constexpr bool PREF = VREG && WPE == 1 && FOLD == 1;
  static constexpr bool HREG = THREADS <= 256 || L2 == 14;
  static constexpr bool HOIST = (THREADS <= 256 && FOLD != 2) || L2 == 14;
  // phi(q) too loaded a feature ahead (where the registers allow it without
  // spills)
  static constexpr bool NEXTQ = L2 == 12;
};

// Work-groups are dispatched round-robin over the 8 XCDs (each with its own
// L2).  Renumber them so that every XCD runs a contiguous range of logical
// blocks: units of one head then share an L2.  A bijection on [0, nblocks).
__device__ __forceinline__ int xcd_block(int b, int nblocks) {
  constexpr int kXcd = 8;
  const int per = nblocks / kXcd, rem = nblocks % kXcd;
  const int xcd = b % kXcd, slot = b / kXcd;
  return (xcd < rem) ? xcd * (per + 1) + slot : rem * (per + 1) + (xcd - rem) * per + slot;
}

// Reads through a raw buffer resource (gfx9 descriptor: base, byte range,
// word 3 = 0x00020000): a per-lane byte offset (VGPR) plus a wave-uniform
// byte offset (SGPR), with no 64-bit address arithmetic per load.  The range
// check covers the VGPR offset only: a read whose VGPR offset is at or past
// `bytes` returns zero, but the SGPR offset is added unchecked, so callers keep
// the sum inside the buffer themselves.
struct BufRd {
  __amdgpu_buffer_rsrc_t r;
  __device__ __forceinline__ BufRd(const void* base, uint32_t bytes)
      : r(__builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0, static_cast<int>(bytes), 0x00020000)) {}
  __device__ __forceinline__ float f32(uint32_t voff, uint32_t soff) const {
    return __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(r, voff, soff, 0));
  }
  __device__ __forceinline__ uint16_t u16(uint32_t voff, uint32_t soff) const {
    return __builtin_amdgcn_raw_buffer_load_b16(r, voff, soff, 0);
  }
  // (The 8-byte result is bit-cast whole: taking its two halves apart by index
  // lowers to a single 4-byte load.)
  __device__ __forceinline__ float2 f64(uint32_t voff, uint32_t soff) const {
    return __builtin_bit_cast(float2, __builtin_amdgcn_raw_buffer_load_b64(r, voff, soff, 0));
  }
};

__device__ __forceinline__ float to_f32(float v) { return v; }
__device__ __forceinline__ float to_f32(uint16_t v) { return __uint_as_float(static_cast<uint32_t>(v) << 16); }

// Reduction over the lanes of one wave that belong to the same unit of T
// threads (T a power of two; units are aligned to T inside the work-group).
// Every lane of the unit receives the result.
template <int T, typename Op>
__device__ __forceinline__ float wave_unit_reduce(float v, Op op) {
#pragma unroll
  for (int off = 1; off < (T < 64 ? T : 64); off <<= 1) v = op(v, __shfl_xor(v, off));
  return v;
}

// Reduction over all T threads of a unit.  `red` is LDS holding one float per
// wave of the work-group.  Every thread of the work-group must call it (it
// contains barriers when T > 64).
template <int T, typename Op>
__device__ __forceinline__ float unit_reduce(float v, float* red, Op op) {
  v = wave_unit_reduce<T>(v, op);
  if constexpr (T > 64) {
    const int wave = threadIdx.x >> 6;
    if ((threadIdx.x & 63) == 0) red[wave] = v;
    __syncthreads();
    const int first = (threadIdx.x / T) * (T / 64);
    v = red[first];
#pragma unroll
    for (int w = 1; w < T / 64; ++w) v = op(v, red[first + w]);
    __syncthreads();
  }
  return v;
}

struct OpMax {
  __device__ __forceinline__ float operator()(float a, float b) const { return fmaxf(a, b); }
};
struct OpAdd {
  __device__ __forceinline__ float operator()(float a, float b) const { return a + b; }
};

// FFT error model.  The rounding error of the zero-padded FFT product
// y = C a (both spectrum halves, fp32) obeys, at every output i,
//   |dy_i| <= kGamma * u * log2(L) * ( ||h||_2 ||x||_2 / sqrt(L) * s + |y_i| )
// for a packed channel pair x = a0/s0 + i a1/s1 and channel scale s in
// {s0, s1}; L = 2N, u = 2^-24, h the length-L circulant kernel.  The
// constant is measured on adversarial inputs (heavy-tailed channels of very
// different scales, causal and spiked kernels) by the GPU test of the model.
constexpr float kGamma = 8.0f;
constexpr float kUnitRoundoff = 5.9604645e-8f;
// A row of Eq. (10) is certified when its bounded normwise relative error is
// at most kTau; otherwise it is evaluated exactly.
constexpr float kTau = 1.0e-4f;

}  // namespace krpe
