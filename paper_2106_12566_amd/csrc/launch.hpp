// Host-side launchers of the kernels in kernels.hip and the workspace layouts.
#pragma once

#include <hip/hip_runtime.h>

#include <cstddef>
#include <cstdint>

namespace krpe {

// Workspace of krpe_attention_fwd (byte offsets, 256-aligned).
struct AttnLayout {
  int l2;            // log2 N, N = next power of two >= n
  size_t tw;         // float2 [2N]            W_{2N}^k
  size_t hs;         // float2 [H][2][N]       spectrum halves of c, / 2N
  size_t hnorm;      // float2 [H]             (||h||_1, ||h||_2)
  size_t phiq;       // float  [BH][m][N]      phi(q), feature-major, zero beyond n
  size_t phik;       // float  [BH][m][N]      phi(k)
  size_t part;       // float  [BH][2][d+1][n] per-half numerators / denominator
  size_t bnd;        // float  [BH][pairs][n]  sum_l phi_l(q_i) ||x_{l,pair}||_2
  size_t colmax;     // float  [BH][d]         max_j |v_{j,c}|
  size_t fix;        // uint   [BH + 1 + BH n] rows queued per head, total; then the
                     //                        queued row indices of each head
  size_t total;
};
AttnLayout attn_layout(int B, int H, int n, int d, int m);

struct ConvLayout {
  int l2;
  size_t tw, hs, total;
};
ConvLayout conv_layout(int H, int n);

hipError_t launch_twiddles(float2* tw, int l2, hipStream_t st);
hipError_t launch_spectrum(int l2, const float* b, const float2* tw, float2* Hs, float2* hnorm, int H, int n,
                           hipStream_t st);
// nsrc sources (1 or 2) x0/x1 -> phi0/phi1.  feature_major: phi[bh][l][ld] for
// positions < ld (zero beyond n); otherwise phi[bh][i][m].  fix_counts, if not
// NULL, gets its BH + 1 entries cleared.
hipError_t launch_feature_map(bool bf16, const void* x0, const void* x1, const float* W, float* phi0,
                              float* phi1, int nsrc, bool feature_major, int ld, int BH, int H, int n, int d,
                              int m, unsigned* fix_counts, hipStream_t st);
hipError_t launch_conv(int l2, bool bf16, const float* phiq, const float* phik, const void* v,
                       const float2* Hs, const float2* tw, float* part, float* bnd, float* colmax, int BH,
                       int H, int n, int d, int m, hipStream_t st);
hipError_t launch_combine(const float* part, const float* bnd, const float* colmax, const float2* hnorm,
                          float* z, unsigned* fix, int BH, int H, int n, int l2, int d, hipStream_t st);
hipError_t launch_fixup(const float* phiq, const float* phik, const void* v, bool bf16, const float* b,
                        float* z, const unsigned* fix, int BH, int H, int n, int ld, int d, int m,
                        hipStream_t st);
hipError_t launch_toeplitz(int l2, const float* a, float* y, const float2* Hs, const float2* tw, int BH, int H,
                           int C, int n, hipStream_t st);

}  // namespace krpe
