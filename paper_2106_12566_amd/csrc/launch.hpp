// Host-side launchers of the kernels in kernels.hip and the workspace layouts.
#pragma once

#include <hip/hip_runtime.h>

#include <cstddef>
#include <cstdint>

namespace krpe {

// Workspace of krpe_attention_fwd (byte offsets, 256-aligned).
struct AttnLayout {
  int l2;            // log2 N, N = next power of two >= n
  int ksplit;        // position slices of the channel-norm products
  int fsplit;        // feature splits of the convolution (conv_fsplit)
  size_t tw;         // float2 [2N]              W_{2N}^k
  size_t hs;         // float2 [H][S][2N/S]      spectrum of c by residue class, / 2N
  size_t hnorm;      // float2 [H]               (||h||_1, ||h||_2)
  size_t phiq;       // float  [BH][m][N]        phi(q), feature-major, zero beyond n
  size_t phik;       // float  [BH][m][N]        phi(k)
  size_t vsc;        // float2 [BH][pairs][N]    scaled column pairs of v' = [v, 1]
  size_t colmax;     // float  [BH][d+1]         column scales of v'
  size_t vmax;       // float  [BH][chunks][d]   column maxima per chunk of positions
  size_t x2;         // float  [BH][ks][m][pairs] squared norms of the packed channels
  size_t wb;         // float2 [BH][m+1]         bound weights of the certification
  size_t part;       // float  [BH][fsplit][splits][d+1][n] numerators / denominator per feature and class split
  size_t psum;       // float  [BH][d+1][n]      their sums (fsplit > 1 only)
  size_t fix;        // uint   [BH + 1]          rows queued per head, then their total
  size_t fixmask;    // uint64 [BH][ceil(n/64)]  queued rows: bit i % 64 of word i / 64
  size_t fixpart;    // double [BH][slots][32][d+1] key-share partial sums of the exact rows
  size_t fixplan;    // int32: the queued rows and work items of the exact rows (fix_plan_bytes)
  size_t brange;     // int2   [H]               range of finite b per head
  size_t cexp;       // float  [H][2n-1]         c = exp(b) (exact rows)
  size_t total;
};
AttnLayout attn_layout(int B, int H, int n, int d, int m);

// Workspace of krpe_attention_bwd: the forward's workspace first, then the
// backward's buffers (cmax = max(M, d + 1) columns, M the features).
struct BwdLayout {
  AttnLayout f;
  size_t zf;         // float  [BH][n][d]        z of the forward pass
  size_t den;        // float  [BH][n]           its denominators
  size_t brev;       // float  [H][2n-1]         reversed bias (transposed Toeplitz matrix)
  size_t hsr;        // float2 [H][S][2N/S]      its spectrum
  size_t gh;         // float  [BH][d+1][N]      [dL/dnumerator, dL/ddenominator], feature-major
  size_t vh;         // float  [BH][d+1][N]      [v, 1], feature-major
  size_t vsc;        // float2 [BH][cmax/2][N]   scaled column pairs of each product
  size_t colmax;     // float  [BH][cmax]
  size_t vmax;       // float  [BH][chunks][cmax]
  size_t part;       // float  [BH][splits][cmax][n] class splits of each product
  size_t gpk, vpk;   // float2 [BH][(d+2)/2][N]  Gh, V' as column pairs (gradient of b)
  size_t spart;      // float2 [BH][(d+2)/2][2N] correlation spectra per column pair
  size_t sh, ycorr;  // float2 [H][2N]           their sum per head, and its inverse per class
  size_t total;
};
BwdLayout bwd_layout(int B, int H, int n, int d, int M);

// Workspace of krpe_attention_fwd for n > 2^kMaxLog2N on the FFT route
// (blocks of nbk positions, nb blocks, Ntot = nb nbk).
struct LongLayout {
  int nb, nbk, Ntot, ksplit, fsplit;
  size_t fix;          // uint   [BH + 1]          (first, as in AttnLayout)
  size_t tw;           // float2 [2 nbk]
  size_t hs;           // float2 [nb][H][2 nbk]   spectra of query block I against each key block
  size_t hnorm;        // float2 [nb][H]          their norms
  size_t hunit;        // float2 [H]              ones
  size_t bwin;         // float  [nb][H][2 nbk - 1] their bias windows
  size_t phiq, phik;   // float  [BH][M][Ntot]    whole sequence (exact rows)
  size_t phiqb, phikb; // float  [nb][BH][M][nbk] per block
  size_t vsc;          // float2 [nb][BH][pairs][nbk]
  size_t colmax;       // float  [nb][BH][d+1]
  size_t vmax;         // float  [BH][chunks][d]
  size_t x2;           // float  [BH][ks][M][pairs]
  size_t wbj, wbi;     // float2 [nb][BH][M+1], [BH][M+1]
  size_t part;         // float  [BH][nb][fsplit][splits][d+1][nbk]
  size_t psum;         // float  [BH][d+1][nbk]   their sums
  size_t zb;           // float  [BH][nbk][d]
  size_t maskb, maskf; // uint64 [BH][nbk/64], [BH][ceil(n/64)]
  size_t fixpart;      // double [BH][slots][32][d+1]
  size_t fixplan;      // int32 (fix_plan_bytes)
  size_t brange;       // int2   [H]
  size_t cexp;         // float  [H][2n-1]       c = exp(b) (exact rows)
  size_t total;
};
LongLayout long_layout(int B, int H, int n, int d, int M);
// Feature splits of a forward convolution launch over nkb key blocks.
int conv_fsplit(int l2, int BH, int cols, int M, int nkb);

// Workspace of krpe_toeplitz_conv.
// Workspace of krpe_toeplitz_conv.  For n > 2^kMaxLog2N the Toeplitz matrix is
// taken in nb x nb blocks of nbk = 2^kMaxLog2N positions (nb = 1 otherwise):
// hs, hnorm and bwin then hold the spectra, norms and bias windows of one
// block row, vsc and colmax the channels of every key block.
struct ConvLayout {
  int l2, nb, nbk;
  size_t tw, hs, hnorm, bwin, ones, vsc, colmax, vmax, part, total;
};
ConvLayout conv_layout(int B, int H, int C, int n);

int conv_splits(int l2);
// Work units of one launch_conv at these sizes (no key blocks, no feature split).
int conv_units(int l2, int BH, int cols);
int gram_splits(int BH, int m, int N);

// Entries (float2) of the twiddle table of length 2^l2: W_{2N}^k, k < 2N, and
// for N >= 8192 the per-thread and per-pass tables after it.
int twiddle_slots(int l2);
hipError_t launch_twiddles(float2* tw, int l2, hipStream_t st);
hipError_t launch_spectrum(int l2, const float* b, const float2* tw, float2* Hs, float2* hnorm, int H, int n,
                           hipStream_t st);
// nsrc sources (1 or 2) x0/x1 -> phi0/phi1.  feature_major: phi[bh][l][ld] for
// positions < ld (zero beyond n); otherwise phi[bh][i][m].  fix_counts, if not
// NULL, gets its BH + 1 entries cleared.  nprf: rows of x are divided by their
// l2 norm first.
hipError_t launch_feature_map(bool bf16, const void* x0, const void* x1, const float* W, float* phi0,
                              float* phi1, int nsrc, bool feature_major, int ld, int BH, int H, int n, int d,
                              int m, unsigned* fix_counts, bool nprf, int kind, hipStream_t st);
// v'(pos, c) = v[bh * bh_stride + pos * sp + c * sc] for c < ncols, 1 for c == ncols if with_ones;
// pmax: scratch of BH * vmax_chunks(n) * ncols floats.
int vmax_chunks(int n);
hipError_t launch_vprep(bool bf16, const void* v, long long sp, long long sc, long long bh_stride, int ncols,
                        bool with_ones, int BH, int n, int N, float* pmax, float* colmax, float2* vsc,
                        hipStream_t st);
hipError_t launch_conv(int l2, const float* phiq, const float* phik, long long phi_bh_stride, const float2* vsc,
                       const float* colmax, const float2* Hs, const float2* tw, float* part, int BH, int H, int n,
                       int cols, int m, hipStream_t st);
// launch_conv over nkb key blocks and fsplit feature splits (the unit layout
// of k_conv_contract); hnorm (or nullptr) lets all-zero blocks of C skip.
hipError_t launch_conv_split(int l2, const float* phiq, const float* phik, long long phi_bh_stride,
                             const float2* vsc, const float* colmax, const float2* Hs, const float2* hnorm,
                             const float2* tw, float* part, int BH, int H, int n, int cols, int m, int nkb,
                             int fsplit, hipStream_t st);
hipError_t launch_gram(const float* phik, const float2* vsc, float* X2, int BH, int m, int N, int pairs,
                       int ksplit, hipStream_t st);
// Wb[bh][l] = (A_l, D_l) for l < m, Wb[bh][m] = (max column scale, 0) from the channel norms.
hipError_t launch_bound_weights(const float* X2, const float* colmax, float2* Wb, int BH, int m, int d, int ksplit,
                                hipStream_t st);
// nsplit: partial results per (bh) row of part (conv_splits(l2) times the
// key blocks and feature splits of the convolution launch).
hipError_t launch_combine(const float* part, const float* phiq, const float2* Wb, const float2* hnorm, float* z,
                          float* den_out, unsigned* fix, unsigned long long* fixmask, int BH, int H, int n, int l2,
                          int d, int m, int nsplit, hipStream_t st);
// Work-group slots per head of the exact-row kernels, and their partial sums:
// fixpart holds BH * fix_slots(BH) * 32 * (d + 1) doubles; plan holds
// fix_plan_bytes(BH, n) bytes (the queued rows and the work items).
int fix_slots(int BH);
size_t fix_plan_bytes(int BH, int n);
hipError_t launch_fixup(const float* phiq, const float* phik, const void* v, bool bf16, const float* b,
                        float* z, float* den_out, const unsigned* fix, const unsigned long long* fixmask, int* plan,
                        double* fixpart, int2* brange, float* cexp, int BH, int H, int n, int ld, int d, int m,
                        hipStream_t st);
// The direct route for m <= kDirMaxM features (fp32 values): one wave per 32
// query rows, no cross-wave reduction.  Taken when the rows give at least
// kDirMinWaves waves (one and a half per SIMD): with fewer, each wave walking
// all keys of its rows alone is slower than the exact-row kernel, whose
// work-groups split a group's keys.
constexpr int kDirMaxM = 128;
constexpr long long kDirMinWaves = 1536;
// Whether the direct route runs the row-parallel kernel (else the exact-row
// kernel over a queue of every row).
inline bool direct_rows_path(long long BH, int n, int M) {
  return M <= kDirMaxM && BH * ((n + 31) / 32) >= kDirMinWaves;
}
hipError_t launch_direct_rows(const float* phiq, const float* phik, const float* v, const float* b, float* z,
                              float* den_out, int2* brange, float* cexp, int BH, int H, int n, int ld, int d, int m,
                              hipStream_t st);
hipError_t launch_ones(float* ones, int n, int N, hipStream_t st);
// Long sequences (long_seq.hip): block copies of phi rows, bias windows of a
// block pair, sums over key blocks, certification weights, row masks, rows.
hipError_t launch_block_rows(const float* src, float* dst, int BH, int R, int nbk, int Ntot, int K, hipStream_t st);
hipError_t launch_bias_window(const float* b, float* out, int H, int n, int nbk, int nb, int I, hipStream_t st);
hipError_t launch_wb_accum(float2* wbI, const float2* wbJ, const float2* hnorm, int BH, int H, int M, int nb,
                           hipStream_t st);
hipError_t launch_merge_mask(const unsigned long long* blk, unsigned long long* full, int BH, int tiles_b,
                             int tiles_full, int K, int nbk, hipStream_t st);
hipError_t launch_scatter_rows(const float* zb, float* z, int BH, int n, int nbk, int d, int K, int lenK,
                               hipStream_t st);
hipError_t launch_unit_hnorm(float2* hn, int H, hipStream_t st);
// dst = src (bf16) widened to fp32, count elements.
hipError_t launch_widen_bf16(const void* src, float* dst, long long count, hipStream_t st);
// Queue every row for the exact-row kernel (the direct route).
hipError_t launch_mark_all(unsigned* fix, unsigned long long* fixmask, int BH, int n, hipStream_t st);
// Backward (see kernels.hip): Gh, V' feature-major from G, z, den, v; the
// reversed bias; dv from the class splits of the convolution output; dx from
// dphi (class splits) and phi.
hipError_t launch_bwd_prep(bool bf16, const float* G, const float* z, const float* den, const void* v, float* Gh,
                           float* Vh, int BH, int n, int N, int d, hipStream_t st);
hipError_t launch_reverse_bias(const float* b, float* brev, int n, int H, hipStream_t st);
hipError_t launch_bwd_dv(const float* part, float* dv, int BH, int n, int d, int cols, int nsplit, hipStream_t st);
// db[h][s] = c_t dc_t from Gh, V' (feature-major [bh][cols][N]) and phi; scratch:
// gpk, vpk [BH][pairs][N], spart [BH][pairs][2N], Sh and ycorr [H][2N] (float2).
hipError_t launch_db(int l2, const float* phiq, const float* phik, long long phi_bh_stride, const float* gh,
                     const float* vh, const float2* tw, float2* gpk, float2* vpk, float2* spart, float2* Sh,
                     float2* ycorr, const float* b, float* db, int B, int H, int n, int cols, int m, hipStream_t st);
hipError_t launch_feature_bwd(bool bf16, const void* x, const float* W, const float* phi, const float* part,
                              float* dx, int BH, int H, int n, int N, int d, int m, int nsplit, bool nprf,
                              hipStream_t st);
// y[bh][c][i] (row stride ldy) = sum over s of part[bh][s][c][i], i < n.
hipError_t launch_sum_splits(const float* part, float* y, int BH, int C, int n, int ldy, int nsplit, hipStream_t st);

}  // namespace krpe
