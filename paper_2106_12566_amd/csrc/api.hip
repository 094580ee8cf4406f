// C ABI of libkrpe.so (declared in include/krpe.h): argument validation on the
// host, workspace carving and the launch sequence of each entry point.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>
#include <mutex>
#include <string>

#include "common.hpp"
#include "krpe.h"
#include "launch.hpp"

namespace krpe {
namespace {

thread_local std::string g_last_error;

krpe_status_t fail(krpe_status_t s, const std::string& msg) {
  g_last_error = msg;
  return s;
}

int log2_ceil(int n) {
  int l = 0;
  while ((1 << l) < n) ++l;
  return l;
}

size_t align_up(size_t v) { return (v + 255) & ~static_cast<size_t>(255); }

// Bytes of an array of `rows` rows of N floats that the convolution reads as
// phi rows, plus one row of slack: with buffer reads its loop loads one row
// past a unit's last row (never used), which for the last unit lands here.
size_t phi_bytes(size_t rows, size_t N) { return (rows + 1) * N * sizeof(float); }

bool misaligned(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) != 0; }

struct Range {
  const void* p;
  size_t bytes;
};
bool overlaps(Range a, Range b) {
  if (a.bytes == 0 || b.bytes == 0) return false;
  const uintptr_t a0 = reinterpret_cast<uintptr_t>(a.p), b0 = reinterpret_cast<uintptr_t>(b.p);
  return a0 < b0 + b.bytes && b0 < a0 + a.bytes;
}

size_t dtype_size(int dt) { return dt == KRPE_BF16 ? 2 : 4; }

krpe_status_t hip_check(hipError_t e, const char* what) {
  if (e == hipSuccess) return KRPE_OK;
  return fail(KRPE_ERR_HIP, std::string(what) + ": " + hipGetErrorString(e));
}

krpe_status_t check_dims(int B, int H, int n, int d, int m, bool need_dm, int max_log2n = kMaxLog2N) {
  if (B < 0 || H < 0 || n < 0 || (need_dm && (d < 0 || m < 0))) return fail(KRPE_ERR_SHAPE, "negative size");
  if (n < 1) return fail(KRPE_ERR_SHAPE, "n must be >= 1 (b has 2n-1 entries)");
  if (n > (1 << max_log2n))
    return fail(KRPE_ERR_UNSUPPORTED, "n > " + std::to_string(1 << max_log2n) + " is not supported here");
  if (need_dm) {
    if (d < 1 || m < 1) return fail(KRPE_ERR_SHAPE, "d and m must be >= 1");
    if (d > kMaxD) return fail(KRPE_ERR_UNSUPPORTED, "d > 128 is not supported");
    if (m > kMaxM) return fail(KRPE_ERR_UNSUPPORTED, "m > 1024 is not supported");
  }
  // Row indices (bh * n + i) are kept in 32 bits and grids in 31 bits.
  const long long rows = static_cast<long long>(B) * H * n;
  if (rows >= (1LL << 31)) return fail(KRPE_ERR_UNSUPPORTED, "B * H * n >= 2^31 is not supported");
  return KRPE_OK;
}

constexpr unsigned kKnownFlags =
    KRPE_NPRF | KRPE_FEAT_TRF | KRPE_FEAT_ELU | KRPE_ROUTE_DIRECT | KRPE_ROUTE_FFT | KRPE_HINT_CAUSAL;
constexpr unsigned kBwdFlags = KRPE_NPRF | KRPE_ROUTE_DIRECT | KRPE_ROUTE_FFT | KRPE_HINT_CAUSAL;

// Whether the direct route is the faster one for BH heads of length n with M
// features and d value columns.  Cost model fitted to MI355X timings of both
// routes at 80 shapes (B H = 1, 16, 96; d = 64; M = 32 .. 128; n = 512 ..
// 40000, not causal): each route's time is its work over all heads at a
// measured rate plus a fixed cost (the launch chain and its latency-bound
// small kernels).  Direct: per (query, key) pair and unit of M rounded up to
// a multiple of 64, plus d + 1, 1.74e-14 s on the row-parallel kernel and
// 1.9e-14 s on the exact-row kernel (few heads, or M > 128), plus 7.4e-5 s.
// FFT: per column pair, feature and point of the length-2N transform times
// log2(2N), 1.65e-13 s up to N = 4096, 3.8e-13 s at N = 8192 and 3.1e-13 s
// at N = 16384, over the nb^2 block pairs of a blocked sequence, plus
// 1.5e-4 s.
// All n^2 pairs are counted, as the host does not read b, unless the caller
// states a causal mask (KRPE_HINT_CAUSAL): the direct kernels then visit the
// n (n + 1) / 2 pairs j <= i only (measured at n = 16384, 16 heads, m = 256:
// 11.7 ms direct, 17.8 ms FFT), and a blocked FFT route runs the
// nb (nb + 1) / 2 block pairs on or below the diagonal.  The route bits force
// either route.
bool direct_is_faster(long long BH, int n, int M, int d, bool causal) {
  int l2 = 0;
  while ((1 << l2) < n) ++l2;
  // beyond one transform block the FFT route runs nb^2 block pairs
  const int nb = l2 > kMaxLog2N ? (n + (1 << kMaxLog2N) - 1) >> kMaxLog2N : 1;
  if (l2 > kMaxLog2N) l2 = kMaxLog2N;
  const double L = 2.0 * static_cast<double>(1 << l2);
  const double heads = static_cast<double>(BH);
  const double pairs = causal ? 0.5 * static_cast<double>(n) * (n + 1) : static_cast<double>(n) * n;
  // (both direct kernels run the features in steps of 64)
  const double per_pair = direct_rows_path(BH, n, M) ? 1.74e-14 : 1.9e-14;
  const double direct = per_pair * heads * pairs * (((M + 63) / 64) * 64 + d + 1) + 7.4e-5;
  const double rate = l2 <= 12 ? 1.65e-13 : (l2 == 13 ? 3.8e-13 : 3.1e-13);
  // (a causal mask leaves nb (nb + 1) / 2 of the block pairs live; the others are skipped)
  const double blocks = causal ? 0.5 * nb * (nb + 1) : static_cast<double>(nb) * nb;
  const double fft = rate * heads * M * ((d + 2) / 2) * L * (l2 + 1) * blocks + 1.5e-4;
  return direct < fft;
}

// Route of the forward pass: the FFT convolution (Sec. 3.2) or the direct
// quadratic evaluation of Eq. (10) on MFMA, forced by an option bit or chosen
// by the measured cost model (the direct route is faster for short sequences).
bool use_direct(unsigned flags, long long BH, int n, int M, int d) {
  if (flags & KRPE_ROUTE_DIRECT) return true;
  if (flags & KRPE_ROUTE_FFT) return false;
  return direct_is_faster(BH, n, M, d, (flags & KRPE_HINT_CAUSAL) != 0);
}

// Feature map selected by the option bits, and its number of features M
// (the row count of phi): m for PRF, 2m for TRF, d for elu + 1 (which needs
// m == d).
krpe_status_t feature_kind(unsigned flags, int d, int m, int* kind, int* M) {
  if (flags & ~kKnownFlags) return fail(KRPE_ERR_UNSUPPORTED, "unknown flag bits");
  if ((flags & KRPE_FEAT_TRF) && (flags & KRPE_FEAT_ELU))
    return fail(KRPE_ERR_UNSUPPORTED, "KRPE_FEAT_TRF and KRPE_FEAT_ELU are exclusive");
  if ((flags & KRPE_ROUTE_DIRECT) && (flags & KRPE_ROUTE_FFT))
    return fail(KRPE_ERR_UNSUPPORTED, "KRPE_ROUTE_DIRECT and KRPE_ROUTE_FFT are exclusive");
  *kind = (flags & KRPE_FEAT_TRF) ? kFeatTrf : (flags & KRPE_FEAT_ELU) ? kFeatElu : kFeatPrf;
  *M = *kind == kFeatTrf ? 2 * m : (*kind == kFeatElu ? d : m);
  if (*kind == kFeatElu && m != d) return fail(KRPE_ERR_SHAPE, "KRPE_FEAT_ELU needs m == d");
  if (*M > kMaxM) return fail(KRPE_ERR_UNSUPPORTED, "more than 1024 features is not supported");
  return KRPE_OK;
}

krpe_status_t record(void* const* events, int i, hipStream_t st) {
  if (!events || !events[i]) return KRPE_OK;
  return hip_check(hipEventRecord(static_cast<hipEvent_t>(events[i]), st), "hipEventRecord");
}

}  // namespace

// Feature splits of the forward convolution: the m features of a unit are
// split into contiguous ranges (each its own partial result) until the launch
// has about four units per CU, keeping at least 8 features per range (few
// (batch, head) rows).  Otherwise, for the transforms of N = 512 .. 8192
// (512 resident units: 256 CUs x 2 work-groups), two ranges when that fills
// the launch's last round of units better: one round in 32 left idle is worth
// the doubled partial results (workload of 96 heads at n = 4096: 12.4 rounds,
// 8.15 -> 8.05 ms).  At N = 16384 (one 512-thread work-group per CU) two
// ranges measured faster at every shape with M >= 64 tried, by more than the
// last round explains (16 heads, m = 256: 21.5 -> 18.5 ms; n = 65536 in
// 4 x 4 blocks: 214 -> 190 ms); four were no faster than two.
int conv_fsplit(int l2, int BH, int cols, int M, int nkb) {
  if (l2 > kMaxLog2N) return 1;
  const long long units = static_cast<long long>(conv_units(l2, BH, cols)) * nkb;
  int fs = 1;
  while (units * fs < 1024 && M / (2 * fs) >= 8) fs *= 2;
  if (fs == 1 && l2 == kMaxLog2N && M >= 64) return 2;
  if (fs == 1 && l2 >= 9 && l2 <= 13 && M >= 64) {
    constexpr long long kResident = 512;
    auto idle = [](long long u) { return static_cast<double>((u + kResident - 1) / kResident * kResident - u) / u; };
    if (idle(units) > 1.0 / 32 && idle(2 * units) < idle(units)) fs = 2;
  }
  return fs;
}

AttnLayout attn_layout(int B, int H, int n, int d, int m) {
  AttnLayout L{};
  L.l2 = log2_ceil(n);
  L.fsplit = conv_fsplit(L.l2, B * H, d + 1, m, 1);
  const size_t N = static_cast<size_t>(1) << L.l2;
  const size_t bh = static_cast<size_t>(B) * H;
  const size_t cols = static_cast<size_t>(d) + 1, pairs = (cols + 1) / 2;
  L.ksplit = gram_splits(static_cast<int>(bh), m, static_cast<int>(N));
  size_t off = 0;
  auto take = [&off](size_t bytes) {
    const size_t at = off;
    off = align_up(off + bytes);
    return at;
  };
  L.fix = take((bh + 1) * sizeof(unsigned));  // first: its offset does not depend on the sizes
  L.tw = take(static_cast<size_t>(twiddle_slots(L.l2)) * sizeof(float2));
  L.hs = take(static_cast<size_t>(H) * 2 * N * sizeof(float2));
  L.hnorm = take(static_cast<size_t>(H) * sizeof(float2));
  L.phiq = take(phi_bytes(bh * m, N));
  L.phik = take(phi_bytes(bh * m, N));
  L.vsc = take(bh * pairs * N * sizeof(float2));
  L.colmax = take(bh * cols * sizeof(float));
  L.vmax = take(bh * vmax_chunks(n) * static_cast<size_t>(d) * sizeof(float));
  L.x2 = take(bh * L.ksplit * m * pairs * sizeof(float));
  L.wb = take(bh * (static_cast<size_t>(m) + 1) * sizeof(float2));
  L.part = take(bh * L.fsplit * conv_splits(L.l2) * cols * n * sizeof(float));
  L.psum = take(L.fsplit > 1 && bh * ((static_cast<size_t>(n) + 63) / 64) < 4096 ? bh * cols * n * sizeof(float) : 0);
  L.fixmask = take(bh * ((static_cast<size_t>(n) + 63) / 64) * sizeof(unsigned long long));
  L.fixpart = take(bh * fix_slots(static_cast<int>(bh)) * 32 * cols * sizeof(double));
  L.fixplan = take(fix_plan_bytes(static_cast<int>(bh), n));
  L.brange = take(static_cast<size_t>(H) * sizeof(int2));
  L.cexp = take(static_cast<size_t>(H) * (2 * static_cast<size_t>(n) - 1) * sizeof(float));
  L.total = off;
  return L;
}

BwdLayout bwd_layout(int B, int H, int n, int d, int M) {
  BwdLayout L{};
  L.f = attn_layout(B, H, n, d, M);
  const size_t N = static_cast<size_t>(1) << L.f.l2;
  const size_t bh = static_cast<size_t>(B) * H;
  const size_t cmax = static_cast<size_t>(M > d + 1 ? M : d + 1), pairs = (cmax + 1) / 2;
  size_t off = L.f.total;
  auto take = [&off](size_t bytes) {
    const size_t at = off;
    off = align_up(off + bytes);
    return at;
  };
  L.zf = take(bh * n * d * sizeof(float));
  L.den = take(bh * n * sizeof(float));
  L.brev = take(static_cast<size_t>(H) * (2 * n - 1) * sizeof(float));
  L.hsr = take(static_cast<size_t>(H) * 2 * N * sizeof(float2));
  L.gh = take(phi_bytes(bh * (d + 1), N));
  L.vh = take(phi_bytes(bh * (d + 1), N));
  L.vsc = take(bh * pairs * N * sizeof(float2));
  L.colmax = take(bh * cmax * sizeof(float));
  L.vmax = take(bh * vmax_chunks(n) * cmax * sizeof(float));
  L.part = take(bh * conv_splits(L.f.l2) * cmax * n * sizeof(float));
  const size_t gpairs = static_cast<size_t>(d + 2) / 2;
  L.gpk = take(bh * gpairs * N * sizeof(float2));
  L.vpk = take(bh * gpairs * N * sizeof(float2));
  L.spart = take(bh * gpairs * 2 * N * sizeof(float2));
  L.sh = take(static_cast<size_t>(H) * 2 * N * sizeof(float2));
  L.ycorr = take(static_cast<size_t>(H) * 2 * N * sizeof(float2));
  L.total = off;
  return L;
}

LongLayout long_layout(int B, int H, int n, int d, int M) {
  LongLayout L{};
  L.nbk = 1 << kMaxLog2N;
  L.nb = (n + L.nbk - 1) / L.nbk;
  L.Ntot = L.nb * L.nbk;
  const size_t bh = static_cast<size_t>(B) * H, nbk = static_cast<size_t>(L.nbk), nb = static_cast<size_t>(L.nb);
  const size_t cols = static_cast<size_t>(d) + 1, pairs = (cols + 1) / 2;
  L.ksplit = gram_splits(static_cast<int>(bh), M, L.nbk);
  L.fsplit = conv_fsplit(kMaxLog2N, B * H, d + 1, M, L.nb);
  size_t off = 0;
  auto take = [&off](size_t bytes) {
    const size_t at = off;
    off = align_up(off + bytes);
    return at;
  };
  L.fix = take((bh + 1) * sizeof(unsigned));
  L.tw = take(static_cast<size_t>(twiddle_slots(kMaxLog2N)) * sizeof(float2));
  L.hs = take(nb * H * 2 * nbk * sizeof(float2));
  L.hnorm = take(nb * H * sizeof(float2));
  L.hunit = take(static_cast<size_t>(H) * sizeof(float2));
  L.bwin = take(nb * H * (2 * nbk - 1) * sizeof(float));
  L.phiq = take(bh * M * static_cast<size_t>(L.Ntot) * sizeof(float));
  L.phik = take(bh * M * static_cast<size_t>(L.Ntot) * sizeof(float));
  L.phiqb = take(nb * bh * M * nbk * sizeof(float));
  L.phikb = take(nb * bh * M * nbk * sizeof(float));
  L.vsc = take(nb * bh * pairs * nbk * sizeof(float2));
  L.colmax = take(nb * bh * cols * sizeof(float));
  L.vmax = take(bh * vmax_chunks(L.nbk) * static_cast<size_t>(d) * sizeof(float));
  L.x2 = take(bh * L.ksplit * M * pairs * sizeof(float));
  L.wbj = take(nb * bh * (static_cast<size_t>(M) + 1) * sizeof(float2));
  L.wbi = take(bh * (static_cast<size_t>(M) + 1) * sizeof(float2));
  L.part = take(bh * nb * L.fsplit * conv_splits(kMaxLog2N) * cols * nbk * sizeof(float));
  L.psum = take(bh * cols * nbk * sizeof(float));
  L.zb = take(bh * nbk * d * sizeof(float));
  L.maskb = take(bh * (nbk / 64) * sizeof(unsigned long long));
  L.maskf = take(bh * ((static_cast<size_t>(n) + 63) / 64) * sizeof(unsigned long long));
  L.fixpart = take(bh * fix_slots(static_cast<int>(bh)) * 32 * cols * sizeof(double));
  L.fixplan = take(fix_plan_bytes(static_cast<int>(bh), n));
  L.brange = take(static_cast<size_t>(H) * sizeof(int2));
  L.cexp = take(static_cast<size_t>(H) * (2 * static_cast<size_t>(n) - 1) * sizeof(float));
  L.total = off;
  return L;
}

// Workspace of the forward pass for these sizes (the blocked layout for long
// sequences on the FFT route, else the one-transform layout).
size_t fwd_workspace(int B, int H, int n, int d, int M, bool direct) {
  if (n > (1 << kMaxLog2N) && !direct) return long_layout(B, H, n, d, M).total;
  return attn_layout(B, H, n, d, M).total;
}

ConvLayout conv_layout(int B, int H, int C, int n) {
  ConvLayout L{};
  const bool blocked = n > (1 << kMaxLog2N);
  L.l2 = blocked ? kMaxLog2N : log2_ceil(n);
  L.nbk = blocked ? 1 << kMaxLog2N : n;
  L.nb = blocked ? (n + L.nbk - 1) / L.nbk : 1;
  const size_t N = static_cast<size_t>(1) << L.l2, nb = static_cast<size_t>(L.nb);
  const size_t bh = static_cast<size_t>(B) * H;
  const size_t pairs = (static_cast<size_t>(C) + 1) / 2;
  size_t off = 0;
  auto take = [&off](size_t bytes) {
    const size_t at = off;
    off = align_up(off + bytes);
    return at;
  };
  L.tw = take(static_cast<size_t>(twiddle_slots(L.l2)) * sizeof(float2));
  L.hs = take(nb * H * 2 * N * sizeof(float2));
  L.hnorm = take(blocked ? nb * H * sizeof(float2) : 0);
  L.bwin = take(blocked ? nb * H * (2 * N - 1) * sizeof(float) : 0);
  L.ones = take(phi_bytes(1, N));
  L.vsc = take(nb * bh * pairs * N * sizeof(float2));
  L.colmax = take(nb * bh * C * sizeof(float));
  L.vmax = take(bh * vmax_chunks(L.nbk) * static_cast<size_t>(C) * sizeof(float));
  // (a blocked product sums nb key blocks x the class splits per row)
  const size_t nsplit = nb * static_cast<size_t>(conv_splits(L.l2));
  L.part = take(nsplit > 1 ? bh * nsplit * C * static_cast<size_t>(L.nbk) * sizeof(float) : 0);
  L.total = off;
  return L;
}

// The forward launch sequence of Eq. (10) on a carved workspace: z, and the
// row denominators into den_out when not NULL (the backward pass needs them).
krpe_status_t run_forward(const AttnLayout& L, char* w, const void* q, const void* k, const void* v, bool bf16,
                          const float* b, const float* W, float* z, float* den_out, int BHi, int H, int n, int d,
                          int m, int M, int kind, bool nprf, bool direct, hipStream_t st, void* const* events) {
  float2* tw = reinterpret_cast<float2*>(w + L.tw);
  float2* Hs = reinterpret_cast<float2*>(w + L.hs);
  float2* hnorm = reinterpret_cast<float2*>(w + L.hnorm);
  float* phiq = reinterpret_cast<float*>(w + L.phiq);
  float* phik = reinterpret_cast<float*>(w + L.phik);
  float2* vsc = reinterpret_cast<float2*>(w + L.vsc);
  float* colmax = reinterpret_cast<float*>(w + L.colmax);
  float* vmax = reinterpret_cast<float*>(w + L.vmax);
  float* x2 = reinterpret_cast<float*>(w + L.x2);
  float2* wb = reinterpret_cast<float2*>(w + L.wb);
  float* part = reinterpret_cast<float*>(w + L.part);
  unsigned* fix = reinterpret_cast<unsigned*>(w + L.fix);
  unsigned long long* fixmask = reinterpret_cast<unsigned long long*>(w + L.fixmask);
  double* fixpart = reinterpret_cast<double*>(w + L.fixpart);
  int* fixplan = reinterpret_cast<int*>(w + L.fixplan);
  int2* brange = reinterpret_cast<int2*>(w + L.brange);
  float* cexp = reinterpret_cast<float*>(w + L.cexp);
  const int N = 1 << L.l2;
  const int pairs = (d + 2) / 2;

  if (direct) {
    // phi(q), phi(k), then every row evaluated directly: by the row-parallel
    // kernel, or by the exact-row kernel over a queue of every row.  The queue
    // is marked on both paths: its count is the number of rows evaluated
    // exactly that krpe_attention_fwd_stats reports.
    for (int e = 0; e < 2; ++e)
      if (krpe_status_t s = record(events, e, st)) return s;
    if (krpe_status_t s = hip_check(launch_feature_map(bf16, q, k, W, phiq, phik, 2, true, N, BHi, H, n, d, m,
                                                       nullptr, nprf, kind, st),
                                    "feature map launch"))
      return s;
    for (int e = 2; e < 4; ++e)
      if (krpe_status_t s = record(events, e, st)) return s;
    if (krpe_status_t s = hip_check(launch_mark_all(fix, fixmask, BHi, n, st), "queue launch")) return s;
    // bf16 values widened once into the (here unused) column-pair buffer,
    // which holds at least BH n d floats
    const void* vv = v;
    if (bf16) {
      float* vw = reinterpret_cast<float*>(vsc);
      if (krpe_status_t s = hip_check(launch_widen_bf16(v, vw, static_cast<long long>(BHi) * n * d, st),
                                      "widen launch"))
        return s;
      vv = vw;
    }
    if (direct_rows_path(BHi, n, M)) {
      if (krpe_status_t s = hip_check(launch_direct_rows(phiq, phik, static_cast<const float*>(vv), b, z, den_out,
                                                         brange, cexp, BHi, H, n, N, d, M, st),
                                      "direct launch"))
        return s;
    } else if (krpe_status_t s = hip_check(launch_fixup(phiq, phik, vv, false, b, z, den_out, fix, fixmask, fixplan,
                                                        fixpart, brange, cexp, BHi, H, n, N, d, M, st),
                                           "direct launch")) {
      return s;
    }
    return record(events, 4, st);
  }
  if (krpe_status_t s = record(events, 0, st)) return s;
  if (krpe_status_t s = hip_check(launch_twiddles(tw, L.l2, st), "twiddle launch")) return s;
  if (krpe_status_t s = hip_check(launch_spectrum(L.l2, b, tw, Hs, hnorm, H, n, st), "spectrum launch")) return s;
  if (krpe_status_t s = record(events, 1, st)) return s;
  if (krpe_status_t s = hip_check(launch_feature_map(bf16, q, k, W, phiq, phik, 2, true, N, BHi, H, n, d, m, fix,
                                                     nprf, kind, st),
                                  "feature map launch"))
    return s;
  if (krpe_status_t s = hip_check(launch_vprep(bf16, v, d, 1, static_cast<long long>(n) * d, d, true, BHi, n, N,
                                               vmax, colmax, vsc, st),
                                  "column launch"))
    return s;
  if (krpe_status_t s = record(events, 2, st)) return s;
  if (krpe_status_t s = hip_check(launch_conv_split(L.l2, phiq, phik, static_cast<long long>(M) * N, vsc, colmax, Hs,
                                                    nullptr, tw, part, BHi, H, n, d + 1, M, 1, L.fsplit, st),
                                  "conv launch"))
    return s;
  if (krpe_status_t s = record(events, 3, st)) return s;
  if (krpe_status_t s = hip_check(launch_gram(phik, vsc, x2, BHi, M, N, pairs, L.ksplit, st), "norm launch"))
    return s;
  if (krpe_status_t s = hip_check(launch_bound_weights(x2, colmax, wb, BHi, M, d, L.ksplit, st), "bound launch"))
    return s;
  // feature splits: with few (batch, head) rows their partial results are
  // summed first, at full parallelism; the ratio kernel sums them otherwise
  const float* sums = part;
  int nsum = L.fsplit * conv_splits(L.l2);
  if (L.fsplit > 1 && static_cast<long long>(BHi) * ((n + 63) / 64) < 4096) {
    float* psum = reinterpret_cast<float*>(w + L.psum);
    if (krpe_status_t s = hip_check(launch_sum_splits(part, psum, BHi, d + 1, n, n, nsum, st), "sum launch"))
      return s;
    sums = psum;
    nsum = 1;
  }
  if (krpe_status_t s = hip_check(launch_combine(sums, phiq, wb, hnorm, z, den_out, fix, fixmask, BHi, H, n, L.l2, d, M,
                                                 nsum, st),
                                  "combine launch"))
    return s;
  if (krpe_status_t s = hip_check(launch_fixup(phiq, phik, v, bf16, b, z, den_out, fix, fixmask, fixplan, fixpart,
                                               brange, cexp, BHi, H, n, N, d, M, st),
                                  "fixup launch"))
    return s;
  return record(events, 4, st);
}

// Forward pass of Eq. (10) for n > 2^kMaxLog2N on the FFT route: query block
// I's numerators and denominator summed over the key blocks J, each block
// pair one convolution run with the Toeplitz block's bias window; the rows
// certified per block with weights summed over J; the rest evaluated
// directly over the whole sequence.
krpe_status_t run_forward_long(const LongLayout& L, char* w, const void* q, const void* k, const void* v, bool bf16,
                               const float* b, const float* W, float* z, int BHi, int H, int n, int d, int m, int M,
                               int kind, bool nprf, hipStream_t st, void* const* events) {
  auto F = [&](size_t o) { return reinterpret_cast<float*>(w + o); };
  auto F2 = [&](size_t o) { return reinterpret_cast<float2*>(w + o); };
  unsigned* fix = reinterpret_cast<unsigned*>(w + L.fix);
  const int nbk = L.nbk, nb = L.nb, cols = d + 1, pairs = (d + 2) / 2, splits = conv_splits(kMaxLog2N);
  const size_t bhM = static_cast<size_t>(BHi) * M, esz = bf16 ? 2 : 4;
  const int tiles_full = (n + 63) / 64;
  auto len_of = [&](int K) { return n - K * nbk < nbk ? n - K * nbk : nbk; };

  if (krpe_status_t s = record(events, 0, st)) return s;
  if (krpe_status_t s = hip_check(launch_twiddles(F2(L.tw), kMaxLog2N, st), "twiddle launch")) return s;
  if (krpe_status_t s = hip_check(launch_unit_hnorm(F2(L.hunit), H, st), "norm launch")) return s;
  if (krpe_status_t s = record(events, 1, st)) return s;
  if (krpe_status_t s = hip_check(launch_feature_map(bf16, q, k, W, F(L.phiq), F(L.phik), 2, true, L.Ntot, BHi, H, n,
                                                     d, m, fix, nprf, kind, st),
                                  "feature map launch"))
    return s;
  for (int K = 0; K < nb; ++K) {
    float* pqb = F(L.phiqb) + static_cast<size_t>(K) * bhM * nbk;
    float* pkb = F(L.phikb) + static_cast<size_t>(K) * bhM * nbk;
    if (krpe_status_t s = hip_check(launch_block_rows(F(L.phiq), pqb, BHi, M, nbk, L.Ntot, K, st), "block launch"))
      return s;
    if (krpe_status_t s = hip_check(launch_block_rows(F(L.phik), pkb, BHi, M, nbk, L.Ntot, K, st), "block launch"))
      return s;
    // key block K: value column pairs, channel norms and bound weights
    const char* vk = static_cast<const char*>(v) + static_cast<size_t>(K) * nbk * d * esz;
    float2* vscK = F2(L.vsc) + static_cast<size_t>(K) * BHi * pairs * nbk;
    float* colK = F(L.colmax) + static_cast<size_t>(K) * BHi * cols;
    if (krpe_status_t s = hip_check(launch_vprep(bf16, vk, d, 1, static_cast<long long>(n) * d, d, true, BHi,
                                                 len_of(K), nbk, F(L.vmax), colK, vscK, st),
                                    "column launch"))
      return s;
    if (krpe_status_t s = hip_check(launch_gram(pkb, vscK, F(L.x2), BHi, M, nbk, pairs, L.ksplit, st), "norm launch"))
      return s;
    if (krpe_status_t s = hip_check(launch_bound_weights(F(L.x2), colK, F2(L.wbj) + static_cast<size_t>(K) * BHi * (M + 1),
                                                         BHi, M, d, L.ksplit, st),
                                    "bound launch"))
      return s;
  }
  if (krpe_status_t s = record(events, 2, st)) return s;
  for (int I = 0; I < nb; ++I) {
    const int lenI = len_of(I);
    const float* pqb = F(L.phiqb) + static_cast<size_t>(I) * bhM * nbk;
    // the nb blocks of C in block row I: windows, spectra, then every key
    // block in one convolution launch (blocks of C that are all zero skip)
    if (krpe_status_t s = hip_check(launch_bias_window(b, F(L.bwin), H, n, nbk, nb, I, st), "bias launch")) return s;
    if (krpe_status_t s = hip_check(launch_spectrum(kMaxLog2N, F(L.bwin), F2(L.tw), F2(L.hs), F2(L.hnorm), nb * H,
                                                    nbk, st),
                                    "spectrum launch"))
      return s;
    if (krpe_status_t s = hip_check(launch_conv_split(kMaxLog2N, pqb, F(L.phikb), static_cast<long long>(M) * nbk,
                                                      F2(L.vsc), F(L.colmax), F2(L.hs), F2(L.hnorm), F2(L.tw),
                                                      F(L.part), BHi, H, lenI, cols, M, nb, L.fsplit, st),
                                    "conv launch"))
      return s;
    if (krpe_status_t s = hip_check(launch_wb_accum(F2(L.wbi), F2(L.wbj), F2(L.hnorm), BHi, H, M, nb, st),
                                    "weight launch"))
      return s;
    unsigned long long* maskb = reinterpret_cast<unsigned long long*>(w + L.maskb);
    if (krpe_status_t s = hip_check(launch_sum_splits(F(L.part), F(L.psum), BHi, cols, lenI, lenI, nb * L.fsplit * splits, st),
                                    "sum launch"))
      return s;
    if (krpe_status_t s = hip_check(launch_combine(F(L.psum), pqb, F2(L.wbi), F2(L.hunit), F(L.zb), nullptr, fix, maskb,
                                                   BHi, H, lenI, kMaxLog2N, d, M, 1, st),
                                    "combine launch"))
      return s;
    if (krpe_status_t s = hip_check(launch_merge_mask(maskb, reinterpret_cast<unsigned long long*>(w + L.maskf), BHi,
                                                      (lenI + 63) / 64, tiles_full, I, nbk, st),
                                    "mask launch"))
      return s;
    if (krpe_status_t s = hip_check(launch_scatter_rows(F(L.zb), z, BHi, n, nbk, d, I, lenI, st), "rows launch"))
      return s;
  }
  if (krpe_status_t s = record(events, 3, st)) return s;
  if (krpe_status_t s = hip_check(launch_fixup(F(L.phiq), F(L.phik), v, bf16, b, z, nullptr, fix,
                                               reinterpret_cast<unsigned long long*>(w + L.maskf),
                                               reinterpret_cast<int*>(w + L.fixplan),
                                               reinterpret_cast<double*>(w + L.fixpart),
                                               reinterpret_cast<int2*>(w + L.brange), F(L.cexp), BHi, H, n, L.Ntot, d,
                                               M, st),
                                  "fixup launch"))
    return s;
  return record(events, 4, st);
}

// ------------------------------------------------ no-allocation scratch --
// Workspace of krpe_toeplitz_conv_noalloc: a file-scope device array, one copy
// per GPU the library runs on, held from the library's load until the process
// ends.  Host code uses it only through the device address that
// hipGetSymbolAddress returns (looked up once per device, with that device
// current): the array's name on the host is a stand-in, not that address.
constexpr size_t kScratchBytes = static_cast<size_t>(KRPE_NOALLOC_SCRATCH_BYTES);
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices];  // device address of `scratch` per device, once looked up

// Device address of the scratch array on the device `stream` belongs to (the
// current device for the null stream).  The first call on a device makes that
// device current for the lookup and restores the caller's.
krpe_status_t scratch_address(hipStream_t stream, void** out) {
  int cur = 0;
  if (krpe_status_t s = hip_check(hipGetDevice(&cur), "hipGetDevice")) return s;
  int dev = cur;
  if (stream) {
    hipDevice_t sd = 0;
    if (krpe_status_t s = hip_check(hipStreamGetDevice(stream, &sd), "hipStreamGetDevice")) return s;
    dev = static_cast<int>(sd);
  }
  if (dev < 0 || dev >= kMaxDevices) return fail(KRPE_ERR_UNSUPPORTED, "device index beyond the scratch table");
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    if (dev != cur)
      if (krpe_status_t s = hip_check(hipSetDevice(dev), "hipSetDevice")) return s;
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (dev != cur) (void)hipSetDevice(cur);
    if (krpe_status_t s = hip_check(e, "hipGetSymbolAddress(scratch)")) return s;
    if (!p) return fail(KRPE_ERR_HIP, "hipGetSymbolAddress(scratch) returned NULL");
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return KRPE_OK;
}
}  // namespace

// The Toeplitz product of krpe_toeplitz_conv on a given workspace.
krpe_status_t toeplitz_conv(const float* b, const float* a, float* y, int B, int H, int C, int n, void* ws,
                            size_t ws_bytes, void* stream) {
  if (C < 0) return fail(KRPE_ERR_SHAPE, "negative size");
  if (krpe_status_t s = check_dims(B, H, n, 0, 0, false, kMaxLongLog2N)) return s;
  if (static_cast<long long>(B) * H * C * n >= (1LL << 31))
    return fail(KRPE_ERR_UNSUPPORTED, "B * H * C * n >= 2^31 is not supported");
  const size_t bh = static_cast<size_t>(B) * H;
  if (bh == 0 || C == 0) return KRPE_OK;
  if (!b || !a || !y) return fail(KRPE_ERR_NULL, "b, a and y must be non-NULL");
  if (misaligned(b) || misaligned(a) || misaligned(y) || misaligned(ws))
    return fail(KRPE_ERR_ALIGN, "b, a, y, ws must be 16-byte aligned");
  const ConvLayout L = conv_layout(B, H, C, n);
  if (!ws || ws_bytes < L.total)
    return fail(KRPE_ERR_WORKSPACE, "workspace needs " + std::to_string(L.total) + " bytes");
  const Range ry{y, bh * C * n * sizeof(float)};
  const Range rws{ws, ws_bytes};
  const Range ra{a, bh * C * n * sizeof(float)};
  const Range rb{b, static_cast<size_t>(H) * (2 * n - 1) * sizeof(float)};
  if (overlaps(ry, ra) || overlaps(ry, rb) || overlaps(ry, rws) || overlaps(rws, ra) || overlaps(rws, rb))
    return fail(KRPE_ERR_ALIAS, "y or the workspace overlaps an input");
  hipStream_t st = static_cast<hipStream_t>(stream);
  char* w = static_cast<char*>(ws);
  float2* tw = reinterpret_cast<float2*>(w + L.tw);
  float2* Hs = reinterpret_cast<float2*>(w + L.hs);
  float* ones = reinterpret_cast<float*>(w + L.ones);
  float2* vsc = reinterpret_cast<float2*>(w + L.vsc);
  float* colmax = reinterpret_cast<float*>(w + L.colmax);
  float* vmax = reinterpret_cast<float*>(w + L.vmax);
  float* part = reinterpret_cast<float*>(w + L.part);
  const int BHi = static_cast<int>(bh);
  const int N = 1 << L.l2;
  const int splits = conv_splits(L.l2);
  // The product runs through the attention's convolution kernel with one
  // feature equal to 1 everywhere: a_c plays the role of the value column c.
  if (L.nb > 1) {
    // Blocks of nbk positions (Eqs. (12)-(13) per block of C): y_I =
    // sum_J C_IJ a_J, block row I as one launch over the nb key blocks J
    // (blocks of C that are all zero, e.g. above the diagonal under a causal
    // mask, skip their transforms), its partial sums added into y_I.
    const int nbk = L.nbk, nb = L.nb;
    const size_t pairs = (static_cast<size_t>(C) + 1) / 2;
    auto len_of = [&](int K) { return n - K * nbk < nbk ? n - K * nbk : nbk; };
    float* bwin = reinterpret_cast<float*>(w + L.bwin);
    float2* hnorm = reinterpret_cast<float2*>(w + L.hnorm);
    if (krpe_status_t s = hip_check(launch_twiddles(tw, L.l2, st), "twiddle launch")) return s;
    if (krpe_status_t s = hip_check(launch_ones(ones, nbk, nbk, st), "ones launch")) return s;
    for (int J = 0; J < nb; ++J) {
      // key block J's channels, zero past its length
      if (krpe_status_t s = hip_check(launch_vprep(false, a + static_cast<size_t>(J) * nbk, 1, n,
                                                   static_cast<long long>(C) * n, C, false, BHi, len_of(J), nbk,
                                                   vmax, colmax + static_cast<size_t>(J) * bh * C,
                                                   vsc + static_cast<size_t>(J) * bh * pairs * nbk, st),
                                      "column launch"))
        return s;
    }
    for (int I = 0; I < nb; ++I) {
      const int lenI = len_of(I);
      if (krpe_status_t s = hip_check(launch_bias_window(b, bwin, H, n, nbk, nb, I, st), "bias launch")) return s;
      if (krpe_status_t s = hip_check(launch_spectrum(L.l2, bwin, tw, Hs, hnorm, nb * H, nbk, st), "spectrum launch"))
        return s;
      if (krpe_status_t s = hip_check(launch_conv_split(L.l2, ones, ones, 0, vsc, colmax, Hs, hnorm, tw, part, BHi, H,
                                                        lenI, C, 1, nb, 1, st),
                                      "conv launch"))
        return s;
      if (krpe_status_t s = hip_check(launch_sum_splits(part, y + static_cast<size_t>(I) * nbk, BHi, C, lenI, n,
                                                        nb * splits, st),
                                      "sum launch"))
        return s;
    }
    return KRPE_OK;
  }
  if (krpe_status_t s = hip_check(launch_twiddles(tw, L.l2, st), "twiddle launch")) return s;
  if (krpe_status_t s = hip_check(launch_spectrum(L.l2, b, tw, Hs, nullptr, H, n, st), "spectrum launch")) return s;
  if (krpe_status_t s = hip_check(launch_ones(ones, n, N, st), "ones launch")) return s;
  if (krpe_status_t s = hip_check(launch_vprep(false, a, 1, n, static_cast<long long>(C) * n, C, false, BHi, n, N,
                                               vmax, colmax, vsc, st),
                                  "column launch"))
    return s;
  if (krpe_status_t s = hip_check(launch_conv(L.l2, ones, ones, 0, vsc, colmax, Hs, tw, splits > 1 ? part : y, BHi,
                                              H, n, C, 1, st),
                                  "conv launch"))
    return s;
  if (splits > 1) return hip_check(launch_sum_splits(part, y, BHi, C, n, n, splits, st), "sum launch");
  return KRPE_OK;
}

}  // namespace krpe

using namespace krpe;

extern "C" {

int krpe_abi_version(void) { return 6; }

const char* krpe_status_str(int s) {
  switch (s) {
    case KRPE_OK: return "ok";
    case KRPE_ERR_NULL: return "null pointer";
    case KRPE_ERR_SHAPE: return "invalid shape";
    case KRPE_ERR_UNSUPPORTED: return "unsupported size";
    case KRPE_ERR_DTYPE: return "unknown dtype";
    case KRPE_ERR_WORKSPACE: return "workspace missing or too small";
    case KRPE_ERR_ALIAS: return "output overlaps an input or the workspace";
    case KRPE_ERR_HIP: return "HIP runtime error";
    case KRPE_ERR_ALIGN: return "pointer not 16-byte aligned";
    default: return "unknown status";
  }
}

const char* krpe_last_error(void) { return g_last_error.c_str(); }

krpe_status_t krpe_feature_map_ex(const void* x, int x_dtype, const float* W, float* phi, int B, int H, int n,
                                  int d, int m, unsigned flags, void* stream) {
  g_last_error.clear();
  if (krpe_status_t s = check_dims(B, H, n, d, m, true, kMaxLongLog2N)) return s;
  int kind = kFeatPrf, M = m;
  if (krpe_status_t s = feature_kind(flags, d, m, &kind, &M)) return s;
  if (x_dtype != KRPE_F32 && x_dtype != KRPE_BF16) return fail(KRPE_ERR_DTYPE, "x_dtype must be F32 or BF16");
  const size_t bh = static_cast<size_t>(B) * H;
  if (bh == 0) return KRPE_OK;
  const bool needW = kind != kFeatElu;
  if (!x || (needW && !W) || !phi) return fail(KRPE_ERR_NULL, "x, W (but for elu + 1) and phi must be non-NULL");
  if (misaligned(x) || (needW && misaligned(W)) || misaligned(phi))
    return fail(KRPE_ERR_ALIGN, "x, W, phi must be 16-byte aligned");
  const Range rphi{phi, bh * n * M * sizeof(float)};
  if (overlaps(rphi, {x, bh * n * d * dtype_size(x_dtype)}) ||
      (needW && overlaps(rphi, {W, static_cast<size_t>(H) * m * d * sizeof(float)})))
    return fail(KRPE_ERR_ALIAS, "phi overlaps x or W");
  hipStream_t st = static_cast<hipStream_t>(stream);
  return hip_check(launch_feature_map(x_dtype == KRPE_BF16, x, x, W, phi, phi, 1, false, M, static_cast<int>(bh),
                                      H, n, d, m, nullptr, (flags & KRPE_NPRF) != 0, kind, st),
                   "feature map launch");
}

krpe_status_t krpe_feature_map(const void* x, int x_dtype, const float* W, float* phi, int B, int H, int n, int d,
                               int m, void* stream) {
  return krpe_feature_map_ex(x, x_dtype, W, phi, B, H, n, d, m, 0u, stream);
}

size_t krpe_toeplitz_conv_workspace(int B, int H, int C, int n) {
  if (B < 0 || H < 0 || C < 0 || n < 1 || n > (1 << kMaxLongLog2N)) return 0;
  return conv_layout(B, H, C, n).total;
}

krpe_status_t krpe_toeplitz_conv(const float* b, const float* a, float* y, int B, int H, int C, int n, void* ws,
                                 size_t ws_bytes, void* stream) {
  g_last_error.clear();
  return toeplitz_conv(b, a, y, B, H, C, n, ws, ws_bytes, stream);
}

krpe_status_t krpe_toeplitz_conv_noalloc(const float* b, const float* a, float* y, int B, int H, int C, int n,
                                         void* stream) {
  g_last_error.clear();
  // sizes first (no HIP call for a rejected request), then the workspace
  if (C < 0) return fail(KRPE_ERR_SHAPE, "negative size");
  if (krpe_status_t s = check_dims(B, H, n, 0, 0, false, kMaxLongLog2N)) return s;
  if (static_cast<long long>(B) * H * C * n >= (1LL << 31))
    return fail(KRPE_ERR_UNSUPPORTED, "B * H * C * n >= 2^31 is not supported");
  if (static_cast<size_t>(B) * H == 0 || C == 0) return KRPE_OK;
  const size_t need = conv_layout(B, H, C, n).total;
  if (need > kScratchBytes)
    return fail(KRPE_ERR_UNSUPPORTED, "these sizes need " + std::to_string(need) +
                                          " bytes of workspace, more than the " + std::to_string(kScratchBytes) +
                                          " of the static scratch: use krpe_toeplitz_conv with a workspace");
  void* ws = nullptr;
  if (krpe_status_t s = scratch_address(static_cast<hipStream_t>(stream), &ws)) return s;
  return toeplitz_conv(b, a, y, B, H, C, n, ws, kScratchBytes, stream);
}

size_t krpe_attention_fwd_workspace_ex(int B, int H, int n, int d, int m, unsigned flags) {
  if (B < 0 || H < 0 || n < 1 || n > (1 << kMaxLongLog2N) || d < 1 || d > kMaxD || m < 1 || m > kMaxM) return 0;
  int kind = kFeatPrf, M = m;
  if (feature_kind(flags, d, m, &kind, &M) != KRPE_OK) return 0;
  return fwd_workspace(B, H, n, d, M, use_direct(flags, static_cast<long long>(B) * H, n, M, d));
}

size_t krpe_attention_fwd_workspace(int B, int H, int n, int d, int m) {
  return krpe_attention_fwd_workspace_ex(B, H, n, d, m, 0u);
}

krpe_status_t krpe_attention_fwd_profiled(const void* q, const void* k, const void* v, int qkv_dtype, const float* b,
                                          const float* W, float* z, int B, int H, int n, int d, int m, unsigned flags,
                                          void* ws, size_t ws_bytes, void* stream, void* const* events) {
  g_last_error.clear();
  if (krpe_status_t s = check_dims(B, H, n, d, m, true, kMaxLongLog2N)) return s;
  int kind = kFeatPrf, M = m;
  if (krpe_status_t s = feature_kind(flags, d, m, &kind, &M)) return s;
  if (qkv_dtype != KRPE_F32 && qkv_dtype != KRPE_BF16) return fail(KRPE_ERR_DTYPE, "qkv_dtype must be F32 or BF16");
  const size_t bh = static_cast<size_t>(B) * H;
  if (bh == 0) return KRPE_OK;
  const bool needW = kind != kFeatElu;
  if (!q || !k || !v || !b || (needW && !W) || !z)
    return fail(KRPE_ERR_NULL, "q, k, v, b, W (but for elu + 1) and z must be non-NULL");
  if (misaligned(q) || misaligned(k) || misaligned(v) || misaligned(b) || (needW && misaligned(W)) ||
      misaligned(z) || misaligned(ws))
    return fail(KRPE_ERR_ALIGN, "all pointers must be 16-byte aligned");
  const bool direct = use_direct(flags, static_cast<long long>(B) * H, n, M, d);
  const size_t need = fwd_workspace(B, H, n, d, M, direct);
  if (!ws || ws_bytes < need) return fail(KRPE_ERR_WORKSPACE, "workspace needs " + std::to_string(need) + " bytes");
  const size_t qkv_bytes = bh * n * d * dtype_size(qkv_dtype);
  const Range ins[] = {{q, qkv_bytes},
                       {k, qkv_bytes},
                       {v, qkv_bytes},
                       {b, static_cast<size_t>(H) * (2 * n - 1) * sizeof(float)},
                       {W, needW ? static_cast<size_t>(H) * m * d * sizeof(float) : 0}};
  const Range rz{z, bh * n * d * sizeof(float)};
  const Range rws{ws, ws_bytes};
  if (overlaps(rz, rws)) return fail(KRPE_ERR_ALIAS, "z overlaps the workspace");
  for (const Range& r : ins)
    if (overlaps(rz, r) || overlaps(rws, r)) return fail(KRPE_ERR_ALIAS, "z or the workspace overlaps an input");

  if (n > (1 << kMaxLog2N) && !direct)
    return run_forward_long(long_layout(B, H, n, d, M), static_cast<char*>(ws), q, k, v, qkv_dtype == KRPE_BF16, b,
                            W, z, static_cast<int>(bh), H, n, d, m, M, kind, (flags & KRPE_NPRF) != 0,
                            static_cast<hipStream_t>(stream), events);
  return run_forward(attn_layout(B, H, n, d, M), static_cast<char*>(ws), q, k, v, qkv_dtype == KRPE_BF16, b, W, z,
                     nullptr, static_cast<int>(bh), H, n, d, m, M, kind, (flags & KRPE_NPRF) != 0, direct,
                     static_cast<hipStream_t>(stream), events);
}

krpe_status_t krpe_attention_fwd_ex(const void* q, const void* k, const void* v, int qkv_dtype, const float* b,
                                    const float* W, float* z, int B, int H, int n, int d, int m, unsigned flags,
                                    void* ws, size_t ws_bytes, void* stream) {
  return krpe_attention_fwd_profiled(q, k, v, qkv_dtype, b, W, z, B, H, n, d, m, flags, ws, ws_bytes, stream,
                                     nullptr);
}

krpe_status_t krpe_attention_fwd(const void* q, const void* k, const void* v, int qkv_dtype, const float* b,
                                 const float* W, float* z, int B, int H, int n, int d, int m, void* ws,
                                 size_t ws_bytes, void* stream) {
  return krpe_attention_fwd_profiled(q, k, v, qkv_dtype, b, W, z, B, H, n, d, m, 0u, ws, ws_bytes, stream, nullptr);
}

int krpe_attention_fwd_route(int B, int H, int n, int d, int m, unsigned flags) {
  if (B < 1 || H < 1 || n < 1 || n > (1 << kMaxLongLog2N) || d < 1 || d > kMaxD || m < 1 || m > kMaxM) return 0;
  int kind = kFeatPrf, M = m;
  if (feature_kind(flags, d, m, &kind, &M) != KRPE_OK) return 0;
  return use_direct(flags, static_cast<long long>(B) * H, n, M, d) ? static_cast<int>(KRPE_ROUTE_DIRECT)
                                                                   : static_cast<int>(KRPE_ROUTE_FFT);
}

size_t krpe_attention_bwd_workspace(int B, int H, int n, int d, int m, unsigned flags) {
  if (B < 0 || H < 0 || n < 1 || n > (1 << kMaxLog2N) || d < 1 || d > kMaxD || m < 1 || m > kMaxM) return 0;
  if (flags & ~kBwdFlags) return 0;
  return bwd_layout(B, H, n, d, m).total;
}

krpe_status_t krpe_attention_bwd(const void* q, const void* k, const void* v, int qkv_dtype, const float* b,
                                 const float* W, const float* dz, float* dq, float* dk, float* dv, float* db, int B,
                                 int H, int n, int d, int m, unsigned flags, void* ws, size_t ws_bytes,
                                 void* stream) {
  g_last_error.clear();
  if (krpe_status_t s = check_dims(B, H, n, d, m, true)) return s;
  if (flags & ~kBwdFlags)
    return fail(KRPE_ERR_UNSUPPORTED, "the backward pass takes KRPE_NPRF, the route bits and KRPE_HINT_CAUSAL (PRF features)");
  if ((flags & KRPE_ROUTE_DIRECT) && (flags & KRPE_ROUTE_FFT))
    return fail(KRPE_ERR_UNSUPPORTED, "KRPE_ROUTE_DIRECT and KRPE_ROUTE_FFT are exclusive");
  if (qkv_dtype != KRPE_F32 && qkv_dtype != KRPE_BF16) return fail(KRPE_ERR_DTYPE, "qkv_dtype must be F32 or BF16");
  const size_t bh = static_cast<size_t>(B) * H;
  if (bh == 0) return KRPE_OK;
  if (!q || !k || !v || !b || !W || !dz || !dq || !dk || !dv)
    return fail(KRPE_ERR_NULL, "q, k, v, b, W, dz, dq, dk and dv must be non-NULL");
  const void* ptrs[] = {q, k, v, b, W, dz, dq, dk, dv, ws};
  for (const void* p : ptrs)
    if (misaligned(p)) return fail(KRPE_ERR_ALIGN, "all pointers must be 16-byte aligned");
  const BwdLayout L = bwd_layout(B, H, n, d, m);
  if (!ws || ws_bytes < L.total)
    return fail(KRPE_ERR_WORKSPACE, "workspace needs " + std::to_string(L.total) + " bytes");
  const size_t qkv_bytes = bh * n * d * dtype_size(qkv_dtype), g_bytes = bh * n * d * sizeof(float);
  const Range ins[] = {{q, qkv_bytes},
                       {k, qkv_bytes},
                       {v, qkv_bytes},
                       {b, static_cast<size_t>(H) * (2 * n - 1) * sizeof(float)},
                       {W, static_cast<size_t>(H) * m * d * sizeof(float)},
                       {dz, g_bytes}};
  if (misaligned(db)) return fail(KRPE_ERR_ALIGN, "all pointers must be 16-byte aligned");
  const Range outs[] = {{dq, g_bytes}, {dk, g_bytes}, {dv, g_bytes}, {ws, ws_bytes},
                        {db, db ? static_cast<size_t>(H) * (2 * n - 1) * sizeof(float) : 0}};
  for (int o = 0; o < 5; ++o) {
    for (const Range& r : ins)
      if (overlaps(outs[o], r)) return fail(KRPE_ERR_ALIAS, "an output or the workspace overlaps an input");
    for (int o2 = o + 1; o2 < 5; ++o2)
      if (overlaps(outs[o], outs[o2])) return fail(KRPE_ERR_ALIAS, "outputs overlap each other or the workspace");
  }

  hipStream_t st = static_cast<hipStream_t>(stream);
  char* w = static_cast<char*>(ws);
  const int BHi = static_cast<int>(bh);
  const bool bf16 = qkv_dtype == KRPE_BF16, nprf = (flags & KRPE_NPRF) != 0;
  const int N = 1 << L.f.l2, splits = conv_splits(L.f.l2);
  float* zf = reinterpret_cast<float*>(w + L.zf);
  float* den = reinterpret_cast<float*>(w + L.den);
  float* brev = reinterpret_cast<float*>(w + L.brev);
  float2* hsr = reinterpret_cast<float2*>(w + L.hsr);
  float* gh = reinterpret_cast<float*>(w + L.gh);
  float* vh = reinterpret_cast<float*>(w + L.vh);
  float2* vsc = reinterpret_cast<float2*>(w + L.vsc);
  float* colmax = reinterpret_cast<float*>(w + L.colmax);
  float* vmax = reinterpret_cast<float*>(w + L.vmax);
  float* part = reinterpret_cast<float*>(w + L.part);
  const float2* tw = reinterpret_cast<const float2*>(w + L.f.tw);
  const float2* Hs = reinterpret_cast<const float2*>(w + L.f.hs);
  const float* phiq = reinterpret_cast<const float*>(w + L.f.phiq);
  const float* phik = reinterpret_cast<const float*>(w + L.f.phik);
  const long long fstride = static_cast<long long>(m) * N, gstride = static_cast<long long>(d + 1) * N;

  // forward: phi(q), phi(k), z and the denominators
  const bool direct = use_direct(flags, static_cast<long long>(B) * H, n, m, d);
  if (krpe_status_t s = run_forward(L.f, w, q, k, v, bf16, b, W, zf, den, BHi, H, n, d, m, m, kFeatPrf, nprf, direct,
                                    st, nullptr))
    return s;
  if (direct) {
    // the direct forward needs no transforms; the backward's products do
    float2* twm = reinterpret_cast<float2*>(w + L.f.tw);
    float2* Hsm = reinterpret_cast<float2*>(w + L.f.hs);
    if (krpe_status_t s = hip_check(launch_twiddles(twm, L.f.l2, st), "twiddle launch")) return s;
    if (krpe_status_t s = hip_check(launch_spectrum(L.f.l2, b, twm, Hsm, nullptr, H, n, st), "spectrum launch"))
      return s;
  }
  if (krpe_status_t s = hip_check(launch_bwd_prep(bf16, dz, zf, den, v, gh, vh, BHi, n, N, d, st), "prep launch"))
    return s;
  if (krpe_status_t s = hip_check(launch_reverse_bias(b, brev, n, H, st), "bias launch")) return s;
  if (krpe_status_t s = hip_check(launch_spectrum(L.f.l2, brev, tw, hsr, nullptr, H, n, st), "spectrum launch"))
    return s;
  // dv = sum_l phi_l(k) o C^T (phi_l(q) o Gh_c)
  if (krpe_status_t s = hip_check(launch_vprep(false, gh, 1, N, gstride, d + 1, false, BHi, n, N, vmax, colmax, vsc,
                                               st),
                                  "column launch"))
    return s;
  if (krpe_status_t s = hip_check(launch_conv(L.f.l2, phik, phiq, fstride, vsc, colmax, hsr, tw, part, BHi, H, n,
                                              d + 1, m, st),
                                  "conv launch"))
    return s;
  if (krpe_status_t s = hip_check(launch_bwd_dv(part, dv, BHi, n, d, d + 1, splits, st), "dv launch")) return s;
  // db_t = c_t sum_lc corr(phi_l(q) o Gh_c, phi_l(k) o V'_c)(t)
  if (db) {
    if (krpe_status_t s = hip_check(
            launch_db(L.f.l2, phiq, phik, fstride, gh, vh, tw, reinterpret_cast<float2*>(w + L.gpk),
                      reinterpret_cast<float2*>(w + L.vpk), reinterpret_cast<float2*>(w + L.spart),
                      reinterpret_cast<float2*>(w + L.sh), reinterpret_cast<float2*>(w + L.ycorr), b, db, B, H, n,
                      d + 1, m, st),
            "db launch"))
      return s;
  }
  // dphi_l(q) = sum_c Gh_c o C (V'_c o phi_l(k)), then dq
  if (krpe_status_t s = hip_check(launch_vprep(false, phik, 1, N, fstride, m, false, BHi, n, N, vmax, colmax, vsc,
                                               st),
                                  "column launch"))
    return s;
  if (krpe_status_t s = hip_check(launch_conv(L.f.l2, gh, vh, gstride, vsc, colmax, Hs, tw, part, BHi, H, n, m, d + 1,
                                              st),
                                  "conv launch"))
    return s;
  if (krpe_status_t s = hip_check(launch_feature_bwd(bf16, q, W, phiq, part, dq, BHi, H, n, N, d, m, splits, nprf,
                                                     st),
                                  "feature launch"))
    return s;
  // dphi_l(k) = sum_c V'_c o C^T (Gh_c o phi_l(q)), then dk
  if (krpe_status_t s = hip_check(launch_vprep(false, phiq, 1, N, fstride, m, false, BHi, n, N, vmax, colmax, vsc,
                                               st),
                                  "column launch"))
    return s;
  if (krpe_status_t s = hip_check(launch_conv(L.f.l2, vh, gh, gstride, vsc, colmax, hsr, tw, part, BHi, H, n, m,
                                              d + 1, st),
                                  "conv launch"))
    return s;
  return hip_check(launch_feature_bwd(bf16, k, W, phik, part, dk, BHi, H, n, N, d, m, splits, nprf, st),
                   "feature launch");
}

krpe_status_t krpe_attention_fwd_stats(const void* ws, size_t ws_bytes, int B, int H, int n, int d, int m,
                                       unsigned* fixed_rows, void* stream) {
  g_last_error.clear();
  if (krpe_status_t s = check_dims(B, H, n, d, m, true, kMaxLongLog2N)) return s;
  if (!fixed_rows) return fail(KRPE_ERR_NULL, "fixed_rows must be non-NULL");
  *fixed_rows = 0;
  if (static_cast<size_t>(B) * H == 0) return KRPE_OK;
  if (!ws) return fail(KRPE_ERR_NULL, "ws must be non-NULL");
  // The counters sit at the start of the workspace whatever the feature map.
  const AttnLayout L = attn_layout(B, H, n, d, m);
  if (ws_bytes < L.fix + (static_cast<size_t>(B) * H + 1) * sizeof(unsigned))
    return fail(KRPE_ERR_WORKSPACE, "workspace smaller than these sizes need");
  hipStream_t st = static_cast<hipStream_t>(stream);
  if (krpe_status_t s = hip_check(hipStreamSynchronize(st), "hipStreamSynchronize")) return s;
  return hip_check(
      hipMemcpy(fixed_rows, static_cast<const char*>(ws) + L.fix + static_cast<size_t>(B) * H * sizeof(unsigned),
                sizeof(unsigned), hipMemcpyDeviceToHost),
      "hipMemcpy");
}

}  // extern "C"
