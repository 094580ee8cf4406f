// The convolution kernel at N = 2^kMaxLog2N (n up to 16384, and every block
// pair of a longer sequence), compiled on its own: the build gives this
// translation unit the maximum-ILP instruction scheduler, measured faster
// for this length only (the shorter lengths in kernels.hip keep the default).
#include "conv.hpp"

namespace krpe {

hipError_t conv_launch_top(const float* phiq, const float* phik, long long phi_bh_stride, const float2* vsc,
                           const float* colmax, const float2* Hs, const float2* hnorm, const float2* tw, float* part,
                           int BH, int H, int n, int cols, int m, int nkb, int fsplit, hipStream_t st) {
  return conv_launch<kMaxLog2N>(phiq, phik, phi_bh_stride, vsc, colmax, Hs, hnorm, tw, part, BH, H, n, cols, m, nkb,
                                fsplit, st);
}

}  // namespace krpe
