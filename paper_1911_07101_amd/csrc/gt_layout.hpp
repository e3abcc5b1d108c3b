// Register/LDS layout of one transform inside the blind-rotation kernels.
//
// The ring product works on the folded polynomial of n = N/2 complex points
// (coefficients j and j + n of a real polynomial form point j).  A transform
// of 2^LOGN points is spread over T = 2^LOGN / E threads holding E = 2^LOGE
// points each.  The transform (Cooley-Tukey forward, Gentleman-Sande inverse,
// one twiddle per butterfly block) is split into passes; pass p owns a window
// of LOGE index bits starting at bit w(p), and thread t's element e is point
//
//     j = (t mod 2^w) | (e << w) | ((t >> w) << (w + LOGE)),
//
// so every butterfly of the stages whose bit lies in the window is in
// registers.  Between passes the points are transposed through LDS.
// Pass 0 (window at the top) is the coefficient layout j = t + T*e used for
// rotation, decomposition and the accumulator; the last pass (window at bit 0)
// is the transform-domain layout, in which the bootstrapping key is stored.
#pragma once
#include <cstdint>

#ifdef __HIPCC__
#include <hip/hip_runtime.h>
#define GL_HD __host__ __device__ __forceinline__
#else
#define GL_HD inline
#endif

namespace gt {

// complex points per thread of the ring transform (log2)
constexpr int kRingLogE = 2;

template <int LOGN_, int LOGE_>
struct Layout {
  static constexpr int LOGN = LOGN_;
  static constexpr int N = 1 << LOGN;
  static constexpr int LOGE = LOGE_;
  static constexpr int E = 1 << LOGE;
  static constexpr int LOGT = LOGN - LOGE;
  static constexpr int T = 1 << LOGT;
  static constexpr int NPASS = (LOGN + LOGE - 1) / LOGE;

  // stages handled in pass p: bits [lo(p), hi(p)); window start w(p)
  static constexpr GL_HD int hi(int p) { return LOGN - p * LOGE; }
  static constexpr GL_HD int lo(int p) { return LOGN - (p + 1) * LOGE > 0 ? LOGN - (p + 1) * LOGE : 0; }
  static constexpr GL_HD int win(int p) { return lo(p) < LOGN - LOGE ? lo(p) : LOGN - LOGE; }

  static GL_HD int jmap(int t, int e, int w) {
    return (t & ((1 << w) - 1)) | (e << w) | ((t >> w) << (w + LOGE));
  }
  // point index of (t, e) in the transform-domain layout
  static GL_HD int jfinal(int t, int e) { return jmap(t, e, win(NPASS - 1)); }
};

// the ring transform for ring degree 2^LOGN_RING: 2^(LOGN_RING-1) complex points
template <int LOGN_RING>
using RingLayout = Layout<LOGN_RING - 1, kRingLogE>;

}  // namespace gt
