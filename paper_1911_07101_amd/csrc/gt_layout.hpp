// Register/LDS layout of one polynomial inside the blind-rotation kernels.
//
// A ciphertext's polynomial of N = 2^LOGN coefficients is spread over
// T = N / E threads holding E = 2^LOGE values each.  The negacyclic NTT
// (Cooley-Tukey forward, Gentleman-Sande inverse, twiddles in bit-reversed
// order) is split into passes; pass p owns a window of LOGE index bits
// starting at bit w(p), and thread t's element e is coefficient
//
//     j = (t mod 2^w) | (e << w) | ((t >> w) << (w + LOGE)),
//
// so every butterfly of the stages whose bit lies in the window is in
// registers.  Between passes the polynomial is transposed through LDS.
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

// log2 of the values per thread for a ring of degree 2^logn (host and device)
constexpr GL_HD int log_values_per_thread(int logn) { return logn >= 9 ? 3 : logn - 6; }

template <int LOGN_>
struct Layout {
  static constexpr int LOGN = LOGN_;
  static constexpr int N = 1 << LOGN;
  // 8 values per thread (4 at N = 256): the four transform-domain
  // accumulators of an external product then take 64 registers per thread
  static constexpr int LOGE = log_values_per_thread(LOGN);
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
  // coefficient index of (t, e) in the transform-domain layout
  static GL_HD int jfinal(int t, int e) { return jmap(t, e, win(NPASS - 1)); }
};

}  // namespace gt
