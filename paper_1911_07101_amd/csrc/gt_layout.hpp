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

// log2 of the complex points per thread of the ring transform: 8 points when
// the key is split into two parts (a lane's four transform-domain accumulators
// then take 128 registers), 4 points with three parts (six accumulators)
GL_HD constexpr int ring_log_e(int parts) { return parts == 2 ? 3 : 2; }

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

  // LDS slot of point j in the transpose scratch.  8 points per thread: one
  // pad slot after every 8 points; the slot of jmap(t, e, w) is then an
  // affine function of e (for w = 0 or w >= 3) and every group of 8
  // consecutive lanes touches 8 distinct 16-byte bank groups in each pass
  // layout.  4 points per thread: the low 4 bits are XORed with bits 1..4,
  // which is conflict-free for every pass layout of 128..1024 points.
  static GL_HD int slot(int j) {
    if constexpr (LOGE == 3)
      return j + (j >> 3);
    else
      return j ^ (((j >> 1) ^ (j >> 2)) & 15);
  }
  static constexpr int SCR = LOGE == 3 ? N + N / 8 : N;  // scratch slots per polynomial
  // slot(jmap(t, e, w)) = slot(jmap(t, 0, w)) + e * slot_stride(w) when affine(w)
  static constexpr GL_HD bool affine(int w) { return LOGE == 3 && (w == 0 || w >= 3); }
  static constexpr GL_HD int slot_stride(int w) { return w == 0 ? 1 : (1 << w) + (1 << (w - 3)); }
};

// the ring transform for ring degree 2^LOGN_RING (2^(LOGN_RING-1) complex
// points) with the key split into S parts
template <int LOGN_RING, int S>
using RingLayout = Layout<LOGN_RING - 1, ring_log_e(S)>;

}  // namespace gt
