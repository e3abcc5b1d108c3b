// HIP kernels of the TFHE activation path for gfx950 (MI355X).
//
//   prep_kernel            gate pre-combination (Section 3.1 gates; NOT is free)
//                          and modulus switch of every LWE word to Z_{2N}
//   mux_combine_kernel     OR of a multiplexer's two exclusive halves
//   lut_leaf_kernel        first multiplexer-tree level over constant leaves
//   blind_rotate_kernel    accumulator init, n CMux external products,
//                          SampleExtract; one wave per ciphertext (N <= 1024)
//   blind_rotate_split_kernel  the same with two waves per ciphertext, each
//                          computing one half of every transform (N = 2048)
//   keyswitch_init_kernel, keyswitch_mfma_kernel  LWE key switching back to
//                          dimension n for t = 8, base 4: (0, b), then an exact
//                          int8 product on the matrix cores added to it
//   keyswitch_kernel       the same for any other digit count and base
//   relu_sign_kernel       trivial 0 for the sign bit of the ReLU output
//   cmux_abar_kernel       modulus-switched inputs of a one-CMux stage check
//   not_kernel             NOT without bootstrapping
//   pack_init_kernel, pack_ks_fft_kernel, pack_ks_kernel  functional key
//                          switching of LWE samples into one ring sample (on
//                          the transform for N <= 1024, else directly)
//   sample_extract_kernel  LWE samples of chosen coefficients of ring samples
//   negacyclic_mul_kernel  standalone ring product (checks the transform)
//
// The external product's negacyclic products are computed with a complex
// fp64 transform of the folded polynomial (N/2 points) and rounded back to
// integers; the key is split into signed parts small enough that the
// transform's worst-case error stays below 1/8, so the rounded result equals
// the exact product (bound in gt_host.cpp, transform_error_bound).
//
// Blind rotation layout (gt_layout.hpp): a ciphertext's transforms are held
// by N/16 lanes with 8 complex points each when the key has two parts: one
// wave at N = 1024, two at N = 2048.  The accumulator (two u32 polynomials),
// a transpose scratch per wave and copies of the twiddle tables live in LDS;
// the transform-domain accumulators of an external product ((mask, body) x
// key parts) live in registers.  The bootstrapping key is read from global
// memory in the transform-domain layout, one 16-byte point per load,
// coalesced across the wave and shared by the block's ciphertexts through L1.
#include <hip/hip_runtime.h>

#include <type_traits>

#include "gt_internal.h"
#include "gt_layout.hpp"

namespace gt {

namespace {

constexpr uint32_t kMu = 0x20000000u;  // 1/8



template <int B, int E, class F>
__device__ __forceinline__ void static_for(F&& f) {
  if constexpr (B < E) {
    f(std::integral_constant<int, B>{});
    static_for<B + 1, E>(f);
  }
}

// ----------------------------------------------------------- complex fp64
__device__ __forceinline__ double2 cmul(double2 a, double2 w) {
  return make_double2(fma(a.x, w.x, -(a.y * w.y)), fma(a.x, w.y, a.y * w.x));
}
__device__ __forceinline__ double2 cadd(double2 a, double2 b) { return make_double2(a.x + b.x, a.y + b.y); }
__device__ __forceinline__ double2 csub(double2 a, double2 b) { return make_double2(a.x - b.x, a.y - b.y); }
__device__ __forceinline__ void cmac(double2& acc, double2 a, double2 w) {
  acc.x = fma(a.x, w.x, acc.x);
  acc.x = fma(-a.y, w.y, acc.x);
  acc.y = fma(a.x, w.y, acc.y);
  acc.y = fma(a.y, w.x, acc.y);
}

// v is within 1/2 of an integer k with |k| < 2^51: adding 1.5 * 2^52 rounds it
// to k + 1.5 * 2^52, whose mantissa field is k + 2^51, so the low 32 bits of
// the double's bit pattern are k mod 2^32
__device__ __forceinline__ uint32_t round_low32(double v) {
  const double s = v + 6755399441055744.0;
  return static_cast<uint32_t>(__double_as_longlong(s));
}

// Make LDS writes of all threads of a polynomial visible to its other threads.
// A polynomial held by one wave needs only ordering: a wave's LDS operations
// are performed in issue order, so a wavefront-scope fence emits no wait and
// only keeps the compiler from moving LDS accesses across it.  A polynomial
// spread over several waves needs the block barrier.
template <int T>
__device__ __forceinline__ void poly_sync() {
  if constexpr (T <= 64) {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  } else {
    __syncthreads();
  }
}

// Position of twiddle k in the LDS copy of the twiddle table.  Stage s owns
// k in [n/2^(s+1), n/2^s); in a pass other than the first, thread t reads the
// stage's entries m = (t >> w) * G + g, g < G, so they are stored [g][t >> w]
// to make the threads of a wave read consecutive entries.  First-pass
// twiddles are the same for every thread, are read from global memory through
// the scalar cache, and keep their natural place.
template <class Lay>
__host__ __device__ constexpr int tw_lds_slot(int k) {
  if (k == 0) return 0;
  int lg = 0;
  while ((2 << lg) <= k) lg++;           // floor(log2 k)
  const int s = Lay::LOGN - 1 - lg;      // stage of k
  int p = 0;
  while (!(Lay::lo(p) <= s && s < Lay::hi(p))) p++;
  if (p == 0) return k;
  const int b = s - Lay::win(p);
  const int G = Lay::E >> (b + 1);
  const int start = Lay::N >> (s + 1);
  const int m = k - start;
  const int rows = start / G;
  return start + (m % G) * rows + m / G;
}

template <class Lay, int WFROM, int WTO, bool PRIO>
__device__ __forceinline__ void transpose(double2 (&x)[Lay::E], int t, double2* scr) {
  // one base address per layout where the slots are affine in e (immediate offsets)
  double2* wr = scr + Lay::slot(Lay::jmap(t, 0, WFROM));
  double2* rd = scr + Lay::slot(Lay::jmap(t, 0, WTO));
  // PRIO: the wave's instruction-issue priority is raised while it issues
  // the transpose's LDS operations, so that they are queued before the other
  // waves' arithmetic and their latency overlaps it
  if constexpr (PRIO) __builtin_amdgcn_s_setprio(3);
  static_for<0, Lay::E>([&](auto EI) {
    constexpr int e = decltype(EI)::value;
    if constexpr (Lay::affine(WFROM))
      wr[e * Lay::slot_stride(WFROM)] = x[e];
    else
      scr[Lay::slot(Lay::jmap(t, e, WFROM))] = x[e];
  });
  poly_sync<Lay::T>();
  static_for<0, Lay::E>([&](auto EI) {
    constexpr int e = decltype(EI)::value;
    if constexpr (Lay::affine(WTO))
      x[e] = rd[e * Lay::slot_stride(WTO)];
    else
      x[e] = scr[Lay::slot(Lay::jmap(t, e, WTO))];
  });
  if constexpr (PRIO) __builtin_amdgcn_s_setprio(0);
  poly_sync<Lay::T>();
}

// Twiddle g of stage s (bit b of the window at w) for thread t: pass 0's are
// the same for every thread (tw_uniform, global memory, read through the
// scalar cache), the others come from tw, an LDS copy laid out by
// tw_lds_slot (TW_PERMUTED) or a natural-order table.
// `tree` selects the tree whose pass-0 twiddles tw_uniform holds: 1 for a
// transform of the whole tree, 2 + h for the subtree under node 2 + h of a
// tree twice as large (its node m at the stage's level is node m + (1 + h)
// times the level's first index there).
template <class Lay, bool TW_PERMUTED, int p, int s, int g>
__device__ __forceinline__ double2 twiddle(int t, const double2* __restrict__ tw,
                                           const double2* __restrict__ tw_uniform, int tree) {
  constexpr int N = Lay::N, LOGE = Lay::LOGE, E = Lay::E;
  constexpr int w = Lay::win(p);
  constexpr int b = s - w;
  constexpr int G = E >> (b + 1);
  if constexpr (p == 0)
    return tw_uniform[(N >> (s + 1)) * tree + g];
  else if constexpr (TW_PERMUTED)
    return tw[(N >> (s + 1)) + g * ((N >> (s + 1)) / G) + (t >> w)];
  else
    return tw[(N >> (s + 1)) + ((t >> w) << (LOGE - b - 1)) + g];
}

// signed bit field [pos, pos + width) of x, 0 < width < 32, in one
// instruction.  Written as inline assembly: the compiler's own bit-field
// intrinsic has been seen followed by an unsigned int-to-double conversion
// here, which would turn negative digits positive.
__device__ __forceinline__ int32_t signed_field(uint32_t x, uint32_t pos, uint32_t width) {
  int32_t r;
  asm("v_bfe_i32 %0, %1, %2, %3" : "=v"(r) : "v"(x), "s"(pos), "v"(width));
  return r;
}

// Cooley-Tukey butterfly (xe, xe2) <- (u + w v, u - w v): a = u + w v in four
// FMAs, b = 2u - a in two
__device__ __forceinline__ void ct_butterfly(double2& xe, double2& xe2, double2 w) {
  const double2 u = xe, v = xe2;
  const double2 a = make_double2(fma(w.x, v.x, fma(-w.y, v.y, u.x)), fma(w.x, v.y, fma(w.y, v.x, u.y)));
  xe = a;
  xe2 = make_double2(fma(2.0, u.x, -a.x), fma(2.0, u.y, -a.y));
}

// Forward transform of the folded polynomial over C[X]/(X^n - i)
// (Cooley-Tukey butterflies; the block of point j at stage s splits tree node
// k = n/2^(s+1) + j/2^(s+1) and multiplies by tw[k]).  In: pass-0 (coefficient)
// layout; out: last-pass (transform) layout.  Each stage fetches its own
// twiddles (one per butterfly group of the thread).
struct NoHook {
  __device__ void operator()() const {}
};

// hook() runs after the butterflies of pass HOOK_PASS (between that pass and
// the next transpose)
template <class Lay, bool TW_PERMUTED, bool PRIO = false, int HOOK_PASS = -1, class Hook = NoHook>
__device__ __forceinline__ void fft_forward(double2 (&x)[Lay::E], int t, double2* scr,
                                            const double2* __restrict__ tw,
                                            const double2* __restrict__ tw_uniform, int tree = 1,
                                            Hook hook = {}) {
  constexpr int E = Lay::E;
  static_for<0, Lay::NPASS>([&](auto PI) {
    constexpr int p = decltype(PI)::value;
    constexpr int w = Lay::win(p);
    constexpr int NS = Lay::hi(p) - Lay::lo(p);
    // the first stage's twiddles are requested before the pass's transpose and
    // the other stages' right after it, so that their round trips overlap the
    // transpose and the first stage instead of following each other.  A
    // thread's twiddles g and g + 1 (g even) belong to sibling tree nodes 2k
    // and 2k + 1, whose twiddles differ by the factor zeta^{N/2} = i: only
    // the even ones are read, the odd ones are i times them (exact: a swap
    // and a sign, which the butterflies' FMAs take as source modifiers)
    double2 z[NS][E / 2];
    auto fetch = [&](auto SI) {
      constexpr int s = Lay::hi(p) - 1 - decltype(SI)::value;
      constexpr int G = E >> (s - w + 1);
      static_for<0, G>([&](auto GI) {
        constexpr int g = decltype(GI)::value;
        if constexpr ((g & 1) == 0)
          z[decltype(SI)::value][g] = twiddle<Lay, TW_PERMUTED, p, s, g>(t, tw, tw_uniform, tree);
        else
          z[decltype(SI)::value][g] = make_double2(-z[decltype(SI)::value][g - 1].y, z[decltype(SI)::value][g - 1].x);
      });
    };
    fetch(std::integral_constant<int, 0>{});
    if constexpr (p > 0) transpose<Lay, Lay::win(p - 1), w, PRIO>(x, t, scr);
    static_for<1, NS>(fetch);
    static_for<0, NS>([&](auto SI) {
      constexpr int s = Lay::hi(p) - 1 - decltype(SI)::value;
      constexpr int b = s - w;
      constexpr int G = E >> (b + 1);
      static_for<0, G>([&](auto GI) {
        constexpr int g = decltype(GI)::value;
        static_for<0, (1 << b)>([&](auto LI) {
          constexpr int e = (g << (b + 1)) | decltype(LI)::value;
          constexpr int e2 = e | (1 << b);
          ct_butterfly(x[e], x[e2], z[decltype(SI)::value][g]);
        });
      });
    });
    if constexpr (p == HOOK_PASS) hook();
  });
}

// Butterfly of the inverse's stages s < 3 in the pass whose window starts at
// bit 0: the twiddle w^{-g} of order 2^(s+1) is e^{-i pi q/4}, q = g 2^(2-s),
// a constant (1 and -i take no multiplication)
template <int s, int g>
__device__ __forceinline__ void dit_const_butterfly(double2& xe, double2& xe2) {
  constexpr int q = g << (2 - s);
  constexpr double r = 0.70710678118654757;  // 1/sqrt(2) rounded to nearest
  const double2 u = xe, v = xe2;
  if constexpr (q == 0) {
    xe = cadd(u, v);
    xe2 = csub(u, v);
  } else if constexpr (q == 2) {  // -i v = (v.y, -v.x)
    xe = make_double2(u.x + v.y, u.y - v.x);
    xe2 = make_double2(u.x - v.y, u.y + v.x);
  } else {
    ct_butterfly(xe, xe2, make_double2(q == 1 ? r : -r, -r));
  }
}

// Inverse transforms without the 1/n factor of polynomials x[K0 .. K0+K).
// The forward transform leaves at tree position j the value at the root
// zeta0 w^m of X^n = i with m the bit reversal of j (w = e^{2 pi i/n},
// zeta0 = e^{i pi/(2n)}), so the inverse is a cyclic inverse DFT by
// decimation in time (bit-reversed in, natural out; stage s is the butterfly
// (u, v) -> (u + t v, u - t v) on positions j, j + 2^s with
// t = e^{-2 pi i (j mod 2^s) / 2^(s+1)}) followed by the twist zeta0^{-k} of
// output k, which the caller applies.  The twiddles of stage s are
// entry 2^s - 1 + c of the table itw, c = j mod 2^s, read as itw(lane part
// of the index, constant part); the polynomials share them, and one
// polynomial's transpose is in flight while another's butterflies run.
// In: transform layout; out: coefficient layout.
template <class Lay, int K0, int K, bool PRIO = false, int M, class Tab>
__device__ __forceinline__ void fft_inverse(double2 (&x)[M][Lay::E], int t, double2* scr, const Tab& itw) {
  static_assert(K0 + K <= M, "polynomial range");
  constexpr int E = Lay::E;
  static_for<0, Lay::NPASS>([&](auto PI) {
    constexpr int p = Lay::NPASS - 1 - decltype(PI)::value;
    constexpr int w = Lay::win(p);
    constexpr int NS = Lay::hi(p) - Lay::lo(p);
    // stage twiddles of the pass (none in the pass whose window starts at bit
    // 0: constants there), requested before its transposes.  Twiddle g + NG/2
    // of a stage (NG = 2^b per thread) has the angle index c + 2^(s-1) of
    // twiddle g, so it is -i times it: only the first half is read
    double2 zp[NS][E / 2];
    if constexpr (w != 0) {
      const int lane = t & ((1 << w) - 1);
      static_for<0, NS>([&](auto SI) {
        constexpr int s = Lay::lo(p) + decltype(SI)::value;
        constexpr int NG = 1 << (s - w);
        static_for<0, NG>([&](auto GI) {
          constexpr int g = decltype(GI)::value;
          if constexpr (NG == 1 || g < NG / 2)
            zp[decltype(SI)::value][g] = itw(lane, (1 << s) - 1 + (g << w));
          else
            zp[decltype(SI)::value][g] =
                make_double2(zp[decltype(SI)::value][g - NG / 2].y, -zp[decltype(SI)::value][g - NG / 2].x);
        });
      });
    }
    if constexpr (p < Lay::NPASS - 1)
      static_for<K0, K0 + K>([&](auto KI) { transpose<Lay, Lay::win(p + 1), w, PRIO>(x[decltype(KI)::value], t, scr); });
    static_for<0, NS>([&](auto SI) {
      constexpr int s = Lay::lo(p) + decltype(SI)::value;
      constexpr int b = s - w;
      constexpr int NG = 1 << b;  // twiddles per thread: one per value of the element bits below b
      if constexpr (w == 0) {
        static_for<K0, K0 + K>([&](auto KI) {
          constexpr int k = decltype(KI)::value;
          static_for<0, E>([&](auto EI) {
            constexpr int e = decltype(EI)::value;
            if constexpr ((e & NG) == 0) dit_const_butterfly<s, e & (NG - 1)>(x[k][e], x[k][e | NG]);
          });
        });
      } else {
        // position j mod 2^s = (t mod 2^w) | ((e mod 2^b) << w)
        static_for<K0, K0 + K>([&](auto KI) {
          constexpr int k = decltype(KI)::value;
          static_for<0, E>([&](auto EI) {
            constexpr int e = decltype(EI)::value;
            if constexpr ((e & NG) == 0) ct_butterfly(x[k][e], x[k][e | NG], zp[decltype(SI)::value][e & (NG - 1)]);
          });
        });
      }
    });
  });
}

// coefficient j of X^e * p for e in [0, 2N), p in LDS: p[(j - e) mod N],
// negated when the index wrapped or when e >= N (X^N = -1), without branches
template <int N>
__device__ __forceinline__ uint32_t rot_coef(const uint32_t* p, uint32_t e, int j) {
  const int src = j - static_cast<int>(e & (N - 1));
  const uint32_t v = p[src & (N - 1)];
  const uint32_t m = static_cast<uint32_t>(src >> 31) ^ (0u - ((e / N) & 1u));
  return (v ^ m) - m;
}


// ------------------------------------------------------------ prep kernel
__device__ __forceinline__ uint16_t mod_switch(uint32_t x, int N) {
  const uint64_t twoN = 2u * static_cast<uint64_t>(N);
  return static_cast<uint16_t>((((static_cast<uint64_t>(x) * twoN) + 0x80000000ull) >> 32) & (twoN - 1));
}

struct GateCoef {
  uint32_t konst;
  int32_t wa, wb;
};

__device__ __forceinline__ GateCoef gate_coef(int gate) {
  switch (gate) {
    case TFHE_NAND: return {kMu, -1, -1};
    case TFHE_AND: return {0u - kMu, 1, 1};
    case TFHE_OR: return {kMu, 1, 1};
    case TFHE_NOR: return {0u - kMu, -1, -1};
    case TFHE_XOR: return {2u * kMu, 2, 2};
    case TFHE_XNOR: return {0u - 2u * kMu, -2, -2};
    case TFHE_ANDNY: return {0u - kMu, -1, 1};
    case TFHE_ANDYN: return {0u - kMu, 1, -1};
    case TFHE_ORNY: return {kMu, -1, 1};
    default: return {kMu, 1, -1};  // TFHE_ORYN
  }
}

__global__ __launch_bounds__(256) void prep_kernel(PrepArgs a, int n, int N, uint16_t* __restrict__ abar) {
  const int64_t idx = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  const int64_t total = a.B * (n + 1);
  if (idx >= total) return;
  const int64_t c = idx / (n + 1);
  const int k = static_cast<int>(idx - c * (n + 1));
  const int64_t row = n + 1;
  uint32_t x;
  if (a.mode == kModePlain) {
    x = a.ca[c * row + k];
  } else {
    const uint32_t* pa;
    const uint32_t* pb;
    int gate = a.gate;
    if (a.mode == kModeRelu) {
      const int64_t g = a.gate_begin + c;
      const int64_t v = g / (a.bits - 1), i = g - v * (a.bits - 1);
      pa = a.ca + (v * a.bits + (a.bits - 1)) * row;  // sign bit
      pb = a.ca + (v * a.bits + i) * row;
      gate = TFHE_ANDNY;
    } else if (a.mode == kModeIRelu) {
      const int64_t g = a.gate_begin + c;
      const int64_t v = g / a.bits;
      pa = a.ca + (v * a.sign_bits + (a.sign_bits - 1)) * row;  // sign bit of u
      pb = a.cb + g * row;                                       // error bit g % bits of value v
      gate = TFHE_ANDNY;
    } else if (a.mode == kModeMux || a.mode == kModeMuxTree) {
      // multiplexer e = c mod M: first half AND(selector, if-true), second
      // half AND(NOT selector, if-false)
      const int64_t M = a.B / 2;
      const bool second = c >= M;
      const int64_t e = second ? c - M : c;
      if (a.mode == kModeMux) {
        pa = a.ca + e * row;
        pb = (second ? a.cc : a.cb) + e * row;
      } else {
        // node j of group (v, o) at this level: children 2j (selector bit 0)
        // and 2j + 1 (selector bit 1) of the level below, selector bit
        // `level` of value v
        const int64_t grp = e / a.group, j = e - grp * a.group;
        const int64_t v = grp / a.out_bits;
        pa = a.ca + (v * a.bits + a.level) * row;
        pb = a.cb + (grp * 2 * a.group + 2 * j + (second ? 0 : 1)) * row;
      }
      gate = second ? TFHE_ANDNY : TFHE_AND;
    } else {
      pa = a.ca + c * row;
      pb = a.cb + c * row;
    }
    const GateCoef gc = gate_coef(gate);
    x = static_cast<uint32_t>(gc.wa) * pa[k] + static_cast<uint32_t>(gc.wb) * pb[k] +
        (k == n ? gc.konst : 0u);
  }
  abar[idx] = mod_switch(x, N);
}

// ext[e] += ext[M + e] + (0, 1/8): the OR of a multiplexer's two halves, of
// which at most one is true (N + 1 words per sample)
__global__ __launch_bounds__(256) void mux_combine_kernel(uint32_t* __restrict__ ext, int N, int64_t M) {
  const int64_t idx = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  const int64_t row = N + 1;
  if (idx >= M * row) return;
  const int k = static_cast<int>(idx % row);
  ext[idx] += ext[M * row + idx] + (k == N ? kMu : 0u);
}

struct LutTable {
  uint32_t s[64];
};

// First level of a multiplexer tree over constant leaves: node (v, o, j)
// chooses between bit o of table[2j] (x[v][0] false) and of table[2j + 1]
// (x[v][0] true), i.e. a constant, x[v][0] or NOT x[v][0]; no bootstrap
__global__ __launch_bounds__(256) void lut_leaf_kernel(const uint32_t* __restrict__ x, int n, int32_t msg_bits,
                                                       LutTable table, int32_t out_bits, int64_t V,
                                                       uint32_t* __restrict__ nodes) {
  const int64_t idx = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  const int64_t row = n + 1;
  const int64_t W = int64_t{1} << (msg_bits - 1);
  if (idx >= V * out_bits * W * row) return;
  const int64_t node = idx / row;
  const int k = static_cast<int>(idx - node * row);
  const int64_t j = node % W, grp = node / W;
  const int o = static_cast<int>(grp % out_bits);
  const int64_t v = grp / out_bits;
  const uint32_t b0 = (table.s[2 * j] >> o) & 1u, b1 = (table.s[2 * j + 1] >> o) & 1u;
  uint32_t w;
  if (b0 == b1) {
    w = k == n ? (b0 ? kMu : 0u - kMu) : 0u;
  } else {
    const uint32_t xs = x[(v * msg_bits) * row + k];
    w = b1 ? xs : 0u - xs;
  }
  nodes[idx] = w;
}

// ------------------------------------------------------ blind rotation
// Ring degree 2^LOGN, key coefficients split into S signed parts.
template <int LOGN, int S, int WPB>
struct BrCfg {
  using Lay = RingLayout<LOGN, S>;
  static constexpr int NR = 1 << LOGN;  // ring degree
  static constexpr int NC = Lay::N;     // complex points, NR / 2
  static constexpr int E = Lay::E, T = Lay::T;
  static constexpr int O = 2 * S;       // transform-domain accumulators: (mask, body) x parts
  static constexpr int SHIFT = S == 2 ? 16 : 11;
  // ciphertexts per block: WPB waves' worth (at least one ciphertext).  A
  // large batch takes 8 waves per block (8 ciphertexts at N = 1024, 4 at
  // N = 2048 with two waves each; one block per CU: its ciphertexts run the
  // same CMux and share its key reads in L1, measured 4 % faster than two
  // blocks of 4 at N = 1024 and 2.6 % faster than three blocks of 1 at
  // N = 2048); a batch too small to give every CU a block of 8 waves takes
  // smaller blocks, which spread it over more CUs (launch_br)
  static constexpr int CPB = WPB * 64 / T > 0 ? WPB * 64 / T : 1;
  static constexpr int THREADS = CPB * T;
  static constexpr int SCR = Lay::SCR;
  // the inverse's stage twiddles (NC - 1) get an LDS copy when a ciphertext
  // takes one wave; at N = 2048 they do not fit beside four ciphertexts and
  // are read from global memory (L1).  The twist (read once per output point
  // and CMux) is always read from global memory.
  static constexpr bool ITW_LDS = CPB > 1 && T <= 64;
  static constexpr int LDS_BYTES = NC * 16 + CPB * SCR * 16 + CPB * 2 * NR * 4 + (ITW_LDS ? (NC - 1) * 16 : 0);
  static_assert(LDS_BYTES <= 160 * 1024, "block exceeds the CU's LDS");
  // compiled for two waves per SIMD (256 VGPRs per wave); blocks of at most
  // 4 waves run with at most one wave per SIMD (launch_br) and are compiled
  // for one (the compiler may then also use accumulation registers: 256
  // gates 8.94 -> 8.31 ms)
  static constexpr int MIN_WAVES = WPB <= 4 ? 1 : 2;
};

// 16-byte load through a buffer resource (base and size uniform, offset per
// lane): no per-lane 64-bit address arithmetic, and an offset past the size
// returns zero instead of faulting
__device__ __forceinline__ double2 load_b128(__amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t soff) {
  typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
  const u32x4 v = __builtin_amdgcn_raw_buffer_load_b128(r, voff, soff, 0);
  double2 d;
  __builtin_memcpy(&d, &v, sizeof d);
  return d;
}

// entry lane + k of a complex table: in LDS or global memory by pointer, or
// through a buffer resource (lane offset in a VGPR, the constant k folded
// into the instruction's offset)
struct PtrTable {
  const double2* p;
  __device__ __forceinline__ double2 operator()(int lane, int k) const { return p[lane + k]; }
};
struct BufTable {
  __amdgpu_buffer_rsrc_t r;
  __device__ __forceinline__ double2 operator()(int lane, int k) const {
    return load_b128(r, static_cast<uint32_t>(lane) * 16u, static_cast<uint32_t>(k) * 16u);
  }
};

template <int LOGN, int S, int WPB>
__global__ __launch_bounds__((BrCfg<LOGN, S, WPB>::THREADS), (BrCfg<LOGN, S, WPB>::MIN_WAVES)) void blind_rotate_kernel(
    const double2* __restrict__ bk, const double2* __restrict__ tw_g, const uint16_t* __restrict__ abar,
    const uint32_t* __restrict__ testvec, uint32_t* __restrict__ extract, int n, int l, int bg_bit,
    int64_t B, const uint32_t* __restrict__ acc_in, uint32_t* __restrict__ acc_out) {
  using C = BrCfg<LOGN, S, WPB>;
  using Lay = typename C::Lay;
  constexpr int NR = C::NR, NC = C::NC, E = C::E, T = C::T, CPB = C::CPB, O = C::O;
  // Blocks of at most 4 waves are launched for batches that give every SIMD
  // at most one wave.  Marking the accumulation registers used takes the
  // wave's allocation past half the register file, so that the hardware
  // places at most one wave per SIMD: without it a wave that fits in 256
  // registers lets the dispatcher put up to six one-wave blocks on some CUs
  // (their LDS allows it) and two waves on one SIMD, while other CUs idle
  // (blind rotation of 1024 gates: 13.1 -> 10.0 ms, 3000 gates: 28.9 -> 25.9 ms)
  if constexpr (C::MIN_WAVES == 1) asm volatile("" ::: "a255");
  __shared__ double2 s_tw[NC];
  __shared__ double2 s_scr[CPB * Lay::SCR];
  __shared__ uint32_t s_acc[CPB * 2 * NR];
  __shared__ double2 s_itw[C::ITW_LDS ? NC - 1 : 1];

  const int slot = threadIdx.x / T;
  const int t = threadIdx.x % T;
  int64_t c = static_cast<int64_t>(blockIdx.x) * CPB + slot;
  const bool active = c < B;
  if (!active) c = B - 1;  // idle slots repeat the last sample and write nothing

  // tw_g: [0, NC) the forward's tree twiddles, [NC, 2NC - 1) the inverse's
  // stage twiddles, [2NC, 3NC) the twist
  for (int k = threadIdx.x; k < NC; k += C::THREADS) s_tw[tw_lds_slot<Lay>(k)] = tw_g[k];
  if constexpr (C::ITW_LDS)
    for (int k = threadIdx.x; k < NC - 1; k += C::THREADS) s_itw[k] = tw_g[NC + k];
  const auto itw = [&] {
    if constexpr (C::ITW_LDS)
      return PtrTable{s_itw};
    else
      return BufTable{__builtin_amdgcn_make_buffer_rsrc(const_cast<double2*>(tw_g + NC), 0, NC * 16, 0x00020000)};
  }();
  const BufTable twist{__builtin_amdgcn_make_buffer_rsrc(const_cast<double2*>(tw_g + 2 * NC), 0, NC * 16, 0x00020000)};
  __syncthreads();
  double2* scr = s_scr + slot * Lay::SCR;
  uint32_t* acc_a = s_acc + slot * 2 * NR;
  uint32_t* acc_b = acc_a + NR;
  const uint16_t* ab = abar + c * (n + 1);

  // ACC = (0, X^{-bbar} v); thread t owns ring coefficients t + T*e and t + T*e + NR/2.
  // A stage check (acc_in given) starts from the caller's accumulator instead.
  if (acc_in != nullptr) {
    const uint32_t* src = acc_in + c * 2 * NR;
#pragma unroll
    for (int e = 0; e < E; e++)
#pragma unroll
      for (int h = 0; h < 2; h++) {
        const int j = t + T * e + h * NC;
        acc_a[j] = src[j];
        acc_b[j] = src[NR + j];
      }
    poly_sync<T>();
  } else {
    const uint32_t bbar = ab[n];
    const uint32_t e0 = (2u * NR - bbar) & (2u * NR - 1);
#pragma unroll
    for (int e = 0; e < E; e++)
#pragma unroll
      for (int h = 0; h < 2; h++) {
        const int j = t + T * e + h * NC;
        acc_a[j] = 0u;
        uint32_t v;
        if (testvec == nullptr) {
          const int src = j - static_cast<int>(e0 & (NR - 1));
          const uint32_t m = static_cast<uint32_t>(src >> 31) ^ (0u - ((e0 / NR) & 1u));
          v = (kMu ^ m) - m;
        } else {
          v = rot_coef<NR>(testvec, e0, j);
        }
        acc_b[j] = v;
      }
    poly_sync<T>();
  }

  // signed gadget decomposition: adding the offset (Bg/2 in every digit
  // position, plus the rounding bit below the last digit) turns each signed
  // digit d into the unsigned field d + Bg/2; flipping the field's top bit
  // (flip) then makes the field's sign extension equal to d
  const uint32_t half = 1u << (bg_bit - 1);
  uint32_t offset = 0, flip = 0;
  for (int j = 1; j <= l; j++) {
    offset += half << (32 - j * bg_bit);
    flip |= half << (32 - j * bg_bit);
  }
  if (l * bg_bit < 32) offset += 1u << (31 - l * bg_bit);
  const size_t bk_step = static_cast<size_t>(2 * l) * O * NC;  // points per CMux
  // key of one CMux: [2l][O][E][T] points; lane t reads point (r, o, e, t)
  const uint32_t voff = static_cast<uint32_t>(t) * 16u;

  // One block barrier per CMux keeps the block's ciphertexts on the same
  // CMux: they then read the same key points close together in time, which
  // the L1 cache serves.  The block's second half of waves takes it later,
  // after pass 1 of the third digit polynomial's forward transform (of the
  // last, with fewer than three digits per polynomial), so that the two
  // waves sharing a SIMD run about two digit transforms apart and one's
  // transposes overlap the other's arithmetic (A/B on one machine: 28.34 ->
  // 27.89 ms per 4096 bootstraps; offsets of one pass, one transform, one
  // and a half transforms gave 0.2 % .. 1.1 %).
  constexpr bool kCmuxBarrier = CPB > 1 && T <= 64;
  const bool late = kCmuxBarrier && slot >= CPB / 2;
  const int late_digit = l > 2 ? 2 : l - 1;  // every wave takes exactly one barrier per CMux
  for (int i = 0; i < n; i++) {
    if constexpr (kCmuxBarrier) {
      if (!late) __syncthreads();
    }
    const uint32_t a_i = ab[i];
    const __amdgpu_buffer_rsrc_t bkr =
        __builtin_amdgcn_make_buffer_rsrc(const_cast<double2*>(bk + static_cast<size_t>(i) * bk_step), 0,
                                          static_cast<int>(bk_step * 16), 0x00020000);
    double2 acc[O][E];
#pragma unroll
    for (int o = 0; o < O; o++)
#pragma unroll
      for (int e = 0; e < E; e++) acc[o][e] = make_double2(0.0, 0.0);

    for (int q = 0; q < 2; q++) {
      const uint32_t* P = q ? acc_b : acc_a;
      // recompute the rotation indices and coefficient positions for each q
      // instead of keeping 4E of them live across the transforms (the empty
      // asm hides the values of a_i and t)
      uint32_t a_q = a_i;
      int t_q = t;
      asm volatile("" : "+v"(a_q), "+v"(t_q));
      // D = X^{a_i} P - P (plus the decomposition offset) at coefficients
      // t + T*e (h = 0) and t + T*e + NR/2 (h = 1): point e's real and imaginary part
      uint32_t D[2][E];
#pragma unroll
      for (int e = 0; e < E; e++)
#pragma unroll
        for (int h = 0; h < 2; h++) {
          const int j = t_q + T * e + h * NC;
          D[h][e] = (rot_coef<NR>(P, a_q, j) - P[j] + offset) ^ flip;
        }
      for (int jj = 0; jj < l; jj++) {
        // digit jj is the signed field of bits [32 - (jj+1) bg_bit, 32 - jj bg_bit)
        // (bg_bit < 32: the transform bound admits no wider digit)
        const uint32_t dpos = static_cast<uint32_t>(32 - (jj + 1) * bg_bit), dw = static_cast<uint32_t>(bg_bit);
        // key row r = q*l + jj; its first output's points are requested
        // before the transform so that their latency overlaps it
        const uint32_t row = static_cast<uint32_t>((q * l + jj) * O * NC) * 16u;
        double2 w[E];
#pragma unroll
        for (int e = 0; e < E; e++) w[e] = load_b128(bkr, voff, row + static_cast<uint32_t>(e * T * 16));
        double2 x[E];
#pragma unroll
        for (int e = 0; e < E; e++)
          x[e] = make_double2(static_cast<double>(signed_field(D[0][e], dpos, dw)),
                              static_cast<double>(signed_field(D[1][e], dpos, dw)));
        const bool barrier_here = late && q == 0 && jj == late_digit;
        fft_forward<Lay, true, false, 1>(x, t, scr, s_tw, tw_g, 1, [&] {
          if (barrier_here) __syncthreads();
        });
#pragma unroll
        for (int o = 0; o < O; o++) {
          if (o > 0) {
#pragma unroll
            for (int e = 0; e < E; e++) w[e] = load_b128(bkr, voff, row + static_cast<uint32_t>((o * E + e) * T * 16));
          }
#pragma unroll
          for (int e = 0; e < E; e++) cmac(acc[o][e], x[e], w[e]);
        }
      }
    }

    // inverse transforms two at a time (O is even)
    static_for<0, O / 2>([&](auto PI) { fft_inverse<Lay, 2 * decltype(PI)::value, 2>(acc, t, scr, itw); });
    // twist, then every output is within 1/8 of an integer (the transform's
    // error bound): round, take it mod 2^32 and recombine the key parts
    int t_r = t;
    asm volatile("" : "+v"(t_r));
#pragma unroll
    for (int e = 0; e < E; e++) {
      const int j = t_r + T * e;
      const double2 tau = twist(t_r, T * e);
      uint32_t ra0 = 0u, ra1 = 0u, rb0 = 0u, rb1 = 0u;
#pragma unroll
      for (int sp = S - 1; sp >= 0; sp--) {
        const double2 va = cmul(acc[sp][e], tau), vb = cmul(acc[S + sp][e], tau);
        ra0 = (ra0 << C::SHIFT) + round_low32(va.x);
        ra1 = (ra1 << C::SHIFT) + round_low32(va.y);
        rb0 = (rb0 << C::SHIFT) + round_low32(vb.x);
        rb1 = (rb1 << C::SHIFT) + round_low32(vb.y);
      }
      acc_a[j] += ra0;
      acc_a[j + NC] += ra1;
      acc_b[j] += rb0;
      acc_b[j + NC] += rb1;
    }
    poly_sync<T>();
  }

  // SampleExtract of coefficient 0: (A_0, -A_{N-1}, ..., -A_1, B_0), or for a
  // stage check (acc_out given) the whole accumulator
  if (active && acc_out != nullptr) {
    uint32_t* dst = acc_out + c * 2 * NR;
    int t_x = t;
    asm volatile("" : "+v"(t_x));
#pragma unroll
    for (int e = 0; e < E; e++)
#pragma unroll
      for (int h = 0; h < 2; h++) {
        const int j = t_x + T * e + h * NC;
        dst[j] = acc_a[j];
        dst[NR + j] = acc_b[j];
      }
  } else if (active) {
    uint32_t* out = extract + c * (NR + 1);
    int t_x = t;  // hidden so that no coefficient position stays live over the CMux loop
    asm volatile("" : "+v"(t_x));
#pragma unroll
    for (int e = 0; e < E; e++)
#pragma unroll
      for (int h = 0; h < 2; h++) {
        const int j = t_x + T * e + h * NC;
        out[j] = j == 0 ? acc_a[0] : 0u - acc_a[NR - j];
      }
    if (t == 0) out[NR] = acc_b[0];
  }
}

// ------------------------------------------ blind rotation, split transforms
// Ring degree 2^LOGN whose transform spans two waves (T = 128 lanes).  The
// forward transform's first stage splits C[X]/(X^n - i) into the halves
// modulo X^{n/2} - tw[1] and X^{n/2} + tw[1]; wave h of a ciphertext computes
// half h of every transform: that stage's output for its half, from input
// points of both halves (read from the accumulator in LDS, which both waves
// see), then the transform of the subtree under tree node 2 + h on its own,
// with wave-local transposes.  The tree positions of half h are
// n/2 * h + j', so the transform-domain layout (and the key) is the one of the
// undivided transform.  The inverse transforms the halves separately; its
// last stage combines them: each wave finishes both halves for half of the
// points, exchanging the other half of its points with its partner through
// LDS two accumulators at a time.  A CMux then takes O/2 + 1 block barriers
// instead of two per transpose.
// SW: waves per SIMD the kernel is compiled for.  Blocks of one ciphertext
// come in two kinds: SW = 1 for batches that give every SIMD at most one
// wave (two blocks per CU), SW = 2 for up to three blocks per CU (their LDS).
template <int LOGN, int S, int WPB, int SW = 2>
struct BrSplitCfg {
  using Lay = RingLayout<LOGN, S>;
  using Sub = Layout<Lay::LOGN - 1, Lay::LOGE>;
  static_assert(Lay::T == 128 && Sub::T == 64, "two waves per ciphertext");
  static constexpr int NR = 1 << LOGN, NC = Lay::N, HN = Sub::N, E = Sub::E;
  static constexpr int O = 2 * S;
  static constexpr int SHIFT = S == 2 ? 16 : 11;
  static constexpr int CPB = WPB / 2;
  static constexpr int THREADS = CPB * 128;
  static constexpr int LDS_BYTES = 2 * HN * 16 + CPB * 2 * Sub::SCR * 16 + CPB * 2 * NR * 4;
  static_assert(CPB >= 1 && LDS_BYTES <= 160 * 1024, "block exceeds the CU's LDS");
  static_assert(SW == 2 || CPB == 1, "one wave per SIMD only for blocks of one ciphertext");
  static constexpr int MIN_WAVES = SW;
};

template <int LOGN, int S, int WPB, int SW>
__global__ __launch_bounds__((BrSplitCfg<LOGN, S, WPB, SW>::THREADS),
                             (BrSplitCfg<LOGN, S, WPB, SW>::MIN_WAVES)) void blind_rotate_split_kernel(
    const double2* __restrict__ bk, const double2* __restrict__ tw_g, const uint16_t* __restrict__ abar,
    const uint32_t* __restrict__ testvec, uint32_t* __restrict__ extract, int n, int l, int bg_bit,
    int64_t B, const uint32_t* __restrict__ acc_in, uint32_t* __restrict__ acc_out) {
  using C = BrSplitCfg<LOGN, S, WPB, SW>;
  using Sub = typename C::Sub;
  constexpr int NR = C::NR, NC = C::NC, HN = C::HN, E = C::E, CPB = C::CPB, O = C::O;
  constexpr int TOP = C::Lay::LOGN - 1;  // the splitting stage
  // one wave per SIMD: the allocation is taken past half the register file
  // so that the hardware places no second wave on the SIMD (as in the
  // one-wave blocks of blind_rotate_kernel): 384 lookups 14.8 -> 12.6 ms
  if constexpr (SW == 1) asm volatile("" ::: "a255");
  __shared__ double2 s_tw[2 * HN];
  __shared__ double2 s_scr[CPB * 2 * Sub::SCR];
  __shared__ uint32_t s_acc[CPB * 2 * NR];

  const int slot = threadIdx.x / 128;
  const int tc = threadIdx.x % 128;  // thread within the ciphertext
  const int h = __builtin_amdgcn_readfirstlane(tc >> 6);  // the half this wave computes
  const int t = tc & 63;
  int64_t c = static_cast<int64_t>(blockIdx.x) * CPB + slot;
  const bool active = c < B;
  if (!active) c = B - 1;  // idle slots repeat the last sample and write nothing

  // subtree tables: node m of the subtree under node 2 + hh is tree node
  // m + (1 + hh) 2^floor(log2 m); each stored in the subtree's LDS order
  for (int k = threadIdx.x; k < 2 * HN; k += C::THREADS) {
    const int hh = k / HN, m = k % HN;
    const int top = m > 0 ? 1 << (31 - __builtin_clz(static_cast<unsigned>(m))) : 0;
    s_tw[hh * HN + tw_lds_slot<Sub>(m)] = tw_g[m + (1 + hh) * top];
  }
  double2* scr = s_scr + (slot * 2 + h) * Sub::SCR;
  double2* partner = s_scr + (slot * 2 + (1 - h)) * Sub::SCR;
  const double2* tw_half = s_tw + h * HN;
  uint32_t* acc_a = s_acc + slot * 2 * NR;
  uint32_t* acc_b = acc_a + NR;
  const uint16_t* ab = abar + c * (n + 1);
  const BufTable itw{__builtin_amdgcn_make_buffer_rsrc(const_cast<double2*>(tw_g + NC), 0, NC * 16, 0x00020000)};
  const BufTable twist{__builtin_amdgcn_make_buffer_rsrc(const_cast<double2*>(tw_g + 2 * NC), 0, NC * 16, 0x00020000)};
  const double2 tw1 = tw_g[1];
  const double2 split_w = h ? make_double2(-tw1.x, -tw1.y) : tw1;

  // ACC = (0, X^{-bbar} v), or for a stage check (acc_in given) the caller's accumulator
  if (acc_in != nullptr) {
    const uint32_t* src = acc_in + c * 2 * NR;
    for (int j = tc; j < NR; j += 128) {
      acc_a[j] = src[j];
      acc_b[j] = src[NR + j];
    }
  } else {
    const uint32_t bbar = ab[n];
    const uint32_t e0 = (2u * NR - bbar) & (2u * NR - 1);
    for (int j = tc; j < NR; j += 128) {
      uint32_t v;
      if (testvec == nullptr) {
        const int src = j - static_cast<int>(e0 & (NR - 1));
        const uint32_t m = static_cast<uint32_t>(src >> 31) ^ (0u - ((e0 / NR) & 1u));
        v = (kMu ^ m) - m;
      } else {
        v = rot_coef<NR>(testvec, e0, j);
      }
      acc_a[j] = 0u;
      acc_b[j] = v;
    }
  }
  __syncthreads();

  const uint32_t half = 1u << (bg_bit - 1);
  uint32_t offset = 0, flip = 0;
  for (int j = 1; j <= l; j++) {
    offset += half << (32 - j * bg_bit);
    flip |= half << (32 - j * bg_bit);
  }
  if (l * bg_bit < 32) offset += 1u << (31 - l * bg_bit);
  const size_t bk_step = static_cast<size_t>(2 * l) * O * NC;
  const uint32_t voff = static_cast<uint32_t>(tc) * 16u;
  const bool packed_second = l == 2 && bg_bit <= 10;

  for (int i = 0; i < n; i++) {
    const uint32_t a_i = ab[i];
    const __amdgpu_buffer_rsrc_t bkr =
        __builtin_amdgcn_make_buffer_rsrc(const_cast<double2*>(bk + static_cast<size_t>(i) * bk_step), 0,
                                          static_cast<int>(bk_step * 16), 0x00020000);
    double2 acc[O][E];
#pragma unroll
    for (int o = 0; o < O; o++)
#pragma unroll
      for (int e = 0; e < E; e++) acc[o][e] = make_double2(0.0, 0.0);

    for (int q = 0; q < 2; q++) {
      const uint32_t* P = q ? acc_b : acc_a;
      // With two digits of at most 10 bits the second digit of each of the
      // lane's 4E coefficients is kept packed (three fields to a register)
      // from the first digit's pass.  For the mask polynomial (q = 0), right
      // after the CMux's closing barrier, each wave forms D = X^{a_i} P - P
      // (plus the decomposition offset) only at its own half's coefficients
      // and writes the words to region h of its own and of its partner's
      // transpose scratch (idle before the transforms): each scratch then
      // holds both halves' words, region hh for half hh, and each wave reads
      // them from its own; both digits are fields of one word, so one
      // exchange serves both digit passes.  The body polynomial's digits are
      // computed by each wave at both halves' coefficients from the
      // accumulator: exchanging them too took one more barrier between the
      // waves' transforms and was 2.7 % slower than this (A/B on one
      // machine, 8192 lookups: 133.6 ms, against 135.9 ms exchanging
      // neither polynomial and 137.3 ms exchanging both).  Other gadgets
      // recompute D from the accumulator for every digit.
      uint32_t pk[(4 * E + 2) / 3];
      const bool xq = packed_second && q == 0;
      if (xq) {
        uint32_t a_q = a_i;
        int t_q = t;
        asm volatile("" : "+v"(a_q), "+v"(t_q));
        __builtin_amdgcn_s_setprio(3);
        uint4* mine = reinterpret_cast<uint4*>(scr) + 64 * (E / 2) * h + t;
        uint4* theirs = reinterpret_cast<uint4*>(partner) + 64 * (E / 2) * h + t;
#pragma unroll
        for (int m = 0; m < E / 2; m++) {
          uint32_t d[4];
#pragma unroll
          for (int k = 0; k < 4; k++) {  // (e, im) = (2m + k / 2, k % 2)
            const int j = t_q + 64 * (2 * m + k / 2) + h * HN + (k % 2) * NC;
            d[k] = (rot_coef<NR>(P, a_q, j) - P[j] + offset) ^ flip;
          }
          const uint4 v = make_uint4(d[0], d[1], d[2], d[3]);
          mine[64 * m] = v;
          theirs[64 * m] = v;
        }
        __builtin_amdgcn_s_setprio(0);
        __syncthreads();
      }
      for (int jj = 0; jj < l; jj++) {
        const uint32_t dpos = static_cast<uint32_t>(32 - (jj + 1) * bg_bit), dw = static_cast<uint32_t>(bg_bit);
        const uint32_t row = static_cast<uint32_t>((q * l + jj) * O * NC) * 16u;
        // The splitting stage: this half's output u + w v (half 0) or
        // u - w v (half 1) of point j' = t + 64 e, u and v the values of
        // half 0 and half 1 there, i.e. coefficients j' + HN hh (real part)
        // and j' + HN hh + NC (imaginary part), hh = 0, 1.
        auto split = [&](const double (&dg)[2][2]) {
          const double2 u = make_double2(dg[0][0], dg[0][1]), v = make_double2(dg[1][0], dg[1][1]);
          return make_double2(fma(split_w.x, v.x, fma(-split_w.y, v.y, u.x)),
                              fma(split_w.x, v.y, fma(split_w.y, v.x, u.y)));
        };
        double2 x[E];
        if (packed_second && jj == 1) {
          // the second digits, kept from the first digit's pass
#pragma unroll
          for (int e = 0; e < E; e++) {
            double dg[2][2];
#pragma unroll
            for (int hh = 0; hh < 2; hh++)
#pragma unroll
              for (int im = 0; im < 2; im++) {
                const int k = (e * 2 + hh) * 2 + im;
                dg[hh][im] = static_cast<double>(signed_field(pk[k / 3], 10u * (k % 3), dw));
              }
            x[e] = split(dg);
          }
        } else if (xq) {
          // the first digits from both halves' words; the second digits'
          // fields packed for the next pass
          const uint32_t dpos2 = dpos - dw;
          const uint4* words = reinterpret_cast<const uint4*>(scr) + t;
#pragma unroll
          for (int m = 0; m < E / 2; m++) {
            const uint4 w0 = words[64 * m], w1 = words[64 * (E / 2 + m)];
            const uint32_t half_words[2][4] = {{w0.x, w0.y, w0.z, w0.w}, {w1.x, w1.y, w1.z, w1.w}};
#pragma unroll
            for (int ee = 0; ee < 2; ee++) {
              const int e = 2 * m + ee;
              double dg[2][2];
#pragma unroll
              for (int hh = 0; hh < 2; hh++)
#pragma unroll
                for (int im = 0; im < 2; im++) {
                  const uint32_t D = half_words[hh][2 * ee + im];
                  dg[hh][im] = static_cast<double>(signed_field(D, dpos, dw));
                  const int k = (e * 2 + hh) * 2 + im;
                  const uint32_t f = __builtin_amdgcn_ubfe(D, dpos2, dw);
                  pk[k / 3] = k % 3 ? pk[k / 3] | (f << (10u * (k % 3))) : f;
                }
              x[e] = split(dg);
            }
          }
        } else {
          // digit jj of D at both halves' coefficients, from the accumulator
          uint32_t a_q = a_i;
          int t_q = t;
          asm volatile("" : "+v"(a_q), "+v"(t_q));
          // raised issue priority while the digits' LDS reads are issued (as
          // in the transposes), where the two waves of a ciphertext wait on
          // each other at the block barriers
          __builtin_amdgcn_s_setprio(3);
#pragma unroll
          for (int e = 0; e < E; e++) {
            double dg[2][2];
#pragma unroll
            for (int hh = 0; hh < 2; hh++)
#pragma unroll
              for (int im = 0; im < 2; im++) {
                const int j = t_q + 64 * e + hh * HN + im * NC;
                const uint32_t D = (rot_coef<NR>(P, a_q, j) - P[j] + offset) ^ flip;
                dg[hh][im] = static_cast<double>(signed_field(D, dpos, dw));
                if (packed_second) {
                  const int k = (e * 2 + hh) * 2 + im;
                  const uint32_t f = __builtin_amdgcn_ubfe(D, dpos - dw, dw);
                  pk[k / 3] = k % 3 ? pk[k / 3] | (f << (10u * (k % 3))) : f;
                }
              }
            x[e] = split(dg);
          }
          __builtin_amdgcn_s_setprio(0);
        }
        // the key row's first output points, requested before the transform
        // so that their latency overlaps it
        double2 w[E];
#pragma unroll
        for (int e = 0; e < E; e++) w[e] = load_b128(bkr, voff, row + static_cast<uint32_t>(e * 128 * 16));
        fft_forward<Sub, true, true>(x, t, scr, tw_half, tw_g, 2 + h);
#pragma unroll
        for (int o = 0; o < O; o++) {
          if (o > 0) {
#pragma unroll
            for (int e = 0; e < E; e++)
              w[e] = load_b128(bkr, voff, row + static_cast<uint32_t>((o * E + e) * 128 * 16));
          }
#pragma unroll
          for (int e = 0; e < E; e++) cmac(acc[o][e], x[e], w[e]);
        }
      }
    }

    // inverse transforms of this half, two at a time
    static_for<0, O / 2>([&](auto PI) { fft_inverse<Sub, 2 * decltype(PI)::value, 2, true>(acc, t, scr, itw); });
    // the inverse's last stage: point j' of half 0 becomes u + t_j' v, of
    // half 1 u - t_j' v (u, v: the halves' values at j', t_j' = e^{-2 pi i j'/n}).
    // Wave h finishes both halves for its slice of the points j' = t + 64 e,
    // e in [h E/2, h E/2 + E/2): it sends the other slice of its half to the
    // partner and receives the partner's values at its own slice.  Two
    // accumulators at a time go through LDS (E points per lane), the first
    // pair through the writer's own scratch, the second through the
    // partner's: a wave overwrites a region only after it has itself read
    // what was last written there, so one barrier per pair suffices.
    int t_x = t;
    asm volatile("" : "+v"(t_x));
    auto finish = [&](auto HI) {
      constexpr int H = decltype(HI)::value, HE = E / 2;
      constexpr int MINE = H * HE, OTHER = (1 - H) * HE;
      double2 tk[HE];  // the stage's twiddles at this slice, the same for every accumulator
#pragma unroll
      for (int e = 0; e < HE; e++) tk[e] = itw(t_x, (1 << TOP) - 1 + 64 * (MINE + e));
      // twist, round (every output is within 1/8 of an integer), recombine
      // the key parts of polynomial q and add to both halves' coefficients
      // at this slice
      auto accumulate = [&](auto QI) {
        constexpr int q = decltype(QI)::value;
        uint32_t* dstp = q ? acc_b : acc_a;
#pragma unroll
        for (int e = 0; e < HE; e++)
#pragma unroll
          for (int hh = 0; hh < 2; hh++) {
            const int slot_e = hh ? OTHER + e : MINE + e;
            const int j = t_x + 64 * (MINE + e) + hh * HN;
            const double2 tau = twist(t_x, 64 * (MINE + e) + hh * HN);
            uint32_t r0 = 0u, r1 = 0u;
#pragma unroll
            for (int sp = S - 1; sp >= 0; sp--) {
              const double2 v = cmul(acc[q * S + sp][slot_e], tau);
              r0 = (r0 << C::SHIFT) + round_low32(v.x);
              r1 = (r1 << C::SHIFT) + round_low32(v.y);
            }
            // an LDS atomic add without return (ds_add_u32): no read round
            // trip before the block barrier that follows (every word has one
            // writer, so this is a plain addition; 133.7 -> 130.9 ms per 8192
            // lookups against read, add, write)
            __hip_atomic_fetch_add(&dstp[j], r0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
            __hip_atomic_fetch_add(&dstp[j + NC], r1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
          }
      };
      static_for<0, O / 2>([&](auto KI) {
        constexpr int k = decltype(KI)::value;
        double2* dst = (k & 1) ? partner : scr;
        const double2* src = (k & 1) ? scr : partner;
        static_for<0, 2>([&](auto PI) {
          constexpr int pi = decltype(PI)::value;
#pragma unroll
          for (int e = 0; e < HE; e++) dst[(pi * HE + e) * 64 + t_x] = acc[2 * k + pi][OTHER + e];
        });
        __syncthreads();
        static_for<0, 2>([&](auto PI) {
          constexpr int pi = decltype(PI)::value, o = 2 * k + pi;
#pragma unroll
          for (int e = 0; e < HE; e++) {
            const double2 pv = src[(pi * HE + e) * 64 + t_x];
            double2 u = H ? pv : acc[o][MINE + e], v = H ? acc[o][MINE + e] : pv;
            ct_butterfly(u, v, tk[e]);
            acc[o][MINE + e] = u;   // half 0's point j'
            acc[o][OTHER + e] = v;  // half 1's point j'
          }
        });
        // with two key parts the first pair is the mask's, the second the body's
        if constexpr (S == 2) accumulate(std::integral_constant<int, k>{});
      });
      if constexpr (S != 2) {
        accumulate(std::integral_constant<int, 0>{});
        accumulate(std::integral_constant<int, 1>{});
      }
    };
    // two copies, one per half; the distinct empty asm statements keep the
    // compiler from merging them into one path that selects between the
    // register slices (which would hold both slices' values at once)
    if (h == 0) {
      asm volatile("; last stage, half 0");
      finish(std::integral_constant<int, 0>{});
      asm volatile("; last stage, half 0 done");
    } else {
      asm volatile("; last stage, half 1");
      finish(std::integral_constant<int, 1>{});
      asm volatile("; last stage, half 1 done");
    }
    __syncthreads();
  }

  // SampleExtract of coefficient 0: (A_0, -A_{N-1}, ..., -A_1, B_0), or for a
  // stage check (acc_out given) the whole accumulator
  if (active && acc_out != nullptr) {
    uint32_t* dst = acc_out + c * 2 * NR;
    for (int j = tc; j < NR; j += 128) {
      dst[j] = acc_a[j];
      dst[NR + j] = acc_b[j];
    }
  } else if (active) {
    uint32_t* out = extract + c * (NR + 1);
    for (int j = tc; j < NR; j += 128) out[j] = j == 0 ? acc_a[0] : 0u - acc_a[NR - j];
    if (tc == 0) out[NR] = acc_b[0];
  }
}

// ------------------------------------------------------- key switching
// Output sample of batch entry c: c itself, or for the activation units the
// gate's place in the [V][bits] output tensor (forward ReLU: bit
// g % (bits-1) of value g / (bits-1); backward iReLU: entry g of [V][bits]).
__device__ __forceinline__ int64_t out_index(int mode, int64_t c, int32_t bits, int64_t gate_begin) {
  const int64_t g = gate_begin + c;
  if (mode == kModeRelu) {
    const int64_t v = g / (bits - 1);
    return v * bits + (g - v * (bits - 1));
  }
  return mode == kModeIRelu ? g : c;
}

// One wave per block covers 64 output columns of KS_CB samples.  Each lane
// keeps the running output word of its column for every sample.  For each
// input coefficient i the block stages the key rows of all t digits and all
// non-zero digit values, plus an all-zero row for digit value 0, in LDS
// ([t][base][64] words); the (wave-uniform) digit of each sample then selects
// its row with one LDS read and one subtraction.  The key rows are read from
// global memory once per block and shared by the KS_CB samples.
constexpr int KS_CB = 32;    // samples per block
constexpr int KS_COLS = 64;  // output columns per block (one wave)
constexpr int KS_ICH = 16;   // input coefficients staged per round
constexpr int KS_MAXROWS = 64;  // t * 2^basebit rows of one coefficient, at most

// Any digit count and base with ks_t * 2^basebit <= MAXROWS (the specialised
// kernel below covers t = 8, base 4).
template <int MAXROWS>
__global__ __launch_bounds__(64) void keyswitch_kernel(const uint32_t* __restrict__ in,
                                                       const uint32_t* __restrict__ ksk,
                                                       uint32_t* __restrict__ out, int n, int N,
                                                       int ks_t, int basebit, int64_t B, int mode,
                                                       int32_t bits, int64_t gate_begin) {
  __shared__ uint32_t s_in[KS_CB][KS_ICH];
  __shared__ uint32_t s_rows[2][MAXROWS][KS_COLS];
  const int lane = threadIdx.x;
  const int64_t c0 = static_cast<int64_t>(blockIdx.x) * KS_CB;
  const int col = blockIdx.y * KS_COLS + lane;
  const bool col_ok = col <= n;
  const int prec = ks_t * basebit;
  const uint32_t round = prec < 32 ? (1u << (31 - prec)) : 0u;
  const int base = 1 << basebit;
  const int vals = base - 1;
  const size_t row = static_cast<size_t>(n) + 1;
  const int nrows = ks_t * base;  // rows staged per coefficient, value 0 included

  uint32_t acc[KS_CB];
#pragma unroll
  for (int k = 0; k < KS_CB; k++) {
    const int64_t c = c0 + k;
    acc[k] = (col == n && c < B) ? in[c * (N + 1) + N] : 0u;
  }

  // rows of coefficient i, (j, v) at j * base + v, fetched into registers
  // one coefficient ahead and written to LDS after the current one is used
  uint32_t pf[MAXROWS];
  auto fetch = [&](int i) {
    const uint32_t* krow_i = ksk + static_cast<size_t>(i) * ks_t * vals * row + col;
#pragma unroll
    for (int r = 0; r < MAXROWS; r++) {
      const int j = r >> basebit, v = r & (base - 1);
      pf[r] = (r < nrows && v != 0 && col_ok) ? krow_i[(static_cast<size_t>(j) * vals + (v - 1)) * row] : 0u;
    }
  };
  auto put = [&](int b) {
#pragma unroll
    for (int r = 0; r < MAXROWS; r++)
      if (r < nrows) s_rows[b][r][lane] = pf[r];
  };

  for (int i0 = 0; i0 < N; i0 += KS_ICH) {
    __syncthreads();
    for (int idx = lane; idx < KS_CB * KS_ICH; idx += KS_COLS) {
      const int k = idx / KS_ICH, ii = idx % KS_ICH;
      const int64_t c = c0 + k;
      s_in[k][ii] = (c < B && i0 + ii < N) ? in[c * (N + 1) + i0 + ii] : 0u;
    }
    const int iend = min(KS_ICH, N - i0);
    fetch(i0);
    put(0);
    __syncthreads();
    for (int ii = 0; ii < iend; ii++) {
      const int b = ii & 1;
      const bool more = ii + 1 < iend;
      if (more) fetch(i0 + ii + 1);
      const uint32_t* rows = &s_rows[b][0][lane];
#pragma unroll 4
      for (int k = 0; k < KS_CB; k++) {
        const uint32_t x = __builtin_amdgcn_readfirstlane(s_in[k][ii]);
        const uint32_t r = prec == 32 ? x : (x + round) >> (32 - prec);
        for (int j = 0; j < ks_t; j++) {
          const uint32_t v = (r >> ((ks_t - 1 - j) * basebit)) & static_cast<uint32_t>(vals);
          acc[k] -= rows[(j * base + v) * KS_COLS];
        }
      }
      if (more) put(b ^ 1);
      __syncthreads();
    }
  }

  if (!col_ok) return;
#pragma unroll
  for (int k = 0; k < KS_CB; k++) {
    const int64_t c = c0 + k;
    if (c >= B) break;
    out[out_index(mode, c, bits, gate_begin) * row + col] = acc[k];
  }
}

// Key switching for t = 8 digits of 2 bits on the matrix cores.  With
// V[c][k] the indicator that digit j of sample c's rounded coefficient a_i
// has value v, for the 24 slots k = (i, j, v) of each input coefficient
// (8 digits x the values 1..3: value 0 selects no key row), key switching
// is the matrix product
//   out[c] = (0, b_c) - sum_k V[c][k] KSK[k]
// with a 0/1 left factor.  The key is held as four signed byte planes
// (ksk_to_mfma_host), so that each plane's product is an exact int8 x int8
// product accumulated in int32 (at most 8 N non-zero terms of magnitude at
// most 128 per output, far below 2^31), and the four products recombine
// exactly mod 2^32.  The 96 slots of four consecutive coefficients
// 4G + q make three v_mfma_i32_32x32x32_i8 (key tiles T = 3G + m): lane l
// of a wave (sample l % 32 of 32, column l % 32 of a 32-column block) holds
// 16 slots, those of coefficient q = h (m = 0) or h + 2 (m = 1) for values
// 1 and 2, and those of value 3 of both (m = 2), h = l / 32.  The
// indicator bytes come from the digits spread one per byte (digits 7..4 of
// the rounded coefficient in the bytes of the low word, 3..0 in the high)
// and one byte permutation per word and value.
// A block of KSM_WAVES waves covers KSM_SAMPLES samples and 32 KSM_NB
// columns over the input coefficients [i_begin, i_end); a wave covers 64 of
// the samples (two MFMA row groups sharing each key fragment) and one
// column block.  Each key tile (KSM_NB column blocks x 4 planes x 64 lanes
// x 16 bytes) is staged through LDS once per block (double-buffered, one
// barrier per tile, the fragments read one tile ahead of their products and
// the tile fetched five ahead), and the inputs are staged through LDS
// KSM_CH coefficients at a time.  The coefficient range is split over
// several blocks when that fills the GPU better: every block adds its exact
// partial sum mod 2^32 to an output that keyswitch_init_kernel set to
// (0, b), so the result does not depend on the order of the additions.
constexpr int KSM_WAVES = 4;                      // waves per block
constexpr int KSM_NB = 2;                         // 32-column blocks per block (ksk_mfma_nb pads to it)
constexpr int KSM_THREADS = 64 * KSM_WAVES;
constexpr int KSM_SG = 2;                         // 32-sample groups per wave
constexpr int KSM_SAMPLES = 128;                  // samples per block
constexpr int KSM_TILE = KSM_NB * 4 * 64;         // 16-byte units of one key tile
constexpr int KSM_UPT = KSM_TILE / KSM_THREADS;   // units each thread stages
constexpr int KSM_CH = 8;                         // input coefficients staged per round
constexpr int KSM_STEPS = KSM_CH / 4 * 3;         // key tiles per round
constexpr int KSM_RING = 3;                       // key tiles in flight in registers
static_assert(KSM_WAVES == KSM_NB * KSM_SAMPLES / (32 * KSM_SG), "waves tile the block's samples x columns");
static_assert(KSM_TILE % KSM_THREADS == 0, "whole units per thread");
static_assert(KSM_STEPS % KSM_RING == 0 && KSM_STEPS % 2 == 0, "ring and LDS buffer indices repeat every round");

typedef int32_t i32x4 __attribute__((ext_vector_type(4)));
typedef int32_t i32x16 __attribute__((ext_vector_type(16)));

struct KsmGrid {
  int nb_total;      // 32-column blocks of the key layout
  int col_tiles;     // nb_total / KSM_NB
  int sample_tiles;  // ceil(B / KSM_SAMPLES)
  int coef_len;      // input coefficients per block, a multiple of KSM_CH
};

// the 2-bit fields of the byte b, one per byte: field f of b in byte f
__device__ __forceinline__ uint32_t spread_digits(uint32_t b) {
  return (b | (b << 6) | (b << 12) | (b << 18)) & 0x03030303u;
}

// byte f of the result is 1 where byte f of the spread digits d equals v
// (v_perm_b32 picks byte d_f of the table, whose byte v is 1)
template <int V>
__device__ __forceinline__ int32_t digit_indicator(uint32_t d) {
  return static_cast<int32_t>(__builtin_amdgcn_perm(0u, 1u << (8 * V), d));
}

__global__ __launch_bounds__(KSM_THREADS, 2) void keyswitch_mfma_kernel(const uint32_t* __restrict__ in,
                                                                     const i32x4* __restrict__ kmf,
                                                                     uint32_t* __restrict__ out, int n, int N,
                                                                     int64_t B, int mode, int32_t bits,
                                                                     int64_t gate_begin, KsmGrid g) {
  __shared__ i32x4 s_b[2][KSM_TILE];
  __shared__ i32x4 s_x[2][KSM_SAMPLES * 3];  // [buffer][sample][12 words, 8 used]
  // Workgroups are handed to the 8 XCDs in turn (workgroup b to XCD b mod 8),
  // and each XCD has its own L2.  The logical tile index L runs over the
  // workgroups of one XCD before the next (a bijection on [0, G) for any G),
  // so that the sample tiles of one key tile, and the key tiles of one
  // coefficient range, share an L2: the key and the inputs are then fetched
  // from HBM about once per launch instead of once per XCD.
  const unsigned G = gridDim.x, xcd = blockIdx.x % 8u, q8 = G / 8u, r8 = G % 8u;
  const unsigned L = xcd * q8 + min(xcd, r8) + blockIdx.x / 8u;
  const int st = static_cast<int>(L % g.sample_tiles);
  const int ct = static_cast<int>((L / g.sample_tiles) % g.col_tiles);
  const int kr = static_cast<int>(L / (static_cast<unsigned>(g.sample_tiles) * g.col_tiles));
  const int i_begin = kr * g.coef_len;
  const int i_end = min(N, i_begin + g.coef_len);
  const int tid = threadIdx.x, w = tid / 64, l = tid % 64;
  const bool hi = l >= 32;  // this lane's coefficients of each four: 1 and 3 (else 0 and 2)
  // wave w: samples [64 (w % 2), +64) of the block's tile as two groups of
  // 32, column block w / 2 of the tile's KSM_NB
  const int ws = w % 2, wc = w / 2;
  // inputs: thread tid loads words 4 (tid % 2) .. +3 of the round's KSM_CH
  // from row tid / 2 of the block's samples
  static_assert(KSM_CH == 8 && KSM_THREADS == 2 * KSM_SAMPLES, "one 16-byte load per thread per round");
  const int xs = tid / 2, xh = tid % 2;
  const uint32_t* x_row;
  {
    const int64_t c = static_cast<int64_t>(st) * KSM_SAMPLES + xs;
    x_row = in + (c < B ? c : B - 1) * (N + 1) + 4 * xh;
  }
  const int nb0 = ct * KSM_NB;

  // key tile units: thread tid stages unit tid + KSM_THREADS u (column block
  // nb0 + u, plane and lane tid / 64, tid % 64)
  const int t_begin = i_begin / 4 * 3, t_last = N / 4 * 3 - 1;
  i32x4 breg[KSM_RING][KSM_UPT];
  auto fetch = [&](int t, i32x4 (&dst)[KSM_UPT]) {
#pragma unroll
    for (int u = 0; u < KSM_UPT; u++)
      dst[u] = kmf[(static_cast<int64_t>(min(t, t_last)) * g.nb_total + nb0) * 256 + KSM_THREADS * u + tid];
  };
  // the first two tiles go to LDS now; breg[s % KSM_RING] holds the tile of
  // offset s + 2 from t_begin at step s
#pragma unroll
  for (int d = 0; d < 2; d++) {
    fetch(t_begin + d, breg[d]);
#pragma unroll
    for (int u = 0; u < KSM_UPT; u++) s_b[d][KSM_THREADS * u + tid] = breg[d][u];
  }
#pragma unroll
  for (int d = 0; d < KSM_RING; d++) fetch(t_begin + 2 + d, breg[d]);
  // (coef_len and N are multiples of KSM_CH, so a round ends before word N)
  i32x4 xv;
  __builtin_memcpy(&xv, x_row + i_begin, 16);
  s_x[0][3 * xs + xh] = xv;
  uint32_t xc[KSM_SG][KSM_CH];
  uint32_t sp[KSM_SG][4];  // spread digits: low and high word of this lane's two coefficients
  int xb = 0;
  // this wave's key fragments (4 planes of its column block): fr[s & 1] holds
  // tile s's, read from LDS one step before its products
  i32x4 fr[2][4];
  __syncthreads();
#pragma unroll
  for (int pl = 0; pl < 4; pl++) fr[0][pl] = s_b[0][(wc * 4 + pl) * 64 + l];

  i32x16 acc[KSM_SG][4];
#pragma unroll
  for (int gi = 0; gi < KSM_SG; gi++)
#pragma unroll
    for (int pl = 0; pl < 4; pl++)
#pragma unroll
      for (int r = 0; r < 16; r++) acc[gi][pl][r] = 0;

#pragma unroll 1
  for (int i0 = i_begin; i0 < i_end; i0 += KSM_CH) {
    const bool more = i0 + KSM_CH < i_end;
    const int t0 = i0 / 4 * 3;
    if (more) __builtin_memcpy(&xv, x_row + i0 + KSM_CH, 16);
    static_for<0, KSM_STEPS>([&](auto SI) {
      constexpr int s = decltype(SI)::value;
      constexpr int b = s & 1;  // (t - t_begin) & 1: rounds start at even offsets
      constexpr int grp = s / 3, m = s % 3;
      const int t = t0 + s;
      // Step of tile t: after the barrier, read the fragments of tile t + 1
      // (it went to LDS one step ago), then stage tile t + 2 in the buffer
      // that held t's (read one step ago, before this barrier) and fetch
      // tile t + 5; the products of t use the fragments read one step ago.
      if constexpr (s == KSM_STEPS - 1)
        if (more) s_x[xb ^ 1][3 * xs + xh] = xv;
      __syncthreads();
#pragma unroll
      for (int pl = 0; pl < 4; pl++) fr[b ^ 1][pl] = s_b[b ^ 1][(wc * 4 + pl) * 64 + l];
#pragma unroll
      for (int u = 0; u < KSM_UPT; u++) s_b[b][KSM_THREADS * u + tid] = breg[s % KSM_RING][u];
      fetch(t + 2 + KSM_RING, breg[s % KSM_RING]);
      if constexpr (s == 0) {
#pragma unroll
        for (int gi = 0; gi < KSM_SG; gi++) {
          const int sl = 32 * (KSM_SG * ws + gi) + (l % 32);
#pragma unroll
          for (int q = 0; q < 2; q++) {
            const i32x4 v = s_x[xb][3 * sl + q];
#pragma unroll
            for (int e = 0; e < 4; e++) xc[gi][4 * q + e] = static_cast<uint32_t>(v[e]);
          }
        }
      }
      if constexpr (m == 0) {
        // this lane's coefficients 4 grp + (0 or 1) and 4 grp + (2 or 3),
        // rounded to 16 bits (ties up), their digits spread one per byte
#pragma unroll
        for (int gi = 0; gi < KSM_SG; gi++)
#pragma unroll
          for (int q = 0; q < 2; q++) {
            const uint32_t x = hi ? xc[gi][4 * grp + 2 * q + 1] : xc[gi][4 * grp + 2 * q];
            const uint32_t r = (x + 0x8000u) >> 16;
            sp[gi][2 * q] = spread_digits(r & 0xffu);
            sp[gi][2 * q + 1] = spread_digits(r >> 8);
          }
      }
      i32x4 a[KSM_SG];
#pragma unroll
      for (int gi = 0; gi < KSM_SG; gi++) {
        if constexpr (m < 2) {
          a[gi][0] = digit_indicator<1>(sp[gi][2 * m]);
          a[gi][1] = digit_indicator<1>(sp[gi][2 * m + 1]);
          a[gi][2] = digit_indicator<2>(sp[gi][2 * m]);
          a[gi][3] = digit_indicator<2>(sp[gi][2 * m + 1]);
        } else {
#pragma unroll
          for (int e = 0; e < 4; e++) a[gi][e] = digit_indicator<3>(sp[gi][e]);
        }
      }
#pragma unroll
      for (int pl = 0; pl < 4; pl++)
#pragma unroll
        for (int gi = 0; gi < KSM_SG; gi++)
          acc[gi][pl] = __builtin_amdgcn_mfma_i32_32x32x32_i8(a[gi], fr[b][pl], acc[gi][pl], 0, 0, 0);
    });
    xb ^= 1;
  }

  // output register r of lane l: sample 8 (r / 4) + 4 (l / 32) + r % 4 of
  // the group, column l % 32 of the wave's column block
  const int row = n + 1;
  const int col = (nb0 + wc) * 32 + (l % 32);
  if (col > n) return;
  static_for<0, 16>([&](auto RI) {
    constexpr int r = decltype(RI)::value;
    // one output row at a time (keeps the accumulators' copies out of VGPRs)
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int gi = 0; gi < KSM_SG; gi++) {
      const int64_t cs = static_cast<int64_t>(st) * KSM_SAMPLES + 32 * (KSM_SG * ws + gi) + 8 * (r / 4) +
                         4 * (l / 32) + (r % 4);
      if (cs >= B) continue;
      uint32_t sum = 0u;
#pragma unroll
      for (int pl = 0; pl < 4; pl++) sum += static_cast<uint32_t>(acc[gi][pl][r]) << (8 * pl);
      atomicAdd(out + out_index(mode, cs, bits, gate_begin) * row + col, 0u - sum);
    }
  });
}

// out = (0^n, b) for every sample: the starting value of the key switching
// on the matrix cores, whose blocks add their partial sums to it
__global__ __launch_bounds__(256) void keyswitch_init_kernel(const uint32_t* __restrict__ in, uint32_t* __restrict__ out,
                                                             int n, int N, int64_t B, int mode, int32_t bits,
                                                             int64_t gate_begin) {
  const int64_t idx = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (idx >= B * (n + 1)) return;
  const int64_t c = idx / (n + 1);
  const int k = static_cast<int>(idx - c * (n + 1));
  out[out_index(mode, c, bits, gate_begin) * (n + 1) + k] = k == n ? in[c * (N + 1) + N] : 0u;
}

__global__ __launch_bounds__(256) void relu_sign_kernel(uint32_t* __restrict__ y, int n, int32_t bits,
                                                        int64_t v_begin, int64_t count) {
  const int64_t idx = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (idx >= count * (n + 1)) return;
  const int64_t v = v_begin + idx / (n + 1);
  const int k = static_cast<int>(idx % (n + 1));
  y[(v * bits + bits - 1) * (n + 1) + k] = k == n ? 0u - kMu : 0u;
}

// modulus-switched inputs of a one-CMux stage check: row c is (abar[c] mod 2N, 0)
__global__ __launch_bounds__(256) void cmux_abar_kernel(const uint32_t* __restrict__ a, int N, int64_t B,
                                                        uint16_t* __restrict__ abar) {
  const int64_t c = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (c >= B) return;
  abar[2 * c] = static_cast<uint16_t>(a[c] & static_cast<uint32_t>(2 * N - 1));
  abar[2 * c + 1] = 0;
}

__global__ __launch_bounds__(256) void not_kernel(const uint32_t* __restrict__ in,
                                                  uint32_t* __restrict__ out, int64_t words) {
  const int64_t idx = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (idx < words) out[idx] = 0u - in[idx];
}

// ------------------------------------- TFHE side of the cryptosystem switch
// Functional key switching with the packing morphism (Section 3.2, step 2):
// Z LWE samples of dimension n become one TRLWE sample (A, B) whose phase is
// sum_z phase_z X^z.  out = (0, sum_z b_z X^z) - sum_{z,i,j} X^z PKS[i][j][v]
// over the non-zero digits v of the rounded a_{z,i}.  pack_init writes the
// first term; pack_ks_kernel adds the rest, one block per (TRLWE, chunk of
// PKS_IC input coefficients), each thread owning 2N/256 output words, and
// adds its partial sums to out with 32-bit atomic adds (exact mod 2^32, so
// the result does not depend on their order).
constexpr int PKS_IC = 8;       // input coefficients per block
constexpr int PKS_ZMAX = 2048;  // Z <= N <= 2048

__global__ __launch_bounds__(256) void pack_init_kernel(const uint32_t* __restrict__ lwe, int n, int N, int Z,
                                                        int64_t B, uint32_t* __restrict__ out) {
  const int64_t idx = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (idx >= B * 2 * N) return;
  const int64_t b = idx / (2 * N);
  const int k = static_cast<int>(idx - b * 2 * N);
  uint32_t w = 0u;
  if (k >= N && k - N < Z) w = lwe[(b * Z + (k - N)) * (n + 1) + n];
  out[idx] = w;
}

template <int N>
__global__ __launch_bounds__(256) void pack_ks_kernel(const uint32_t* __restrict__ lwe,
                                                      const uint32_t* __restrict__ pks, int n, int Z, int t,
                                                      int basebit, uint32_t* __restrict__ out) {
  constexpr int W = 2 * N / 256;  // output words per thread: k = threadIdx.x + 256 * w
  __shared__ uint16_t s_r[PKS_IC][PKS_ZMAX];  // rounded a_{z,i} (t * basebit <= 16 bits)
  __shared__ uint32_t s_key[3][2 * N];        // entries (i, j, v = 1..3) of the packing key
  const int64_t b = blockIdx.x;
  const int i0 = blockIdx.y * PKS_IC;
  const int ic = min(PKS_IC, n - i0);
  const int prec = t * basebit, vals = (1 << basebit) - 1;
  const uint32_t round = prec < 32 ? (1u << (31 - prec)) : 0u;
  for (int idx = threadIdx.x; idx < ic * Z; idx += 256) {
    const int ii = idx / Z, z = idx - ii * Z;
    const uint32_t a = lwe[(b * Z + z) * (n + 1) + i0 + ii];
    s_r[ii][z] = static_cast<uint16_t>((a + round) >> (32 - prec));
  }
  uint32_t acc[W];
#pragma unroll
  for (int w = 0; w < W; w++) acc[w] = 0u;
  for (int ii = 0; ii < ic; ii++) {
    for (int j = 0; j < t; j++) {
      __syncthreads();  // s_r written / the previous entries no longer read
      const uint32_t* e = pks + (static_cast<size_t>(i0 + ii) * t + j) * vals * 2 * N;
      for (int idx = threadIdx.x; idx < vals * 2 * N; idx += 256) s_key[idx / (2 * N)][idx % (2 * N)] = e[idx];
      __syncthreads();
      const int sh = (t - 1 - j) * basebit;
      for (int z = 0; z < Z; z++) {
        const uint32_t v = (static_cast<uint32_t>(s_r[ii][z]) >> sh) & static_cast<uint32_t>(vals);
        if (v == 0) continue;  // uniform across the block
        const uint32_t* key = s_key[v - 1];
#pragma unroll
        for (int w = 0; w < W; w++) {
          const int k = threadIdx.x + 256 * w;  // word k of (A, B): polynomial k / N, coefficient k % N
          const int c = k & (N - 1), base = k - c;
          const int src = c - z;  // X^z moves coefficient src to c, negated when it wrapped
          const uint32_t x = key[base + (src & (N - 1))];
          acc[w] -= src < 0 ? 0u - x : x;
        }
      }
    }
  }
#pragma unroll
  for (int w = 0; w < W; w++) atomicAdd(out + b * 2 * N + threadIdx.x + 256 * w, acc[w]);
}

// The same on the transform (N <= 1024): sum_{z,i,j} X^z PKS[i][j][v_{z,i,j}]
// = sum_{i,j,v} M_{i,j,v} PKS[i][j][v], M_{i,j,v} = sum of X^z over the
// samples z whose digit j of the rounded a_{z,i} is v: one negacyclic
// product of a 0/1 polynomial by each key entry, computed as in the external
// product (the entry in the transform domain in two 16-bit parts, the
// products summed there, one inverse transform and one rounding per block,
// exact because the sum's worst-case error stays below 1/8 for up to
// pks_ic_max input coefficients).  A block takes IC input coefficients of
// CPB TRLWE outputs, one per T lanes; its waves read the same key entries
// close together in time, which L1 then serves; each adds its exact partial
// sum to out with 32-bit atomics after pack_init_kernel.  Workgroups are
// remapped so that the blocks of one coefficient range run on one XCD (its
// L2 then holds the range's key entries for all of them).
template <int LOGN, int WPB>
__global__ __launch_bounds__((BrCfg<LOGN, 2, WPB>::THREADS), (BrCfg<LOGN, 2, WPB>::MIN_WAVES)) void pack_ks_fft_kernel(
    const double2* __restrict__ pkf, const double2* __restrict__ tw_g, const uint32_t* __restrict__ lwe, int n,
    int Z, int t_digits, int basebit, int IC, int groups, int64_t B, uint32_t* __restrict__ out) {
  using C = BrCfg<LOGN, 2, WPB>;
  using Lay = typename C::Lay;
  constexpr int NR = C::NR, NC = C::NC, E = C::E, T = C::T, CPB = C::CPB, O = C::O;
  if constexpr (C::MIN_WAVES == 1) asm volatile("" ::: "a255");
  __shared__ double2 s_tw[NC];
  __shared__ double2 s_scr[CPB * Lay::SCR];
  __shared__ double2 s_itw[C::ITW_LDS ? NC - 1 : 1];

  const unsigned G = gridDim.x, xcd = blockIdx.x % 8u, q8 = G / 8u, r8 = G % 8u;
  const unsigned L = xcd * q8 + min(xcd, r8) + blockIdx.x / 8u;
  const int grp = static_cast<int>(L % static_cast<unsigned>(groups));
  const int i0 = static_cast<int>(L / static_cast<unsigned>(groups)) * IC;
  const int i1 = min(n, i0 + IC);
  const int slot = threadIdx.x / T;
  const int t = threadIdx.x % T;
  int64_t b = static_cast<int64_t>(grp) * CPB + slot;
  const bool active = b < B;
  if (!active) b = B - 1;  // idle slots repeat the last output and write nothing

  for (int k = threadIdx.x; k < NC; k += C::THREADS) s_tw[tw_lds_slot<Lay>(k)] = tw_g[k];
  if constexpr (C::ITW_LDS)
    for (int k = threadIdx.x; k < NC - 1; k += C::THREADS) s_itw[k] = tw_g[NC + k];
  const auto itw = [&] {
    if constexpr (C::ITW_LDS)
      return PtrTable{s_itw};
    else
      return BufTable{__builtin_amdgcn_make_buffer_rsrc(const_cast<double2*>(tw_g + NC), 0, NC * 16, 0x00020000)};
  }();
  const BufTable twist{__builtin_amdgcn_make_buffer_rsrc(const_cast<double2*>(tw_g + 2 * NC), 0, NC * 16, 0x00020000)};
  __syncthreads();
  double2* scr = s_scr + slot * Lay::SCR;

  const int vals = (1 << basebit) - 1, R = t_digits * vals, prec = t_digits * basebit;
  const uint32_t round = 1u << (31 - prec);  // prec <= 16
  // this output's Z input samples through a buffer resource: an offset past
  // the last sample (z >= Z) reads 0, which rounds to 0 and matches no digit v >= 1
  const __amdgpu_buffer_rsrc_t lr = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint32_t*>(lwe + b * Z * (n + 1)), 0, Z * (n + 1) * 4, 0x00020000);
  const size_t key_step = static_cast<size_t>(R) * O * NC;  // points per input coefficient
  const uint32_t voff = static_cast<uint32_t>(t) * 16u;
  double2 acc[O][E];
#pragma unroll
  for (int o = 0; o < O; o++)
#pragma unroll
    for (int e = 0; e < E; e++) acc[o][e] = make_double2(0.0, 0.0);

  for (int i = i0; i < i1; i++) {
    const __amdgpu_buffer_rsrc_t kr = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<double2*>(pkf + static_cast<size_t>(i) * key_step), 0, static_cast<int>(key_step * 16), 0x00020000);
    // rounded a_{z,i} at this lane's coefficients z = t + T e (real part of
    // point e) and z + N/2 (imaginary part); the lane's offset is recomputed
    // here (the empty asm hides t) rather than kept live across the loop
    int t_q = t;
    asm volatile("" : "+v"(t_q));
    const uint32_t lane_off = static_cast<uint32_t>((t_q * (n + 1) + i) * 4);
    uint32_t r[2][E];
#pragma unroll
    for (int e = 0; e < E; e++)
#pragma unroll
      for (int h = 0; h < 2; h++) {
        const uint32_t z_off = static_cast<uint32_t>((T * e + h * NC) * (n + 1) * 4);
        const uint32_t a = static_cast<uint32_t>(__builtin_amdgcn_raw_buffer_load_b32(lr, lane_off, z_off, 0));
        r[h][e] = (a + round) >> (32 - prec);
      }
    for (int j = 0; j < t_digits; j++) {
      const uint32_t sh = static_cast<uint32_t>((t_digits - 1 - j) * basebit);
      for (int v = 1; v <= vals; v++) {
        const uint32_t row = static_cast<uint32_t>((j * vals + v - 1) * O * NC) * 16u;
        // one-wave blocks (the whole register file) request the first
        // output's key points before the transform; two waves per SIMD have
        // no registers for them there
        double2 w[E];
        if constexpr (C::MIN_WAVES == 1) {
#pragma unroll
          for (int e = 0; e < E; e++) w[e] = load_b128(kr, voff, row + static_cast<uint32_t>(e * T * 16));
        }
        double2 x[E];
#pragma unroll
        for (int e = 0; e < E; e++)
          x[e] = make_double2(((r[0][e] >> sh) & static_cast<uint32_t>(vals)) == static_cast<uint32_t>(v) ? 1.0 : 0.0,
                              ((r[1][e] >> sh) & static_cast<uint32_t>(vals)) == static_cast<uint32_t>(v) ? 1.0 : 0.0);
        fft_forward<Lay, true>(x, t, scr, s_tw, tw_g, 1);
#pragma unroll
        for (int o = 0; o < O; o++) {
          if (o > 0 || C::MIN_WAVES != 1) {
#pragma unroll
            for (int e = 0; e < E; e++) w[e] = load_b128(kr, voff, row + static_cast<uint32_t>((o * E + e) * T * 16));
          }
#pragma unroll
          for (int e = 0; e < E; e++) cmac(acc[o][e], x[e], w[e]);
        }
      }
    }
  }

  static_for<0, O / 2>([&](auto PI) { fft_inverse<Lay, 2 * decltype(PI)::value, 2>(acc, t, scr, itw); });
  if (!active) return;
  uint32_t* dst = out + b * 2 * NR;
  int t_r = t;
  asm volatile("" : "+v"(t_r));
#pragma unroll
  for (int e = 0; e < E; e++) {
    const int j = t_r + T * e;
    const double2 tau = twist(t_r, T * e);
    uint32_t ra0 = 0u, ra1 = 0u, rb0 = 0u, rb1 = 0u;
#pragma unroll
    for (int sp = 1; sp >= 0; sp--) {
      const double2 va = cmul(acc[sp][e], tau), vb = cmul(acc[2 + sp][e], tau);
      ra0 = (ra0 << 16) + round_low32(va.x);
      ra1 = (ra1 << 16) + round_low32(va.y);
      rb0 = (rb0 << 16) + round_low32(vb.x);
      rb1 = (rb1 << 16) + round_low32(vb.y);
    }
    atomicAdd(dst + j, 0u - ra0);
    atomicAdd(dst + j + NC, 0u - ra1);
    atomicAdd(dst + NR + j, 0u - rb0);
    atomicAdd(dst + NR + j + NC, 0u - rb1);
  }
}

// SampleExtract of coefficients 0 .. K-1 (Section 3.2, step 3): out[b][i] =
// (a'_0 .. a'_{N-1}, B_i), a'_j = A_{i-j} (j <= i) or -A_{N+i-j} (j > i)
__global__ __launch_bounds__(256) void sample_extract_kernel(const uint32_t* __restrict__ trlwe, int N, int64_t B,
                                                             int K, uint32_t* __restrict__ out) {
  const int64_t idx = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  const int64_t row = N + 1;
  if (idx >= B * K * row) return;
  const int64_t s = idx / row;
  const int j = static_cast<int>(idx - s * row);
  const int64_t b = s / K;
  const int i = static_cast<int>(s - b * K);
  const uint32_t* A = trlwe + b * 2 * N;
  uint32_t w;
  if (j == N) w = A[N + i];
  else w = j <= i ? A[i - j] : 0u - A[N + i - j];
  out[idx] = w;
}

// Standalone negacyclic product c = d * b in Z_{2^32}[X]/(X^N+1) with the blind
// rotation's transform code: d small signed digits, b split into S parts on
// the device and transformed there.  One polynomial per T threads.
template <int LOGN, int S>
__global__ __launch_bounds__(256) void negacyclic_mul_kernel(const double2* __restrict__ tw,
                                                             const int32_t* __restrict__ d,
                                                             const uint32_t* __restrict__ b,
                                                             uint32_t* __restrict__ c, int64_t B) {
  using Lay = RingLayout<LOGN, S>;
  constexpr int NR = 1 << LOGN, NC = Lay::N, E = Lay::E, T = Lay::T, CPB = 256 / T;
  constexpr int SHIFT = S == 2 ? 16 : 11;
  __shared__ double2 s_scr[CPB * Lay::SCR];
  const int slot = threadIdx.x / T;
  const int t = threadIdx.x % T;
  int64_t k = static_cast<int64_t>(blockIdx.x) * CPB + slot;
  const bool active = k < B;
  if (!active) k = B - 1;
  double2* scr = s_scr + slot * Lay::SCR;
  double2 xd[E], xb[S][E];
#pragma unroll
  for (int e = 0; e < E; e++) {
    const int j = t + T * e;
    xd[e] = make_double2(static_cast<double>(d[k * NR + j]), static_cast<double>(d[k * NR + j + NC]));
    int64_t rest0 = static_cast<int32_t>(b[k * NR + j]);
    int64_t rest1 = static_cast<int32_t>(b[k * NR + j + NC]);
#pragma unroll
    for (int sp = 0; sp < S; sp++) {
      int64_t p0 = rest0, p1 = rest1;
      if (sp + 1 < S) {
        const int64_t hb = int64_t{1} << (SHIFT - 1), mask = (int64_t{1} << SHIFT) - 1;
        p0 = ((rest0 + hb) & mask) - hb;
        p1 = ((rest1 + hb) & mask) - hb;
        rest0 = (rest0 - p0) >> SHIFT;
        rest1 = (rest1 - p1) >> SHIFT;
      }
      xb[sp][e] = make_double2(static_cast<double>(p0), static_cast<double>(p1));
    }
  }
  fft_forward<Lay, false>(xd, t, scr, tw, tw);
  static_for<0, S>([&](auto SP) {
    constexpr int sp = decltype(SP)::value;
    fft_forward<Lay, false>(xb[sp], t, scr, tw, tw);
#pragma unroll
    for (int e = 0; e < E; e++) {
      const double2 pr = cmul(xd[e], xb[sp][e]);
      xb[sp][e] = make_double2(pr.x / NC, pr.y / NC);  // exact: NC is a power of two
    }
    fft_inverse<Lay, sp, 1>(xb, t, scr, PtrTable{tw + NC});
  });
  if (!active) return;
#pragma unroll
  for (int e = 0; e < E; e++) {
    const int j = t + T * e;
    const double2 tau = tw[2 * NC + j];
    uint32_t r0 = 0u, r1 = 0u;
#pragma unroll
    for (int sp = S - 1; sp >= 0; sp--) {
      const double2 v = cmul(xb[sp][e], tau);
      r0 = (r0 << SHIFT) + round_low32(v.x);
      r1 = (r1 << SHIFT) + round_low32(v.y);
    }
    c[k * NR + j] = r0;
    c[k * NR + j + NC] = r1;
  }
}

inline int launch_status(const char* what) {
  hipError_t err = hipGetLastError();
  if (err != hipSuccess) return fail(TFHE_EHIP, "%s launch failed: %s", what, hipGetErrorString(err));
  return TFHE_OK;
}

// key rows and CMux count of a launch: the eval key's, or a stage check's
inline const double2* br_key(const tfhe_eval_key* ek, const BrIo& io) {
  return reinterpret_cast<const double2*>(io.bk ? io.bk : ek->bk_fft);
}
inline int br_steps(const tfhe_eval_key* ek, const BrIo& io) { return io.bk ? io.n : ek->p.n; }

template <int LOGN, int S, int WPB>
int launch_br_blocks(const tfhe_eval_key* ek, const Workspace& ws, const uint32_t* testvec, int64_t B,
                     hipStream_t st, const BrIo& io) {
  using C = BrCfg<LOGN, S, WPB>;
  const int64_t blocks = (B + C::CPB - 1) / C::CPB;
  hipLaunchKernelGGL((blind_rotate_kernel<LOGN, S, WPB>), dim3(static_cast<unsigned>(blocks)), dim3(C::THREADS),
                     0, st, br_key(ek, io), reinterpret_cast<const double2*>(ek->tw), ws.abar, testvec,
                     ws.extract, br_steps(ek, io), ek->p.l, ek->p.bg_bit, B, io.acc_in, io.acc_out);
  return launch_status("blind_rotate_kernel");
}

template <int LOGN, int S, int WPB, int SW = 2>
int launch_br_split(const tfhe_eval_key* ek, const Workspace& ws, const uint32_t* testvec, int64_t B,
                    hipStream_t st, const BrIo& io) {
  using C = BrSplitCfg<LOGN, S, WPB, SW>;
  const int64_t blocks = (B + C::CPB - 1) / C::CPB;
  hipLaunchKernelGGL((blind_rotate_split_kernel<LOGN, S, WPB, SW>), dim3(static_cast<unsigned>(blocks)),
                     dim3(C::THREADS), 0, st, br_key(ek, io), reinterpret_cast<const double2*>(ek->tw), ws.abar,
                     testvec, ws.extract, br_steps(ek, io), ek->p.l, ek->p.bg_bit, B, io.acc_in, io.acc_out);
  return launch_status("blind_rotate_split_kernel");
}

// the part of a launch's buffers after its first `head` ciphertexts
inline Workspace ws_tail(const tfhe_eval_key* ek, const Workspace& ws, const BrIo& io, int64_t head) {
  return Workspace{ws.abar + head * (br_steps(ek, io) + 1), ws.extract + head * (ek->p.N + 1)};
}
inline BrIo io_tail(const tfhe_eval_key* ek, const BrIo& io, int64_t head) {
  BrIo r = io;
  if (r.acc_in) r.acc_in += head * 2 * ek->p.N;
  if (r.acc_out) r.acc_out += head * 2 * ek->p.N;
  return r;
}

// Block shape by how many blocks a CU runs at once.  Blocks of one wave are
// compiled for one wave per SIMD, so a CU runs four side by side: a batch
// that fits four per CU takes them (the shortest CMux chain), a larger one
// blocks of 8 waves (two per SIMD, one block per CU, shared key reads in L1).
// A ciphertext of two waves likewise takes blocks of one ciphertext while
// three per CU (their LDS) hold the batch, else blocks of four.  Against the
// largest block that still gave every CU one: 600 gates 10.31 -> 9.6 ms,
// 1024 9.64 -> 9.30, 1500 19.55 -> 13.60 (one round of 8-wave blocks instead
// of two of 4-wave ones), 1000 lookups at N = 2048 27.2 -> 17.0 ms.  A batch
// whose last round of 8-wave blocks would be partly filled runs that tail as
// a second launch of one-wave blocks when four per CU hold it (2100 gates
// 29.9 -> 24.1 ms, 3000 28.8 -> 24.2, 53,760 382.6 -> 378.6; lookups at
// N = 2048 as one-ciphertext blocks, three per CU: 1102 35.6 -> 30.3 ms,
// 8292 153.0 -> 148.9).
template <int LOGN, int S>
int launch_br(const tfhe_eval_key* ek, const Workspace& ws, const uint32_t* testvec, int64_t B,
              hipStream_t st, const BrIo& io) {
  constexpr int T = BrCfg<LOGN, S, 8>::T;
  const int64_t cus = ek->cus > 0 ? ek->cus : 256;
  auto blocks = [&](int64_t b, int cpb) { return (b + cpb - 1) / cpb; };
  if constexpr (T <= 64) {
    constexpr int C1 = BrCfg<LOGN, S, 1>::CPB;
    if (blocks(B, C1) <= 4 * cus) return launch_br_blocks<LOGN, S, 1>(ek, ws, testvec, B, st, io);
    // full rounds of 8-wave blocks (one per CU); a last round that one-wave
    // blocks hold (four per CU) runs as those instead of as a partly filled
    // round of 8-wave blocks
    const int64_t round = int64_t{BrCfg<LOGN, S, 8>::CPB} * cus;
    const int64_t tail = B % round;
    if (tail == 0 || blocks(tail, C1) > 4 * cus) return launch_br_blocks<LOGN, S, 8>(ek, ws, testvec, B, st, io);
    const int64_t head = B - tail;
    if (int rc = launch_br_blocks<LOGN, S, 8>(ek, ws, testvec, head, st, io)) return rc;
    return launch_br_blocks<LOGN, S, 1>(ek, ws_tail(ek, ws, io, head), testvec, tail, st, io_tail(ek, io, head));
  } else if constexpr (T == 128) {
    // blocks of one ciphertext: one wave per SIMD while two per CU hold the
    // batch, else up to three per CU
    auto one_ct = [&](const Workspace& w, int64_t b, const BrIo& bio) {
      return b <= 2 * cus ? launch_br_split<LOGN, S, 2, 1>(ek, w, testvec, b, st, bio)
                          : launch_br_split<LOGN, S, 2>(ek, w, testvec, b, st, bio);
    };
    constexpr int C1 = BrSplitCfg<LOGN, S, 2>::CPB;
    if (blocks(B, C1) <= 3 * cus) return one_ct(ws, B, io);
    // as above: a partly filled last round runs as one-ciphertext blocks
    const int64_t round = int64_t{BrSplitCfg<LOGN, S, 8>::CPB} * cus;
    const int64_t tail = B % round;
    if (tail == 0 || blocks(tail, C1) > 3 * cus) return launch_br_split<LOGN, S, 8>(ek, ws, testvec, B, st, io);
    const int64_t head = B - tail;
    if (int rc = launch_br_split<LOGN, S, 8>(ek, ws, testvec, head, st, io)) return rc;
    return one_ct(ws_tail(ek, ws, io, head), tail, io_tail(ek, io, head));
  } else {
    return launch_br_blocks<LOGN, S, T / 64>(ek, ws, testvec, B, st, io);
  }
}

template <int LOGN, int S>
int launch_mul(const tfhe_eval_key* ek, const int32_t* d, const uint32_t* b, uint32_t* c, int64_t B,
               hipStream_t st) {
  constexpr int CPB = 256 / RingLayout<LOGN, S>::T;
  const int64_t blocks = (B + CPB - 1) / CPB;
  hipLaunchKernelGGL((negacyclic_mul_kernel<LOGN, S>), dim3(static_cast<unsigned>(blocks)), dim3(256), 0, st,
                     reinterpret_cast<const double2*>(ek->tw), d, b, c, B);
  return launch_status("negacyclic_mul_kernel");
}

template <template <int, int> class F, class... A>
int dispatch_ring(const tfhe_eval_key* ek, A... args) {
  const int N = ek->p.N, S = ek->parts;
#define GT_CASE(LOGN, SP) \
  if (N == (1 << LOGN) && S == SP) return F<LOGN, SP>::run(ek, args...);
  GT_CASE(8, 2) GT_CASE(8, 3) GT_CASE(9, 2) GT_CASE(9, 3) GT_CASE(10, 2) GT_CASE(10, 3) GT_CASE(11, 2)
  GT_CASE(11, 3)
#undef GT_CASE
  return fail(TFHE_EUNSUPPORTED, "no kernel for N=%d with %d key parts", N, S);
}

template <int LOGN, int S>
struct BrRun {
  static int run(const tfhe_eval_key* ek, const Workspace& ws, const uint32_t* tv, int64_t B, hipStream_t st,
                 const BrIo& io) {
    return launch_br<LOGN, S>(ek, ws, tv, B, st, io);
  }
};
template <int LOGN, int S>
struct MulRun {
  static int run(const tfhe_eval_key* ek, const int32_t* d, const uint32_t* b, uint32_t* c, int64_t B,
                 hipStream_t st) {
    return launch_mul<LOGN, S>(ek, d, b, c, B, st);
  }
};

}  // namespace

int64_t workspace_bytes(const tfhe_params& p, int64_t B) {
  const int64_t a = ((B * (p.n + 1) * 2) + 255) / 256 * 256;
  const int64_t x = ((B * (p.N + 1) * 4) + 255) / 256 * 256;
  return a + x;
}

Workspace carve_workspace(const tfhe_params& p, void* ws, int64_t B) {
  const int64_t a = ((B * (p.n + 1) * 2) + 255) / 256 * 256;
  Workspace w;
  w.abar = static_cast<uint16_t*>(ws);
  w.extract = reinterpret_cast<uint32_t*>(static_cast<char*>(ws) + a);
  return w;
}

int launch_prep(const tfhe_eval_key* ek, const PrepArgs& a, const Workspace& ws, void* stream) {
  const int64_t total = a.B * (ek->p.n + 1);
  const int64_t blocks = (total + 255) / 256;
  hipLaunchKernelGGL(prep_kernel, dim3(static_cast<unsigned>(blocks)), dim3(256), 0,
                     static_cast<hipStream_t>(stream), a, ek->p.n, ek->p.N, ws.abar);
  return launch_status("prep_kernel");
}

int launch_blind_rotate(const tfhe_eval_key* ek, const Workspace& ws, const uint32_t* testvec,
                        int64_t B, void* stream, const BrIo* io) {
  const BrIo none{};
  return dispatch_ring<BrRun>(ek, ws, testvec, B, static_cast<hipStream_t>(stream), io ? *io : none);
}

int launch_keyswitch(const tfhe_eval_key* ek, const uint32_t* in, uint32_t* out, int64_t B, int mode,
                     int32_t bits, int64_t gate_begin, void* stream) {
  const tfhe_params& p = ek->p;
  if (p.ks_t * (1 << p.ks_basebit) > KS_MAXROWS)
    return fail(TFHE_EUNSUPPORTED, "key switching with t * 2^basebit = %d > %d rows per coefficient",
                p.ks_t * (1 << p.ks_basebit), KS_MAXROWS);
  dim3 grid(static_cast<unsigned>((B + KS_CB - 1) / KS_CB), static_cast<unsigned>((p.n + 1 + KS_COLS - 1) / KS_COLS));
  hipStream_t st = static_cast<hipStream_t>(stream);
  if (ks_uses_mfma(p)) {
    // split the input coefficients over k blocks per (sample tile, column
    // tile) so that the rounds of resident blocks (two per CU) are full:
    // the smallest ceil(tiles k / resident) ceil(N / k) for k <= 8
    const int64_t cus = ek->cus > 0 ? ek->cus : 256;
    KsmGrid g;
    g.nb_total = ksk_mfma_nb(p);
    g.col_tiles = g.nb_total / KSM_NB;
    const int64_t sample_tiles = (B + KSM_SAMPLES - 1) / KSM_SAMPLES;
    g.sample_tiles = static_cast<int>(sample_tiles);
    const int64_t tiles = sample_tiles * g.col_tiles, resident = 2 * cus;
    int64_t best_k = 1, best = -1;
    for (int64_t k = 1; k <= 8 && k <= p.N; k++) {
      const int64_t len = (p.N + k - 1) / k, ranges = (p.N + len - 1) / len;
      const int64_t cost = (tiles * ranges + resident - 1) / resident * len;
      if (best < 0 || cost < best) best = cost, best_k = k;
    }
    g.coef_len = static_cast<int>(((p.N + best_k - 1) / best_k + KSM_CH - 1) / KSM_CH * KSM_CH);
    const int64_t ranges = (p.N + g.coef_len - 1) / g.coef_len;
    const int64_t blocks = tiles * ranges;
    hipLaunchKernelGGL(keyswitch_init_kernel, dim3(static_cast<unsigned>((B * (p.n + 1) + 255) / 256)), dim3(256), 0,
                       st, in, out, p.n, p.N, B, mode, bits, gate_begin);
    if (int rc = launch_status("keyswitch_init_kernel")) return rc;
    hipLaunchKernelGGL(keyswitch_mfma_kernel, dim3(static_cast<unsigned>(blocks)), dim3(KSM_THREADS), 0, st, in,
                       reinterpret_cast<const i32x4*>(ek->ksk_mfma), out, p.n, p.N, B, mode, bits, gate_begin, g);
  } else if (p.ks_t * (1 << p.ks_basebit) <= 32)
    hipLaunchKernelGGL((keyswitch_kernel<32>), grid, dim3(KS_COLS), 0, st, in, ek->ksk, out, p.n, p.N,
                       p.ks_t, p.ks_basebit, B, mode, bits, gate_begin);
  else
    hipLaunchKernelGGL((keyswitch_kernel<64>), grid, dim3(KS_COLS), 0, st, in, ek->ksk, out, p.n, p.N,
                       p.ks_t, p.ks_basebit, B, mode, bits, gate_begin);
  return launch_status("keyswitch_kernel");
}

int launch_relu_sign(const tfhe_eval_key* ek, uint32_t* y, int32_t bits, int64_t v_begin, int64_t v_end,
                     void* stream) {
  const int64_t count = v_end - v_begin;
  if (count <= 0) return TFHE_OK;
  const int64_t blocks = (count * (ek->p.n + 1) + 255) / 256;
  hipLaunchKernelGGL(relu_sign_kernel, dim3(static_cast<unsigned>(blocks)), dim3(256), 0,
                     static_cast<hipStream_t>(stream), y, ek->p.n, bits, v_begin, count);
  return launch_status("relu_sign_kernel");
}

int launch_cmux_abar(const tfhe_eval_key* ek, const uint32_t* a, int64_t B, uint16_t* abar, void* stream) {
  hipLaunchKernelGGL(cmux_abar_kernel, dim3(static_cast<unsigned>((B + 255) / 256)), dim3(256), 0,
                     static_cast<hipStream_t>(stream), a, ek->p.N, B, abar);
  return launch_status("cmux_abar_kernel");
}

int launch_not(int32_t dim, const uint32_t* in, uint32_t* out, int64_t count, void* stream) {
  const int64_t words = count * (dim + 1);
  const int64_t blocks = (words + 255) / 256;
  hipLaunchKernelGGL(not_kernel, dim3(static_cast<unsigned>(blocks)), dim3(256), 0,
                     static_cast<hipStream_t>(stream), in, out, words);
  return launch_status("not_kernel");
}

int launch_mux_combine(const tfhe_eval_key* ek, uint32_t* ext, int64_t M, void* stream) {
  const int64_t words = M * (ek->p.N + 1);
  if (words == 0) return TFHE_OK;
  hipLaunchKernelGGL(mux_combine_kernel, dim3(static_cast<unsigned>((words + 255) / 256)), dim3(256), 0,
                     static_cast<hipStream_t>(stream), ext, ek->p.N, M);
  return launch_status("mux_combine_kernel");
}

int launch_lut_leaf(const tfhe_eval_key* ek, const uint32_t* x, int32_t msg_bits, const uint32_t* table,
                    int32_t out_bits, int64_t V, uint32_t* nodes, void* stream) {
  if (msg_bits < 1 || msg_bits > 6) return fail(TFHE_EUNSUPPORTED, "table lookup over %d bits", msg_bits);
  LutTable t{};
  for (int k = 0; k < (1 << msg_bits); k++) t.s[k] = table[k];
  const int64_t words = V * out_bits * (int64_t{1} << (msg_bits - 1)) * (ek->p.n + 1);
  if (words == 0) return TFHE_OK;
  hipLaunchKernelGGL(lut_leaf_kernel, dim3(static_cast<unsigned>((words + 255) / 256)), dim3(256), 0,
                     static_cast<hipStream_t>(stream), x, ek->p.n, msg_bits, t, out_bits, V, nodes);
  return launch_status("lut_leaf_kernel");
}

// The packing key switch on the transform: at N = 1024 blocks of 8 waves when
// the batch fills one (their outputs share the key reads in L1), else
// one-wave blocks;
// IC input coefficients per block, at most pks_ic_max, chosen so that the
// rounds of resident blocks times a block's work (IC t (base - 1) forward
// transforms and four inverse ones) is least.
template <int WPB, int LOGN>
int launch_pack_fft_blocks(const tfhe_eval_key* ek, const uint32_t* lwe, int32_t Z, uint32_t* out, int64_t B,
                           hipStream_t st) {
  using C = BrCfg<LOGN, 2, WPB>;
  const tfhe_params& p = ek->p;
  const int vals = (1 << p.ks_basebit) - 1, R = p.ks_t * vals;
  const int64_t cus = ek->cus > 0 ? ek->cus : 256;
  const int64_t groups = (B + C::CPB - 1) / C::CPB;
  const int64_t resident = cus * (WPB == 8 ? 1 : 4);
  int64_t best_ic = 1, best = -1;
  for (int64_t ic = 1; ic <= ek->pks_ic_max; ic++) {
    const int64_t blocks = groups * ((p.n + ic - 1) / ic);
    const int64_t cost = (blocks + resident - 1) / resident * (ic * R + 4);
    if (best < 0 || cost < best) best = cost, best_ic = ic;
  }
  const int64_t blocks = groups * ((p.n + best_ic - 1) / best_ic);
  if (blocks > 0x7fffffff) return fail(TFHE_EINVAL, "too many TRLWE outputs for one launch");
  hipLaunchKernelGGL((pack_ks_fft_kernel<LOGN, WPB>), dim3(static_cast<unsigned>(blocks)), dim3(C::THREADS), 0, st,
                     reinterpret_cast<const double2*>(ek->pks_fft), reinterpret_cast<const double2*>(ek->tw), lwe,
                     p.n, Z, p.ks_t, p.ks_basebit, static_cast<int>(best_ic), static_cast<int>(groups), B, out);
  return launch_status("pack_ks_fft_kernel");
}

template <int LOGN>
int launch_pack_fft(const tfhe_eval_key* ek, const uint32_t* lwe, int32_t Z, uint32_t* out, int64_t B,
                    hipStream_t st) {
  // (blocks of 8 waves at N < 1024 would spill registers: one-wave blocks
  // there hold 64 / T outputs each)
  if constexpr (LOGN == 10)
    if (B >= 8) return launch_pack_fft_blocks<8, LOGN>(ek, lwe, Z, out, B, st);
  return launch_pack_fft_blocks<1, LOGN>(ek, lwe, Z, out, B, st);
}

int launch_pack_keyswitch(const tfhe_eval_key* ek, const uint32_t* lwe, int32_t Z, uint32_t* out, int64_t B,
                          void* stream) {
  const tfhe_params& p = ek->p;
  if (p.ks_t * p.ks_basebit > 16 || (1 << p.ks_basebit) - 1 > 3)
    return fail(TFHE_EUNSUPPORTED, "packing key switching needs t * basebit <= 16 and basebit <= 2");
  hipStream_t st = static_cast<hipStream_t>(stream);
  const int64_t words = B * 2 * p.N;
  hipLaunchKernelGGL(pack_init_kernel, dim3(static_cast<unsigned>((words + 255) / 256)), dim3(256), 0, st, lwe,
                     p.n, p.N, Z, B, out);
  int rc = launch_status("pack_init_kernel");
  if (rc) return rc;
  if (ek->pks_fft != nullptr) {
    switch (p.N) {
      case 256: return launch_pack_fft<8>(ek, lwe, Z, out, B, st);
      case 512: return launch_pack_fft<9>(ek, lwe, Z, out, B, st);
      case 1024: return launch_pack_fft<10>(ek, lwe, Z, out, B, st);
      default: break;
    }
  }
  dim3 grid(static_cast<unsigned>(B), static_cast<unsigned>((p.n + PKS_IC - 1) / PKS_IC));
  switch (p.N) {
    case 256: hipLaunchKernelGGL(pack_ks_kernel<256>, grid, dim3(256), 0, st, lwe, ek->pks, p.n, Z, p.ks_t, p.ks_basebit, out); break;
    case 512: hipLaunchKernelGGL(pack_ks_kernel<512>, grid, dim3(256), 0, st, lwe, ek->pks, p.n, Z, p.ks_t, p.ks_basebit, out); break;
    case 1024: hipLaunchKernelGGL(pack_ks_kernel<1024>, grid, dim3(256), 0, st, lwe, ek->pks, p.n, Z, p.ks_t, p.ks_basebit, out); break;
    case 2048: hipLaunchKernelGGL(pack_ks_kernel<2048>, grid, dim3(256), 0, st, lwe, ek->pks, p.n, Z, p.ks_t, p.ks_basebit, out); break;
    default: return fail(TFHE_EUNSUPPORTED, "packing key switching for N=%d", p.N);
  }
  return launch_status("pack_ks_kernel");
}

int launch_sample_extract(int32_t N, const uint32_t* trlwe, int64_t B, int32_t K, uint32_t* out, void* stream) {
  const int64_t words = B * K * (N + 1);
  hipLaunchKernelGGL(sample_extract_kernel, dim3(static_cast<unsigned>((words + 255) / 256)), dim3(256), 0,
                     static_cast<hipStream_t>(stream), trlwe, N, B, K, out);
  return launch_status("sample_extract_kernel");
}

int launch_negacyclic_mul(const tfhe_eval_key* ek, const int32_t* d, const uint32_t* b, uint32_t* c,
                          int64_t B, void* stream) {
  return dispatch_ring<MulRun>(ek, d, b, c, B, static_cast<hipStream_t>(stream));
}

}  // namespace gt
