// HIP kernels of the TFHE activation path for gfx950 (MI355X).
//
//   prep_kernel          gate pre-combination (Section 3.1 gates; NOT is free)
//                        and modulus switch of every LWE word to Z_{2N}
//   blind_rotate_kernel  accumulator init, n CMux external products with exact
//                        negacyclic products (fp64 NTT mod P), SampleExtract
//   keyswitch_kernel     LWE key switching back to dimension n
//   relu_sign_kernel     trivial 0 for the sign bit of the ReLU output
//   not_kernel           NOT without bootstrapping
//   negacyclic_mul_kernel  standalone exact product (checks the transform)
//
// Blind rotation layout: one polynomial of a ciphertext is held by T = N/E
// threads with E values each (gt_layout.hpp); T = 64 (one wave) for
// N <= 1024 and 128 for N = 2048.  A 256-thread block carries 256/T
// ciphertexts.  The accumulator (two u32 polynomials) and a transpose scratch
// of N doubles per ciphertext live in LDS; the four transform-domain
// accumulators of an external product (mask/body x high/low key halves) live
// in registers.  The bootstrapping key is read straight from global memory in
// the transform-domain layout, coalesced across the T threads, and shared by
// all ciphertexts in flight through L2.
#include <hip/hip_runtime.h>

#include <type_traits>

#include "gt_internal.h"
#include "gt_layout.hpp"
#include "gt_modp.hpp"

namespace gt {

namespace {

constexpr uint32_t kMu = 0x20000000u;  // 1/8

// minimum waves per SIMD the blind-rotation kernel is compiled for (sets its
// register budget: 2 -> 256 VGPRs, 3 -> 168)
#ifndef GT_BR_WAVES_PER_SIMD
#define GT_BR_WAVES_PER_SIMD 2
#endif

template <int B, int E, class F>
__device__ __forceinline__ void static_for(F&& f) {
  if constexpr (B < E) {
    f(std::integral_constant<int, B>{});
    static_for<B + 1, E>(f);
  }
}

// Make LDS writes of all threads of a polynomial visible to its other threads.
// A polynomial held by a single wave needs only ordering (a wave's LDS
// operations complete in order); a polynomial spread over two waves needs the
// block barrier.
template <int T>
__device__ __forceinline__ void poly_sync() {
  if constexpr (T <= 64) {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
  } else {
    __syncthreads();
  }
}

// bank swizzle of the transpose scratch: with 8 values per thread every pass
// layout at N = 512..2048 reads and writes 64-bit elements without bank
// conflicts (checked for 32 and 64 banks of 4 bytes); it permutes only the low
// 5 bits, so it stays inside the polynomial
__device__ __forceinline__ int swz(int j) { return j ^ (((j >> 3) ^ (j >> 7)) & 31); }

// Position of twiddle k in the LDS copy of a twiddle table.  Stage s owns
// k in [N/2^(s+1), N/2^s); in a pass other than the first, thread t reads the
// stage's entries m = (t >> w) * G + g, g < G, so they are stored [g][t >> w]
// to make the threads of a wave read consecutive words.  First-pass twiddles
// are read uniformly from global memory and keep their natural place.
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

template <class Lay, int WFROM, int WTO>
__device__ __forceinline__ void transpose(double (&x)[Lay::E], int t, double* scr) {
  static_for<0, Lay::E>([&](auto EI) {
    constexpr int e = decltype(EI)::value;
    scr[swz(Lay::jmap(t, e, WFROM))] = x[e];
  });
  poly_sync<Lay::T>();
  static_for<0, Lay::E>([&](auto EI) {
    constexpr int e = decltype(EI)::value;
    x[e] = scr[swz(Lay::jmap(t, e, WTO))];
  });
  poly_sync<Lay::T>();
}

// Offset of stage k's twiddles within a pass's batch: the stages before it
// (descending bits for the forward transform, ascending for the inverse) use
// E >> (b + 1) twiddles each, b the stage's bit within the pass window.
template <class Lay>
constexpr int tw_offset(int p, int k, bool fwd) {
  int off = 0;
  for (int q = 0; q < k; q++) {
    const int s = fwd ? Lay::hi(p) - 1 - q : Lay::lo(p) + q;
    off += Lay::E >> (s - Lay::win(p) + 1);
  }
  return off;
}

// Forward negacyclic NTT (Cooley-Tukey butterflies, twiddle psi^brv(k) for the
// block of coefficient j at stage s: k = N/2^(s+1) + j/2^(s+1)).  In: pass-0
// (coefficient) layout; out: last-pass (transform) layout.  |in| < 2^10 gives
// |out| < 2^43 (each stage adds at most 0.75P + 2^35).  The twiddles of a pass
// are fetched together before its butterflies: pass 0's are the same for every
// thread (tw_uniform, read through the scalar cache), the others come from
// tw: an LDS copy laid out by tw_lds_slot (TW_PERMUTED) or a natural-order
// table in global memory.  SMALL_IN: inputs are below 2^10 in magnitude, so the first
// stage's products are exact without the low part.
template <class Lay, bool SMALL_IN, bool TW_PERMUTED>
__device__ __forceinline__ void ntt_forward(double (&x)[Lay::E], int t, double* scr,
                                            const double* __restrict__ tw,
                                            const double* __restrict__ tw_uniform) {
  constexpr int N = Lay::N, LOGE = Lay::LOGE, E = Lay::E;
  static_for<0, Lay::NPASS>([&](auto PI) {
    constexpr int p = decltype(PI)::value;
    constexpr int w = Lay::win(p);
    constexpr int NS = Lay::hi(p) - Lay::lo(p);
    if constexpr (p > 0) transpose<Lay, Lay::win(p - 1), w>(x, t, scr);
    // twiddles of all stages of the pass: stage si uses z[off(si) .. off(si) + G(si))
    double z[E];
    static_for<0, NS>([&](auto SI) {
      constexpr int s = Lay::hi(p) - 1 - decltype(SI)::value;
      constexpr int b = s - w;
      constexpr int G = E >> (b + 1);
      constexpr int off = tw_offset<Lay>(p, decltype(SI)::value, true);
      static_for<0, G>([&](auto GI) {
        constexpr int g = decltype(GI)::value;
        if constexpr (p == 0)
          z[off + g] = tw_uniform[(N >> (s + 1)) + g];
        else if constexpr (TW_PERMUTED)
          z[off + g] = tw[(N >> (s + 1)) + g * ((N >> (s + 1)) / G) + (t >> w)];
        else
          z[off + g] = tw[(N >> (s + 1)) + ((t >> w) << (LOGE - b - 1)) + g];
      });
    });
    static_for<0, NS>([&](auto SI) {
      constexpr int s = Lay::hi(p) - 1 - decltype(SI)::value;
      constexpr int b = s - w;
      constexpr int G = E >> (b + 1);
      constexpr int off = tw_offset<Lay>(p, decltype(SI)::value, true);
      constexpr bool small = SMALL_IN && p == 0 && decltype(SI)::value == 0;
      static_for<0, G>([&](auto GI) {
        constexpr int g = decltype(GI)::value;
        static_for<0, (1 << b)>([&](auto LI) {
          constexpr int e = (g << (b + 1)) | decltype(LI)::value;
          constexpr int e2 = e | (1 << b);
          const double u = x[e];
          const double v = small ? mulmod_small(x[e2], z[off + g]) : mulmod(x[e2], z[off + g]);
          x[e] = u + v;
          x[e2] = u - v;
        });
      });
    });
  });
}

// Inverse transform without the 1/N factor (Gentleman-Sande butterflies,
// twiddle psi^-brv(k)).  In: transform layout, |in| <= P/2 + 1; out:
// coefficient layout, |out| < 2^(38 + LOGN) (sums double per stage).
template <class Lay, bool TW_PERMUTED>
__device__ __forceinline__ void ntt_inverse(double (&x)[Lay::E], int t, double* scr,
                                            const double* __restrict__ tw,
                                            const double* __restrict__ tw_uniform) {
  constexpr int N = Lay::N, LOGE = Lay::LOGE, E = Lay::E;
  static_for<0, Lay::NPASS>([&](auto PI) {
    constexpr int p = Lay::NPASS - 1 - decltype(PI)::value;
    constexpr int w = Lay::win(p);
    constexpr int NS = Lay::hi(p) - Lay::lo(p);
    if constexpr (p < Lay::NPASS - 1) transpose<Lay, Lay::win(p + 1), w>(x, t, scr);
    // stage si (ascending bit s = lo + si) uses z[off(si) .. off(si) + G(si))
    double z[E];
    static_for<0, NS>([&](auto SI) {
      constexpr int s = Lay::lo(p) + decltype(SI)::value;
      constexpr int b = s - w;
      constexpr int G = E >> (b + 1);
      constexpr int off = tw_offset<Lay>(p, decltype(SI)::value, false);
      static_for<0, G>([&](auto GI) {
        constexpr int g = decltype(GI)::value;
        if constexpr (p == 0)
          z[off + g] = tw_uniform[(N >> (s + 1)) + g];
        else if constexpr (TW_PERMUTED)
          z[off + g] = tw[(N >> (s + 1)) + g * ((N >> (s + 1)) / G) + (t >> w)];
        else
          z[off + g] = tw[(N >> (s + 1)) + ((t >> w) << (LOGE - b - 1)) + g];
      });
    });
    static_for<0, NS>([&](auto SI) {
      constexpr int s = Lay::lo(p) + decltype(SI)::value;
      constexpr int b = s - w;
      constexpr int G = E >> (b + 1);
      constexpr int off = tw_offset<Lay>(p, decltype(SI)::value, false);
      static_for<0, G>([&](auto GI) {
        constexpr int g = decltype(GI)::value;
        static_for<0, (1 << b)>([&](auto LI) {
          constexpr int e = (g << (b + 1)) | decltype(LI)::value;
          constexpr int e2 = e | (1 << b);
          const double u = x[e];
          const double v = x[e2];
          x[e] = u + v;
          x[e2] = mulmod(u - v, z[off + g]);
        });
      });
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

__global__ __launch_bounds__(256) void prep_kernel(int mode, int gate, const uint32_t* __restrict__ ca,
                                                   const uint32_t* __restrict__ cb, int n, int N,
                                                   int64_t B, int32_t bits, int64_t gate_begin,
                                                   uint16_t* __restrict__ abar) {
  const int64_t idx = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  const int64_t total = B * (n + 1);
  if (idx >= total) return;
  const int64_t c = idx / (n + 1);
  const int k = static_cast<int>(idx - c * (n + 1));
  uint32_t x;
  if (mode == kModePlain) {
    x = ca[c * (n + 1) + k];
  } else {
    const uint32_t* pa;
    const uint32_t* pb;
    if (mode == kModeRelu) {
      const int64_t g = gate_begin + c;
      const int64_t v = g / (bits - 1), i = g - v * (bits - 1);
      pa = ca + (v * bits + (bits - 1)) * (n + 1);  // sign bit
      pb = ca + (v * bits + i) * (n + 1);
    } else {
      pa = ca + c * (n + 1);
      pb = cb + c * (n + 1);
    }
    const GateCoef gc = gate_coef(mode == kModeRelu ? static_cast<int>(TFHE_ANDNY) : gate);
    x = static_cast<uint32_t>(gc.wa) * pa[k] + static_cast<uint32_t>(gc.wb) * pb[k] +
        (k == n ? gc.konst : 0u);
  }
  abar[idx] = mod_switch(x, N);
}

// ------------------------------------------------------ blind rotation
template <int LOGN>
struct BrCfg {
  using Lay = Layout<LOGN>;
  static constexpr int N = Lay::N, E = Lay::E, T = Lay::T;
  // ciphertexts per block: a block's barriers couple the waves of all its
  // ciphertexts, so fewer per block means less waiting on the slowest wave
#ifdef GT_BR_CPB
  static constexpr int CPB = GT_BR_CPB;
#else
  static constexpr int CPB = T >= 256 ? 1 : 256 / T;
#endif
  static constexpr int THREADS = CPB * T;
  static constexpr bool kTwLds = true;               // twiddle tables in LDS
};

template <int LOGN>
__global__ __launch_bounds__(BrCfg<LOGN>::THREADS, GT_BR_WAVES_PER_SIMD) void blind_rotate_kernel(
    const double* __restrict__ bk, const double* __restrict__ tw_fwd_g,
    const double* __restrict__ tw_inv_g, const uint16_t* __restrict__ abar,
    const uint32_t* __restrict__ testvec, uint32_t* __restrict__ extract, int n, int l, int bg_bit,
    int64_t B) {
  using C = BrCfg<LOGN>;
  using Lay = typename C::Lay;
  constexpr int N = C::N, E = C::E, T = C::T, CPB = C::CPB;
  __shared__ double s_tw[C::kTwLds ? 2 * N : 1];
  __shared__ double s_scr[CPB * N];
  __shared__ uint32_t s_acc[CPB * 2 * N];

  const int slot = threadIdx.x / T;
  const int t = threadIdx.x % T;
  int64_t c = static_cast<int64_t>(blockIdx.x) * CPB + slot;
  const bool active = c < B;
  if (!active) c = B - 1;  // idle slots repeat the last sample and write nothing

  const double* twf;
  const double* twi;
  if constexpr (C::kTwLds) {
    for (int k = threadIdx.x; k < N; k += C::THREADS) {
      const int slot = tw_lds_slot<Lay>(k);
      s_tw[slot] = tw_fwd_g[k];
      s_tw[N + slot] = tw_inv_g[k];
    }
    __syncthreads();
    twf = s_tw;
    twi = s_tw + N;
  } else {
    twf = tw_fwd_g;
    twi = tw_inv_g;
  }
  double* scr = s_scr + slot * N;
  uint32_t* acc_a = s_acc + slot * 2 * N;
  uint32_t* acc_b = acc_a + N;
  const uint16_t* ab = abar + c * (n + 1);

  // ACC = (0, X^{-bbar} v)
  {
    const uint32_t bbar = ab[n];
    const uint32_t e0 = (2u * N - bbar) & (2u * N - 1);
    for (int e = 0; e < E; e++) {
      const int j = t + T * e;
      acc_a[j] = 0u;
      uint32_t v;
      if (testvec == nullptr) {
        const int src = j - static_cast<int>(e0 & (N - 1));
        const uint32_t m = static_cast<uint32_t>(src >> 31) ^ (0u - ((e0 / N) & 1u));
        v = (kMu ^ m) - m;
      } else {
        v = rot_coef<N>(testvec, e0, j);
      }
      acc_b[j] = v;
    }
    poly_sync<T>();
  }

  const uint32_t half = 1u << (bg_bit - 1);
  const uint32_t dmask = (1u << bg_bit) - 1u;
  uint32_t offset = 0;
  for (int j = 1; j <= l; j++) offset += half << (32 - j * bg_bit);
  if (l * bg_bit < 32) offset += 1u << (31 - l * bg_bit);
  const size_t bk_step = static_cast<size_t>(2 * l) * 4 * N;

  for (int i = 0; i < n; i++) {
    const uint32_t a_i = ab[i];
    const double* bki = bk + static_cast<size_t>(i) * bk_step;
    double acc[4][E];
#pragma unroll
    for (int o = 0; o < 4; o++)
#pragma unroll
      for (int e = 0; e < E; e++) acc[o][e] = 0.0;

    for (int q = 0; q < 2; q++) {
      const uint32_t* P = q ? acc_b : acc_a;
      uint32_t D[E];
#pragma unroll
      for (int e = 0; e < E; e++) {
        const int j = t + T * e;
        D[e] = rot_coef<N>(P, a_i, j) - P[j] + offset;
      }
      for (int jj = 0; jj < l; jj++) {
        const int shift = 32 - (jj + 1) * bg_bit;
        double x[E];
#pragma unroll
        for (int e = 0; e < E; e++)
          x[e] = static_cast<double>(static_cast<int32_t>((D[e] >> shift) & dmask) - static_cast<int32_t>(half));
        // key row r = q*l + jj: four output polynomials, each stored as
        // [E/2][T][2] so a thread's pair of values is one 16-byte load
        const double2* bkr =
            reinterpret_cast<const double2*>(bki + static_cast<size_t>(q * l + jj) * 4 * N) + t;
        ntt_forward<Lay, true, C::kTwLds>(x, t, scr, twf, tw_fwd_g);
        double2 w[E / 2];
#pragma unroll
        for (int h = 0; h < E / 2; h++) w[h] = bkr[h * T];
#pragma unroll
        for (int o = 0; o < 4; o++) {
          double2 wn[E / 2];
          if (o < 3) {
#pragma unroll
            for (int h = 0; h < E / 2; h++) wn[h] = bkr[(o + 1) * (N / 2) + h * T];
          }
#pragma unroll
          for (int h = 0; h < E / 2; h++) {
            acc[o][2 * h] += mulmod(x[2 * h], w[h].x);
            acc[o][2 * h + 1] += mulmod(x[2 * h + 1], w[h].y);
          }
          if (o < 3) {
#pragma unroll
            for (int h = 0; h < E / 2; h++) w[h] = wn[h];
          }
        }
      }
    }

#pragma unroll
    for (int o = 0; o < 4; o++) {
#pragma unroll
      for (int e = 0; e < E; e++) acc[o][e] = reduce(acc[o][e]);
      ntt_inverse<Lay, C::kTwLds>(acc[o], t, scr, twi, tw_inv_g);
#pragma unroll
      for (int e = 0; e < E; e++) acc[o][e] = reduce(acc[o][e]);
    }
#pragma unroll
    for (int e = 0; e < E; e++) {
      const int j = t + T * e;
      acc_a[j] += (low32(acc[0][e]) << 16) + low32(acc[1][e]);
      acc_b[j] += (low32(acc[2][e]) << 16) + low32(acc[3][e]);
    }
    poly_sync<T>();
  }

  // SampleExtract of coefficient 0: (A_0, -A_{N-1}, ..., -A_1, B_0)
  if (active) {
    uint32_t* out = extract + c * (N + 1);
    for (int e = 0; e < E; e++) {
      const int j = t + T * e;
      out[j] = j == 0 ? acc_a[0] : 0u - acc_a[N - j];
    }
    if (t == 0) out[N] = acc_b[0];
  }
}

// ------------------------------------------------------- key switching
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

// KT > 0: digit count and base fixed at compile time (the digit loop unrolls);
// KT = 0: runtime ks_t / basebit.  MAXROWS >= ks_t * 2^basebit.
template <int MAXROWS, int KT, int KBB>
__global__ __launch_bounds__(64) void keyswitch_kernel(const uint32_t* __restrict__ in,
                                                       const uint32_t* __restrict__ ksk,
                                                       uint32_t* __restrict__ out, int n, int N,
                                                       int ks_t_rt, int basebit_rt, int64_t B, int mode,
                                                       int32_t bits, int64_t gate_begin) {
  __shared__ uint32_t s_in[KS_CB][KS_ICH];
  __shared__ uint32_t s_rows[2][MAXROWS][KS_COLS];
  const int ks_t = KT > 0 ? KT : ks_t_rt;
  const int basebit = KT > 0 ? KBB : basebit_rt;
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
      if constexpr (KT > 0) {
#pragma unroll 8
        for (int k = 0; k < KS_CB; k++) {
          const uint32_t x = __builtin_amdgcn_readfirstlane(s_in[k][ii]);
          const uint32_t r = prec == 32 ? x : (x + round) >> (32 - prec);
          uint32_t sum = 0u;
#pragma unroll
          for (int j = 0; j < KT; j++) {
            const uint32_t v = (r >> ((KT - 1 - j) * KBB)) & ((1u << KBB) - 1u);
            sum += rows[((j << KBB) + v) * KS_COLS];
          }
          acc[k] -= sum;
        }
      } else {
#pragma unroll 4
        for (int k = 0; k < KS_CB; k++) {
          const uint32_t x = __builtin_amdgcn_readfirstlane(s_in[k][ii]);
          const uint32_t r = prec == 32 ? x : (x + round) >> (32 - prec);
          for (int j = 0; j < ks_t; j++) {
            const uint32_t v = (r >> ((ks_t - 1 - j) * basebit)) & static_cast<uint32_t>(vals);
            acc[k] -= rows[(j * base + v) * KS_COLS];
          }
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
    int64_t dst = c;
    if (mode == kModeRelu) {
      const int64_t g = gate_begin + c;
      const int64_t v = g / (bits - 1), bit = g - v * (bits - 1);
      dst = v * bits + bit;
    }
    out[dst * row + col] = acc[k];
  }
}

// Key switching for t = 8 digits of 2 bits (16-bit precision).  A block of 4
// waves covers 64 output columns of 4 x 32 samples.  For each input
// coefficient i the block builds, in LDS, the pair tables
//   PT[p][u][col] = KSK[i][2p][u >> 2] + KSK[i][2p+1][u & 3]   (row of value 0 = 0)
// for the 4 digit pairs p and the 16 pair values u; a sample then needs 4
// table reads for the 8 digits.  Tables are double-buffered across i; the key
// rows are fetched one coefficient ahead.  Every table read, add and the
// final subtraction are exact mod 2^32.
constexpr int KS8_WAVES = 4;
#ifndef GT_KS8_CB
#define GT_KS8_CB 16
#endif
constexpr int KS8_CB = GT_KS8_CB;  // samples per wave

__global__ __launch_bounds__(256) void keyswitch_t8b2_kernel(const uint32_t* __restrict__ in,
                                                             const uint32_t* __restrict__ ksk,
                                                             uint32_t* __restrict__ out, int n, int N,
                                                             int64_t B, int mode, int32_t bits,
                                                             int64_t gate_begin) {
  constexpr int ROWS = 24;              // 8 digits x 3 non-zero values
  constexpr int TAB = 64;               // 4 pairs x 16 pair values
  __shared__ uint32_t s_tab[2][TAB][KS_COLS];
  __shared__ uint32_t s_in[KS8_WAVES * KS8_CB][KS_ICH];
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int col = blockIdx.y * KS_COLS + lane;
  const bool col_ok = col <= n;
  const int64_t c0 = static_cast<int64_t>(blockIdx.x) * (KS8_WAVES * KS8_CB);
  const int64_t cw = c0 + wave * KS8_CB;
  const size_t row = static_cast<size_t>(n) + 1;

  uint32_t acc[KS8_CB];
#pragma unroll
  for (int k = 0; k < KS8_CB; k++) {
    const int64_t c = cw + k;
    acc[k] = (col == n && c < B) ? in[c * (N + 1) + N] : 0u;
  }

  // thread (wave, lane) fetches key rows wave*6 .. wave*6+5 of its column and
  // builds table entries (pair = wave, all 16 values) -- the two digit rows a
  // pair needs are rows 6*wave .. 6*wave+5, exactly this thread's fetch
  uint32_t kr[6];
  auto fetch = [&](int i) {
    const uint32_t* base = ksk + static_cast<size_t>(i) * ROWS * row + col;
#pragma unroll
    for (int q = 0; q < 6; q++) kr[q] = col_ok ? base[static_cast<size_t>(wave * 6 + q) * row] : 0u;
  };
  auto build = [&](int b) {
    // kr[0..2]: digit 2*wave, values 1..3; kr[3..5]: digit 2*wave+1, values 1..3
#pragma unroll
    for (int u = 0; u < 16; u++) {
      const int v1 = u >> 2, v2 = u & 3;
      const uint32_t a = v1 ? kr[v1 - 1] : 0u;
      const uint32_t c = v2 ? kr[2 + v2] : 0u;
      s_tab[b][wave * 16 + u][lane] = a + c;
    }
  };

  fetch(0);
  for (int i0 = 0; i0 < N; i0 += KS_ICH) {
    __syncthreads();
    for (int idx = threadIdx.x; idx < KS8_WAVES * KS8_CB * KS_ICH; idx += 256) {
      const int k = idx / KS_ICH, ii = idx % KS_ICH;
      const int64_t c = c0 + k;
      s_in[k][ii] = (c < B && i0 + ii < N) ? in[c * (N + 1) + i0 + ii] : 0u;
    }
    const int iend = min(KS_ICH, N - i0);
    for (int ii = 0; ii < iend; ii++) {
      const int i = i0 + ii;
      const int b = i & 1;
      build(b);
      if (i + 1 < N) fetch(i + 1);
      __syncthreads();
      const uint32_t* tab = &s_tab[b][0][lane];
#pragma unroll 8
      for (int k = 0; k < KS8_CB; k++) {
        const uint32_t x = __builtin_amdgcn_readfirstlane(s_in[wave * KS8_CB + k][ii]);
        const uint32_t r = (x + 0x8000u) >> 16;  // round to 16 bits, ties up
        const uint32_t s0 = tab[(0 * 16 + ((r >> 12) & 15)) * KS_COLS];
        const uint32_t s1 = tab[(1 * 16 + ((r >> 8) & 15)) * KS_COLS];
        const uint32_t s2 = tab[(2 * 16 + ((r >> 4) & 15)) * KS_COLS];
        const uint32_t s3 = tab[(3 * 16 + (r & 15)) * KS_COLS];
        acc[k] -= (s0 + s1) + (s2 + s3);
      }
    }
  }

  if (!col_ok) return;
#pragma unroll
  for (int k = 0; k < KS8_CB; k++) {
    const int64_t c = cw + k;
    if (c >= B) break;
    int64_t dst = c;
    if (mode == kModeRelu) {
      const int64_t g = gate_begin + c;
      const int64_t v = g / (bits - 1), bit = g - v * (bits - 1);
      dst = v * bits + bit;
    }
    out[dst * row + col] = acc[k];
  }
}

__global__ __launch_bounds__(256) void relu_sign_kernel(uint32_t* __restrict__ y, int n, int32_t bits,
                                                        int64_t v_begin, int64_t count) {
  const int64_t idx = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (idx >= count * (n + 1)) return;
  const int64_t v = v_begin + idx / (n + 1);
  const int k = static_cast<int>(idx % (n + 1));
  y[(v * bits + bits - 1) * (n + 1) + k] = k == n ? 0u - kMu : 0u;
}

__global__ __launch_bounds__(256) void not_kernel(const uint32_t* __restrict__ in,
                                                  uint32_t* __restrict__ out, int64_t words) {
  const int64_t idx = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (idx < words) out[idx] = 0u - in[idx];
}

// Standalone exact negacyclic product c = d * b in Z_{2^32}[X]/(X^N+1), one
// polynomial per T threads, with the blind rotation's transform code.
template <int LOGN>
__global__ __launch_bounds__(256) void negacyclic_mul_kernel(const double* __restrict__ twf,
                                                             const double* __restrict__ twi,
                                                             const int32_t* __restrict__ d,
                                                             const uint32_t* __restrict__ b,
                                                             uint32_t* __restrict__ c, int64_t B) {
  using Lay = Layout<LOGN>;
  constexpr int N = Lay::N, E = Lay::E, T = Lay::T, CPB = 256 / T;
  __shared__ double s_scr[CPB * N];
  const int slot = threadIdx.x / T;
  const int t = threadIdx.x % T;
  int64_t k = static_cast<int64_t>(blockIdx.x) * CPB + slot;
  const bool active = k < B;
  if (!active) k = B - 1;
  double* scr = s_scr + slot * N;
  double xd[E], xh[E], xl[E];
  for (int e = 0; e < E; e++) {
    const int j = t + T * e;
    xd[e] = static_cast<double>(d[k * N + j]);
    const int32_t sv = static_cast<int32_t>(b[k * N + j]);
    const int32_t lo = ((sv + 32768) & 0xFFFF) - 32768;
    const int32_t hi = static_cast<int32_t>((static_cast<int64_t>(sv) - lo) / 65536);
    xh[e] = static_cast<double>(hi);
    xl[e] = static_cast<double>(lo);
  }
  ntt_forward<Lay, true, false>(xd, t, scr, twf, twf);
  ntt_forward<Lay, false, false>(xh, t, scr, twf, twf);
  ntt_forward<Lay, false, false>(xl, t, scr, twf, twf);
  // N^-1 mod P, folded into the products
  double ninv = 1.0;
  {
    // P = 1 mod 2^14, so N^-1 = P - (P - 1) / N
    ninv = kP - (kP - 1.0) / static_cast<double>(N);
  }
  for (int e = 0; e < E; e++) {
    const double de = mulmod(xd[e], ninv);
    xh[e] = reduce(mulmod(de, xh[e]));
    xl[e] = reduce(mulmod(de, xl[e]));
  }
  ntt_inverse<Lay, false>(xh, t, scr, twi, twi);
  ntt_inverse<Lay, false>(xl, t, scr, twi, twi);
  if (!active) return;
  for (int e = 0; e < E; e++) {
    const int j = t + T * e;
    c[k * N + j] = (low32(reduce(xh[e])) << 16) + low32(reduce(xl[e]));
  }
}

inline int launch_status(const char* what) {
  hipError_t err = hipGetLastError();
  if (err != hipSuccess) return fail(TFHE_EHIP, "%s launch failed: %s", what, hipGetErrorString(err));
  return TFHE_OK;
}

template <int LOGN>
int launch_br(const tfhe_eval_key* ek, const Workspace& ws, const uint32_t* testvec, int64_t B,
              hipStream_t st) {
  using C = BrCfg<LOGN>;
  const int64_t blocks = (B + C::CPB - 1) / C::CPB;
  hipLaunchKernelGGL(blind_rotate_kernel<LOGN>, dim3(static_cast<unsigned>(blocks)), dim3(C::THREADS), 0, st,
                     ek->bk_ntt, ek->tw_fwd, ek->tw_inv, ws.abar, testvec, ws.extract, ek->p.n,
                     ek->p.l, ek->p.bg_bit, B);
  return launch_status("blind_rotate_kernel");
}

template <int LOGN>
int launch_mul(const tfhe_eval_key* ek, const int32_t* d, const uint32_t* b, uint32_t* c, int64_t B,
               hipStream_t st) {
  constexpr int CPB = 256 / Layout<LOGN>::T;
  const int64_t blocks = (B + CPB - 1) / CPB;
  hipLaunchKernelGGL(negacyclic_mul_kernel<LOGN>, dim3(static_cast<unsigned>(blocks)), dim3(256), 0, st,
                     ek->tw_fwd, ek->tw_inv, d, b, c, B);
  return launch_status("negacyclic_mul_kernel");
}

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
                     static_cast<hipStream_t>(stream), a.mode, a.gate, a.ca, a.cb, ek->p.n, ek->p.N,
                     a.B, a.bits, a.gate_begin, ws.abar);
  return launch_status("prep_kernel");
}

int launch_blind_rotate(const tfhe_eval_key* ek, const Workspace& ws, const uint32_t* testvec,
                        int64_t B, void* stream) {
  hipStream_t st = static_cast<hipStream_t>(stream);
  switch (ek->p.N) {
    case 256: return launch_br<8>(ek, ws, testvec, B, st);
    case 512: return launch_br<9>(ek, ws, testvec, B, st);
    case 1024: return launch_br<10>(ek, ws, testvec, B, st);
    case 2048: return launch_br<11>(ek, ws, testvec, B, st);
    default: return fail(TFHE_EUNSUPPORTED, "N=%d has no blind-rotation kernel", ek->p.N);
  }
}

int launch_keyswitch(const tfhe_eval_key* ek, const uint32_t* in, uint32_t* out, int64_t B, int mode,
                     int32_t bits, int64_t gate_begin, void* stream) {
  const tfhe_params& p = ek->p;
  if (p.ks_t * (1 << p.ks_basebit) > KS_MAXROWS)
    return fail(TFHE_EUNSUPPORTED, "key switching with t * 2^basebit = %d > %d rows per coefficient",
                p.ks_t * (1 << p.ks_basebit), KS_MAXROWS);
  dim3 grid(static_cast<unsigned>((B + KS_CB - 1) / KS_CB), static_cast<unsigned>((p.n + 1 + KS_COLS - 1) / KS_COLS));
  hipStream_t st = static_cast<hipStream_t>(stream);
  if (p.ks_t == 8 && p.ks_basebit == 2) {
    dim3 g8(static_cast<unsigned>((B + KS8_WAVES * KS8_CB - 1) / (KS8_WAVES * KS8_CB)),
            static_cast<unsigned>((p.n + 1 + KS_COLS - 1) / KS_COLS));
    hipLaunchKernelGGL(keyswitch_t8b2_kernel, g8, dim3(256), 0, st, in, ek->ksk, out, p.n, p.N, B, mode,
                       bits, gate_begin);
  } else if (p.ks_t * (1 << p.ks_basebit) <= 32)
    hipLaunchKernelGGL((keyswitch_kernel<32, 0, 0>), grid, dim3(KS_COLS), 0, st, in, ek->ksk, out, p.n, p.N,
                       p.ks_t, p.ks_basebit, B, mode, bits, gate_begin);
  else
    hipLaunchKernelGGL((keyswitch_kernel<64, 0, 0>), grid, dim3(KS_COLS), 0, st, in, ek->ksk, out, p.n, p.N,
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

int launch_not(int32_t dim, const uint32_t* in, uint32_t* out, int64_t count, void* stream) {
  const int64_t words = count * (dim + 1);
  const int64_t blocks = (words + 255) / 256;
  hipLaunchKernelGGL(not_kernel, dim3(static_cast<unsigned>(blocks)), dim3(256), 0,
                     static_cast<hipStream_t>(stream), in, out, words);
  return launch_status("not_kernel");
}

int launch_negacyclic_mul(const tfhe_eval_key* ek, const int32_t* d, const uint32_t* b, uint32_t* c,
                          int64_t B, void* stream) {
  hipStream_t st = static_cast<hipStream_t>(stream);
  switch (ek->p.N) {
    case 256: return launch_mul<8>(ek, d, b, c, B, st);
    case 512: return launch_mul<9>(ek, d, b, c, B, st);
    case 1024: return launch_mul<10>(ek, d, b, c, B, st);
    case 2048: return launch_mul<11>(ek, d, b, c, B, st);
    default: return fail(TFHE_EUNSUPPORTED, "N=%d has no product kernel", ek->p.N);
  }
}

}  // namespace gt
