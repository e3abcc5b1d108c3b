// Host-side (client) cryptography of the library: the counter-based generator,
// key generation, encryption, and the one-time conversion of the
// bootstrapping key into the transform domain of the blind-rotation kernels.
//
// Built without floating-point contraction: the Gaussian noise is computed by
// glibc's scalar log/cos/sqrt exactly as written, so that keys are a pure
// function of the seed.
#include <algorithm>
#include <cmath>
#include <cstdint>
#include <cstring>
#include <thread>
#include <vector>

#include "gt_internal.h"
#include "gt_layout.hpp"

namespace gt {

// ---------------------------------------------------------------- generator
// SplitMix64 (Steele, Lea, Flood 2014): output k of the stream whose state is
// x is mix(x + (k + 1) * 0x9E3779B97F4A7C15).  Word idx under (seed, tag) is
// output idx of the stream whose state is output tag of the seed's stream.
static inline uint64_t splitmix_mix(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}
static inline uint64_t splitmix_at(uint64_t state, uint64_t k) {
  return splitmix_mix(state + (k + 1) * 0x9E3779B97F4A7C15ull);
}
uint64_t rand_word(uint64_t seed, uint32_t tag, uint64_t idx) {
  return splitmix_at(splitmix_at(seed, tag), idx);
}
static inline uint32_t rand_torus(uint64_t seed, uint32_t tag, uint64_t idx) {
  return static_cast<uint32_t>(rand_word(seed, tag, idx) >> 32);
}

// rounded Gaussian of standard deviation alpha (torus units), Box-Muller
// cosine branch on 53-bit uniforms u1 in (0, 1], u2 in [0, 1)
uint32_t rand_noise(uint64_t seed, uint32_t tag, uint64_t idx, double alpha) {
  const uint64_t w1 = rand_word(seed, tag, 2 * idx);
  const uint64_t w2 = rand_word(seed, tag, 2 * idx + 1);
  const double u1 = static_cast<double>((w1 >> 11) + 1) * 0x1p-53;
  const double u2 = static_cast<double>(w2 >> 11) * 0x1p-53;
  const double radius = std::sqrt(-2.0 * std::log(u1));
  const double cosine = std::cos(6.283185307179586 * u2);
  const double z = radius * cosine;
  const double scale = alpha * 4294967296.0;
  const double x = z * scale;
  return static_cast<uint32_t>(static_cast<uint64_t>(std::llround(x)));
}

// ---------------------------------------------------------------- threading
void parallel_for(int64_t count, int64_t grain, void (*fn)(int64_t, int64_t, void*), void* ctx) {
  unsigned hw = std::thread::hardware_concurrency();
  int64_t workers = std::max<int64_t>(1, std::min<int64_t>(hw ? hw : 1, 64));
  workers = std::min<int64_t>(workers, (count + grain - 1) / std::max<int64_t>(grain, 1));
  if (workers <= 1) {
    if (count > 0) fn(0, count, ctx);
    return;
  }
  std::vector<std::thread> pool;
  const int64_t chunk = (count + workers - 1) / workers;
  for (int64_t w = 0; w < workers; w++) {
    const int64_t b = w * chunk, e = std::min(count, b + chunk);
    if (b < e) pool.emplace_back(fn, b, e, ctx);
  }
  for (auto& th : pool) th.join();
}

// ---------------------------------------------------------------- keys
namespace {

struct KeygenCtx {
  tfhe_secret_key* sk;
};

// body = A * S + E for binary S: the sum of X^m * A over the set bits m of S
void trlwe_body(int N, const uint32_t* A, const uint32_t* S, uint32_t* body) {
  std::fill(body, body + N, 0u);
  for (int m = 0; m < N; m++) {
    if (!S[m]) continue;
    // X^m * A: coefficient k moves to k + m, wrapping with a sign flip
    for (int k = 0; k < N - m; k++) body[k + m] += A[k];
    for (int k = N - m; k < N; k++) body[k + m - N] -= A[k];
  }
}

void bk_rows(int64_t begin, int64_t end, void* vctx) {
  tfhe_secret_key& sk = *static_cast<KeygenCtx*>(vctx)->sk;
  const tfhe_params& p = sk.p;
  const int N = p.N, l = p.l, L2 = 2 * p.l;
  std::vector<uint32_t> body(N);
  for (int64_t ir = begin; ir < end; ir++) {
    const int i = static_cast<int>(ir / L2), r = static_cast<int>(ir % L2);
    uint32_t* A = sk.bk.data() + ir * 2 * N;
    uint32_t* Bp = A + N;
    const uint64_t base = static_cast<uint64_t>(ir) * static_cast<uint64_t>(N);
    for (int m = 0; m < N; m++) A[m] = rand_torus(sk.seed, kTagBkMask, base + m);
    trlwe_body(N, A, sk.S.data(), body.data());
    for (int m = 0; m < N; m++) Bp[m] = body[m] + rand_noise(sk.seed, kTagBkNoise, base + m, p.alpha_bk);
    const int q = r / l, j = r % l + 1;
    const uint32_t g = sk.s[i] << (32 - j * p.bg_bit);
    (q == 0 ? A : Bp)[0] += g;
  }
}

void lwe_encrypt(const std::vector<uint32_t>& key, uint32_t mu, uint64_t seed, uint32_t tag_mask,
                 uint64_t mask0, uint32_t tag_noise, uint64_t noise_idx, double alpha,
                 uint32_t* ct) {
  const int dim = static_cast<int>(key.size());
  uint32_t b = mu + rand_noise(seed, tag_noise, noise_idx, alpha);
  for (int k = 0; k < dim; k++) {
    ct[k] = rand_torus(seed, tag_mask, mask0 + k);
    b += ct[k] * key[k];
  }
  ct[dim] = b;
}

void ksk_rows(int64_t begin, int64_t end, void* vctx) {
  tfhe_secret_key& sk = *static_cast<KeygenCtx*>(vctx)->sk;
  const tfhe_params& p = sk.p;
  const int n = p.n, t = p.ks_t, bb = p.ks_basebit, vals = (1 << bb) - 1;
  for (int64_t u = begin; u < end; u++) {
    const int i = static_cast<int>(u / (static_cast<int64_t>(t) * vals));
    const int j = static_cast<int>((u / vals) % t);
    const uint32_t v = static_cast<uint32_t>(u % vals) + 1u;
    const uint32_t msg = v * sk.S[i] * (1u << (32 - (j + 1) * bb));
    lwe_encrypt(sk.s, msg, sk.seed, kTagKskMask, static_cast<uint64_t>(u) * n, kTagKskNoise,
                static_cast<uint64_t>(u), p.alpha_ks, sk.ksk.data() + u * (n + 1));
  }
}

// packing key entry u = (i, j, v): TRLWE sample under S of the constant
// polynomial v * s_i * 2^(32 - (j+1)*basebit)
void pks_rows(int64_t begin, int64_t end, void* vctx) {
  tfhe_secret_key& sk = *static_cast<KeygenCtx*>(vctx)->sk;
  const tfhe_params& p = sk.p;
  const int N = p.N, t = p.ks_t, bb = p.ks_basebit, vals = (1 << bb) - 1;
  std::vector<uint32_t> body(N);
  for (int64_t u = begin; u < end; u++) {
    const int i = static_cast<int>(u / (static_cast<int64_t>(t) * vals));
    const int j = static_cast<int>((u / vals) % t);
    const uint32_t v = static_cast<uint32_t>(u % vals) + 1u;
    uint32_t* A = sk.pks.data() + u * 2 * N;
    uint32_t* Bp = A + N;
    const uint64_t base = static_cast<uint64_t>(u) * static_cast<uint64_t>(N);
    for (int m = 0; m < N; m++) A[m] = rand_torus(sk.seed, kTagPksMask, base + m);
    trlwe_body(N, A, sk.S.data(), body.data());
    for (int m = 0; m < N; m++) Bp[m] = body[m] + rand_noise(sk.seed, kTagPksNoise, base + m, p.alpha_bk);
    Bp[0] += v * sk.s[i] * (1u << (32 - (j + 1) * bb));
  }
}

}  // namespace

void packing_keygen_host(tfhe_secret_key& sk) {
  const tfhe_params& p = sk.p;
  const int64_t entries = static_cast<int64_t>(p.n) * p.ks_t * ((1 << p.ks_basebit) - 1);
  sk.pks.assign(static_cast<size_t>(entries) * 2 * p.N, 0u);
  KeygenCtx ctx{&sk};
  parallel_for(entries, 8, pks_rows, &ctx);
}

void keygen_host(tfhe_secret_key& sk) {
  const tfhe_params& p = sk.p;
  sk.s.resize(p.n);
  sk.S.resize(p.N);
  for (int i = 0; i < p.n; i++) sk.s[i] = static_cast<uint32_t>(rand_word(sk.seed, kTagLweKey, i) & 1u);
  for (int j = 0; j < p.N; j++) sk.S[j] = static_cast<uint32_t>(rand_word(sk.seed, kTagRlweKey, j) & 1u);
  sk.bk.assign(static_cast<size_t>(p.n) * 2 * p.l * 2 * p.N, 0u);
  const int64_t vals = (1 << p.ks_basebit) - 1;
  sk.ksk.assign(static_cast<size_t>(p.N) * p.ks_t * vals * (p.n + 1), 0u);
  KeygenCtx ctx{&sk};
  parallel_for(static_cast<int64_t>(p.n) * 2 * p.l, 8, bk_rows, &ctx);
  parallel_for(static_cast<int64_t>(p.N) * p.ks_t * vals, 256, ksk_rows, &ctx);
}

namespace {
struct EncCtx {
  const tfhe_secret_key* sk;
  uint64_t seed;
  const uint32_t* mu;
  int64_t first;
  uint32_t* ct;
};
void enc_rows(int64_t begin, int64_t end, void* vctx) {
  const EncCtx& c = *static_cast<EncCtx*>(vctx);
  const int n = c.sk->p.n;
  for (int64_t k = begin; k < end; k++) {
    const uint64_t idx = static_cast<uint64_t>(c.first + k);
    lwe_encrypt(c.sk->s, c.mu[k], c.seed, kTagEncMask, idx * n, kTagEncNoise, idx, c.sk->p.alpha_lwe,
                c.ct + k * (n + 1));
  }
}
}  // namespace

void encrypt_host(const tfhe_secret_key& sk, uint64_t seed, const uint32_t* mu, int64_t first,
                  int64_t count, uint32_t* ct) {
  EncCtx ctx{&sk, seed, mu, first, ct};
  parallel_for(count, 1024, enc_rows, &ctx);
}

// ------------------------------------------------- transform-domain key
// The ring product is computed as a complex transform of the folded
// polynomial z_j = a_j + i a_{j+n} (n = N/2) over C[X]/(X^n - i): R[X]/(X^N+1)
// and C[X]/(X^n - i) are isomorphic as real algebras (X^n = i is a square
// root of X^N = -1), and z evaluated at the n roots of X^n - i gives a at
// those roots.  The Cooley-Tukey tree splits node k, X^m - zeta^R(k) with
// zeta = exp(i pi / N), into X^(m/2) -/+ zeta^(R(k)/2); R(1) = n and, since
// -1 = zeta^N, R(2k) = R(k)/2, R(2k+1) = R(k)/2 + N.  The butterfly of node k
// multiplies by tw[k] = zeta^(R(k)/2).
//
// The host builds the twiddles and the transformed key in long double and
// rounds once to double.
namespace {

inline int ilog2(int x) {
  int r = 0;
  while ((1 << r) < x) r++;
  return r;
}

// exponents e(k) = R(k)/2 of the twiddles, k in [1, n)
std::vector<long> twiddle_exponents(int N) {
  const int n = N / 2;
  std::vector<long> R(2 * static_cast<size_t>(n), 0), e(n, 0);
  R[1] = n;
  for (int k = 1; k < n; k++) {
    R[2 * k] = R[k] / 2;
    R[2 * k + 1] = R[k] / 2 + N;
  }
  for (int k = 1; k < n; k++) e[k] = R[k] / 2;
  return e;
}

struct ComplexL {
  long double re, im;
};

std::vector<ComplexL> twiddles_long(int N) {
  const int n = N / 2;
  const std::vector<long> ex = twiddle_exponents(N);
  const long double pi = 3.141592653589793238462643383279502884L;
  std::vector<ComplexL> tw(n);
  tw[0] = {1.0L, 0.0L};
  for (int k = 1; k < n; k++) {
    const long double ang = pi * static_cast<long double>(ex[k]) / static_cast<long double>(N);
    tw[k] = {cosl(ang), sinl(ang)};
  }
  return tw;
}

// in-place forward transform (Cooley-Tukey, natural order in, tree order out)
void transform_forward_long(std::vector<ComplexL>& x, const std::vector<ComplexL>& tw) {
  const int n = static_cast<int>(x.size());
  int k = 1;
  for (int len = n / 2; len >= 1; len >>= 1) {
    for (int start = 0; start < n; start += 2 * len, k++) {
      const ComplexL w = tw[k];
      for (int j = start; j < start + len; j++) {
        const ComplexL v = x[j + len];
        const ComplexL t = {w.re * v.re - w.im * v.im, w.re * v.im + w.im * v.re};
        x[j + len] = {x[j].re - t.re, x[j].im - t.im};
        x[j] = {x[j].re + t.re, x[j].im + t.im};
      }
    }
  }
}

// split a signed 32-bit coefficient into `parts` signed pieces of
// 32/parts-bit weight: value = sum_s piece_s * 2^(s * shift)
void split_coefficient(int32_t v, int parts, int64_t* piece) {
  const int shift = key_part_shift(parts);
  int64_t rest = v;
  for (int s = 0; s < parts; s++) {
    if (s == parts - 1) {
      piece[s] = rest;
      break;
    }
    const int64_t half = int64_t{1} << (shift - 1);
    const int64_t mask = (int64_t{1} << shift) - 1;
    const int64_t low = ((rest + half) & mask) - half;
    piece[s] = low;
    rest = (rest - low) >> shift;
  }
}

struct BkCtx {
  int N;
  int parts;
  const uint32_t* bk;
  double* out;
  const std::vector<ComplexL>* tw;
};

void bk_convert_rows(int64_t begin, int64_t end, void* vctx) {
  const BkCtx& c = *static_cast<BkCtx*>(vctx);
  const int N = c.N, n = N / 2;
  const int S = c.parts;
  const int loge = ring_log_e(S);
  const int E = 1 << loge, T = n >> loge;
  std::vector<std::vector<ComplexL>> z(S, std::vector<ComplexL>(n));
  int64_t piece_lo[4], piece_hi[4];
  for (int64_t row = begin; row < end; row++) {  // row = (TRLWE row) * 2 + q
    const uint32_t* src = c.bk + row * N;
    for (int j = 0; j < n; j++) {
      split_coefficient(static_cast<int32_t>(src[j]), S, piece_lo);
      split_coefficient(static_cast<int32_t>(src[j + n]), S, piece_hi);
      for (int s = 0; s < S; s++)
        z[s][j] = {static_cast<long double>(piece_lo[s]), static_cast<long double>(piece_hi[s])};
    }
    const int64_t ir = row / 2, q = row % 2;
    for (int s = 0; s < S; s++) {
      transform_forward_long(z[s], *c.tw);
      // output slot o = q * S + s of [i][r][o][e][t] (complex), scaled by 1/n
      double* dst = c.out + ((ir * 2 * S + q * S + s) * static_cast<int64_t>(n)) * 2;
      for (int t = 0; t < T; t++)
        for (int e = 0; e < E; e++) {
          const int j = e | (t << loge);  // point held by (t, e) after the forward transform
          const int slot = e * T + t;
          dst[2 * slot] = static_cast<double>(z[s][j].re / static_cast<long double>(n));
          dst[2 * slot + 1] = static_cast<double>(z[s][j].im / static_cast<long double>(n));
        }
    }
  }
}

}  // namespace

int key_part_shift(int parts) { return parts == 2 ? 16 : 11; }

int key_part_bits(int parts) { return parts == 2 ? 15 : 10; }

// Worst-case error of one output coefficient of z = sum_{r<R} x_r * y_r
// (x_r the digits, |x| <= D; y_r one key part, |y| <= Y = 2^b; in the
// external product R = 2l and D = Bg/2)
// computed as the library does: X_r = fl(F x_r) on the device, K_r = the
// key's transform F y_r / n computed in long double and rounded once,
// P = fl(sum_r X_r K_r) pointwise, z^ = fl(G P) with G the unscaled inverse.
// F is a radix-2 transform of n = N/2 points with F/sqrt(n) unitary, and
// (Higham, Accuracy and Stability of Numerical Algorithms, Thm 24.2)
// ||fl(F v) - F v||_2 <= eps ||F v||_2, eps = m eta / (1 - m eta),
// eta = mu + gamma4 (sqrt2 + mu), m = log2 n, mu <= u the twiddle error.
// G is a radix-2 cyclic inverse transform (m stages) followed by a diagonal
// of unit-modulus twists, one more multiplication stage of the same kind,
// so ||fl(G P) - G P||_2 <= eps' ||G P||_2, eps' = (m+1) eta / (1 - (m+1) eta).
// Then, with ||.||_1 of a Hadamard product bounded by Cauchy-Schwarz,
//   ||z^ - z||_inf <= ||fl(G P) - G P||_2 + ||G (P - P_exact)||_inf
//                  <= eps' (||z||_2 + sqrt(n) E_P) + E_P,
//   E_P = ||P - P_exact||_1
//       <= R [eps (1 + u2) + u2 + gamma_2R (1 + eps)(1 + u2)] ||x||_2 ||y||_2
// (forward error of the digits; key rounding u2 = 2u; a complex product-sum
// of R terms with two roundings per term and component), ||x||_2 <= D sqrt N,
// ||y||_2 <= Y sqrt N, and ||z||_2 <= R ||x||_1 ||y||_2 <= R D N Y sqrt N
// (Young's inequality for the negacyclic convolution).  The device's
// butterflies (a = u + w v in four FMAs, b = 2u - a in two, in both
// directions) have a per-stage relative error of at most mu + 3.02u to first
// order, below the theorem's eta, so eta covers them; the twist is one
// complex product per point, also within eta.
double transform_error_bound_rows(int ring_n, int parts, double R, double D) {
  const double u = std::ldexp(1.0, -53), u2 = 2 * u;
  const int n = ring_n / 2;
  const double m = ilog2(n);
  const double gamma4 = 4 * u / (1 - 4 * u);
  const double eta = u + gamma4 * (std::sqrt(2.0) + u);
  const double eps = m * eta / (1 - m * eta);
  const double eps_inv = (m + 1) * eta / (1 - (m + 1) * eta);
  const double g2R = 2 * R * u / (1 - 2 * R * u);
  const double Y = std::ldexp(1.0, key_part_bits(parts));
  const double N = ring_n, sN = std::sqrt(N);
  const double x1 = D * N, x2 = D * sN, y2 = Y * sN;
  const double z2 = R * x1 * y2;
  const double ep = R * (eps * (1 + u2) + u2 + g2R * (1 + eps) * (1 + u2)) * x2 * y2;
  return eps_inv * (z2 + std::sqrt(static_cast<double>(n)) * ep) + ep;
}

double transform_error_bound(const tfhe_params& p, int parts) {
  return transform_error_bound_rows(p.N, parts, 2.0 * p.l, std::ldexp(1.0, p.bg_bit - 1));
}

int key_parts(const tfhe_params& p) {
  for (int parts = 2; parts <= 3; parts++)
    if (transform_error_bound(p, parts) <= 0.125) return parts;
  return 0;
}

void trlwe_rows_to_transform_host(int N, int parts, int64_t rows, const uint32_t* src, double* out) {
  const std::vector<ComplexL> tw = twiddles_long(N);
  BkCtx ctx{N, parts, src, out, &tw};
  parallel_for(rows * 2, 16, bk_convert_rows, &ctx);
}

void bk_to_transform_host(const tfhe_params& p, int parts, const uint32_t* bk, double* out) {
  trlwe_rows_to_transform_host(p.N, parts, static_cast<int64_t>(p.n) * 2 * p.l, bk, out);
}

bool ks_uses_mfma(const tfhe_params& p) { return p.ks_t == 8 && p.ks_basebit == 2; }

int64_t ksk_mfma_bytes(const tfhe_params& p) { return static_cast<int64_t>(p.N) / 4 * 3 * ksk_mfma_nb(p) * 4 * 64 * 16; }

namespace {
struct KmfCtx {
  const tfhe_params* p;
  const uint32_t* ksk;
  int8_t* out;
};

// groups [begin, end) of four input coefficients
void kmf_rows(int64_t begin, int64_t end, void* vctx) {
  const KmfCtx& c = *static_cast<KmfCtx*>(vctx);
  const int n = c.p->n;
  const int64_t row = n + 1, nbs = ksk_mfma_nb(*c.p);
  for (int64_t grp = begin; grp < end; grp++)
    for (int m = 0; m < 3; m++) {
      const int64_t t = 3 * grp + m;
      for (int64_t nb = 0; nb < nbs; nb++)
        for (int l = 0; l < 64; l++) {
          const int64_t col = nb * 32 + l % 32;
          const int h = l / 32;
          for (int s = 0; s < 16; s++) {
            const int q = m < 2 ? h + 2 * m : h + 2 * (s / 8);
            const int v = m < 2 ? 1 + s / 8 : 3;
            const int w = m < 2 ? (s / 4) % 2 : (s % 8) / 4;
            const int j = 7 - s % 4 - 4 * w;
            const int64_t i = 4 * grp + q;
            int64_t x = col <= n ? c.ksk[((i * 8 + j) * 3 + (v - 1)) * row + col] : 0;
            // signed base-256 digits, the top one taken mod 256 (2^32 = 0)
            for (int beta = 0; beta < 4; beta++) {
              const int64_t b = ((x & 255) ^ 128) - 128;
              x = (x - b) >> 8;
              c.out[(((t * nbs + nb) * 4 + beta) * 64 + l) * 16 + s] = static_cast<int8_t>(b);
            }
          }
        }
    }
}
}  // namespace

void ksk_to_mfma_host(const tfhe_params& p, const uint32_t* ksk, int8_t* out) {
  KmfCtx ctx{&p, ksk, out};
  parallel_for(p.N / 4, 2, kmf_rows, &ctx);
}

void twiddles_host(int N, double* tw) {
  const int n = N / 2;
  const long double pi = 3.141592653589793238462643383279502884L;
  auto put = [tw](int slot, long double re, long double im) {
    tw[2 * slot] = static_cast<double>(re);
    tw[2 * slot + 1] = static_cast<double>(im);
  };
  // [0, n): the forward's tree twiddles
  const std::vector<ComplexL> t = twiddles_long(N);
  for (int k = 0; k < n; k++) put(k, t[k].re, t[k].im);
  // [n, 2n - 1): inverse stage s, entry c < 2^s at n + 2^s - 1 + c:
  // e^{-2 pi i c / 2^(s+1)}; slot 2n - 1 is unused
  for (int half = 1; half < n; half *= 2)
    for (int c = 0; c < half; c++) {
      const long double ang = -pi * static_cast<long double>(c) / static_cast<long double>(half);
      put(n + half - 1 + c, cosl(ang), sinl(ang));
    }
  put(2 * n - 1, 1.0L, 0.0L);
  // [2n, 3n): the twist zeta0^{-k} = e^{-i pi k / N} of output k
  for (int k = 0; k < n; k++) {
    const long double ang = -pi * static_cast<long double>(k) / static_cast<long double>(N);
    put(2 * n + k, cosl(ang), sinl(ang));
  }
}

}  // namespace gt
