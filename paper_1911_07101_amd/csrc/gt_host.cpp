// Host-side (client) cryptography of the library: the counter-based generator,
// key generation, encryption, and the one-time conversion of the
// bootstrapping key into the transform domain of the blind-rotation kernels.
//
// Built without floating-point contraction: the Gaussian noise is computed by
// glibc's scalar log/cos/sqrt exactly as written, so that keys are a pure
// function of the seed.
#include <algorithm>
#include <cmath>
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

}  // namespace

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
// Exact integer arithmetic mod P on the host (128-bit products); the device
// reaches the same residues with its fp64 error-free arithmetic.
namespace {

constexpr uint64_t kPrimeU = 549755731969ull;  // the NTT prime (see gt_modp.hpp)

inline uint64_t mulmod_u64(uint64_t a, uint64_t b) {
  return static_cast<uint64_t>((static_cast<unsigned __int128>(a) * b) % kPrimeU);
}
inline uint64_t powmod_u64(uint64_t a, uint64_t e) {
  uint64_t r = 1;
  while (e) {
    if (e & 1) r = mulmod_u64(r, a);
    a = mulmod_u64(a, a);
    e >>= 1;
  }
  return r;
}
inline int ilog2(int x) {
  int r = 0;
  while ((1 << r) < x) r++;
  return r;
}
inline uint32_t bitrev(uint32_t x, int bits) {
  uint32_t r = 0;
  for (int b = 0; b < bits; b++) r |= ((x >> b) & 1u) << (bits - 1 - b);
  return r;
}
// psi: a primitive 2N-th root of unity.  7 is a quadratic non-residue mod P,
// so 7^((P-1)/2N) has order exactly 2N.
uint64_t root_2n(int N) { return powmod_u64(7, (kPrimeU - 1) / (2 * static_cast<uint64_t>(N))); }

struct TwiddleTable {
  std::vector<uint64_t> fwd;  // psi^brv(k)
  std::vector<uint64_t> inv;  // psi^-brv(k)
  explicit TwiddleTable(int N) : fwd(N), inv(N) {
    const int logn = ilog2(N);
    const uint64_t psi = root_2n(N);
    const uint64_t psi_inv = powmod_u64(psi, kPrimeU - 2);
    for (int k = 0; k < N; k++) {
      fwd[k] = powmod_u64(psi, bitrev(k, logn));
      inv[k] = powmod_u64(psi_inv, bitrev(k, logn));
    }
  }
};

// in-place forward negacyclic NTT (Cooley-Tukey, natural order in,
// bit-reversed order out); x holds residues in [0, P)
void ntt_forward_u64(std::vector<uint64_t>& x, const TwiddleTable& tw) {
  const int N = static_cast<int>(x.size());
  int k = 1;
  for (int len = N / 2; len >= 1; len >>= 1) {
    for (int start = 0; start < N; start += 2 * len, k++) {
      const uint64_t z = tw.fwd[k];
      for (int j = start; j < start + len; j++) {
        const uint64_t t = mulmod_u64(z, x[j + len]);
        x[j + len] = (x[j] + kPrimeU - t) % kPrimeU;
        x[j] = (x[j] + t) % kPrimeU;
      }
    }
  }
}

struct BkCtx {
  const tfhe_params* p;
  const uint32_t* bk;
  double* out;
  const TwiddleTable* tw;
};

void bk_convert_rows(int64_t begin, int64_t end, void* vctx) {
  const BkCtx& c = *static_cast<BkCtx*>(vctx);
  const int N = c.p->N;
  const int logn = ilog2(N);
  const int loge = log_values_per_thread(logn);
  const int E = 1 << loge, T = N >> loge;
  const uint64_t ninv = powmod_u64(static_cast<uint64_t>(N), kPrimeU - 2);
  std::vector<uint64_t> hi(N), lo(N);
  for (int64_t row = begin; row < end; row++) {  // row = (i * 2l + r) * 2 + q
    const uint32_t* src = c.bk + row * N;
    for (int m = 0; m < N; m++) {
      // signed 16-bit halves: coefficient = hi * 2^16 + lo, lo in [-2^15, 2^15)
      const int64_t sv = static_cast<int32_t>(src[m]);
      const int64_t l16 = ((sv + 32768) & 0xFFFF) - 32768;
      const int64_t h16 = (sv - l16) / 65536;
      hi[m] = static_cast<uint64_t>((h16 + static_cast<int64_t>(kPrimeU)) % static_cast<int64_t>(kPrimeU));
      lo[m] = static_cast<uint64_t>((l16 + static_cast<int64_t>(kPrimeU)) % static_cast<int64_t>(kPrimeU));
    }
    ntt_forward_u64(hi, *c.tw);
    ntt_forward_u64(lo, *c.tw);
    // output slots o = 2q (high half), 2q + 1 (low half) of [i][r][o][e][t]
    const int64_t ir = row / 2, q = row % 2;
    double* dst_hi = c.out + (ir * 4 + 2 * q) * N;
    double* dst_lo = dst_hi + N;
    // thread t's values e = 2h, 2h+1 are adjacent: layout [E/2][T][2]
    for (int t = 0; t < T; t++)
      for (int e = 0; e < E; e++) {
        const int j = e | (t << loge);  // transform-domain index held by (t, e)
        const int slot = (e >> 1) * 2 * T + 2 * t + (e & 1);
        dst_hi[slot] = static_cast<double>(mulmod_u64(hi[j], ninv));
        dst_lo[slot] = static_cast<double>(mulmod_u64(lo[j], ninv));
      }
  }
}

}  // namespace

void bk_to_transform_host(const tfhe_params& p, const uint32_t* bk, double* out) {
  TwiddleTable tw(p.N);
  BkCtx ctx{&p, bk, out, &tw};
  parallel_for(static_cast<int64_t>(p.n) * 2 * p.l * 2, 16, bk_convert_rows, &ctx);
}

void twiddles_host(int N, double* fwd, double* inv) {
  TwiddleTable tw(N);
  for (int k = 0; k < N; k++) {
    fwd[k] = static_cast<double>(tw.fwd[k]);
    inv[k] = static_cast<double>(tw.inv[k]);
  }
}

}  // namespace gt
