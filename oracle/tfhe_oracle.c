/*
 * TEST INFRASTRUCTURE ONLY -- CPU oracle of the TFHE activation path.
 * See tfhe_oracle.h for the scope.  Everything here is written for a reader
 * checking it against the mathematics, not for speed.
 *
 * Sources: the paper (Glyph, arXiv 1911.07101) names the operations --
 * TLWE / TRLWE / TRGSW samples and key switching (Section 3.2), SampleExtract
 * (Section 3.2, step 3 of the BGV-to-TFHE switch), gates with bootstrapping,
 * the free NOT gate and the forward ReLU unit (Section 3.1) -- and defers
 * their definitions to TFHE (Chillotti et al., J. Cryptology, cited in
 * Section 2).  The integer conventions (rounding, digit order, key-switch
 * table layout, generator) are the readings listed in the design notes.
 */
#include "tfhe_oracle.h"

#include <math.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

#define MU_GATE 0x20000000u /* 1/8 on the torus */

/* ------------------------------------------------------------------------
 * Counter-based generator.  SplitMix64 (Steele, Lea, Flood, OOPSLA 2014):
 * the k-th output of a stream whose state starts at x is mix(x + (k+1)*gamma).
 * A (seed, tag) pair selects the stream whose state is the tag-th output of
 * the stream started at seed; word idx of that stream is its idx-th output.
 * ---------------------------------------------------------------------- */
static uint64_t mix64(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBULL;
  return z ^ (z >> 31);
}

uint64_t oracle_stream_output(uint64_t state, uint64_t k) {
  return mix64(state + (k + 1) * 0x9E3779B97F4A7C15ULL);
}

uint64_t oracle_word(uint64_t seed, uint32_t tag, uint64_t idx) {
  return oracle_stream_output(oracle_stream_output(seed, tag), idx);
}

/* a uniform torus element is the high half of a word */
static uint32_t torus_word(uint64_t seed, uint32_t tag, uint64_t idx) {
  return (uint32_t)(oracle_word(seed, tag, idx) >> 32);
}

/* Box-Muller (cosine branch) on two 53-bit uniforms: u1 in (0,1], u2 in [0,1) */
double oracle_gauss(uint64_t seed, uint32_t tag, uint64_t idx) {
  uint64_t w1 = oracle_word(seed, tag, 2 * idx);
  uint64_t w2 = oracle_word(seed, tag, 2 * idx + 1);
  double u1 = (double)((w1 >> 11) + 1) * 0x1p-53;
  double u2 = (double)(w2 >> 11) * 0x1p-53;
  double r = sqrt(-2.0 * log(u1));
  double c = cos(6.283185307179586 * u2);
  return r * c;
}

/* rounded Gaussian torus noise of standard deviation alpha (torus units) */
uint32_t oracle_noise(uint64_t seed, uint32_t tag, uint64_t idx, double alpha) {
  double scale = alpha * 4294967296.0;
  double x = oracle_gauss(seed, tag, idx) * scale;
  long long e = llround(x);
  return (uint32_t)(uint64_t)e;
}

/* ------------------------------------------------------------------------
 * Ring arithmetic in Z_{2^32}[X]/(X^N+1)  (TRLWE plaintext ring, Section 3.2)
 * ---------------------------------------------------------------------- */

/* schoolbook negacyclic product: c_j = sum_{m<=j} a_m b_{j-m} - sum_{m>j} a_m b_{N+j-m} */
void oracle_negacyclic_mul(int32_t N, const uint32_t* a, const uint32_t* b, uint32_t* c) {
  for (int32_t j = 0; j < N; j++) {
    uint32_t acc = 0;
    for (int32_t m = 0; m <= j; m++) acc += a[m] * b[j - m];
    for (int32_t m = j + 1; m < N; m++) acc -= a[m] * b[N + j - m];
    c[j] = acc;
  }
}

/* out = X^e * p for e in [0, 2N): coefficient m moves to m+e; an index that
 * lands in [N, 2N) wraps to index - N with its sign flipped (X^N = -1) */
void oracle_rotate(int32_t N, const uint32_t* p, uint32_t e, uint32_t* out) {
  uint32_t twoN = 2u * (uint32_t)N;
  for (int32_t m = 0; m < N; m++) {
    uint32_t t = ((uint32_t)m + e) % twoN;
    if (t < (uint32_t)N)
      out[t] = p[m];
    else
      out[t - (uint32_t)N] = 0u - p[m];
  }
}

/* signed gadget decomposition of one torus element into l digits in
 * [-Bg/2, Bg/2), most significant first: x ~ sum_j d_j 2^(32 - j*bg_bit),
 * rounded to the nearest multiple of 2^(32 - l*bg_bit) (ties upward) */
void oracle_decompose(int32_t l, int32_t bg_bit, uint32_t x, int32_t* digits) {
  uint32_t half = 1u << (bg_bit - 1);
  uint32_t offset = 0;
  for (int32_t j = 1; j <= l; j++) offset += half << (32 - j * bg_bit);
  if (l * bg_bit < 32) offset += 1u << (31 - l * bg_bit);
  uint32_t y = x + offset;
  uint32_t mask = (1u << bg_bit) - 1u;
  for (int32_t j = 1; j <= l; j++)
    digits[j - 1] = (int32_t)((y >> (32 - j * bg_bit)) & mask) - (int32_t)half;
}

/* modulus switch of a torus element to Z_{2N}: round(x * 2N / 2^32) mod 2N */
uint32_t oracle_mod_switch(uint32_t x, int32_t N) {
  uint64_t twoN = 2u * (uint64_t)N;
  uint64_t v = ((uint64_t)x * twoN + 0x80000000ULL) >> 32;
  return (uint32_t)(v % twoN);
}

/* oracle_mod_switch of count words (a loop, for batches) */
void oracle_mod_switch_batch(const uint32_t* x, int64_t count, int32_t N, uint32_t* out) {
  for (int64_t k = 0; k < count; k++) out[k] = oracle_mod_switch(x[k], N);
}

/* ------------------------------------------------------------------------
 * Keys
 * ---------------------------------------------------------------------- */
int64_t oracle_bk_words(const oracle_params* p) {
  return (int64_t)p->n * 2 * p->l * 2 * p->N;
}

int64_t oracle_ksk_words(const oracle_params* p) {
  int64_t base = 1ll << p->ks_basebit;
  return (int64_t)p->N * p->ks_t * (base - 1) * (p->n + 1);
}

/* LWE encryption of one torus value: (a, <a,key> + mu + e) */
static void lwe_encrypt_one(int32_t dim, const uint32_t* key, uint32_t mu, uint64_t seed,
                            uint32_t tag_mask, uint64_t mask_index0, uint32_t tag_noise,
                            uint64_t noise_index, double alpha, uint32_t* ct) {
  uint32_t b = mu + oracle_noise(seed, tag_noise, noise_index, alpha);
  for (int32_t k = 0; k < dim; k++) {
    ct[k] = torus_word(seed, tag_mask, mask_index0 + (uint64_t)k);
    b += ct[k] * key[k];
  }
  ct[dim] = b;
}

/*
 * Key generation from one seed.
 *   s  : n binary LWE key bits;  S : N binary TRLWE key coefficients.
 *   bk : n TRGSW samples, BK_i = Z + s_i * H  (TRGSW encrypts integer
 *        polynomials, Section 3.2).  Row r = q*l + (j-1) of BK_i is the TRLWE
 *        sample (A, A*S + E) with s_i * 2^(32 - j*bg_bit) added to coefficient
 *        0 of polynomial q (q = 0: mask A, q = 1: body).  Layout
 *        [i][r][q][N].
 *   ksk: for each i < N, j < t and v in [1, base): the LWE sample under s of
 *        v * S_i * 2^(32 - (j+1)*basebit).  Layout [i][j][v-1][n+1].  There is
 *        no v = 0 entry (it would encrypt zero and is never read).
 */
void oracle_keygen(const oracle_params* p, uint64_t seed, uint32_t* s, uint32_t* S,
                   uint32_t* bk, uint32_t* ksk) {
  const int32_t n = p->n, N = p->N, l = p->l, L2 = 2 * p->l;
  for (int32_t i = 0; i < n; i++) s[i] = (uint32_t)(oracle_word(seed, ORACLE_TAG_LWE_KEY, (uint64_t)i) & 1u);
  for (int32_t j = 0; j < N; j++) S[j] = (uint32_t)(oracle_word(seed, ORACLE_TAG_RLWE_KEY, (uint64_t)j) & 1u);

#pragma omp parallel for schedule(dynamic)
  for (int64_t ir = 0; ir < (int64_t)n * L2; ir++) {
    int32_t i = (int32_t)(ir / L2), r = (int32_t)(ir % L2);
    uint32_t* A = bk + ir * 2 * N;
    uint32_t* Bp = A + N;
    uint64_t base_index = (uint64_t)ir * (uint64_t)N;
    for (int32_t m = 0; m < N; m++) A[m] = torus_word(seed, ORACLE_TAG_BK_MASK, base_index + (uint64_t)m);
    oracle_negacyclic_mul(N, A, S, Bp);
    for (int32_t m = 0; m < N; m++)
      Bp[m] += oracle_noise(seed, ORACLE_TAG_BK_NOISE, base_index + (uint64_t)m, p->alpha_bk);
    int32_t q = r / l, j = r % l + 1;
    uint32_t g = s[i] << (32 - j * p->bg_bit);
    if (q == 0) A[0] += g; else Bp[0] += g;
  }

  const int32_t t = p->ks_t, bb = p->ks_basebit, base = 1 << bb;
#pragma omp parallel for schedule(static)
  for (int64_t u = 0; u < (int64_t)N * t * (base - 1); u++) {
    int32_t i = (int32_t)(u / ((int64_t)t * (base - 1)));
    int32_t j = (int32_t)((u / (base - 1)) % t);
    uint32_t v = (uint32_t)(u % (base - 1)) + 1u;
    uint32_t msg = v * S[i] * (1u << (32 - (j + 1) * bb));
    lwe_encrypt_one(n, s, msg, seed, ORACLE_TAG_KSK_MASK, (uint64_t)u * (uint64_t)n,
                    ORACLE_TAG_KSK_NOISE, (uint64_t)u, p->alpha_ks, ksk + u * (n + 1));
  }
}

/* fresh LWE encryptions; ciphertext c uses generator index first_index + c */
void oracle_encrypt(int32_t dim, const uint32_t* key, uint64_t seed, double alpha,
                    const uint32_t* mu, int64_t first_index, int64_t count, uint32_t* ct) {
#pragma omp parallel for schedule(static)
  for (int64_t c = 0; c < count; c++) {
    uint64_t idx = (uint64_t)(first_index + c);
    lwe_encrypt_one(dim, key, mu[c], seed, ORACLE_TAG_ENC_MASK, idx * (uint64_t)dim,
                    ORACLE_TAG_ENC_NOISE, idx, alpha, ct + c * (dim + 1));
  }
}

/* decryption phase b - <a, key>  (Section 2: p = sigma(c, k)) */
void oracle_phase(int32_t dim, const uint32_t* key, const uint32_t* ct, int64_t count,
                  uint32_t* phase) {
  for (int64_t c = 0; c < count; c++) {
    const uint32_t* x = ct + c * (dim + 1);
    uint32_t v = x[dim];
    for (int32_t k = 0; k < dim; k++) v -= x[k] * key[k];
    phase[c] = v;
  }
}

/* ------------------------------------------------------------------------
 * Bootstrapping steps
 * ---------------------------------------------------------------------- */

/* linear pre-combination of two encrypted bits (true = +1/8, false = -1/8)
 * so that the bootstrap's sign test computes the gate */
void oracle_gate_combine(const oracle_params* p, int32_t gate, const uint32_t* ca,
                         const uint32_t* cb, uint32_t* out) {
  const int32_t n = p->n;
  int32_t wa, wb;
  uint32_t konst;
  switch (gate) {
    case ORACLE_NAND:  konst = MU_GATE;        wa = -1; wb = -1; break;
    case ORACLE_AND:   konst = 0u - MU_GATE;   wa = 1;  wb = 1;  break;
    case ORACLE_OR:    konst = MU_GATE;        wa = 1;  wb = 1;  break;
    case ORACLE_NOR:   konst = 0u - MU_GATE;   wa = -1; wb = -1; break;
    case ORACLE_XOR:   konst = 2u * MU_GATE;   wa = 2;  wb = 2;  break;
    case ORACLE_XNOR:  konst = 0u - 2u * MU_GATE; wa = -2; wb = -2; break;
    case ORACLE_ANDNY: konst = 0u - MU_GATE;   wa = -1; wb = 1;  break;
    case ORACLE_ANDYN: konst = 0u - MU_GATE;   wa = 1;  wb = -1; break;
    case ORACLE_ORNY:  konst = MU_GATE;        wa = -1; wb = 1;  break;
    case ORACLE_ORYN:  konst = MU_GATE;        wa = 1;  wb = -1; break;
    default: konst = 0; wa = 0; wb = 0; break;
  }
  for (int32_t k = 0; k <= n; k++)
    out[k] = (uint32_t)wa * ca[k] + (uint32_t)wb * cb[k] + (k == n ? konst : 0u);
}

/* NOT without bootstrapping (Section 3.1): negate every word */
void oracle_not(int32_t dim, const uint32_t* in, uint32_t* out, int64_t count) {
  for (int64_t k = 0; k < count * (dim + 1); k++) out[k] = 0u - in[k];
}

/*
 * One CMux step of the blind rotation: with D = X^abar * ACC - ACC,
 * ACC <- ACC + sum_r Dec(D)_r * BK_i[r], where Dec splits each coefficient of
 * D's mask polynomial into digit polynomials r = 0..l-1 and of its body into
 * r = l..2l-1, and each digit polynomial multiplies both polynomials of row r.
 */
void oracle_cmux(const oracle_params* p, const uint32_t* bk_i, uint32_t abar, uint32_t* acc) {
  const int32_t N = p->N, l = p->l, L2 = 2 * p->l;
  uint32_t* rot = (uint32_t*)malloc(sizeof(uint32_t) * (size_t)N);
  uint32_t* D = (uint32_t*)malloc(sizeof(uint32_t) * 2 * (size_t)N);
  uint32_t* dig = (uint32_t*)malloc(sizeof(uint32_t) * (size_t)L2 * (size_t)N);
  uint32_t* prod = (uint32_t*)malloc(sizeof(uint32_t) * (size_t)N);
  int32_t d[32];
  for (int32_t q = 0; q < 2; q++) {
    oracle_rotate(N, acc + q * N, abar, rot);
    for (int32_t m = 0; m < N; m++) D[q * N + m] = rot[m] - acc[q * N + m];
  }
  for (int32_t q = 0; q < 2; q++)
    for (int32_t m = 0; m < N; m++) {
      oracle_decompose(l, p->bg_bit, D[q * N + m], d);
      for (int32_t j = 0; j < l; j++) dig[(q * l + j) * N + m] = (uint32_t)d[j];
    }
  for (int32_t r = 0; r < L2; r++)
    for (int32_t q = 0; q < 2; q++) {
      oracle_negacyclic_mul(N, dig + r * N, bk_i + (r * 2 + q) * N, prod);
      for (int32_t m = 0; m < N; m++) acc[q * N + m] += prod[m];
    }
  free(rot); free(D); free(dig); free(prod);
}

/* blind rotation: ACC = (0, X^{-bbar} v), then one CMux per mask element;
 * the result is a TRLWE sample of X^{-phi} v with phi = bbar - sum abar_i s_i */
void oracle_blind_rotate(const oracle_params* p, const uint32_t* bk, const uint32_t* lwe,
                         const uint32_t* testvec, uint32_t* acc) {
  const int32_t n = p->n, N = p->N;
  uint32_t bbar = oracle_mod_switch(lwe[n], N);
  memset(acc, 0, sizeof(uint32_t) * (size_t)N);
  oracle_rotate(N, testvec, (2u * (uint32_t)N - bbar) % (2u * (uint32_t)N), acc + N);
  for (int32_t i = 0; i < n; i++) {
    uint32_t abar = oracle_mod_switch(lwe[i], N);
    oracle_cmux(p, bk + (int64_t)i * 2 * p->l * 2 * N, abar, acc);
  }
}

/* SampleExtract of coefficient 0 (Section 3.2, step 3): the LWE sample
 * (A_0, -A_{N-1}, ..., -A_1, B_0) under the key (S_0 .. S_{N-1}) */
void oracle_sample_extract(int32_t N, const uint32_t* acc, uint32_t* out) {
  out[0] = acc[0];
  for (int32_t j = 1; j < N; j++) out[j] = 0u - acc[N - j];
  out[N] = acc[N];
}

/*
 * LWE key switching (Section 3.2, "through key-switching") from dimension N
 * under S to dimension n under s: round each a'_i to t*basebit bits, split it
 * into t base-2^basebit digits (most significant first) and subtract the
 * table entry of every non-zero digit from (0, b').
 */
void oracle_keyswitch(const oracle_params* p, const uint32_t* ksk, const uint32_t* in,
                      uint32_t* out, int64_t count) {
  const int32_t n = p->n, N = p->N, t = p->ks_t, bb = p->ks_basebit;
  const int32_t base = 1 << bb, prec = t * bb;
  const uint32_t round = prec < 32 ? (1u << (31 - prec)) : 0u;
#pragma omp parallel for schedule(static)
  for (int64_t c = 0; c < count; c++) {
    const uint32_t* x = in + c * (N + 1);
    uint32_t* y = out + c * (n + 1);
    for (int32_t k = 0; k < n; k++) y[k] = 0;
    y[n] = x[N];
    for (int32_t i = 0; i < N; i++) {
      uint32_t r = prec == 32 ? x[i] : (x[i] + round) >> (32 - prec);
      for (int32_t j = 0; j < t; j++) {
        uint32_t v = (r >> ((t - 1 - j) * bb)) & (uint32_t)(base - 1);
        if (v == 0) continue;
        const uint32_t* row = ksk + (((int64_t)i * t + j) * (base - 1) + (v - 1)) * (n + 1);
        for (int32_t k = 0; k <= n; k++) y[k] -= row[k];
      }
    }
  }
}

/*
 * Test vector of a programmable bootstrap for a table of 2^msg_bits entries
 * (the paper's 3-bit table lookup, Section 3.1 "Forward Softmax").  Message m
 * is encoded as m * 2^(31 - msg_bits) (one padding bit).  Coefficient j holds
 * lut[floor((j + N/2^(msg_bits+1)) * 2^msg_bits / N)] when that index is in
 * range, otherwise -lut[0] (the negacyclic wrap of messages just below 0).
 */
void oracle_lut_testvec(int32_t N, int32_t msg_bits, const uint32_t* lut, uint32_t* tv) {
  const int64_t M = 1ll << msg_bits;
  const int32_t shift = 31 - msg_bits;
  for (int32_t j = 0; j < N; j++) {
    int64_t idx = (((int64_t)j + (int64_t)N / (2 * M)) * M) / N;
    tv[j] = idx < M ? lut[idx] << shift : 0u - (lut[0] << shift);
  }
}

/* bootstrap of one LWE sample up to (not including) key switching */
static void bootstrap_one(const oracle_params* p, const uint32_t* bk, const uint32_t* lwe,
                          const uint32_t* testvec, uint32_t* extracted) {
  uint32_t* acc = (uint32_t*)malloc(sizeof(uint32_t) * 2 * (size_t)p->N);
  oracle_blind_rotate(p, bk, lwe, testvec, acc);
  oracle_sample_extract(p->N, acc, extracted);
  free(acc);
}

void oracle_bootstrap_no_ks(const oracle_params* p, const uint32_t* bk, const uint32_t* in,
                            const uint32_t* testvec, uint32_t* out, int64_t count) {
#pragma omp parallel for schedule(dynamic)
  for (int64_t c = 0; c < count; c++)
    bootstrap_one(p, bk, in + c * (p->n + 1), testvec, out + c * (p->N + 1));
}

/* gate bootstrapping: combine, bootstrap with v = 1/8 everywhere, extract,
 * key switch back to dimension n */
void oracle_gate_bootstrap(const oracle_params* p, const uint32_t* bk, const uint32_t* ksk,
                           int32_t gate, const uint32_t* ca, const uint32_t* cb,
                           uint32_t* out, int64_t count) {
  const int32_t n = p->n, N = p->N;
  uint32_t* tv = (uint32_t*)malloc(sizeof(uint32_t) * (size_t)N);
  for (int32_t j = 0; j < N; j++) tv[j] = MU_GATE;
#pragma omp parallel for schedule(dynamic)
  for (int64_t c = 0; c < count; c++) {
    uint32_t* comb = (uint32_t*)malloc(sizeof(uint32_t) * (size_t)(n + 1));
    uint32_t* ext = (uint32_t*)malloc(sizeof(uint32_t) * (size_t)(N + 1));
    oracle_gate_combine(p, gate, ca + c * (n + 1), cb + c * (n + 1), comb);
    bootstrap_one(p, bk, comb, tv, ext);
    oracle_keyswitch(p, ksk, ext, out + c * (n + 1), 1);
    free(comb); free(ext);
  }
  free(tv);
}

void oracle_lut_bootstrap(const oracle_params* p, const uint32_t* bk, const uint32_t* ksk,
                          const uint32_t* in, const uint32_t* testvec, uint32_t* out,
                          int64_t count) {
  const int32_t n = p->n, N = p->N;
#pragma omp parallel for schedule(dynamic)
  for (int64_t c = 0; c < count; c++) {
    uint32_t* ext = (uint32_t*)malloc(sizeof(uint32_t) * (size_t)(N + 1));
    bootstrap_one(p, bk, in + c * (n + 1), testvec, ext);
    oracle_keyswitch(p, ksk, ext, out + c * (n + 1), 1);
    free(ext);
  }
}

/*
 * Forward ReLU unit (Section 3.1): for a value of `bits` bit-ciphertexts
 * (LSB first, the last one is the sign), output bit i < bits-1 is
 * AND(NOT sign, bit i) -- one bootstrapped gate -- and the output sign is a
 * trivial encryption of 0.  Gate g of the whole tensor is bit g % (bits-1) of
 * value g / (bits-1); out[c] receives gate gate_ids[c].
 */
void oracle_relu_gates(const oracle_params* p, const uint32_t* bk, const uint32_t* ksk,
                       const uint32_t* x, int32_t bits, const int64_t* gate_ids,
                       int64_t count, uint32_t* out) {
  const int32_t n = p->n;
  const int64_t stride = (int64_t)bits * (n + 1);
  uint32_t* sign = (uint32_t*)malloc(sizeof(uint32_t) * (size_t)count * (size_t)(n + 1));
  uint32_t* bit = (uint32_t*)malloc(sizeof(uint32_t) * (size_t)count * (size_t)(n + 1));
  for (int64_t c = 0; c < count; c++) {
    int64_t v = gate_ids[c] / (bits - 1), i = gate_ids[c] % (bits - 1);
    memcpy(sign + c * (n + 1), x + v * stride + (int64_t)(bits - 1) * (n + 1), sizeof(uint32_t) * (size_t)(n + 1));
    memcpy(bit + c * (n + 1), x + v * stride + i * (n + 1), sizeof(uint32_t) * (size_t)(n + 1));
  }
  oracle_gate_bootstrap(p, bk, ksk, ORACLE_ANDNY, sign, bit, out, count);
  free(sign); free(bit);
}

int oracle_threads(void) {
#ifdef _OPENMP
  return omp_get_max_threads();
#else
  return 1;
#endif
}

/* Threads of the calling thread's later parallel regions (n >= 1), for
 * timing the oracle on one core; the results do not depend on it. */
void oracle_set_threads(int n) {
#ifdef _OPENMP
  if (n >= 1) omp_set_num_threads(n);
#else
  (void)n;
#endif
}

/* ------------------------------------------------------------------------
 * TFHE side of the cryptosystem switch (Section 3.2: step 2, functional key
 * switching from T^N to T_N[X]; step 3, SampleExtract of K coefficients;
 * step 4, functional bootstrapping onto multiples of p^-r)
 * ---------------------------------------------------------------------- */

int64_t oracle_pks_words(const oracle_params* p) {
  return (int64_t)p->n * p->ks_t * ((1 << p->ks_basebit) - 1) * 2 * p->N;
}

/* Packing key: entry u = (i, j, v), v in [1, base), is a TRLWE sample (A, B)
 * under S of the constant polynomial v * s_i * 2^(32 - (j+1)*basebit):
 * A uniform, B = A * S + e + message in coefficient 0, e a rounded Gaussian
 * of deviation alpha_bk per coefficient. */
void oracle_packing_keygen(const oracle_params* p, uint64_t seed, const uint32_t* s,
                           const uint32_t* S, uint32_t* pks) {
  const int32_t n = p->n, N = p->N, t = p->ks_t, bb = p->ks_basebit, vals = (1 << bb) - 1;
#pragma omp parallel for schedule(dynamic)
  for (int64_t u = 0; u < (int64_t)n * t * vals; u++) {
    const int32_t i = (int32_t)(u / ((int64_t)t * vals));
    const int32_t j = (int32_t)((u / vals) % t);
    const uint32_t v = (uint32_t)(u % vals) + 1u;
    uint32_t* A = pks + u * 2 * N;
    uint32_t* B = A + N;
    const uint64_t base_index = (uint64_t)u * (uint64_t)N;
    for (int32_t m = 0; m < N; m++) A[m] = torus_word(seed, ORACLE_TAG_PKS_MASK, base_index + (uint64_t)m);
    oracle_negacyclic_mul(N, A, S, B);
    for (int32_t m = 0; m < N; m++)
      B[m] += oracle_noise(seed, ORACLE_TAG_PKS_NOISE, base_index + (uint64_t)m, p->alpha_bk);
    B[0] += v * s[i] * (1u << (32 - (j + 1) * bb));
  }
}

/* Functional key switching with the packing morphism (mu_0..mu_{Z-1}) ->
 * sum_z mu_z X^z: Z LWE samples (dimension n, key s) become one TRLWE
 * sample (A, B) under S whose phase is sum_z phase_z X^z, plus key noise
 * and the rounding of each a_{z,i} to t*basebit bits.  Start from
 * (0, sum_z b_z X^z) and, for every sample z, coefficient i and non-zero
 * digit v_{z,i,j} of the rounded a_{z,i} (most significant first),
 * subtract X^z times the key entry (i, j, v). */
void oracle_pack_keyswitch(const oracle_params* p, const uint32_t* pks, const uint32_t* lwe,
                           int32_t Z, uint32_t* out) {
  const int32_t n = p->n, N = p->N, t = p->ks_t, bb = p->ks_basebit, vals = (1 << bb) - 1;
  const int32_t prec = t * bb;
  const uint32_t round = prec < 32 ? (1u << (31 - prec)) : 0u;
  uint32_t* A = out;
  uint32_t* B = out + N;
  uint32_t* rot = (uint32_t*)malloc(sizeof(uint32_t) * 2 * (size_t)N);
  for (int32_t k = 0; k < 2 * N; k++) out[k] = 0;
  for (int32_t z = 0; z < Z; z++) {
    const uint32_t* c = lwe + (int64_t)z * (n + 1);
    B[z] += c[n];
    for (int32_t i = 0; i < n; i++) {
      const uint32_t r = prec == 32 ? c[i] : (c[i] + round) >> (32 - prec);
      for (int32_t j = 0; j < t; j++) {
        const uint32_t v = (r >> ((t - 1 - j) * bb)) & (uint32_t)vals;
        if (v == 0) continue;
        const uint32_t* e = pks + (((int64_t)i * t + j) * vals + (v - 1)) * 2 * N;
        oracle_rotate(N, e, (uint32_t)z, rot);
        oracle_rotate(N, e + N, (uint32_t)z, rot + N);
        for (int32_t k = 0; k < N; k++) {
          A[k] -= rot[k];
          B[k] -= rot[N + k];
        }
      }
    }
  }
  free(rot);
}

/* SampleExtract of coefficient idx of (A, B): the LWE sample under the key
 * (S_0 .. S_{N-1}) with a'_j = A_{idx-j} for j <= idx, -A_{N+idx-j} for
 * j > idx, and b' = B_idx (coefficient idx of B - A*S is b' - <a', S>) */
void oracle_sample_extract_at(int32_t N, const uint32_t* acc, int32_t idx, uint32_t* out) {
  for (int32_t j = 0; j < N; j++) out[j] = j <= idx ? acc[idx - j] : 0u - acc[N + idx - j];
  out[N] = acc[N + idx];
}

/* Test vector of a programmable bootstrap onto arbitrary torus values
 * (step 4 maps messages onto multiples of p^-r): as oracle_lut_testvec, with
 * values[m] (torus words) in place of lut[m] * 2^(31 - msg_bits). */
void oracle_torus_testvec(int32_t N, int32_t msg_bits, const uint32_t* values, uint32_t* tv) {
  const int64_t M = 1ll << msg_bits;
  for (int32_t j = 0; j < N; j++) {
    int64_t idx = (((int64_t)j + (int64_t)N / (2 * M)) * M) / N;
    tv[j] = idx < M ? values[idx] : 0u - values[0];
  }
}
