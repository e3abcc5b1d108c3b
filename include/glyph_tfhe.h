/*
 * glyph_tfhe.h -- C ABI of the MI355X TFHE activation library.
 *
 * Glyph (Lou, Feng, Fox, Jiang; arXiv 1911.07101) evaluates the nonlinear
 * activations of encrypted DNN training with TFHE: a ReLU is one NOT without
 * bootstrapping plus one bootstrapped AND per lower bit (Section 3.1,
 * "Forward ReLU"), and table lookups are TFHE bootstraps (Section 3.1,
 * "Forward Softmax"; functional bootstrapping in the cryptosystem switch,
 * Section 3.2).  One gate bootstrap is: modulus switch of the LWE sample to
 * Z_{2N}, blind rotation by n CMux external products (TRGSW key x TRLWE
 * accumulator, gadget-decomposed, negacyclic in Z_{2^32}[X]/(X^N+1)),
 * SampleExtract (Section 3.2, step 3) and LWE key switching (Section 3.2).
 *
 * Conventions (all calls):
 *   - Torus elements are uint32_t; value x stands for x / 2^32; every torus
 *     operation is mod 2^32.
 *   - An LWE sample of dimension d is d+1 consecutive words [a_0 .. a_{d-1}, b];
 *     a batch is row-major [count][d+1] with no padding.
 *   - An encrypted bit is +1/8 (true) or -1/8 (false) on the torus.
 *   - Every call returns 0 (TFHE_OK) or a negative TFHE_E* code;
 *     tfhe_last_error() gives a message for the calling thread's last failure.
 *   - "Client-side" calls (key generation, encryption, decryption, key export)
 *     work on host memory and hold the secret key.  "Server-side" calls
 *     (bootstraps, key switching, ReLU) take device pointers, enqueue work on
 *     the given HIP stream (NULL = the legacy default stream) and return
 *     without synchronising; they never allocate, copy to or from the host, or
 *     read secret key material (the stage check tfhe_debug_cmux_batch alone
 *     uploads a caller-given key row and waits for its stream).
 *   - Inputs, outputs and the workspace of one server-side call must not
 *     overlap (TFHE_EINVAL otherwise).  Concurrent calls on different streams
 *     are safe when they use different workspaces.
 *   - A server-side call launches one-dimensional grids with one work-item per
 *     word of its widest buffer, and a grid dimension holds at most 2^32 - 1
 *     work-items: a call whose count times words per item exceeds 2^32 - 256
 *     returns TFHE_EINVAL before any launch (a bootstrap call: B * (n + 1),
 *     i.e. at most 6.8 million ciphertexts at n = 630).  Split larger batches;
 *     the ReLU units take gate windows for this.
 */
#ifndef GLYPH_TFHE_H
#define GLYPH_TFHE_H
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum {
  TFHE_OK = 0,
  TFHE_EINVAL = -1,       /* bad argument: NULL pointer, negative count, unknown gate,
                             workspace too small, misaligned pointer, a count too
                             large for one launch */
  TFHE_EUNSUPPORTED = -2, /* parameter set outside what the kernels are built for */
  TFHE_ENOMEM = -3,       /* host or device allocation failed (key generation only) */
  TFHE_EHIP = -4,         /* a HIP runtime call or kernel launch failed */
  TFHE_EDEVICE = -5       /* the device is not a gfx950 GPU or does not exist */
};

/* TFHE parameters with k = 1 (one mask polynomial).
 * Supported: N in {256, 512, 1024, 2048}; 1 <= n <= 4096; 2 <= bg_bit,
 * l * bg_bit <= 32; ks_t * ks_basebit <= 32 and ks_t * 2^ks_basebit <= 64 (the
 * key rows of one coefficient fit the key-switch kernel's LDS stage).  The
 * ring products are computed with a floating-point transform and rounded;
 * the parameters must keep its worst-case error below 1/8 with the key split
 * into 16-bit or 11-bit signed parts (it holds for all the parameter sets
 * the library is tested on, with 16-bit parts; it fails for example at
 * N = 2048 with bg_bit = 24); otherwise key generation returns
 * TFHE_EUNSUPPORTED. */
typedef struct {
  int32_t n;          /* LWE dimension */
  int32_t N;          /* TRLWE ring degree */
  int32_t l;          /* bootstrapping-key gadget length */
  int32_t bg_bit;     /* log2 of the gadget base */
  int32_t ks_t;       /* key-switching digits */
  int32_t ks_basebit; /* log2 of the key-switching base */
  double alpha_lwe;   /* std. dev. of fresh-encryption noise (torus units) */
  double alpha_bk;    /* std. dev. of bootstrapping-key noise */
  double alpha_ks;    /* std. dev. of key-switching-key noise */
} tfhe_params;

typedef struct tfhe_secret_key tfhe_secret_key; /* host only: LWE key s, TRLWE key S */
typedef struct tfhe_eval_key tfhe_eval_key;     /* device: bootstrapping + key-switching keys */

/* two-input gates with bootstrapping (TFHE's gate set; the paper's ReLU uses
 * ANDNY = AND(NOT a, b), Section 3.1) */
enum tfhe_gate {
  TFHE_NAND = 0, TFHE_AND = 1, TFHE_OR = 2, TFHE_NOR = 3, TFHE_XOR = 4, TFHE_XNOR = 5,
  TFHE_ANDNY = 6, TFHE_ANDYN = 7, TFHE_ORNY = 8, TFHE_ORYN = 9
};

const char* tfhe_strerror(int rc);
const char* tfhe_last_error(void);

/* ---------------------------------------------------------------- keys ---- */

/* Generate all keys deterministically from `seed` (Section 2: the user holds
 * the private key, the server evaluates with public material only).
 *   s (n bits), S (N bits): binary secret keys.
 *   Bootstrapping key: n TRGSW samples of s_i under S, rows r = q*l + (j-1)
 *     carrying s_i * 2^(32 - j*bg_bit) on polynomial q (0 = mask, 1 = body).
 *   Key-switching key: LWE samples under s of v * S_i * 2^(32-(j+1)*basebit)
 *     for i < N, j < ks_t, v in [1, 2^basebit).
 * The evaluation key is uploaded to `device` (precomputed into the transform
 * domain of the blind-rotation kernels); the secret key stays on the host.
 * Both handles are owned by the caller and released with the *_free calls. */
int tfhe_keygen_from_seed(const tfhe_params* params, uint64_t seed, int device,
                          tfhe_secret_key** sk_out, tfhe_eval_key** ek_out);

/* The two halves of tfhe_keygen_from_seed: the client-side key generation
 * (host only, no device needed) and the upload of the evaluation key derived
 * from it to `device`.  tfhe_keygen_from_seed(p, seed, dev, &sk, &ek) equals
 * tfhe_secret_keygen(p, seed, &sk) followed by tfhe_eval_key_upload(sk, dev, &ek). */
int tfhe_secret_keygen(const tfhe_params* params, uint64_t seed, tfhe_secret_key** sk_out);
int tfhe_eval_key_upload(const tfhe_secret_key* sk, int device, tfhe_eval_key** ek_out);
void tfhe_secret_key_free(tfhe_secret_key* sk);

/* Exactness of the ring products (host only, no device needed).  The blind
 * rotation multiplies digit polynomials by the key in a floating-point
 * transform and rounds the results; the key's coefficients are split into
 * `*key_parts` signed parts (2 of 16 bits or 3 of 11 bits) so that the
 * worst-case transform error of every output coefficient, `*error_bound`,
 * stays below 1/8 (the rounding then returns the exact integer).  Returns
 * TFHE_EUNSUPPORTED (with the 3-part bound) when no split achieves it. */
int tfhe_transform_error_bound(const tfhe_params* params, int32_t* key_parts, double* error_bound);
void tfhe_eval_key_free(tfhe_eval_key* ek);
int tfhe_eval_key_params(const tfhe_eval_key* ek, tfhe_params* out);

/* Copy keys out (host buffers; any pointer may be NULL to skip it): the
 * private keys k of Section 2 ("FHE": the user keeps them) and the public
 * evaluation material derived from them -- the TRGSW bootstrapping key and
 * the key-switching key of Section 3.2 -- so that a client, or a check, can
 * recompute any step on its own.
 *   s [n], S [N] (0/1 words); bk [n][2l][2][N] (coefficient domain, rows as
 *   in tfhe_keygen_from_seed); ksk [N][ks_t][2^basebit - 1][n+1].
 * Each buffer must hold the stated number of words; the call reads only the
 * secret key handle and returns TFHE_EINVAL if it is NULL. */
int tfhe_export_keys(const tfhe_secret_key* sk, uint32_t* s, uint32_t* S, uint32_t* bk,
                     uint32_t* ksk);

/* --------------------------------------------------- client side (host) ---- */

/* Encryption c = E(p, k) of Section 2 ("FHE") for TFHE's LWE samples
 * (TLWE, Section 3.2): fresh encryptions under s of the torus messages
 * mu[0..count), each (a, <a, s> + mu + e) with a uniform and e a rounded
 * Gaussian of deviation alpha_lwe.  Ciphertext c is a pure function of
 * (key, seed, first_index + c), so a large input can be produced in
 * independent pieces.  mu: [count] host, ct: [count][n+1] host, written by
 * the call.  count = 0 is a no-op; NULL buffers or a negative count or index
 * return TFHE_EINVAL. */
int tfhe_encrypt_torus(const tfhe_secret_key* sk, uint64_t seed, const uint32_t* mu,
                       int64_t first_index, int64_t count, uint32_t* ct);

/* Decryption p = D(c, k) of Section 2 ("FHE") up to the final rounding: the
 * phase b - <a, key> of count LWE samples, which is the message plus the
 * noise (a bit decrypts to true when the phase, read as a signed 32-bit
 * value, is positive).  key_kind 0: the LWE key s, rows of n+1 words;
 * 1: the TRLWE key S read as an LWE key of dimension N, rows of N+1 words
 * (samples produced by SampleExtract, Section 3.2 step 3).  ct:
 * [count][dim+1] host, phase: [count] host.  The row width is fixed by
 * key_kind, so ct must hold count rows of that width. */
int tfhe_decrypt_phase(const tfhe_secret_key* sk, int key_kind, const uint32_t* ct,
                       int64_t count, uint32_t* phase);

/* Test polynomial of a table-lookup bootstrap over 2^msg_bits entries
 * (message m encoded as m * 2^(31-msg_bits), one padding bit): coefficient j
 * holds lut[floor((j + N/2^(msg_bits+1)) * 2^msg_bits / N)] * 2^(31-msg_bits)
 * when that index is below 2^msg_bits, else -lut[0] * 2^(31-msg_bits).
 * lut entries must be < 2^msg_bits; N >= 2^(msg_bits+1).  tv: [N] host. */
int tfhe_lut_testvec(int32_t N, int32_t msg_bits, const uint32_t* lut, uint32_t* tv);

/* ------------------------------------------------- server side (device) ---- */

/* Device workspace in bytes that a bootstrap call over `batch` samples needs
 * (256-byte aligned pointer required).  The workspace holds the modulus-
 * switched inputs and the extracted samples between kernels. */
int64_t tfhe_workspace_bytes(const tfhe_eval_key* ek, int64_t batch);

/* Gate bootstrapping (Section 3.1, "TFHE homomorphic gates with
 * bootstrapping"): out[c] = LWE_s(gate(ca[c], cb[c])) for c < B.
 * ca, cb, out: [B][n+1] device.  The two inputs are combined linearly, the
 * sum is bootstrapped with the constant test polynomial 1/8, extracted and
 * key-switched back to dimension n.  B = 0 is a no-op. */
int tfhe_gate_bootstrap_batch(const tfhe_eval_key* ek, int gate, const uint32_t* ca,
                              const uint32_t* cb, uint32_t* out, int64_t B, void* workspace,
                              int64_t workspace_bytes, void* stream);

/* Table-lookup (programmable) bootstrap with key switching, the TFHE table
 * lookup of the softmax unit (Section 3.1, "Forward Softmax") and the
 * functional bootstrapping of the cryptosystem switch (Section 3.2, steps 3
 * and 4): out[c] encrypts the test polynomial's value selected by in[c]'s
 * phase -- coefficient 0 of X^{-phi} testvec, phi the phase switched to
 * Z_{2N}.  in, out: [B][n+1] device; testvec: [N] device (see
 * tfhe_lut_testvec, tfhe_torus_testvec).  B = 0 is a no-op. */
int tfhe_lut_bootstrap_batch(const tfhe_eval_key* ek, const uint32_t* in, const uint32_t* testvec,
                             uint32_t* out, int64_t B, void* workspace, int64_t workspace_bytes,
                             void* stream);

/* Blind rotation and SampleExtract without key switching: out[c] is an LWE
 * sample of dimension N under S ([B][N+1] device).  testvec NULL selects the
 * gate polynomial (1/8 everywhere).  Exposed so each stage can be checked. */
int tfhe_bootstrap_extract_batch(const tfhe_eval_key* ek, const uint32_t* in,
                                 const uint32_t* testvec, uint32_t* out, int64_t B,
                                 void* workspace, int64_t workspace_bytes, void* stream);

/* LWE key switching (Section 3.2) from dimension N under S to dimension n
 * under s: each a_i is rounded to ks_t*ks_basebit bits, split into ks_t
 * digits (most significant first) and the key entries of the non-zero digits
 * are subtracted from (0, b).  in: [B][N+1], out: [B][n+1], device.  With
 * t = 8 digits of base 4 the sum runs on the matrix cores (an exact int8
 * product of the one-hot digits with the key's byte planes, whose partial
 * sums over coefficient ranges are added to out with device-scope atomics:
 * the result does not depend on their order). */
int tfhe_keyswitch_batch(const tfhe_eval_key* ek, const uint32_t* in, uint32_t* out, int64_t B,
                         void* stream);

/* Glyph forward ReLU unit (Section 3.1): x holds V encrypted values of
 * `bits` two's-complement bits, LSB first, [V][bits][n+1] device.  Output bit
 * i < bits-1 of value v is AND(NOT x[v][bits-1], x[v][i]) -- the NOT costs no
 * bootstrap -- and output bit bits-1 is a trivial encryption of 0.
 * Gate g of the whole tensor is bit g % (bits-1) of value g / (bits-1); a
 * call computes gates [gate_begin, gate_end) (a streaming window) and writes
 * the sign words of every value it touches.  y: [V][bits][n+1] device. */
int glyph_relu_batch(const tfhe_eval_key* ek, const uint32_t* x, uint32_t* y, int64_t V,
                     int32_t bits, int64_t gate_begin, int64_t gate_end, void* workspace,
                     int64_t workspace_bytes, void* stream);

/* Glyph backward iReLU unit (Section 3.1, "Backward iReLU"): the error of
 * the layer below is the error delta where the forward pre-activation u was
 * non-negative, and zero where it was negative.  u: [V][u_bits][n+1] device
 * (the forward input; only its sign word, bit u_bits-1, is read); delta,
 * out: [V][bits][n+1] device, two's complement LSB first.  Output bit i of
 * value v is AND(NOT u[v][u_bits-1], delta[v][i]) for every i < bits -- the
 * error's sign bit included, so a negative error becomes 0 where u < 0 (the
 * paper counts bits-1 AND gates for the unit; the sign bit needs one too).
 * Gate g is bit g % bits of value g / bits; a call computes gates
 * [gate_begin, gate_end) and writes exactly their output words.  out must
 * not alias u or delta. */
int glyph_irelu_batch(const tfhe_eval_key* ek, const uint32_t* u, int32_t u_bits, const uint32_t* delta,
                      uint32_t* out, int64_t V, int32_t bits, int64_t gate_begin, int64_t gate_end,
                      void* workspace, int64_t workspace_bytes, void* stream);

/* TFHE homomorphic multiplexer, the building block of the paper's softmax
 * unit (Section 3.1, "Forward Softmax"): out[e] encrypts c[e] ? a[e] : b[e]
 * for encrypted bits.  Each multiplexer takes two bootstraps without key
 * switching -- AND(c, a) and AND(NOT c, b) -- whose dimension-N results are
 * added with the constant 1/8 (at most one of them is true) and key-switched
 * once.  c, a, b, out: [B][n+1] device; the workspace must hold
 * tfhe_workspace_bytes(ek, 2 * B). */
int tfhe_mux_batch(const tfhe_eval_key* ek, const uint32_t* c, const uint32_t* a, const uint32_t* b,
                   uint32_t* out, int64_t B, void* workspace, int64_t workspace_bytes, void* stream);

/* Table lookup by a tree of multiplexers, the paper's 3-bit softmax
 * exponentiation unit (Section 3.1, "Forward Softmax", generalised): value v
 * is msg_bits encrypted bits x[v][0..msg_bits) (LSB first) selecting entry
 * k = sum x[v][i] 2^i of the public table[2^msg_bits] (host memory, entries
 * below 2^out_bits); out[v][o] encrypts bit o of table[k].  The first tree
 * level selects between two constants with x[v][0] and needs no bootstrap
 * (its node is a constant, x[v][0] or NOT x[v][0]); each further level is
 * one batch of multiplexers over all values, output bits and nodes:
 * (2^(msg_bits-1) - 1) * out_bits multiplexers per value.  x:
 * [V][msg_bits][n+1], out: [V][out_bits][n+1] device; 1 <= msg_bits <= 6,
 * 1 <= out_bits <= 32; the workspace must hold
 * glyph_mux_lut_workspace_bytes(ek, V, msg_bits, out_bits) bytes. */
int glyph_mux_lut_batch(const tfhe_eval_key* ek, const uint32_t* x, int32_t msg_bits, const uint32_t* table,
                        int32_t out_bits, uint32_t* out, int64_t V, void* workspace,
                        int64_t workspace_bytes, void* stream);

/* Workspace bytes of glyph_mux_lut_batch (negative error code on bad input). */
int64_t glyph_mux_lut_workspace_bytes(const tfhe_eval_key* ek, int64_t V, int32_t msg_bits,
                                      int32_t out_bits);

/* ---- TFHE side of the cryptosystem switch (Section 3.2) ----------------
 * From BGV to TFHE, step 2 packs LWE samples into a TRLWE sample by
 * functional key switching and step 3 extracts LWE samples of its
 * coefficients; from TFHE to BGV, step 4 bootstraps onto multiples of
 * p^-r (a programmable bootstrap with tfhe_torus_testvec).  The BGV side of
 * either direction is not part of this library. */

/* Client side: build the packing key from the secret key (entry (i, j, v),
 * v in [1, 2^ks_basebit), is a TRLWE sample under S of the constant
 * polynomial v * s_i * 2^(32 - (j+1)*ks_basebit), noise alpha_bk) and add it
 * to the eval key on its device.  n * ks_t * (2^ks_basebit - 1) * 2N words
 * (124 MB at n = 630, N = 1024), and for N <= 1024 the same entries in the
 * transform domain, split into two 16-bit parts, that the key switch runs
 * on: n * ks_t * (2^ks_basebit - 1) * 4 * N/2 complex doubles (495 MB at
 * n = 630, N = 1024).  A second call is a no-op.  sk must be the secret key
 * the eval key was made from (checked against a digest of the eval key's
 * public key-switching key: TFHE_EINVAL otherwise). */
int tfhe_packing_key_upload(tfhe_secret_key* sk, tfhe_eval_key* ek);

/* Client side: copy the packing key (built on first use) to host memory,
 * [n][ks_t][2^ks_basebit - 1][2][N] words. */
int tfhe_export_packing_key(tfhe_secret_key* sk, uint32_t* pks);

/* Step 2: functional key switching with the packing morphism.  lwe:
 * [B][Z][n+1] device, Z <= N samples per output under s; out: [B][2][N]
 * device, TRLWE samples (A, B) under S whose phase is sum_z phase_z X^z up to
 * the rounding of each a_{z,i} to ks_t * ks_basebit bits and the key noise.
 * The result is exact mod 2^32: for N <= 1024 the sum of key entries rotated
 * by X^z is computed as products of 0/1 polynomials by the key entries on
 * the transform, whose worst-case error stays below 1/8 before rounding.
 * Needs the packing key (tfhe_packing_key_upload), ks_t * ks_basebit <= 16
 * and ks_basebit <= 2.  out must not alias lwe. */
int tfhe_pack_keyswitch_batch(const tfhe_eval_key* ek, const uint32_t* lwe, int32_t Z, uint32_t* out,
                              int64_t B, void* stream);

/* Step 3: SampleExtract of coefficients 0 .. K-1 of B TRLWE samples
 * ([B][2][N] device) into [B][K][N+1] device LWE samples under S: sample i
 * is (a'_0 .. a'_{N-1}, B_i) with a'_j = A_{i-j} for j <= i and -A_{N+i-j}
 * for j > i; its phase is coefficient i of B - A*S. */
int tfhe_sample_extract_batch(int32_t N, const uint32_t* trlwe, int64_t B, int32_t K, uint32_t* out,
                              void* stream);

/* Host: test polynomial of a programmable bootstrap onto arbitrary torus
 * values (step 4 uses multiples of p^-r): as tfhe_lut_testvec with
 * values[m] (2^msg_bits torus words) in place of lut[m] * 2^(31-msg_bits). */
int tfhe_torus_testvec(int32_t N, int32_t msg_bits, const uint32_t* values, uint32_t* tv);

/* NOT without bootstrapping (Section 3.1): out = -in word by word.
 * in, out: [count][dim+1] device. */
int tfhe_not_batch(int32_t dim, const uint32_t* in, uint32_t* out, int64_t count, void* stream);

/* Exact negacyclic product in Z_{2^32}[X]/(X^N+1) of small signed digit
 * polynomials by torus polynomials, computed by the same transform code as
 * the blind rotation (digits in [-2^(bg-1), 2^(bg-1)) for the key's bg; the
 * other factor is any uint32 polynomial).  d: [B][N] int32, b: [B][N],
 * c: [B][N], device.  Exposed so the transform can be checked at extreme
 * magnitudes against a schoolbook product. */
int tfhe_negacyclic_mul_batch(const tfhe_eval_key* ek, const int32_t* d, const uint32_t* b,
                              uint32_t* c, int64_t B, void* stream);

/* ------------------------------------------------ allocation-free call ---- */

/* Bytes of the device array that tfhe_gate_bootstrap_batch_noalloc uses as
 * its workspace: one copy per device, held from the library's first use on
 * that device until the process ends. */
#define TFHE_NOALLOC_SCRATCH_BYTES (64ll << 20)

/* tfhe_gate_bootstrap_batch for callers that cannot allocate device memory
 * -- code under HIP graph capture, tight serving loops, harnesses that forbid
 * allocation: the same kernels and results, with the workspace taken from a
 * file-scope device array of TFHE_NOALLOC_SCRATCH_BYTES instead of from the
 * caller.  The caller passes inputs and output as for
 * tfhe_gate_bootstrap_batch (ca, cb, out: [B][n+1] device).  The call
 * allocates nothing and records no stage-timing events; the first call on a
 * device also looks up the array's address there.
 * Limit: tfhe_workspace_bytes(ek, B) <= TFHE_NOALLOC_SCRATCH_BYTES (12,515
 * gates at n = 630, N = 1024; 6,919 at n = 750, N = 2048); a larger batch
 * returns TFHE_EINVAL, as do the argument errors of tfhe_gate_bootstrap_batch.
 * Every call on a device shares that device's array: calls that can run at
 * the same time on one device (on different streams, or unordered from
 * different threads) race and corrupt each other's results.  Nothing in the
 * array needs clearing between calls: every word is written before it is
 * read. */
int tfhe_gate_bootstrap_batch_noalloc(const tfhe_eval_key* ek, int gate, const uint32_t* ca,
                                      const uint32_t* cb, uint32_t* out, int64_t B, void* stream);

/* ------------------------------------------------------- stage checks ---- *
 * Single stages of the blind rotation, run by the production kernels in
 * their production launch shapes, so that a fault can be located in one step
 * and any chosen input -- worst cases included -- driven through them. */

/* The modulus switch of Section 3.2's bootstrapping (the first step of every
 * gate bootstrap), after the gate's linear pre-combination (Section 3.1,
 * gates with bootstrapping): out[c][k] = round(x[c][k] * 2N / 2^32) mod 2N,
 * ties rounded up, where x is ca itself (gate = -1) or the combination of
 * ca and cb for gate (a tfhe_gate value).  ca, cb: [B][n+1] device (cb is
 * ignored for gate = -1); out: [B][n+1] device uint16 words, the layout the
 * blind rotation reads.  B = 0 is a no-op. */
int tfhe_debug_mod_switch_batch(const tfhe_eval_key* ek, int gate, const uint32_t* ca, const uint32_t* cb,
                                uint16_t* out, int64_t B, void* stream);

/* Device workspace in bytes of tfhe_debug_cmux_batch over B accumulators. */
int64_t tfhe_debug_cmux_workspace_bytes(const tfhe_eval_key* ek, int64_t B);

/* One CMux step of the blind rotation: the external product of a TRGSW
 * sample by a TRLWE accumulator (Section 3.2, TRGSW x TRLWE), i.e. for every
 * accumulator c < B
 *   acc_out[c] = ACC + sum_r Dec(X^{abar[c]} ACC - ACC)_r * bk_row[r],  ACC = acc_in[c],
 * with the signed gadget decomposition Dec into l digits per polynomial and
 * the negacyclic products exact in Z_{2^32}[X]/(X^N+1).  bk_row is one row
 * of the bootstrapping key in the coefficient domain, [2l][2][N] host words
 * (any values: a chosen key exercises the transform's worst case); it is
 * converted to the transform domain exactly as tfhe_eval_key_upload
 * converts the eval key's rows.  abar: [B] device, each taken mod 2N;
 * acc_in, acc_out: [B][2][N] device (mask polynomial, then body).  The same
 * blind-rotation kernel as every bootstrap runs, with one CMux step, in the
 * launch shape a bootstrap batch of B takes.  The key row is uploaded from
 * host memory, so the call waits for the stream before returning (not for
 * production use).  B = 0 is a no-op. */
int tfhe_debug_cmux_batch(const tfhe_eval_key* ek, const uint32_t* bk_row, const uint32_t* abar,
                          const uint32_t* acc_in, uint32_t* acc_out, int64_t B, void* workspace,
                          int64_t workspace_bytes, void* stream);

/* ---------------------------------------------------------- profiling ---- */

/* Stage timing with HIP events.  While enabled (enable = 1), every server-side
 * call records an event pair around each kernel it launches, on the call's
 * stream.  tfhe_stage_times waits for the recorded events, returns the summed
 * milliseconds and launch counts of the three stages -- index 0: input
 * combination and modulus switch, 1: blind rotation with SampleExtract,
 * 2: key switching -- and clears the record.  enable = 0 stops recording.
 * Host-side state, shared by all threads; not for use during graph capture. */
int tfhe_stage_timing(int enable);
int tfhe_stage_times(double* ms /*[3]*/, int64_t* launches /*[3]*/);

/* VALU issue-rate probe, the measurement behind the blind rotation's
 * roofline peak (64 lane-operations per CU per clock for full-rate
 * instructions).  Launches waves / 4 blocks of 4 waves on `stream` (the
 * current device); every wave runs iters rounds of 16 instructions of one
 * kind on 8 independent chains -- 0: v_fma_f64, 1: v_add_u32,
 * 2: v_cvt_f64_i32, 3: v_bfe_i32, 4: v_mul_lo_u32 -- and each lane
 * writes one word to out[waves * 64] (device) so that no work is dropped.
 * The caller times the launch.  Errors: TFHE_EINVAL for kind outside 0..4,
 * waves not a positive multiple of 4 up to 2^20, iters outside [1, 2^24],
 * or out NULL; TFHE_EHIP if the launch fails. */
int tfhe_probe_valu_rate(int kind, int64_t waves, int64_t iters, uint32_t* out, void* stream);

#ifdef __cplusplus
}
#endif
#endif
