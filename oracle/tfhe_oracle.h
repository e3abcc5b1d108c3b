/*
 * TEST INFRASTRUCTURE ONLY -- the CPU oracle of the TFHE activation path.
 *
 * A plain, slow, obviously-correct implementation of TFHE gate bootstrapping
 * (modulus switch, blind rotation by CMux external products, sample
 * extraction, LWE key switching), the Glyph forward ReLU unit built from it
 * (paper, Section 3.1 "Forward ReLU") and the programmable (look-up-table)
 * bootstrap that stands in for the paper's TFHE table-lookup softmax
 * (Section 3.1 "Forward Softmax"; functional bootstrapping, Section 3.2).
 * Negacyclic products are done by schoolbook multiplication in
 * Z_{2^32}[X]/(X^N+1); nothing here is blocked, fused or transformed.
 *
 * Only tests/, __graft_entry__.smoke() and bench.py's cpu_baseline leg may
 * load or call this library.  The GPU library shares no code with it: the two
 * agree only through the written conventions (rounding, digit order, layouts,
 * the counter-based generator) which each side implements on its own.
 *
 * Torus elements are uint32_t (value x stands for x / 2^32); every torus
 * operation is taken mod 2^32.  LWE samples are [a_0 .. a_{dim-1}, b].
 */
#ifndef TFHE_ORACLE_H
#define TFHE_ORACLE_H
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct {
  int32_t n;          /* LWE dimension */
  int32_t N;          /* ring degree of T_N[X] = T[X]/(X^N+1) (k = 1) */
  int32_t l;          /* gadget length of the bootstrapping key */
  int32_t bg_bit;     /* log2 of the gadget base Bg */
  int32_t ks_t;       /* key-switch digit count */
  int32_t ks_basebit; /* log2 of the key-switch base */
  double alpha_lwe;   /* std. dev. (torus units) of fresh LWE noise */
  double alpha_bk;    /* std. dev. of bootstrapping-key noise */
  double alpha_ks;    /* std. dev. of key-switching-key noise */
} oracle_params;

/* gate codes; the numbering is shared with the GPU library's header by
 * convention only (it is restated there, not included) */
enum {
  ORACLE_NAND = 0, ORACLE_AND, ORACLE_OR, ORACLE_NOR, ORACLE_XOR, ORACLE_XNOR,
  ORACLE_ANDNY, ORACLE_ANDYN, ORACLE_ORNY, ORACLE_ORYN
};

/* domain tags of the counter-based generator */
enum {
  ORACLE_TAG_LWE_KEY = 1, ORACLE_TAG_RLWE_KEY = 2, ORACLE_TAG_BK_MASK = 3,
  ORACLE_TAG_BK_NOISE = 4, ORACLE_TAG_KSK_MASK = 5, ORACLE_TAG_KSK_NOISE = 6,
  ORACLE_TAG_ENC_MASK = 7, ORACLE_TAG_ENC_NOISE = 8, ORACLE_TAG_PKS_MASK = 9,
  ORACLE_TAG_PKS_NOISE = 10
};

/* ---- randomness ------------------------------------------------------- */
uint64_t oracle_stream_output(uint64_t state, uint64_t k);
uint64_t oracle_word(uint64_t seed, uint32_t tag, uint64_t idx);
double oracle_gauss(uint64_t seed, uint32_t tag, uint64_t idx);
uint32_t oracle_noise(uint64_t seed, uint32_t tag, uint64_t idx, double alpha);

/* ---- polynomial arithmetic in Z_{2^32}[X]/(X^N+1) ---------------------- */
void oracle_negacyclic_mul(int32_t N, const uint32_t* a, const uint32_t* b, uint32_t* c);
void oracle_rotate(int32_t N, const uint32_t* p, uint32_t e, uint32_t* out);
void oracle_decompose(int32_t l, int32_t bg_bit, uint32_t x, int32_t* digits);
uint32_t oracle_mod_switch(uint32_t x, int32_t N);
void oracle_mod_switch_batch(const uint32_t* x, int64_t count, int32_t N, uint32_t* out);

/* ---- keys, encryption, decryption ------------------------------------ */
int64_t oracle_bk_words(const oracle_params* p);   /* n * 2l * 2 * N */
int64_t oracle_ksk_words(const oracle_params* p);  /* N * t * (base-1) * (n+1) */
void oracle_keygen(const oracle_params* p, uint64_t seed, uint32_t* s, uint32_t* S,
                   uint32_t* bk, uint32_t* ksk);
void oracle_encrypt(int32_t dim, const uint32_t* key, uint64_t seed, double alpha,
                    const uint32_t* mu, int64_t first_index, int64_t count, uint32_t* ct);
void oracle_phase(int32_t dim, const uint32_t* key, const uint32_t* ct, int64_t count,
                  uint32_t* phase);

/* ---- the bootstrapping steps ----------------------------------------- */
void oracle_gate_combine(const oracle_params* p, int32_t gate, const uint32_t* ca,
                         const uint32_t* cb, uint32_t* out);
void oracle_blind_rotate(const oracle_params* p, const uint32_t* bk, const uint32_t* lwe,
                         const uint32_t* testvec, uint32_t* acc);
void oracle_cmux(const oracle_params* p, const uint32_t* bk_i, uint32_t abar, uint32_t* acc);
void oracle_sample_extract(int32_t N, const uint32_t* acc, uint32_t* out);
void oracle_keyswitch(const oracle_params* p, const uint32_t* ksk, const uint32_t* in,
                      uint32_t* out, int64_t count);
void oracle_lut_testvec(int32_t N, int32_t msg_bits, const uint32_t* lut, uint32_t* tv);

/* ---- batched end-to-end operations (OpenMP across ciphertexts) -------- */
void oracle_gate_bootstrap(const oracle_params* p, const uint32_t* bk, const uint32_t* ksk,
                           int32_t gate, const uint32_t* ca, const uint32_t* cb,
                           uint32_t* out, int64_t count);
void oracle_bootstrap_no_ks(const oracle_params* p, const uint32_t* bk, const uint32_t* in,
                            const uint32_t* testvec, uint32_t* out, int64_t count);
void oracle_lut_bootstrap(const oracle_params* p, const uint32_t* bk, const uint32_t* ksk,
                          const uint32_t* in, const uint32_t* testvec, uint32_t* out,
                          int64_t count);
void oracle_relu_gates(const oracle_params* p, const uint32_t* bk, const uint32_t* ksk,
                       const uint32_t* x, int32_t bits, const int64_t* gate_ids,
                       int64_t count, uint32_t* out);
void oracle_not(int32_t dim, const uint32_t* in, uint32_t* out, int64_t count);
int oracle_threads(void);
/* Threads of the calling thread's later parallel regions (n >= 1); timing only. */
void oracle_set_threads(int n);

/* ---- TFHE side of the cryptosystem switch (Section 3.2) ---------------- */
int64_t oracle_pks_words(const oracle_params* p);  /* n * t * (base-1) * 2 * N */
void oracle_packing_keygen(const oracle_params* p, uint64_t seed, const uint32_t* s,
                           const uint32_t* S, uint32_t* pks);
void oracle_pack_keyswitch(const oracle_params* p, const uint32_t* pks, const uint32_t* lwe,
                           int32_t Z, uint32_t* out);
void oracle_sample_extract_at(int32_t N, const uint32_t* acc, int32_t idx, uint32_t* out);
void oracle_torus_testvec(int32_t N, int32_t msg_bits, const uint32_t* values, uint32_t* tv);

#ifdef __cplusplus
}
#endif
#endif
