// Internal declarations shared by the library's translation units.
#pragma once
#include <cstdint>
#include <string>
#include <vector>

#include "glyph_tfhe.h"

struct tfhe_secret_key {
  tfhe_params p;
  uint64_t seed;
  std::vector<uint32_t> s;    // [n] 0/1
  std::vector<uint32_t> S;    // [N] 0/1
  std::vector<uint32_t> bk;   // [n][2l][2][N] coefficient domain
  std::vector<uint32_t> ksk;  // [N][t][base-1][n+1]
  std::vector<uint32_t> pks;  // packing key [n][t][base-1][2][N], built on request
};

struct tfhe_eval_key {
  tfhe_params p;
  int device;
  int parts;        // the key's coefficients are split into 2 (16-bit) or 3 (11-bit) signed parts
  int cus;          // compute units of the device (the blind rotation sizes its blocks by it)
  double* bk_fft;   // device [n][2l][2*parts][N/2] complex (re, im), transform layout, times 2/N
  double* tw;       // device [3][N/2] complex: forward tree twiddles, inverse stage twiddles, twist
  uint32_t* ksk;    // device [N][t][base-1][n+1], for key switching other than t = 8, base 4 (else NULL)
  int8_t* ksk_mfma; // device, t = 8 and base 4: the key as signed byte planes in matrix-core operand
                    // order (ksk_mfma_host), else NULL
  int64_t ksk_mfma_bytes;
  uint32_t* pks;    // device packing key [n][t][base-1][2][N], or NULL until uploaded
  double* pks_fft;  // the packing key in the transform layout with two parts,
                    // [n][t (base-1)][4][N/2] complex, for N <= 1024 (else NULL)
  int pks_ic_max;   // input coefficients whose products may be summed before one rounding
  int64_t bk_bytes;
  int64_t ksk_bytes;
  int64_t pks_bytes;
  int64_t pks_fft_bytes;
  uint64_t key_tag;  // digest of the start of the key-switching key (public material), which ties
                     // a packing key to the secret key this eval key was made from
};

namespace gt {

// error reporting (thread-local message)
int fail(int rc, const char* fmt, ...);
int check_params(const tfhe_params& p);

// tfhe_gate_bootstrap_batch; timing = false records no stage-timing events
int gate_bootstrap(const tfhe_eval_key* ek, int gate, const uint32_t* ca, const uint32_t* cb, uint32_t* out,
                   int64_t B, void* workspace, int64_t workspace_bytes, void* stream, bool timing);

// generator tags
enum : uint32_t {
  kTagLweKey = 1, kTagRlweKey = 2, kTagBkMask = 3, kTagBkNoise = 4,
  kTagKskMask = 5, kTagKskNoise = 6, kTagEncMask = 7, kTagEncNoise = 8, kTagPksMask = 9, kTagPksNoise = 10
};

// host-side cryptography (gt_host.cpp)
uint64_t rand_word(uint64_t seed, uint32_t tag, uint64_t idx);
uint32_t rand_noise(uint64_t seed, uint32_t tag, uint64_t idx, double alpha);
void keygen_host(tfhe_secret_key& sk);
void packing_keygen_host(tfhe_secret_key& sk);
void encrypt_host(const tfhe_secret_key& sk, uint64_t seed, const uint32_t* mu, int64_t first,
                  int64_t count, uint32_t* ct);
int key_part_shift(int parts);
int key_part_bits(int parts);
// worst-case error of a sum of R products of digits |x| <= D by key parts
// at ring degree N (the external product: R = 2l, D = Bg/2)
double transform_error_bound_rows(int N, int parts, double R, double D);
double transform_error_bound(const tfhe_params& p, int parts);
int key_parts(const tfhe_params& p);  // 2 or 3, 0 if no split keeps the bound
// TRLWE samples [rows][2][N] (u32) to the transform layout of the
// bootstrapping key: [rows][2 parts][N/2] complex, output slot q * parts + s
void trlwe_rows_to_transform_host(int N, int parts, int64_t rows, const uint32_t* src, double* out);
void bk_to_transform_host(const tfhe_params& p, int parts, const uint32_t* bk, double* out);

// Key switching with t = 8 digits of 2 bits runs on the matrix cores: the
// key is uploaded as signed byte planes, without the rows of digit value 0
// (which select nothing).  The 96 key rows (j, v = 1..3) of four input
// coefficients 4G + q make three tiles t = 3G + m.  For tile t, 32-column
// block nb, byte plane beta and lane l of a 64-lane operand, 16 bytes at
// (((t * NB + nb) * 4 + beta) * 64 + l) * 16, NB = ksk_mfma_nb(p); byte s
// is byte plane beta of KSK[4G + q][j][v - 1][col] with col = 32 nb + l % 32
// (0 when col > n), h = l / 32 and
//   m = 0, 1: q = h + 2 m, v = 1 + s / 8, w = (s / 4) % 2,
//   m = 2:    q = h + 2 (s / 8), v = 3, w = (s % 8) / 4,
// j = 7 - s % 4 - 4 w.  The signed bytes b_0..b_3 in [-128, 128) of a key
// word x satisfy sum_beta b_beta 2^(8 beta) = x mod 2^32.
// 32-column blocks of the layout, padded to whole pairs (a kernel block
// covers two)
inline int ksk_mfma_nb(const tfhe_params& p) { return (p.n + 1 + 63) / 64 * 2; }
bool ks_uses_mfma(const tfhe_params& p);
int64_t ksk_mfma_bytes(const tfhe_params& p);
void ksk_to_mfma_host(const tfhe_params& p, const uint32_t* ksk, int8_t* out);
void twiddles_host(int N, double* tw);
void parallel_for(int64_t count, int64_t grain, void (*fn)(int64_t, int64_t, void*), void* ctx);

// device launchers (gt_kernels.hip); return TFHE_OK or TFHE_EHIP
struct Workspace {
  uint16_t* abar;     // [B][n+1] modulus-switched inputs
  uint32_t* extract;  // [B][N+1] extracted samples
};
int64_t workspace_bytes(const tfhe_params& p, int64_t B);
Workspace carve_workspace(const tfhe_params& p, void* ws, int64_t B);

enum InputMode : int {
  kModeGate = 0,      // two-input gate on (ca[c], cb[c])
  kModePlain = 1,     // ca[c] as is
  kModeRelu = 2,      // forward ReLU gates over x = ca
  kModeIRelu = 3,     // backward iReLU gates: sign of u = ca, error bits cb
  kModeMux = 4,       // multiplexer halves: AND(ca, cb), AND(NOT ca, cc)
  kModeMuxTree = 5,   // one level of a multiplexer tree (see prep_kernel)
};

// Inputs of the preparation kernel (gate combination and modulus switch).
// In the multiplexer modes B counts the two halves of every multiplexer.
struct PrepArgs {
  int mode;
  int gate;
  const uint32_t* ca;  // gate: first operand; plain: the input; relu: x; irelu: u; mux: selectors
  const uint32_t* cb;  // gate: second operand; irelu: delta; mux: if-true; mux tree: the level's children
  int64_t B;
  int32_t bits = 0;           // relu: bits of x; irelu: bits of delta; mux tree: selector bits per value
  int64_t gate_begin = 0;     // relu, irelu
  int32_t sign_bits = 0;      // irelu: bits of u (its sign is bit sign_bits - 1)
  const uint32_t* cc = nullptr;  // mux: if-false
  int64_t group = 0;          // mux tree: nodes per (value, output bit) at this level
  int32_t out_bits = 0;       // mux tree: output bits per value
  int32_t level = 0;          // mux tree: selector bit of this level
};

// Stage-check inputs and outputs of the blind rotation (all NULL / 0 on the
// production path): the same kernels, in the same launch shapes, then start
// from the caller's accumulators, run `n` CMux steps over the given
// transform-domain key rows, and write the whole accumulators back instead
// of their SampleExtract.
struct BrIo {
  const uint32_t* acc_in = nullptr;  // [B][2][N] accumulators in place of (0, X^{-bbar} v)
  uint32_t* acc_out = nullptr;       // [B][2][N] final accumulators in place of SampleExtract
  const double* bk = nullptr;        // transform-domain key rows in place of the eval key's
  int n = 0;                         // CMux steps in place of the LWE dimension
};

int launch_prep(const tfhe_eval_key* ek, const PrepArgs& a, const Workspace& ws, void* stream);
int launch_blind_rotate(const tfhe_eval_key* ek, const Workspace& ws, const uint32_t* testvec,
                        int64_t B, void* stream, const BrIo* io = nullptr);
int launch_keyswitch(const tfhe_eval_key* ek, const uint32_t* in, uint32_t* out, int64_t B,
                     int mode, int32_t bits, int64_t gate_begin, void* stream);
int launch_relu_sign(const tfhe_eval_key* ek, uint32_t* y, int32_t bits, int64_t v_begin,
                     int64_t v_end, void* stream);
int launch_not(int32_t dim, const uint32_t* in, uint32_t* out, int64_t count, void* stream);
// abar[2c] = a[c] mod 2N, abar[2c + 1] = 0 for c < B (inputs of a one-CMux stage check)
int launch_cmux_abar(const tfhe_eval_key* ek, const uint32_t* a, int64_t B, uint16_t* abar, void* stream);
// ext[e] += ext[M + e] + (0, 1/8) for e < M (the multiplexer's OR of its halves)
int launch_mux_combine(const tfhe_eval_key* ek, uint32_t* ext, int64_t M, void* stream);
// first level of a multiplexer tree over constant leaves table[k]: node
// (v, o, j) selects bit o of table[2j + x[v][0]]
int launch_lut_leaf(const tfhe_eval_key* ek, const uint32_t* x, int32_t msg_bits, const uint32_t* table,
                    int32_t out_bits, int64_t V, uint32_t* nodes, void* stream);
int launch_pack_keyswitch(const tfhe_eval_key* ek, const uint32_t* lwe, int32_t Z, uint32_t* out, int64_t B,
                          void* stream);
int launch_sample_extract(int32_t N, const uint32_t* trlwe, int64_t B, int32_t K, uint32_t* out, void* stream);
int launch_negacyclic_mul(const tfhe_eval_key* ek, const int32_t* d, const uint32_t* b,
                          uint32_t* c, int64_t B, void* stream);

}  // namespace gt
