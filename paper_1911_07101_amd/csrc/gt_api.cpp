// C ABI of the library (declared in include/glyph_tfhe.h): argument checks,
// key handles, workspace carving and kernel launches.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <initializer_list>
#include <mutex>
#include <new>
#include <vector>

#include "gt_internal.h"

namespace gt {

namespace {
thread_local char g_msg[512] = "";
}

int fail(int rc, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  std::vsnprintf(g_msg, sizeof(g_msg), fmt, ap);
  va_end(ap);
  return rc;
}

int check_params(const tfhe_params& p) {
  if (p.N != 256 && p.N != 512 && p.N != 1024 && p.N != 2048)
    return fail(TFHE_EUNSUPPORTED, "N=%d: supported ring degrees are 256, 512, 1024, 2048", p.N);
  if (p.n < 1 || p.n > 4096) return fail(TFHE_EUNSUPPORTED, "n=%d outside [1, 4096]", p.n);
  if (p.l < 1 || p.bg_bit < 2 || p.l * p.bg_bit > 32)
    return fail(TFHE_EUNSUPPORTED, "gadget l=%d bg_bit=%d: need bg_bit >= 2 and l*bg_bit <= 32", p.l,
                p.bg_bit);
  // the fp64 transform must reproduce every product exactly after rounding
  if (key_parts(p) == 0)
    return fail(TFHE_EUNSUPPORTED,
                "l=%d bg_bit=%d N=%d: the transform error bound exceeds 1/8 even with 11-bit key parts",
                p.l, p.bg_bit, p.N);
  if (p.ks_basebit < 1 || p.ks_basebit > 6 || p.ks_t < 1 || p.ks_t * p.ks_basebit > 32 ||
      p.ks_t * (1 << p.ks_basebit) > 64)
    return fail(TFHE_EUNSUPPORTED,
                "key switching t=%d basebit=%d: need t*basebit <= 32 and t*2^basebit <= 64", p.ks_t,
                p.ks_basebit);
  if (!(p.alpha_lwe >= 0.0) || !(p.alpha_bk >= 0.0) || !(p.alpha_ks >= 0.0))
    return fail(TFHE_EINVAL, "noise parameters must be >= 0");
  return TFHE_OK;
}

}  // namespace gt

using namespace gt;

namespace {

int hip_fail(hipError_t e, const char* what) {
  return fail(TFHE_EHIP, "%s: %s", what, hipGetErrorString(e));
}

// The one-dimensional launches put one work-item on each word (or sample)
// and HIP takes at most 2^32 - 1 work-items in a grid dimension.  Every
// server-side call bounds count * words_per_item by this before it forms
// any product of counts, so none of them can overflow either.
constexpr int64_t kMaxItems = (int64_t{1} << 32) - 256;

int check_count(int64_t count, int64_t words_per_item, const char* what) {
  if (count > kMaxItems / words_per_item)
    return fail(TFHE_EINVAL, "%lld %s of %lld words each exceed the %lld words of one launch; split the call",
                static_cast<long long>(count), what, static_cast<long long>(words_per_item),
                static_cast<long long>(kMaxItems));
  return TFHE_OK;
}

bool aligned(const void* p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

// make the eval key's device current for the duration of a call
struct DeviceGuard {
  int prev = -1;
  bool ok = true;
  explicit DeviceGuard(int dev) {
    if (hipGetDevice(&prev) != hipSuccess) prev = -1;
    if (prev != dev) ok = hipSetDevice(dev) == hipSuccess;
  }
  ~DeviceGuard() {
    int cur = -1;
    if (prev >= 0 && hipGetDevice(&cur) == hipSuccess && cur != prev) (void)hipSetDevice(prev);
  }
};

// FNV-1a over the first 2^16 words of the key-switching key and its length:
// keys from different seeds differ there, and the key-switching key is part
// of the eval key, so the digest reveals nothing secret
uint64_t key_tag(const tfhe_secret_key& sk) {
  uint64_t h = 1469598103934665603ull;
  auto mix = [&](uint64_t v) {
    for (int b = 0; b < 8; b++) {
      h ^= (v >> (8 * b)) & 0xffu;
      h *= 1099511628211ull;
    }
  };
  mix(sk.ksk.size());
  const size_t m = std::min<size_t>(sk.ksk.size(), size_t{1} << 16);
  for (size_t k = 0; k < m; k++) mix(sk.ksk[k]);
  return h;
}

int check_ws(const tfhe_eval_key* ek, void* ws, int64_t ws_bytes, int64_t B) {
  if (ws == nullptr) return fail(TFHE_EINVAL, "workspace is NULL");
  if (!aligned(ws, 256)) return fail(TFHE_EINVAL, "workspace must be 256-byte aligned");
  const int64_t need = workspace_bytes(ek->p, B);
  if (ws_bytes < need)
    return fail(TFHE_EINVAL, "workspace of %lld bytes is smaller than the %lld bytes needed",
                static_cast<long long>(ws_bytes), static_cast<long long>(need));
  return TFHE_OK;
}

struct PhaseCtx {
  const std::vector<uint32_t>* key;
  const uint32_t* ct;
  uint32_t* phase;
};

void phase_rows(int64_t begin, int64_t end, void* vctx) {
  const PhaseCtx& c = *static_cast<PhaseCtx*>(vctx);
  const int64_t dim = static_cast<int64_t>(c.key->size());
  const uint32_t* key = c.key->data();
  for (int64_t k = begin; k < end; k++) {
    const uint32_t* x = c.ct + k * (dim + 1);
    uint32_t v = x[dim];
    for (int64_t m = 0; m < dim; m++) v -= x[m] * key[m];
    c.phase[k] = v;
  }
}

// ---- stage timing (event pairs recorded around each launch while enabled)
struct StageEvent {
  int stage;
  hipEvent_t start, stop;
};
std::mutex g_prof_mu;
bool g_prof_on = false;
std::vector<StageEvent> g_prof_events;

struct StageScope {
  StageEvent ev{};
  bool on = false;
  hipStream_t st;
  StageScope(int stage, void* stream, bool allowed = true) : st(static_cast<hipStream_t>(stream)) {
    if (!allowed) return;
    std::lock_guard<std::mutex> lk(g_prof_mu);
    if (!g_prof_on) return;
    ev.stage = stage;
    if (hipEventCreate(&ev.start) != hipSuccess) return;
    if (hipEventCreate(&ev.stop) != hipSuccess) {
      (void)hipEventDestroy(ev.start);
      return;
    }
    on = hipEventRecord(ev.start, st) == hipSuccess;
  }
  ~StageScope() {
    if (!on) return;
    (void)hipEventRecord(ev.stop, st);
    std::lock_guard<std::mutex> lk(g_prof_mu);
    g_prof_events.push_back(ev);
  }
};

int check_u32(const void* p, const char* name) {
  if (p == nullptr) return fail(TFHE_EINVAL, "%s is NULL", name);
  if (!aligned(p, 4)) return fail(TFHE_EINVAL, "%s is not 4-byte aligned", name);
  return TFHE_OK;
}

// One device buffer of a call, [p, p + bytes).
struct Span {
  const void* p;
  int64_t bytes;
  const char* name;
};

bool overlap(const Span& a, const Span& b) {
  if (a.p == nullptr || b.p == nullptr || a.bytes <= 0 || b.bytes <= 0) return false;
  const uintptr_t a0 = reinterpret_cast<uintptr_t>(a.p), b0 = reinterpret_cast<uintptr_t>(b.p);
  return a0 < b0 + static_cast<uintptr_t>(b.bytes) && b0 < a0 + static_cast<uintptr_t>(a.bytes);
}

// Inputs, outputs and workspace of one call must not overlap: the kernels
// read inputs of some samples after they have written outputs of others
// (a ReLU window, for instance, writes the sign words of values that the
// next window's gates still read).  Every written buffer (`out`) is checked
// against every other buffer of the call.
int check_disjoint(std::initializer_list<Span> in, std::initializer_list<Span> out) {
  for (const Span* o = out.begin(); o != out.end(); ++o) {
    for (const Span& i : in)
      if (overlap(*o, i)) return fail(TFHE_EINVAL, "%s overlaps %s", o->name, i.name);
    for (const Span* o2 = o + 1; o2 != out.end(); ++o2)
      if (overlap(*o, *o2)) return fail(TFHE_EINVAL, "%s overlaps %s", o->name, o2->name);
  }
  return TFHE_OK;
}

int64_t lwe_bytes(int64_t count, int32_t dim) { return count * (int64_t{dim} + 1) * 4; }

}  // namespace

extern "C" {

const char* tfhe_strerror(int rc) {
  switch (rc) {
    case TFHE_OK: return "ok";
    case TFHE_EINVAL: return "invalid argument";
    case TFHE_EUNSUPPORTED: return "unsupported parameters";
    case TFHE_ENOMEM: return "out of memory";
    case TFHE_EHIP: return "HIP runtime error";
    case TFHE_EDEVICE: return "no usable gfx950 device";
    default: return "unknown error";
  }
}

const char* tfhe_last_error(void) { return g_msg; }

int tfhe_secret_keygen(const tfhe_params* params, uint64_t seed, tfhe_secret_key** sk_out) {
  if (params == nullptr || sk_out == nullptr) return fail(TFHE_EINVAL, "NULL argument to tfhe_secret_keygen");
  *sk_out = nullptr;
  int rc = check_params(*params);
  if (rc) return rc;
  tfhe_secret_key* sk = new (std::nothrow) tfhe_secret_key();
  if (!sk) return fail(TFHE_ENOMEM, "host allocation failed");
  sk->p = *params;
  sk->seed = seed;
  try {
    keygen_host(*sk);
  } catch (const std::bad_alloc&) {
    delete sk;
    return fail(TFHE_ENOMEM, "host allocation failed during key generation");
  }
  *sk_out = sk;
  return TFHE_OK;
}

int tfhe_eval_key_upload(const tfhe_secret_key* sk, int device, tfhe_eval_key** ek_out) {
  if (sk == nullptr || ek_out == nullptr) return fail(TFHE_EINVAL, "NULL argument to tfhe_eval_key_upload");
  *ek_out = nullptr;
  int ndev = 0;
  if (hipGetDeviceCount(&ndev) != hipSuccess || device < 0 || device >= ndev)
    return fail(TFHE_EDEVICE, "device %d does not exist (%d visible)", device, ndev);
  hipDeviceProp_t prop;
  if (hipGetDeviceProperties(&prop, device) != hipSuccess) return fail(TFHE_EDEVICE, "cannot query device %d", device);
  if (std::strncmp(prop.gcnArchName, "gfx950", 6) != 0)
    return fail(TFHE_EDEVICE, "device %d is %s; the kernels are built for gfx950", device, prop.gcnArchName);

  const tfhe_params& p = sk->p;
  tfhe_eval_key* ek = new (std::nothrow) tfhe_eval_key();
  if (!ek) return fail(TFHE_ENOMEM, "host allocation failed");
  ek->p = p;
  ek->device = device;
  ek->cus = prop.multiProcessorCount > 0 ? prop.multiProcessorCount : 256;
  ek->parts = key_parts(p);
  ek->bk_fft = nullptr;
  ek->tw = nullptr;
  ek->ksk = nullptr;
  ek->ksk_mfma = nullptr;
  ek->pks = nullptr;
  ek->pks_bytes = 0;
  ek->pks_fft = nullptr;
  ek->pks_fft_bytes = 0;
  ek->pks_ic_max = 0;
  ek->key_tag = key_tag(*sk);
  // [n][2l][2 * parts][N/2] complex doubles
  ek->bk_bytes = static_cast<int64_t>(p.n) * 2 * p.l * 2 * ek->parts * (p.N / 2) * 16;
  // the key-switching key: as byte planes for the matrix-core key switching
  // (t = 8, base 4), as is otherwise
  const bool mfma_ks = ks_uses_mfma(p);
  ek->ksk_bytes = mfma_ks ? 0 : static_cast<int64_t>(sk->ksk.size()) * 4;
  ek->ksk_mfma_bytes = mfma_ks ? ksk_mfma_bytes(p) : 0;
  // forward tree twiddles, inverse stage twiddles, twist: N/2 complex each
  const int64_t tw_bytes = static_cast<int64_t>(3 * (p.N / 2)) * 16;

  std::vector<double> bk_host, tw(static_cast<size_t>(3 * p.N));
  std::vector<int8_t> kmf_host;
  try {
    bk_host.resize(static_cast<size_t>(ek->bk_bytes / 8));
    kmf_host.resize(static_cast<size_t>(ek->ksk_mfma_bytes));
  } catch (const std::bad_alloc&) {
    delete ek;
    return fail(TFHE_ENOMEM, "host allocation failed for the transformed keys");
  }
  bk_to_transform_host(p, ek->parts, sk->bk.data(), bk_host.data());
  twiddles_host(p.N, tw.data());
  if (mfma_ks) ksk_to_mfma_host(p, sk->ksk.data(), kmf_host.data());

  int rc = TFHE_OK;
  hipError_t e;
  DeviceGuard g(device);
  if (!g.ok) {
    rc = fail(TFHE_EDEVICE, "cannot select device %d", device);
    goto fail_out;
  }
  if ((e = hipMalloc(&ek->bk_fft, ek->bk_bytes)) != hipSuccess) { rc = fail(TFHE_ENOMEM, "hipMalloc(bk): %s", hipGetErrorString(e)); goto fail_out; }
  if ((e = hipMalloc(&ek->tw, tw_bytes)) != hipSuccess) { rc = fail(TFHE_ENOMEM, "hipMalloc(twiddles): %s", hipGetErrorString(e)); goto fail_out; }
  if ((e = hipMemcpy(ek->bk_fft, bk_host.data(), ek->bk_bytes, hipMemcpyHostToDevice)) != hipSuccess) { rc = hip_fail(e, "copy bk"); goto fail_out; }
  if ((e = hipMemcpy(ek->tw, tw.data(), tw_bytes, hipMemcpyHostToDevice)) != hipSuccess) { rc = hip_fail(e, "copy twiddles"); goto fail_out; }
  if (mfma_ks) {
    if ((e = hipMalloc(&ek->ksk_mfma, ek->ksk_mfma_bytes)) != hipSuccess) { rc = fail(TFHE_ENOMEM, "hipMalloc(ksk): %s", hipGetErrorString(e)); goto fail_out; }
    if ((e = hipMemcpy(ek->ksk_mfma, kmf_host.data(), ek->ksk_mfma_bytes, hipMemcpyHostToDevice)) != hipSuccess) { rc = hip_fail(e, "copy ksk"); goto fail_out; }
  } else {
    if ((e = hipMalloc(&ek->ksk, ek->ksk_bytes)) != hipSuccess) { rc = fail(TFHE_ENOMEM, "hipMalloc(ksk): %s", hipGetErrorString(e)); goto fail_out; }
    if ((e = hipMemcpy(ek->ksk, sk->ksk.data(), ek->ksk_bytes, hipMemcpyHostToDevice)) != hipSuccess) { rc = hip_fail(e, "copy ksk"); goto fail_out; }
  }
  *ek_out = ek;
  return TFHE_OK;

fail_out:
  tfhe_eval_key_free(ek);
  return rc;
}

int tfhe_keygen_from_seed(const tfhe_params* params, uint64_t seed, int device,
                          tfhe_secret_key** sk_out, tfhe_eval_key** ek_out) {
  if (params == nullptr || sk_out == nullptr || ek_out == nullptr)
    return fail(TFHE_EINVAL, "NULL argument to tfhe_keygen_from_seed");
  *sk_out = nullptr;
  *ek_out = nullptr;
  tfhe_secret_key* sk = nullptr;
  int rc = tfhe_secret_keygen(params, seed, &sk);
  if (rc) return rc;
  rc = tfhe_eval_key_upload(sk, device, ek_out);
  if (rc) {
    delete sk;
    return rc;
  }
  *sk_out = sk;
  return TFHE_OK;
}

void tfhe_secret_key_free(tfhe_secret_key* sk) { delete sk; }

int tfhe_transform_error_bound(const tfhe_params* params, int32_t* parts_out, double* error_bound) {
  if (!params || !parts_out || !error_bound) return fail(TFHE_EINVAL, "NULL argument");
  if (params->N < 256 || params->N > 2048 || (params->N & (params->N - 1)) || params->l < 1 ||
      params->bg_bit < 2 || params->bg_bit > 30)
    return fail(TFHE_EUNSUPPORTED, "N, l or bg_bit out of range");
  const int parts = key_parts(*params);
  *parts_out = parts ? parts : 3;
  *error_bound = transform_error_bound(*params, *parts_out);
  return parts ? TFHE_OK : fail(TFHE_EUNSUPPORTED, "error bound %.3g exceeds 1/8", *error_bound);
}

void tfhe_eval_key_free(tfhe_eval_key* ek) {
  if (!ek) return;
  DeviceGuard g(ek->device);
  if (ek->bk_fft) (void)hipFree(ek->bk_fft);
  if (ek->tw) (void)hipFree(ek->tw);
  if (ek->ksk) (void)hipFree(ek->ksk);
  if (ek->ksk_mfma) (void)hipFree(ek->ksk_mfma);
  if (ek->pks) (void)hipFree(ek->pks);
  if (ek->pks_fft) (void)hipFree(ek->pks_fft);
  delete ek;
}

int tfhe_eval_key_params(const tfhe_eval_key* ek, tfhe_params* out) {
  if (!ek || !out) return fail(TFHE_EINVAL, "NULL argument");
  *out = ek->p;
  return TFHE_OK;
}

int tfhe_export_keys(const tfhe_secret_key* sk, uint32_t* s, uint32_t* S, uint32_t* bk, uint32_t* ksk) {
  if (!sk) return fail(TFHE_EINVAL, "NULL secret key");
  if (s) std::memcpy(s, sk->s.data(), sk->s.size() * 4);
  if (S) std::memcpy(S, sk->S.data(), sk->S.size() * 4);
  if (bk) std::memcpy(bk, sk->bk.data(), sk->bk.size() * 4);
  if (ksk) std::memcpy(ksk, sk->ksk.data(), sk->ksk.size() * 4);
  return TFHE_OK;
}

int tfhe_packing_key_upload(tfhe_secret_key* sk, tfhe_eval_key* ek) {
  if (!sk || !ek) return fail(TFHE_EINVAL, "NULL argument to tfhe_packing_key_upload");
  const tfhe_params &a = sk->p, &b = ek->p;
  if (a.n != b.n || a.N != b.N || a.l != b.l || a.bg_bit != b.bg_bit || a.ks_t != b.ks_t ||
      a.ks_basebit != b.ks_basebit || a.alpha_bk != b.alpha_bk)
    return fail(TFHE_EINVAL, "secret key and eval key have different parameters");
  if (key_tag(*sk) != ek->key_tag)
    return fail(TFHE_EINVAL, "the eval key was not made from this secret key");
  if (ek->pks) return TFHE_OK;
  try {
    if (sk->pks.empty()) packing_keygen_host(*sk);
  } catch (const std::bad_alloc&) {
    return fail(TFHE_ENOMEM, "host allocation failed for the packing key");
  }
  // For N <= 1024 the key switch runs on the transform (pack_ks_fft_kernel):
  // each entry is a product of a 0/1 polynomial by a key polynomial split
  // into two 16-bit parts, and the products of up to ic_max input
  // coefficients (t (base - 1) entries each) are summed before one rounding,
  // ic_max the largest count (at most 64) whose worst-case error stays
  // below 1/8.
  const tfhe_params& p = ek->p;
  const int vals = (1 << p.ks_basebit) - 1;
  const int64_t rows = static_cast<int64_t>(p.n) * p.ks_t * vals;
  int ic_max = 0;
  if (p.N <= 1024 && p.ks_t * p.ks_basebit <= 16 && vals <= 3)
    while (ic_max < 64 && ic_max < p.n &&
           transform_error_bound_rows(p.N, 2, static_cast<double>(ic_max + 1) * p.ks_t * vals, 1.0) <= 0.125)
      ic_max++;
  std::vector<double> fft_host;
  try {
    if (ic_max > 0) {
      fft_host.resize(static_cast<size_t>(rows) * 2 * 2 * p.N);
      trlwe_rows_to_transform_host(p.N, 2, rows, sk->pks.data(), fft_host.data());
    }
  } catch (const std::bad_alloc&) {
    return fail(TFHE_ENOMEM, "host allocation failed for the packing key's transform");
  }
  DeviceGuard g(ek->device);
  if (!g.ok) return fail(TFHE_EDEVICE, "cannot select device %d", ek->device);
  const int64_t bytes = static_cast<int64_t>(sk->pks.size()) * 4;
  const int64_t fft_bytes = static_cast<int64_t>(fft_host.size()) * 8;
  uint32_t* d = nullptr;
  double* df = nullptr;
  hipError_t e;
  if ((e = hipMalloc(&d, bytes)) != hipSuccess) return fail(TFHE_ENOMEM, "hipMalloc(pks): %s", hipGetErrorString(e));
  if ((e = hipMemcpy(d, sk->pks.data(), bytes, hipMemcpyHostToDevice)) != hipSuccess) {
    (void)hipFree(d);
    return hip_fail(e, "copy pks");
  }
  if (fft_bytes > 0) {
    if ((e = hipMalloc(&df, fft_bytes)) != hipSuccess) {
      (void)hipFree(d);
      return fail(TFHE_ENOMEM, "hipMalloc(pks transform): %s", hipGetErrorString(e));
    }
    if ((e = hipMemcpy(df, fft_host.data(), fft_bytes, hipMemcpyHostToDevice)) != hipSuccess) {
      (void)hipFree(d);
      (void)hipFree(df);
      return hip_fail(e, "copy pks transform");
    }
  }
  ek->pks = d;
  ek->pks_bytes = bytes;
  ek->pks_fft = df;
  ek->pks_fft_bytes = fft_bytes;
  ek->pks_ic_max = df ? ic_max : 0;
  return TFHE_OK;
}

int tfhe_export_packing_key(tfhe_secret_key* sk, uint32_t* pks) {
  if (!sk || !pks) return fail(TFHE_EINVAL, "NULL argument to tfhe_export_packing_key");
  try {
    if (sk->pks.empty()) packing_keygen_host(*sk);
  } catch (const std::bad_alloc&) {
    return fail(TFHE_ENOMEM, "host allocation failed for the packing key");
  }
  std::memcpy(pks, sk->pks.data(), sk->pks.size() * 4);
  return TFHE_OK;
}

int tfhe_encrypt_torus(const tfhe_secret_key* sk, uint64_t seed, const uint32_t* mu, int64_t first_index,
                       int64_t count, uint32_t* ct) {
  if (!sk) return fail(TFHE_EINVAL, "NULL secret key");
  if (count < 0 || first_index < 0) return fail(TFHE_EINVAL, "negative count or index");
  if (count == 0) return TFHE_OK;
  if (!mu || !ct) return fail(TFHE_EINVAL, "NULL buffer");
  encrypt_host(*sk, seed, mu, first_index, count, ct);
  return TFHE_OK;
}

int tfhe_decrypt_phase(const tfhe_secret_key* sk, int key_kind, const uint32_t* ct, int64_t count,
                       uint32_t* phase) {
  if (!sk) return fail(TFHE_EINVAL, "NULL secret key");
  if (key_kind != 0 && key_kind != 1) return fail(TFHE_EINVAL, "key_kind must be 0 or 1");
  if (count < 0) return fail(TFHE_EINVAL, "negative count");
  if (count == 0) return TFHE_OK;
  if (!ct || !phase) return fail(TFHE_EINVAL, "NULL buffer");
  PhaseCtx ctx{key_kind == 0 ? &sk->s : &sk->S, ct, phase};
  parallel_for(count, 4096, phase_rows, &ctx);
  return TFHE_OK;
}

int tfhe_torus_testvec(int32_t N, int32_t msg_bits, const uint32_t* values, uint32_t* tv) {
  if (!values || !tv) return fail(TFHE_EINVAL, "NULL buffer");
  if (msg_bits < 1 || msg_bits > 30 || N < (2 << msg_bits) || (N & (N - 1)) != 0)
    return fail(TFHE_EINVAL, "need N a power of two with N >= 2^(msg_bits+1), 1 <= msg_bits <= 30");
  const int64_t M = int64_t{1} << msg_bits;
  const int64_t box = N / M;  // coefficients per table entry
  for (int32_t j = 0; j < N; j++) {
    const int64_t idx = (j + box / 2) / box;
    tv[j] = idx < M ? values[idx] : 0u - values[0];
  }
  return TFHE_OK;
}

int tfhe_lut_testvec(int32_t N, int32_t msg_bits, const uint32_t* lut, uint32_t* tv) {
  if (!lut || !tv) return fail(TFHE_EINVAL, "NULL buffer");
  if (msg_bits < 1 || msg_bits > 30 || N < (2 << msg_bits) || (N & (N - 1)) != 0)
    return fail(TFHE_EINVAL, "need N a power of two with N >= 2^(msg_bits+1), 1 <= msg_bits <= 30");
  const int64_t M = int64_t{1} << msg_bits;
  const int shift = 31 - msg_bits;
  for (int64_t k = 0; k < M; k++)
    if (lut[k] >= static_cast<uint32_t>(M)) return fail(TFHE_EINVAL, "lut[%lld] = %u is not below 2^%d",
                                                         static_cast<long long>(k), lut[k], msg_bits);
  const int64_t box = N / M;  // coefficients per table entry
  for (int32_t j = 0; j < N; j++) {
    const int64_t idx = (j + box / 2) / box;
    tv[j] = idx < M ? lut[idx] << shift : 0u - (lut[0] << shift);
  }
  return TFHE_OK;
}

int64_t tfhe_workspace_bytes(const tfhe_eval_key* ek, int64_t batch) {
  if (!ek || batch < 0) return fail(TFHE_EINVAL, "bad argument to tfhe_workspace_bytes");
  if (int rc = check_count(batch, 1, "ciphertexts")) return rc;
  return workspace_bytes(ek->p, batch);
}

// timing: whether the stage-timing events (tfhe_stage_timing) may be recorded
static int bootstrap_common(const tfhe_eval_key* ek, const PrepArgs& a, const uint32_t* testvec,
                            uint32_t* out, int out_mode, void* ws, int64_t ws_bytes, void* stream,
                            bool keyswitch, bool timing = true) {
  int rc = check_ws(ek, ws, ws_bytes, a.B);
  if (rc) return rc;
  DeviceGuard g(ek->device);
  if (!g.ok) return fail(TFHE_EDEVICE, "cannot select device %d", ek->device);
  Workspace w = carve_workspace(ek->p, ws, a.B);
  {
    StageScope sc(0, stream, timing);
    if ((rc = launch_prep(ek, a, w, stream))) return rc;
  }
  {
    StageScope sc(1, stream, timing);
    if ((rc = launch_blind_rotate(ek, w, testvec, a.B, stream))) return rc;
  }
  if (!keyswitch) {
    hipError_t e = hipMemcpyAsync(out, w.extract, static_cast<size_t>(a.B) * (ek->p.N + 1) * 4,
                                  hipMemcpyDeviceToDevice, static_cast<hipStream_t>(stream));
    return e == hipSuccess ? TFHE_OK : hip_fail(e, "copy extracted samples");
  }
  StageScope sc(2, stream, timing);
  return launch_keyswitch(ek, w.extract, out, a.B, out_mode, a.bits, a.gate_begin, stream);
}

static int gate_bootstrap_impl(const tfhe_eval_key* ek, int gate, const uint32_t* ca, const uint32_t* cb,
                               uint32_t* out, int64_t B, void* workspace, int64_t workspace_bytes_, void* stream,
                               bool timing) {
  if (!ek) return fail(TFHE_EINVAL, "NULL eval key");
  if (B < 0) return fail(TFHE_EINVAL, "negative batch");
  if (int rc = check_count(B, ek->p.n + 1, "ciphertexts")) return rc;
  if (gate < TFHE_NAND || gate > TFHE_ORYN) return fail(TFHE_EINVAL, "unknown gate %d", gate);
  if (B == 0) return TFHE_OK;
  int rc;
  if ((rc = check_u32(ca, "ca")) || (rc = check_u32(cb, "cb")) || (rc = check_u32(out, "out"))) return rc;
  const int64_t w = lwe_bytes(B, ek->p.n);
  if ((rc = check_disjoint({{ca, w, "ca"}, {cb, w, "cb"}},
                           {{out, w, "out"}, {workspace, workspace_bytes(ek->p, B), "workspace"}})))
    return rc;
  PrepArgs a{kModeGate, gate, ca, cb, B, 0, 0};
  return bootstrap_common(ek, a, nullptr, out, kModeGate, workspace, workspace_bytes_, stream, true, timing);
}

int tfhe_gate_bootstrap_batch(const tfhe_eval_key* ek, int gate, const uint32_t* ca, const uint32_t* cb,
                              uint32_t* out, int64_t B, void* workspace, int64_t workspace_bytes_,
                              void* stream) {
  return gate_bootstrap_impl(ek, gate, ca, cb, out, B, workspace, workspace_bytes_, stream, true);
}

int tfhe_lut_bootstrap_batch(const tfhe_eval_key* ek, const uint32_t* in, const uint32_t* testvec,
                             uint32_t* out, int64_t B, void* workspace, int64_t workspace_bytes_,
                             void* stream) {
  if (!ek) return fail(TFHE_EINVAL, "NULL eval key");
  if (B < 0) return fail(TFHE_EINVAL, "negative batch");
  if (int rc = check_count(B, ek->p.n + 1, "ciphertexts")) return rc;
  if (B == 0) return TFHE_OK;
  int rc;
  if ((rc = check_u32(in, "in")) || (rc = check_u32(testvec, "testvec")) || (rc = check_u32(out, "out")))
    return rc;
  const int64_t w = lwe_bytes(B, ek->p.n);
  if ((rc = check_disjoint({{in, w, "in"}, {testvec, int64_t{ek->p.N} * 4, "testvec"}},
                           {{out, w, "out"}, {workspace, workspace_bytes(ek->p, B), "workspace"}})))
    return rc;
  PrepArgs a{kModePlain, 0, in, nullptr, B, 0, 0};
  return bootstrap_common(ek, a, testvec, out, kModePlain, workspace, workspace_bytes_, stream, true);
}

int tfhe_bootstrap_extract_batch(const tfhe_eval_key* ek, const uint32_t* in, const uint32_t* testvec,
                                 uint32_t* out, int64_t B, void* workspace, int64_t workspace_bytes_,
                                 void* stream) {
  if (!ek) return fail(TFHE_EINVAL, "NULL eval key");
  if (B < 0) return fail(TFHE_EINVAL, "negative batch");
  if (int rc = check_count(B, ek->p.n + 1, "ciphertexts")) return rc;
  if (B == 0) return TFHE_OK;
  int rc;
  if ((rc = check_u32(in, "in")) || (rc = check_u32(out, "out"))) return rc;
  if (testvec && !aligned(testvec, 4)) return fail(TFHE_EINVAL, "testvec is not 4-byte aligned");
  if ((rc = check_disjoint({{in, lwe_bytes(B, ek->p.n), "in"}, {testvec, int64_t{ek->p.N} * 4, "testvec"}},
                           {{out, lwe_bytes(B, ek->p.N), "out"}, {workspace, workspace_bytes(ek->p, B), "workspace"}})))
    return rc;
  PrepArgs a{kModePlain, 0, in, nullptr, B, 0, 0};
  return bootstrap_common(ek, a, testvec, out, kModePlain, workspace, workspace_bytes_, stream, false);
}

int tfhe_keyswitch_batch(const tfhe_eval_key* ek, const uint32_t* in, uint32_t* out, int64_t B, void* stream) {
  if (!ek) return fail(TFHE_EINVAL, "NULL eval key");
  if (B < 0) return fail(TFHE_EINVAL, "negative batch");
  if (int rc = check_count(B, ek->p.N + 1, "samples")) return rc;
  if (B == 0) return TFHE_OK;
  int rc;
  if ((rc = check_u32(in, "in")) || (rc = check_u32(out, "out"))) return rc;
  if ((rc = check_disjoint({{in, lwe_bytes(B, ek->p.N), "in"}}, {{out, lwe_bytes(B, ek->p.n), "out"}}))) return rc;
  DeviceGuard g(ek->device);
  if (!g.ok) return fail(TFHE_EDEVICE, "cannot select device %d", ek->device);
  StageScope sc(2, stream);
  return launch_keyswitch(ek, in, out, B, kModePlain, 0, 0, stream);
}

int glyph_relu_batch(const tfhe_eval_key* ek, const uint32_t* x, uint32_t* y, int64_t V, int32_t bits,
                     int64_t gate_begin, int64_t gate_end, void* workspace, int64_t workspace_bytes_,
                     void* stream) {
  if (!ek) return fail(TFHE_EINVAL, "NULL eval key");
  if (V < 0 || bits < 2 || bits > 64) return fail(TFHE_EINVAL, "need V >= 0 and 2 <= bits <= 64");
  if (int rc = check_count(V, bits, "values")) return rc;
  const int64_t total = V * (bits - 1);
  if (gate_begin < 0 || gate_end < gate_begin || gate_end > total)
    return fail(TFHE_EINVAL, "gate window [%lld, %lld) outside [0, %lld)", static_cast<long long>(gate_begin),
                static_cast<long long>(gate_end), static_cast<long long>(total));
  const int64_t B = gate_end - gate_begin;
  if (int rc = check_count(B, ek->p.n + 1, "gates")) return rc;
  if (B == 0) return TFHE_OK;
  int rc;
  if ((rc = check_u32(x, "x")) || (rc = check_u32(y, "y"))) return rc;
  const int64_t w = lwe_bytes(V * bits, ek->p.n);
  if ((rc = check_disjoint({{x, w, "x"}}, {{y, w, "y"}, {workspace, workspace_bytes(ek->p, B), "workspace"}})))
    return rc;
  PrepArgs a{kModeRelu, TFHE_ANDNY, x, nullptr, B, bits, gate_begin};
  rc = bootstrap_common(ek, a, nullptr, y, kModeRelu, workspace, workspace_bytes_, stream, true);
  if (rc) return rc;
  const int64_t v_begin = gate_begin / (bits - 1);
  const int64_t v_end = (gate_end - 1) / (bits - 1) + 1;
  DeviceGuard g(ek->device);
  return launch_relu_sign(ek, y, bits, v_begin, v_end, stream);
}

int glyph_irelu_batch(const tfhe_eval_key* ek, const uint32_t* u, int32_t u_bits, const uint32_t* delta,
                      uint32_t* out, int64_t V, int32_t bits, int64_t gate_begin, int64_t gate_end,
                      void* workspace, int64_t workspace_bytes_, void* stream) {
  if (!ek) return fail(TFHE_EINVAL, "NULL eval key");
  if (V < 0 || bits < 1 || bits > 64 || u_bits < 1 || u_bits > 64)
    return fail(TFHE_EINVAL, "need V >= 0, 1 <= bits <= 64 and 1 <= u_bits <= 64");
  if (int rc = check_count(V, bits, "values")) return rc;
  const int64_t total = V * bits;
  if (gate_begin < 0 || gate_end < gate_begin || gate_end > total)
    return fail(TFHE_EINVAL, "gate window [%lld, %lld) outside [0, %lld)", static_cast<long long>(gate_begin),
                static_cast<long long>(gate_end), static_cast<long long>(total));
  const int64_t B = gate_end - gate_begin;
  if (int rc = check_count(B, ek->p.n + 1, "gates")) return rc;
  if (B == 0) return TFHE_OK;
  int rc;
  if ((rc = check_u32(u, "u")) || (rc = check_u32(delta, "delta")) || (rc = check_u32(out, "out"))) return rc;
  const int64_t w = lwe_bytes(V * bits, ek->p.n);
  if ((rc = check_disjoint({{u, lwe_bytes(V * u_bits, ek->p.n), "u"}, {delta, w, "delta"}},
                           {{out, w, "out"}, {workspace, workspace_bytes(ek->p, B), "workspace"}})))
    return rc;
  PrepArgs a{kModeIRelu, TFHE_ANDNY, u, delta, B, bits, gate_begin, u_bits};
  return bootstrap_common(ek, a, nullptr, out, kModeIRelu, workspace, workspace_bytes_, stream, true);
}

// Multiplexers: a.B = 2M samples (the two halves of M multiplexers) are
// prepared and blind-rotated with the gate polynomial, the halves of each
// multiplexer are added with (0, 1/8) and the M sums key-switched into out.
static int mux_common(const tfhe_eval_key* ek, const PrepArgs& a, uint32_t* out, void* ws, int64_t ws_bytes,
                      void* stream) {
  int rc = check_ws(ek, ws, ws_bytes, a.B);
  if (rc) return rc;
  DeviceGuard g(ek->device);
  if (!g.ok) return fail(TFHE_EDEVICE, "cannot select device %d", ek->device);
  Workspace w = carve_workspace(ek->p, ws, a.B);
  const int64_t M = a.B / 2;
  {
    StageScope sc(0, stream);
    if ((rc = launch_prep(ek, a, w, stream))) return rc;
  }
  {
    StageScope sc(1, stream);
    if ((rc = launch_blind_rotate(ek, w, nullptr, a.B, stream))) return rc;
    if ((rc = launch_mux_combine(ek, w.extract, M, stream))) return rc;
  }
  StageScope sc(2, stream);
  return launch_keyswitch(ek, w.extract, out, M, kModePlain, 0, 0, stream);
}

int tfhe_mux_batch(const tfhe_eval_key* ek, const uint32_t* c, const uint32_t* a, const uint32_t* b,
                   uint32_t* out, int64_t B, void* workspace, int64_t workspace_bytes_, void* stream) {
  if (!ek) return fail(TFHE_EINVAL, "NULL eval key");
  if (B < 0) return fail(TFHE_EINVAL, "negative batch");
  // 2B halves are bootstrapped (n + 1 words each), B sums combined (N + 1)
  if (int rc = check_count(B, 2 * (std::max(ek->p.n, ek->p.N) + 1), "multiplexers")) return rc;
  if (B == 0) return TFHE_OK;
  int rc;
  if ((rc = check_u32(c, "c")) || (rc = check_u32(a, "a")) || (rc = check_u32(b, "b")) ||
      (rc = check_u32(out, "out")))
    return rc;
  const int64_t w = lwe_bytes(B, ek->p.n);
  if ((rc = check_disjoint({{c, w, "c"}, {a, w, "a"}, {b, w, "b"}},
                           {{out, w, "out"}, {workspace, workspace_bytes(ek->p, 2 * B), "workspace"}})))
    return rc;
  PrepArgs pa{};
  pa.mode = kModeMux;
  pa.ca = c;
  pa.cb = a;
  pa.cc = b;
  pa.B = 2 * B;
  return mux_common(ek, pa, out, workspace, workspace_bytes_, stream);
}

// Workspace of glyph_mux_lut_batch: the tree's first two levels of nodes and
// the bootstrap workspace of its widest bootstrapped level.
struct MuxLutLayout {
  int64_t a_off, b_off, ws_off, total, nodes_a, nodes_b, widest;
};

// words per value of the widest launch of a multiplexer tree: its leaves,
// out_bits * 2^(msg_bits - 1) samples of n + 1 words, which also bound the
// bootstrapped levels' samples (n + 1 words) and sums (N + 1 words)
static int64_t mux_lut_words(const tfhe_params& p, int32_t msg_bits, int32_t out_bits) {
  return int64_t{out_bits} * (int64_t{1} << (msg_bits - 1)) * (std::max(p.n, p.N) + 1);
}

static MuxLutLayout mux_lut_layout(const tfhe_params& p, int64_t V, int32_t msg_bits, int32_t out_bits) {
  MuxLutLayout L{};
  const int64_t row = (p.n + 1) * 4;
  L.nodes_a = msg_bits >= 2 ? V * out_bits * (int64_t{1} << (msg_bits - 1)) : 0;
  L.nodes_b = msg_bits >= 3 ? V * out_bits * (int64_t{1} << (msg_bits - 2)) : 0;
  L.widest = msg_bits >= 2 ? 2 * V * out_bits * (int64_t{1} << (msg_bits - 2)) : 0;
  auto up = [](int64_t x) { return (x + 255) / 256 * 256; };
  L.a_off = 0;
  L.b_off = up(L.nodes_a * row);
  L.ws_off = L.b_off + up(L.nodes_b * row);
  L.total = L.ws_off + (L.widest ? workspace_bytes(p, L.widest) : 0);
  return L;
}

int64_t glyph_mux_lut_workspace_bytes(const tfhe_eval_key* ek, int64_t V, int32_t msg_bits, int32_t out_bits) {
  if (!ek || V < 0 || msg_bits < 1 || msg_bits > 6 || out_bits < 1 || out_bits > 32)
    return fail(TFHE_EINVAL, "bad argument to glyph_mux_lut_workspace_bytes");
  if (int rc = check_count(V, mux_lut_words(ek->p, msg_bits, out_bits), "values")) return rc;
  return mux_lut_layout(ek->p, V, msg_bits, out_bits).total;
}

int glyph_mux_lut_batch(const tfhe_eval_key* ek, const uint32_t* x, int32_t msg_bits, const uint32_t* table,
                        int32_t out_bits, uint32_t* out, int64_t V, void* workspace, int64_t workspace_bytes_,
                        void* stream) {
  if (!ek) return fail(TFHE_EINVAL, "NULL eval key");
  if (V < 0 || msg_bits < 1 || msg_bits > 6 || out_bits < 1 || out_bits > 32)
    return fail(TFHE_EINVAL, "need V >= 0, 1 <= msg_bits <= 6, 1 <= out_bits <= 32");
  if (int rc = check_count(V, mux_lut_words(ek->p, msg_bits, out_bits), "values")) return rc;
  if (!table) return fail(TFHE_EINVAL, "NULL table");
  for (int k = 0; k < (1 << msg_bits); k++)
    if (out_bits < 32 && (table[k] >> out_bits) != 0)
      return fail(TFHE_EINVAL, "table entry %d does not fit in %d bits", k, out_bits);
  if (V == 0) return TFHE_OK;
  int rc;
  if ((rc = check_u32(x, "x")) || (rc = check_u32(out, "out"))) return rc;
  const MuxLutLayout L = mux_lut_layout(ek->p, V, msg_bits, out_bits);
  if (!workspace) return fail(TFHE_EINVAL, "workspace is NULL");
  if (!aligned(workspace, 256)) return fail(TFHE_EINVAL, "workspace must be 256-byte aligned");
  if (workspace_bytes_ < L.total)
    return fail(TFHE_EINVAL, "workspace of %lld bytes is smaller than the %lld bytes needed",
                static_cast<long long>(workspace_bytes_), static_cast<long long>(L.total));
  if ((rc = check_disjoint({{x, lwe_bytes(V * msg_bits, ek->p.n), "x"}},
                           {{out, lwe_bytes(V * out_bits, ek->p.n), "out"}, {workspace, L.total, "workspace"}})))
    return rc;
  char* base = static_cast<char*>(workspace);
  uint32_t* nodes[2] = {reinterpret_cast<uint32_t*>(base + L.a_off), reinterpret_cast<uint32_t*>(base + L.b_off)};
  {
    DeviceGuard g(ek->device);
    if (!g.ok) return fail(TFHE_EDEVICE, "cannot select device %d", ek->device);
    if ((rc = launch_lut_leaf(ek, x, msg_bits, table, out_bits, V, msg_bits == 1 ? out : nodes[0], stream)))
      return rc;
  }
  // levels 2 .. msg_bits: level k reads the nodes of level k-1 and writes
  // 2^(msg_bits-k) nodes per (value, output bit), the last level into out
  for (int k = 2; k <= msg_bits; k++) {
    PrepArgs pa{};
    pa.mode = kModeMuxTree;
    pa.ca = x;
    pa.cb = nodes[k & 1];
    pa.bits = msg_bits;
    pa.group = int64_t{1} << (msg_bits - k);
    pa.out_bits = out_bits;
    pa.level = k - 1;
    pa.B = 2 * V * out_bits * pa.group;
    uint32_t* dst = k == msg_bits ? out : nodes[(k + 1) & 1];
    if ((rc = mux_common(ek, pa, dst, base + L.ws_off, L.total - L.ws_off, stream))) return rc;
  }
  return TFHE_OK;
}

int tfhe_pack_keyswitch_batch(const tfhe_eval_key* ek, const uint32_t* lwe, int32_t Z, uint32_t* out, int64_t B,
                              void* stream) {
  if (!ek) return fail(TFHE_EINVAL, "NULL eval key");
  if (!ek->pks) return fail(TFHE_EINVAL, "the eval key has no packing key (call tfhe_packing_key_upload)");
  if (B < 0 || Z < 1 || Z > ek->p.N) return fail(TFHE_EINVAL, "need B >= 0 and 1 <= Z <= N");
  // B * 2N words initialised, then B blocks of 256 work-items
  if (int rc = check_count(B, std::max(2 * ek->p.N, 256), "ciphertexts")) return rc;
  if (B == 0) return TFHE_OK;
  int rc;
  if ((rc = check_u32(lwe, "lwe")) || (rc = check_u32(out, "out"))) return rc;
  if ((rc = check_disjoint({{lwe, lwe_bytes(B * Z, ek->p.n), "lwe"}}, {{out, B * 2 * ek->p.N * 4, "out"}})))
    return rc;
  DeviceGuard g(ek->device);
  if (!g.ok) return fail(TFHE_EDEVICE, "cannot select device %d", ek->device);
  return launch_pack_keyswitch(ek, lwe, Z, out, B, stream);
}

int tfhe_sample_extract_batch(int32_t N, const uint32_t* trlwe, int64_t B, int32_t K, uint32_t* out,
                              void* stream) {
  if (N < 2 || N > 4096 || (N & (N - 1))) return fail(TFHE_EINVAL, "N must be a power of two in [2, 4096]");
  if (B < 0 || K < 1 || K > N) return fail(TFHE_EINVAL, "need B >= 0 and 1 <= K <= N");
  if (int rc = check_count(B, int64_t{K} * (N + 1), "ciphertexts")) return rc;
  if (B == 0) return TFHE_OK;
  int rc;
  if ((rc = check_u32(trlwe, "trlwe")) || (rc = check_u32(out, "out"))) return rc;
  if ((rc = check_disjoint({{trlwe, B * 2 * N * 4, "trlwe"}}, {{out, lwe_bytes(B * K, N), "out"}}))) return rc;
  return launch_sample_extract(N, trlwe, B, K, out, stream);
}

int tfhe_not_batch(int32_t dim, const uint32_t* in, uint32_t* out, int64_t count, void* stream) {
  if (dim < 1 || count < 0) return fail(TFHE_EINVAL, "need dim >= 1 and count >= 0");
  if (int rc = check_count(count, int64_t{dim} + 1, "samples")) return rc;
  if (count == 0) return TFHE_OK;
  int rc;
  if ((rc = check_u32(in, "in")) || (rc = check_u32(out, "out"))) return rc;
  if ((rc = check_disjoint({{in, lwe_bytes(count, dim), "in"}}, {{out, lwe_bytes(count, dim), "out"}}))) return rc;
  return launch_not(dim, in, out, count, stream);
}

int tfhe_negacyclic_mul_batch(const tfhe_eval_key* ek, const int32_t* d, const uint32_t* b, uint32_t* c,
                              int64_t B, void* stream) {
  if (!ek) return fail(TFHE_EINVAL, "NULL eval key");
  if (B < 0) return fail(TFHE_EINVAL, "negative batch");
  if (int rc = check_count(B, ek->p.N, "products")) return rc;
  if (B == 0) return TFHE_OK;
  int rc;
  if ((rc = check_u32(d, "d")) || (rc = check_u32(b, "b")) || (rc = check_u32(c, "c"))) return rc;
  const int64_t w = B * ek->p.N * 4;
  if ((rc = check_disjoint({{d, w, "d"}, {b, w, "b"}}, {{c, w, "c"}}))) return rc;
  DeviceGuard g(ek->device);
  if (!g.ok) return fail(TFHE_EDEVICE, "cannot select device %d", ek->device);
  return launch_negacyclic_mul(ek, d, b, c, B, stream);
}

int tfhe_debug_mod_switch_batch(const tfhe_eval_key* ek, int gate, const uint32_t* ca, const uint32_t* cb,
                                uint16_t* out, int64_t B, void* stream) {
  if (!ek) return fail(TFHE_EINVAL, "NULL eval key");
  if (B < 0) return fail(TFHE_EINVAL, "negative batch");
  if (int rc = check_count(B, ek->p.n + 1, "samples")) return rc;
  if (gate < -1 || gate > TFHE_ORYN) return fail(TFHE_EINVAL, "gate %d is neither -1 nor a gate", gate);
  if (B == 0) return TFHE_OK;
  int rc;
  if ((rc = check_u32(ca, "ca")) || (gate >= 0 && (rc = check_u32(cb, "cb")))) return rc;
  if (out == nullptr || !aligned(out, 2)) return fail(TFHE_EINVAL, "out is NULL or not 2-byte aligned");
  const int64_t w = lwe_bytes(B, ek->p.n);
  if ((rc = check_disjoint({{ca, w, "ca"}, {gate >= 0 ? cb : nullptr, w, "cb"}}, {{out, w / 2, "out"}}))) return rc;
  DeviceGuard g(ek->device);
  if (!g.ok) return fail(TFHE_EDEVICE, "cannot select device %d", ek->device);
  PrepArgs a{gate < 0 ? kModePlain : kModeGate, gate < 0 ? 0 : gate, ca, gate < 0 ? nullptr : cb, B, 0, 0};
  Workspace ws{out, nullptr};
  StageScope sc(0, stream);
  return launch_prep(ek, a, ws, stream);
}

// workspace of tfhe_debug_cmux_batch: the key row in the transform domain,
// then the modulus-switched inputs [B][2] u16
static int64_t debug_cmux_key_bytes(const tfhe_eval_key* ek) {
  const int64_t b = int64_t{2} * ek->p.l * 2 * ek->parts * (ek->p.N / 2) * 16;
  return (b + 255) / 256 * 256;
}

int64_t tfhe_debug_cmux_workspace_bytes(const tfhe_eval_key* ek, int64_t B) {
  if (!ek || B < 0) return fail(TFHE_EINVAL, "bad argument to tfhe_debug_cmux_workspace_bytes");
  if (int rc = check_count(B, 2 * int64_t{ek->p.N}, "accumulators")) return rc;
  return debug_cmux_key_bytes(ek) + (B * 4 + 255) / 256 * 256;
}

int tfhe_debug_cmux_batch(const tfhe_eval_key* ek, const uint32_t* bk_row, const uint32_t* abar,
                          const uint32_t* acc_in, uint32_t* acc_out, int64_t B, void* workspace,
                          int64_t workspace_bytes_, void* stream) {
  if (!ek) return fail(TFHE_EINVAL, "NULL eval key");
  if (B < 0) return fail(TFHE_EINVAL, "negative batch");
  if (int rc = check_count(B, 2 * int64_t{ek->p.N}, "accumulators")) return rc;
  if (B == 0) return TFHE_OK;
  if (!bk_row) return fail(TFHE_EINVAL, "bk_row is NULL");
  int rc;
  if ((rc = check_u32(abar, "abar")) || (rc = check_u32(acc_in, "acc_in")) || (rc = check_u32(acc_out, "acc_out")))
    return rc;
  if (!workspace || !aligned(workspace, 256)) return fail(TFHE_EINVAL, "workspace is NULL or not 256-byte aligned");
  const int64_t need = tfhe_debug_cmux_workspace_bytes(ek, B);
  if (workspace_bytes_ < need)
    return fail(TFHE_EINVAL, "workspace of %lld bytes is smaller than the %lld bytes needed",
                static_cast<long long>(workspace_bytes_), static_cast<long long>(need));
  const int64_t acc_bytes = B * 2 * ek->p.N * 4;
  if ((rc = check_disjoint({{abar, B * 4, "abar"}, {acc_in, acc_bytes, "acc_in"}},
                           {{acc_out, acc_bytes, "acc_out"}, {workspace, need, "workspace"}})))
    return rc;
  // the key row in the transform domain, as the eval key's rows are made
  tfhe_params p1 = ek->p;
  p1.n = 1;
  std::vector<double> row;
  try {
    row.resize(static_cast<size_t>(debug_cmux_key_bytes(ek) / 8));
  } catch (const std::bad_alloc&) {
    return fail(TFHE_ENOMEM, "host allocation failed for the key row");
  }
  bk_to_transform_host(p1, ek->parts, bk_row, row.data());
  DeviceGuard g(ek->device);
  if (!g.ok) return fail(TFHE_EDEVICE, "cannot select device %d", ek->device);
  hipStream_t st = static_cast<hipStream_t>(stream);
  char* base = static_cast<char*>(workspace);
  uint16_t* ab = reinterpret_cast<uint16_t*>(base + debug_cmux_key_bytes(ek));
  hipError_t e = hipMemcpyAsync(base, row.data(), row.size() * 8, hipMemcpyHostToDevice, st);
  if (e != hipSuccess) return hip_fail(e, "copy key row");
  // the host copy of the key row must outlive the upload: every return from
  // here on waits for the stream first
  auto finish = [&](int result) {
    const hipError_t se = hipStreamSynchronize(st);
    if (result != TFHE_OK) return result;
    return se == hipSuccess ? TFHE_OK : hip_fail(se, "stage check");
  };
  if ((rc = launch_cmux_abar(ek, abar, B, ab, stream))) return finish(rc);
  BrIo io;
  io.acc_in = acc_in;
  io.acc_out = acc_out;
  io.bk = reinterpret_cast<const double*>(base);
  io.n = 1;
  {
    StageScope sc(1, stream);
    if ((rc = launch_blind_rotate(ek, Workspace{ab, nullptr}, nullptr, B, stream, &io))) return finish(rc);
  }
  return finish(TFHE_OK);
}

int tfhe_stage_timing(int enable) {
  std::lock_guard<std::mutex> lk(g_prof_mu);
  g_prof_on = enable != 0;
  return TFHE_OK;
}

int tfhe_stage_times(double* ms, int64_t* launches) {
  if (!ms || !launches) return fail(TFHE_EINVAL, "NULL argument");
  std::vector<StageEvent> evs;
  {
    std::lock_guard<std::mutex> lk(g_prof_mu);
    evs.swap(g_prof_events);
  }
  for (int k = 0; k < 3; k++) {
    ms[k] = 0.0;
    launches[k] = 0;
  }
  int rc = TFHE_OK;
  for (auto& ev : evs) {
    float t = 0.f;
    hipError_t e = hipEventSynchronize(ev.stop);
    if (e == hipSuccess) e = hipEventElapsedTime(&t, ev.start, ev.stop);
    if (e != hipSuccess && rc == TFHE_OK) rc = hip_fail(e, "stage event");
    if (e == hipSuccess && ev.stage >= 0 && ev.stage < 3) {
      ms[ev.stage] += t;
      launches[ev.stage] += 1;
    }
    (void)hipEventDestroy(ev.start);
    (void)hipEventDestroy(ev.stop);
  }
  return rc;
}

}  // extern "C"

int gt::gate_bootstrap(const tfhe_eval_key* ek, int gate, const uint32_t* ca, const uint32_t* cb, uint32_t* out,
                       int64_t B, void* workspace, int64_t workspace_bytes, void* stream, bool timing) {
  return gate_bootstrap_impl(ek, gate, ca, cb, out, B, workspace, workspace_bytes, stream, timing);
}
