// Gate bootstrapping for callers that cannot allocate device memory.
//
// tfhe_gate_bootstrap_batch takes its workspace (the modulus-switched inputs
// and the extracted samples between the kernels) from the caller.  The entry
// point here takes it from a file-scope device array instead, so that code
// under HIP graph capture, tight serving loops and harnesses that forbid
// allocation can bootstrap without any allocation.  Each device holds its
// own copy of the array, at its own address, from the time the library's
// code is loaded on it until the process ends.
#include <hip/hip_runtime.h>

#include <mutex>

#include "gt_internal.h"

namespace {

constexpr int64_t kScratchBytes = TFHE_NOALLOC_SCRATCH_BYTES;

// In host code `scratch` names a host-side stand-in, not device memory: it is
// never passed to a kernel or a copy.  Host code uses the device address
// that hipGetSymbolAddress returns for the current device.
__device__ __align__(256) unsigned char scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_mu;
void* g_scratch[kMaxDevices] = {};

// Address of `scratch` on `device`, looked up on the first call on that
// device (with the device current) and kept.
int scratch_address(int device, void** out) {
  if (device < 0 || device >= kMaxDevices)
    return gt::fail(TFHE_EDEVICE, "device %d is outside the %d devices the no-allocation entry serves", device,
                    kMaxDevices);
  std::lock_guard<std::mutex> lk(g_mu);
  if (g_scratch[device] == nullptr) {
    int prev = -1;
    if (hipGetDevice(&prev) != hipSuccess) prev = -1;
    if (prev != device && hipSetDevice(device) != hipSuccess)
      return gt::fail(TFHE_EDEVICE, "cannot select device %d", device);
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (prev >= 0 && prev != device) (void)hipSetDevice(prev);
    if (e != hipSuccess || p == nullptr)
      return gt::fail(TFHE_EHIP, "device address of the no-allocation workspace on device %d: %s", device,
                      hipGetErrorString(e));
    g_scratch[device] = p;
  }
  *out = g_scratch[device];
  return TFHE_OK;
}

}  // namespace

extern "C" int tfhe_gate_bootstrap_batch_noalloc(const tfhe_eval_key* ek, int gate, const uint32_t* ca,
                                                 const uint32_t* cb, uint32_t* out, int64_t B, void* stream) {
  if (!ek) return gt::fail(TFHE_EINVAL, "NULL eval key");
  if (B < 0) return gt::fail(TFHE_EINVAL, "negative batch");
  // the per-gate workspace is under 10 KB for every supported ring, so this
  // bound also keeps the size computation below from overflowing
  if (B > kScratchBytes) return gt::fail(TFHE_EINVAL, "batch of %lld gates exceeds the no-allocation workspace",
                                         static_cast<long long>(B));
  if (B == 0) return TFHE_OK;
  const int64_t need = gt::workspace_bytes(ek->p, B);
  if (need > kScratchBytes)
    return gt::fail(TFHE_EINVAL,
                    "a batch of %lld gates needs %lld bytes of workspace; the no-allocation entry holds %lld "
                    "(split the batch or use tfhe_gate_bootstrap_batch)",
                    static_cast<long long>(B), static_cast<long long>(need), static_cast<long long>(kScratchBytes));
  void* ws = nullptr;
  if (int rc = scratch_address(ek->device, &ws)) return rc;
  // every workspace word is written before it is read (modulus-switched
  // inputs by the first kernel, extracted samples by the second), so nothing
  // is cleared between calls
  return gt::gate_bootstrap(ek, gate, ca, cb, out, B, ws, kScratchBytes, stream, false);
}
