// VALU issue-rate probe.
//
// The blind rotation's roofline counts lane-operations against 64 per CU per
// clock (4 SIMDs x 16 lanes, one wave64 instruction per 4 cycles): the rate
// of full-rate VALU instructions.  Its work is fp64 FMAs, additions and
// products, 32-bit integer operations, signed bit-field extractions and
// int-to-double conversions.  This probe measures the issue rate of each of
// these kinds directly: every wave runs `iters` rounds of 16 instructions of
// one kind on 8 independent chains (inline assembly, so the count is exact),
// with enough waves to fill every SIMD, and the caller times the launch.  The
// 32-bit integer multiply is measured beside them.
#include <hip/hip_runtime.h>

#include "gt_internal.h"

namespace {

constexpr int kProbeThreads = 256;  // 4 waves per block

template <int KIND>
__global__ __launch_bounds__(kProbeThreads) void valu_rate_kernel(uint32_t* __restrict__ out, int64_t iters,
                                                                   uint32_t seed) {
  const uint32_t tid = blockIdx.x * kProbeThreads + threadIdx.x;
  const uint32_t s = seed ^ tid;
  if constexpr (KIND == 0) {  // v_fma_f64
    double x[8];
    const double a = 1.0 + 1e-9 * static_cast<double>(s & 7), b = 1e-3 * static_cast<double>(s & 15);
#pragma unroll
    for (int u = 0; u < 8; u++) x[u] = static_cast<double>(u + (s & 3));
    for (int64_t k = 0; k < iters; k++)
#pragma unroll
      for (int u = 0; u < 16; u++) asm volatile("v_fma_f64 %0, %0, %1, %2" : "+v"(x[u % 8]) : "v"(a), "v"(b));
    double t = 0.0;
#pragma unroll
    for (int u = 0; u < 8; u++) t += x[u];
    out[tid] = static_cast<uint32_t>(__double_as_longlong(t));
  } else if constexpr (KIND == 2) {  // v_cvt_f64_i32
    double d[8];
    int32_t v[8];
#pragma unroll
    for (int u = 0; u < 8; u++) v[u] = static_cast<int32_t>(s + u);
    for (int64_t k = 0; k < iters; k++)
#pragma unroll
      for (int u = 0; u < 16; u++) asm volatile("v_cvt_f64_i32 %0, %1" : "=v"(d[u % 8]) : "v"(v[u % 8]));
    double t = 0.0;
#pragma unroll
    for (int u = 0; u < 8; u++) t += d[u];
    out[tid] = static_cast<uint32_t>(__double_as_longlong(t));
  } else {  // 32-bit integer kinds
    uint32_t x[8];
    const uint32_t y = s | 1u, pos = s & 7u, width = 10u;
#pragma unroll
    for (int u = 0; u < 8; u++) x[u] = s * 2654435761u + static_cast<uint32_t>(u);
    for (int64_t k = 0; k < iters; k++)
#pragma unroll
      for (int u = 0; u < 16; u++) {
        if constexpr (KIND == 1)
          asm volatile("v_add_u32 %0, %0, %1" : "+v"(x[u % 8]) : "v"(y));
        else if constexpr (KIND == 3)
          asm volatile("v_bfe_i32 %0, %0, %1, %2" : "+v"(x[u % 8]) : "v"(pos), "v"(width));
        else
          asm volatile("v_mul_lo_u32 %0, %0, %1" : "+v"(x[u % 8]) : "v"(y));
      }
    uint32_t t = 0u;
#pragma unroll
    for (int u = 0; u < 8; u++) t ^= x[u];
    out[tid] = t;
  }
}

}  // namespace

extern "C" int tfhe_probe_valu_rate(int kind, int64_t waves, int64_t iters, uint32_t* out, void* stream) {
  if (kind < 0 || kind > 4) return gt::fail(TFHE_EINVAL, "probe kind %d is not one of 0..4", kind);
  if (waves <= 0 || waves % 4 != 0 || waves > (int64_t{1} << 20))
    return gt::fail(TFHE_EINVAL, "waves must be a positive multiple of 4 up to 2^20, got %lld",
                    static_cast<long long>(waves));
  if (iters <= 0 || iters > (int64_t{1} << 24))
    return gt::fail(TFHE_EINVAL, "iters must be in [1, 2^24], got %lld", static_cast<long long>(iters));
  if (out == nullptr) return gt::fail(TFHE_EINVAL, "NULL output buffer");
  const dim3 grid(static_cast<unsigned>(waves / 4)), block(kProbeThreads);
  hipStream_t st = static_cast<hipStream_t>(stream);
  const uint32_t seed = 0x9e3779b9u;
  switch (kind) {
    case 0: hipLaunchKernelGGL(valu_rate_kernel<0>, grid, block, 0, st, out, iters, seed); break;
    case 1: hipLaunchKernelGGL(valu_rate_kernel<1>, grid, block, 0, st, out, iters, seed); break;
    case 2: hipLaunchKernelGGL(valu_rate_kernel<2>, grid, block, 0, st, out, iters, seed); break;
    case 3: hipLaunchKernelGGL(valu_rate_kernel<3>, grid, block, 0, st, out, iters, seed); break;
    default: hipLaunchKernelGGL(valu_rate_kernel<4>, grid, block, 0, st, out, iters, seed); break;
  }
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return gt::fail(TFHE_EHIP, "valu_rate_kernel: %s", hipGetErrorString(e));
  return TFHE_OK;
}
