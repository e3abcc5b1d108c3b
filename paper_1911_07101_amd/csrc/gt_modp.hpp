// Exact arithmetic modulo the NTT prime P = 549755731969 (= 2^39 - 5 * 2^14 + 1,
// so P = 1 mod 2^14) carried in IEEE double precision.
//
// Why doubles: the negacyclic products of blind rotation are computed exactly
// with a number-theoretic transform mod P.  On CDNA4, fp64 FMA issues at full
// rate, so a modular product costs six fp64 instructions (error-free product
// plus a rounded quotient) instead of the ~28 integer instructions a 64-bit
// integer modulus needs on a 32-bit integer ALU.
//
// Every value is an integer held exactly in a double (|x| < 2^53).  Residues
// are kept lazily in a symmetric range and reduced only where the bounds below
// require it.
//
//   mulmod(a, w): for |a| < 2^51 and |w| < P returns r = a*w (mod P) with
//     |r| < 0.75 P + 2^(e-53) where 2^e > |a*w|.
//     h = fl(a*w) and l = a*w - h (exact, by FMA) split the product; q is the
//     nearest integer to h * fl(1/P) (|h/P| < 2^51 so the magic-constant
//     rounding is exact and |q - h/P| <= 3/4); h - q*P is an integer below
//     0.75 P in magnitude and the FMA produces it exactly; adding l is exact.
//   reduce(x): for |x| < 2^52 returns r = x (mod P) with |r| <= P/2 + 1.
//
// Shared by the HIP kernels and the host-side unit test of this header.
#pragma once
#include <cmath>
#include <cstdint>

#ifdef __HIPCC__
#include <hip/hip_runtime.h>
#define GT_HD __host__ __device__ __forceinline__
#else
#define GT_HD inline
#endif

namespace gt {

constexpr uint64_t kPrime = 549755731969ull;
constexpr double kP = 549755731969.0;
constexpr double kPinv = 1.0 / 549755731969.0;
constexpr double kMagic = 6755399441055744.0;  // 1.5 * 2^52: adding it rounds to an integer

GT_HD double quotient(double x) { return std::fma(x, kPinv, kMagic) - kMagic; }

GT_HD double mulmod(double a, double w) {
  double h = a * w;
  double l = std::fma(a, w, -h);
  double q = quotient(h);
  return std::fma(-q, kP, h) + l;
}

// a*w mod P when |a*w| < 2^53 (the product is exact, no low part)
GT_HD double mulmod_small(double a, double w) {
  double h = a * w;
  double q = quotient(h);
  return std::fma(-q, kP, h);
}

GT_HD double reduce(double x) {
  double q = quotient(x);
  return std::fma(-q, kP, x);
}

// x mod 2^32 of an exact integer |x| < 2^52, as uint32
GT_HD uint32_t low32(double x) {
  double q = std::floor(x * 0x1p-32);
  double r = std::fma(-q, 4294967296.0, x);  // in [0, 2^32), exact
  return (uint32_t)r;
}

}  // namespace gt
