// Exact Q_eps rounding shared by the quantizer and the banded candidate
// index: q = round-half-even of the exact real x / s, x float32, s = 2 eps
// binary64.
//
// A binary64 estimate q0 = rint(x * (1/s)) is within 2^-20 of x/s for
// |x/s| < 2^31, so the nearest integer is q0 or a neighbour.  The remainder
// e = x - q0*s is formed by one fused multiply-add; round-to-nearest is
// monotone, so RN(e) < eps proves e < eps, RN(e) > eps proves e > eps, and only
// RN(e) == +-eps needs the sign of x - (q0 +- 1/2) s, which a second fused
// multiply-add gives exactly (a single rounding keeps the sign, and zero only
// for an exact zero, i.e. a true tie).
//
// Fast path: p = x * float32(1/s) is within 2^-22 (|p| + 1) of x/s (two
// float32 roundings), so when |p - rint(p)| is at most 1/2 - 2^-21 (|p| + 1) no
// half-integer can separate p from x/s and rint(p) is the exact answer.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace lam {

// Exact round-half-even of x / s, see the file comment.
__device__ __forceinline__ int32_t q_round(float xf, double s, double inv_s, double eps) {
  const double xd = (double)xf;
  double q0 = rint(xd * inv_s);
  const double t = fma(-q0, s, xd);
  if (t > eps) {
    q0 += 1.0;
  } else if (t < -eps) {
    q0 -= 1.0;
  } else if (t == eps) {
    const double d = fma(-(q0 + 0.5), s, xd);
    const bool odd = ((long long)q0 & 1LL) != 0;
    if (d > 0.0 || (d == 0.0 && odd)) q0 += 1.0;
  } else if (t == -eps) {
    const double d = fma(-(q0 - 0.5), s, xd);
    const bool odd = ((long long)q0 & 1LL) != 0;
    if (d < 0.0 || (d == 0.0 && odd)) q0 -= 1.0;
  }
  return (int32_t)q0;
}

// float32 fast path with the binary64 method as the fallback (file comment).
__device__ __forceinline__ int32_t q_round_fast(float x, float inv_s32, double s, double inv_s, double eps) {
  const float p = x * inv_s32;
  const float q0 = rintf(p);
  const float thr = fmaf(-0x1p-21f, fabsf(p), 0.5f - 0x1p-21f);
  if (fabsf(p - q0) <= thr) return (int32_t)q0;
  return q_round(x, s, inv_s, eps);
}

}  // namespace lam
