// Exact fixed-point arithmetic for the merge predicate
//   sum_d (a_d - b_d)^2 <= 2 - 2 tau        (Eq. identity, squared form, inclusive)
// on the exact real values of float32 rows a, b and the binary64 tau.  It is
// used only for pairs whose binary64 distance lies within rounding distance of
// delta^2, by one wave per pair on the device; the right-hand side is formed
// once per store on the host.
//
// Every float32 v with |v| < 2^8 (the ingest rejects larger coordinates) is an
// integer multiple of 2^-149, so V = |v| * 2^149 is an integer below 2^157 and
// fits three 64-bit limbs.  A squared difference is below 2^316 and a sum over
// at most 2^16 coordinates below 2^332, within six limbs (384 bits); the right
// side floor((2 - 2 tau) * 2^298) < 2^300 uses the same six limbs.  Limbs are
// little-endian.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace lam {

constexpr int kExactLimbs = 6;

struct Big6 {
  uint64_t w[kExactLimbs];
};

__host__ __device__ inline void big_zero(Big6& a) {
#pragma unroll
  for (int i = 0; i < kExactLimbs; ++i) a.w[i] = 0u;
}

// a += b (no overflow for the magnitudes above)
__host__ __device__ inline void big_add(Big6& a, const Big6& b) {
  uint64_t carry = 0u;
#pragma unroll
  for (int i = 0; i < kExactLimbs; ++i) {
    const uint64_t s = a.w[i] + b.w[i];
    const uint64_t c1 = s < a.w[i] ? 1u : 0u;
    const uint64_t t = s + carry;
    const uint64_t c2 = t < s ? 1u : 0u;
    a.w[i] = t;
    carry = c1 + c2;
  }
}

// a -= b, requires a >= b
__host__ __device__ inline void big_sub(Big6& a, const Big6& b) {
  uint64_t borrow = 0u;
#pragma unroll
  for (int i = 0; i < kExactLimbs; ++i) {
    const uint64_t d = a.w[i] - b.w[i];
    const uint64_t b1 = a.w[i] < b.w[i] ? 1u : 0u;
    const uint64_t t = d - borrow;
    const uint64_t b2 = d < borrow ? 1u : 0u;
    a.w[i] = t;
    borrow = b1 + b2;
  }
}

__host__ __device__ inline int big_cmp(const Big6& a, const Big6& b) {
#pragma unroll
  for (int i = kExactLimbs - 1; i >= 0; --i)
    if (a.w[i] != b.w[i]) return a.w[i] < b.w[i] ? -1 : 1;
  return 0;
}

// m * 2^s for m < 2^64, 0 <= s < 384 - 64.  Every limb is selected with a
// constant index, so the limbs stay in registers (a run-time index would put
// the array in scratch memory).
__host__ __device__ inline Big6 big_shifted(uint64_t m, int s) {
  const int limb = s >> 6, bit = s & 63;
  const uint64_t lo = m << bit;
  const uint64_t hi = bit != 0 ? m >> (64 - bit) : 0u;
  Big6 r;
#pragma unroll
  for (int i = 0; i < kExactLimbs; ++i) r.w[i] = (i == limb ? lo : 0u) | (i == limb + 1 ? hi : 0u);
  return r;
}

__host__ __device__ inline uint64_t mul_hi64(uint64_t a, uint64_t b) {
#if defined(__HIP_DEVICE_COMPILE__)
  return __umul64hi(a, b);
#else
  return (uint64_t)(((unsigned __int128)a * b) >> 64);
#endif
}

// |v| * 2^149 as an integer (float32 bit pattern u, |v| < 2^8)
__host__ __device__ inline Big6 big_fixed149(uint32_t u) {
  const uint32_t e = (u >> 23) & 0xffu;
  const uint64_t m = u & 0x7fffffu;
  if (e == 0u) return big_shifted(m, 0);
  return big_shifted(m | 0x800000u, (int)e - 1);
}

// (a_d - b_d)^2 * 2^298, exactly, for float32 bit patterns ua, ub
__host__ __device__ inline Big6 big_sq_diff(uint32_t ua, uint32_t ub) {
  Big6 A = big_fixed149(ua), B = big_fixed149(ub);
  Big6 d;
  if ((ua >> 31) == (ub >> 31)) {
    if (big_cmp(A, B) >= 0) {
      d = A;
      big_sub(d, B);
    } else {
      d = B;
      big_sub(d, A);
    }
  } else {
    d = A;
    big_add(d, B);
  }
  // d < 2^158 lives in limbs 0..2; the square in limbs 0..5
  Big6 r;
  big_zero(r);
#pragma unroll
  for (int i = 0; i < 3; ++i) {
    uint64_t carry = 0u;
#pragma unroll
    for (int j = 0; j < 3; ++j) {
      const uint64_t lo = d.w[i] * d.w[j];
      const uint64_t hi = mul_hi64(d.w[i], d.w[j]);
      // r[i+j] += lo + carry, the overflow and hi go to the next limb
      uint64_t s = r.w[i + j] + lo;
      uint64_t c = s < lo ? 1u : 0u;
      const uint64_t t = s + carry;
      c += t < s ? 1u : 0u;
      r.w[i + j] = t;
      carry = hi + c;   // d_i d_j + r + carry < 2^128, so this high word cannot wrap
    }
#pragma unroll
    for (int k = i + 3; k < kExactLimbs; ++k) {   // constant indices: the limbs stay in registers
      const uint64_t s = r.w[k] + carry;
      carry = s < carry ? 1u : 0u;
      r.w[k] = s;
    }
  }
  return r;
}

// floor((2 - 2 tau) * 2^298) for a binary64 tau in (-1, 1] (host only)
Big6 exact_threshold(double tau);

}  // namespace lam
