// Exact decision of the merge predicate sum_d (a_d - b_d)^2 <= 2 - 2 tau
// (Eq. identity, squared form, inclusive) on the exact real values of float32
// rows a, b and the binary64 tau.  Used only for pairs whose binary64 distance
// lies within rounding distance of delta^2.
//
// Every float32 v with |v| < 2^8 is an integer multiple of 2^-149, so
// V = v * 2^149 is an integer below 2^157.  The sum S = sum (A_d - B_d)^2 is
// an integer below 2^(316 + 12) for d <= 4096, and the predicate is
// S <= floor((2 - 2 tau) * 2^298).  Integers are held in 8 little-endian
// 64-bit limbs (512 bits), which covers both sides.
#include <cmath>
#include <cstdint>
#include <cstring>

#include "lam_internal.h"

namespace lam {
namespace {

constexpr int kL = 8;
struct Big {
  uint64_t w[kL] = {};
};

void add(Big& a, const Big& b) {
  unsigned __int128 c = 0;
  for (int i = 0; i < kL; ++i) {
    c += (unsigned __int128)a.w[i] + b.w[i];
    a.w[i] = (uint64_t)c;
    c >>= 64;
  }
}

// a -= b, requires a >= b
void sub(Big& a, const Big& b) {
  uint64_t borrow = 0;
  for (int i = 0; i < kL; ++i) {
    const unsigned __int128 t = (unsigned __int128)a.w[i] - b.w[i] - borrow;
    a.w[i] = (uint64_t)t;
    borrow = (uint64_t)(t >> 64) ? 1 : 0;
  }
}

int cmp(const Big& a, const Big& b) {
  for (int i = kL - 1; i >= 0; --i)
    if (a.w[i] != b.w[i]) return a.w[i] < b.w[i] ? -1 : 1;
  return 0;
}

// m * 2^s for m < 2^64, s >= 0
Big shifted(uint64_t m, int s) {
  Big r;
  const int limb = s / 64, bit = s % 64;
  if (limb < kL) r.w[limb] = m << bit;
  if (bit && limb + 1 < kL) r.w[limb + 1] = m >> (64 - bit);
  return r;
}

// |v| * 2^149 as an integer, and the sign of v
Big fixed149(float v, bool* neg) {
  uint32_t u;
  memcpy(&u, &v, 4);
  *neg = (u >> 31) != 0;
  const uint32_t e = (u >> 23) & 0xffu;
  const uint64_t m = u & 0x7fffffu;
  if (e == 0) return shifted(m, 0);
  return shifted(m | 0x800000u, (int)e - 1);
}

Big mul(const Big& a, const Big& b) {
  Big r;
  for (int i = 0; i < kL; ++i) {
    if (!a.w[i]) continue;
    unsigned __int128 c = 0;
    for (int j = 0; i + j < kL; ++j) {
      c += (unsigned __int128)a.w[i] * b.w[j] + r.w[i + j];
      r.w[i + j] = (uint64_t)c;
      c >>= 64;
    }
  }
  return r;
}

}  // namespace

bool exact_within(const float* a, const float* b, int d, double tau) {
  Big s;
  for (int k = 0; k < d; ++k) {
    bool na, nb;
    Big A = fixed149(a[k], &na), B = fixed149(b[k], &nb);
    Big diff;
    if (na == nb) {
      if (cmp(A, B) >= 0) { diff = A; sub(diff, B); }
      else { diff = B; sub(diff, A); }
    } else {
      diff = A;
      add(diff, B);
    }
    add(s, mul(diff, diff));
  }
  // floor((2 - 2 tau) * 2^298) = 2^299 - 2 tau 2^298, tau = f * 2^e, f in [0.5, 1)
  Big r = shifted(1, 299);
  if (tau != 0.0) {
    int e = 0;
    const double f = std::frexp(std::fabs(tau), &e);
    const uint64_t mt = (uint64_t)std::ldexp(f, 53);   // |tau| = mt * 2^(e - 53)
    const int sh = e - 53 + 299;                        // 2|tau| 2^298 = mt * 2^sh
    Big t;
    if (sh >= 0) {
      t = shifted(mt, sh);
    } else {
      const int q = -sh;
      const uint64_t fl = q >= 64 ? 0u : (mt >> q);
      const bool frac = q >= 64 ? (mt != 0) : (mt & ((1ull << q) - 1ull)) != 0;
      // tau > 0: floor(2^299 - y) = 2^299 - ceil(y);  tau < 0: floor(2^299 + y) = 2^299 + floor(y)
      t = shifted(tau > 0.0 ? fl + (frac ? 1u : 0u) : fl, 0);
    }
    if (tau > 0.0) sub(r, t);
    else add(r, t);
  }
  return cmp(s, r) <= 0;
}

}  // namespace lam
