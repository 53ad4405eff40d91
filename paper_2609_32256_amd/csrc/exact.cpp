// Host side of the exact merge predicate (fixed-point arithmetic in exact.h):
// the right-hand side floor((2 - 2 tau) * 2^298) as an integer, computed once
// per store.
#include "exact.h"

#include <cmath>

namespace lam {

Big6 exact_threshold(double tau) {
  // floor((2 - 2 tau) * 2^298) = 2^299 - 2 tau 2^298, |tau| = mt * 2^(e - 53), mt < 2^53
  Big6 r = big_shifted(1, 299);
  if (tau == 0.0) return r;
  int e = 0;
  const double f = std::frexp(std::fabs(tau), &e);
  const uint64_t mt = (uint64_t)std::ldexp(f, 53);
  const int sh = e - 53 + 299;   // 2 |tau| 2^298 = mt * 2^sh
  Big6 t;
  if (sh >= 0) {
    t = big_shifted(mt, sh);
  } else {
    const int q = -sh;
    const uint64_t fl = q >= 64 ? 0u : (mt >> q);
    const bool frac = q >= 64 ? (mt != 0) : (mt & ((1ull << q) - 1ull)) != 0;
    // tau > 0: floor(2^299 - y) = 2^299 - ceil(y); tau < 0: floor(2^299 + y) = 2^299 + floor(y)
    t = big_shifted(tau > 0.0 ? fl + (frac ? 1u : 0u) : fl, 0);
  }
  if (tau > 0.0)
    big_sub(r, t);
  else
    big_add(r, t);
  return r;
}

}  // namespace lam
