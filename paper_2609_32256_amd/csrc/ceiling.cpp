// Removal ceiling and the measured bracket on the delta-entropy (Theorem
// "removal ceiling", Corollary "measured bracket"): greedy first-occurrence run
// over the same stream at radius delta (threshold tau) and at radius 2 delta
// (threshold 4 tau - 3).  The second pass returns a 2 delta-packing, whose size
// bounds the retained size of any delta-bounded compactor from below, so
//   rho*(delta) <= 1 - |R(2 delta)| / |S|   and
//   log2 |R(2 delta)| <= H_delta(S) <= log2 |R(delta)|.
// Both passes are ordinary ingests (exact decisions); this file only runs them.
#include <algorithm>
#include <cmath>

#include "lam_internal.h"

extern "C" {

lam_status lam_removal_ceiling(lam_ctx* ctx, const float* x_dev, int64_t n, int32_t dim, double tau,
                               int64_t batch, lam_ceiling_stats* out) {
  LAM_CHECK(ctx != nullptr && out != nullptr, LAM_EINVAL, "ctx or out is NULL");
  LAM_CHECK(n > 0 && x_dev != nullptr, LAM_EINVAL, "need at least one row");
  LAM_CHECK(batch > 0, LAM_EINVAL, "batch must be positive");
  LAM_CHECK(std::isfinite(tau) && tau > 0.5 && tau <= 1.0, LAM_EINVAL,
            "tau must be in (1/2, 1] so that the 2 delta pass has 4 tau - 3 in (-1, 1]");
  // exact: 4 tau is a power-of-two scaling and 4 tau - 3 is exact by Sterbenz
  // (4 tau and 3 lie within a factor of two of each other)
  const double tau2 = 4.0 * tau - 3.0;
  lam_store* s1 = nullptr;
  lam_store* s2 = nullptr;
  lam_status s = lam_store_create(ctx, dim, tau, n, &s1);
  if (s == LAM_OK) s = lam_store_create(ctx, dim, tau2, n, &s2);
  // the representatives are not needed: both passes write them to one scratch slot
  if (s == LAM_OK) s = ctx->scratch[lam::kScratchCeilingRep].ensure((size_t)std::min<int64_t>(batch, n) * 8);
  int64_t* rep = ctx->scratch[lam::kScratchCeilingRep].as<int64_t>();
  for (int64_t b0 = 0; s == LAM_OK && b0 < n; b0 += batch) {
    const int64_t nb = std::min<int64_t>(batch, n - b0);
    s = lam_dedup_ingest(ctx, s1, x_dev + b0 * dim, nb, rep, nullptr, nullptr);
    if (s == LAM_OK) s = lam_dedup_ingest(ctx, s2, x_dev + b0 * dim, nb, rep, nullptr, nullptr);
  }
  lam_store_info i1{}, i2{};
  if (s == LAM_OK) s = lam_store_get_info(s1, &i1);
  if (s == LAM_OK) s = lam_store_get_info(s2, &i2);
  lam_store_destroy(s1);
  lam_store_destroy(s2);
  if (s != LAM_OK) return s;
  lam_ceiling_stats r{};
  r.n = n;
  r.kept = i1.size;
  r.kept_2delta = i2.size;
  r.tau = tau;
  r.tau_2delta = tau2;
  r.removal = 1.0 - (double)i1.size / (double)n;
  r.ceiling = 1.0 - (double)i2.size / (double)n;
  r.frac_of_ceiling = r.ceiling > 0.0 ? r.removal / r.ceiling : 0.0;
  r.bits_lo = std::log2((double)i2.size);
  r.bits_hi = std::log2((double)i1.size);
  r.delta_hat = i1.delta_hat_run;
  r.delta_hat_2delta = i2.delta_hat_run;
  *out = r;
  return LAM_OK;
}

}  // extern "C"
