// The streaming-bandwidth anchor: the triad c = a + s b over float32 arrays,
// which the paper measures on its platform to state every bandwidth figure
// against a measured ceiling as well as the published one (Appendix
// "Measured hardware constants", Table "anchors": 3 x 512 MB arrays).  Bytes
// moved are 12 per element (two reads, one write).
#include <hip/hip_ext.h>

#include <algorithm>

#include "lam_internal.h"

namespace lam {
namespace {

constexpr int kTriadThreads = 256;

typedef float f4 __attribute__((ext_vector_type(4)));

// One 16-byte vector per thread over a grid that covers the arrays once,
// loads and stores marked non-temporal (each element is touched once): the
// fastest of the layouts measured on MI355X (grid-stride loops with 2 to 16 K
// workgroups and 1 to 8 vectors per trip, plain or non-temporal, and
// contiguous ranges per workgroup were 5 to 30 % slower).  The tail of n % 4
// elements is done by thread 0.
__global__ __launch_bounds__(kTriadThreads) void k_triad(const float* __restrict__ a, const float* __restrict__ b,
                                                         float* __restrict__ c, int64_t n, float s) {
  const int64_t n4 = n / 4;
  const int64_t i = (int64_t)blockIdx.x * kTriadThreads + threadIdx.x;
  if (i < n4) {
    const f4 x = __builtin_nontemporal_load(reinterpret_cast<const f4*>(a) + i);
    const f4 y = __builtin_nontemporal_load(reinterpret_cast<const f4*>(b) + i);
    __builtin_nontemporal_store(x + s * y, reinterpret_cast<f4*>(c) + i);
  }
  if (blockIdx.x == 0 && threadIdx.x == 0)
    for (int64_t t = n4 * 4; t < n; ++t) c[t] = a[t] + s * b[t];
}

}  // namespace

lam_status launch_triad(lam_ctx* ctx, const float* a, const float* b, float* c, int64_t n, float s) {
  if (n == 0) return LAM_OK;
  hipEvent_t e0, e1;   // timed by the launch itself when profiled ("triad")
  LAM_TRY(prof_launch_events(ctx, "triad", &e0, &e1));
  const int64_t n4 = std::max<int64_t>(n / 4, 1);
  const int64_t grid = (n4 + kTriadThreads - 1) / kTriadThreads;
  LAM_CHECK(grid < (1LL << 31), LAM_EINVAL, "n too large for one triad launch");
  hipExtLaunchKernelGGL(k_triad, dim3((unsigned)grid), dim3(kTriadThreads), 0, ctx->stream, e0, e1, 0, a, b, c, n, s);
  LAM_HIP(hipGetLastError());
  return LAM_OK;
}

}  // namespace lam
