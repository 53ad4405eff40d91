// The C ABI of liblam (include/lam.h): argument checks, context and store
// lifetime, the scratch arena, per-kernel event timing, and the Q_eps entry
// points.  The dedup and scoring pipelines live in dedup.hip and score.hip.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <new>

#include "lam_internal.h"

namespace lam {

static thread_local char g_err[512] = "";

void set_error(const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof g_err, fmt, ap);
  va_end(ap);
}

lam_status DevBuf::ensure(size_t need) {
  if (need <= bytes && p != nullptr) return LAM_OK;
  release();
  size_t sz = need < 256 ? 256 : need;
  sz = (sz + 255) & ~size_t(255);
  hipError_t e = hipMalloc(&p, sz);
  if (e != hipSuccess) {
    p = nullptr;
    bytes = 0;
    set_error("hipMalloc(%zu) failed: %s", sz, hipGetErrorString(e));
    return LAM_ENOMEM;
  }
  bytes = sz;
  return LAM_OK;
}

void DevBuf::release() {
  if (p) (void)hipFree(p);
  p = nullptr;
  bytes = 0;
}

// Makes the context's device current for the scope of one API call.
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

// Whether launches of kernel `name` are timed: every kernel, or those named in
// the comma-separated list of lam_ctx_profile_only.
static bool prof_selected(const lam_ctx* ctx, const char* name) {
  if (!ctx->profiling) return false;
  if (ctx->prof_only.empty()) return true;
  const std::string& l = ctx->prof_only;
  const size_t n = strlen(name);
  for (size_t p = 0; p <= l.size();) {
    size_t e = l.find(',', p);
    if (e == std::string::npos) e = l.size();
    if (e - p == n && l.compare(p, n, name) == 0) return true;
    p = e + 1;
  }
  return false;
}

lam_status prof_begin(lam_ctx* ctx, const char* name, size_t* slot) {
  *slot = (size_t)-1;
  if (!prof_selected(ctx, name)) return LAM_OK;
  ProfRec r{name, nullptr, nullptr};
  for (hipEvent_t* ev : {&r.a, &r.b}) {
    if (!ctx->event_pool.empty()) {
      *ev = ctx->event_pool.back();
      ctx->event_pool.pop_back();
    } else {
      // timing events only: no system-scope fence (nothing on the host
      // reads device memory through them), which would flush the L2 at each
      // record and hold up the next kernel
      LAM_HIP(hipEventCreateWithFlags(ev, hipEventDisableSystemFence));
    }
  }
  LAM_HIP(hipEventRecord(r.a, ctx->stream));
  ctx->prof.push_back(r);
  *slot = ctx->prof.size() - 1;
  return LAM_OK;
}

// Timing of one launch by the launch itself: the two events go to
// hipExtLaunchKernel, which stamps them at the kernel's start and end, so no
// marker packets sit between this kernel and its neighbours.  Both stay null
// unless this kernel is being profiled.
lam_status prof_launch_events(lam_ctx* ctx, const char* name, hipEvent_t* start, hipEvent_t* stop) {
  *start = *stop = nullptr;
  if (!prof_selected(ctx, name)) return LAM_OK;
  ProfRec r{name, nullptr, nullptr};
  for (hipEvent_t* ev : {&r.a, &r.b}) {
    if (!ctx->event_pool.empty()) {
      *ev = ctx->event_pool.back();
      ctx->event_pool.pop_back();
    } else {
      LAM_HIP(hipEventCreateWithFlags(ev, hipEventDisableSystemFence));
    }
  }
  ctx->prof.push_back(r);
  *start = r.a;
  *stop = r.b;
  return LAM_OK;
}

lam_status prof_end(lam_ctx* ctx, size_t slot) {
  if (slot >= ctx->prof.size()) return LAM_OK;
  LAM_HIP(hipEventRecord(ctx->prof[slot].b, ctx->stream));
  return LAM_OK;
}

// Clears the context's status words with a kernel (not a memset node), so that
// the sequence stays valid inside a captured stream.
__global__ void k_zero_words(uint32_t* p, int n) {
  int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = 0u;
}

lam_status clear_flags(lam_ctx* ctx) {
  ctx->flags_zero = false;   // the caller's kernels write them next
  hipLaunchKernelGGL(k_zero_words, dim3(1), dim3(64), 0, ctx->stream,
                     reinterpret_cast<uint32_t*>(ctx->flags_dev), (int)(sizeof(DevFlags) / 4));
  LAM_HIP(hipGetLastError());
  return LAM_OK;
}

lam_status read_flags(lam_ctx* ctx) {
  LAM_HIP(hipMemcpyAsync(ctx->flags_host, ctx->flags_dev, sizeof(DevFlags), hipMemcpyDeviceToHost, ctx->stream));
  LAM_HIP(hipStreamSynchronize(ctx->stream));
  return LAM_OK;
}

// Shared body of lam_quantize and lam_store_quantize.
// known_valid: the caller knows every |x| to be finite and at most a positive
// absmax (a store's rows against the store's exact maximum), so no status word
// can be set and the encode is not waited for.
lam_status quantize_impl(lam_ctx* ctx, const float* x, int64_t n, double eps, float absmax, int mode,
                         uint32_t* codes, uint64_t cap, lam_qparams* out, DevBuf* grow_into,
                         bool store_path = false, bool known_valid = false) {
  lam_qparams p{};
  // argument checks that do not depend on the data
  LAM_TRY(qeps_plan_host(eps, 0.0f, mode, n, &p));
  LAM_CHECK(std::isfinite(absmax), LAM_EINVAL, "absmax must be finite");
  if (!ctx->flags_zero) LAM_TRY(clear_flags(ctx));   // (already zero after an ingest or a clean quantize)
  ctx->flags_zero = false;
  float a = absmax;
  if (!(absmax > 0.0f)) {
    LAM_TRY(launch_absmax(ctx, x, n, &ctx->flags_dev->absmax_bits, store_path ? "store_absmax" : "qeps_absmax"));
    LAM_TRY(read_flags(ctx));
    const uint32_t bits = ctx->flags_host->absmax_bits;
    LAM_CHECK(bits < 0x7f800000u, LAM_EINVAL, "input holds NaN or Inf");
    memcpy(&a, &bits, 4);
  }
  LAM_TRY(qeps_plan_host(eps, a, mode, n, &p));
  if (grow_into) {
    LAM_TRY(grow_into->ensure(p.code_bytes));
    codes = grow_into->as<uint32_t>();
    cap = grow_into->bytes;
  }
  LAM_CHECK(codes != nullptr || n == 0, LAM_EINVAL, "codes buffer is NULL");
  LAM_CHECK(cap >= p.code_bytes, LAM_EINVAL, "codes capacity %llu < %llu bytes needed",
            (unsigned long long)cap, (unsigned long long)p.code_bytes);
  LAM_TRY(launch_encode(ctx, x, n, p, codes, &ctx->flags_dev->nonfinite, store_path ? "store_encode" : "qeps_encode"));
  if (known_valid && absmax > 0.0f) {
    ctx->flags_zero = true;   // cleared above and left untouched by valid input
    if (out) *out = p;
    return LAM_OK;
  }
  LAM_TRY(read_flags(ctx));
  LAM_CHECK(ctx->flags_host->nonfinite == 0, LAM_EINVAL, "input holds NaN or Inf (%u elements)",
            ctx->flags_host->nonfinite);
  LAM_CHECK(ctx->flags_host->out_of_range == 0, LAM_ERANGE, "%u elements exceed the declared absmax %g",
            ctx->flags_host->out_of_range, (double)a);
  // a declared absmax and valid input leave every status word at zero, which
  // the next call need not clear again (the host copy is exact: the stream was
  // synchronised after the encode)
  static const DevFlags kZero{};
  ctx->flags_zero = memcmp(ctx->flags_host, &kZero, sizeof(DevFlags)) == 0;
  if (out) *out = p;
  return LAM_OK;
}

}  // namespace lam

using namespace lam;

extern "C" {

int lam_abi_version(void) { return LAM_ABI_VERSION; }

const char* lam_status_name(lam_status s) {
  switch (s) {
    case LAM_OK: return "LAM_OK";
    case LAM_EINVAL: return "LAM_EINVAL";
    case LAM_ERANGE: return "LAM_ERANGE";
    case LAM_ENOMEM: return "LAM_ENOMEM";
    case LAM_ECAPACITY: return "LAM_ECAPACITY";
    case LAM_EDEVICE: return "LAM_EDEVICE";
    case LAM_ESTATE: return "LAM_ESTATE";
  }
  return "LAM_UNKNOWN";
}

const char* lam_last_error(void) { return g_err; }

lam_status lam_ctx_create(int device, void* hip_stream, lam_ctx** out) {
  LAM_CHECK(out != nullptr, LAM_EINVAL, "out is NULL");
  *out = nullptr;
  int ndev = 0;
  LAM_HIP(hipGetDeviceCount(&ndev));
  LAM_CHECK(device >= 0 && device < ndev, LAM_EINVAL, "device %d out of range (%d devices)", device, ndev);
  DeviceGuard g(device);
  LAM_CHECK(g.ok, LAM_EDEVICE, "hipSetDevice(%d) failed", device);
  lam_ctx* c = new (std::nothrow) lam_ctx();
  LAM_CHECK(c != nullptr, LAM_ENOMEM, "out of host memory");
  c->device = device;
  c->stream = static_cast<hipStream_t>(hip_stream);
  if (hipMalloc(&c->flags_dev, sizeof(DevFlags)) != hipSuccess ||
      hipHostMalloc(&c->flags_host, sizeof(DevFlags), hipHostMallocCoherent) != hipSuccess ||
      hipHostGetDevicePointer(reinterpret_cast<void**>(&c->flags_host_dev), c->flags_host, 0) != hipSuccess) {
    if (c->flags_dev) (void)hipFree(c->flags_dev);
    if (c->flags_host) (void)hipHostFree(c->flags_host);
    delete c;
    set_error("could not allocate the context status words");
    return LAM_ENOMEM;
  }
  memset(c->flags_host, 0, sizeof(DevFlags));
  // the allocation-free scoring call's workspace on this device (once per device)
  const lam_status ns = noalloc_setup(device);
  if (ns != LAM_OK) {
    lam_ctx_destroy(c);
    return ns;
  }
  *out = c;
  return LAM_OK;
}

void lam_ctx_destroy(lam_ctx* ctx) {
  if (!ctx) return;
  DeviceGuard g(ctx->device);
  (void)hipStreamSynchronize(ctx->stream);
  for (auto& b : ctx->scratch) b.release();
  for (auto& r : ctx->prof) {
    (void)hipEventDestroy(r.a);
    (void)hipEventDestroy(r.b);
  }
  for (auto e : ctx->event_pool) (void)hipEventDestroy(e);
  if (ctx->flags_dev) (void)hipFree(ctx->flags_dev);
  if (ctx->flags_host) (void)hipHostFree(ctx->flags_host);
  delete ctx;
}

lam_status lam_ctx_synchronize(lam_ctx* ctx) {
  LAM_CHECK(ctx != nullptr, LAM_EINVAL, "ctx is NULL");
  DeviceGuard g(ctx->device);
  LAM_HIP(hipStreamSynchronize(ctx->stream));
  return LAM_OK;
}

lam_status lam_ctx_profile(lam_ctx* ctx, int enable) {
  LAM_CHECK(ctx != nullptr, LAM_EINVAL, "ctx is NULL");
  ctx->profiling = enable != 0;
  return LAM_OK;
}

lam_status lam_ctx_set_screen_tile(lam_ctx* ctx, int policy) {
  LAM_CHECK(ctx != nullptr, LAM_EINVAL, "ctx is NULL");
  LAM_CHECK(policy == LAM_SCREEN_TILE_AUTO || policy == LAM_SCREEN_TILE_SMALL || policy == LAM_SCREEN_TILE_LARGE,
            LAM_EINVAL, "screen tile policy %d is not one of 0, 1, 2", policy);
  ctx->screen_tile = policy;
  return LAM_OK;
}

lam_status lam_ctx_profile_only(lam_ctx* ctx, const char* kernel) {
  LAM_CHECK(ctx != nullptr, LAM_EINVAL, "ctx is NULL");
  ctx->prof_only = kernel ? kernel : "";
  return LAM_OK;
}

lam_status lam_ctx_profile_reset(lam_ctx* ctx) {
  LAM_CHECK(ctx != nullptr, LAM_EINVAL, "ctx is NULL");
  DeviceGuard g(ctx->device);
  LAM_HIP(hipStreamSynchronize(ctx->stream));
  for (auto& r : ctx->prof) {
    ctx->event_pool.push_back(r.a);
    ctx->event_pool.push_back(r.b);
  }
  ctx->prof.clear();
  return LAM_OK;
}

lam_status lam_ctx_profile_read(lam_ctx* ctx, const char* kernel, double* total_ms, int64_t* launches) {
  LAM_CHECK(ctx != nullptr && kernel != nullptr, LAM_EINVAL, "ctx or kernel name is NULL");
  DeviceGuard g(ctx->device);
  LAM_HIP(hipStreamSynchronize(ctx->stream));
  double sum = 0.0;
  int64_t cnt = 0;
  for (auto& r : ctx->prof) {
    if (strcmp(r.name, kernel) != 0) continue;
    float ms = 0.0f;
    LAM_HIP(hipEventElapsedTime(&ms, r.a, r.b));
    sum += ms;
    ++cnt;
  }
  if (total_ms) *total_ms = sum;
  if (launches) *launches = cnt;
  return LAM_OK;
}

lam_status lam_qeps_plan(double eps, float absmax, int mode, int64_t n, lam_qparams* out) {
  return qeps_plan_host(eps, absmax, mode, n, out);
}

lam_status lam_quantize(lam_ctx* ctx, const float* x_dev, int64_t n, double eps, float absmax, int mode,
                        uint32_t* codes_dev, uint64_t codes_cap_bytes, lam_qparams* out) {
  LAM_CHECK(ctx != nullptr, LAM_EINVAL, "ctx is NULL");
  LAM_CHECK(n >= 0, LAM_EINVAL, "n must be >= 0");
  LAM_CHECK(x_dev != nullptr || n == 0, LAM_EINVAL, "x is NULL");
  LAM_CHECK(((uintptr_t)x_dev & 3u) == 0 && ((uintptr_t)codes_dev & 3u) == 0, LAM_EINVAL,
            "x and codes must be 4-byte aligned");
  DeviceGuard g(ctx->device);
  return quantize_impl(ctx, x_dev, n, eps, absmax, mode, codes_dev, codes_cap_bytes, out, nullptr);
}

lam_status lam_quantize_async(lam_ctx* ctx, const float* x_dev, int64_t n, double eps, float absmax, int mode,
                              uint32_t* codes_dev, uint64_t codes_cap_bytes, uint32_t* status_dev,
                              lam_qparams* out) {
  LAM_CHECK(ctx != nullptr, LAM_EINVAL, "ctx is NULL");
  LAM_CHECK(n >= 0, LAM_EINVAL, "n must be >= 0");
  LAM_CHECK(x_dev != nullptr || n == 0, LAM_EINVAL, "x is NULL");
  LAM_CHECK(status_dev != nullptr, LAM_EINVAL, "status is NULL");
  LAM_CHECK(((uintptr_t)x_dev & 3u) == 0 && ((uintptr_t)codes_dev & 3u) == 0 && ((uintptr_t)status_dev & 3u) == 0,
            LAM_EINVAL, "x, codes and status must be 4-byte aligned");
  LAM_CHECK(std::isfinite(absmax) && absmax > 0.0f, LAM_EINVAL, "an asynchronous encode needs a declared absmax > 0");
  lam_qparams p{};
  LAM_TRY(qeps_plan_host(eps, absmax, mode, n, &p));
  LAM_CHECK(codes_dev != nullptr || n == 0, LAM_EINVAL, "codes buffer is NULL");
  LAM_CHECK(codes_cap_bytes >= p.code_bytes, LAM_EINVAL, "codes capacity %llu < %llu bytes needed",
            (unsigned long long)codes_cap_bytes, (unsigned long long)p.code_bytes);
  DeviceGuard g(ctx->device);
  LAM_TRY(launch_encode(ctx, x_dev, n, p, codes_dev, status_dev, "qeps_encode"));
  if (out) *out = p;
  return LAM_OK;
}

lam_status lam_dequantize(lam_ctx* ctx, const uint32_t* codes_dev, const lam_qparams* p, float* xhat_dev) {
  LAM_CHECK(ctx != nullptr && p != nullptr, LAM_EINVAL, "ctx or params is NULL");
  LAM_CHECK(p->n >= 0 && p->bits >= 1 && p->bits <= 32, LAM_EINVAL, "bad params (n=%lld, bits=%d)",
            (long long)p->n, p->bits);
  LAM_CHECK(std::isfinite(p->step) && p->step > 0.0, LAM_EINVAL, "bad step");
  LAM_CHECK(p->code_bytes == 4u * (((uint64_t)p->n * (uint64_t)p->bits + 31u) / 32u), LAM_EINVAL,
            "code_bytes does not match n and bits");
  LAM_CHECK((codes_dev != nullptr && xhat_dev != nullptr) || p->n == 0, LAM_EINVAL, "NULL buffer");
  LAM_CHECK(((uintptr_t)xhat_dev & 3u) == 0 && ((uintptr_t)codes_dev & 3u) == 0, LAM_EINVAL,
            "buffers must be 4-byte aligned");
  DeviceGuard g(ctx->device);
  return launch_decode(ctx, codes_dev, *p, xhat_dev);
}

namespace {

lam_status store_create(lam_ctx* ctx, int32_t dim, double tau, int64_t capacity, double eps_band,
                        int32_t band_width, lam_store** out) {
  LAM_CHECK(ctx != nullptr && out != nullptr, LAM_EINVAL, "ctx or out is NULL");
  *out = nullptr;
  LAM_CHECK(dim > 0 && dim % 32 == 0 && dim <= 4096, LAM_EINVAL, "dim must be a multiple of 32 in [32, 4096]");
  LAM_CHECK(std::isfinite(tau) && tau > -1.0 && tau <= 1.0, LAM_EINVAL, "tau must be in (-1, 1]");
  LAM_CHECK(capacity > 0 && capacity < (1LL << 31), LAM_EINVAL, "capacity must be in [1, 2^31)");
  if (band_width > 0) {
    LAM_CHECK(dim % band_width == 0, LAM_EINVAL, "band_width must divide dim");
    LAM_CHECK(std::isfinite(eps_band) && eps_band >= 0x1p-23 && eps_band <= 0x1p40, LAM_EINVAL,
              "eps_band must be in [2^-23, 2^40]");
    LAM_CHECK(capacity * (int64_t)(dim / band_width) < (1LL << 31), LAM_EINVAL,
              "capacity * (dim / band_width) must be below 2^31");
  }
  DeviceGuard g(ctx->device);
  lam_store* st = new (std::nothrow) lam_store();
  LAM_CHECK(st != nullptr, LAM_ENOMEM, "out of host memory");
  st->ctx = ctx;
  st->dim = dim;
  st->tau = tau;
  st->d2 = 2.0 - 2.0 * tau;
  st->capacity = capacity;
  if (band_width > 0) {
    st->lsh_r = band_width;
    st->lsh_nb = dim / band_width;
    st->lsh_eps = eps_band;
  }
  lam_status s = store_alloc(st);
  if (s != LAM_OK) {
    store_free(st);
    delete st;
    return s;
  }
  *out = st;
  return LAM_OK;
}

}  // namespace

lam_status lam_store_create(lam_ctx* ctx, int32_t dim, double tau, int64_t capacity, lam_store** out) {
  return store_create(ctx, dim, tau, capacity, 0.0, 0, out);
}

lam_status lam_store_create_banded(lam_ctx* ctx, int32_t dim, double tau, int64_t capacity, double eps_band,
                                   int32_t band_width, lam_store** out) {
  LAM_CHECK(band_width > 0, LAM_EINVAL, "band_width must be positive");
  return store_create(ctx, dim, tau, capacity, eps_band, band_width, out);
}

void lam_store_destroy(lam_store* st) {
  if (!st) return;
  DeviceGuard g(st->ctx->device);
  (void)hipStreamSynchronize(st->ctx->stream);
  store_free(st);
  delete st;
}

lam_status lam_store_get_info(const lam_store* st, lam_store_info* out) {
  LAM_CHECK(st != nullptr && out != nullptr, LAM_EINVAL, "store or out is NULL");
  {
    DeviceGuard g(st->ctx->device);
    LAM_TRY(store_settle(const_cast<lam_store*>(st)));
  }
  lam_store_info i{};
  i.size = st->size;
  i.capacity = st->capacity;
  i.n_seen = st->n_seen;
  i.dim = st->dim;
  i.quantized = (st->codes != nullptr && st->coded_rows == st->size) ? 1 : 0;
  i.tau = st->tau;
  i.delta_hat_run = st->delta_hat_run;
  i.q = st->q;
  *out = i;
  return LAM_OK;
}

lam_status lam_dedup_ingest(lam_ctx* ctx, lam_store* st, const float* x_dev, int64_t n, int64_t* rep_dev,
                            float* max_cos_dev, lam_ingest_stats* stats) {
  LAM_CHECK(ctx != nullptr && st != nullptr, LAM_EINVAL, "ctx or store is NULL");
  LAM_CHECK(st->ctx->device == ctx->device, LAM_EINVAL, "store belongs to another device");
  LAM_CHECK(n >= 0, LAM_EINVAL, "n must be >= 0");
  LAM_CHECK((x_dev != nullptr && rep_dev != nullptr) || n == 0, LAM_EINVAL, "x or rep is NULL");
  LAM_CHECK(((uintptr_t)x_dev & 15u) == 0, LAM_EINVAL, "x must be 16-byte aligned");
  LAM_CHECK(n <= st->capacity, LAM_ECAPACITY, "a batch of %lld rows exceeds the store's capacity %lld",
            (long long)n, (long long)st->capacity);
  DeviceGuard g(ctx->device);
  return dedup_ingest(ctx, st, x_dev, n, rep_dev, max_cos_dev, stats);
}

lam_status lam_store_quantize(lam_ctx* ctx, lam_store* st, double eps, float absmax, int mode,
                              lam_qparams* out) {
  LAM_CHECK(ctx != nullptr && st != nullptr, LAM_EINVAL, "ctx or store is NULL");
  DeviceGuard g(ctx->device);
  // the store's max |x| and max ||x||^2 / 2 are kept by the appends, so
  // neither needs a pass over the rows here
  LAM_TRY(store_maxima(st));
  const int64_t n = st->size * (int64_t)st->dim;
  DevBuf holder{st->codes, st->codes_cap};
  lam_qparams p{};
  st->blk_rows = -1;   // any block encoding describes the previous codes
  float a = absmax;
  if (!(absmax > 0.0f) && st->absmax_bits != 0u) memcpy(&a, &st->absmax_bits, 4);   // the exact maximum
  if (absmax > 0.0f && std::isfinite(absmax)) {
    // the rows were checked finite at ingest; against a declared absmax the
    // store's exact maximum decides ERANGE before any code is written
    uint32_t ab = 0u;
    memcpy(&ab, &absmax, 4);
    if (st->absmax_bits > ab) {
      float mx = 0.0f;
      memcpy(&mx, &st->absmax_bits, 4);
      st->coded_rows = -1;
      LAM_CHECK(false, LAM_ERANGE, "the store's largest |x| (%g) exceeds the declared absmax %g", (double)mx,
                (double)absmax);
    }
  }
  lam_status s = quantize_impl(ctx, st->x32, n, eps, a, mode, nullptr, 0, &p, &holder, true, true);
  st->codes = holder.as<uint32_t>();
  st->codes_cap = holder.bytes;
  if (s != LAM_OK) {
    st->coded_rows = -1;
    return s;
  }
  st->q = p;
  st->coded_rows = st->size;
  st->hn_max = st->hnmax_bits;
  if (out) *out = p;
  return LAM_OK;
}

lam_status lam_store_clear(lam_ctx* ctx, lam_store* st) {
  LAM_CHECK(ctx != nullptr && st != nullptr, LAM_EINVAL, "ctx or store is NULL");
  DeviceGuard g(ctx->device);
  // the device bookkeeping is zeroed by the next ingest's first kernel (no
  // launch of its own); until then nothing on the device reads it
  st->meta_reset = true;
  LAM_TRY(lsh_reset(ctx, st, 0));
  st->pending = false;   // errors of earlier calls that did not wait are dropped with the contents
  st->blk_rows = -1;
  st->size_ub = 0;
  st->size = 0;
  st->n_seen = 0;
  st->maxima_known = false;
  st->delta_hat_run = 0.0;
  st->coded_rows = -1;
  st->q = lam_qparams{};
  return LAM_OK;
}

lam_status lam_store_dequantize(lam_ctx* ctx, const lam_store* st, float* xhat_dev) {
  LAM_CHECK(ctx != nullptr && st != nullptr, LAM_EINVAL, "ctx or store is NULL");
  {
    DeviceGuard g(ctx->device);
    LAM_TRY(store_settle(const_cast<lam_store*>(st)));
  }
  LAM_CHECK(st->codes != nullptr && st->coded_rows == st->size, LAM_ESTATE, "store is not quantized");
  LAM_CHECK(xhat_dev != nullptr || st->size == 0, LAM_EINVAL, "xhat is NULL");
  LAM_CHECK(((uintptr_t)xhat_dev & 3u) == 0, LAM_EINVAL, "xhat must be 4-byte aligned");
  DeviceGuard g(ctx->device);
  return launch_decode(ctx, st->codes, st->q, xhat_dev, "store_decode");
}

lam_status lam_store_export(lam_ctx* ctx, const lam_store* st, int64_t* ids_dev, uint32_t* codes_dev,
                            uint64_t codes_cap_bytes) {
  LAM_CHECK(ctx != nullptr && st != nullptr, LAM_EINVAL, "ctx or store is NULL");
  DeviceGuard g(ctx->device);
  LAM_TRY(store_settle(const_cast<lam_store*>(st)));
  if (ids_dev && st->size > 0)
    LAM_HIP(hipMemcpyAsync(ids_dev, st->ids, (size_t)st->size * 8, hipMemcpyDeviceToDevice, ctx->stream));
  if (codes_dev) {
    LAM_CHECK(st->codes != nullptr && st->coded_rows == st->size, LAM_ESTATE, "store is not quantized");
    LAM_CHECK(codes_cap_bytes >= st->q.code_bytes, LAM_EINVAL, "codes capacity too small");
    if (st->q.code_bytes)
      LAM_HIP(hipMemcpyAsync(codes_dev, st->codes, st->q.code_bytes, hipMemcpyDeviceToDevice, ctx->stream));
  }
  return LAM_OK;
}

lam_status lam_score_topk(lam_ctx* ctx, const lam_store* st, const float* q_dev, int64_t nq, int32_t k,
                          float* scores_dev, int64_t* ids_dev, float* bound_dev) {
  LAM_CHECK(ctx != nullptr && st != nullptr, LAM_EINVAL, "ctx or store is NULL");
  LAM_CHECK(nq >= 0, LAM_EINVAL, "nq must be >= 0");
  LAM_CHECK(k >= 1 && k <= 64, LAM_EINVAL, "k must be in [1, 64]");
  LAM_CHECK((q_dev != nullptr && scores_dev != nullptr && ids_dev != nullptr) || nq == 0, LAM_EINVAL,
            "NULL buffer");
  LAM_CHECK(((uintptr_t)q_dev & 15u) == 0, LAM_EINVAL, "q must be 16-byte aligned");
  {
    DeviceGuard g(ctx->device);
    LAM_TRY(store_settle(const_cast<lam_store*>(st)));
  }
  LAM_CHECK(st->codes != nullptr && st->coded_rows == st->size, LAM_ESTATE,
            "store must be quantized (lam_store_quantize) after its last ingest");
  DeviceGuard g(ctx->device);
  return score_topk(ctx, st, q_dev, nq, k, scores_dev, ids_dev, bound_dev);
}

lam_status lam_score_topk_noalloc(lam_ctx* ctx, const lam_store* st, const float* q_dev, int64_t nq, int32_t k,
                                  float* scores_dev, int64_t* ids_dev, float* bound_dev) {
  LAM_CHECK(ctx != nullptr && st != nullptr, LAM_EINVAL, "ctx or store is NULL");
  LAM_CHECK(nq >= 0, LAM_EINVAL, "nq must be >= 0");
  LAM_CHECK(k >= 1 && k <= 64, LAM_EINVAL, "k must be in [1, 64]");
  LAM_CHECK((q_dev != nullptr && scores_dev != nullptr && ids_dev != nullptr) || nq == 0, LAM_EINVAL,
            "NULL buffer");
  LAM_CHECK(((uintptr_t)q_dev & 15u) == 0, LAM_EINVAL, "q must be 16-byte aligned");
  LAM_CHECK(!st->pending, LAM_ESTATE,
            "ingest calls that did not wait are still in flight: settle the store first (lam_store_get_info)");
  LAM_CHECK(st->codes != nullptr && st->coded_rows == st->size, LAM_ESTATE,
            "store must be quantized (lam_store_quantize) after its last ingest");
  DeviceGuard g(ctx->device);
  return score_topk_noalloc(ctx, st, q_dev, nq, k, scores_dev, ids_dev, bound_dev);
}

lam_status lam_triad(lam_ctx* ctx, const float* a_dev, const float* b_dev, float* c_dev, int64_t n, float s) {
  LAM_CHECK(ctx != nullptr, LAM_EINVAL, "ctx is NULL");
  LAM_CHECK(n >= 0, LAM_EINVAL, "n must be >= 0");
  LAM_CHECK(n == 0 || (a_dev && b_dev && c_dev), LAM_EINVAL, "NULL buffer");
  LAM_CHECK((((uintptr_t)a_dev | (uintptr_t)b_dev | (uintptr_t)c_dev) & 15u) == 0, LAM_EINVAL,
            "arrays must be 16-byte aligned");
  DeviceGuard g(ctx->device);
  return launch_triad(ctx, a_dev, b_dev, c_dev, n, s);
}

lam_status lam_store_block_encode(lam_ctx* ctx, lam_store* st, lam_block_stats* out) {
  LAM_CHECK(ctx != nullptr && st != nullptr, LAM_EINVAL, "ctx or store is NULL");
  DeviceGuard g(ctx->device);
  LAM_TRY(store_settle(st));
  LAM_CHECK(st->codes != nullptr && st->coded_rows == st->size, LAM_ESTATE,
            "store must be quantized (lam_store_quantize) after its last ingest");
  return block_encode(ctx, st, out);
}

static bool blocks_current(const lam_store* st) {
  return st->codes != nullptr && st->coded_rows == st->size && st->blk_rows == st->size;
}

lam_status lam_store_block_decode(lam_ctx* ctx, const lam_store* st, float* xhat_dev) {
  LAM_CHECK(ctx != nullptr && st != nullptr, LAM_EINVAL, "ctx or store is NULL");
  DeviceGuard g(ctx->device);
  LAM_TRY(store_settle(const_cast<lam_store*>(st)));
  LAM_CHECK(blocks_current(st), LAM_ESTATE, "store has no block encoding of its current codes");
  LAM_CHECK(xhat_dev != nullptr || st->size == 0, LAM_EINVAL, "xhat is NULL");
  return block_decode(ctx, st, xhat_dev, nullptr);
}

lam_status lam_store_block_export(lam_ctx* ctx, const lam_store* st, uint8_t* widths_dev, uint64_t* row_off_dev,
                                  uint32_t* data_dev, uint64_t data_cap_bytes) {
  LAM_CHECK(ctx != nullptr && st != nullptr, LAM_EINVAL, "ctx or store is NULL");
  DeviceGuard g(ctx->device);
  LAM_TRY(store_settle(const_cast<lam_store*>(st)));
  LAM_CHECK(blocks_current(st), LAM_ESTATE, "store has no block encoding of its current codes");
  const int64_t m = st->blk_rows;
  const size_t nb = (size_t)st->dim / 32;
  if (widths_dev && m > 0)
    LAM_HIP(hipMemcpyAsync(widths_dev, st->blk_w, (size_t)m * nb, hipMemcpyDeviceToDevice, ctx->stream));
  if (row_off_dev)
    LAM_HIP(hipMemcpyAsync(row_off_dev, st->blk_row_off, (size_t)(m + 1) * 8, hipMemcpyDeviceToDevice, ctx->stream));
  if (data_dev) {
    LAM_CHECK(data_cap_bytes >= st->blk_words * 4, LAM_EINVAL, "data capacity too small");
    if (st->blk_words)
      LAM_HIP(hipMemcpyAsync(data_dev, st->blk_data, st->blk_words * 4, hipMemcpyDeviceToDevice, ctx->stream));
  }
  return LAM_OK;
}

lam_status lam_score_topk_blocks(lam_ctx* ctx, const lam_store* st, const float* q_dev, int64_t nq, int32_t k,
                                 float* scores_dev, int64_t* ids_dev, float* bound_dev) {
  LAM_CHECK(ctx != nullptr && st != nullptr, LAM_EINVAL, "ctx or store is NULL");
  LAM_CHECK(nq >= 0, LAM_EINVAL, "nq must be >= 0");
  LAM_CHECK(k >= 1 && k <= 64, LAM_EINVAL, "k must be in [1, 64]");
  LAM_CHECK((q_dev != nullptr && scores_dev != nullptr && ids_dev != nullptr) || nq == 0, LAM_EINVAL,
            "NULL buffer");
  LAM_CHECK(((uintptr_t)q_dev & 15u) == 0, LAM_EINVAL, "q must be 16-byte aligned");
  DeviceGuard g(ctx->device);
  LAM_TRY(store_settle(const_cast<lam_store*>(st)));
  LAM_CHECK(blocks_current(st), LAM_ESTATE, "store has no block encoding of its current codes");
  // the blocks are expanded back to the fixed-width stream the fused scorer reads
  LAM_TRY(ctx->scratch[kScratchExpand].ensure(std::max<uint64_t>(st->q.code_bytes, 4)));
  uint32_t* codes = ctx->scratch[kScratchExpand].as<uint32_t>();
  LAM_TRY(block_decode(ctx, st, nullptr, codes));
  return score_topk(ctx, st, q_dev, nq, k, scores_dev, ids_dev, bound_dev, codes);
}

lam_status lam_score_topk_certified(lam_ctx* ctx, const lam_store* st, const float* q_dev, int64_t nq, int32_t k,
                                    float* scores_dev, int64_t* ids_dev, float* bound_dev, uint8_t* certified_dev,
                                    float* margin_dev) {
  LAM_CHECK(ctx != nullptr && st != nullptr, LAM_EINVAL, "ctx or store is NULL");
  LAM_CHECK(nq >= 0, LAM_EINVAL, "nq must be >= 0");
  LAM_CHECK(k >= 1 && k <= 63, LAM_EINVAL, "k must be in [1, 63]");
  LAM_CHECK((q_dev != nullptr && scores_dev != nullptr && ids_dev != nullptr && certified_dev != nullptr) || nq == 0,
            LAM_EINVAL, "NULL buffer");
  LAM_CHECK(((uintptr_t)q_dev & 15u) == 0, LAM_EINVAL, "q must be 16-byte aligned");
  {
    DeviceGuard g(ctx->device);
    LAM_TRY(store_settle(const_cast<lam_store*>(st)));
  }
  LAM_CHECK(st->codes != nullptr && st->coded_rows == st->size, LAM_ESTATE,
            "store must be quantized (lam_store_quantize) after its last ingest");
  DeviceGuard g(ctx->device);
  return score_certify(ctx, st, q_dev, nq, k, scores_dev, ids_dev, bound_dev, certified_dev, margin_dev);
}

}  // extern "C"
