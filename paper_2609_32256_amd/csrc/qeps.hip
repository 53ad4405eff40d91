// Q_eps, the error-bounded quantizer of Section 2.2 ("Three layers", L1):
// q = round(x / 2eps) per coordinate, packed to the narrowest two's-complement
// width b, and its decode x_hat = float32(float64(q * 2eps)).
//
// Rounding.  The quotient is the exact real x / s (x float32, s = 2 eps
// binary64), rounded half to even.  A binary64 estimate q0 = rint(x * (1/s))
// is within 2^-20 of x/s for |x/s| < 2^31, so the nearest integer is q0 or a
// neighbour.  The remainder e = x - q0*s is formed by one fused multiply-add;
// round-to-nearest is monotone, so RN(e) < eps proves e < eps, RN(e) > eps
// proves e > eps, and only RN(e) == +-eps needs the sign of x - (q0 +- 1/2) s,
// which a second fused multiply-add gives exactly (a single rounding keeps the
// sign, and zero only for an exact zero, i.e. a true tie).
//
// Memory layout.  A tile of 4096 elements (256 threads x 16) is read with
// coalesced float4 loads, quantized in registers, and parked in LDS as int32;
// each thread then assembles whole output words (bits [32w, 32w+32) of the
// tile's stream) from LDS and stores them coalesced.  4096*b bits is a whole
// number of words, so tiles never share a word.  Decode mirrors this.
// Bytes per element: encode 4 + b/8, decode b/8 + 4 -- an HBM-bound stream.
#include <cmath>
#include <cstring>

#include "lam_internal.h"

namespace lam {
namespace {

constexpr int kThreads = 256;
constexpr int kPerThread = 16;
constexpr int kTile = kThreads * kPerThread;  // 4096 elements

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

__device__ __forceinline__ void wave_flag(bool bad, uint32_t* counter) {
  const unsigned long long m = __ballot(bad);
  if (m != 0ull && (threadIdx.x & 63) == 0) atomicAdd(counter, (uint32_t)__popcll(m));
}

template <bool VEC>
__global__ __launch_bounds__(kThreads) void k_absmax(const float* __restrict__ x, int64_t n,
                                                     uint32_t* __restrict__ out) {
  uint32_t m = 0;
  const int64_t stride = (int64_t)gridDim.x * kThreads;
  int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  if (VEC) {
    const int64_t n4 = n >> 2;
    const uint4* x4 = reinterpret_cast<const uint4*>(x);
    for (int64_t j = i; j < n4; j += stride) {
      const uint4 v = x4[j];
      m = max(m, max(max(v.x & 0x7fffffffu, v.y & 0x7fffffffu), max(v.z & 0x7fffffffu, v.w & 0x7fffffffu)));
    }
    for (int64_t j = (n4 << 2) + i; j < n; j += stride) m = max(m, __float_as_uint(x[j]) & 0x7fffffffu);
  } else {
    for (int64_t j = i; j < n; j += stride) m = max(m, __float_as_uint(x[j]) & 0x7fffffffu);
  }
  for (int o = 32; o > 0; o >>= 1) m = max(m, (uint32_t)__shfl_xor((int)m, o));
  // one atomic per block: a few hundred updates of one address, not one per wave
  __shared__ uint32_t wm[kThreads / 64];
  if ((threadIdx.x & 63) == 0) wm[threadIdx.x >> 6] = m;
  __syncthreads();
  if (threadIdx.x == 0) {
    uint32_t b = wm[0];
    for (int w = 1; w < kThreads / 64; ++w) b = max(b, wm[w]);
    atomicMax(out, b);
  }
}

template <int B, bool VEC>
__global__ __launch_bounds__(kThreads) void k_encode(const float* __restrict__ x, int64_t n, double s,
                                                     double inv_s, double eps, float absmax,
                                                     uint32_t* __restrict__ codes, uint64_t nwords,
                                                     uint32_t* __restrict__ flags) {
  __shared__ int32_t lq[kTile + 40];
  const int t = threadIdx.x;
  const int64_t tile = blockIdx.x;
  const int64_t base = tile * (int64_t)kTile;
  bool nonfinite = false, range = false;
#pragma unroll
  for (int j = 0; j < kPerThread / 4; ++j) {
    const int le = j * (kThreads * 4) + t * 4;
    const int64_t e = base + le;
    float v[4];
    if (VEC && e + 3 < n) {
      const float4 f = *reinterpret_cast<const float4*>(x + e);
      v[0] = f.x; v[1] = f.y; v[2] = f.z; v[3] = f.w;
    } else {
#pragma unroll
      for (int r = 0; r < 4; ++r) v[r] = (e + r < n) ? x[e + r] : 0.0f;
    }
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const float a = fabsf(v[r]);
      nonfinite |= !(a <= 3.402823466e38f);
      range |= a > absmax;
      lq[le + r] = q_round(v[r], s, inv_s, eps);
    }
  }
  if (t < 40) lq[kTile + t] = 0;
  __syncthreads();

  constexpr int kWords = kTile * B / 32;           // 128 * B words per tile
  constexpr uint32_t kMask = (B == 32) ? 0xffffffffu : ((1u << B) - 1u);
  constexpr int kSpan = (32 + B - 1) / B + 1;       // elements touching one word
  const uint64_t w0 = (uint64_t)tile * kWords;
  for (int w = t; w < kWords; w += kThreads) {
    if (w0 + w >= nwords) break;
    const int bit = w * 32;
    const int e = bit / B;
    const int sh = e * B - bit;  // in (-B, 0]
    uint32_t acc = 0;
#pragma unroll
    for (int r = 0; r < kSpan; ++r) {
      const int s2 = sh + r * B;
      if (s2 < 32) {
        const uint32_t u = (uint32_t)lq[e + r] & kMask;
        acc |= (s2 >= 0) ? (u << s2) : (u >> (-s2));
      }
    }
    codes[w0 + w] = acc;
  }
  wave_flag(nonfinite, &flags[0]);
  wave_flag(range, &flags[1]);
}

template <int B, bool VEC>
__global__ __launch_bounds__(kThreads) void k_decode(const uint32_t* __restrict__ codes, int64_t n,
                                                     uint64_t nwords, double s, float* __restrict__ xhat) {
  constexpr int kWords = kTile * B / 32;
  __shared__ uint32_t lw[kWords + 2];
  const int t = threadIdx.x;
  const int64_t tile = blockIdx.x;
  const uint64_t w0 = (uint64_t)tile * kWords;
  for (int w = t; w < kWords + 2; w += kThreads) lw[w] = (w0 + w < nwords) ? codes[w0 + w] : 0u;
  __syncthreads();
  const int64_t base = tile * (int64_t)kTile;
#pragma unroll
  for (int j = 0; j < kPerThread / 4; ++j) {
    const int le = j * (kThreads * 4) + t * 4;
    float v[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int bit = (le + r) * B;
      const int wi = bit >> 5, off = bit & 31;
      const uint64_t pair = ((uint64_t)lw[wi + 1] << 32) | lw[wi];
      const uint32_t u = (uint32_t)(pair >> off);
      const int32_t q = (int32_t)(u << (32 - B)) >> (32 - B);
      v[r] = (float)((double)q * s);
    }
    const int64_t e = base + le;
    if (VEC && e + 3 < n) {
      *reinterpret_cast<float4*>(xhat + e) = make_float4(v[0], v[1], v[2], v[3]);
    } else {
#pragma unroll
      for (int r = 0; r < 4; ++r)
        if (e + r < n) xhat[e + r] = v[r];
    }
  }
}

// Host-side exact rounding, same method as q_round (std::fma is correctly
// rounded), used for the width plan M = Q_eps(A).
double host_round_quotient(double x, double s) {
  const double eps = s * 0.5;
  double q0 = std::nearbyint(x / s);
  const double t = std::fma(-q0, s, x);
  if (t > eps) {
    q0 += 1.0;
  } else if (t < -eps) {
    q0 -= 1.0;
  } else if (t == eps) {
    const double d = std::fma(-(q0 + 0.5), s, x);
    if (d > 0.0 || (d == 0.0 && std::fmod(q0, 2.0) != 0.0)) q0 += 1.0;
  } else if (t == -eps) {
    const double d = std::fma(-(q0 - 0.5), s, x);
    if (d < 0.0 || (d == 0.0 && std::fmod(q0, 2.0) != 0.0)) q0 -= 1.0;
  }
  return q0;
}

template <int B>
void encode_dispatch(int b, bool vec, dim3 grid, hipStream_t st, const float* x, int64_t n, double s,
                     double eps, float absmax, uint32_t* codes, uint64_t nwords, uint32_t* flags) {
  if (b == B) {
    if (vec)
      hipLaunchKernelGGL((k_encode<B, true>), grid, dim3(kThreads), 0, st, x, n, s, 1.0 / s, eps, absmax,
                         codes, nwords, flags);
    else
      hipLaunchKernelGGL((k_encode<B, false>), grid, dim3(kThreads), 0, st, x, n, s, 1.0 / s, eps, absmax,
                         codes, nwords, flags);
    return;
  }
  if constexpr (B < 32) encode_dispatch<B + 1>(b, vec, grid, st, x, n, s, eps, absmax, codes, nwords, flags);
}

template <int B>
void decode_dispatch(int b, bool vec, dim3 grid, hipStream_t st, const uint32_t* codes, int64_t n,
                     uint64_t nwords, double s, float* xhat) {
  if (b == B) {
    if (vec)
      hipLaunchKernelGGL((k_decode<B, true>), grid, dim3(kThreads), 0, st, codes, n, nwords, s, xhat);
    else
      hipLaunchKernelGGL((k_decode<B, false>), grid, dim3(kThreads), 0, st, codes, n, nwords, s, xhat);
    return;
  }
  if constexpr (B < 32) decode_dispatch<B + 1>(b, vec, grid, st, codes, n, nwords, s, xhat);
}

}  // namespace

lam_status qeps_plan_host(double eps, float absmax, int mode, int64_t n, lam_qparams* out) {
  LAM_CHECK(out != nullptr, LAM_EINVAL, "qparams output is NULL");
  LAM_CHECK(std::isfinite(eps) && eps >= std::ldexp(1.0, -60) && eps <= std::ldexp(1.0, 20), LAM_EINVAL,
            "eps must be finite and in [2^-60, 2^20] (got %g)", eps);
  LAM_CHECK(std::isfinite(absmax) && absmax >= 0.0f, LAM_EINVAL, "absmax must be finite and >= 0");
  LAM_CHECK(n >= 0, LAM_EINVAL, "n must be >= 0");
  LAM_CHECK(mode == LAM_PACK_BITS || mode == LAM_PACK_BYTES, LAM_EINVAL, "unknown pack mode %d", mode);
  const double s = 2.0 * eps;
  const double ratio = (double)absmax / s;
  LAM_CHECK(ratio < 2147483647.0, LAM_ERANGE, "code range too wide: absmax/(2 eps) = %g >= 2^31", ratio);
  const double m = host_round_quotient((double)absmax, s);
  LAM_CHECK(m <= 2147483647.0, LAM_ERANGE, "max code %g does not fit 32 bits", m);
  const uint32_t M = (uint32_t)m;
  int b = 1;
  while (b < 32 && ((1u << (b - 1)) - 1u) < M) ++b;   // smallest b with 2^(b-1) - 1 >= M
  if (mode == LAM_PACK_BYTES) b = (b <= 8) ? 8 : (b <= 16 ? 16 : 32);
  lam_qparams p{};
  p.eps = eps;
  p.step = s;
  p.absmax = absmax;
  p.bits = b;
  p.mode = mode;
  p.max_code = (int32_t)M;
  p.n = n;
  const uint64_t words = ((uint64_t)n * (uint64_t)b + 31u) / 32u;
  p.code_bytes = words * 4u;
  *out = p;
  return LAM_OK;
}

lam_status launch_absmax(lam_ctx* ctx, const float* x, int64_t n, uint32_t* absmax_bits_dev, const char* prof_name) {
  if (n == 0) return LAM_OK;
  const bool vec = ((uintptr_t)x & 15u) == 0;
  const int64_t work = vec ? (n + 3) / 4 : n;
  const int blocks = (int)std::min<int64_t>(1024, (work + kThreads - 1) / kThreads);
  ProfScope ps(ctx, prof_name);
  if (vec)
    hipLaunchKernelGGL(k_absmax<true>, dim3(blocks), dim3(kThreads), 0, ctx->stream, x, n, absmax_bits_dev);
  else
    hipLaunchKernelGGL(k_absmax<false>, dim3(blocks), dim3(kThreads), 0, ctx->stream, x, n, absmax_bits_dev);
  LAM_HIP(hipGetLastError());
  return LAM_OK;
}

lam_status launch_encode(lam_ctx* ctx, const float* x, int64_t n, const lam_qparams& p, uint32_t* codes,
                         uint32_t* flags2, const char* prof_name) {
  if (n == 0) return LAM_OK;
  LAM_CHECK(p.bits >= 1 && p.bits <= 32, LAM_EINVAL, "bad code width %d", p.bits);
  const bool vec = ((uintptr_t)x & 15u) == 0;
  const int64_t tiles = (n + kTile - 1) / kTile;
  LAM_CHECK(tiles < (1LL << 31), LAM_EINVAL, "too many elements");
  const uint64_t nwords = p.code_bytes / 4u;
  ProfScope ps(ctx, prof_name);
  encode_dispatch<1>(p.bits, vec, dim3((unsigned)tiles), ctx->stream, x, n, p.step, p.eps, p.absmax, codes,
                     nwords, flags2);
  LAM_HIP(hipGetLastError());
  return LAM_OK;
}

lam_status launch_decode(lam_ctx* ctx, const uint32_t* codes, const lam_qparams& p, float* xhat, const char* prof_name) {
  if (p.n == 0) return LAM_OK;
  LAM_CHECK(p.bits >= 1 && p.bits <= 32, LAM_EINVAL, "bad code width %d", p.bits);
  const bool vec = ((uintptr_t)xhat & 15u) == 0;
  const int64_t tiles = (p.n + kTile - 1) / kTile;
  LAM_CHECK(tiles < (1LL << 31), LAM_EINVAL, "too many elements");
  ProfScope ps(ctx, prof_name);
  decode_dispatch<1>(p.bits, vec, dim3((unsigned)tiles), ctx->stream, codes, p.n, (uint64_t)(p.code_bytes / 4u),
                     p.step, xhat);
  LAM_HIP(hipGetLastError());
  return LAM_OK;
}

}  // namespace lam
