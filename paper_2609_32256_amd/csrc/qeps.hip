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
// Most elements never need binary64: p = x * float32(1/s) is within
// 2^-22 (|p| + 1) of x/s (two float32 roundings), so when |p - rint(p)| is at
// most 1/2 - 2^-21 (|p| + 1) no half-integer can separate p from x/s and
// rint(p) is the exact answer.  Only the remaining elements (near a tie, or
// |p| beyond float32's exact range) take the binary64 path above.
//
// Memory layout.  A tile of 8192 elements (256 threads x 32) is read with
// coalesced float4 loads and quantized; the codes are parked in LDS (one pad
// word per 32 so that a thread reading its own 32 consecutive codes hits
// distinct banks), each thread packs its 32 codes into b words in registers
// with compile-time shifts, and the packed words go back through LDS to
// coalesced stores.  32 codes are exactly b words, so threads and tiles never
// share a word.  Decode loads a tile's words into LDS, extracts each code with
// a funnel shift, and (for b <= 12) maps it through a per-workgroup table of
// float32(float64(c * s)).  Bytes per element: encode 4 + b/8, decode b/8 + 4
// -- an HBM-bound stream.
#include <cmath>
#include <cstring>

#include <hip/hip_ext.h>

#include "lam_internal.h"
#include "qround.h"

namespace lam {
namespace {

constexpr int kThreads = 256;
constexpr int kPerThread = 32;
constexpr int kTile = kThreads * kPerThread;  // 8192 elements
constexpr int kPadded = kTile + kTile / 32;    // one pad word per 32 codes
// Cache policy of the encoder's streaming traffic: its input is read once and
// its codes are written once, so both are marked non-temporal (the buffer
// load's policy operand; the stores use the non-temporal builtin).  This took
// the 2^26-value encode from 98 to 66 us; the decoder is faster without it.
constexpr int kNonTemporal = 2;

// Buffer resource over `bytes` bytes from base: loads at offsets past the
// bound return zeros without touching memory, so a load never needs a branch
// (a load under a branch makes the compiler wait for every outstanding load,
// which serialises a prefetching loop).  gfx9 raw buffer: stride 0, 32-bit data
// format word.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t span_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes, 0x00020000);
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
    // float4 loads, four per trip and all in flight together; each trip reads
    // a window of 4 * stride float4 through a resource that ends at the data,
    // so the tail reads zeros (which do not change the maximum)
    const int64_t n4 = n >> 2;
    for (int64_t j0 = (int64_t)blockIdx.x * kThreads; j0 < n4; j0 += 4 * stride) {
      const int64_t left = n4 - j0;
      const uint32_t nbytes = (uint32_t)((left < 4 * stride ? left : 4 * stride) * 16);
      const __amdgpu_buffer_rsrc_t rs = span_rsrc(x + j0 * 4, nbytes);
      uint4 v[4];
#pragma unroll
      for (int u = 0; u < 4; ++u)
        v[u] = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(
                                             rs, (uint32_t)(u * stride + threadIdx.x) * 16u, 0, 0));
#pragma unroll
      for (int u = 0; u < 4; ++u)
        m = max(m, max(max(v[u].x & 0x7fffffffu, v[u].y & 0x7fffffffu),
                       max(v[u].z & 0x7fffffffu, v[u].w & 0x7fffffffu)));
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

// Quantize, pack and store one tile whose values are in v (thread t holds
// elements j * 1024 + 4t .. +3 of the tile for j = 0..7).  FULL: all kTile
// elements exist.
template <int B, bool FULL>
__device__ __forceinline__ void encode_tile(const float4 (&v4)[kPerThread / 4], int64_t tile, int64_t n,
                                            float inv_s32, double s, double inv_s, double eps, float absmax,
                                            uint32_t* __restrict__ codes, uint64_t nwords,
                                            uint32_t* __restrict__ flags, uint32_t* lq) {
  constexpr uint32_t kMask = (B == 32) ? 0xffffffffu : ((1u << B) - 1u);
  const int t = threadIdx.x;
  const int64_t base = tile * (int64_t)kTile;
  bool bad = false;   // NaN, Inf or |x| > absmax (absmax is finite)
#pragma unroll
  for (int j = 0; j < kPerThread / 4; ++j) {
    const int le = j * (kThreads * 4) + t * 4;
    const float v[4] = {v4[j].x, v4[j].y, v4[j].z, v4[j].w};
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const bool real = FULL || base + le + r < n;
      bad |= real && !(fabsf(v[r]) <= absmax);
      const int li = le + r;
      lq[li + (li >> 5)] = (uint32_t)q_round_fast(v[r], inv_s32, s, inv_s, eps) & kMask;
    }
  }
  __syncthreads();
  // pack this thread's 32 consecutive codes into B words
  uint32_t w[B];
#pragma unroll
  for (int i = 0; i < B; ++i) w[i] = 0u;
#pragma unroll
  for (int k = 0; k < 32; ++k) {
    const uint32_t u = lq[t * 33 + k];
    const int bit = k * B, wi = bit >> 5, off = bit & 31;
    w[wi] |= u << off;
    if (off + B > 32) w[wi + 1] |= u >> (32 - off);
  }
  __syncthreads();
  // words back through LDS (same one-per-32 padding) for coalesced stores
#pragma unroll
  for (int i = 0; i < B; ++i) {
    const int wi = t * B + i;
    lq[wi + (wi >> 5)] = w[i];
  }
  __syncthreads();
  constexpr int kWords = kThreads * B;              // words per tile
  const uint64_t w0 = (uint64_t)tile * kWords;
#pragma unroll
  for (int i = t; i < kWords; i += kThreads)
    if (FULL || w0 + i < nwords) __builtin_nontemporal_store(lq[i + (i >> 5)], &codes[w0 + i]);
  if (__ballot(bad) != 0ull) {
    // classify the rare failures from the values at hand: non-finite (EINVAL)
    // vs merely above absmax (ERANGE)
    bool nonfinite = false, range = false;
#pragma unroll
    for (int j = 0; j < kPerThread / 4; ++j) {
      const int le = j * (kThreads * 4) + t * 4;
      const float v[4] = {v4[j].x, v4[j].y, v4[j].z, v4[j].w};
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        if (!(FULL || base + le + r < n)) continue;
        const float a = fabsf(v[r]);
        nonfinite |= !(a <= 3.402823466e38f);
        range |= a > absmax;
      }
    }
    wave_flag(nonfinite, &flags[0]);
    wave_flag(range, &flags[1]);
  }
}

// One tile per workgroup (the grid covers the tiles once): its eight float4
// loads per thread are issued together through a buffer resource, marked
// non-temporal.  The partial last tile, and every tile of an input that is
// not 16-byte aligned, take the element-wise path.  (A persistent grid of
// 1,024 or 2,048 workgroups that loads the next tile while encoding the
// current one measured 12 to 24 % slower on MI355X, as grid-stride loops did
// for the plain triad.)
template <int B, bool VEC>
__global__ __launch_bounds__(kThreads) void k_encode(const float* __restrict__ x, int64_t n, float inv_s32,
                                                     double s, double inv_s, double eps, float absmax,
                                                     uint32_t* __restrict__ codes, uint64_t nwords,
                                                     uint32_t* __restrict__ flags) {
  __shared__ uint32_t lq[kPadded];
  const int t = threadIdx.x;
  const int64_t tile = blockIdx.x;
  const int64_t nfull = VEC ? n / kTile : 0;
  float4 v[kPerThread / 4];
  if (tile < nfull) {
    const __amdgpu_buffer_rsrc_t rs = span_rsrc(x + tile * (int64_t)kTile, kTile * 4u);
#pragma unroll
    for (int j = 0; j < kPerThread / 4; ++j)
      v[j] = __builtin_bit_cast(float4, __builtin_amdgcn_raw_buffer_load_b128(
                                            rs, (uint32_t)(j * (kThreads * 4) + t * 4) * 4u, 0, kNonTemporal));
    encode_tile<B, true>(v, tile, n, inv_s32, s, inv_s, eps, absmax, codes, nwords, flags, lq);
    return;
  }
  const int64_t b0 = tile * (int64_t)kTile;
#pragma unroll
  for (int j = 0; j < kPerThread / 4; ++j) {
    const int64_t e = b0 + j * (kThreads * 4) + t * 4;
    v[j].x = (e < n) ? x[e] : 0.0f;
    v[j].y = (e + 1 < n) ? x[e + 1] : 0.0f;
    v[j].z = (e + 2 < n) ? x[e + 2] : 0.0f;
    v[j].w = (e + 3 < n) ? x[e + 3] : 0.0f;
  }
  encode_tile<B, false>(v, tile, n, inv_s32, s, inv_s, eps, absmax, codes, nwords, flags, lq);
}

template <int B, bool VEC>
__global__ __launch_bounds__(kThreads) void k_decode(const uint32_t* __restrict__ codes, int64_t n,
                                                     uint64_t nwords, double s, float* __restrict__ xhat) {
  constexpr int kWords = kTile * B / 32;
  constexpr bool kLut = B <= 12;                    // decode table of 2^B entries
  constexpr int kLutN = kLut ? (1 << (B > 12 ? 0 : B)) : 1;
  __shared__ uint32_t lw[kWords + 2];
  __shared__ float lut[kLutN];
  const int t = threadIdx.x;
  const int64_t tile = blockIdx.x;
  const uint64_t w0 = (uint64_t)tile * kWords;
  {
    // all of this thread's loads in flight before the first LDS store; words
    // past the tile's end (and past the stream) read as zero from the bound
    constexpr int kIt = (kWords + 2 + kThreads - 1) / kThreads;
    const uint64_t avail = nwords > w0 ? nwords - w0 : 0u;
    const uint32_t nw = (uint32_t)(avail < (uint64_t)(kWords + 2) ? avail : (uint64_t)(kWords + 2));
    const __amdgpu_buffer_rsrc_t rs = span_rsrc(codes + w0, nw * 4u);
    uint32_t tmp[kIt];
#pragma unroll
    for (int i = 0; i < kIt; ++i)
      tmp[i] = (uint32_t)__builtin_amdgcn_raw_buffer_load_b32(rs, (uint32_t)(t + i * kThreads) * 4u, 0, 0);
#pragma unroll
    for (int i = 0; i < kIt; ++i) {
      const int w = t + i * kThreads;
      if (w < kWords + 2) lw[w] = tmp[i];
    }
  }
  if (kLut) {
    // entry c + 2^(B-1) holds float32(float64(c * s)), the decode definition
    for (int c = t; c < kLutN; c += kThreads) lut[c] = (float)((double)(c - kLutN / 2) * s);
  }
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
      const uint32_t u = __builtin_amdgcn_alignbit(lw[wi + 1], lw[wi], (uint32_t)off);
      if (kLut) {
        v[r] = lut[(u ^ (1u << (B - 1))) & (uint32_t)(kLutN - 1)];   // offset binary index
      } else {
        const int32_t q = (int32_t)(u << (32 - B)) >> (32 - B);
        v[r] = (float)((double)q * s);
      }
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

// e0 / e1: events the launch itself stamps at the kernel's start and end
// (null unless the kernel is being timed)
template <int B>
void encode_dispatch(int b, bool vec, dim3 grid, hipStream_t st, hipEvent_t e0, hipEvent_t e1, const float* x,
                     int64_t n, double s, double eps, float absmax, uint32_t* codes, uint64_t nwords,
                     uint32_t* flags) {
  if (b == B) {
    if (vec)
      hipExtLaunchKernelGGL((k_encode<B, true>), grid, dim3(kThreads), 0, st, e0, e1, 0, x, n, (float)(1.0 / s), s,
                            1.0 / s, eps, absmax, codes, nwords, flags);
    else
      hipExtLaunchKernelGGL((k_encode<B, false>), grid, dim3(kThreads), 0, st, e0, e1, 0, x, n, (float)(1.0 / s), s,
                            1.0 / s, eps, absmax, codes, nwords, flags);
    return;
  }
  if constexpr (B < 32) encode_dispatch<B + 1>(b, vec, grid, st, e0, e1, x, n, s, eps, absmax, codes, nwords, flags);
}

template <int B>
void decode_dispatch(int b, bool vec, dim3 grid, hipStream_t st, hipEvent_t e0, hipEvent_t e1, const uint32_t* codes,
                     int64_t n, uint64_t nwords, double s, float* xhat) {
  if (b == B) {
    if (vec)
      hipExtLaunchKernelGGL((k_decode<B, true>), grid, dim3(kThreads), 0, st, e0, e1, 0, codes, n, nwords, s, xhat);
    else
      hipExtLaunchKernelGGL((k_decode<B, false>), grid, dim3(kThreads), 0, st, e0, e1, 0, codes, n, nwords, s, xhat);
    return;
  }
  if constexpr (B < 32) decode_dispatch<B + 1>(b, vec, grid, st, e0, e1, codes, n, nwords, s, xhat);
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
  hipEvent_t e0, e1;   // timed by the launch itself when profiled
  LAM_TRY(prof_launch_events(ctx, prof_name, &e0, &e1));
  const unsigned grid = (unsigned)tiles;   // one tile per workgroup
  encode_dispatch<1>(p.bits, vec, dim3(grid), ctx->stream, e0, e1, x, n, p.step, p.eps, p.absmax, codes,
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
  hipEvent_t e0, e1;   // timed by the launch itself when profiled
  LAM_TRY(prof_launch_events(ctx, prof_name, &e0, &e1));
  decode_dispatch<1>(p.bits, vec, dim3((unsigned)tiles), ctx->stream, e0, e1, codes, p.n,
                     (uint64_t)(p.code_bytes / 4u), p.step, xhat);
  LAM_HIP(hipGetLastError());
  return LAM_OK;
}

}  // namespace lam
