// MFMA tile machinery shared by the similarity screen and the scoring kernel.
//
// A workgroup of 256 threads (4 waves of 64) computes a 128 x 128 block of
// C = A . B^T where A and B are row-major with the reduction dimension
// contiguous ("K-major" on both sides).  Waves sit on a 2 x 2 grid; each wave
// owns 64 x 64 of C as 2 x 2 tiles of v_mfma_f32_32x32x16_f16 (CDNA4), i.e.
// 64 fp32 accumulators per lane.  Operands are staged through LDS in K-slabs
// of 64 halves per row, double-buffered, with rows padded by 8 halves so that
// the 32 rows read by one fragment load fall on distinct LDS banks.
//
// Fragment layout of the 32x32x16 instruction (wave64):
//   A operand: lane l supplies A[i = l % 32][k = 8 * (l / 32) + e], e = 0..7
//   B operand: lane l supplies B[k = 8 * (l / 32) + e][j = l % 32]
//   C:         lane l, register r holds C[i][j] with j = l % 32 and
//              i = 8 * (r / 4) + 4 * (l / 32) + (r % 4).
// The reduction index a lane supplies only has to agree between A and B, so
// both fragments are read as 8 consecutive halves of one LDS row.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace lam {

typedef _Float16 half8 __attribute__((ext_vector_type(8)));
typedef float floatx16 __attribute__((ext_vector_type(16)));

constexpr int kTB = 128;          // rows of A and of B per workgroup tile
constexpr int kBK = 64;           // reduction slab per LDS stage (halves)
constexpr int kLdk = kBK + 8;     // padded LDS row length (halves)
constexpr int kWG = 256;          // threads per workgroup

struct SlabRegs {
  uint4 v[4];  // 4 x 16 B per thread = one 128 x 64 fp16 slab per workgroup
};

// Loads rows [0, rows) x halves [k0, k0 + 64) of a row-major fp16 matrix with
// leading dimension ld (halves); rows past `rows` and columns past `kmax` read
// as zero.
__device__ __forceinline__ void slab_load(const _Float16* __restrict__ base, int rows, int64_t ld, int k0,
                                          int kmax, SlabRegs& r) {
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int c = threadIdx.x + kWG * q;
    const int row = c >> 3, col = (c & 7) * 8;
    uint4 v = make_uint4(0u, 0u, 0u, 0u);
    if (row < rows && k0 + col < kmax)
      v = *reinterpret_cast<const uint4*>(base + (int64_t)row * ld + k0 + col);
    r.v[q] = v;
  }
}

__device__ __forceinline__ void slab_store(_Float16* __restrict__ s, const SlabRegs& r) {
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int c = threadIdx.x + kWG * q;
    const int row = c >> 3, col = (c & 7) * 8;
    *reinterpret_cast<uint4*>(s + row * kLdk + col) = r.v[q];
  }
}

__device__ __forceinline__ half8 frag_load(const _Float16* __restrict__ s, int row0, int kk) {
  const int lane = threadIdx.x & 63;
  return *reinterpret_cast<const half8*>(s + (row0 + (lane & 31)) * kLdk + kk * 16 + (lane >> 5) * 8);
}

// Row of C (within a 32x32 tile) held in accumulator register r of this lane.
__device__ __forceinline__ int acc_row(int r, int lane) { return 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3); }

// 128x128 block of C = A . B^T over reduction length kdim.  A rows [0, ra),
// B rows [0, rb) (zero beyond).  lds must hold 2 * 2 * 128 * kLdk halves.
__device__ __forceinline__ void gemm_block_f16(const _Float16* __restrict__ A, int ra,
                                               const _Float16* __restrict__ B, int rb, int64_t ld, int kdim,
                                               _Float16* lds, floatx16 (&acc)[2][2]) {
  // slab buffers: A at 0 / 1, B at 2 / 3
  auto buf = [&](int i) -> _Float16* { return lds + i * (kTB * kLdk); };
  const int wave = threadIdx.x >> 6;
  const int wm = wave >> 1, wn = wave & 1;
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int b = 0; b < 2; ++b)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[a][b][r] = 0.0f;

  SlabRegs ra_, rb_;
  slab_load(A, ra, ld, 0, kdim, ra_);
  slab_load(B, rb, ld, 0, kdim, rb_);
  slab_store(buf(0), ra_);
  slab_store(buf(2), rb_);
  __syncthreads();
  int cur = 0;
  for (int k0 = 0; k0 < kdim; k0 += kBK) {
    const bool more = k0 + kBK < kdim;
    if (more) {
      slab_load(A, ra, ld, k0 + kBK, kdim, ra_);
      slab_load(B, rb, ld, k0 + kBK, kdim, rb_);
    }
#pragma unroll
    for (int kk = 0; kk < kBK / 16; ++kk) {
      half8 fa[2], fb[2];
#pragma unroll
      for (int t = 0; t < 2; ++t) {
        fa[t] = frag_load(buf(cur), wm * 64 + t * 32, kk);
        fb[t] = frag_load(buf(2 + cur), wn * 64 + t * 32, kk);
      }
#pragma unroll
      for (int a = 0; a < 2; ++a)
#pragma unroll
        for (int b = 0; b < 2; ++b)
          acc[a][b] = __builtin_amdgcn_mfma_f32_32x32x16_f16(fa[a], fb[b], acc[a][b], 0, 0, 0);
    }
    if (more) {
      slab_store(buf(cur ^ 1), ra_);
      slab_store(buf(2 + (cur ^ 1)), rb_);
    }
    __syncthreads();
    cur ^= 1;
  }
}

// ---------------------------------------------------------------------------
// Generalised block: WM x WN waves, each owning TI x TJ tiles of 32 x 32, so a
// workgroup computes (WM*TI*32) x (WN*TJ*32) of C = A . B^T.  Larger per-wave
// tiles read fewer LDS bytes per MFMA: (TI + TJ) / (TI * TJ) KB.
template <int WM_, int WN_, int TI_, int TJ_>
struct Tile {
  static constexpr int WM = WM_, WN = WN_, TI = TI_, TJ = TJ_;
  static constexpr int kWaves = WM * WN;
  static constexpr int kThreads = 64 * kWaves;
  static constexpr int BM = WM * TI * 32;   // A rows per workgroup
  static constexpr int BN = WN * TJ * 32;   // B rows per workgroup
  static constexpr int kChunksA = BM * (kBK / 8);   // 16-byte chunks of one A slab
  static constexpr int kChunksB = BN * (kBK / 8);
  static constexpr int kPerA = kChunksA / kThreads;
  static constexpr int kPerB = kChunksB / kThreads;
  static constexpr int kLdsHalves = 2 * (BM + BN) * kLdk;   // double-buffered slabs
  static_assert(kChunksA % kThreads == 0 && kChunksB % kThreads == 0, "slab must split evenly");
};

template <int N>
__device__ __forceinline__ void slab_load_n(const _Float16* __restrict__ base, int rows, int64_t ld, int k0, int kmax,
                                            uint4 (&r)[N], int nthreads) {
#pragma unroll
  for (int q = 0; q < N; ++q) {
    const int c = threadIdx.x + nthreads * q;
    const int row = c >> 3, col = (c & 7) * 8;
    uint4 v = make_uint4(0u, 0u, 0u, 0u);
    if (row < rows && k0 + col < kmax) v = *reinterpret_cast<const uint4*>(base + (int64_t)row * ld + k0 + col);
    r[q] = v;
  }
}

template <int N>
__device__ __forceinline__ void slab_store_n(_Float16* __restrict__ s, const uint4 (&r)[N], int nthreads) {
#pragma unroll
  for (int q = 0; q < N; ++q) {
    const int c = threadIdx.x + nthreads * q;
    const int row = c >> 3, col = (c & 7) * 8;
    *reinterpret_cast<uint4*>(s + row * kLdk + col) = r[q];
  }
}

// C tile of one workgroup; lds holds C::kLdsHalves halves.  acc[ti][tj] holds
// rows wm*TI*32 + ti*32 + acc_row(r, lane) of A and column wn*TJ*32 + tj*32 +
// lane%32 of B, with wm = wave / WN, wn = wave % WN.
template <class C>
__device__ __forceinline__ void gemm_tile(const _Float16* __restrict__ A, int ra, const _Float16* __restrict__ B,
                                          int rb, int64_t ld, int kdim, _Float16* lds,
                                          floatx16 (&acc)[C::TI][C::TJ]) {
  _Float16* sa0 = lds;
  _Float16* sb0 = lds + 2 * C::BM * kLdk;
  auto sa = [&](int i) -> _Float16* { return sa0 + i * (C::BM * kLdk); };
  auto sb = [&](int i) -> _Float16* { return sb0 + i * (C::BN * kLdk); };
  const int wave = threadIdx.x >> 6;
  const int wm = wave / C::WN, wn = wave % C::WN;
#pragma unroll
  for (int a = 0; a < C::TI; ++a)
#pragma unroll
    for (int b = 0; b < C::TJ; ++b)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[a][b][r] = 0.0f;
  uint4 ra_[C::kPerA], rb_[C::kPerB];
  slab_load_n<C::kPerA>(A, ra, ld, 0, kdim, ra_, C::kThreads);
  slab_load_n<C::kPerB>(B, rb, ld, 0, kdim, rb_, C::kThreads);
  slab_store_n<C::kPerA>(sa(0), ra_, C::kThreads);
  slab_store_n<C::kPerB>(sb(0), rb_, C::kThreads);
  __syncthreads();
  int cur = 0;
  for (int k0 = 0; k0 < kdim; k0 += kBK) {
    const bool more = k0 + kBK < kdim;
    if (more) {
      slab_load_n<C::kPerA>(A, ra, ld, k0 + kBK, kdim, ra_, C::kThreads);
      slab_load_n<C::kPerB>(B, rb, ld, k0 + kBK, kdim, rb_, C::kThreads);
    }
#pragma unroll
    for (int kk = 0; kk < kBK / 16; ++kk) {
      half8 fa[C::TI], fb[C::TJ];
#pragma unroll
      for (int t = 0; t < C::TI; ++t) fa[t] = frag_load(sa(cur), wm * C::TI * 32 + t * 32, kk);
#pragma unroll
      for (int t = 0; t < C::TJ; ++t) fb[t] = frag_load(sb(cur), wn * C::TJ * 32 + t * 32, kk);
#pragma unroll
      for (int a = 0; a < C::TI; ++a)
#pragma unroll
        for (int b = 0; b < C::TJ; ++b)
          acc[a][b] = __builtin_amdgcn_mfma_f32_32x32x16_f16(fa[a], fb[b], acc[a][b], 0, 0, 0);
    }
    if (more) {
      slab_store_n<C::kPerA>(sa(cur ^ 1), ra_, C::kThreads);
      slab_store_n<C::kPerB>(sb(cur ^ 1), rb_, C::kThreads);
    }
    __syncthreads();
    cur ^= 1;
  }
}

// Workgroup index remapped so that consecutive logical tiles run on the same
// XCD (the hardware deals workgroups to the 8 XCDs round-robin), letting tiles
// that share operand rows share that XCD's L2.
// A bijection of [0, nblocks): XCD x = bid % 8 receives the contiguous range
// starting at x * q + min(x, rem).
__host__ __device__ inline int64_t xcd_remap(int64_t bid, int64_t nblocks) {
  const int64_t q = nblocks / 8, rem = nblocks % 8;
  const int64_t x = bid % 8;
  return x * q + (x < rem ? x : rem) + bid / 8;
}

// Order-preserving map of float to uint32 for atomicMax.
__device__ __forceinline__ uint32_t f2ord(float f) {
  const uint32_t u = __float_as_uint(f);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}
__host__ __device__ inline float ord2f(uint32_t o) {
  const uint32_t u = (o & 0x80000000u) ? (o & 0x7fffffffu) : ~o;
  float f;
  __builtin_memcpy(&f, &u, 4);
  return f;
}

}  // namespace lam
