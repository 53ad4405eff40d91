// MFMA tile machinery shared by the similarity screen and the scoring kernel.
//
// A workgroup of WM x WN waves computes a block of C = A . B^T where A and B
// are row-major with the reduction dimension contiguous ("K-major" on both
// sides); each wave owns TI x TJ tiles of v_mfma_f32_32x32x16_f16 (CDNA4),
// i.e. 16 * TI * TJ fp32 accumulators per lane.  Operands are staged through
// LDS in K-slabs of 64 halves per row (two stages), with rows padded by 8
// halves so that the 32 rows read by one fragment load fall on distinct LDS
// banks.
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

// Slab loads go through buffer resources: a descriptor bounds the tile's rows
// in bytes and the hardware returns zeros for an offset past the bound, so a
// chunk outside the tile costs no branch (an offset select instead).  Keeping
// every load off divergent branches also lets the compiler count outstanding
// loads exactly rather than waiting for all of them.
constexpr uint32_t kOffOOB = 0x80000000u;   // beyond every tile's bound

__device__ __forceinline__ __amdgpu_buffer_rsrc_t tile_rsrc(const _Float16* base, int rows, int64_t ld) {
  // gfx9 raw buffer: stride 0, num_records in bytes, 32-bit data format word
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<_Float16*>(base), (short)0, (int)(rows * ld * 2), 0x00020000);
}

// Per-row float32 terms of a tile through a buffer resource (zeros past
// `count` rows), for the same reason as the slab loads.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t f32_rsrc(const float* base, int count) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<float*>(base), (short)0, count * 4, 0x00020000);
}

__device__ __forceinline__ float buf_f32(__amdgpu_buffer_rsrc_t rs, bool ok, int idx) {
  return __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rs, ok ? (uint32_t)idx * 4u : kOffOOB, 0, 0));
}

__device__ __forceinline__ uint4 chunk_load(__amdgpu_buffer_rsrc_t rs, bool ok, int64_t off_halves) {
  const uint32_t off = ok ? (uint32_t)(off_halves * 2) : kOffOOB;
  return __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(rs, off, 0, 0));
}

// Loads rows [0, rows) x halves [k0, k0 + 64) of a row-major fp16 matrix with
// leading dimension ld (halves); rows past `rows` and columns past `kmax` read
// as zero.  rows * ld * 2 must fit in 31 bits.
__device__ __forceinline__ void slab_load(const _Float16* __restrict__ base, int rows, int64_t ld, int k0,
                                          int kmax, SlabRegs& r) {
  const __amdgpu_buffer_rsrc_t rs = tile_rsrc(base, rows, ld);
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int c = threadIdx.x + kWG * q;
    const int row = c >> 3, col = (c & 7) * 8;
    r.v[q] = chunk_load(rs, row < rows && k0 + col < kmax, (int64_t)row * ld + k0 + col);
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

// ---------------------------------------------------------------------------
// Block shape: WM x WN waves, each owning TI x TJ tiles of 32 x 32, so a
// workgroup computes (WM*TI*32) x (WN*TJ*32) of C = A . B^T.  Larger per-wave
// tiles read fewer LDS bytes per MFMA: (TI + TJ) / (TI * TJ) KB.
template <int WM_, int WN_, int TI_, int TJ_, int MW_ = 2>
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
  static constexpr int kLdsHalves = 2 * (BM + BN) * kLdk;   // two K-slab stages of A and B
  // waves per SIMD the register budget is held to (512 / MW registers per lane)
  static constexpr int kMinWaves = MW_;
  static_assert(kChunksA % kThreads == 0 && kChunksB % kThreads == 0, "slab must split evenly");
};

template <int N>
__device__ __forceinline__ void slab_load_n(__amdgpu_buffer_rsrc_t rs, int rows, int64_t ld, int k0, int kmax,
                                            uint4 (&r)[N], int nthreads) {
#pragma unroll
  for (int q = 0; q < N; ++q) {
    const int c = threadIdx.x + nthreads * q;
    const int row = c >> 3, col = (c & 7) * 8;
    r[q] = chunk_load(rs, row < rows && k0 + col < kmax, (int64_t)row * ld + k0 + col);
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

// C tile of one workgroup; lds holds C::kLdsHalves halves (two K-slab stages
// of A and B).  acc[ti][tj] holds rows wm*TI*32 + ti*32 + acc_row(r, lane) of A
// and column wn*TJ*32 + tj*32 + lane%32 of B, with wm = wave / WN, wn = wave %
// WN.
//
// Pipeline: global loads run two slabs ahead of the MFMAs in two register
// sets (three slabs ahead in three sets when NS > 0 and SETS = 3; one slab
// ahead in one set when SETS = 1, for tiles whose accumulators leave no room
// for more: the loads of slab s + 2 are issued once slab s + 1 is in LDS, so
// they have one slab's MFMAs to land); slab s is multiplied from LDS stage
// s % 2 while slab s + 1 is written to the other stage, so one barrier per
// slab suffices and the LDS writes overlap the MFMAs.  With NS > 0 the
// reduction has exactly NS slabs (kdim = 64 NS) and the loop is unrolled,
// which lets the compiler wait for exactly the loads each LDS store needs
// (across a loop back edge it waits for all of them), and loads past the last
// slab are dropped at compile time.  NS = 0 takes kdim at run time; there the
// loads past the last slab are issued too (they fall outside the buffer
// bound, read zeros and touch no memory), so that no load sits behind a
// branch.  go_on() runs once the first slabs' loads are in flight; if it
// returns false the tile is abandoned and gemm_tile returns false.
template <class C, int NS = 0, int SETS = 3, class Go>
__device__ __forceinline__ bool gemm_tile(const _Float16* __restrict__ A, int ra, const _Float16* __restrict__ B,
                                          int rb, int64_t ld, int kdim, _Float16* lds,
                                          floatx16 (&acc)[C::TI][C::TJ], Go&& go_on) {
  auto sa = [&](int i) -> _Float16* { return lds + i * ((C::BM + C::BN) * kLdk); };
  auto sb = [&](int i) -> _Float16* { return lds + i * ((C::BM + C::BN) * kLdk) + C::BM * kLdk; };
  const int wave = threadIdx.x >> 6;
  const int wm = wave / C::WN, wn = wave % C::WN;
#pragma unroll
  for (int a = 0; a < C::TI; ++a)
#pragma unroll
    for (int b = 0; b < C::TJ; ++b)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[a][b][r] = 0.0f;
  auto compute = [&](int st) {
#pragma unroll
    for (int kk = 0; kk < kBK / 16; ++kk) {
      half8 fa[C::TI], fb[C::TJ];
#pragma unroll
      for (int t = 0; t < C::TI; ++t) fa[t] = frag_load(sa(st), wm * C::TI * 32 + t * 32, kk);
#pragma unroll
      for (int t = 0; t < C::TJ; ++t) fb[t] = frag_load(sb(st), wn * C::TJ * 32 + t * 32, kk);
#pragma unroll
      for (int a = 0; a < C::TI; ++a)
#pragma unroll
        for (int b = 0; b < C::TJ; ++b)
          acc[a][b] = __builtin_amdgcn_mfma_f32_32x32x16_f16(fa[a], fb[b], acc[a][b], 0, 0, 0);
    }
  };
  const __amdgpu_buffer_rsrc_t rsA = tile_rsrc(A, ra, ld), rsB = tile_rsrc(B, rb, ld);
  static_assert(SETS == 3 || (SETS == 1 && NS > 0), "three register sets, or one with an unrolled reduction");
  // (NS > 0: the caller guarantees kdim = 64 NS <= ld)
  if constexpr (NS > 0) {
    // exactly NS slabs: loads past the last slab are not issued
    auto load = [&](int slab, uint4 (&xa)[C::kPerA], uint4 (&xb)[C::kPerB]) {
      if (slab < NS) {
        slab_load_n<C::kPerA>(rsA, ra, ld, slab * kBK, kdim, xa, C::kThreads);
        slab_load_n<C::kPerB>(rsB, rb, ld, slab * kBK, kdim, xb, C::kThreads);
      }
    };
    if constexpr (SETS == 1) {
      uint4 xa[C::kPerA], xb[C::kPerB];
      load(0, xa, xb);
      if (!go_on()) return false;
      slab_store_n<C::kPerA>(sa(0), xa, C::kThreads);
      slab_store_n<C::kPerB>(sb(0), xb, C::kThreads);
      load(1, xa, xb);
      __syncthreads();
#pragma unroll
      for (int s = 0; s < NS; ++s) {
        compute(s & 1);
        if (s + 1 < NS) {
          slab_store_n<C::kPerA>(sa((s + 1) & 1), xa, C::kThreads);
          slab_store_n<C::kPerB>(sb((s + 1) & 1), xb, C::kThreads);
          load(s + 2, xa, xb);
        }
        __syncthreads();
      }
      return true;
    } else {
      // three register sets, so each slab's loads are issued three slabs
      // before its LDS store (set and stage indices are compile-time
      // constants after unrolling)
      uint4 xa[3][C::kPerA], xb[3][C::kPerB];
#pragma unroll
      for (int u = 0; u < 3; ++u) load(u, xa[u], xb[u]);
      if (!go_on()) return false;
      slab_store_n<C::kPerA>(sa(0), xa[0], C::kThreads);
      slab_store_n<C::kPerB>(sb(0), xb[0], C::kThreads);
      load(3, xa[0], xb[0]);
      __syncthreads();
#pragma unroll
      for (int s = 0; s < NS; ++s) {
        compute(s & 1);
        if (s + 1 < NS) {
          const int u = (s + 1) % 3;
          slab_store_n<C::kPerA>(sa((s + 1) & 1), xa[u], C::kThreads);
          slab_store_n<C::kPerB>(sb((s + 1) & 1), xb[u], C::kThreads);
          load(s + 4, xa[u], xb[u]);
        }
        __syncthreads();
      }
      return true;
    }
  }
  const int S = (kdim + kBK - 1) / kBK;
  uint4 a0[C::kPerA], b0[C::kPerB], a1[C::kPerA], b1[C::kPerB];
  slab_load_n<C::kPerA>(rsA, ra, ld, 0, kdim, a0, C::kThreads);
  slab_load_n<C::kPerB>(rsB, rb, ld, 0, kdim, b0, C::kThreads);
  slab_load_n<C::kPerA>(rsA, ra, ld, kBK, kdim, a1, C::kThreads);
  slab_load_n<C::kPerB>(rsB, rb, ld, kBK, kdim, b1, C::kThreads);
  // the caller may stop here (its check's own loads overlap the first slabs')
  if (!go_on()) return false;
  slab_store_n<C::kPerA>(sa(0), a0, C::kThreads);
  slab_store_n<C::kPerB>(sb(0), b0, C::kThreads);
  slab_load_n<C::kPerA>(rsA, ra, ld, 2 * kBK, kdim, a0, C::kThreads);
  slab_load_n<C::kPerB>(rsB, rb, ld, 2 * kBK, kdim, b0, C::kThreads);
  __syncthreads();
#pragma unroll
  for (int s = 0; s < (NS > 0 ? NS : S); s += 2) {
    // even slab s from stage 0; slab s + 1 (a1/b1) goes to stage 1
    compute(0);
    slab_store_n<C::kPerA>(sa(1), a1, C::kThreads);
    slab_store_n<C::kPerB>(sb(1), b1, C::kThreads);
    slab_load_n<C::kPerA>(rsA, ra, ld, (s + 3) * kBK, kdim, a1, C::kThreads);
    slab_load_n<C::kPerB>(rsB, rb, ld, (s + 3) * kBK, kdim, b1, C::kThreads);
    __syncthreads();
    if (s + 1 >= S) break;
    // odd slab s + 1 from stage 1; slab s + 2 (a0/b0) goes to stage 0
    compute(1);
    slab_store_n<C::kPerA>(sa(0), a0, C::kThreads);
    slab_store_n<C::kPerB>(sb(0), b0, C::kThreads);
    slab_load_n<C::kPerA>(rsA, ra, ld, (s + 4) * kBK, kdim, a0, C::kThreads);
    slab_load_n<C::kPerB>(rsB, rb, ld, (s + 4) * kBK, kdim, b0, C::kThreads);
    __syncthreads();
  }
  return true;
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

__device__ __forceinline__ int xcd_remap32(int bid, int nblocks) {
  const int q = nblocks >> 3, rem = nblocks & 7;
  const int x = bid & 7;
  return x * q + (x < rem ? x : rem) + (bid >> 3);
}

// Workgroup index -> logical tile for a grid made of groups of P consecutive
// logical tiles that share operand rows: XCD x = bid % 8 takes whole groups,
// x, x + 8, x + 16, ..., each group's tiles in order, so a group stays in one
// L2 while the groups are dealt round-robin over the XCDs (tiles at the end of
// the logical order, e.g. tiles that turn out to be empty, are spread over all
// XCDs rather than all falling to the last).  The grid's tail of fewer than 8
// whole groups is split into contiguous ranges as by xcd_remap32.  A bijection
// of [0, nblocks).
__device__ __forceinline__ int group_interleave(int bid, int nblocks, int P) {
  const int span = 8 * P;
  const int full = nblocks / span;
  if (bid < full * span) {
    const int i = bid >> 3;
    return (i / P) * span + (bid & 7) * P + i % P;
  }
  return full * span + xcd_remap32(bid - full * span, nblocks - full * span);
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
