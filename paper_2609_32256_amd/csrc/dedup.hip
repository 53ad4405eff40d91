// The epsilon error-bounded near-duplicate test (Section 2.3, Algorithm
// "admit") with exhaustive candidates, as a batched GPU pipeline.
//
// Semantics (exact, independent of batching): arrivals are taken in global
// order; arrival i is dropped iff some retained row y has
// sum_d (x_i,d - y_d)^2 <= 2 - 2 tau (Eq. identity; squared l2 on the float32
// rows as exact reals, inclusive), and its representative is the lowest such
// y (Appendix "Representative selection"); otherwise it is retained.
//
// Pipeline for one call (rows are processed in chunks of at most 4096, which
// by the semantics above changes nothing):
//   prep      -- validate rows, fp16 copy scaled by 2^8, ||x||^2/2, error term
//   screen S  -- fp16 MFMA  C = store . chunk^T ; each pair is classified
//                against delta^2 with a rigorous bound E on the screen's error:
//                definitely in, definitely out, or ambiguous.  Per arrival the
//                lowest definite store row is kept (atomicMin); ambiguous rows
//                below it go to a pair list.
//   screen B  -- the same on the chunk's lower triangle (j < i); definite
//                pairs set bits of an n x n edge bitmap, ambiguous ones go to
//                the pair list.
//   verify    -- each ambiguous pair is re-decided in binary64 (one wave per
//                pair); a pair within rounding distance of delta^2 is decided
//                by the same wave on exact integers (exact.h: six 64-bit limbs
//                hold the squared distance scaled to an integer).
//   resolve   -- in a workgroup of 1,024 threads: a row with a store hit is
//                dropped, a row with no in-chunk edge is kept; the others copy
//                their earlier in-chunk neighbours into LDS lists and decide in
//                rounds (a row decides once every earlier neighbour has: it
//                takes the lowest kept one, or is kept when none is).  When
//                the lists overflow LDS, one wave walks the chunk in arrival
//                order with the kept mask in its registers instead.
//   append    -- kept rows join the store; for dropped rows ||x - rep||^2 in
//                binary64 feeds the measured bound delta_hat.
// The resolve and the append are one launch (k_resolve_append): each
// workgroup resolves the chunk's rows up to its own last one in its LDS and
// appends its 16 rows.  The banded store keeps them apart (k_resolve,
// k_lsh_insert, k_append), since its index insertion sits between them.
//
// Error bound of the screen (dot-product units), for rows a, b:
//   |c16 - a.b| <= K1 (||a||^2 + ||b||^2)/2 + K2 (||a||_1 + ||b||_1) + K3
// from fp16 input rounding (relative 2^-11, or 2^-22 absolute for scaled
// subnormals even if flushed), exact fp16 products in fp32, and fp32
// accumulation in any order (gamma_D with 2u per addition); the AM-GM step
// ||a|| ||b|| <= (||a||^2 + ||b||^2)/2 makes it a sum of per-row terms, and the
// per-row term also absorbs the float32 roundings of the epilogue.
#include <hip/hip_ext.h>

#include <cmath>
#include <cstdlib>
#include <cstring>
#include <vector>

#include "exact.h"
#include "lam_internal.h"
#include "mfma_tile.h"
#include "qround.h"
#include "wave.h"

namespace lam {

namespace {

constexpr int kChunk = 4096;           // rows per resolve (64 lanes x 64 bits)
constexpr int kNone = 0x7fffffff;       // "no store hit"
constexpr int kGroupA = 8;              // store tiles per group in the screen's tile order
constexpr float kScale = 256.0f;        // fp16 operands hold x * 2^8
// Largest accepted |x| (exclusive): 2^8 x rounds to a finite float16 exactly
// when 2^8 |x| < 65520 (the midpoint between the largest finite value 65504
// and 2^16), i.e. |x| < 2^8 - 2^-4.
constexpr float kXLimit = 255.9375f;
constexpr float kInvScale2 = 1.0f / 65536.0f;

enum Scratch { S_X16 = 0, S_ROWF, S_CHUNK, S_BITMAP, S_PAIRS, S_STATUS, S_G };

// Device bookkeeping of a store.  Kernels keep it current, so calls that do
// not wait for the device need no host round trip: the host reads it when a
// call needs exact values (lam_store_get_info, capacity near full, ...).
struct StoreMeta {
  int32_t m;                       // retained rows
  uint32_t err_calls;              // calls since the host last looked that had invalid input
  int64_t n_seen;                  // arrivals taken so far (global id of the next arrival)
  unsigned long long dhat2_bits;   // max merged squared distance of the run (binary64 bits)
  uint32_t err_bits;               // bit 0: non-finite input, bit 1: a coordinate with |x| >= kXLimit
  uint32_t absmax_bits;            // max |x| over the retained rows (float32 bits; non-negative
                                   // floats order as their bits), the store codec's width input
  uint32_t hnmax_bits;             // max ||x||^2 / 2 over the retained rows (float32 bits)
  uint32_t pad;
};

// Chunk-level counters (in the S_CHUNK scratch, after the per-row arrays).
struct ChunkCounters {
  uint32_t npairs;        // ambiguous pairs appended in this chunk
  uint32_t n_escalate;
  // one 64-bit word, added to with one atomic per append workgroup:
  uint32_t blocks_done;   // append workgroups finished (last one exports the status words)
  uint32_t kept;          // rows of the chunk kept, summed by the workgroups of k_resolve_append
};
static_assert(offsetof(ChunkCounters, blocks_done) % 8 == 0 &&
                  offsetof(ChunkCounters, kept) == offsetof(ChunkCounters, blocks_done) + 4,
              "blocks_done and kept form one little-endian 64-bit word");

__device__ __forceinline__ bool skip_all(const DevFlags* f) {
  return (f->nonfinite | f->out_of_range | f->pair_overflow) != 0u;
}

// Smallest |d^2 - delta^2| among the pairs the exact test decided: kept as the
// complement of the binary64 bits (non-negative doubles order as their bits),
// so that the zeroed status word means "none".
__device__ __forceinline__ void note_margin(DevFlags* f, double m) {
  if (m < 1e300) atomicMax(&f->margin_inv, ~(unsigned long long)__double_as_longlong(m));
}

__device__ __forceinline__ float round_up_f32(double d) {
  float f = (float)d;
  if ((double)f < d) f = __uint_as_float(f >= 0.0f ? __float_as_uint(f) + 1u : __float_as_uint(f) - 1u);
  return f;
}
__device__ __forceinline__ float round_down_f32(double d) {
  float f = (float)d;
  if ((double)f > d) f = __uint_as_float(f > 0.0f ? __float_as_uint(f) - 1u : (f == 0.0f ? 0x80000001u : __float_as_uint(f) + 1u));
  return f;
}

// ------------------------------------------------------------------ prep
// Per-chunk state: the first store hit, the in-chunk edge flag, the order-
// encoded max cosine and the row's edge bitmap words.  Rows of the first chunk
// are initialised by k_prep, the others by k_chunk_init.
struct ChunkState {
  int32_t* firstHit;
  uint32_t* hasEdge;
  uint32_t* maxcos;
  uint64_t* bitmap;
  int W;
  int nB;                  // rows of the first chunk
  ChunkCounters* cc;
  StoreMeta* meta;
  int32_t m_first;         // store size at the start of the call, or -1 to leave it
  int32_t reset_meta;      // the store was cleared since its last ingest: zero its bookkeeping first
};

__device__ __forceinline__ void init_chunk_row(const ChunkState& c, int64_t r, int lane) {
  for (int w = lane; w < c.W; w += 64) c.bitmap[r * c.W + w] = 0ull;
  if (lane == 0) {
    c.firstHit[r] = kNone;
    c.hasEdge[r] = 0u;
    c.maxcos[r] = 0x007fffffu;  // order-encoded -inf
  }
}

constexpr int kPrepVec = 4;   // float4 of a row per lane held in registers (D <= 1,024)

__global__ __launch_bounds__(256) void k_prep(const float* __restrict__ x, int64_t n, int D,
                                              _Float16* __restrict__ x16, float* __restrict__ hn,
                                              float* __restrict__ eterm, double K1, double K2, double K3h,
                                              DevFlags* __restrict__ flags, ChunkState cs) {
  const int lane = threadIdx.x & 63;
  const int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  const float* p = x + row * D;
  // For D <= 1,024 the row's loads are issued first, through a buffer resource
  // (no memory touched past the row, nor for a row past n), so their latency
  // overlaps the chunk-state stores below.
  const bool vec = D <= 256 * kPrepVec;
  float4 v4[kPrepVec];
  {
    const __amdgpu_buffer_rsrc_t rs = f32_rsrc(p, (vec && row < n) ? D : 0);
#pragma unroll
    for (int u = 0; u < kPrepVec; ++u)
      v4[u] = __builtin_bit_cast(float4, __builtin_amdgcn_raw_buffer_load_b128(rs, (uint32_t)(u * 256 + lane * 4) * 4u, 0, 0));
  }
  if (blockIdx.x == 0 && threadIdx.x == 0) {
    cs.cc->npairs = 0u;
    cs.cc->n_escalate = 0u;
    cs.cc->blocks_done = 0u;
    cs.cc->kept = 0u;
    if (cs.reset_meta) *cs.meta = StoreMeta{};       // lam_store_clear, applied by the next ingest
    if (cs.m_first >= 0) cs.meta->m = cs.m_first;   // a retried call starts from the store as it was
  }
  if (row < cs.nB) init_chunk_row(cs, row, lane);
  if (row >= n) return;
  _Float16* q = x16 + row * D;
  double na = 0.0, l1 = 0.0;
  bool nf = false, rng = false;
  auto take = [&](const float4& v, int d) {
    const float c[4] = {v.x, v.y, v.z, v.w};
    _Float16 h[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const float a = fabsf(c[r]);
      nf |= !(a <= 3.402823466e38f);
      rng |= !(a < kXLimit);
      na = fma((double)c[r], (double)c[r], na);
      l1 += (double)a;
      h[r] = (_Float16)(c[r] * kScale);
    }
    uint2 packed;
    __builtin_memcpy(&packed, h, 8);
    *reinterpret_cast<uint2*>(q + d) = packed;
  };
  if (vec) {
#pragma unroll
    for (int u = 0; u < kPrepVec; ++u) {
      const int d = u * 256 + lane * 4;
      if (d >= D) break;
      take(v4[u], d);
    }
  } else {
    for (int d = lane * 4; d < D; d += 256) take(*reinterpret_cast<const float4*>(p + d), d);
  }
  na = wave_sum_f64(na);
  l1 = wave_sum_f64(l1);
  const unsigned long long bn = __ballot(nf), br = __ballot(rng);
  if (lane == 0) {
    if (bn) atomicAdd(&flags->nonfinite, 1u);
    if (br) atomicAdd(&flags->out_of_range, 1u);
    hn[row] = (float)(0.5 * na);
    const double et = K1 * 0.5 * na + K2 * l1 + K3h + 0x1p-23 * (na + 1.0);
    eterm[row] = round_up_f32(et);
  }
}

// ------------------------------------------------------------------ chunk init
// Clears the chunk state for the second and later chunks of a call.
__global__ void k_chunk_init(ChunkState cs) {
  const int lane = threadIdx.x & 63;
  const int64_t waves = (int64_t)gridDim.x * (blockDim.x >> 6);
  for (int64_t r = (int64_t)blockIdx.x * (blockDim.x >> 6) + (threadIdx.x >> 6); r < cs.nB; r += waves)
    init_chunk_row(cs, r, lane);
  if (blockIdx.x == 0 && threadIdx.x == 0) {
    cs.cc->npairs = 0u;
    cs.cc->n_escalate = 0u;
    cs.cc->blocks_done = 0u;
    cs.cc->kept = 0u;
  }
}

// ------------------------------------------------------------------ screens
struct ScreenArgs {
  const _Float16* As;       // store rows (fp16 x 2^8)
  const float* hnS;         // ||y||^2 / 2 of store rows
  const float* etS;         // error term of store rows
  const StoreMeta* meta;    // store size
  int m_exact;              // store size when the host knows it, else -1 (read meta)
  int capA;                 // store capacity (rows that may be read before the size is known)
  const _Float16* B;        // chunk rows (arrivals)
  const float* hnB;         // ||b||^2 / 2 of chunk rows
  const float* etB;         // error term of chunk rows
  int nB;
  int D;
  int ntB;                  // chunk tiles
  int64_t nb0;              // workgroups screening against the store (first in the grid)
  int64_t nb1;              // workgroups screening inside the chunk (lower triangle)
  double half_d2;           // delta^2 / 2
  int32_t* firstHit;        // store screen
  uint32_t* maxcos;         // store screen, order-encoded (WANT_MAX)
  uint64_t* bitmap;         // chunk screen
  int W;                    // bitmap words per row
  uint32_t* hasEdge;
  float* G;                 // chunk screen dot matrix (WANT_MAX), ldG = nB
  int2* pairs;
  uint32_t pair_cap;
  ChunkCounters* cc;
  DevFlags* flags;
};

// Lists the ambiguous pairs (i, row_of(e)) for the set bits e of `bits`: one
// atomic reserves the lane's whole run of list entries (one per pair had put
// a round trip per pair on the tile's critical path).
template <class RowOf>
__device__ __forceinline__ void push_pairs(const ScreenArgs& a, int i, int kind, uint64_t bits, RowOf&& row_of) {
  const uint32_t cnt = (uint32_t)__popcll(bits);
  if (cnt == 0u) return;
  const uint32_t idx0 = atomicAdd(&a.cc->npairs, cnt);
  atomicAdd(&a.flags->n_pairs, cnt);
  uint32_t idx = idx0;
  while (bits) {
    const int e = __builtin_ctzll(bits);
    bits &= bits - 1ull;
    if (idx < a.pair_cap) a.pairs[idx] = make_int2(i | (kind << 31), row_of(e));
    ++idx;
  }
  if (idx0 + cnt > a.pair_cap) {
    atomicOr(&a.flags->pair_overflow, 1u);
    atomicMax(&a.flags->pairs_needed, idx0 + cnt);   // capacity that would have sufficed
  }
}

// One launch screens a chunk against the store (workgroups [0, nb0), MODE 0:
// A = store rows, B = chunk rows) and against itself (workgroups
// [nb0, nb0 + nb1), MODE 1: A = B = chunk rows, pairs ia < ib only).  The
// A side of the error bound is the largest per-row term among the tile's own
// A rows.
// NS > 0: the reduction has exactly NS slabs of 64 (D = 64 NS), fully
// unrolled; NS = 0: any D.  Each is its own kernel, so each gets its own
// register allocation (the unrolled ones need no scratch memory).
template <class C, bool WANT_MAX, int NS, int SETS = 3>
__global__ __launch_bounds__(C::kThreads, C::kMinWaves) void k_screen(ScreenArgs a) {
  static_assert(C::BM == C::BN, "the in-chunk triangle needs square tiles");
  static_assert(C::BM <= C::kThreads, "one thread per A row for the row terms");
  __shared__ _Float16 lds[C::kLdsHalves];
  __shared__ __attribute__((aligned(16))) float hbA[C::BM];
  __shared__ float emx[C::kWaves];
  // (no early exit on the status words: the screen writes only chunk scratch,
  // and every kernel that writes caller outputs or the store checks them)
  const int bid = (int)blockIdx.x;
  const int nb0 = (int)a.nb0;
  const int MODE = bid < nb0 ? 0 : 1;
  int ta, tb;
  if (MODE == 0) {
    // Grouped order: a group is gA store tiles against every chunk tile,
    // swept store tile fastest, and one XCD takes a whole group, so the tiles
    // in flight on one XCD (two per CU, 64 in all: 8 store tiles and 8 chunk
    // tiles either way -- one group of gA = 8, or eight groups of one store
    // tile when the chunk has at most 8 tiles) stay inside its L2 and each
    // store tile leaves HBM once.  With the store size known the grid is
    // exact and each XCD takes a contiguous range of groups; when the grid
    // covers an upper bound of the size, groups go round-robin to the XCDs so
    // that the empty tiles at its end are shared out instead of idling the
    // last XCDs.
    const bool exact = a.m_exact >= 0;
    const int gA = (exact || a.ntB > 8) ? kGroupA : 1;
    const int per_group = gA * a.ntB;
    const int logical = exact ? xcd_remap32(bid, nb0) : group_interleave(bid, nb0, per_group);
    const int ntA = nb0 / a.ntB;
    const int g = logical / per_group, l = logical - g * per_group;
    const int ta0 = g * gA;
    const int gsize = min(gA, ntA - ta0);
    ta = ta0 + l % gsize;
    tb = l / gsize;
  } else {
    // lower-triangular tile pairs ta <= tb, row-major over tb
    const int64_t logical = xcd_remap(bid - nb0, a.nb1);
    int t = (int)((sqrt(8.0 * (double)logical + 1.0) - 1.0) * 0.5);
    while ((int64_t)(t + 1) * (t + 2) / 2 <= logical) ++t;
    while ((int64_t)t * (t + 1) / 2 > logical) --t;
    tb = t;
    ta = (int)(logical - (int64_t)t * (t + 1) / 2);
  }
  const _Float16* A = MODE == 0 ? a.As : a.B;
  const float* hnA = MODE == 0 ? a.hnS : a.hnB;
  const float* etA = MODE == 0 ? a.etS : a.etB;
  const int rowsB = min(C::BN, a.nB - tb * C::BN);
  // When the host does not know the store size, loads start against the
  // capacity bound and the size is read while they are in flight; tiles past
  // it stop before the main loop.  Rows between size and capacity only reach
  // accumulators the epilogue masks out.
  const bool known = MODE == 1 || a.m_exact >= 0;
  const int nA0 = MODE == 1 ? a.nB : (known ? a.m_exact : a.capA);
  const int rowsLim = min(C::BM, nA0 - ta * C::BM);
  if (rowsLim <= 0 || rowsB <= 0) return;
  int rowsA = rowsLim;
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int wn0 = wave % C::WN;

  // Row terms of both sides: loaded before the GEMM, used after it, so their
  // latency hides behind the first slabs.
  const __amdgpu_buffer_rsrc_t rhA = f32_rsrc(hnA + (int64_t)ta * C::BM, rowsLim);
  const __amdgpu_buffer_rsrc_t reA = f32_rsrc(etA + (int64_t)ta * C::BM, rowsLim);
  const __amdgpu_buffer_rsrc_t rhB = f32_rsrc(a.hnB + (int64_t)tb * C::BN, rowsB);
  const __amdgpu_buffer_rsrc_t reB = f32_rsrc(a.etB + (int64_t)tb * C::BN, rowsB);
  const float hA = buf_f32(rhA, (int)threadIdx.x < rowsLim, threadIdx.x);
  float eA = buf_f32(reA, (int)threadIdx.x < rowsLim, threadIdx.x);
  float hB[C::TJ], eB[C::TJ];
#pragma unroll
  for (int tj = 0; tj < C::TJ; ++tj) {
    const int ibl = wn0 * C::TJ * 32 + tj * 32 + (lane & 31);
    hB[tj] = buf_f32(rhB, ibl < rowsB, ibl);
    eB[tj] = buf_f32(reB, ibl < rowsB, ibl);
  }

  floatx16 acc[C::TI][C::TJ];
  const _Float16* tA = A + (int64_t)ta * C::BM * a.D;
  const _Float16* tB = a.B + (int64_t)tb * C::BN * a.D;
  // Called by gemm_tile once the first slabs' loads are issued and before it
  // waits for any: the store size when the host does not know it, then the
  // A side's row terms into LDS and each wave's largest error term among the
  // tile's rows (the error bound uses the tile's largest), all while the
  // slabs load.  gemm_tile ends with a barrier, so the epilogue sees them.
  auto go_on = [&]() {
    if (!known) {
      rowsA = min(C::BM, a.meta->m - ta * C::BM);
      if (rowsA <= 0) return false;
    }
    if ((int)threadIdx.x < C::BM) hbA[threadIdx.x] = hA;
    const float e = wave_max_f32((int)threadIdx.x < rowsA ? eA : 0.0f);
    if (lane == 0) emx[wave] = e;
    return true;
  };
  if (!gemm_tile<C, NS, SETS>(tA, rowsLim, tB, rowsB, a.D, a.D, lds, acc, go_on)) return;
  const int wm = wave / C::WN, wn = wave % C::WN;
  float ebA = emx[0];
#pragma unroll
  for (int w = 1; w < C::kWaves; ++w) ebA = fmaxf(ebA, emx[w]);
#pragma unroll
  for (int tj = 0; tj < C::TJ; ++tj) {
    const int ibl = wn * C::TJ * 32 + tj * 32 + (lane & 31);
    const int ib = tb * C::BN + ibl;
    const bool vB = ibl < rowsB;
    float thrAmb = 3.0e38f, thrIn = 3.0e38f;
    if (vB) {
      const double base = (double)hB[tj] - a.half_d2;
      const double e = (double)eB[tj] + (double)ebA;
      thrAmb = round_down_f32(base - e);
      thrIn = round_up_f32(base + e);
    }
    float mx = -3.0e38f, cmax = -3.0e38f;
    // A tile with every A row valid, against the store or below the chunk's
    // diagonal (ta < tb: every A row precedes every B row): no element needs
    // a validity test (a lane past rowsB has thrAmb = 3e38, which no finite
    // mx reaches)
    const bool full = !WANT_MAX && rowsA == C::BM && (MODE == 0 || ta < tb);
#pragma unroll
    for (int ti = 0; ti < C::TI; ++ti) {
      // the row terms of this lane's 16 rows of the 32 x 32 tile: four
      // consecutive rows per 16-byte LDS read, all read (every entry of hbA is
      // written) before any is used, so no read waits behind a row's validity
      const int rb = wm * C::TI * 32 + ti * 32;
      // with four or more blocks per wave, keep each block's reads with its
      // use (hoisted together they would not fit beside the accumulators)
      if constexpr (C::TI * C::TJ >= 4) __builtin_amdgcn_sched_barrier(0);
      float4 h4[4];
#pragma unroll
      for (int g = 0; g < 4; ++g) h4[g] = *reinterpret_cast<const float4*>(&hbA[rb + acc_row(4 * g, lane)]);
      if (full) {
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const float4 hg = h4[r >> 2];
          const float hv = (r & 3) == 0 ? hg.x : (r & 3) == 1 ? hg.y : (r & 3) == 2 ? hg.z : hg.w;
          mx = fmaxf(mx, acc[ti][tj][r] * kInvScale2 - hv);
        }
        continue;
      }
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int ial = rb + acc_row(r, lane);
        const int ia = ta * C::BM + ial;
        const bool valid = vB && ial < rowsA && (MODE == 0 || ia < ib);
        const float4 hg = h4[r >> 2];
        const float hv = (r & 3) == 0 ? hg.x : (r & 3) == 1 ? hg.y : (r & 3) == 2 ? hg.z : hg.w;
        const float dot = acc[ti][tj][r] * kInvScale2;
        const float v = dot - hv;
        mx = valid ? fmaxf(mx, v) : mx;
        if (WANT_MAX) {
          if (MODE == 0) cmax = valid ? fmaxf(cmax, dot) : cmax;
          else if (valid) a.G[(int64_t)ib * a.nB + ia] = dot;
        }
      }
    }
    if (WANT_MAX && MODE == 0 && vB && cmax > -3.0e38f) atomicMax(&a.maxcos[ib], f2ord(cmax));
    const bool hot = mx >= thrAmb;
    if (__ballot(hot) == 0ull) continue;
    // Rare path.  Classify this lane's elements into bit masks (bit e = ti*16 + r;
    // A rows increase with e), then walk the set bits -- the accumulators are
    // only ever indexed statically.
    static_assert(C::TI * 16 <= 64, "one 64-bit mask per lane and B column");
    uint64_t cand = 0ull, def = 0ull;
#pragma unroll
    for (int ti = 0; ti < C::TI; ++ti) {
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int ial = wm * C::TI * 32 + ti * 32 + acc_row(r, lane);
        const int ia = ta * C::BM + ial;
        const bool valid = vB && ial < rowsA && (MODE == 0 || ia < ib);
        const float v = acc[ti][tj][r] * kInvScale2 - hbA[ial];
        const uint64_t bit = 1ull << (ti * 16 + r);
        cand |= (valid && v >= thrAmb) ? bit : 0ull;
        def |= (valid && v >= thrIn) ? bit : 0ull;
      }
    }
    if (!hot) continue;
    auto row_of = [&](int e) { return ta * C::BM + wm * C::TI * 32 + (e >> 4) * 32 + acc_row(e & 15, lane); };
    if (MODE == 0) {
      // lowest definite row, and the ambiguous rows below it
      const int edef = def ? __builtin_ctzll(def) : 64;
      push_pairs(a, ib, 0, cand & ~def & (edef < 64 ? ((1ull << edef) - 1ull) : ~0ull), row_of);
      if (edef < 64) atomicMin(&a.firstHit[ib], row_of(edef));
    } else {
      // a lane's rows are 64 consecutive rows from a multiple of 64, so its
      // definite edges fall in one bitmap word: one atomic for all of them
      static_assert(C::TI * 32 == 64 && C::BM % 64 == 0, "a lane's A rows fill one bitmap word");
      if (def) {
        uint64_t word = 0ull, d = def;
        while (d) {
          const int e = __builtin_ctzll(d);
          d &= d - 1ull;
          word |= 1ull << (row_of(e) & 63);
        }
        atomicOr(reinterpret_cast<unsigned long long*>(&a.bitmap[(int64_t)ib * a.W + (row_of(0) >> 6)]), word);
        a.hasEdge[ib] = 1u;
      }
      push_pairs(a, ib, 1, cand & ~def, row_of);
    }
  }
}

// 128 x 128, eight waves of 64 x 32 held to 128 registers, so that LDS (two
// 37 KB stages) and registers both allow two workgroups (four waves per SIMD)
// per CU: the short reductions (D = 768) are latency-bound, and this
// occupancy took the subset stream's screen from 1.16 to 1.01 ms against
// four waves of 64 x 64 at two waves per SIMD.
using ScreenTile = Tile<2, 4, 2, 1, 4>;

// 256 x 256, sixteen waves of 64 x 64 (64 accumulators per lane, held to 128
// registers) at four waves per SIMD: one workgroup per CU (two 74 KB
// stages), half the global loads per flop of the 128 x 128 tile and a third
// fewer LDS bytes per MFMA, with one slab of loads in flight in registers.
// Faster when a launch holds many tiles (the steady state of large stores);
// a lone tile takes more than twice as long, so small launches keep
// ScreenTile.  (Eight waves of 128 x 64 run as fast but need every register
// of two waves per SIMD and spill on the rare path.)
using ScreenTileL = Tile<4, 4, 2, 2, 4>;
constexpr int64_t kLargeTileMinTiles = 768;   // automatic choice: large tiles from this many

// ------------------------------------------------------------------ merge predicate of one pair
// sum_d (a_d - b_d)^2 <= delta^2 for float32 rows a, b (16-byte aligned, D a
// multiple of 4) by a group of G lanes of one wave: the squared distance in
// binary64 (error below (D + 2) u64 d^2 in any order); a pair within that
// distance of delta^2 is decided on exact integers (exact.h), so every
// decision is the exact one.  Every lane of the group returns the decision;
// *escalated tells whether the exact path ran and *margin is |s - delta^2| for
// the binary64 sum s.  The G lanes of a group must run it together.
template <int G>
__device__ bool pair_within(const float* pa, const float* pb, int D, double d2, const Big6& thr, bool* escalated,
                            double* margin) {
  static_assert(G == 16 || G == 32 || G == 64, "a group is a power of two within one wave");
  const int gl = (int)threadIdx.x & (G - 1);
  double s = 0.0;
  for (int d = gl * 4; d < D; d += 4 * G) {
    const float4 u = *reinterpret_cast<const float4*>(pa + d);
    const float4 v = *reinterpret_cast<const float4*>(pb + d);
    const double t0 = (double)u.x - (double)v.x, t1 = (double)u.y - (double)v.y;
    const double t2 = (double)u.z - (double)v.z, t3 = (double)u.w - (double)v.w;
    s = fma(t0, t0, s);
    s = fma(t1, t1, s);
    s = fma(t2, t2, s);
    s = fma(t3, t3, s);
  }
  if constexpr (G == 64) {
    s = wave_sum_f64(s);   // a whole wave: every lane holds the sum
  } else {
    for (int o = G / 2; o > 0; o >>= 1) s += __shfl_xor(s, o);   // every lane of the group holds the sum
  }
  const double tol = (double)(D + 8) * 2.5e-16 * fmax(d2, s) + 1e-300;
  *margin = fabs(s - d2);
  if (*margin > tol) {
    *escalated = false;
    return s <= d2;
  }
  Big6 acc;
  big_zero(acc);
  for (int d = gl * 4; d < D; d += 4 * G) {
    const uint4 u = *reinterpret_cast<const uint4*>(pa + d);
    const uint4 v = *reinterpret_cast<const uint4*>(pb + d);
    big_add(acc, big_sq_diff(u.x, v.x));
    big_add(acc, big_sq_diff(u.y, v.y));
    big_add(acc, big_sq_diff(u.z, v.z));
    big_add(acc, big_sq_diff(u.w, v.w));
  }
  for (int o = G / 2; o > 0; o >>= 1) {
    Big6 other;
#pragma unroll
    for (int l = 0; l < kExactLimbs; ++l) other.w[l] = (uint64_t)__shfl_xor((unsigned long long)acc.w[l], o);
    big_add(acc, other);
  }
  *escalated = true;
  return big_cmp(acc, thr) <= 0;
}

// ------------------------------------------------------------------ banded candidates
// Algorithm "admit" with a band index (Section 2.2, L1): the codes of a row at
// the band step are cut into bands of r coordinates; a retained row is a
// candidate of an arrival when some band holds equal codes in both.  A 64-bit
// key of (band, codes) finds equal bands through open-addressing indexes (one
// over the retained rows, one over the chunk); the codes themselves are
// compared before a pair counts, so key collisions never make candidates.
//
// One workgroup per arrival collects its distinct candidates in an LDS set,
// then decides them with the merge predicate: retained rows first, where the
// lowest one within delta is the representative (a candidate above the lowest
// hit found so far is skipped); only when none is within are the chunk's
// earlier arrivals decided, for the in-order resolve.  An arrival with more
// candidates than the set holds instead lists each pair once, for its lowest
// equal band, for the separate verification kernel.
constexpr int kAdmitThreads = 256;
constexpr int kSetSlots = 4096;               // LDS candidate set (a power of two)
constexpr int kSetMax = 3072;                 // entries before an arrival takes the pair list
constexpr uint32_t kSetEmpty = 0xffffffffu;
constexpr uint32_t kChunkBit = 0x80000000u;   // set entry of a chunk row (else a store position)
static_assert(kSetMax + kAdmitThreads < kSetSlots, "the set always keeps an empty slot");

struct LshArgs {
  const float* xc;            // chunk rows (float32)
  const float* xs;            // store rows (float32)
  // the screen's operands: fp16 rows x 2^8 and the per-row terms ||x||^2 / 2
  // and error term, of the chunk and of the store
  const _Float16* xc16;
  const float* hnc;
  const float* etc;
  const _Float16* xs16;
  const float* hns;
  const float* ets;
  double half_d2;             // delta^2 / 2
  int nB;
  int D;
  int r, nb;                  // band width, bands per row
  double s, inv_s, eps;       // band step 2 eps, its inverse, eps
  float inv_s32;
  unsigned long long* ckey;   // chunk band keys (nB x nb)
  // the store's index
  const unsigned long long* skey;
  const int32_t* shead;
  const int32_t* snext;
  const unsigned long long* srowkey;
  uint64_t smask;
  // the chunk's own index (rebuilt per chunk)
  unsigned long long* bkey;
  int32_t* bhead;
  int32_t* bnext;
  uint64_t bmask;
  uint64_t bslots;            // slots of the chunk's index
  const StoreMeta* meta;
  int m_exact;                // store size when known, else -1
  // decisions
  double d2;                  // delta^2 in binary64
  Big6 thr;                   // exact right-hand side (exact.h)
  int32_t* firstHit;
  uint64_t* bitmap;
  int W;
  uint32_t* hasEdge;
  // pair list of arrivals whose candidates overflow the set
  int2* pairs;
  uint32_t pair_cap;
  ChunkCounters* cc;
  DevFlags* flags;
};

__device__ __forceinline__ unsigned long long mix64(unsigned long long z) {
  z += 0x9e3779b97f4a7c15ull;
  z = (z ^ (z >> 30)) * 0xbf58476d1ce4e5b9ull;
  z = (z ^ (z >> 27)) * 0x94d049bb133111ebull;
  return z ^ (z >> 31);
}

__device__ __forceinline__ int32_t band_code(const LshArgs& a, float v) {
  return q_round_fast(v, a.inv_s32, a.s, a.inv_s, a.eps);
}

// band b of float32 row q has the codes held in code[] (the arrival's)
__device__ __forceinline__ bool band_matches(const LshArgs& a, const int32_t* code, const float* q, int b) {
  for (int t = b * a.r; t < (b + 1) * a.r; ++t)
    if (band_code(a, q[t]) != code[t]) return false;
  return true;
}

// Slot holding key h in an index (linear probing), or -1 if absent.
__device__ __forceinline__ int64_t find_slot(const unsigned long long* keys, uint64_t mask, unsigned long long h) {
  uint64_t sl = h & mask;
  for (;;) {
    const unsigned long long k = keys[sl];
    if (k == h) return (int64_t)sl;
    if (k == 0ull) return -1;
    sl = (sl + 1) & mask;
  }
}

// Inserts entry e under key h (an index is at most half full, so a free or
// matching slot is always found).
__device__ __forceinline__ void index_insert(unsigned long long* keys, int32_t* head, int32_t* next, uint64_t mask,
                                             unsigned long long h, int32_t e) {
  uint64_t sl = h & mask;
  for (;;) {
    const unsigned long long k = atomicCAS(&keys[sl], 0ull, h);
    if (k == 0ull || k == h) break;
    sl = (sl + 1) & mask;
  }
  next[e] = atomicExch(&head[sl], e);
}

// Band keys of the chunk's rows; the same grid clears the chunk's index.
__global__ __launch_bounds__(256) void k_lsh_keys(LshArgs a) {
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if ((uint64_t)t < a.bslots) {
    a.bkey[t] = 0ull;
    a.bhead[t] = -1;
  }
  if (t >= (int64_t)a.nB * a.nb) return;
  const int i = (int)(t / a.nb), b = (int)(t % a.nb);
  const float* p = a.xc + (int64_t)i * a.D + b * a.r;
  unsigned long long h = mix64((unsigned long long)b + 1ull);
  for (int k = 0; k < a.r; ++k) h = mix64(h ^ (unsigned long long)(uint32_t)band_code(a, p[k]));
  a.ckey[t] = h ? h : 1ull;   // 0 marks an empty slot
}

// The chunk's own index over all its rows (cleared by k_lsh_keys).
__global__ __launch_bounds__(256) void k_lsh_index_chunk(LshArgs a) {
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= (int64_t)a.nB * a.nb) return;
  index_insert(a.bkey, a.bhead, a.bnext, a.bmask, a.ckey[t], (int32_t)t);
}

// Walks the store's and the chunk's lists of arrival i's band b and hands each
// row whose band codes equal the arrival's to f(entry) (entry: store position,
// or kChunkBit | chunk row j for j < i).  Stops early when f returns false.
template <class F>
__device__ __forceinline__ void band_rows(const LshArgs& a, int i, int b, int m, const int32_t* code, F&& f) {
  const unsigned long long h = a.ckey[(int64_t)i * a.nb + b];
  if (m > 0) {
    const int64_t sl = find_slot(a.skey, a.smask, h);
    for (int32_t e = sl >= 0 ? a.shead[sl] : -1; e >= 0; e = a.snext[e]) {
      const int pos = e / a.nb;
      if (e - pos * a.nb != b || pos >= m) continue;
      if (band_matches(a, code, a.xs + (int64_t)pos * a.D, b) && !f((uint32_t)pos)) return;
    }
  }
  const int64_t sl = find_slot(a.bkey, a.bmask, h);
  for (int32_t e = sl >= 0 ? a.bhead[sl] : -1; e >= 0; e = a.bnext[e]) {
    const int j = e / a.nb;
    if (e - j * a.nb != b || j >= i) continue;
    if (band_matches(a, code, a.xc + (int64_t)j * a.D, b) && !f(kChunkBit | (uint32_t)j)) return;
  }
}

__device__ __forceinline__ uint32_t set_hash(uint32_t v) { return (v * 0x9e3779b1u) >> (32 - 12); }

// Decision of one candidate pair by a group of G lanes: the fp16 screen's dot
// (exact products, float32 sums in any order) against the same error bound as
// the MFMA screen, with the binary64 and exact test (pair_within) only for a
// pair the bound leaves ambiguous.  a = the arrival (chunk row i), b = the
// candidate.  *tested tells whether pair_within ran.
template <int G>
__device__ bool screened_within(const LshArgs& a, int i, const float* pb32, const _Float16* pb16, float hn_b,
                                float et_b, bool* escalated, double* margin, bool* tested) {
  const int gl = (int)threadIdx.x & (G - 1);
  const _Float16* pa16 = a.xc16 + (int64_t)i * a.D;
  float acc = 0.0f;
  for (int d = gl * 8; d < a.D; d += 8 * G) {
    const half8 u = *reinterpret_cast<const half8*>(pa16 + d);
    const half8 v = *reinterpret_cast<const half8*>(pb16 + d);
#pragma unroll
    for (int e = 0; e < 8; ++e) acc = fmaf((float)u[e], (float)v[e], acc);
  }
  for (int o = G / 2; o > 0; o >>= 1) acc += __shfl_xor(acc, o);
  const float v = acc * kInvScale2 - hn_b;
  const double base = (double)a.hnc[i] - a.half_d2;
  const double e = (double)a.etc[i] + (double)et_b;
  *tested = false;
  if (v >= round_up_f32(base + e)) return true;
  if (v < round_down_f32(base - e)) return false;
  *tested = true;
  return pair_within<G>(a.xc + (int64_t)i * a.D, pb32, a.D, a.d2, a.thr, escalated, margin);
}
static_assert(kSetSlots == 1 << 12, "set_hash yields 12 bits");

__global__ __launch_bounds__(kAdmitThreads) void k_lsh_admit(LshArgs a) {
  extern __shared__ int32_t s_code[];   // the arrival's band codes (D)
  __shared__ uint32_t set[kSetSlots];
  __shared__ uint32_t list[kSetMax + kAdmitThreads];
  __shared__ uint32_t n_set, n_store, n_chunk;
  __shared__ int32_t hit, skip;
  const int i = (int)blockIdx.x;
  const int tid = (int)threadIdx.x;
  // one reading of the status words for the whole workgroup (another
  // workgroup's pair-list overflow may set them meanwhile)
  if (tid == 0) skip = skip_all(a.flags) ? 1 : 0;
  __syncthreads();
  if (skip) return;
  const int m = a.m_exact >= 0 ? a.m_exact : a.meta->m;
  const float* p = a.xc + (int64_t)i * a.D;
  for (int d = tid; d < a.D; d += kAdmitThreads) s_code[d] = band_code(a, p[d]);
  for (int k = tid; k < kSetSlots; k += kAdmitThreads) set[k] = kSetEmpty;
  if (tid == 0) {
    n_set = 0u;
    n_store = 0u;
    n_chunk = 0u;
    hit = kNone;
  }
  __syncthreads();

  // 1. distinct candidates into the set (at most kSetMax + one per thread:
  //    an insert starts only while the count is below kSetMax)
  volatile uint32_t* vn = &n_set;
  for (int b = tid; b < a.nb && *vn < (uint32_t)kSetMax; b += kAdmitThreads) {
    band_rows(a, i, b, m, s_code, [&](uint32_t v) {
      if (*vn >= (uint32_t)kSetMax) return false;
      uint32_t sl = set_hash(v);
      for (;;) {
        const uint32_t old = atomicCAS(&set[sl], kSetEmpty, v);
        if (old == kSetEmpty) {
          atomicAdd(&n_set, 1u);
          break;
        }
        if (old == v) break;
        sl = (sl + 1) & (kSetSlots - 1);
      }
      return true;
    });
  }
  __syncthreads();

  if (n_set >= (uint32_t)kSetMax) {
    // 1'. too many candidates: each pair once, for its lowest equal band, to
    //     the pair list (decided by k_verify)
    for (int b = tid; b < a.nb; b += kAdmitThreads) {
      band_rows(a, i, b, m, s_code, [&](uint32_t v) {
        const bool chunk = (v & kChunkBit) != 0u;
        const int y = (int)(v & ~kChunkBit);
        const float* q = (chunk ? a.xc : a.xs) + (int64_t)y * a.D;
        for (int b2 = 0; b2 < b; ++b2)
          if (band_matches(a, s_code, q, b2)) return true;   // listed by band b2
        const uint32_t idx = atomicAdd(&a.cc->npairs, 1u);
        atomicAdd(&a.flags->n_pairs, 1u);
        atomicAdd(&a.flags->n_cand, 1ull);
        if (idx < a.pair_cap) {
          a.pairs[idx] = make_int2(i | ((chunk ? 1 : 0) << 31), y);
        } else {
          atomicOr(&a.flags->pair_overflow, 1u);
          atomicMax(&a.flags->pairs_needed, idx + 1u);
        }
        return true;
      });
    }
    return;
  }
  if (tid == 0) atomicAdd(&a.flags->n_cand, (unsigned long long)n_set);

  // 2. the set as two lists: store positions from the front, chunk rows from the back
  for (int k = tid; k < kSetSlots; k += kAdmitThreads) {
    const uint32_t v = set[k];
    if (v == kSetEmpty) continue;
    if (v & kChunkBit)
      list[kSetMax + kAdmitThreads - 1 - atomicAdd(&n_chunk, 1u)] = v & ~kChunkBit;
    else
      list[atomicAdd(&n_store, 1u)] = v;
  }
  __syncthreads();
  const int ns = (int)n_store, nc = (int)n_chunk;

  // 3. retained candidates, by groups of kGroup lanes (a wave's groups take
  //    consecutive entries): the lowest within delta is the representative,
  //    so a candidate above the lowest hit so far is skipped.  (Each reading
  //    of hit is the same for every lane of a group: they read it in one
  //    instruction.)
  constexpr int kGroup = 16, kGroups = kAdmitThreads / kGroup;
  const int grp = tid / kGroup;
  const bool glead = (tid & (kGroup - 1)) == 0;
  volatile int32_t* vh = &hit;
  uint32_t esc = 0u;
  double mmin = 1e308;
  for (int k = grp; k < ns; k += kGroups) {
    const int y = (int)list[k];
    if (y >= *vh) continue;
    bool e = false, tested = false;
    double mg = 1e308;
    const bool in = screened_within<kGroup>(a, i, a.xs + (int64_t)y * a.D, a.xs16 + (int64_t)y * a.D, a.hns[y],
                                            a.ets[y], &e, &mg, &tested);
    esc += e ? 1u : 0u;
    if (tested) mmin = fmin(mmin, mg);
    if (in && glead) atomicMin(&hit, y);
  }
  __syncthreads();
  if (hit != kNone) {
    if (tid == 0) a.firstHit[i] = hit;
  } else {
    // 4. no retained row within delta: the chunk's earlier arrivals, for the resolve
    const uint32_t* cl = list + kSetMax + kAdmitThreads - nc;
    for (int k = grp; k < nc; k += kGroups) {
      const int j = (int)cl[k];
      bool e = false, tested = false;
      double mg = 1e308;
      const bool in = screened_within<kGroup>(a, i, a.xc + (int64_t)j * a.D, a.xc16 + (int64_t)j * a.D, a.hnc[j],
                                              a.etc[j], &e, &mg, &tested);
      esc += e ? 1u : 0u;
      if (tested) mmin = fmin(mmin, mg);
      if (in && glead) {
        atomicOr(reinterpret_cast<unsigned long long*>(&a.bitmap[(int64_t)i * a.W + (j >> 6)]), 1ull << (j & 63));
        a.hasEdge[i] = 1u;
      }
    }
  }
  if (glead && esc) {
    atomicAdd(&a.cc->n_escalate, esc);
    atomicAdd(&a.flags->n_escalate, esc);
  }
  if (glead) note_margin(a.flags, mmin);
}

// Kept rows of the chunk join the store's index under their store positions.
__global__ __launch_bounds__(256) void k_lsh_insert(LshArgs a, const int32_t* __restrict__ pos,
                                                    unsigned long long* skey, int32_t* shead, int32_t* snext,
                                                    unsigned long long* srowkey) {
  if (skip_all(a.flags)) return;
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= (int64_t)a.nB * a.nb) return;
  const int i = (int)(t / a.nb), b = (int)(t % a.nb);
  const int p = pos[i];
  if (p < 0) return;
  const unsigned long long h = a.ckey[t];
  const int32_t e = p * a.nb + b;
  srowkey[e] = h;
  index_insert(skey, shead, snext, a.smask, h, e);
}

// Empties the store's index, then (second kernel) puts back the entries of the
// first rows of the store from their recorded band keys.
__global__ __launch_bounds__(256) void k_lsh_clear_index(unsigned long long* key, int32_t* head, uint64_t slots) {
  const uint64_t stride = (uint64_t)gridDim.x * blockDim.x;
  for (uint64_t t = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; t < slots; t += stride) {
    key[t] = 0ull;
    head[t] = -1;
  }
}

__global__ __launch_bounds__(256) void k_lsh_reinsert(unsigned long long* key, int32_t* head, int32_t* next,
                                                      const unsigned long long* rowkey, uint64_t mask,
                                                      int64_t n_entries) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < n_entries; e += stride)
    index_insert(key, head, next, mask, rowkey[e], (int32_t)e);
}

// ------------------------------------------------------------------ verify
struct VerifyArgs {
  const int2* pairs;
  uint32_t* status;       // 0 out, 1 in, 3 skipped (above the row's definite hit)
  const ChunkCounters* cc;
  uint32_t pair_cap;
  const float* xc;        // chunk rows, float32 (caller memory)
  const float* xs;        // store rows, float32
  int D;
  double d2;              // delta^2 in binary64
  Big6 thr;               // floor((2 - 2 tau) * 2^298), the exact right-hand side
  int32_t* firstHit;
  uint64_t* bitmap;
  int W;
  uint32_t* hasEdge;
  DevFlags* flags;
  ChunkCounters* ccw;
};

// One wave per listed pair, decided by the merge predicate (pair_within).
__global__ __launch_bounds__(256) void k_verify(VerifyArgs a) {
  // the pair count is loaded with the status words (both decide the exit), so
  // the two do not take dependent round trips
  const uint32_t np = a.cc->npairs;
  if ((np == 0u) | skip_all(a.flags)) return;
  const uint32_t n = min(np, a.pair_cap);
  const int lane = threadIdx.x & 63;
  const uint32_t wid = (blockIdx.x * blockDim.x + threadIdx.x) >> 6;
  const uint32_t nw = (gridDim.x * blockDim.x) >> 6;
  double mmin = 1e308;
  for (uint32_t p = wid; p < n; p += nw) {
    const int2 e = a.pairs[p];
    const int kind = (int)((uint32_t)e.x >> 31);
    const int i = e.x & 0x7fffffff;
    const int y = e.y;
    if (kind == 0 && y >= *reinterpret_cast<volatile const int32_t*>(&a.firstHit[i])) {
      if (lane == 0) a.status[p] = 3u;
      continue;
    }
    const float* pa = a.xc + (int64_t)i * a.D;
    const float* pb = (kind == 0 ? a.xs : a.xc) + (int64_t)y * a.D;
    bool escalated = false;
    double mg;
    const bool in = pair_within<64>(pa, pb, a.D, a.d2, a.thr, &escalated, &mg);
    mmin = fmin(mmin, mg);
    if (escalated && lane == 0) {
      atomicAdd(&a.ccw->n_escalate, 1u);
      atomicAdd(&a.flags->n_escalate, 1u);
    }
    if (lane != 0) continue;
    if (in) {
      if (kind == 0) {
        atomicMin(&a.firstHit[i], y);
      } else {
        atomicOr(reinterpret_cast<unsigned long long*>(&a.bitmap[(int64_t)i * a.W + (y >> 6)]), 1ull << (y & 63));
        a.hasEdge[i] = 1u;
      }
    }
    a.status[p] = in ? 1u : 0u;
  }
  if (lane == 0) note_margin(a.flags, mmin);
}

// ------------------------------------------------------------------ resolve
struct ResolveArgs {
  int nB;
  int W;
  const int32_t* firstHit;
  const uint32_t* hasEdge;
  const uint64_t* bitmap;
  const int64_t* store_ids;
  StoreMeta* meta;
  int64_t c0;               // offset of the chunk in the call (global id = meta->n_seen + c0 + row)
  int64_t* rep;             // caller output for the chunk (global ids, -1 kept)
  int32_t* pos;             // store position of kept rows, -1 if dropped
  int32_t* rep_row;         // >= 0 store row, <= -2 chunk row (-(j+2)), -1 kept
  uint64_t* kept_words;     // kept mask of the chunk (64 words)
  DevFlags* flags;
};

constexpr int kResolveThreads = 1024;
static_assert(kChunk % kResolveThreads == 0, "whole rows per thread");
constexpr int kEdgeCap = 20480;    // in-chunk candidate entries held in LDS (list form)
constexpr int kBitsCap = 8704;     // candidate bitmap words of active rows held in LDS (bitmap form)

// LDS of the in-chunk resolve.  rrow: the decision of each row as rep_row
// encodes it; posv: the store position of each kept row (-1 if dropped).
// The active rows' in-chunk candidates are held in one of two forms: their
// bitmap words as loaded (bitmap form, when they fit), or ascending lists.
struct ResolveLds {
  uint8_t st[kChunk];        // 0 undecided, 1 kept, 2 dropped
  union {
    struct {
      uint16_t edges[kEdgeCap];
      uint32_t eoff[kChunk];
      uint16_t elen[kChunk];
      uint16_t ecur[kChunk];
    } ls;                    // list form: active row i's candidates at edges[eoff[i], eoff[i] + elen[i])
    struct {
      unsigned long long bits[kBitsCap];
      uint8_t first[kChunk];
    } bm;                    // bitmap form: active row k's words at bits[k W, k W + W); first word to look at
  };
  unsigned long long dropped[kChunk / 64];   // rows known to be dropped, one bit each
  uint16_t active[kChunk];
  int32_t rrow[kChunk];
  int32_t posv[kChunk];
  uint32_t n_active, n_edges, total;
  uint32_t pend[3];          // round r sets pend[r % 3] while a row waits
  int wsum[kResolveThreads / 64];
};

// Fallback when the candidate lists do not fit in LDS: one wave walks the
// undecided rows in arrival order; lane L keeps bits [64L, 64L + 64) of the
// kept mask in a register, and a row takes the lowest kept candidate of its
// bitmap row.
__device__ void resolve_sequential(const ResolveArgs& a, ResolveLds& L, int n) {
  volatile uint8_t* st = L.st;
  const int lane = threadIdx.x & 63;
  const int nblk = (n + 63) >> 6;
  uint64_t kept = 0ull;
  for (int w = 0; w < nblk; ++w) {
    const int r = w * 64 + lane;
    const uint64_t b = __ballot(r < n && st[r] == 1);
    if (lane == w) kept = b;
  }
  for (int blk = 0; blk < nblk; ++blk) {
    const int r = blk * 64 + lane;
    uint64_t act = __ballot(r < n && st[r] == 0);
    while (act) {
      const int b = __builtin_ctzll(act);
      act &= act - 1ull;
      const int i = blk * 64 + b;
      const int nw = (i + 63) >> 6;   // words holding bits j < i
      const uint64_t e = (lane < nw) ? a.bitmap[(int64_t)i * a.W + lane] : 0ull;
      const uint64_t u = e & kept;
      const uint64_t any = __ballot(u != 0ull);
      if (any) {
        const int F = __builtin_ctzll(any);
        const uint64_t uf = __shfl(u, F);
        const int j = F * 64 + __builtin_ctzll(uf);
        if (lane == 0) {
          st[i] = 2;
          L.rrow[i] = -(j + 2);
        }
      } else {
        if (lane == blk) kept |= 1ull << b;
        if (lane == 0) {
          st[i] = 1;
          L.rrow[i] = -1;
        }
      }
    }
  }
}

// In-order resolve of the first n rows of a chunk by one workgroup of T
// threads, into L (the decision of a row depends only on rows before it).
//  A. Rows with a store hit are dropped (their representative is the lowest
//     store row); rows with no in-chunk edge are kept.  Neither depends on any
//     other row of the chunk.  The rest are "active".
//  B. Each active row's in-chunk candidates (bits j < i of its bitmap row) are
//     copied into LDS: the bitmap words themselves when all active rows' words
//     fit (bitmap form), else as ascending lists.  (Expanding dense words into
//     lists bit by bit serialised the lanes holding them: clustered streams
//     put dozens of candidates in one word.)
//  C. Rounds: an undecided active row looks for its lowest candidate that is
//     not dropped (the bitmap words masked by the dropped rows, or the list
//     walked past them); that candidate decides it (kept -> the row is dropped
//     with that representative), or makes it wait if still undecided; a row
//     with no such candidate is kept.  A decision is taken only once every
//     earlier candidate is decided, so it is the one the sequential walk
//     takes, and the lowest undecided row can always decide, so the rounds
//     end.
//  D. Kept rows get consecutive store positions from m0, in arrival order;
//     L.total is the number kept among the n rows.
// The first phase's loads (hits and edge flags) are issued by the caller
// with the others that open its kernel; hit_r / edge_r hold rows
// tid + u T.  Returns with every thread past a barrier.
template <int T>
__device__ void resolve_core(const ResolveArgs& a, ResolveLds& L, int n, int m0, const int32_t (&hit_r)[kChunk / T],
                             const uint32_t (&edge_r)[kChunk / T]) {
  volatile uint8_t* st = L.st;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  if (tid == 0) {
    L.n_active = 0u;
    L.n_edges = 0u;
    L.pend[0] = 0u;   // the first round's flag (later ones are cleared a round ahead)
  }
  __syncthreads();
#pragma unroll
  for (int u = 0; u < kChunk / T; ++u) {
    const int r = tid + u * T;
    if (r >= n) break;
    const int32_t hit = hit_r[u];
    if (hit != kNone) {
      st[r] = 2;
      L.rrow[r] = hit;
    } else if (edge_r[u] == 0u) {
      st[r] = 1;
      L.rrow[r] = -1;
    } else {
      st[r] = 0;
      L.active[atomicAdd(&L.n_active, 1u)] = (uint16_t)r;
    }
  }
  // the rows dropped so far (store hits), one word per 64 rows
#pragma unroll
  for (int u = 0; u < kChunk / T; ++u) {
    const int r = tid + u * T;   // a wave's lanes hold 64 consecutive rows
    const uint64_t b = __ballot(r < n && hit_r[u] != kNone);
    if (lane == 0) L.dropped[(u * T) / 64 + wave] = b;
  }
  __syncthreads();
  const int na = (int)L.n_active;
  // B. A row's bitmap words (bits j < i) are read by G lanes, G = W rounded up
  //    to a power of two, so a wave covers 64 / G rows at once; four such sets
  //    are loaded before any is used, which keeps several loads in flight.
  const int G = a.W <= 1 ? 1 : 1 << (32 - __clz(a.W - 1));
  const int sub = lane / G, wl = lane % G;
  const int rstep = (T / 64) * (64 / G);
  if ((int64_t)na * a.W <= kBitsCap) {
    volatile unsigned long long* dropped = L.dropped;
    for (int kb = wave * (64 / G); kb < na; kb += 4 * rstep) {
      uint64_t e[4];
      int ir[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int k = kb + u * rstep + sub;
        ir[u] = k < na ? (int)L.active[k] : -1;
        const int nw = (ir[u] + 63) >> 6;
        e[u] = (ir[u] >= 0 && wl < nw) ? a.bitmap[(int64_t)ir[u] * a.W + wl] : 0ull;
      }
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int k = kb + u * rstep + sub;
        if (ir[u] >= 0 && wl < a.W) L.bm.bits[k * a.W + wl] = e[u];
        const uint64_t nz = __ballot(e[u] != 0ull);
        if (wl == 0 && ir[u] >= 0) {
          const uint64_t gm = (G == 64) ? nz : (nz >> (sub * G)) & ((1ull << G) - 1ull);
          L.bm.first[k] = gm ? (uint8_t)__builtin_ctzll(gm) : (uint8_t)a.W;
        }
      }
    }
    __syncthreads();
    // one barrier per round: round r raises pend[r % 3] and clears pend[(r + 1)
    // % 3], which every thread last read before the previous barrier
    if (na <= T) {
      // one active row per thread: its index, whether it is still open, its
      // current word index and that word stay in registers across rounds
      // (only the row's own thread changes them), so a round reads only the
      // dropped words and the candidates' states
      const bool mine = tid < na;
      const int i = mine ? (int)L.active[tid] : 0;
      const int nw = (i + 63) >> 6;
      int w = mine ? (int)L.bm.first[tid] : 0;
      uint64_t cur = (mine && w < nw) ? L.bm.bits[tid * a.W + w] : 0ull;
      bool open = mine;
      for (int r = 0;; ++r) {
        if (tid == 0) L.pend[(r + 1) % 3] = 0u;
        if (open) {
          int dec = 0;   // 0 keep, 1 drop, -1 wait
          int j = -1;
          while (w < nw) {
            uint64_t x = cur & ~dropped[w];
            while (x) {
              const int c = w * 64 + __builtin_ctzll(x);
              const uint8_t sc = st[c];
              if (sc == 2) {   // dropped since the word was read
                x &= x - 1ull;
                continue;
              }
              dec = (sc == 1) ? 1 : -1;
              j = c;
              break;
            }
            if (j >= 0) break;
            ++w;   // the word holds only dropped candidates
            cur = w < nw ? L.bm.bits[tid * a.W + w] : 0ull;
          }
          if (dec == 1) {
            st[i] = 2;
            L.rrow[i] = -(j + 2);
            atomicOr(&L.dropped[i >> 6], 1ull << (i & 63));
            open = false;
          } else if (dec == 0) {
            st[i] = 1;
            L.rrow[i] = -1;
            open = false;
          } else {
            L.pend[r % 3] = 1u;
          }
        }
        __syncthreads();
        if (L.pend[r % 3] == 0u) break;
      }
    } else for (int r = 0;; ++r) {
      if (tid == 0) L.pend[(r + 1) % 3] = 0u;
      for (int k = tid; k < na; k += T) {
        const int i = L.active[k];
        if (st[i] != 0) continue;
        const int nw = (i + 63) >> 6;
        int dec = 0;   // 0 keep, 1 drop, -1 wait
        int j = -1;
        int w = L.bm.first[k];
        for (; w < nw; ++w) {
          uint64_t x = L.bm.bits[k * a.W + w] & ~dropped[w];
          while (x) {
            const int c = w * 64 + __builtin_ctzll(x);
            const uint8_t sc = st[c];
            if (sc == 2) {   // dropped since the word was read
              x &= x - 1ull;
              continue;
            }
            dec = (sc == 1) ? 1 : -1;
            j = c;
            break;
          }
          if (j >= 0) break;
        }
        if (dec == 1) {
          st[i] = 2;
          L.rrow[i] = -(j + 2);
          atomicOr(&L.dropped[i >> 6], 1ull << (i & 63));
        } else if (dec == 0) {
          st[i] = 1;
          L.rrow[i] = -1;
        } else {
          L.bm.first[k] = (uint8_t)w;   // the words before it hold only dropped candidates
          L.pend[r % 3] = 1u;
        }
      }
      __syncthreads();
      if (L.pend[r % 3] == 0u) break;
    }
  } else {
    for (int kb = wave * (64 / G); kb < na; kb += 4 * rstep) {
      uint64_t e[4];
      int ir[4];
  #pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int k = kb + u * rstep + sub;
        ir[u] = k < na ? (int)L.active[k] : -1;
        const int nw = (ir[u] + 63) >> 6;
        e[u] = (ir[u] >= 0 && wl < nw) ? a.bitmap[(int64_t)ir[u] * a.W + wl] : 0ull;
      }
  #pragma unroll
      for (int u = 0; u < 4; ++u) {
        uint64_t eu = e[u];
        const int c = __popcll(eu);
        int incl = c;
        for (int o = 1; o < G; o <<= 1) {
          const int t = __shfl_up(incl, o, G);
          if (wl >= o) incl += t;
        }
        const int tot = __shfl(incl, sub * G + G - 1);
        uint32_t base = 0u;
        if (wl == 0 && ir[u] >= 0) base = atomicAdd(&L.n_edges, (uint32_t)tot);
        base = __shfl(base, sub * G);
        if (ir[u] >= 0) {
          if (base + (uint32_t)tot <= (uint32_t)kEdgeCap) {
            uint32_t p = base + (uint32_t)(incl - c);
            while (eu) {
              L.ls.edges[p++] = (uint16_t)(wl * 64 + __builtin_ctzll(eu));
              eu &= eu - 1ull;
            }
          }
          if (wl == 0) {
            L.ls.eoff[ir[u]] = base;
            L.ls.elen[ir[u]] = (uint16_t)tot;
            L.ls.ecur[ir[u]] = 0;
          }
        }
      }
    }
    __syncthreads();
    if (L.n_edges > (uint32_t)kEdgeCap) {
      if (wave == 0) resolve_sequential(a, L, n);
    } else {
      for (int r = 0;; ++r) {   // one barrier per round, as in the bitmap form
        if (tid == 0) L.pend[(r + 1) % 3] = 0u;
        for (int k = tid; k < na; k += T) {
          const int i = L.active[k];
          if (st[i] != 0) continue;
          const int len = L.ls.elen[i];
          const uint32_t b0 = L.ls.eoff[i];
          int p = L.ls.ecur[i];
          int dec = -1;   // -1 wait, 0 keep, 1 drop
          int j = -1;
          for (; p < len; ++p) {
            j = L.ls.edges[b0 + p];
            const uint8_t s = st[j];
            if (s == 2) continue;
            dec = (s == 1) ? 1 : -1;
            break;
          }
          if (p == len) dec = 0;
          L.ls.ecur[i] = (uint16_t)p;
          if (dec == 1) {
            st[i] = 2;
            L.rrow[i] = -(j + 2);
          } else if (dec == 0) {
            st[i] = 1;
            L.rrow[i] = -1;
          } else {
            L.pend[r % 3] = 1u;
          }
        }
        __syncthreads();
        if (L.pend[r % 3] == 0u) break;
      }
    }
  }
  __syncthreads();
  // D. store positions: exclusive scan of kept flags, whole rows per thread
  // (one row per thread: the wave's ballot gives the counts)
  if (n <= T) {
    const bool kp = tid < n && st[tid] == 1;
    const uint64_t bal = __ballot(kp);
    if (lane == 0) L.wsum[wave] = __popcll(bal);
    __syncthreads();
    int base = 0, total = 0;
#pragma unroll
    for (int w = 0; w < T / 64; ++w) {
      const int v = L.wsum[w];
      base += w < wave ? v : 0;
      total += v;
    }
    if (tid == 0) L.total = (uint32_t)total;
    if (tid < n) L.posv[tid] = kp ? m0 + base + __popcll(bal & ((1ull << lane) - 1ull)) : -1;
    __syncthreads();
    return;
  }
  const int per = (n + T - 1) / T;
  const int r0 = tid * per, r1 = min(n, r0 + per);
  int c = 0;
  for (int r = r0; r < r1; ++r) c += (st[r] == 1) ? 1 : 0;
  int x = c;
  for (int o = 1; o < 64; o <<= 1) {
    const int t = __shfl_up(x, o);
    if (lane >= o) x += t;
  }
  if (lane == 63) L.wsum[wave] = x;
  __syncthreads();
  if (tid == 0) {
    int acc = 0;
    for (int w = 0; w < T / 64; ++w) {
      const int t = L.wsum[w];
      L.wsum[w] = acc;
      acc += t;
    }
    L.total = (uint32_t)acc;
  }
  __syncthreads();
  int pos = m0 + L.wsum[wave] + x - c;
  for (int r = r0; r < r1; ++r) L.posv[r] = (st[r] == 1) ? pos++ : -1;
  __syncthreads();
}

// The resolve as a kernel of its own (one workgroup): decisions to rep, pos,
// rep_row and the kept mask in global memory, the store size advanced.
__global__ __launch_bounds__(kResolveThreads) void k_resolve(ResolveArgs a) {
  __shared__ ResolveLds L;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  // the first phase's loads (hits and edge flags of this thread's rows, the
  // status words, the store's counts) are all issued before any is used
  constexpr int kRowsPerThread = kChunk / kResolveThreads;
  int32_t hit_r[kRowsPerThread];
  uint32_t edge_r[kRowsPerThread];
#pragma unroll
  for (int u = 0; u < kRowsPerThread; ++u) {
    const int r = min(tid + u * kResolveThreads, a.nB - 1);
    hit_r[u] = a.firstHit[r];
    edge_r[u] = a.hasEdge[r];
  }
  const bool skip = skip_all(a.flags);
  const int m0 = a.meta->m;
  const int64_t gbase = a.meta->n_seen + a.c0;   // updated only at the end of a call
  if (skip) return;   // (the status words do not change while this single workgroup runs)
  resolve_core<kResolveThreads>(a, L, a.nB, m0, hit_r, edge_r);
  for (int r = tid; r < a.nB; r += kResolveThreads) {
    const int32_t rr = L.rrow[r];
    a.rep[r] = rr >= 0 ? a.store_ids[rr] : (rr == -1 ? -1 : gbase + (-rr - 2));
    a.rep_row[r] = rr;
    a.pos[r] = L.posv[r];
  }
  for (int w = wave; w < 64; w += kResolveThreads / 64) {
    const int r = w * 64 + lane;
    const uint64_t b = __ballot(r < a.nB && L.st[r] == 1);
    if (lane == 0) a.kept_words[w] = b;
  }
  if (tid == 0) {
    a.meta->m = m0 + (int)L.total;
    atomicAdd(&a.flags->n_kept, L.total);
  }
}

// ------------------------------------------------------------------ append
struct AppendArgs {
  const float* xc;
  const _Float16* x16c;
  const float* hnc;
  const float* etc;
  const int32_t* pos;
  const int32_t* rep_row;
  int64_t c0;               // offset of the chunk in the call
  int D;
  float* xs;
  _Float16* x16s;
  float* hns;
  float* ets;
  int64_t* ids;
  DevFlags* flags;
  ChunkCounters* cc;
  StoreMeta* meta;
  int64_t n_call;           // rows of the whole call
  int last_chunk;           // the call's last chunk: fold the call into the store's bookkeeping
  int async_call;           // no host check follows: a full pair list is reported as an error
  DevFlags* flags_out;      // host-mapped copy of the status words, or NULL
};

constexpr int kAppendRows = 4;  // rows per workgroup of k_append (one wave each)
constexpr int kAppendVec = 4;   // float4 of a row per lane held in registers (D <= 1,024)

// Loads row r of the chunk into registers (D <= 1,024: the whole row, zeros
// past it, through a buffer resource; otherwise nothing, and append_row reads
// the row itself).
__device__ __forceinline__ void append_load(const AppendArgs& a, int r, float4 (&v)[kAppendVec]) {
  const bool vec = a.D <= 256 * kAppendVec;
  const int lane = threadIdx.x & 63;
  const __amdgpu_buffer_rsrc_t rs = f32_rsrc(a.xc + (int64_t)r * a.D, vec ? a.D : 0);
#pragma unroll
  for (int u = 0; u < kAppendVec; ++u)
    v[u] = __builtin_bit_cast(float4, __builtin_amdgcn_raw_buffer_load_b128(rs, (uint32_t)(u * 256 + lane * 4) * 4u, 0, 0));
}

// One wave's work for chunk row r (its data in v, from append_load): a kept
// row (store position p >= 0) is copied into the store, with its terms and
// global id, and raises amax / hmax (|x| and ||x||^2 / 2 as float bits); for a
// dropped row ||x - x_rep||^2 (rr: the representative as rep_row encodes it)
// is summed in binary64 in a fixed order into dmax (every lane).
__device__ __forceinline__ void append_row(const AppendArgs& a, int r, int p, int rr, float hn, float et,
                                           int64_t gbase, const float4 (&v)[kAppendVec], double& dmax,
                                           uint32_t& amax, uint32_t& hmax) {
  const int lane = threadIdx.x & 63;
  const bool vec = a.D <= 256 * kAppendVec;
  const float* src = a.xc + (int64_t)r * a.D;
  if (p >= 0) {
    float* dst = a.xs + (int64_t)p * a.D;
    _Float16* d16 = a.x16s + (int64_t)p * a.D;
    hmax = max(hmax, __float_as_uint(hn));
    auto absbits = [](const float4& x) {
      return max(max(__float_as_uint(x.x) & 0x7fffffffu, __float_as_uint(x.y) & 0x7fffffffu),
                 max(__float_as_uint(x.z) & 0x7fffffffu, __float_as_uint(x.w) & 0x7fffffffu));
    };
    if (vec) {
      // the fp16 operand is formed as the prep forms it, fl16(2^8 x)
#pragma unroll
      for (int u = 0; u < kAppendVec; ++u) {
        const int d = u * 256 + lane * 4;
        if (d >= a.D) break;
        amax = max(amax, absbits(v[u]));
        *reinterpret_cast<float4*>(dst + d) = v[u];
        const _Float16 h[4] = {(_Float16)(v[u].x * kScale), (_Float16)(v[u].y * kScale),
                               (_Float16)(v[u].z * kScale), (_Float16)(v[u].w * kScale)};
        uint2 packed;
        __builtin_memcpy(&packed, h, 8);
        *reinterpret_cast<uint2*>(d16 + d) = packed;
      }
    } else {
      for (int d = lane * 4; d < a.D; d += 256) {
        const float4 x = *reinterpret_cast<const float4*>(src + d);
        amax = max(amax, absbits(x));
        *reinterpret_cast<float4*>(dst + d) = x;
      }
      const _Float16* s16 = a.x16c + (int64_t)r * a.D;
      for (int d = lane * 8; d < a.D; d += 512)
        *reinterpret_cast<uint4*>(d16 + d) = *reinterpret_cast<const uint4*>(s16 + d);
    }
    if (lane == 0) {
      a.hns[p] = hn;
      a.ets[p] = et;
      a.ids[p] = gbase + r;
    }
  } else {
    const float* b = (rr >= 0) ? a.xs + (int64_t)rr * a.D : a.xc + (int64_t)(-rr - 2) * a.D;
    double s = 0.0;
    auto acc4 = [&](const float4& x, const float4& y) {
      const double t0 = (double)x.x - (double)y.x, t1 = (double)x.y - (double)y.y;
      const double t2 = (double)x.z - (double)y.z, t3 = (double)x.w - (double)y.w;
      s = fma(t0, t0, s);
      s = fma(t1, t1, s);
      s = fma(t2, t2, s);
      s = fma(t3, t3, s);
    };
    if (vec) {
      const __amdgpu_buffer_rsrc_t rb = f32_rsrc(b, a.D);
#pragma unroll
      for (int u = 0; u < kAppendVec; ++u)
        acc4(v[u], __builtin_bit_cast(float4, __builtin_amdgcn_raw_buffer_load_b128(
                                                  rb, (uint32_t)(u * 256 + lane * 4) * 4u, 0, 0)));
    } else {
      for (int d = lane * 4; d < a.D; d += 256)
        acc4(*reinterpret_cast<const float4*>(src + d), *reinterpret_cast<const float4*>(b + d));
    }
    dmax = fmax(dmax, wave_sum_f64(s));
  }
}

// A workgroup's maxima go to the status words and the store's bookkeeping
// (one atomic each, only when they rise); am0 / hm0: the store's maxima as the
// workgroup read them at its start.  parts: 3 x kWaves words of LDS.
template <int kWaves>
__device__ __forceinline__ void append_maxima(const AppendArgs& a, double dmax, uint32_t amax, uint32_t hmax,
                                              uint32_t am0, uint32_t hm0, double* part, uint32_t* apart,
                                              uint32_t* hpart) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  amax = wave_max_u32(amax);
  if (lane == 0) {
    part[wave] = dmax;
    apart[wave] = amax;
    hpart[wave] = hmax;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    double m = part[0];
    uint32_t am = apart[0], hm = hpart[0];
    for (int w = 1; w < kWaves; ++w) {
      m = fmax(m, part[w]);
      am = max(am, apart[w]);
      hm = max(hm, hpart[w]);
    }
    // A call that waits gathers its delta_hat in the status words, read back
    // by the host; a call that does not goes straight to the store's
    // bookkeeping (rows are appended only by calls that go through, and skip
    // is uniform over the call, so an invalid call leaves it as it was).
    if (m > 0.0)
      atomicMax(a.async_call ? &a.meta->dhat2_bits : reinterpret_cast<unsigned long long*>(&a.flags->dhat2_bits),
                (unsigned long long)__double_as_longlong(m));
    if (am > am0) atomicMax(&a.meta->absmax_bits, am);
    if (hm > hm0) atomicMax(&a.meta->hnmax_bits, hm);
    // When the last workgroup reads the status words' maximum (a call that
    // waits), this workgroup is counted only once its maxima have been
    // performed: the wait covers the atomics issued above.  Device-scope
    // atomics are performed where every XCD sees them, so the last workgroup,
    // which reads the status words with device-scope atomic loads, needs no
    // cache write-back or invalidation (fences here cost 1.7 us per call).
    // Nothing of this launch reads the bookkeeping's maxima, so a call that
    // does not wait does not wait here (its row stores are not waited for).
    if (!a.async_call) __builtin_amdgcn_s_waitcnt(0);
  }
}

// The last workgroup to finish runs `last_work(kept)` (thread 0; kept = the
// rows kept by the launch's workgroups, each adding its own kept_here), and
// on the call's last chunk folds the call into the store's bookkeeping
// (arrival count, and delta_hat of a call that waits, if the call went
// through; an error count if its input was invalid), copies the status words
// to host memory when asked, and clears them for the next call.  A
// workgroup's count and its kept rows go in one 64-bit atomic, so the last
// one knows the total from the value it gets back.  The only words of this
// launch it reads are the status words' maxima of a call that waits, updated
// by atomics that each workgroup has waited for before its count;
// everything else it reads was written by earlier launches.  Called by every
// thread of every workgroup.
template <class F>
__device__ __forceinline__ void append_finish(const AppendArgs& a, bool count_every_chunk, uint32_t kept_here,
                                              F&& last_work) {
  if (!a.last_chunk && !count_every_chunk) return;
  __shared__ bool last;
  __shared__ uint32_t kept_total;
  unsigned long long* done_kept = reinterpret_cast<unsigned long long*>(&a.cc->blocks_done);
  __syncthreads();
  if (threadIdx.x == 0) {
    const unsigned long long prev = atomicAdd(done_kept, ((unsigned long long)kept_here << 32) | 1ull);
    last = (uint32_t)prev == gridDim.x - 1;
    kept_total = (uint32_t)(prev >> 32) + kept_here;
  }
  __syncthreads();
  if (!last) return;
  if (threadIdx.x == 0) {
    last_work(kept_total);
    if (a.flags_out) __builtin_amdgcn_s_waitcnt(0);   // its atomics are performed before the words are exported
  }
  if (!a.last_chunk) {
    if (threadIdx.x == 0) *done_kept = 0ull;
    return;
  }
  constexpr int kWords = (int)(sizeof(DevFlags) / 4);
  uint32_t* f = reinterpret_cast<uint32_t*>(a.flags);
  if (threadIdx.x == 0) {
    // atomic loads: this workgroup may hold the words in its L1 from its start
    auto ld = [](uint32_t* p) { return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT); };
    const uint32_t bad = (ld(&a.flags->nonfinite) ? 1u : 0u) | (ld(&a.flags->out_of_range) ? 2u : 0u);
    const bool overflow = (ld(&a.flags->pair_overflow) & 1u) != 0u;
    if (bad != 0u || (overflow && a.async_call)) {
      a.meta->err_calls += 1u;
      a.meta->err_bits |= bad | (overflow ? 4u : 0u);
    } else if (!overflow) {
      a.meta->n_seen += a.n_call;
      if (!a.async_call) {   // (a call that does not wait put its maximum in the bookkeeping already)
        const unsigned long long d2 =
            __hip_atomic_load(&a.flags->dhat2_bits, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        if (d2 > a.meta->dhat2_bits) a.meta->dhat2_bits = d2;   // non-negative doubles order as their bits
      }
    }
  }
  __syncthreads();
  if (a.flags_out) {   // (uniform) a call that waits: the words go to host memory first
    if ((int)threadIdx.x < kWords) {
      const uint32_t v = __hip_atomic_load(f + threadIdx.x, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      reinterpret_cast<uint32_t*>(a.flags_out)[threadIdx.x] = v;
    }
    __syncthreads();
  }
  if ((int)threadIdx.x < kWords) f[threadIdx.x] = 0u;
  if (threadIdx.x == 0) *done_kept = 0ull;
}

// One wave per row, four rows per workgroup, decisions from k_resolve.  Kept
// rows are copied into the store; for dropped rows ||x - x_rep||^2 is formed
// in binary64 (fixed order) and the workgroup's maximum goes to the measured
// bound with one atomic.
__global__ __launch_bounds__(256) void k_append(AppendArgs a, int nB) {
  const int wave = threadIdx.x >> 6;
  const int r = (int)blockIdx.x * kAppendRows + wave;   // one row per wave
  const int rc = min(r, nB - 1);
  // Every load that depends on no other is issued before any is used: the
  // row's decision, its terms, the status words, the arrival count and (for
  // D <= 1,024) the row itself through a buffer resource (zeros past the row).
  const int p = a.pos[rc];
  const int rr = a.rep_row[rc];
  const float hn = a.hnc[rc], et = a.etc[rc];
  const bool skip = skip_all(a.flags);
  // every workgroup reads n_seen before the last one (below) advances it
  const int64_t gbase = a.meta->n_seen + a.c0;
  const uint32_t am0 = a.meta->absmax_bits, hm0 = a.meta->hnmax_bits;   // the store's maxima so far
  float4 v[kAppendVec];
  append_load(a, rc, v);
  double dmax = 0.0;
  uint32_t amax = 0u, hmax = 0u;
  if (!skip && r < nB) append_row(a, r, p, rr, hn, et, gbase, v, dmax, amax, hmax);
  __shared__ double part[4];
  __shared__ uint32_t apart[4], hpart[4];
  append_maxima<4>(a, dmax, amax, hmax, am0, hm0, part, apart, hpart);
  append_finish(a, false, 0u, [](uint32_t) {});
}

// The in-chunk resolve and the append in one launch.  Workgroup b appends
// rows [16 b, 16 b + 16) of the chunk, one wave per row; it first resolves,
// in its own LDS, every row up to its last one (a decision depends only on
// earlier rows: those with a store hit or without in-chunk candidates are
// immediate, the rest take a few rounds).  This saves a launch and the
// decisions' round trip through global memory.  Every workgroup reads the
// store size at its start and adds its own kept count to the chunk's; the
// last one to finish advances the store size.
constexpr int kAppendGroupThreads = kResolveThreads;
constexpr int kAppendGroupRows = kAppendGroupThreads / 64;

__global__ __launch_bounds__(kAppendGroupThreads) void k_resolve_append(ResolveArgs ra, AppendArgs a, int nB,
                                                                         float* max_cos,
                                                                         const uint32_t* maxcos_store,
                                                                         const float* G) {
  __shared__ ResolveLds L;
  constexpr int T = kAppendGroupThreads;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int r = (int)blockIdx.x * kAppendGroupRows + wave;   // this wave's row
  const int rc = min(r, nB - 1);
  const int nres = min(nB, ((int)blockIdx.x + 1) * kAppendGroupRows);   // rows this workgroup resolves
  // every load that depends on no other first: hits and edge flags of the
  // rows resolved here, the status words, the store's counts, and this
  // wave's row with its terms
  constexpr int kRowsPerThread = kChunk / T;
  int32_t hit_r[kRowsPerThread];
  uint32_t edge_r[kRowsPerThread];
#pragma unroll
  for (int u = 0; u < kRowsPerThread; ++u) {
    const int q = tid + u * T;
    hit_r[u] = q < nres ? ra.firstHit[q] : kNone;
    edge_r[u] = q < nres ? ra.hasEdge[q] : 0u;
  }
  const bool skip = skip_all(a.flags);
  const int m0 = a.meta->m;
  const int64_t gbase = a.meta->n_seen + a.c0;
  const uint32_t am0 = a.meta->absmax_bits, hm0 = a.meta->hnmax_bits;
  const float hn = a.hnc[rc], et = a.etc[rc];
  float4 v[kAppendVec];
  append_load(a, rc, v);
  double dmax = 0.0;
  uint32_t amax = 0u, hmax = 0u;
  uint32_t kept_here = 0u;
  if (!skip) {   // (uniform: the status words do not change during this launch)
    resolve_core<T>(ra, L, nres, m0, hit_r, edge_r);
    if (r < nB) {
      const int rr = L.rrow[r];
      if (lane == 0) ra.rep[r] = rr >= 0 ? ra.store_ids[rr] : (rr == -1 ? -1 : gbase + (-rr - 2));
      append_row(a, r, L.posv[r], rr, hn, et, gbase, v, dmax, amax, hmax);
      if (max_cos) {
        // the largest cosine over the store (from the screen) and over the
        // kept chunk rows before this one
        float mc = ord2f(maxcos_store[r]);
        for (int j = lane; j < r; j += 64)
          if (L.st[j] == 1) mc = fmaxf(mc, G[(int64_t)r * nB + j]);
        for (int o = 32; o > 0; o >>= 1) mc = fmaxf(mc, __shfl_xor(mc, o));
        if (lane == 0) max_cos[r] = mc;
      }
    }
    // kept rows among this workgroup's own
    const int first = (int)blockIdx.x * kAppendGroupRows;
    const uint64_t k = __ballot(lane < nres - first && L.st[first + lane] == 1);
    kept_here = (uint32_t)__popcll(k);
  }
  __shared__ double part[T / 64];
  __shared__ uint32_t apart[T / 64], hpart[T / 64];
  append_maxima<T / 64>(a, dmax, amax, hmax, am0, hm0, part, apart, hpart);
  append_finish(a, true, kept_here, [&](uint32_t total) {
    if (skip) return;
    a.meta->m = m0 + (int)total;
    atomicAdd(&a.flags->n_kept, total);
  });
}

// ------------------------------------------------------------------ max cos
// max over store rows (from the screen) and over kept chunk rows j < i of the
// screened dot product.
__global__ __launch_bounds__(256) void k_maxcos(int nB, const uint32_t* maxcos_store, const float* G,
                                                const uint64_t* kept_words, float* out, DevFlags* flags) {
  if (skip_all(flags)) return;
  const int lane = threadIdx.x & 63;
  const int i = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (i >= nB) return;
  float m = ord2f(maxcos_store[i]);
  for (int j = lane; j < i; j += 64)
    if ((kept_words[j >> 6] >> (j & 63)) & 1ull) m = fmaxf(m, G[(int64_t)i * nB + j]);
  for (int o = 32; o > 0; o >>= 1) m = fmaxf(m, __shfl_xor(m, o));
  if (lane == 0) out[i] = m;
}

}  // namespace

// ------------------------------------------------------------------ store memory

lam_status store_alloc(lam_store* st) {
  const size_t cap = (size_t)st->capacity, D = (size_t)st->dim;
  LAM_HIP(hipMalloc(&st->x32, cap * D * 4));
  LAM_HIP(hipMalloc(&st->x16, cap * D * 2));
  LAM_HIP(hipMalloc(&st->hn, cap * 4));
  LAM_HIP(hipMalloc(&st->et, cap * 4));
  LAM_HIP(hipMalloc(&st->ids, cap * 8));
  LAM_HIP(hipMalloc(&st->stat_dev, sizeof(StoreMeta)));
  LAM_HIP(hipMemset(st->stat_dev, 0, sizeof(StoreMeta)));
  LAM_HIP(hipHostMalloc(&st->meta_host, sizeof(StoreMeta), hipHostMallocDefault));
  if (st->lsh_r > 0) {
    const uint64_t entries = (uint64_t)cap * (uint64_t)st->lsh_nb;
    uint64_t slots = 1;
    while (slots < 2 * entries) slots <<= 1;
    st->lsh_slots = slots;
    LAM_HIP(hipMalloc(&st->lsh_key, slots * 8));
    LAM_HIP(hipMalloc(&st->lsh_head, slots * 4));
    LAM_HIP(hipMalloc(&st->lsh_next, entries * 4));
    LAM_HIP(hipMalloc(&st->lsh_rowkey, entries * 8));
    LAM_HIP(hipMemset(st->lsh_key, 0, slots * 8));
    LAM_HIP(hipMemset(st->lsh_head, 0xff, slots * 4));   // -1: empty list
  }
  LAM_HIP(hipDeviceSynchronize());
  st->thr = exact_threshold(st->tau);
  return LAM_OK;
}

lam_status lsh_reset(lam_ctx* ctx, lam_store* st, int64_t keep_rows) {
  if (st->lsh_r <= 0) return LAM_OK;
  const unsigned g = (unsigned)std::min<uint64_t>((st->lsh_slots + 255) / 256, 8192);
  hipLaunchKernelGGL(k_lsh_clear_index, dim3(g), dim3(256), 0, ctx->stream, st->lsh_key, st->lsh_head,
                     st->lsh_slots);
  LAM_HIP(hipGetLastError());
  const int64_t ne = keep_rows * st->lsh_nb;
  if (ne > 0) {
    const unsigned g2 = (unsigned)std::min<int64_t>((ne + 255) / 256, 8192);
    hipLaunchKernelGGL(k_lsh_reinsert, dim3(g2), dim3(256), 0, ctx->stream, st->lsh_key, st->lsh_head,
                       st->lsh_next, st->lsh_rowkey, (uint64_t)(st->lsh_slots - 1), ne);
    LAM_HIP(hipGetLastError());
  }
  return LAM_OK;
}

void store_free(lam_store* st) {
  for (void* p : {(void*)st->x32, (void*)st->x16, (void*)st->hn, (void*)st->et, (void*)st->ids,
                  (void*)st->stat_dev, (void*)st->codes})
    if (p) (void)hipFree(p);
  for (void* p : {(void*)st->blk_w, (void*)st->blk_row_off, (void*)st->blk_data, (void*)st->lsh_key,
                  (void*)st->lsh_head, (void*)st->lsh_next, (void*)st->lsh_rowkey})
    if (p) (void)hipFree(p);
  st->lsh_key = st->lsh_rowkey = nullptr;
  st->lsh_head = st->lsh_next = nullptr;
  st->blk_w = nullptr;
  st->blk_row_off = nullptr;
  st->blk_data = nullptr;
  st->blk_cap = 0;
  st->blk_rows = -1;
  if (st->meta_host) (void)hipHostFree(st->meta_host);
  st->meta_host = nullptr;
  st->x32 = nullptr;
  st->x16 = nullptr;
  st->hn = st->et = st->stat_dev = nullptr;
  st->ids = nullptr;
  st->codes = nullptr;
}

// ------------------------------------------------------------------ host orchestration
namespace {

struct Consts {
  double K1, K2, K3h;
};

Consts screen_consts(int D) {
  const double uh = std::ldexp(1.0, -11), u = std::ldexp(1.0, -24), eta = std::ldexp(1.0, -22);
  const double g = 2.0 * D * u / (1.0 - 2.0 * D * u);
  Consts c;
  c.K1 = (2.0 * uh + uh * uh + g * (1.0 + uh) * (1.0 + uh)) * 1.01;
  c.K2 = eta * (1.0 + uh) * (1.0 + g) * 1.01;
  c.K3h = 0.5 * D * eta * eta * (1.0 + g) * 1.01;
  return c;
}

// Ambiguous-pair entries (12 bytes each) reserved for a call that does not
// wait for the device: such a call needs room for every pair one chunk can
// produce, n (m + n).
constexpr uint64_t kAsyncPairLimit = 1ull << 26;

}  // namespace

// The device bookkeeping is copied to pinned host memory on the stream of the
// last call that did not wait, behind that call, and read after one wait for
// the stream (an event wait and then a synchronous copy would be two).
lam_status store_settle(lam_store* st) {
  if (!st->pending) return LAM_OK;
  LAM_HIP(hipMemcpyAsync(st->meta_host, st->stat_dev, sizeof(StoreMeta), hipMemcpyDeviceToHost, st->last_stream));
  LAM_HIP(hipStreamSynchronize(st->last_stream));
  StoreMeta m{};
  memcpy(&m, st->meta_host, sizeof m);
  st->pending = false;
  st->size = m.m;
  st->size_ub = m.m;
  st->n_seen = m.n_seen;
  st->absmax_bits = m.absmax_bits;
  st->hnmax_bits = m.hnmax_bits;
  st->maxima_known = true;
  double dh2 = 0.0;
  memcpy(&dh2, &m.dhat2_bits, 8);
  st->delta_hat_run = std::sqrt(dh2);
  if (m.err_calls != 0u) {
    const uint32_t calls = m.err_calls, bits = m.err_bits;
    m.err_calls = 0u;
    m.err_bits = 0u;
    LAM_HIP(hipMemcpy(st->stat_dev, &m, sizeof m, hipMemcpyHostToDevice));
    set_error("%u earlier ingest call(s) that did not wait for the device had %s; they left the store "
              "unchanged and wrote no outputs", calls,
              (bits & 4u) ? "too many ambiguous pairs (internal)"
                          : (bits & 1u) ? "NaN or Inf in the input" : "coordinates with |x| >= 255.9375");
    return LAM_EINVAL;
  }
  return LAM_OK;
}

lam_status store_maxima(lam_store* st) {
  LAM_TRY(store_settle(st));
  if (st->maxima_known) return LAM_OK;
  if (st->meta_reset) {   // cleared, and no ingest since: nothing retained
    st->absmax_bits = 0u;
    st->hnmax_bits = 0u;
    st->maxima_known = true;
    return LAM_OK;
  }
  StoreMeta m{};
  LAM_HIP(hipMemcpy(&m, st->stat_dev, sizeof m, hipMemcpyDeviceToHost));
  st->absmax_bits = m.absmax_bits;
  st->hnmax_bits = m.hnmax_bits;
  st->maxima_known = true;
  return LAM_OK;
}

lam_status dedup_ingest(lam_ctx* ctx, lam_store* st, const float* x, int64_t n, int64_t* rep, float* max_cos,
                        lam_ingest_stats* stats) {
  const int D = st->dim;
  if (n == 0) {
    if (stats) {
      LAM_TRY(store_settle(st));
      *stats = lam_ingest_stats{};
      stats->min_margin_d2 = HUGE_VAL;
      stats->store_size = st->size;
      stats->delta_hat_run = st->delta_hat_run;
    }
    return LAM_OK;
  }
  const int CH = (int)std::min<int64_t>(n, kChunk);
  const int W = (CH + 63) / 64;
  const bool lsh = st->lsh_r > 0;
  LAM_CHECK(!(lsh && max_cos), LAM_EINVAL, "max_cos is not available on a store with a band index");

  // A call without stats does not wait for the device when the ambiguous-pair
  // list can hold every pair its chunks could produce (so it cannot overflow)
  // and the store has room even if every earlier row was kept.  Otherwise the
  // call waits, checks the status words and, on an overflow, repeats with a
  // larger list.
  const int64_t m_ub = st->pending ? st->size_ub : st->size;
  const uint64_t worst = (uint64_t)CH * (uint64_t)(m_ub + n);
  const bool async = stats == nullptr && worst <= kAsyncPairLimit && m_ub + n <= st->capacity;
  if (!async) {
    LAM_TRY(store_settle(st));
    LAM_CHECK(n <= st->capacity - st->size, LAM_ECAPACITY, "store holds %lld of %lld rows; a batch of %lld may not fit",
              (long long)st->size, (long long)st->capacity, (long long)n);
  } else if (ctx->pair_cap < worst) {
    // grow geometrically: every growth reallocates, which waits for the device
    ctx->pair_cap = (uint32_t)std::min<uint64_t>(kAsyncPairLimit, std::max<uint64_t>(worst, 2ull * ctx->pair_cap));
  }
  // the rows this call appends may raise the store's maxima (after the
  // settling above, which reads the maxima of the earlier calls)
  st->maxima_known = false;
  const int64_t m_before = async ? m_ub : st->size;   // exact when waiting, an upper bound otherwise
  const Consts K = screen_consts(D);
  StoreMeta* meta = reinterpret_cast<StoreMeta*>(st->stat_dev);
  const bool want_max = max_cos != nullptr;

  // scratch
  LAM_TRY(ctx->scratch[S_X16].ensure((size_t)n * D * 2));
  LAM_TRY(ctx->scratch[S_ROWF].ensure((size_t)n * 8));
  const size_t chunk_bytes = (size_t)CH * 4 * 6 + 64 * 8 + sizeof(ChunkCounters) + 256;
  LAM_TRY(ctx->scratch[S_CHUNK].ensure(chunk_bytes));
  LAM_TRY(ctx->scratch[S_BITMAP].ensure((size_t)CH * W * 8));
  if (want_max) LAM_TRY(ctx->scratch[S_G].ensure((size_t)CH * CH * 4));
  _Float16* x16c = ctx->scratch[S_X16].as<_Float16>();
  float* hnc = ctx->scratch[S_ROWF].as<float>();
  float* etc = hnc + n;
  char* cb = ctx->scratch[S_CHUNK].as<char>();
  int32_t* firstHit = reinterpret_cast<int32_t*>(cb);
  uint32_t* hasEdge = reinterpret_cast<uint32_t*>(cb + (size_t)CH * 4);
  uint32_t* maxcos = reinterpret_cast<uint32_t*>(cb + (size_t)CH * 8);
  int32_t* pos = reinterpret_cast<int32_t*>(cb + (size_t)CH * 12);
  int32_t* rep_row = reinterpret_cast<int32_t*>(cb + (size_t)CH * 16);
  uint64_t* kept_words = reinterpret_cast<uint64_t*>(cb + (size_t)CH * 24);
  ChunkCounters* cc = reinterpret_cast<ChunkCounters*>(cb + (size_t)CH * 24 + 64 * 8);
  uint64_t* bitmap = ctx->scratch[S_BITMAP].as<uint64_t>();
  float* G = want_max ? ctx->scratch[S_G].as<float>() : nullptr;

  // banded candidates: chunk keys and the chunk's own index
  LshArgs la{};
  if (lsh) {
    const int nb = st->lsh_nb;
    const uint64_t ce = (uint64_t)CH * nb;
    uint64_t bslots = 1;
    while (bslots < 2 * ce) bslots <<= 1;
    LAM_TRY(ctx->scratch[kScratchLsh].ensure(ce * 8 + bslots * 8 + bslots * 4 + ce * 4));
    char* lb = ctx->scratch[kScratchLsh].as<char>();
    la.ckey = reinterpret_cast<unsigned long long*>(lb);
    la.bkey = reinterpret_cast<unsigned long long*>(lb + ce * 8);
    la.bhead = reinterpret_cast<int32_t*>(lb + ce * 8 + bslots * 8);
    la.bnext = reinterpret_cast<int32_t*>(lb + ce * 8 + bslots * 12);
    la.bslots = bslots;
    la.bmask = bslots - 1;
    la.xs = st->x32;
    la.xs16 = st->x16;
    la.hns = st->hn;
    la.ets = st->et;
    la.half_d2 = 0.5 * st->d2;
    la.D = D;
    la.r = st->lsh_r;
    la.nb = nb;
    la.eps = st->lsh_eps;
    la.s = 2.0 * st->lsh_eps;
    la.inv_s = 1.0 / la.s;
    la.inv_s32 = (float)la.inv_s;
    la.skey = st->lsh_key;
    la.shead = st->lsh_head;
    la.snext = st->lsh_next;
    la.srowkey = st->lsh_rowkey;
    la.smask = st->lsh_slots - 1;
    la.meta = meta;
    la.d2 = st->d2;
    la.thr = st->thr;
    la.firstHit = firstHit;
    la.bitmap = bitmap;
    la.W = W;
    la.hasEdge = hasEdge;
    la.cc = cc;
    la.flags = ctx->flags_dev;
  }

  for (int attempt = 0; attempt < 4; ++attempt) {
    const uint32_t cap = ctx->pair_cap;
    LAM_TRY(ctx->scratch[S_PAIRS].ensure((size_t)cap * sizeof(int2)));
    LAM_TRY(ctx->scratch[S_STATUS].ensure((size_t)cap * 4));
    int2* pairs = ctx->scratch[S_PAIRS].as<int2>();
    uint32_t* status = ctx->scratch[S_STATUS].as<uint32_t>();
    // a repeated attempt starts from the store as it was: the band index is
    // rebuilt from the rows retained before the call
    if (lsh && attempt > 0) LAM_TRY(lsh_reset(ctx, st, m_before));

    for (int64_t c0 = 0; c0 < n; c0 += CH) {
      const int nB = (int)std::min<int64_t>(CH, n - c0);
      const float* xc = x + c0 * D;
      const _Float16* x16 = x16c + c0 * D;
      const bool last_chunk = c0 + CH >= n;
      // a waiting call sets the store size (so a repeated attempt starts from
      // the store as it was); otherwise the kernels keep it
      const ChunkState cs{firstHit, hasEdge, maxcos, bitmap, W, nB, cc, meta, async ? -1 : (int32_t)m_before,
                          st->meta_reset ? 1 : 0};
      if (c0 == 0) {
        // the status words must be zero before prep counts into them; the
        // last append of every call leaves them zero
        if (!ctx->flags_zero) LAM_TRY(clear_flags(ctx));
        ctx->flags_zero = false;
        ProfScope ps(ctx, "dedup_prep");
        hipLaunchKernelGGL(k_prep, dim3((unsigned)((n + 3) / 4)), dim3(256), 0, ctx->stream, x, n, D, x16c, hnc,
                           etc, K.K1, K.K2, K.K3h, ctx->flags_dev, cs);
        LAM_HIP(hipGetLastError());
        st->meta_reset = false;
      } else {
        hipLaunchKernelGGL(k_chunk_init, dim3(64), dim3(256), 0, ctx->stream, cs);
        LAM_HIP(hipGetLastError());
      }

      if (lsh) {
        la.xc = xc;
        la.xc16 = x16;
        la.hnc = hnc + c0;
        la.etc = etc + c0;
        la.nB = nB;
        la.m_exact = (!async && c0 == 0) ? (int)m_before : -1;
        la.pairs = pairs;
        la.pair_cap = cap;
        const int64_t ne = (int64_t)nB * la.nb;
        const int64_t nt = std::max<int64_t>(ne, (int64_t)la.bslots);
        {
          ProfScope ps(ctx, "lsh_keys");
          hipLaunchKernelGGL(k_lsh_keys, dim3((unsigned)((nt + 255) / 256)), dim3(256), 0, ctx->stream, la);
          LAM_HIP(hipGetLastError());
          hipLaunchKernelGGL(k_lsh_index_chunk, dim3((unsigned)((ne + 255) / 256)), dim3(256), 0, ctx->stream, la);
          LAM_HIP(hipGetLastError());
        }
        {
          ProfScope ps(ctx, "lsh_admit");
          hipLaunchKernelGGL(k_lsh_admit, dim3((unsigned)nB), dim3(kAdmitThreads), (size_t)D * 4, ctx->stream, la);
          LAM_HIP(hipGetLastError());
        }
      }
      ScreenArgs sa{};
      sa.As = st->x16;
      sa.hnS = st->hn;
      sa.etS = st->et;
      sa.meta = meta;
      sa.m_exact = (!async && c0 == 0) ? (int)m_before : -1;   // otherwise read the kernel-maintained count
      sa.capA = (int)std::min<int64_t>(st->capacity, INT32_MAX);
      sa.B = x16;
      sa.hnB = hnc + c0;
      sa.etB = etc + c0;
      sa.nB = nB;
      sa.D = D;
      sa.half_d2 = 0.5 * st->d2;
      sa.firstHit = firstHit;
      sa.maxcos = maxcos;
      sa.bitmap = bitmap;
      sa.W = W;
      sa.hasEdge = hasEdge;
      sa.G = G;
      sa.pairs = pairs;
      sa.pair_cap = cap;
      sa.cc = cc;
      sa.flags = ctx->flags_dev;
      // against the store (rows retained before this chunk; the kernel reads
      // the exact count, the grid covers an upper bound) and inside the chunk
      const int64_t m_grid = m_before + c0;
      auto grid_of = [&](int rows) {
        const int64_t nt = (nB + rows - 1) / rows;
        return ((m_grid + rows - 1) / rows) * nt + nt * (nt + 1) / 2;
      };
      const bool large_ok = !want_max && (D == 768 || D == 1024);
      const bool large = large_ok && (ctx->screen_tile == LAM_SCREEN_TILE_LARGE ||
                                      (ctx->screen_tile == LAM_SCREEN_TILE_AUTO &&
                                       grid_of(ScreenTileL::BN) >= kLargeTileMinTiles));
      const int tb_rows = large ? ScreenTileL::BN : ScreenTile::BN;
      const int ntBt = (nB + tb_rows - 1) / tb_rows;
      sa.ntB = ntBt;
      sa.nb0 = ((m_grid + tb_rows - 1) / tb_rows) * ntBt;
      sa.nb1 = (int64_t)ntBt * (ntBt + 1) / 2;
      const int64_t grid = sa.nb0 + sa.nb1;
      LAM_CHECK(grid < (1LL << 31), LAM_EINVAL, "screen grid too large");
      if (!lsh) {
        // timed by the launch itself when profiled (the dominant kernel)
        hipEvent_t e0, e1;
        LAM_TRY(prof_launch_events(ctx, "dedup_screen", &e0, &e1));
        // the common dims get a fully unrolled reduction
        const dim3 g((unsigned)grid);
        if (large) {
          const dim3 b(ScreenTileL::kThreads);
          if (D == 768)
            hipExtLaunchKernelGGL((k_screen<ScreenTileL, false, 12, 1>), g, b, 0, ctx->stream, e0, e1, 0, sa);
          else
            hipExtLaunchKernelGGL((k_screen<ScreenTileL, false, 16, 1>), g, b, 0, ctx->stream, e0, e1, 0, sa);
        } else {
          const dim3 b(ScreenTile::kThreads);
          if (want_max)
            hipExtLaunchKernelGGL((k_screen<ScreenTile, true, 0>), g, b, 0, ctx->stream, e0, e1, 0, sa);
          else if (D == 768)
            hipExtLaunchKernelGGL((k_screen<ScreenTile, false, 12>), g, b, 0, ctx->stream, e0, e1, 0, sa);
          else if (D == 1024)
            hipExtLaunchKernelGGL((k_screen<ScreenTile, false, 16>), g, b, 0, ctx->stream, e0, e1, 0, sa);
          else
            hipExtLaunchKernelGGL((k_screen<ScreenTile, false, 0>), g, b, 0, ctx->stream, e0, e1, 0, sa);
        }
        LAM_HIP(hipGetLastError());
      }
      VerifyArgs va{pairs, status, cc, cap, xc, st->x32, D, st->d2, st->thr, firstHit, bitmap, W, hasEdge,
                    ctx->flags_dev, cc};
      {
        ProfScope ps(ctx, "dedup_verify");
        hipLaunchKernelGGL(k_verify, dim3(256), dim3(256), 0, ctx->stream, va);
        LAM_HIP(hipGetLastError());
      }
      ResolveArgs ra{nB, W, firstHit, hasEdge, bitmap, st->ids, meta, c0, rep + c0, pos, rep_row, kept_words,
                     ctx->flags_dev};
      AppendArgs aa{xc, x16, hnc + c0, etc + c0, pos, rep_row, c0, D, st->x32, st->x16, st->hn, st->et, st->ids,
                    ctx->flags_dev, cc, meta, n, last_chunk ? 1 : 0, async ? 1 : 0,
                    (last_chunk && !async) ? ctx->flags_host_dev : nullptr};
      if (!lsh) {
        // resolve, largest cosines and append in one launch
        ProfScope ps(ctx, "dedup_resolve_append");
        hipLaunchKernelGGL(k_resolve_append, dim3((unsigned)((nB + kAppendGroupRows - 1) / kAppendGroupRows)),
                           dim3(kAppendGroupThreads), 0, ctx->stream, ra, aa, nB, want_max ? max_cos + c0 : nullptr,
                           maxcos, G);
        LAM_HIP(hipGetLastError());
        continue;
      }
      {
        ProfScope ps(ctx, "dedup_resolve");
        hipLaunchKernelGGL(k_resolve, dim3(1), dim3(kResolveThreads), 0, ctx->stream, ra);
        LAM_HIP(hipGetLastError());
      }
      if (want_max) {
        hipLaunchKernelGGL(k_maxcos, dim3((unsigned)((nB + 3) / 4)), dim3(256), 0, ctx->stream, nB, maxcos, G,
                           kept_words, max_cos + c0, ctx->flags_dev);
        LAM_HIP(hipGetLastError());
      }
      if (lsh) {
        // kept rows join the store's index before the append of the last
        // chunk hands the status words back (and zeroes them)
        ProfScope ps(ctx, "lsh_insert");
        hipLaunchKernelGGL(k_lsh_insert, dim3((unsigned)(((int64_t)nB * la.nb + 255) / 256)), dim3(256), 0,
                           ctx->stream, la, pos, st->lsh_key, st->lsh_head, st->lsh_next, st->lsh_rowkey);
        LAM_HIP(hipGetLastError());
      }
      {
        ProfScope ps(ctx, "dedup_append");
        hipLaunchKernelGGL(k_append, dim3((unsigned)((nB + kAppendRows - 1) / kAppendRows)), dim3(256), 0,
                           ctx->stream, aa, nB);
        LAM_HIP(hipGetLastError());
      }
    }
    ctx->flags_zero = true;   // the last append clears the status words
    if (async) {
      st->last_stream = ctx->stream;
      st->pending = true;
      st->size_ub = m_before + n;
      return LAM_OK;
    }
    // the last append wrote the status words to host memory
    LAM_HIP(hipStreamSynchronize(ctx->stream));
    const DevFlags f = *ctx->flags_host;
    LAM_CHECK(f.nonfinite == 0, LAM_EINVAL, "input holds NaN or Inf (%u rows)", f.nonfinite);
    LAM_CHECK(f.out_of_range == 0, LAM_EINVAL, "input has coordinates with |x| >= 255.9375 (%u rows)", f.out_of_range);
    if (f.pair_overflow & 1u) {
      ctx->pair_cap = std::max<uint32_t>(ctx->pair_cap * 2u, f.pairs_needed + (f.pairs_needed >> 2));
      continue;
    }
    double dh2 = 0.0;
    memcpy(&dh2, &f.dhat2_bits, 8);
    const double dh_call = std::sqrt(dh2);
    st->size = m_before + f.n_kept;
    st->size_ub = st->size;
    st->n_seen += n;
    st->delta_hat_run = std::max(st->delta_hat_run, dh_call);
    if (stats) {
      stats->n_in = n;
      stats->n_kept = f.n_kept;
      stats->n_dropped = n - f.n_kept;
      stats->store_size = st->size;
      stats->n_ambiguous_pairs = lsh ? (int64_t)f.n_cand : (int64_t)f.n_pairs;
      stats->n_exact_escalations = f.n_escalate;
      double mg = HUGE_VAL;
      if (f.margin_inv != 0ull) {
        const unsigned long long bits = ~f.margin_inv;
        memcpy(&mg, &bits, 8);
      }
      stats->min_margin_d2 = mg;
      stats->delta_hat_call = dh_call;
      stats->delta_hat_run = st->delta_hat_run;
    }
    return LAM_OK;
  }
  set_error("ingest did not converge (ambiguous-pair list kept overflowing)");
  return LAM_EDEVICE;
}

}  // namespace lam
