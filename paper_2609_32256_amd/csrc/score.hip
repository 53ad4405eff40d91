// Retrieval scoring against the quantized store, dequantized on the fly, with
// top-k per query and the per-query bound eps * ||q||_1 (Hoelder applied to
// the per-coordinate bound of Q_eps, Appendix "Rank invariance, in full").
//
// score(j, y) = s * sum_d q_j,d * code_y,d  (s = 2 eps), i.e. q_j . x_hat_y with
// the exact dequantized row.  Codes of at most 12 bits are exact in fp16.
// Codes of 13 to 22 bits are scored as a 12-bit store of 2D columns, each
// code c split as 2^11 (c >> 11) + (c & 2047), against queries [2^11 q, q]:
// the same score term by term (see widen).
// Each query is scaled by a power of two 2^e_j (max |q| into [2^14, 2^15)) and
// split into fp16 hi + lo parts, q 2^e = hi + lo + r with |r| <= 2^-22 |q 2^e|;
// hi*code and lo*code are exact in fp32 and the MFMA accumulates in fp32.  The
// score is acc * float32(s 2^-e_j).
//
// Kernel layout: a workgroup owns 128 queries and a contiguous range ("split")
// of the store, walked in 128-row tiles.  Per tile the codes are unpacked from
// their b-bit words straight into an fp16 LDS slab (no dequantized copy exists
// in HBM) and multiplied with the query slabs on v_mfma_f32_32x32x16_f16.  Wave
// w holds queries [32w, 32w + 32) against all 128 rows of the tile, so every
// query lives in two lanes of one wave; each lane keeps a sorted private list
// of its best KL (score, row) pairs in registers, touched only when a score
// reaches the list's current threshold.  A merge kernel then picks the k best
// per query from all lists by (score desc, id asc).
//
// Stores beyond the sample size take a threshold plan (score_topk) whose
// sample and filter passes multiply the hi part alone -- half the MFMAs --
// with thresholds lowered by twice a per-query bound on the hi part's error;
// the few candidates near the k-th are then rescored exactly.  At D = 768 and
// 1,024 the filter pass is k_filter: one tile per workgroup on the
// similarity screen's pipeline (two LDS stages), 128 x 128 or, for launches
// of many tiles, 256 x 256.
#include <cmath>
#include <cstring>
#include <mutex>

#include "lam_internal.h"
#include "mfma_tile.h"
#include "wave.h"

namespace lam {
namespace {

constexpr int kNoRow = 0x7fffffff;

enum ScoreScratch { S_QHI = 7, S_QLO, S_QMETA, S_PART, S_CAND };

struct QMeta {
  float osc;     // float32(s * 2^-e): multiplies the raw accumulator
  float bound;   // eps * ||q||_1 rounded up, or NaN for an invalid query
  int bad;       // query holds NaN/Inf
  float err;     // >= |hi-only score - rescored score| for every store row (rounded up)
};

__device__ __forceinline__ float ru32(double d) {
  float f = (float)d;
  if ((double)f < d) f = __uint_as_float(__float_as_uint(f) + 1u);   // d >= 0 here
  return f;
}

__device__ __forceinline__ float rd32(double d) {
  float f = (float)d;
  if ((double)f > d) f = nextafterf(f, -INFINITY);
  return f;
}

// Per query: the hi/lo split and the meta block.  err bounds the difference
// between a score from the hi part alone (H) and the rescored one (S), both
// against T = s sum_d q_d code_d, in score units, with R >= s ||code_y|| for
// every row y (row_norm_bound) and h = hi 2^-e the query's hi part in its own
// units; the reported bound is eps times the l1 norm of columns [l1_from, D)
// (all of them, except for the split form of wide codes):
//   hi part:   |s sum_d (q_d - h_d) code_d| <= ||q - h||_2 R (Cauchy-Schwarz;
//              ||q - h||_2 is computed here in binary64);
//   fp32 sum:  g = 2 (D + 64) 2^-24 of s sum |h_d code_d| <= (||q|| + ||q - h||) R
//              (two roundings per addition, in any order);
//   scalings:  osc and the final product, 2^-24 each;
//   S:         the rescoring sums in binary64 and rounds once to float32.
// |H - S| <= |H - T| + |T - S| <= ||q - h|| R + (g + 2^-21)(||q|| + ||q - h||) R.
__global__ __launch_bounds__(256) void k_score_prep(const float* __restrict__ q, int64_t nq, int D, double s,
                                                    double eps, double R, int l1_from,
                                                    _Float16* __restrict__ qhi,
                                                    _Float16* __restrict__ qlo, QMeta* __restrict__ meta,
                                                    uint32_t* __restrict__ cand_cnt, uint32_t* __restrict__ tflag) {
  const int lane = threadIdx.x & 63;
  const int64_t j = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (j >= nq) return;
  // the threshold plan's candidate count of this query and flag of its query
  // tile start at zero (the buffers may hold anything from an earlier call)
  if (cand_cnt && lane == 0) {
    cand_cnt[j] = 0u;
    if (j % kTB == 0) {
      const int64_t nqt = (nq + kTB - 1) / kTB;
      tflag[j / kTB] = 0u;          // the tile's flag
      tflag[nqt + j / kTB] = 0u;    // and its fallback workgroups' completion count
    }
  }
  const float* p = q + j * D;
  float mx = 0.0f;
  double l1 = 0.0, l2 = 0.0;
  bool bad = false;
  // D <= 1,024: the row is loaded once as float4 pieces held in registers (all
  // loads in flight together; the resource ends at the row, so pieces past it
  // read as zero), and both passes below work from them
  constexpr int kVec = 4;
  const bool vec = D <= 256 * kVec;
  float4 v4[kVec];
  {
    const __amdgpu_buffer_rsrc_t rs =
        __builtin_amdgcn_make_buffer_rsrc(const_cast<float*>(p), (short)0, vec ? D * 4 : 0, 0x00020000);
#pragma unroll
    for (int u = 0; u < kVec; ++u)
      v4[u] = __builtin_bit_cast(float4, __builtin_amdgcn_raw_buffer_load_b128(rs, (uint32_t)(u * 256 + lane * 4) * 4u, 0, 0));
  }
  auto take1 = [&](float v, bool in_l1) {
    const float a = fabsf(v);
    bad |= !(a <= 3.402823466e38f);
    mx = fmaxf(mx, a);
    l1 += in_l1 ? (double)a : 0.0;
    l2 = fma((double)v, (double)v, l2);
  };
  if (vec) {
#pragma unroll
    for (int u = 0; u < kVec; ++u) {
      const int d = u * 256 + lane * 4;
      if (d >= D) break;
      const bool in = d >= l1_from;   // (l1_from is a multiple of 32)
      take1(v4[u].x, in);
      take1(v4[u].y, in);
      take1(v4[u].z, in);
      take1(v4[u].w, in);
    }
  } else {
    for (int d = lane; d < D; d += 64) take1(p[d], d >= l1_from);
  }
  mx = wave_max_f32(mx);
  l1 = wave_sum_f64(l1);
  l2 = wave_sum_f64(l2);
  bad = __ballot(bad) != 0ull;
  int e = 0;
  if (!bad && mx > 0.0f) e = 14 - ilogbf(mx);   // max |q| 2^e in [2^14, 2^15)
  const float sc = ldexpf(1.0f, e);
  const double isc = ldexp(1.0, -e);
  double dh2 = 0.0;   // ||q - h||^2
  auto split = [&](float x, _Float16& h, _Float16& l) {
    const float v = bad ? 0.0f : x * sc;     // exact power-of-two scaling
    h = (_Float16)v;
    l = (_Float16)(v - (float)h);
    const double r = bad ? 0.0 : (double)x - (double)(float)h * isc;   // exact in binary64
    dh2 = fma(r, r, dh2);
  };
  if (vec) {
#pragma unroll
    for (int u = 0; u < kVec; ++u) {
      const int d = u * 256 + lane * 4;
      if (d >= D) break;
      const float c[4] = {v4[u].x, v4[u].y, v4[u].z, v4[u].w};
      _Float16 h[4], l[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) split(c[e], h[e], l[e]);
      uint2 ph, pl;
      __builtin_memcpy(&ph, h, 8);
      __builtin_memcpy(&pl, l, 8);
      *reinterpret_cast<uint2*>(qhi + j * D + d) = ph;
      *reinterpret_cast<uint2*>(qlo + j * D + d) = pl;
    }
  } else {
    for (int d = lane; d < D; d += 64) {
      _Float16 h, l;
      split(p[d], h, l);
      qhi[j * D + d] = h;
      qlo[j * D + d] = l;
    }
  }
  dh2 = wave_sum_f64(dh2);
  if (lane == 0) {
    QMeta m;
    m.osc = (float)ldexp(s, -e);
    // (a binary64 sum of D non-negative terms is below the exact one by at most
    // (D - 1) 2^-53 relative, in any order; products and sqrt add 2^-53 each)
    const double up = 1.0 + (double)(D + 4) * 0x1p-52;
    m.bound = bad ? __builtin_nanf("") : ru32(eps * l1 * up);
    m.bad = bad ? 1 : 0;
    const double g = 2.0 * (double)(D + 64) * 0x1p-24;
    const double qn = sqrt(l2) * up;
    const double dh = sqrt(dh2) * up;
    const double E = dh * R + (g + 0x1p-21) * (qn + dh) * R;
    m.err = bad ? 0.0f : ru32(E * (1.0 + 0x1p-20));
    meta[j] = m;
  }
}


struct ScoreArgs {
  const uint32_t* codes;
  int64_t n;                 // store rows
  int D;
  int64_t row_words;         // D * b / 32
  const _Float16* qhi;
  const _Float16* qlo;
  const QMeta* meta;
  int64_t nq;
  int nqt;                   // query tiles of 128
  int64_t tile_begin;        // store tiles [tile_begin, tile_end) scanned by this launch
  int64_t tile_end;
  int splits;                // contiguous tile ranges per query tile
  int64_t tiles_per_split;
  float* part_s;             // list modes: [nq][splits][2][KL]
  int32_t* part_r;
  const float* thr;          // filter mode: per-query threshold
  float* cand_s;             // filter mode: [nq][cap]
  int32_t* cand_r;
  uint32_t* cand_cnt;
  uint32_t cap;
  const uint32_t* tflag;     // fallback mode: query tiles to redo
  // fallback mode: the last workgroup of a query tile merges its flagged queries
  const uint32_t* qflag;     // queries to redo
  uint32_t* tdone;           // per query tile: workgroups finished
  int k;
  float* out_s;
  int64_t* out_i;
  float* out_bound;
  const int64_t* ids;        // store row -> global id
};

__device__ __forceinline__ bool better(float a, int ra, float b, int rb) {
  return a > b || (a == b && ra < rb);
}

// Sorted insertion into a descending register list (entry KL-1 is dropped).
template <int KL>
__device__ __forceinline__ void list_insert(float (&ls)[KL], int (&lr)[KL], float sc, int row) {
  int qpos = 0;
#pragma unroll
  for (int p = 0; p < KL; ++p) qpos += better(ls[p], lr[p], sc, row) ? 1 : 0;
#pragma unroll
  for (int p = KL - 1; p >= 0; --p) {
    const float ps = (p > 0) ? ls[p - 1] : 0.0f;
    const int pr = (p > 0) ? lr[p - 1] : 0;
    ls[p] = (p > qpos) ? ps : (p == qpos ? sc : ls[p]);
    lr[p] = (p > qpos) ? pr : (p == qpos ? row : lr[p]);
  }
}

typedef _Float16 half2v __attribute__((ext_vector_type(2)));

// Unpacks 32 b-bit codes starting at word w (element 0 at bit 0) to fp16.
// Byte codes take an exact shortcut, two codes per step: the byte c + 128
// (c XOR 0x80) becomes the low byte of the fp16 bit pattern 0x6400 | byte,
// which is the value 1024 + c + 128 exactly; one packed fp16 subtraction of
// 1152 leaves c.
template <int B>
__device__ __forceinline__ void unpack32(const uint32_t* __restrict__ w, _Float16* __restrict__ out) {
  if constexpr (B == 8) {
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const uint32_t x = w[i] ^ 0x80808080u;
      // bytes 0..3 of the selection come from x, 4..7 from the constant 0x64646464
      const uint32_t lo = __builtin_amdgcn_perm(0x64646464u, x, 0x04010400u);
      const uint32_t hi = __builtin_amdgcn_perm(0x64646464u, x, 0x04030402u);
      const half2v off = {(_Float16)1152.0f, (_Float16)1152.0f};
      const half2v a = __builtin_bit_cast(half2v, lo) - off;
      const half2v b = __builtin_bit_cast(half2v, hi) - off;
      out[4 * i + 0] = a.x;
      out[4 * i + 1] = a.y;
      out[4 * i + 2] = b.x;
      out[4 * i + 3] = b.y;
    }
    return;
  }
  uint32_t v[B + 1];
#pragma unroll
  for (int i = 0; i < B; ++i) v[i] = w[i];
  v[B] = 0u;
#pragma unroll
  for (int e = 0; e < 32; ++e) {
    const int bit = e * B, wi = bit >> 5, off = bit & 31;
    uint32_t u = v[wi] >> off;
    if (off + B > 32) u |= v[wi + 1] << (32 - off);
    const int32_t c = (int32_t)(u << (32 - B)) >> (32 - B);
    out[e] = (_Float16)(float)c;
  }
}

// NC (16 or 32) b-bit codes from NC * B / 32 whole words (element 0 at bit 0)
// to fp16, as unpack32 does.
template <int B, int NC>
__device__ __forceinline__ void unpack_codes(const uint32_t* __restrict__ w, _Float16* __restrict__ out) {
  static_assert(NC == 16 || NC == 32, "a half or a whole group");
  constexpr int NW = NC * B / 32;
  if constexpr (NC == 32) {
    unpack32<B>(w, out);
  } else if constexpr (B == 8) {
#pragma unroll
    for (int i = 0; i < NW; ++i) {
      const uint32_t x = w[i] ^ 0x80808080u;
      const uint32_t lo = __builtin_amdgcn_perm(0x64646464u, x, 0x04010400u);
      const uint32_t hi = __builtin_amdgcn_perm(0x64646464u, x, 0x04030402u);
      const half2v off = {(_Float16)1152.0f, (_Float16)1152.0f};
      const half2v a = __builtin_bit_cast(half2v, lo) - off;
      const half2v b = __builtin_bit_cast(half2v, hi) - off;
      out[4 * i + 0] = a.x;
      out[4 * i + 1] = a.y;
      out[4 * i + 2] = b.x;
      out[4 * i + 3] = b.y;
    }
  } else {
    uint32_t v[NW + 1];
#pragma unroll
    for (int i = 0; i < NW; ++i) v[i] = w[i];
    v[NW] = 0u;
#pragma unroll
    for (int e = 0; e < NC; ++e) {
      const int bit = e * B, wi = bit >> 5, off = bit & 31;
      uint32_t u = v[wi] >> off;
      if (off + B > 32) u |= v[wi + 1] << (32 - off);
      const int32_t c = (int32_t)(u << (32 - B)) >> (32 - B);
      out[e] = (_Float16)(float)c;
    }
  }
}

// One group of 32 b-bit codes (B consecutive words starting at word w0 of the
// buffer, or zeros when !ok): the widest loads the group's alignment allows
// (a group starts at a multiple of B words), so a lane asks for its bytes in
// one or two pieces rather than B.
template <int B>
__device__ __forceinline__ void load_group(__amdgpu_buffer_rsrc_t rs, bool ok, uint32_t w0, uint32_t (&cw)[B]) {
  if constexpr (B % 4 == 0) {
#pragma unroll
    for (int i = 0; i < B; i += 4) {
      const uint4 v = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(rs, ok ? (w0 + i) * 4u : kOffOOB, 0, 0));
      cw[i] = v.x;
      cw[i + 1] = v.y;
      cw[i + 2] = v.z;
      cw[i + 3] = v.w;
    }
  } else if constexpr (B % 2 == 0) {
#pragma unroll
    for (int i = 0; i < B; i += 2) {
      const uint2 v = __builtin_bit_cast(uint2, __builtin_amdgcn_raw_buffer_load_b64(rs, ok ? (w0 + i) * 4u : kOffOOB, 0, 0));
      cw[i] = v.x;
      cw[i + 1] = v.y;
    }
  } else {
#pragma unroll
    for (int i = 0; i < B; ++i)
      cw[i] = (uint32_t)__builtin_amdgcn_raw_buffer_load_b32(rs, ok ? (w0 + i) * 4u : kOffOOB, 0, 0);
  }
}

// acc[t] (t = 0..3) <- the 128 x 128 tile of raw scores: store rows
// [rbase, rbase + rows) against the workgroup's 128 queries (wave w holds
// queries [32w, 32w + 32), lane j % 32, store rows t*32 + acc_row(r, lane)).
// Codes are unpacked straight into an fp16 LDS slab; queries enter as hi/lo
// (LO), or as the hi part alone.
//
// One LDS stage (codes, hi[, lo]: 2 or 3 x 128 rows of kLdk halves) is refilled
// between two barriers while the next slab's loads are in flight in
// registers; loads go through buffer resources (zeros past the tile) so none
// sits behind a branch.  With one slab in flight, the wait at the top of each
// step is for all outstanding loads, which is exactly the slab being stored.
// Ends with a barrier, so the caller may reuse the LDS.
template <int B, bool LO>
__device__ __forceinline__ void score_tile(const ScoreArgs& a, int64_t rbase, int rows, const _Float16* QH,
                                           const _Float16* QL, int qrows, _Float16* lds, floatx16 (&acc)[4]) {
  _Float16* sc = lds;
  _Float16* sh = lds + kTB * kLdk;
  _Float16* sl = lds + 2 * kTB * kLdk;
  const int wave = threadIdx.x >> 6;
  const int urow = threadIdx.x >> 1, uhalf = threadIdx.x & 1;   // unpack: 2 threads per row
#pragma unroll
  for (int t = 0; t < 4; ++t)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[t][r] = 0.0f;
  const __amdgpu_buffer_rsrc_t rsC = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint32_t*>(a.codes + rbase * a.row_words), (short)0, (int)(rows * a.row_words * 4), 0x00020000);
  const __amdgpu_buffer_rsrc_t rsH = tile_rsrc(QH, qrows, a.D), rsL = tile_rsrc(QL, qrows, a.D);
  auto load_slab = [&](int k0, uint32_t (&cw)[B], uint4 (&rh)[4], uint4 (&rl)[4]) {
    const bool ok = urow < rows && k0 + 32 * uhalf < a.D;
    const uint32_t w0 = (uint32_t)(urow * a.row_words + (int64_t)(k0 / 32 + uhalf) * B);
    load_group<B>(rsC, ok, w0, cw);
    slab_load_n<4>(rsH, qrows, a.D, k0, a.D, rh, kWG);
    if (LO) slab_load_n<4>(rsL, qrows, a.D, k0, a.D, rl, kWG);
  };
  auto compute = [&]() {
#pragma unroll
    for (int kk = 0; kk < kBK / 16; ++kk) {
      const half8 bh = frag_load(sh, wave * 32, kk);
      half8 fa[4];
#pragma unroll
      for (int t = 0; t < 4; ++t) fa[t] = frag_load(sc, t * 32, kk);
#pragma unroll
      for (int t = 0; t < 4; ++t) acc[t] = __builtin_amdgcn_mfma_f32_32x32x16_f16(fa[t], bh, acc[t], 0, 0, 0);
      if (LO) {
        const half8 bl = frag_load(sl, wave * 32, kk);
#pragma unroll
        for (int t = 0; t < 4; ++t) acc[t] = __builtin_amdgcn_mfma_f32_32x32x16_f16(fa[t], bl, acc[t], 0, 0, 0);
      }
    }
  };
  const int S = (a.D + kBK - 1) / kBK;
  uint32_t cw[B];
  uint4 rh[4], rl[4];
  load_slab(0, cw, rh, rl);
  for (int s = 0; s < S; ++s) {
    __syncthreads();   // every wave is done with the previous slab (or tile)
    {
      _Float16 h[32];
      unpack32<B>(cw, h);
      _Float16* dst = sc + urow * kLdk + uhalf * 32;
#pragma unroll
      for (int i = 0; i < 32; i += 8) *reinterpret_cast<uint4*>(dst + i) = *reinterpret_cast<const uint4*>(h + i);
    }
    slab_store_n<4>(sh, rh, kWG);
    if (LO) slab_store_n<4>(sl, rl, kWG);
    __syncthreads();
    load_slab((s + 1) * kBK, cw, rh, rl);   // past the last slab: zeros, no memory touched
    __builtin_amdgcn_sched_barrier(0);      // issue the loads before the MFMAs
    compute();
  }
  __syncthreads();
}

enum { kModeLists = 0, kModeFilter = 1, kModeFallback = 2 };

template <int KL, int SEG>
__device__ void merge_query(int64_t j, int cands, int k, const float* __restrict__ ps,
                            const int32_t* __restrict__ pr, const QMeta* __restrict__ meta,
                            const int64_t* __restrict__ ids, float* __restrict__ out_s, int64_t* __restrict__ out_i,
                            float* __restrict__ bound, float* __restrict__ kth);

// MODE kModeLists / kModeFallback: each lane keeps a sorted private list of its
// best KL (score, row) pairs; the lists go to part_s/part_r.  kModeFallback
// only runs query tiles flagged in tflag.  MODE kModeFilter: every score at or
// above the query's threshold is appended to its candidate buffer.  LO: the
// scores include the query's lo part; without it they are the hi-only scores
// H of the sample and filter passes (within QMeta::err of the rescored ones).
template <int B, int KL, int MODE, bool LO>
__global__ __launch_bounds__(kWG, 2) void k_score(ScoreArgs a) {
  // one slab stage (codes, hi[, lo]: 128 rows each) or the list epilogue's
  // 4 x 64 x 64 scores
  constexpr int kSlab = (LO ? 3 : 2) * kTB * kLdk;
  constexpr int kLists = MODE == kModeFilter ? 0 : 2 * 4 * 64 * 64;
  constexpr int kLdsHalves = kSlab > kLists ? kSlab : kLists;
  __shared__ __attribute__((aligned(16))) _Float16 lds[kLdsHalves];
  const int qt = blockIdx.x % a.nqt;
  const int split = blockIdx.x / a.nqt;
  if (MODE == kModeFallback && a.tflag[qt] == 0u) return;
  const int64_t t0 = a.tile_begin + (int64_t)split * a.tiles_per_split;
  const int64_t t1 = min(a.tile_end, t0 + a.tiles_per_split);
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int64_t qbase = (int64_t)qt * kTB;
  const int qrows = (int)min<int64_t>(kTB, a.nq - qbase);
  const int64_t j = qbase + wave * 32 + (lane & 31);
  const float osc = (j < a.nq) ? a.meta[j].osc : 0.0f;
  const float th = (MODE == kModeFilter && j < a.nq) ? a.thr[j] : 0.0f;
  const _Float16* QH = a.qhi + qbase * a.D;
  const _Float16* QL = a.qlo + qbase * a.D;

  float ls[MODE == kModeFilter ? 1 : KL];
  int lr[MODE == kModeFilter ? 1 : KL];
  if constexpr (MODE != kModeFilter) {
#pragma unroll
    for (int p = 0; p < KL; ++p) {
      ls[p] = -INFINITY;
      lr[p] = kNoRow;
    }
  }

  for (int64_t tile = t0; tile < t1; ++tile) {
    const int64_t rbase = tile * kTB;
    const int rows = (int)min<int64_t>(kTB, a.n - rbase);
    floatx16 acc[4];
    score_tile<B, LO>(a, rbase, rows, QH, QL, qrows, lds, acc);

    // The scale osc is positive, so the largest score is osc times the
    // largest accumulator; only a partial tile needs the row check.
    float amx = -INFINITY;
    if (rows == kTB) {
#pragma unroll
      for (int t = 0; t < 4; ++t)
#pragma unroll
        for (int r = 0; r < 16; ++r) amx = fmaxf(amx, acc[t][r]);
    } else {
#pragma unroll
      for (int t = 0; t < 4; ++t)
#pragma unroll
        for (int r = 0; r < 16; ++r) amx = (t * 32 + acc_row(r, lane) < rows) ? fmaxf(amx, acc[t][r]) : amx;
    }
    const float mx = amx * osc;
    if constexpr (MODE == kModeFilter) {
      const bool hot = j < a.nq && mx >= th;
      if (__ballot(hot) != 0ull && hot) {
        // count this lane's candidates, reserve their slots with one atomic,
        // then write them
        uint32_t c = 0u;
#pragma unroll
        for (int t = 0; t < 4; ++t)
#pragma unroll
          for (int r = 0; r < 16; ++r)
            c += (t * 32 + acc_row(r, lane) < rows && acc[t][r] * osc >= th) ? 1u : 0u;
        uint32_t idx = atomicAdd(&a.cand_cnt[j], c);
#pragma unroll
        for (int t = 0; t < 4; ++t)
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int rl_ = t * 32 + acc_row(r, lane);
            const float sc = acc[t][r] * osc;
            if (rl_ < rows && sc >= th) {
              if (idx < a.cap) {
                a.cand_s[j * a.cap + idx] = sc;
                a.cand_r[j * a.cap + idx] = (int)(rbase + rl_);
              }
              ++idx;
            }
          }
      }
      // no LDS use here: score_tile's barriers protect the slabs
    } else {
    const bool hot = mx >= ls[KL - 1];
    if (__ballot(hot) != 0ull) {
      // Park this wave's 64 scores per lane in LDS (free after the K loop) and
      // let the hot lanes walk them in a plain loop.
      float* wl = reinterpret_cast<float*>(lds) + wave * 64 * 64;
#pragma unroll
      for (int t = 0; t < 4; ++t)
#pragma unroll
        for (int r = 0; r < 16; ++r) wl[(t * 16 + r) * 64 + lane] = acc[t][r] * osc;
      if (hot) {
        for (int e = 0; e < 64; ++e) {
          const int rl_ = (e >> 4) * 32 + acc_row(e & 15, lane);
          if (rl_ >= rows) continue;
          const float sc = wl[e * 64 + lane];
          const int row = (int)(rbase + rl_);
          if (!better(sc, row, ls[KL - 1], lr[KL - 1])) continue;
          list_insert<KL>(ls, lr, sc, row);
        }
      }
    }
    __syncthreads();   // LDS is reused by the next tile's first slab
    }
  }
  if constexpr (MODE != kModeFilter) {
    if (j < a.nq) {
      const int slot = lane >> 5;
      const int64_t o = ((j * a.splits + split) * 2 + slot) * (int64_t)KL;
#pragma unroll
      for (int p = 0; p < KL; ++p) {
        a.part_s[o + p] = ls[p];
        a.part_r[o + p] = lr[p];
      }
    }
  }
  if constexpr (MODE == kModeFallback) {
    // The last of the tile's workgroups to finish merges the lists of the
    // tile's flagged queries (one wave per query), so the pass needs no merge
    // launch of its own.  Runs only for flagged tiles: the fences (release
    // of every workgroup's lists, acquire by the last) cost nothing otherwise.
    __shared__ bool last;
    __threadfence();
    __syncthreads();
    if (threadIdx.x == 0) last = atomicAdd(&a.tdone[qt], 1u) == (uint32_t)(a.splits - 1);
    __syncthreads();
    if (!last) return;
    __threadfence();
    for (int q = wave; q < qrows; q += kWG / 64) {
      const int64_t jq = qbase + q;
      if (a.qflag[jq] == 0u) continue;
      merge_query<KL, KL>(jq, a.splits * 2 * KL, a.k, a.part_s, a.part_r, a.meta, a.ids, a.out_s, a.out_i,
                          a.out_bound, nullptr);
    }
  }
}

// Fold a lane's share of candidates into a sorted register list, then take k
// rounds of the best list head of the wave under (score desc, row asc).  Rows
// are distinct, so the winning head identifies its lane.  Writes the k picks
// (ids mapped to global ids) and/or the k-th score.  The head's order is that
// of the key (order-encoded score, complement of the row): larger is better;
// scores are taken + 0.0f so that -0 and +0 are equal, as in `better`.
template <int KL>
__device__ __forceinline__ void wave_select(int k, float (&ls)[KL], int (&lr)[KL], int64_t j,
                                            const int64_t* __restrict__ ids, float* __restrict__ out_s,
                                            int64_t* __restrict__ out_i, float* __restrict__ kth,
                                            float kth_drop = 0.0f) {
  const int lane = threadIdx.x & 63;
  for (int t = 0; t < k; ++t) {
    const unsigned long long key =
        ((unsigned long long)f2ord(ls[0] + 0.0f) << 32) | (unsigned long long)(uint32_t)~(uint32_t)lr[0];
    const unsigned long long best = wave_max_u64(key);
    const float bs = ord2f((uint32_t)(best >> 32));
    const int br = (int)~(uint32_t)best;
    if (br != kNoRow && lr[0] == br) {        // this lane's head won: pop it
#pragma unroll
      for (int p = 0; p < KL - 1; ++p) {
        ls[p] = ls[p + 1];
        lr[p] = lr[p + 1];
      }
      ls[KL - 1] = -INFINITY;
      lr[KL - 1] = kNoRow;
    }
    if (lane == 0) {
      if (out_s) {
        out_s[j * k + t] = (br == kNoRow) ? -INFINITY : bs;
        out_i[j * k + t] = (br == kNoRow) ? -1 : ids[br];
      }
      if (kth && t == k - 1) kth[j] = (br == kNoRow) ? -INFINITY : rd32((double)bs - (double)kth_drop);
    }
  }
}

__device__ __forceinline__ bool write_bad(const QMeta& m, int64_t j, int k, float* out_s, int64_t* out_i,
                                          float* bound) {
  const int lane = threadIdx.x & 63;
  if (lane == 0 && bound) bound[j] = m.bound;
  if (!m.bad) return false;
  if (out_s)
    for (int t = lane; t < k; t += 64) {
      out_s[j * k + t] = __builtin_nanf("");
      out_i[j * k + t] = -1;
    }
  return true;
}

// One wave per query: the k best of the per-lane lists (segments of SEG sorted
// entries, of which only the first k can matter), each lane folding its share
// into a register list of KL.  With KL >= k and the shares' lists complete this
// is the exact k best; otherwise the k picks are still k distinct entries.
template <int KL, int SEG = KL>
__global__ __launch_bounds__(256) void k_topk_merge(int64_t nq, int cands, int k, const float* __restrict__ ps,
                                                    const int32_t* __restrict__ pr, const QMeta* __restrict__ meta,
                                                    const int64_t* __restrict__ ids, float* __restrict__ out_s,
                                                    int64_t* __restrict__ out_i, float* __restrict__ bound,
                                                    float* __restrict__ kth) {
  const int64_t j = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (j >= nq) return;
  merge_query<KL, SEG>(j, cands, k, ps, pr, meta, ids, out_s, out_i, bound, kth);
}

// One wave: the merge of query j's lists (the body of k_topk_merge).
template <int KL, int SEG>
__device__ void merge_query(int64_t j, int cands, int k, const float* __restrict__ ps,
                            const int32_t* __restrict__ pr, const QMeta* __restrict__ meta,
                            const int64_t* __restrict__ ids, float* __restrict__ out_s, int64_t* __restrict__ out_i,
                            float* __restrict__ bound, float* __restrict__ kth) {
  const int lane = threadIdx.x & 63;
  if (write_bad(meta[j], j, k, out_s, out_i, bound)) {
    if (kth && lane == 0) kth[j] = __builtin_nanf("");
    return;
  }
  const float* s = ps + j * (int64_t)cands;
  const int32_t* r = pr + j * (int64_t)cands;
  float ls[KL];
  int lr[KL];
#pragma unroll
  for (int p = 0; p < KL; ++p) {
    ls[p] = -INFINITY;
    lr[p] = kNoRow;
  }
  // a lane's next entries loaded together before any is used (one load
  // after another's test had put two round trips per entry on the path);
  // four for the sample's unsorted entries, two beside 16-entry lists
  constexpr int kU = (SEG == 1 || KL < 16) ? 4 : 2;
  for (int c0 = lane; c0 < cands; c0 += 64 * kU) {
    float cs[kU];
    int cr[kU];
#pragma unroll
    for (int u = 0; u < kU; ++u) {
      const int c = c0 + 64 * u;
      const bool in = c < cands && (c % SEG) < k;   // not below rank k of its own sorted segment
      cr[u] = in ? r[c] : kNoRow;
      cs[u] = in ? s[c] : -INFINITY;
    }
#pragma unroll
    for (int u = 0; u < kU; ++u) {
      if (cr[u] == kNoRow || !better(cs[u], cr[u], ls[KL - 1], lr[KL - 1])) continue;
      list_insert<KL>(ls, lr, cs[u], cr[u]);
    }
  }
  // the sample's k-th hi-only score, lowered by 2 err: a threshold no row of
  // the final top-k falls below in hi-only terms
  wave_select<KL>(k, ls, lr, j, ids, out_s, out_i, kth, kth ? 2.0f * meta[j].err : 0.0f);
}

// ------------------------------------------------------------------ radix selection (k > 16)
constexpr int kCandCap = 4096;   // candidate buffer entries per query
constexpr int kNoAllocMaxQ = 256;   // queries of one allocation-free scoring call

// The kth largest (1-based) of keys[0, n) in LDS, found one 8-bit digit at a
// time from the top: a histogram of the digit among keys that match the
// digits found so far, then the digit whose suffix count first reaches kth.
// Returns the key; *ties is the number of keys equal to it and *above the
// number of keys above it.  Called by the single wave of a workgroup.
__device__ uint32_t wave_kth_key(const uint32_t* keys, int n, int kth, uint32_t* hist, int* ties, int* above) {
  const int lane = threadIdx.x & 63;
  uint32_t prefix = 0u, mask = 0u;
  int need = kth, tie = 0;
  for (int shift = 24; shift >= 0; shift -= 8) {
    for (int b = lane; b < 256; b += 64) hist[b] = 0u;
    __syncthreads();   // (a workgroup of one wave)
    for (int i = lane; i < n; i += 64) {
      const uint32_t key = keys[i];
      if ((key & mask) == prefix) atomicAdd(&hist[(key >> shift) & 255u], 1u);
    }
    __syncthreads();
    // lane L holds bins 4L .. 4L + 3; suffix sums over the lanes above
    uint32_t h[4];
#pragma unroll
    for (int b = 0; b < 4; ++b) h[b] = hist[4 * lane + b];
    const uint32_t sl = h[0] + h[1] + h[2] + h[3];
    uint32_t incl = sl;
    for (int o = 1; o < 64; o <<= 1) {
      const uint32_t t = __shfl_down(incl, o);
      if (lane + o < 64) incl += t;
    }
    uint32_t acc = incl - sl;   // keys in higher bins than this lane's
    int digit = -1, rest = 0, cnt = 0;
#pragma unroll
    for (int b = 3; b >= 0; --b) {
      if (digit < 0 && acc < (uint32_t)need && acc + h[b] >= (uint32_t)need) {
        digit = 4 * lane + b;
        rest = need - (int)acc;
        cnt = (int)h[b];
      }
      acc += h[b];
    }
    const int src = __builtin_ctzll(__ballot(digit >= 0));   // exactly one lane found it
    digit = __shfl(digit, src);
    need = __shfl(rest, src);
    tie = __shfl(cnt, src);
    prefix |= (uint32_t)digit << shift;
    mask |= 255u << shift;
    __syncthreads();
  }
  *ties = tie;
  *above = kth - need;
  return prefix;
}

// One wave per query: the k best (score desc, row asc) of the candidate
// buffer, by radix selection of the kth score (and, among the scores equal to
// it, of the rows), then a bitonic sort of the k winners across the wave.
__global__ __launch_bounds__(64) void k_cand_select_radix(int64_t nq, uint32_t cap, int k,
                                                          const uint32_t* __restrict__ cnt,
                                                          const float* __restrict__ cs, const int32_t* __restrict__ cr,
                                                          const QMeta* __restrict__ meta,
                                                          const int64_t* __restrict__ ids, float* __restrict__ out_s,
                                                          int64_t* __restrict__ out_i, float* __restrict__ bound,
                                                          uint32_t* __restrict__ qflag, uint32_t* __restrict__ tflag) {
  __shared__ uint32_t keys[kCandCap];
  __shared__ uint32_t hist[256];
  __shared__ uint32_t n_win;
  __shared__ unsigned long long win[64];
  const int lane = threadIdx.x & 63;
  const int64_t j = blockIdx.x;
  if (j >= nq) return;
  const uint32_t c = cnt[j];
  const bool over = c > cap;
  if (lane == 0) {
    qflag[j] = over ? 1u : 0u;
    if (over) atomicOr(&tflag[j / kTB], 1u);
  }
  if (write_bad(meta[j], j, k, out_s, out_i, bound) || over) return;
  const float* sj = cs + j * cap;
  const int32_t* rj = cr + j * cap;
  const int n = (int)c;
  // order keys of the scores (-0 counts as +0, as in the comparison)
  for (int i = lane; i < n; i += 64) keys[i] = f2ord(sj[i] + 0.0f);
  const int kk = min(k, n);
  if (lane == 0) n_win = 0u;
  win[lane] = 0ull;
  __syncthreads();   // (a workgroup of one wave)
  if (kk > 0) {
    int ties = 0, above = 0;
    const uint32_t T = wave_kth_key(keys, n, kk, hist, &ties, &above);
    const int need_t = kk - above;    // entries equal to T to take
    // Entries above T are all taken; of those equal to T, the need_t with the
    // smallest rows: the keys become ~row for the ties (the larger, the
    // smaller the row; every tie key exceeds 0) and 0 for the rest.
    uint32_t R = 0u;
    if (need_t < ties) {
      for (int i = lane; i < n; i += 64) keys[i] = (keys[i] == T) ? ~(uint32_t)rj[i] : 0u;
      __syncthreads();
      int t2 = 0, a2 = 0;
      R = wave_kth_key(keys, n, need_t, hist, &t2, &a2);
    }
    for (int i = lane; i < n; i += 64) {
      const uint32_t ord = f2ord(sj[i] + 0.0f);
      const uint32_t row = (uint32_t)rj[i];
      const bool take = ord > T || (ord == T && (need_t >= ties || ~row >= R));
      if (take) win[atomicAdd(&n_win, 1u)] = ((unsigned long long)ord << 32) | (unsigned long long)(~row);
    }
  }
  __syncthreads();
  // bitonic sort, descending, one key per lane (empty slots hold 0)
  unsigned long long key = win[lane];
  for (int size = 2; size <= 64; size <<= 1) {
    for (int stride = size >> 1; stride > 0; stride >>= 1) {
      const unsigned long long other = __shfl_xor(key, stride);
      const bool desc = (lane & size) == 0;          // the direction of this run
      const bool lower = (lane & stride) == 0;
      key = (desc == lower) ? (key > other ? key : other) : (key < other ? key : other);
    }
  }
  if (lane < k) {
    if (lane < kk) {
      out_s[j * k + lane] = ord2f((uint32_t)(key >> 32));
      out_i[j * k + lane] = ids[~(uint32_t)(key & 0xffffffffull)];
    } else {
      out_s[j * k + lane] = -INFINITY;
      out_i[j * k + lane] = -1;
    }
  }
}

// ------------------------------------------------------------------ filter pass on the screen's pipeline
using FilterTile = Tile<2, 4, 2, 1, 4>;
// 256 x 256 (store rows x queries), sixteen waves of 64 x 64 held to 128
// registers, one workgroup per CU: half the code and query loads per flop of
// FilterTile; for the filter pass of stores with many tiles
using FilterTileL = Tile<4, 4, 2, 2, 4>;
constexpr int kFilterGroupQ = 8;   // query tiles per group in the tile order
constexpr int kSampleEntries = 4;  // entries per query and 128-row store tile of the sample pass
constexpr int64_t kFilterLargeMinTiles = 1024;   // large filter tiles from this many per launch

// The threshold plan's filter pass (hi-only scores H) for D = 64 NS: one
// C::BM x C::BN tile (store rows x queries) per workgroup, each wave 64 rows x
// 32 TJ queries (2 x TJ tiles of v_mfma_f32_32x32x16_f16); K-slabs of 64
// through two LDS stages, one barrier per slab, every load issued three slabs
// before its LDS store (SETS = 3) or one (SETS = 1, for the large tile).  For
// even code widths four threads share a row's 64-code slab (16 codes, B / 2
// whole words each), so every wave unpacks; for odd widths threads 0 to
// 2 BM - 1 take 32 codes (B words) each.  Codes are unpacked straight to fp16
// (exact for B <= 12); the queries' hi part is loaded in 16-byte pieces.  Tile
// order: groups of 8 query tiles against every store tile, query tile
// fastest, each XCD a contiguous range, so an XCD holds its query tiles in L2
// while the codes stream past.  Every row with H >= the query's threshold is
// appended to its candidate buffer, as in k_score's filter mode.
// SAMPLE (FilterTile only): the sample pass of the threshold plan over store
// tiles [0, tile_end) instead: per query and tile, the best H of each of the
// four lanes holding the query (disjoint sets of 32 rows) at entries [4 t,
// 4 t + 4) of the query's partial list.  The k-th best of these entries is the
// H of k distinct rows, so at most the sample's k-th best H: a valid base for
// the threshold (lower only where several of the best rows share a lane).
// a.nqt and a.tile_end count tiles of this kernel's size.
template <class C, int B, int NS, bool SAMPLE, int SETS>
__global__ __launch_bounds__(C::kThreads, C::kMinWaves) void k_filter(ScoreArgs a) {
  static_assert(!SAMPLE || (C::BM == kTB && C::TJ == 1), "the sample pass runs on 128-row tiles of one query block");
  static_assert(SETS == 1 || SETS == 3, "one or three register sets");
  __shared__ _Float16 lds[C::kLdsHalves];
  const int64_t nt = a.tile_end;   // store tiles of this pass (tile_begin = 0)
  // 32-bit index arithmetic: the host keeps the grid (nqt * nt) below 2^31
  const uint32_t logical = (uint32_t)xcd_remap32((int)blockIdx.x, (int)(a.nqt * nt));
  const uint32_t per = (uint32_t)(kFilterGroupQ * nt);
  const uint32_t g = logical / per;
  const uint32_t l = logical - g * per;
  const uint32_t gsize = (uint32_t)min(kFilterGroupQ, a.nqt - (int)g * kFilterGroupQ);
  const int qt = (int)(g * kFilterGroupQ + l % gsize);
  const int64_t rbase = (int64_t)(l / gsize) * C::BM;
  const int rows = (int)min<int64_t>(C::BM, a.n - rbase);
  const int64_t qbase = (int64_t)qt * C::BN;
  const int qrows = (int)min<int64_t>(C::BN, a.nq - qbase);
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / C::WN, wn = wave % C::WN;
  // this lane's queries and their thresholds, loaded before the GEMM
  int64_t j[C::TJ];
  bool jv[C::TJ];
  float th[C::TJ], osc[C::TJ];
#pragma unroll
  for (int y = 0; y < C::TJ; ++y) {
    j[y] = qbase + wn * C::TJ * 32 + y * 32 + (lane & 31);
    jv[y] = j[y] < a.nq;
    th[y] = (jv[y] && !SAMPLE) ? a.thr[j[y]] : 0.0f;
    osc[y] = jv[y] ? a.meta[j[y]].osc : 0.0f;
  }

  auto sa = [&](int i) -> _Float16* { return lds + i * ((C::BM + C::BN) * kLdk); };
  auto sb = [&](int i) -> _Float16* { return lds + i * ((C::BM + C::BN) * kLdk) + C::BM * kLdk; };
  floatx16 acc[C::TI][C::TJ];
#pragma unroll
  for (int x = 0; x < C::TI; ++x)
#pragma unroll
    for (int y = 0; y < C::TJ; ++y)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[x][y][r] = 0.0f;
  const __amdgpu_buffer_rsrc_t rsC = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint32_t*>(a.codes + rbase * a.row_words), (short)0, (int)(rows * a.row_words * 4), 0x00020000);
  const __amdgpu_buffer_rsrc_t rsQ = tile_rsrc(a.qhi + qbase * a.D, qrows, a.D);
  // Code unpacking: for even widths every thread takes 16 codes of its row's
  // 64-code slab (B / 2 whole words: a quarter of the row), so all waves
  // share it; for odd widths threads 0 to 2 BM - 1 take 32 codes (B words)
  // each.  (With half the waves unpacking, the other half waited at every
  // slab's barrier.)
  constexpr bool kQuarter = (B % 2) == 0;
  constexpr int kNW = kQuarter ? B / 2 : B;   // code words per thread and slab
  constexpr int kNC = kQuarter ? 16 : 32;     // codes per thread and slab
  static_assert(!kQuarter || C::kThreads == 4 * C::BM, "four threads per row");
  static_assert(C::kThreads >= 2 * C::BM, "two threads per row for odd widths");
  const int urow = kQuarter ? tid >> 2 : tid >> 1;
  const int upart = kQuarter ? tid & 3 : tid & 1;
  const bool unpacker = kQuarter || tid < 2 * C::BM;
  auto load = [&](int s, uint32_t (&cw)[kNW], uint4 (&qv)[C::kPerB]) {
    const int k0 = s * kBK;
    const bool ok = unpacker && urow < rows && k0 < a.D;
    const uint32_t w0 = (uint32_t)(urow * a.row_words + (int64_t)(k0 / 32) * B + upart * kNW);
    load_group<kNW>(rsC, ok, w0, cw);
    slab_load_n<C::kPerB>(rsQ, qrows, a.D, k0, a.D, qv, C::kThreads);
  };
  auto store = [&](int st, const uint32_t (&cw)[kNW], const uint4 (&qv)[C::kPerB]) {
    if (unpacker) {
      _Float16 h[kNC];
      unpack_codes<B, kNC>(cw, h);
      _Float16* dst = sa(st) + urow * kLdk + upart * kNC;
#pragma unroll
      for (int i = 0; i < kNC; i += 8) *reinterpret_cast<uint4*>(dst + i) = *reinterpret_cast<const uint4*>(h + i);
    }
    slab_store_n<C::kPerB>(sb(st), qv, C::kThreads);
  };
  auto compute = [&](int st) {
#pragma unroll
    for (int kk = 0; kk < kBK / 16; ++kk) {
      half8 fa[C::TI], fb[C::TJ];
#pragma unroll
      for (int t = 0; t < C::TI; ++t) fa[t] = frag_load(sa(st), wm * C::TI * 32 + t * 32, kk);
#pragma unroll
      for (int t = 0; t < C::TJ; ++t) fb[t] = frag_load(sb(st), wn * C::TJ * 32 + t * 32, kk);
#pragma unroll
      for (int x = 0; x < C::TI; ++x)
#pragma unroll
        for (int y = 0; y < C::TJ; ++y)
          acc[x][y] = __builtin_amdgcn_mfma_f32_32x32x16_f16(fa[x], fb[y], acc[x][y], 0, 0, 0);
    }
  };
  if constexpr (SETS == 3) {
    uint32_t cw[3][kNW];
    uint4 qv[3][C::kPerB];
#pragma unroll
    for (int u = 0; u < 3; ++u) load(u, cw[u], qv[u]);
    store(0, cw[0], qv[0]);
    load(3, cw[0], qv[0]);
    __syncthreads();
#pragma unroll
    for (int s = 0; s < NS; ++s) {
      compute(s & 1);
      if (s + 1 < NS) {
        const int u = (s + 1) % 3;
        store((s + 1) & 1, cw[u], qv[u]);
        load(s + 4, cw[u], qv[u]);   // past the last slab: zeros, no memory touched
      }
      __syncthreads();
    }
  } else {
    uint32_t cw[kNW];
    uint4 qv[C::kPerB];
    load(0, cw, qv);
    store(0, cw, qv);
    load(1, cw, qv);
    __syncthreads();
#pragma unroll
    for (int s = 0; s < NS; ++s) {
      compute(s & 1);
      if (s + 1 < NS) {
        store((s + 1) & 1, cw, qv);
        if (s + 2 < NS) load(s + 2, cw, qv);
      }
      __syncthreads();
    }
  }
  if constexpr (SAMPLE) {
    // this lane's best H over its 32 rows (the lowest row among equals)
    float best = -INFINITY;
    int brow = kNoRow;
#pragma unroll
    for (int x = 0; x < C::TI; ++x)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int rl_ = wm * 64 + x * 32 + acc_row(r, lane);   // ascending in (x, r)
        const float sc = acc[x][0][r] * osc[0];
        const bool take = rl_ < rows && sc > best;
        best = take ? sc : best;
        brow = take ? (int)(rbase + rl_) : brow;
      }
    if (jv[0]) {
      const int64_t o = j[0] * (nt * kSampleEntries) + (rbase / kTB) * kSampleEntries + wm * 2 + (lane >> 5);
      a.part_s[o] = best;
      a.part_r[o] = brow;
    }
    return;
  }
  // a tile whose store rows are all valid needs no per-element row test
  const bool full = rows == C::BM;
#pragma unroll
  for (int y = 0; y < C::TJ; ++y) {
    // epilogue: the tile's largest raw accumulator first (osc > 0)
    float amx = -INFINITY;
    if (full) {
#pragma unroll
      for (int x = 0; x < C::TI; ++x)
#pragma unroll
        for (int r = 0; r < 16; ++r) amx = fmaxf(amx, acc[x][y][r]);
    } else {
#pragma unroll
      for (int x = 0; x < C::TI; ++x)
#pragma unroll
        for (int r = 0; r < 16; ++r)
          amx = (wm * C::TI * 32 + x * 32 + acc_row(r, lane) < rows) ? fmaxf(amx, acc[x][y][r]) : amx;
    }
    const bool hot = jv[y] && amx * osc[y] >= th[y];
    if (__ballot(hot) == 0ull || !hot) continue;
    uint32_t c = 0u;
#pragma unroll
    for (int x = 0; x < C::TI; ++x)
#pragma unroll
      for (int r = 0; r < 16; ++r)
        c += (wm * C::TI * 32 + x * 32 + acc_row(r, lane) < rows && acc[x][y][r] * osc[y] >= th[y]) ? 1u : 0u;
    uint32_t idx = atomicAdd(&a.cand_cnt[j[y]], c);
#pragma unroll
    for (int x = 0; x < C::TI; ++x)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int rl_ = wm * C::TI * 32 + x * 32 + acc_row(r, lane);
        const float sc = acc[x][y][r] * osc[y];
        if (rl_ < rows && sc >= th[y]) {
          if (idx < a.cap) {
            a.cand_s[j[y] * a.cap + idx] = sc;
            a.cand_r[j[y] * a.cap + idx] = (int)(rbase + rl_);
          }
          ++idx;
        }
      }
  }
}

// large: the filter pass on FilterTileL (a.nqt and a.tile_end in its tiles)
template <int B, bool SAMPLE>
lam_status launch_filter(int b, int D, bool large, dim3 grid, hipStream_t st, const ScoreArgs& a) {
  if (b == B) {
    if constexpr (!SAMPLE) {
      if (large) {
        if (D == 768)
          hipLaunchKernelGGL((k_filter<FilterTileL, B, 12, false, 1>), grid, dim3(FilterTileL::kThreads), 0, st, a);
        else
          hipLaunchKernelGGL((k_filter<FilterTileL, B, 16, false, 1>), grid, dim3(FilterTileL::kThreads), 0, st, a);
        LAM_HIP(hipGetLastError());
        return LAM_OK;
      }
    }
    if (D == 768) hipLaunchKernelGGL((k_filter<FilterTile, B, 12, SAMPLE, 3>), grid, dim3(FilterTile::kThreads), 0, st, a);
    else hipLaunchKernelGGL((k_filter<FilterTile, B, 16, SAMPLE, 3>), grid, dim3(FilterTile::kThreads), 0, st, a);
    LAM_HIP(hipGetLastError());
    return LAM_OK;
  }
  if constexpr (B < 12) return launch_filter<B + 1, SAMPLE>(b, D, large, grid, st, a);
  set_error("scoring supports codes of at most 12 bits (got %d)", b);
  return LAM_ESTATE;
}

// ------------------------------------------------------------------ rescoring
constexpr int kRescoreCap = 256;     // candidates near the k-th score rescored per query
constexpr int kRescoreThreads = 256;
constexpr int kRescoreLanes = 8;     // lanes per rescored row

// The rescoring of m rows (in LDS) of query j from the codes and the float32
// query, summed in binary64 and rounded once, and a bitonic sort of the keys
// (score desc, row asc); the kk best go to the outputs.
template <int B>
__device__ __forceinline__ void rescore_sort(int64_t j, uint32_t m, int kk, int k, const int32_t* rows,
                                             unsigned long long* keys, const int64_t* __restrict__ ids,
                                             const float* __restrict__ q, double step,
                                             const uint32_t* __restrict__ codes, int64_t row_words, int D,
                                             float* __restrict__ out_s, int64_t* __restrict__ out_i) {
  const int tid = threadIdx.x;
  const float* qj = q + j * D;
  const int slot = tid / kRescoreLanes, sl = tid % kRescoreLanes;
  const int ngroups = D / 32;
  for (uint32_t t0 = 0; t0 < m; t0 += kRescoreThreads / kRescoreLanes) {
    const uint32_t t = t0 + (uint32_t)slot;
    double acc = 0.0;
    if (t < m) {
      const uint32_t* w = codes + (int64_t)rows[t] * row_words;
      for (int g = sl; g < ngroups; g += kRescoreLanes) {
        uint32_t cw[B];
#pragma unroll
        for (int i = 0; i < B; ++i) cw[i] = w[g * B + i];
        float qv[32];
#pragma unroll
        for (int e = 0; e < 32; ++e) qv[e] = qj[g * 32 + e];
        _Float16 h[32];
        unpack32<B>(cw, h);
#pragma unroll
        for (int e = 0; e < 32; ++e) acc = fma((double)qv[e], (double)(float)h[e], acc);
      }
    }
    for (int o = kRescoreLanes / 2; o > 0; o >>= 1) acc += __shfl_xor(acc, o);   // within the row's lanes
    if (t < m && sl == 0)
      keys[t] = ((unsigned long long)f2ord((float)(acc * step) + 0.0f) << 32) | (unsigned long long)(~(uint32_t)rows[t]);
  }
  // bitonic sort of the m keys, descending (score, then ~row); padding keys 0
  uint32_t P = 1u;
  while (P < m) P <<= 1;
  for (uint32_t i = m + tid; i < P; i += kRescoreThreads) keys[i] = 0ull;
  __syncthreads();
  for (uint32_t size = 2; size <= P; size <<= 1) {
    for (uint32_t stride = size >> 1; stride > 0; stride >>= 1) {
      for (uint32_t i = tid; i < P; i += kRescoreThreads) {
        const uint32_t l = i ^ stride;
        if (l > i) {
          const unsigned long long x = keys[i], y = keys[l];
          const bool desc = (i & size) == 0;
          if (desc ? (x < y) : (x > y)) {
            keys[i] = y;
            keys[l] = x;
          }
        }
      }
      __syncthreads();
    }
  }
  for (int t = tid; t < kk; t += kRescoreThreads) {
    out_s[j * k + t] = ord2f((uint32_t)(keys[t] >> 32));
    out_i[j * k + t] = ids[~(uint32_t)(keys[t] & 0xffffffffull)];
  }
}

// One workgroup per query, after the selection of the k best hi-only scores H
// among the candidates.  With h_k the k-th of them, every row of the final
// top-k has H >= h_k - 2 err (k rows have S >= h_k - err, and |H - S| <= err),
// so those candidates are rescored from the codes and the float32 query,
// summed in binary64 and rounded once to float32, and the k best by (S desc,
// row asc) replace the selection's output.  More than kRescoreCap such
// candidates (many near-equal scores) flag the query for the exact fallback
// pass.  Queries already flagged, or invalid, are left as the selection wrote
// them.  Eight lanes share a row (32 rows in flight per workgroup); a lane
// takes whole groups of 32 codes (B words), unpacked as the scoring kernel
// unpacks them (exactly, to fp16).
template <int B>
__global__ __launch_bounds__(kRescoreThreads) void k_rescore(
    int64_t nq, uint32_t cap, int k, const uint32_t* __restrict__ cnt, const float* __restrict__ cs,
    const int32_t* __restrict__ cr, const QMeta* __restrict__ meta, const int64_t* __restrict__ ids,
    const float* __restrict__ q, double step, const uint32_t* __restrict__ codes, int64_t row_words, int D,
    float* __restrict__ out_s, int64_t* __restrict__ out_i, uint32_t* __restrict__ qflag,
    uint32_t* __restrict__ tflag) {
  __shared__ int32_t rows[kRescoreCap];
  __shared__ unsigned long long keys[kRescoreCap];
  __shared__ uint32_t m_sh;
  const int tid = threadIdx.x;
  const int64_t j = blockIdx.x;
  if (j >= nq) return;
  const QMeta mj = meta[j];
  if (qflag[j] != 0u || mj.bad) return;
  const uint32_t c = cnt[j];
  const int kk = (int)min((uint32_t)k, c);
  if (kk == 0) return;
  const float thr = rd32((double)out_s[j * k + kk - 1] - 2.0 * (double)mj.err);
  if (tid == 0) m_sh = 0u;
  __syncthreads();
  for (uint32_t i = tid; i < c; i += kRescoreThreads) {
    if (cs[j * cap + i] >= thr) {
      const uint32_t p = atomicAdd(&m_sh, 1u);
      if (p < (uint32_t)kRescoreCap) rows[p] = cr[j * cap + i];
    }
  }
  __syncthreads();
  const uint32_t m = m_sh;
  if (m > (uint32_t)kRescoreCap) {
    if (tid == 0) {
      qflag[j] = 1u;
      atomicOr(&tflag[j / kTB], 1u);
    }
    return;
  }
  rescore_sort<B>(j, m, kk, k, rows, keys, ids, q, step, codes, row_words, D, out_s, out_i);
}

// The selection and the rescoring in one workgroup per query (k <= 16):
// wave 0 finds the k-th best hi-only score H among the candidates (per-lane
// lists of 16, then k rounds of the wave's best head as in wave_select, only
// the last one kept), and the workgroup then rescores the candidates within
// 2 err of it as k_rescore does.  Also does the selection's other work:
// flags an overflowed buffer, writes the bound, NaN outputs for an invalid
// query, and (-inf, -1) past the candidates.
template <int B>
__global__ __launch_bounds__(kRescoreThreads) void k_select_rescore(
    int64_t nq, uint32_t cap, int k, const uint32_t* __restrict__ cnt, const float* __restrict__ cs,
    const int32_t* __restrict__ cr, const QMeta* __restrict__ meta, const int64_t* __restrict__ ids,
    const float* __restrict__ q, double step, const uint32_t* __restrict__ codes, int64_t row_words, int D,
    float* __restrict__ out_s, int64_t* __restrict__ out_i, float* __restrict__ bound, uint32_t* __restrict__ qflag,
    uint32_t* __restrict__ tflag) {
  constexpr int KL = 16;
  __shared__ int32_t rows[kRescoreCap];
  __shared__ unsigned long long keys[kRescoreCap];
  __shared__ uint32_t m_sh;
  __shared__ float thr_sh;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int64_t j = blockIdx.x;
  if (j >= nq) return;
  const uint32_t c = cnt[j];
  const QMeta mj = meta[j];
  const bool over = c > cap;
  if (tid == 0) {
    qflag[j] = over ? 1u : 0u;
    if (over) atomicOr(&tflag[j / kTB], 1u);
    if (bound) bound[j] = mj.bound;
  }
  if (mj.bad) {
    for (int t = tid; t < k; t += kRescoreThreads) {
      out_s[j * k + t] = __builtin_nanf("");
      out_i[j * k + t] = -1;
    }
    return;
  }
  if (over) return;   // the exact fallback redoes the query
  const int kk = (int)min((uint32_t)k, c);
  for (int t = kk + tid; t < k; t += kRescoreThreads) {   // fewer candidates than k
    out_s[j * k + t] = -INFINITY;
    out_i[j * k + t] = -1;
  }
  if (kk == 0) return;
  // every thread's first two candidates for the threshold test below, loaded
  // while wave 0 selects
  float fs[2];
  int fr[2];
#pragma unroll
  for (int u = 0; u < 2; ++u) {
    const uint32_t i = (uint32_t)(tid + u * kRescoreThreads);
    fs[u] = i < c ? cs[j * cap + i] : 0.0f;
    fr[u] = i < c ? cr[j * cap + i] : 0;
  }
  if (wave == 0) {
    float ls[KL];
    int lr[KL];
#pragma unroll
    for (int p = 0; p < KL; ++p) {
      ls[p] = -INFINITY;
      lr[p] = kNoRow;
    }
    // a lane's first kPre candidates are loaded before any is inserted
    constexpr int kPre = 8;
    float ps[kPre];
    int pr[kPre];
#pragma unroll
    for (int u = 0; u < kPre; ++u) {
      const uint32_t i = (uint32_t)(lane + u * 64);
      ps[u] = i < c ? cs[j * cap + i] : 0.0f;
      pr[u] = i < c ? cr[j * cap + i] : 0;
    }
#pragma unroll
    for (int u = 0; u < kPre; ++u)
      if ((uint32_t)(lane + u * 64) < c && better(ps[u], pr[u], ls[KL - 1], lr[KL - 1]))
        list_insert<KL>(ls, lr, ps[u], pr[u]);
    for (uint32_t i = lane + kPre * 64; i < c; i += 64) {
      const int row = cr[j * cap + i];
      const float sc = cs[j * cap + i];
      if (!better(sc, row, ls[KL - 1], lr[KL - 1])) continue;
      list_insert<KL>(ls, lr, sc, row);
    }
    float hk = -INFINITY;
    for (int t = 0; t < kk; ++t) {
      const unsigned long long key =
          ((unsigned long long)f2ord(ls[0] + 0.0f) << 32) | (unsigned long long)(uint32_t)~(uint32_t)lr[0];
      const unsigned long long best = wave_max_u64(key);
      const int br = (int)~(uint32_t)best;
      hk = ord2f((uint32_t)(best >> 32));
      if (br != kNoRow && lr[0] == br) {
#pragma unroll
        for (int p = 0; p < KL - 1; ++p) {
          ls[p] = ls[p + 1];
          lr[p] = lr[p + 1];
        }
        ls[KL - 1] = -INFINITY;
        lr[KL - 1] = kNoRow;
      }
    }
    if (lane == 0) {
      thr_sh = rd32((double)hk - 2.0 * (double)mj.err);
      m_sh = 0u;
    }
  }
  __syncthreads();
  const float thr = thr_sh;
#pragma unroll
  for (int u = 0; u < 2; ++u) {
    if ((uint32_t)(tid + u * kRescoreThreads) < c && fs[u] >= thr) {
      const uint32_t p = atomicAdd(&m_sh, 1u);
      if (p < (uint32_t)kRescoreCap) rows[p] = fr[u];
    }
  }
  for (uint32_t i = tid + 2 * kRescoreThreads; i < c; i += kRescoreThreads) {
    if (cs[j * cap + i] >= thr) {
      const uint32_t p = atomicAdd(&m_sh, 1u);
      if (p < (uint32_t)kRescoreCap) rows[p] = cr[j * cap + i];
    }
  }
  __syncthreads();
  const uint32_t m = m_sh;
  if (m > (uint32_t)kRescoreCap) {
    if (tid == 0) {
      qflag[j] = 1u;
      atomicOr(&tflag[j / kTB], 1u);
    }
    return;
  }
  rescore_sort<B>(j, m, kk, k, rows, keys, ids, q, step, codes, row_words, D, out_s, out_i);
}

// Lists and fallback give final scores (hi and lo); the filter pass works on
// hi-only scores.
template <int B, int KL>
void launch_mode(int mode, dim3 grid, hipStream_t st, const ScoreArgs& a) {
  if (mode == kModeLists) hipLaunchKernelGGL((k_score<B, KL, kModeLists, true>), grid, dim3(kWG), 0, st, a);
  else if (mode == kModeFilter) hipLaunchKernelGGL((k_score<B, KL, kModeFilter, false>), grid, dim3(kWG), 0, st, a);
  else hipLaunchKernelGGL((k_score<B, KL, kModeFallback, true>), grid, dim3(kWG), 0, st, a);
}

template <int B>
lam_status dispatch_bits(int b, int kl, int mode, dim3 grid, hipStream_t st, const ScoreArgs& a) {
  if (b == B) {
    if (kl == 4) {   // the sample pass: short lists of hi-only scores
      if (mode != kModeLists) {
        set_error("internal: lists of 4 serve the sample pass only");
        return LAM_EINVAL;
      }
      hipLaunchKernelGGL((k_score<B, 4, kModeLists, false>), grid, dim3(kWG), 0, st, a);
    } else if (kl == 16) launch_mode<B, 16>(mode, grid, st, a);
    else launch_mode<B, 64>(mode, grid, st, a);
    return LAM_OK;
  }
  if constexpr (B < 12) return dispatch_bits<B + 1>(b, kl, mode, grid, st, a);
  set_error("scoring supports codes of at most 12 bits (got %d)", b);
  return LAM_ESTATE;
}

// The rescoring after the radix selection (k > 16), or the fused selection
// and rescoring (k <= 16, fused = true; bound written there too).
template <int B>
lam_status launch_rescore(int b, bool fused, dim3 grid, hipStream_t st, int64_t nq, uint32_t cap, int k,
                          const uint32_t* cnt, const float* cs, const int32_t* cr, const QMeta* meta,
                          const int64_t* ids, const float* q, double step, const uint32_t* codes, int64_t row_words,
                          int D, float* out_s, int64_t* out_i, float* bound, uint32_t* qflag, uint32_t* tflag) {
  if (b == B) {
    if (fused)
      hipLaunchKernelGGL((k_select_rescore<B>), grid, dim3(kRescoreThreads), 0, st, nq, cap, k, cnt, cs, cr, meta,
                         ids, q, step, codes, row_words, D, out_s, out_i, bound, qflag, tflag);
    else
      hipLaunchKernelGGL((k_rescore<B>), grid, dim3(kRescoreThreads), 0, st, nq, cap, k, cnt, cs, cr, meta, ids, q,
                         step, codes, row_words, D, out_s, out_i, qflag, tflag);
    LAM_HIP(hipGetLastError());
    return LAM_OK;
  }
  if constexpr (B < 12)
    return launch_rescore<B + 1>(b, fused, grid, st, nq, cap, k, cnt, cs, cr, meta, ids, q, step, codes, row_words, D,
                                 out_s, out_i, bound, qflag, tflag);
  set_error("scoring supports codes of at most 12 bits (got %d)", b);
  return LAM_ESTATE;
}

// Split a tile range over query tiles so that the grid holds about 1024
// workgroups; returns (splits, tiles per split).
void plan_splits(int nqt, int64_t ntiles, int* splits, int64_t* tps, int max_splits) {
  if (ntiles <= 0) {
    *splits = 1;
    *tps = 0;
    return;
  }
  const int64_t want = std::min<int64_t>(max_splits, std::max<int64_t>(1, (1024 + nqt - 1) / nqt));
  int64_t s = std::min<int64_t>(want, ntiles);
  const int64_t t = (ntiles + s - 1) / s;
  *tps = t;
  *splits = (int)((ntiles + t - 1) / t);
}

// ---- codes of 13 to 22 bits
// A code c of b bits is 2^11 (c >> 11) + (c & 2047) with |c >> 11| <= 2^(b-12)
// <= 1,024 and 0 <= c & 2047 <= 2,047: both parts are 12-bit codes, exact in
// fp16.  The split store has 2D columns, column d holding c_d >> 11 and column
// D + d holding c_d & 2047; a query q becomes [2^11 q, q] (exact scalings), so
// that s sum_d' q'_d' code'_d' = s sum_d q_d code_d term by term.
constexpr int kWideMaxBits = 22;
constexpr int kWideShift = 11;

// One thread per 32 columns of a split row (12 words of 12-bit codes).
__global__ __launch_bounds__(256) void k_wide_codes(const uint32_t* __restrict__ src, int64_t n, int D, int b,
                                                    uint32_t* __restrict__ dst) {
  const int G = 2 * D / 32;   // groups of 32 split columns per row
  const int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (t >= n * G) return;
  const int64_t row = t / G;
  const int g = (int)(t - row * G);
  const bool low = g >= D / 32;
  const int d0 = (low ? g - D / 32 : g) * 32;
  const uint32_t* w = src + row * ((int64_t)D * b / 32);
  uint32_t o[12];
#pragma unroll
  for (int i = 0; i < 12; ++i) o[i] = 0u;
#pragma unroll
  for (int e = 0; e < 32; ++e) {
    const int64_t bit = (int64_t)(d0 + e) * b;
    const int wi = (int)(bit >> 5), off = (int)(bit & 31);
    uint32_t u = w[wi] >> off;
    if (off + b > 32) u |= w[wi + 1] << (32 - off);   // the code's bits lie inside the row
    const int32_t c = (int32_t)(u << (32 - b)) >> (32 - b);
    const uint32_t v = (uint32_t)(low ? (c & ((1 << kWideShift) - 1)) : (c >> kWideShift)) & 0xfffu;
    const int ob = e * 12, ow = ob >> 5, oo = ob & 31;
    o[ow] |= v << oo;
    if (oo + 12 > 32) o[ow + 1] |= v >> (32 - oo);
  }
  uint32_t* out = dst + row * ((int64_t)2 * D * 12 / 32) + (int64_t)g * 12;
#pragma unroll
  for (int i = 0; i < 12; ++i) out[i] = o[i];
}

// q' = [2^11 q, q], one thread per element.
__global__ __launch_bounds__(256) void k_wide_queries(const float* __restrict__ q, int64_t nq, int D,
                                                      float* __restrict__ qw) {
  const int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (t >= nq * 2 * D) return;
  const int64_t j = t / (2 * D);
  const int d = (int)(t - j * 2 * D);
  qw[t] = d < D ? q[j * D + d] * (float)(1 << kWideShift) : q[j * D + d - D];
}

}  // namespace

// What the scoring passes read of a store: its coded rows (D columns of b-bit
// codes, step s = 2 eps), their ids, R >= s ||code_y|| for every row y, and
// the first column counted in the reported bound.
struct ScoreView {
  int D;
  int b;
  int64_t n;
  double step;
  double eps;
  double R;
  int l1_from;
  const uint32_t* codes;
  const int64_t* ids;
};

namespace {

// R >= ||x_hat_y||: ||x|| from the largest ||x||^2 / 2 of the coded rows
// (float32, rounded up by one part in 2^22) plus ||x_hat - x|| <= eps sqrt(D).
double row_norm_bound(uint32_t hn_max_bits, double eps, int D) {
  float hn;
  std::memcpy(&hn, &hn_max_bits, 4);
  return std::sqrt(2.0 * (double)hn * (1.0 + 0x1p-22)) * (1.0 + 0x1p-50) +
         eps * std::sqrt((double)D) * (1.0 + 0x1p-50);
}

ScoreView store_view(const lam_store* st, const uint32_t* codes) {
  ScoreView v;
  v.D = st->dim;
  v.b = st->q.bits;
  v.n = st->size;
  v.step = st->q.step;
  v.eps = st->q.eps;
  v.R = row_norm_bound(st->hn_max, st->q.eps, st->dim);
  v.l1_from = 0;
  v.codes = codes ? codes : st->codes;
  v.ids = st->ids;
  return v;
}

// The split form of a store with wide codes and of the queries, in the
// context's arena.  With |c >> 11| <= ||c|| / 2^11 + 1 per column and
// c & 2047 <= 2,047, s ||code'|| <= R / 2^11 + 2^12 eps sqrt(D).
lam_status widen(lam_ctx* ctx, ScoreView& v, const float*& q, int64_t nq) {
  LAM_CHECK(v.b <= kWideMaxBits, LAM_ESTATE,
            "scoring supports codes of at most %d bits (store codes have %d); quantize with a larger eps",
            kWideMaxBits, v.b);
  const int D = v.D;
  LAM_TRY(ctx->scratch[kScratchWideCodes].ensure(std::max<size_t>((size_t)v.n * 2 * D * 12 / 8, 4)));
  LAM_TRY(ctx->scratch[kScratchWideQueries].ensure(std::max<size_t>((size_t)nq * 2 * D * 4, 4)));
  uint32_t* wc = ctx->scratch[kScratchWideCodes].as<uint32_t>();
  float* wq = ctx->scratch[kScratchWideQueries].as<float>();
  const int64_t ng = v.n * (2 * D / 32);
  if (ng > 0) {
    hipLaunchKernelGGL(k_wide_codes, dim3((unsigned)((ng + 255) / 256)), dim3(256), 0, ctx->stream, v.codes, v.n, D,
                       v.b, wc);
    LAM_HIP(hipGetLastError());
  }
  const int64_t ne = nq * 2 * D;
  if (ne > 0) {
    hipLaunchKernelGGL(k_wide_queries, dim3((unsigned)((ne + 255) / 256)), dim3(256), 0, ctx->stream, q, nq, D, wq);
    LAM_HIP(hipGetLastError());
  }
  v.R = (v.R * 0x1p-11 + 4096.0 * v.eps * std::sqrt((double)D) * (1.0 + 0x1p-50)) * (1.0 + 0x1p-50);
  v.D = 2 * D;
  v.b = 12;
  v.l1_from = D;
  v.codes = wc;
  q = wq;
  return LAM_OK;
}

}  // namespace

// Scoring plan.  With at most S store rows (S = k * n / 1024, at least 4,096)
// one pass of per-lane lists gives the exact top-k.  Beyond that (H: scores
// of the hi part alone, within err of the rescored scores S):
//   1. theta_j, the k-th best H of per-lane lists of the 4 best H over the
//      first S rows, minus 2 err_j: k distinct rows have S >= theta_j + err_j,
//      so every row of the final top-k has H >= theta_j (short lists keep
//      this pass cheap -- the insertions, not the MFMAs, dominate it -- at
//      the price of a slightly lower theta_j when one lane holds more than 4
//      of the sample's best k; the splits give at least 2k entries);
//   2. a full scan of H appends every row with H >= theta_j to query j's
//      candidate buffer (about k * n / S = 1,024 entries expected; capacity
//      4,096);
//   3. the k best candidates by H; the candidates within 2 err_j of the k-th
//      of them are rescored exactly and their k best by (S desc, id asc) are
//      the answer (k_rescore);
//   4. a query whose buffer overflowed, or with more than 256 candidates to
//      rescore (many equal scores, say), is redone with exact per-lane lists
//      over the whole store; launched always, it returns at once when nothing
//      was flagged, so the call stays asynchronous.
namespace {

// Scratch of one scoring call: the context's arena (grown on demand), or a
// fixed region carved in order (the allocation-free entry point).
struct ScoreWork {
  char* base = nullptr;   // fixed region; nullptr: the context arena
  size_t bytes = 0;
  size_t used = 0;
  template <class T>
  lam_status take(lam_ctx* ctx, int slot, size_t need, T** out) {
    if (!base) {
      LAM_TRY(ctx->scratch[slot].ensure(need));
      *out = ctx->scratch[slot].as<T>();
      return LAM_OK;
    }
    const size_t at = (used + 255) & ~(size_t)255;
    LAM_CHECK(at + need <= bytes, LAM_ECAPACITY,
              "scoring needs more than the %zu bytes of the fixed workspace", bytes);
    *out = reinterpret_cast<T*>(base + at);
    used = at + need;
    return LAM_OK;
  }
};

// score_topk on the workspace w.  Every buffer is taken before the first
// launch, so a workspace that is too small fails with nothing enqueued.
// max_splits caps the store ranges per query tile of the list passes (their
// candidate lists grow with it); no profiling events are recorded unless prof.
lam_status score_topk_impl(lam_ctx* ctx, const ScoreView& st, const float* q, int64_t nq, int32_t k, float* scores,
                           int64_t* ids, float* bound, ScoreWork& w, int max_splits, bool prof) {
  if (nq == 0) return LAM_OK;
  const int D = st.D;
  const int b = st.b;
  LAM_CHECK(b >= 1 && b <= 12, LAM_ESTATE, "internal: the scoring passes take codes of 1 to 12 bits (got %d)", b);
  const int KL = (k <= 16) ? 16 : 64;
  const int64_t n = st.n;
  const int nqt = (int)((nq + kTB - 1) / kTB);
  const int64_t ntiles = (n + kTB - 1) / kTB;
  // the sample: the store's first max(4,096, k n / 256) rows, so that at
  // most about k n / sample = 256 rows per query pass the filter (a sample of
  // k n / 1,024 rows let about 1,024 through: the corpus call 2.65-2.71 ->
  // 2.57-2.59 ms, 60 K rows at top-50 265 -> 238 us; k n / 128 was no faster)
  const int64_t sample_rows = std::max<int64_t>(4096, ((int64_t)k * n + 255) / 256);
  const int64_t stiles = std::min<int64_t>(ntiles, (sample_rows + kTB - 1) / kTB);
  const bool two_pass = stiles < ntiles;

  int sp1 = 1, sp2 = 1;
  int64_t tps1 = 0, tps2 = 0;
  plan_splits(nqt, stiles, &sp1, &tps1, max_splits);
  plan_splits(nqt, ntiles, &sp2, &tps2, max_splits);
  constexpr int kSampleKL = 4;
  if (two_pass && (int64_t)sp1 * 2 * kSampleKL < 2 * (int64_t)k) {
    const int64_t want = std::min<int64_t>(stiles, (k + kSampleKL - 1) / kSampleKL);
    tps1 = (stiles + want - 1) / want;
    sp1 = (int)((stiles + tps1 - 1) / tps1);
  }
  const int cands_max = std::max(sp1, sp2) * 2 * KL;
  // the sample pass on the filter's pipeline at D = 768 and 1,024 when its
  // entries fit the partial lists' buffer
  const bool filter_sample =
      two_pass && (D == 768 || D == 1024) && stiles * kSampleEntries <= (int64_t)cands_max;
  // the filter pipeline's grids (sample and filter passes) are one workgroup
  // per (query tile, store tile), indexed in 32 bits
  LAM_CHECK(!two_pass || !(D == 768 || D == 1024) || (int64_t)nqt * ntiles < (1LL << 31), LAM_EINVAL,
            "scoring grid too large");
  const uint32_t cap = kCandCap;

  // every buffer first
  _Float16 *qhi = nullptr, *qlo = nullptr;
  QMeta* qmeta = nullptr;
  float* part_s = nullptr;
  float* cand_s = nullptr;
  LAM_TRY(w.take(ctx, S_QHI, (size_t)nq * D * 2, &qhi));
  LAM_TRY(w.take(ctx, S_QLO, (size_t)nq * D * 2, &qlo));
  LAM_TRY(w.take(ctx, S_QMETA, (size_t)nq * sizeof(QMeta), &qmeta));
  LAM_TRY(w.take(ctx, S_PART, (size_t)nq * cands_max * 8, &part_s));
  if (two_pass) LAM_TRY(w.take(ctx, S_CAND, (size_t)nq * cap * 8 + (size_t)nq * 12 + (size_t)nqt * 8 + 256, &cand_s));
  int32_t* part_r = reinterpret_cast<int32_t*>(part_s + (size_t)nq * cands_max);
  int32_t* cand_r = two_pass ? reinterpret_cast<int32_t*>(cand_s + (size_t)nq * cap) : nullptr;
  uint32_t* cand_cnt = two_pass ? reinterpret_cast<uint32_t*>(cand_r + (size_t)nq * cap) : nullptr;
  float* thr = two_pass ? reinterpret_cast<float*>(cand_cnt + nq) : nullptr;
  uint32_t* qflag = two_pass ? reinterpret_cast<uint32_t*>(thr + nq) : nullptr;
  uint32_t* tflag = two_pass ? qflag + nq : nullptr;

  {
    ProfScope ps(ctx, "score_prep", prof);
    hipLaunchKernelGGL(k_score_prep, dim3((unsigned)((nq + 3) / 4)), dim3(256), 0, ctx->stream, q, nq, D, st.step,
                       st.eps, st.R, st.l1_from, qhi, qlo, qmeta, cand_cnt, tflag);
    LAM_HIP(hipGetLastError());
  }

  ScoreArgs a{};
  a.codes = st.codes;
  a.n = n;
  a.D = D;
  a.row_words = (int64_t)D * b / 32;
  a.qhi = qhi;
  a.qlo = qlo;
  a.meta = qmeta;
  a.nq = nq;
  a.nqt = nqt;
  a.part_s = part_s;
  a.part_r = part_r;
  const dim3 gq((unsigned)((nq + 3) / 4));

  if (!two_pass) {
    if (ntiles > 0) {
      a.tile_begin = 0;
      a.tile_end = ntiles;
      a.splits = sp2;
      a.tiles_per_split = tps2;
      ProfScope ps(ctx, "score_mfma", prof);
      LAM_TRY(dispatch_bits<1>(b, KL, kModeLists, dim3((unsigned)(nqt * sp2)), ctx->stream, a));
      LAM_HIP(hipGetLastError());
    }
    ProfScope ps(ctx, "score_merge", prof);
    const int nc = ntiles > 0 ? sp2 * 2 * KL : 0;
    if (KL == 16)
      hipLaunchKernelGGL((k_topk_merge<16>), gq, dim3(256), 0, ctx->stream, nq, nc, k, part_s, part_r, qmeta, st.ids,
                         scores, ids, bound, nullptr);
    else
      hipLaunchKernelGGL((k_topk_merge<64>), gq, dim3(256), 0, ctx->stream, nq, nc, k, part_s, part_r, qmeta, st.ids,
                         scores, ids, bound, nullptr);
    LAM_HIP(hipGetLastError());
    return LAM_OK;
  }

  // (the candidate counts and tile flags were cleared by k_score_prep)
  {  // 1. a k-th best score of the sample -> thresholds
    ProfScope ps(ctx, "score_sample", prof);
    a.tile_begin = 0;
    a.tile_end = stiles;
    a.splits = sp1;
    a.tiles_per_split = tps1;
    if (filter_sample) {
      // one tile per workgroup on the filter's pipeline; entries unsorted (segments of 1)
      LAM_TRY((launch_filter<1, true>(b, D, false, dim3((unsigned)(nqt * stiles)), ctx->stream, a)));
      hipLaunchKernelGGL((k_topk_merge<16, 1>), gq, dim3(256), 0, ctx->stream, nq, (int)stiles * kSampleEntries, k,
                         part_s, part_r, qmeta, st.ids, nullptr, nullptr, nullptr, thr);
    } else {
      LAM_TRY(dispatch_bits<1>(b, kSampleKL, kModeLists, dim3((unsigned)(nqt * sp1)), ctx->stream, a));
      hipLaunchKernelGGL((k_topk_merge<16, kSampleKL>), gq, dim3(256), 0, ctx->stream, nq, sp1 * 2 * kSampleKL, k,
                         part_s, part_r, qmeta, st.ids, nullptr, nullptr, nullptr, thr);
    }
    LAM_HIP(hipGetLastError());
  }
  a.tile_begin = 0;
  a.tile_end = ntiles;
  a.splits = sp2;
  a.tiles_per_split = tps2;
  a.thr = thr;
  a.cand_s = cand_s;
  a.cand_r = cand_r;
  a.cand_cnt = cand_cnt;
  a.cap = cap;
  a.tflag = tflag;
  {  // 2. full scan with the thresholds
    ProfScope ps(ctx, "score_mfma", prof);
    if (D == 768 || D == 1024) {
      // one tile per workgroup on the screen's pipeline: 256 x 256 when the
      // launch holds many of them, else 128 x 128
      const int nqtL = (int)((nq + FilterTileL::BN - 1) / FilterTileL::BN);
      const int64_t ntilesL = (n + FilterTileL::BM - 1) / FilterTileL::BM;
      const bool large = (int64_t)nqtL * ntilesL >= kFilterLargeMinTiles;
      ScoreArgs af = a;
      if (large) {
        af.nqt = nqtL;
        af.tile_end = ntilesL;
      }
      const int64_t grid = (int64_t)af.nqt * af.tile_end;
      LAM_CHECK(grid < (1LL << 31), LAM_EINVAL, "scoring grid too large");
      LAM_TRY((launch_filter<1, false>(b, D, large, dim3((unsigned)grid), ctx->stream, af)));
    } else {
      LAM_TRY(dispatch_bits<1>(b, KL, kModeFilter, dim3((unsigned)(nqt * sp2)), ctx->stream, a));
      LAM_HIP(hipGetLastError());
    }
  }
  {  // 3. select; 4. exact fallback for overflowed buffers (returns at once otherwise)
    ProfScope ps(ctx, "score_merge", prof);
    if (KL != 16) {
      hipLaunchKernelGGL(k_cand_select_radix, dim3((unsigned)nq), dim3(64), 0, ctx->stream, nq, cap, k, cand_cnt, cand_s, cand_r,
                         qmeta, st.ids, scores, ids, bound, qflag, tflag);
      LAM_HIP(hipGetLastError());
    }
    LAM_TRY(launch_rescore<1>(b, KL == 16, dim3((unsigned)nq), ctx->stream, nq, cap, k, cand_cnt, cand_s, cand_r,
                              qmeta, st.ids, q, st.step, a.codes, a.row_words, D, scores, ids, bound, qflag, tflag));
  }
  {
    // exact lists for the flagged query tiles, merged by each tile's last
    // workgroup (returns at once when nothing is flagged)
    ProfScope ps(ctx, "score_fallback", prof);
    a.qflag = qflag;
    a.tdone = tflag + nqt;
    a.k = k;
    a.out_s = scores;
    a.out_i = ids;
    a.out_bound = bound;
    a.ids = st.ids;
    LAM_TRY(dispatch_bits<1>(b, KL, kModeFallback, dim3((unsigned)(nqt * sp2)), ctx->stream, a));
    LAM_HIP(hipGetLastError());
  }
  return LAM_OK;
}

// ------------------------------------------------------------------ allocation-free scoring
// Its scratch memory: one array per device, allocated with the code object,
// held until the process ends.  Sized for kNoAllocMaxQ queries of up to 4,096
// dimensions with at most kNoAllocSplits store ranges per query tile:
// fp16 hi and lo query parts (4 D bytes per query), the query meta block, the
// list passes' candidates (2 x 64 entries of 8 bytes per range) and the
// threshold plan's candidate buffer (kCandCap entries of 8 bytes, 12 bytes
// of counts and flags) -- 112 KB per query, 28 MB at the limits.
constexpr int kNoAllocSplits = 64;
constexpr size_t kNoAllocBytes = (size_t)32 << 20;
static_assert((size_t)kNoAllocMaxQ * (4 * 4096 + 16 + (size_t)kNoAllocSplits * 2 * 64 * 8 + (size_t)kCandCap * 8 + 12) +
                      6 * 256 + 256 <= kNoAllocBytes,
              "the workspace holds a call at the limits");

}  // namespace

static __device__ __align__(256) unsigned char scratch[kNoAllocBytes];

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_noalloc_mu;
void* g_noalloc_ptr[kMaxDevices];   // device address of `scratch` on each device (host code must not use its name)
}  // namespace

lam_status noalloc_setup(int device) {
  LAM_CHECK(device >= 0 && device < kMaxDevices, LAM_EINVAL, "device %d beyond the supported %d", device, kMaxDevices);
  std::lock_guard<std::mutex> lk(g_noalloc_mu);
  if (g_noalloc_ptr[device]) return LAM_OK;
  void* p = nullptr;
  LAM_HIP(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)));   // the current device is `device`
  g_noalloc_ptr[device] = p;
  return LAM_OK;
}

lam_status score_topk(lam_ctx* ctx, const lam_store* st, const float* q, int64_t nq, int32_t k, float* scores,
                      int64_t* ids, float* bound, const uint32_t* codes) {
  if (nq == 0) return LAM_OK;
  ScoreWork w;
  ScoreView v = store_view(st, codes);
  if (v.b > 12) LAM_TRY(widen(ctx, v, q, nq));
  return score_topk_impl(ctx, v, q, nq, k, scores, ids, bound, w, 1 << 30, true);
}

lam_status score_topk_noalloc(lam_ctx* ctx, const lam_store* st, const float* q, int64_t nq, int32_t k, float* scores,
                              int64_t* ids, float* bound) {
  LAM_CHECK(nq <= kNoAllocMaxQ, LAM_EINVAL, "the allocation-free call takes at most %d queries (asked %lld)",
            kNoAllocMaxQ, (long long)nq);
  void* p = nullptr;
  {
    std::lock_guard<std::mutex> lk(g_noalloc_mu);
    p = ctx->device < kMaxDevices ? g_noalloc_ptr[ctx->device] : nullptr;
  }
  LAM_CHECK(p != nullptr, LAM_ESTATE, "the fixed workspace of device %d was not set up", ctx->device);
  LAM_CHECK(st->q.bits <= 12, LAM_ESTATE,
            "the allocation-free call scores codes of at most 12 bits (store codes have %d)", st->q.bits);
  ScoreWork w;
  w.base = static_cast<char*>(p);
  w.bytes = kNoAllocBytes;
  return score_topk_impl(ctx, store_view(st, nullptr), q, nq, k, scores, ids, bound, w, kNoAllocSplits, false);
}

// ------------------------------------------------------------------ certificate
namespace {

// Rank-invariance certificate (Appendix "Rank invariance, in full"): one wave
// per query copies the first k of its top-(k+1) and flags the query when the
// float32 margin between ranks k and k+1 exceeds
//   2 (beta + ||q||_2 delta_hat + e),   e = kappa ||q||_1 (A + eps),
// where e bounds the float32 score's error against the exact dequantized score
// (hi/lo residual 2^-22, float32 accumulation of 2 D terms gamma_2D, output
// scaling 2^-23, all relative to sum |q_d x_hat_d| <= ||q||_1 (A + eps)).  A
// flag therefore implies that the exact margin exceeds 2 (beta + ||q||_2
// delta_hat): no record can cross the rank-k boundary when every score moves
// by at most beta + ||q||_2 delta_hat.  A store with at most k rows certifies
// every valid query (nothing can cross).
__global__ __launch_bounds__(256) void k_certify(int64_t nq, int k, const float* __restrict__ s1,
                                                 const int64_t* __restrict__ i1, const float* __restrict__ b1,
                                                 const float* __restrict__ q, int D, double eps, double dhat,
                                                 double err_per_l1, float* __restrict__ scores,
                                                 int64_t* __restrict__ ids, float* __restrict__ bound,
                                                 uint8_t* __restrict__ cert, float* __restrict__ margin) {
  const int lane = threadIdx.x & 63;
  const int64_t j = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (j >= nq) return;
  const float* p = q + j * D;
  double l1 = 0.0, l2 = 0.0;
  for (int d = lane; d < D; d += 64) {
    const double v = (double)p[d];
    l1 += fabs(v);
    l2 = fma(v, v, l2);
  }
  for (int o = 32; o > 0; o >>= 1) {
    l1 += __shfl_xor(l1, o);
    l2 += __shfl_xor(l2, o);
  }
  const int64_t o1 = j * (k + 1);
  for (int t = lane; t < k; t += 64) {
    scores[j * k + t] = s1[o1 + t];
    ids[j * k + t] = i1[o1 + t];
  }
  if (lane != 0) return;
  if (bound) bound[j] = b1[j];
  const float sk = s1[o1 + k - 1], sk1 = s1[o1 + k];
  const bool valid = !isnan(b1[j]);   // NaN bound: the query row holds NaN/Inf
  const double m = (i1[o1 + k] < 0) ? INFINITY : (double)sk - (double)sk1;
  // rounded up past its own evaluation error: the binary64 sums of D terms are
  // within (D - 1) 2^-53 relative in any order, the few products and the
  // square root add 2^-53 each
  const double thr = 2.0 * (eps * l1 + sqrt(l2) * dhat + err_per_l1 * l1) * (1.0 + (double)(D + 8) * 0x1p-52);
  cert[j] = (valid && m > thr) ? 1 : 0;
  if (margin) margin[j] = valid ? (float)m : __builtin_nanf("");
}

}  // namespace

lam_status score_certify(lam_ctx* ctx, const lam_store* st, const float* q, int64_t nq, int32_t k, float* scores,
                         int64_t* ids, float* bound, uint8_t* certified, float* margin) {
  if (nq == 0) return LAM_OK;
  const int K1 = k + 1;
  const size_t per = (size_t)K1 * (4 + 8);
  LAM_TRY(ctx->scratch[kScratchCertify].ensure((size_t)nq * per + (size_t)nq * 4 + 64));
  char* base = ctx->scratch[kScratchCertify].as<char>();
  int64_t* i1 = reinterpret_cast<int64_t*>(base);
  float* s1 = reinterpret_cast<float*>(base + (size_t)nq * K1 * 8);
  float* b1 = s1 + (size_t)nq * K1;
  LAM_TRY(score_topk(ctx, st, q, nq, K1, s1, i1, b1));
  // error bound of the float32 score per unit of ||q||_1: kappa (A + eps).
  // Wide codes are scored in their split form (2 D columns): twice the terms,
  // and sum |q'_d' x_hat'_d'| <= ||q||_1 (A + eps + 2^12 s) since
  // 2^11 |c >> 11| <= |c| + 2^11 and c & 2047 < 2^11.
  const bool wide = st->q.bits > 12;
  const double Dt = (wide ? 2.0 : 1.0) * st->dim;
  const double u = std::ldexp(1.0, -24);
  const double g2d = 2.0 * Dt * u / (1.0 - 2.0 * Dt * u);
  // (the split residual, the sums, the two scalings; a rescored score is
  // within 2^-24 relative of its binary64 sum, far inside this)
  const double kappa = 1.01 * (std::ldexp(1.0, -22) + g2d + std::ldexp(1.0, -23));
  const double mag = (double)st->q.absmax + st->q.eps + (wide ? 4096.0 * st->q.step : 0.0);
  const double err_per_l1 = kappa * mag;
  hipLaunchKernelGGL(k_certify, dim3((unsigned)((nq + 3) / 4)), dim3(256), 0, ctx->stream, nq, k, s1, i1, b1, q,
                     st->dim, st->q.eps, st->delta_hat_run, err_per_l1, scores, ids, bound, certified, margin);
  LAM_HIP(hipGetLastError());
  return LAM_OK;
}

}  // namespace lam
