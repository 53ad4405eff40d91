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
//                on exact integers on the host (a second, "careful", pass).
//   resolve   -- one wave walks the chunk in arrival order: a row with a store
//                hit is dropped; a row with no in-chunk edge is kept; any other
//                row takes its lowest earlier in-chunk neighbour that was kept,
//                using a 4096-bit kept mask held in the wave's registers.
//   append    -- kept rows join the store; for dropped rows ||x - rep||^2 in
//                binary64 feeds the measured bound delta_hat.
//
// Error bound of the screen (dot-product units), for rows a, b:
//   |c16 - a.b| <= K1 (||a||^2 + ||b||^2)/2 + K2 (||a||_1 + ||b||_1) + K3
// from fp16 input rounding (relative 2^-11, or 2^-22 absolute for scaled
// subnormals even if flushed), exact fp16 products in fp32, and fp32
// accumulation in any order (gamma_D with 2u per addition); the AM-GM step
// ||a|| ||b|| <= (||a||^2 + ||b||^2)/2 makes it a sum of per-row terms, and the
// per-row term also absorbs the float32 roundings of the epilogue.
#include <cmath>
#include <cstring>
#include <vector>

#include "lam_internal.h"
#include "mfma_tile.h"

namespace lam {

namespace {

constexpr int kChunk = 4096;           // rows per resolve (64 lanes x 64 bits)
constexpr int kNone = 0x7fffffff;       // "no store hit"
constexpr float kScale = 256.0f;        // fp16 operands hold x * 2^8
constexpr float kInvScale2 = 1.0f / 65536.0f;

enum Scratch { S_X16 = 0, S_ROWF, S_CHUNK, S_BITMAP, S_PAIRS, S_STATUS, S_G };

struct StoreMeta {
  int32_t m;              // retained rows
  uint32_t ebmax_bits;    // max per-row error term over retained rows (float bits)
  uint32_t l2max_bits;
  uint32_t pad;
};

// Chunk-level counters (in the S_CHUNK scratch, after the per-row arrays).
struct ChunkCounters {
  uint32_t npairs;        // ambiguous pairs appended in this chunk
  uint32_t ebmax_bits;    // max error term over the chunk's rows (batch side)
  uint32_t n_escalate;
  uint32_t pad;
};

__device__ __forceinline__ bool skip_all(const DevFlags* f) {
  return (f->nonfinite | f->out_of_range | f->pair_overflow) != 0u;
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

__device__ __forceinline__ double wave_sum_f64(double v) {
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  return v;
}

// ------------------------------------------------------------------ prep
__global__ __launch_bounds__(256) void k_prep(const float* __restrict__ x, int64_t n, int D,
                                              _Float16* __restrict__ x16, float* __restrict__ hn,
                                              float* __restrict__ eterm, double K1, double K2, double K3h,
                                              DevFlags* __restrict__ flags, uint32_t* __restrict__ ebmax_call) {
  const int lane = threadIdx.x & 63;
  const int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= n) return;
  const float* p = x + row * D;
  _Float16* q = x16 + row * D;
  double na = 0.0, l1 = 0.0;
  bool nf = false, rng = false;
  for (int d = lane * 4; d < D; d += 256) {
    const float4 v = *reinterpret_cast<const float4*>(p + d);
    const float c[4] = {v.x, v.y, v.z, v.w};
    _Float16 h[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const float a = fabsf(c[r]);
      nf |= !(a <= 3.402823466e38f);
      rng |= !(a < 256.0f);
      na = fma((double)c[r], (double)c[r], na);
      l1 += (double)a;
      h[r] = (_Float16)(c[r] * kScale);
    }
    uint2 packed;
    __builtin_memcpy(&packed, h, 8);
    *reinterpret_cast<uint2*>(q + d) = packed;
  }
  na = wave_sum_f64(na);
  l1 = wave_sum_f64(l1);
  const unsigned long long bn = __ballot(nf), br = __ballot(rng);
  if (lane == 0) {
    if (bn) atomicAdd(&flags->nonfinite, 1u);
    if (br) atomicAdd(&flags->out_of_range, 1u);
    hn[row] = (float)(0.5 * na);
    const double et = K1 * 0.5 * na + K2 * l1 + K3h + 0x1p-23 * (na + 1.0);
    const float e = round_up_f32(et);
    eterm[row] = e;
    if (!(bn | br)) atomicMax(ebmax_call, __float_as_uint(e));
  }
}

// ------------------------------------------------------------------ chunk init
__global__ void k_chunk_init(int nB, int W, int32_t* firstHit, uint32_t* hasEdge, uint32_t* maxcos,
                             uint64_t* bitmap, ChunkCounters* cc) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  const int64_t t0 = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  for (int64_t i = t0; i < nB; i += stride) {
    firstHit[i] = kNone;
    hasEdge[i] = 0u;
    maxcos[i] = 0x007fffffu;  // order-encoded -inf
  }
  for (int64_t i = t0; i < (int64_t)nB * W; i += stride) bitmap[i] = 0ull;
  if (t0 == 0) {
    cc->npairs = 0u;
    cc->n_escalate = 0u;
  }
}

__global__ void k_set_meta(StoreMeta* meta, int32_t m) {
  if (threadIdx.x == 0 && blockIdx.x == 0) meta->m = m;
}

// ------------------------------------------------------------------ screens
struct ScreenArgs {
  const _Float16* A;        // rows of the "earlier" side (store rows, or chunk rows)
  const _Float16* B;        // chunk rows (arrivals)
  const float* hnA;         // ||a||^2 / 2 of A rows
  const float* hnB;         // ||b||^2 / 2 of B rows
  const float* etB;         // per-row error term of B rows
  const uint32_t* ebmaxA;   // max error term over A rows (float bits)
  const StoreMeta* meta;    // store size (store screen)
  int nA;                   // A rows (chunk screen) -- store screen reads meta->m
  int nB;
  int D;
  int ntB;                  // B tiles
  int64_t nblocks;
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

__device__ __forceinline__ void push_pair(const ScreenArgs& a, int i, int kind, int y) {
  const uint32_t idx = atomicAdd(&a.cc->npairs, 1u);
  atomicAdd(&a.flags->n_pairs, 1u);
  if (idx < a.pair_cap) {
    a.pairs[idx] = make_int2(i | (kind << 31), y);
  } else {
    atomicOr(&a.flags->pair_overflow, 1u);
    atomicMax(&a.flags->pairs_needed, idx + 1u);   // capacity that would have sufficed
  }
}

// MODE 0: A = store, B = chunk.  MODE 1: A = B = chunk, pairs (ia < ib).
template <int MODE, bool WANT_MAX>
__global__ __launch_bounds__(kWG) void k_screen(ScreenArgs a) {
  __shared__ _Float16 lds[4 * kTB * kLdk];
  __shared__ float hbA[kTB];
  if (skip_all(a.flags)) return;
  const int64_t logical = xcd_remap(blockIdx.x, a.nblocks);
  int ta, tb;
  if (MODE == 0) {
    ta = (int)(logical / a.ntB);
    tb = (int)(logical % a.ntB);
  } else {
    // lower-triangular tile pairs ta <= tb, row-major over tb
    int t = (int)((sqrt(8.0 * (double)logical + 1.0) - 1.0) * 0.5);
    while ((int64_t)(t + 1) * (t + 2) / 2 <= logical) ++t;
    while ((int64_t)t * (t + 1) / 2 > logical) --t;
    tb = t;
    ta = (int)(logical - (int64_t)t * (t + 1) / 2);
  }
  const int nA = (MODE == 0) ? a.meta->m : a.nA;
  const int rowsA = min(kTB, nA - ta * kTB);
  const int rowsB = min(kTB, a.nB - tb * kTB);
  if (rowsA <= 0 || rowsB <= 0) return;
  if (threadIdx.x < kTB) hbA[threadIdx.x] = (threadIdx.x < rowsA) ? a.hnA[ta * kTB + threadIdx.x] : 0.0f;

  floatx16 acc[2][2];
  gemm_block_f16(a.A + (int64_t)ta * kTB * a.D, rowsA, a.B + (int64_t)tb * kTB * a.D, rowsB, a.D, a.D, lds, acc);

  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const float ebA = __uint_as_float(*a.ebmaxA);
#pragma unroll
  for (int tj = 0; tj < 2; ++tj) {
    const int ibl = wn * 64 + tj * 32 + (lane & 31);
    const int ib = tb * kTB + ibl;
    const bool vB = ibl < rowsB;
    float thrAmb = 3.0e38f, thrIn = 3.0e38f;
    if (vB) {
      const double base = (double)a.hnB[ib] - a.half_d2;
      const double e = (double)a.etB[ib] + (double)ebA;
      thrAmb = round_down_f32(base - e);
      thrIn = round_up_f32(base + e);
    }
    float mx = -3.0e38f, cmax = -3.0e38f;
#pragma unroll
    for (int ti = 0; ti < 2; ++ti) {
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int ial = wm * 64 + ti * 32 + acc_row(r, lane);
        const int ia = ta * kTB + ial;
        const bool valid = vB && ial < rowsA && (MODE == 0 || ia < ib);
        const float dot = acc[ti][tj][r] * kInvScale2;
        const float v = dot - hbA[ial];
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
    if (!hot) continue;
    // Rare path: classify this lane's candidates in increasing row order.
    if (MODE == 0) {
      int ydef = kNone;
      for (int ti = 0; ti < 2 && ydef == kNone; ++ti) {
        for (int r = 0; r < 16; ++r) {
          const int ial = wm * 64 + ti * 32 + acc_row(r, lane);
          if (ial >= rowsA) continue;
          const float v = acc[ti][tj][r] * kInvScale2 - hbA[ial];
          if (v < thrAmb) continue;
          const int ia = ta * kTB + ial;
          if (v >= thrIn) { ydef = ia; break; }
          push_pair(a, ib, 0, ia);
        }
      }
      if (ydef != kNone) atomicMin(&a.firstHit[ib], ydef);
    } else {
      for (int ti = 0; ti < 2; ++ti) {
        for (int r = 0; r < 16; ++r) {
          const int ial = wm * 64 + ti * 32 + acc_row(r, lane);
          const int ia = ta * kTB + ial;
          if (ial >= rowsA || ia >= ib) continue;
          const float v = acc[ti][tj][r] * kInvScale2 - hbA[ial];
          if (v < thrAmb) continue;
          if (v >= thrIn) {
            atomicOr(reinterpret_cast<unsigned long long*>(&a.bitmap[(int64_t)ib * a.W + (ia >> 6)]),
                     1ull << (ia & 63));
            a.hasEdge[ib] = 1u;
          } else {
            push_pair(a, ib, 1, ia);
          }
        }
      }
    }
  }
}

// ------------------------------------------------------------------ verify
struct VerifyArgs {
  const int2* pairs;
  uint32_t* status;       // 0 out, 1 in, 2 escalate, 3 skipped
  const ChunkCounters* cc;
  uint32_t pair_cap;
  const float* xc;        // chunk rows, float32 (caller memory)
  const float* xs;        // store rows, float32
  int D;
  double d2;              // delta^2 in binary64
  int32_t* firstHit;
  uint64_t* bitmap;
  int W;
  uint32_t* hasEdge;
  DevFlags* flags;
  ChunkCounters* ccw;
  int careful;
};

__global__ __launch_bounds__(256) void k_verify(VerifyArgs a) {
  if (skip_all(a.flags)) return;
  const uint32_t n = min(a.cc->npairs, a.pair_cap);
  const int lane = threadIdx.x & 63;
  const uint32_t wid = (blockIdx.x * blockDim.x + threadIdx.x) >> 6;
  const uint32_t nw = (gridDim.x * blockDim.x) >> 6;
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
    double s = 0.0;
    for (int d = lane; d < a.D; d += 64) {
      const double t = (double)pa[d] - (double)pb[d];
      s = fma(t, t, s);
    }
    s = wave_sum_f64(s);
    if (lane != 0) continue;
    const double margin = (double)(a.D + 8) * 2.5e-16 * fmax(a.d2, s) + 1e-300;
    uint32_t st;
    if (fabs(s - a.d2) <= margin) {
      st = 2u;
      atomicAdd(&a.ccw->n_escalate, 1u);
      atomicAdd(&a.flags->n_escalate, 1u);
      if (!a.careful) atomicOr(&a.flags->pair_overflow, 2u);
    } else if (s <= a.d2) {
      st = 1u;
      if (kind == 0) {
        atomicMin(&a.firstHit[i], y);
      } else {
        atomicOr(reinterpret_cast<unsigned long long*>(&a.bitmap[(int64_t)i * a.W + (y >> 6)]), 1ull << (y & 63));
        a.hasEdge[i] = 1u;
      }
    } else {
      st = 0u;
    }
    a.status[p] = st;
  }
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
  int64_t gbase;            // global id of chunk row 0
  int64_t* rep;             // caller output for the chunk (global ids, -1 kept)
  int32_t* pos;             // store position of kept rows, -1 if dropped
  int32_t* rep_row;         // >= 0 store row, <= -2 chunk row (-(j+2)), -1 kept
  uint64_t* kept_words;     // kept mask of the chunk (64 words)
  DevFlags* flags;
};

// One wave.  Lane L owns bits [64L, 64L + 64) of the chunk's kept mask.
__global__ __launch_bounds__(64) void k_resolve(ResolveArgs a) {
  if (skip_all(a.flags)) return;
  const int lane = threadIdx.x;
  const int nblk = (a.nB + 63) >> 6;
  uint64_t kept = 0ull;
  for (int blk = 0; blk < nblk; ++blk) {
    const int r = blk * 64 + lane;
    const bool v = r < a.nB;
    const int32_t hit = v ? a.firstHit[r] : kNone;
    const bool edge = v && a.hasEdge[r] != 0u;
    const bool plain_keep = v && hit == kNone && !edge;
    const bool active = v && hit == kNone && edge;
    const uint64_t pk = __ballot(plain_keep);
    if (lane == blk) kept |= pk;
    if (v && hit != kNone) {
      a.rep[r] = a.store_ids[hit];
      a.rep_row[r] = hit;
    } else if (plain_keep) {
      a.rep[r] = -1;
      a.rep_row[r] = -1;
    }
    uint64_t act = __ballot(active);
    // Active rows in increasing order; each needs every earlier row decided,
    // which holds because rows are visited in order and decisions of plain rows
    // (store hit / no edge) do not depend on other rows.
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
          a.rep[i] = a.gbase + j;
          a.rep_row[i] = -(j + 2);
        }
      } else {
        if (lane == blk) kept |= 1ull << b;
        if (lane == 0) {
          a.rep[i] = -1;
          a.rep_row[i] = -1;
        }
      }
    }
  }
  // positions of kept rows
  const int cnt = __popcll(kept);
  int pre = cnt;
  for (int o = 1; o < 64; o <<= 1) {
    const int t = __shfl_up(pre, o);
    if (lane >= o) pre += t;
  }
  pre -= cnt;  // exclusive prefix
  const int total = __shfl(pre + cnt, 63);
  const int m0 = a.meta->m;
  a.kept_words[lane] = kept;
  for (int blk = 0; blk < nblk; ++blk) {
    const int r = blk * 64 + lane;
    const uint64_t w = __shfl(kept, blk);
    const int base = __shfl(pre, blk);
    if (r < a.nB) {
      const bool k = (w >> lane) & 1ull;
      a.pos[r] = k ? m0 + base + __popcll(w & ((1ull << lane) - 1ull)) : -1;
    }
  }
  __syncthreads();
  if (lane == 0) {
    a.meta->m = m0 + total;
    atomicAdd(&a.flags->n_kept, (uint32_t)total);
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
  int64_t gbase;
  int D;
  float* xs;
  _Float16* x16s;
  float* hns;
  int64_t* ids;
  StoreMeta* meta;
  DevFlags* flags;
};

__global__ __launch_bounds__(256) void k_append(AppendArgs a) {
  if (skip_all(a.flags)) return;
  const int r = blockIdx.x;
  const int p = a.pos[r];
  const float* src = a.xc + (int64_t)r * a.D;
  if (p >= 0) {
    float* dst = a.xs + (int64_t)p * a.D;
    for (int d = threadIdx.x * 4; d < a.D; d += 1024)
      *reinterpret_cast<float4*>(dst + d) = *reinterpret_cast<const float4*>(src + d);
    const _Float16* s16 = a.x16c + (int64_t)r * a.D;
    _Float16* d16 = a.x16s + (int64_t)p * a.D;
    for (int d = threadIdx.x * 8; d < a.D; d += 2048)
      *reinterpret_cast<uint4*>(d16 + d) = *reinterpret_cast<const uint4*>(s16 + d);
    if (threadIdx.x == 0) {
      a.hns[p] = a.hnc[r];
      a.ids[p] = a.gbase + r;
      atomicMax(&a.meta->ebmax_bits, __float_as_uint(a.etc[r]));
    }
    return;
  }
  // dropped: ||x - x_rep||^2 in binary64 for the measured bound
  const int rr = a.rep_row[r];
  const float* b = (rr >= 0) ? a.xs + (int64_t)rr * a.D : a.xc + (int64_t)(-rr - 2) * a.D;
  double s = 0.0;
  for (int d = threadIdx.x; d < a.D; d += 256) {
    const double t = (double)src[d] - (double)b[d];
    s = fma(t, t, s);
  }
  s = wave_sum_f64(s);
  __shared__ double part[4];
  if ((threadIdx.x & 63) == 0) part[threadIdx.x >> 6] = s;
  __syncthreads();
  if (threadIdx.x == 0) {
    const double tot = (part[0] + part[1]) + (part[2] + part[3]);
    atomicMax(reinterpret_cast<unsigned long long*>(&a.flags->dhat2_bits),
              (unsigned long long)__double_as_longlong(tot));
  }
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
size_t store_meta_bytes() { return sizeof(StoreMeta); }

lam_status store_alloc(lam_store* st) {
  const size_t cap = (size_t)st->capacity, D = (size_t)st->dim;
  LAM_HIP(hipMalloc(&st->x32, cap * D * 4));
  LAM_HIP(hipMalloc(&st->x16, cap * D * 2));
  LAM_HIP(hipMalloc(&st->hn, cap * 4));
  LAM_HIP(hipMalloc(&st->ids, cap * 8));
  LAM_HIP(hipMalloc(&st->stat_dev, sizeof(StoreMeta)));
  LAM_HIP(hipMemset(st->stat_dev, 0, sizeof(StoreMeta)));
  LAM_HIP(hipDeviceSynchronize());
  return LAM_OK;
}

void store_free(lam_store* st) {
  for (void* p : {(void*)st->x32, (void*)st->x16, (void*)st->hn, (void*)st->l1, (void*)st->nrm, (void*)st->ids,
                  (void*)st->stat_dev, (void*)st->codes})
    if (p) (void)hipFree(p);
  st->x32 = nullptr;
  st->x16 = nullptr;
  st->hn = st->l1 = st->nrm = st->stat_dev = nullptr;
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

// Exact decisions for the pairs the binary64 test could not separate from
// delta^2 (status 2), patched into the chunk's hit/edge state.
lam_status escalate_chunk(lam_ctx* ctx, lam_store* st, const float* xc, int64_t c_rows, int32_t* firstHit,
                          uint64_t* bitmap, int W, uint32_t* hasEdge, const int2* pairs_dev,
                          const uint32_t* status_dev, const ChunkCounters* cc_dev, uint32_t cap) {
  ChunkCounters cc{};
  LAM_HIP(hipMemcpyAsync(&cc, cc_dev, sizeof cc, hipMemcpyDeviceToHost, ctx->stream));
  LAM_HIP(hipStreamSynchronize(ctx->stream));
  if (cc.n_escalate == 0) return LAM_OK;
  const uint32_t n = std::min(cc.npairs, cap);
  std::vector<int2> pairs(n);
  std::vector<uint32_t> status(n);
  LAM_HIP(hipMemcpy(pairs.data(), pairs_dev, n * sizeof(int2), hipMemcpyDeviceToHost));
  LAM_HIP(hipMemcpy(status.data(), status_dev, n * 4, hipMemcpyDeviceToHost));
  const int D = st->dim;
  std::vector<float> ra(D), rb(D);
  for (uint32_t p = 0; p < n; ++p) {
    if (status[p] != 2u) continue;
    const int kind = (int)((uint32_t)pairs[p].x >> 31);
    const int i = pairs[p].x & 0x7fffffff;
    const int y = pairs[p].y;
    (void)c_rows;
    LAM_HIP(hipMemcpy(ra.data(), xc + (int64_t)i * D, D * 4, hipMemcpyDeviceToHost));
    LAM_HIP(hipMemcpy(rb.data(), (kind ? xc : st->x32) + (int64_t)y * D, D * 4, hipMemcpyDeviceToHost));
    if (!exact_within(ra.data(), rb.data(), D, st->tau)) continue;
    if (kind == 0) {
      int32_t cur = 0;
      LAM_HIP(hipMemcpy(&cur, firstHit + i, 4, hipMemcpyDeviceToHost));
      if (y < cur) LAM_HIP(hipMemcpy(firstHit + i, &y, 4, hipMemcpyHostToDevice));
    } else {
      uint64_t w = 0;
      LAM_HIP(hipMemcpy(&w, bitmap + (int64_t)i * W + (y >> 6), 8, hipMemcpyDeviceToHost));
      w |= 1ull << (y & 63);
      LAM_HIP(hipMemcpy(bitmap + (int64_t)i * W + (y >> 6), &w, 8, hipMemcpyHostToDevice));
      const uint32_t one = 1u;
      LAM_HIP(hipMemcpy(hasEdge + i, &one, 4, hipMemcpyHostToDevice));
    }
  }
  return LAM_OK;
}

}  // namespace

lam_status dedup_ingest(lam_ctx* ctx, lam_store* st, const float* x, int64_t n, int64_t* rep, float* max_cos,
                        lam_ingest_stats* stats) {
  const int D = st->dim;
  const int64_t m_before = st->size;
  if (n == 0) {
    if (stats) {
      *stats = lam_ingest_stats{};
      stats->store_size = st->size;
      stats->delta_hat_run = st->delta_hat_run;
    }
    return LAM_OK;
  }
  const int CH = (int)std::min<int64_t>(n, kChunk);
  const int W = (CH + 63) / 64;
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

  bool careful = false;
  for (int attempt = 0; attempt < 4; ++attempt) {
    const uint32_t cap = ctx->pair_cap;
    LAM_TRY(ctx->scratch[S_PAIRS].ensure((size_t)cap * sizeof(int2)));
    LAM_TRY(ctx->scratch[S_STATUS].ensure((size_t)cap * 4));
    int2* pairs = ctx->scratch[S_PAIRS].as<int2>();
    uint32_t* status = ctx->scratch[S_STATUS].as<uint32_t>();

    LAM_TRY(clear_flags(ctx));
    hipLaunchKernelGGL(k_set_meta, dim3(1), dim3(64), 0, ctx->stream, meta, (int32_t)m_before);
    {
      ProfScope ps(ctx, "dedup_prep");
      hipLaunchKernelGGL(k_prep, dim3((unsigned)((n + 3) / 4)), dim3(256), 0, ctx->stream, x, n, D, x16c, hnc, etc,
                         K.K1, K.K2, K.K3h, ctx->flags_dev, &ctx->flags_dev->ebmax_call_bits);
    }
    LAM_HIP(hipGetLastError());

    for (int64_t c0 = 0; c0 < n; c0 += CH) {
      const int nB = (int)std::min<int64_t>(CH, n - c0);
      const int ntB = (nB + kTB - 1) / kTB;
      const float* xc = x + c0 * D;
      const _Float16* x16 = x16c + c0 * D;
      hipLaunchKernelGGL(k_chunk_init, dim3(64), dim3(256), 0, ctx->stream, nB, W, firstHit, hasEdge, maxcos,
                         bitmap, cc);
      LAM_HIP(hipGetLastError());

      ScreenArgs sa{};
      sa.B = x16;
      sa.hnB = hnc + c0;
      sa.etB = etc + c0;
      sa.meta = meta;
      sa.nB = nB;
      sa.D = D;
      sa.ntB = ntB;
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

      // screen against the store (rows retained before this chunk)
      const int64_t m_ub = m_before + c0;
      if (m_ub > 0) {
        ScreenArgs s0 = sa;
        s0.A = st->x16;
        s0.hnA = st->hn;
        s0.ebmaxA = &meta->ebmax_bits;
        const int64_t ntA = (m_ub + kTB - 1) / kTB;
        s0.nblocks = ntA * ntB;
        LAM_CHECK(s0.nblocks < (1LL << 31), LAM_EINVAL, "screen grid too large");
        ProfScope ps(ctx, "dedup_screen_store");
        if (want_max)
          hipLaunchKernelGGL((k_screen<0, true>), dim3((unsigned)s0.nblocks), dim3(kWG), 0, ctx->stream, s0);
        else
          hipLaunchKernelGGL((k_screen<0, false>), dim3((unsigned)s0.nblocks), dim3(kWG), 0, ctx->stream, s0);
        LAM_HIP(hipGetLastError());
      }
      // screen inside the chunk (j < i)
      if (nB > 1) {
        ScreenArgs s1 = sa;
        s1.A = x16;
        s1.hnA = hnc + c0;
        s1.ebmaxA = &ctx->flags_dev->ebmax_call_bits;
        s1.nA = nB;
        s1.nblocks = (int64_t)ntB * (ntB + 1) / 2;
        ProfScope ps(ctx, "dedup_screen_chunk");
        if (want_max)
          hipLaunchKernelGGL((k_screen<1, true>), dim3((unsigned)s1.nblocks), dim3(kWG), 0, ctx->stream, s1);
        else
          hipLaunchKernelGGL((k_screen<1, false>), dim3((unsigned)s1.nblocks), dim3(kWG), 0, ctx->stream, s1);
        LAM_HIP(hipGetLastError());
      }
      VerifyArgs va{pairs, status, cc, cap, xc, st->x32, D, st->d2, firstHit, bitmap, W, hasEdge,
                    ctx->flags_dev, cc, careful ? 1 : 0};
      {
        ProfScope ps(ctx, "dedup_verify");
        hipLaunchKernelGGL(k_verify, dim3(256), dim3(256), 0, ctx->stream, va);
        LAM_HIP(hipGetLastError());
      }
      if (careful)
        LAM_TRY(escalate_chunk(ctx, st, xc, nB, firstHit, bitmap, W, hasEdge, pairs, status, cc, cap));
      ResolveArgs ra{nB, W, firstHit, hasEdge, bitmap, st->ids, meta, st->n_seen + c0, rep + c0, pos, rep_row,
                     kept_words, ctx->flags_dev};
      {
        ProfScope ps(ctx, "dedup_resolve");
        hipLaunchKernelGGL(k_resolve, dim3(1), dim3(64), 0, ctx->stream, ra);
        LAM_HIP(hipGetLastError());
      }
      AppendArgs aa{xc, x16, hnc + c0, etc + c0, pos, rep_row, st->n_seen + c0, D, st->x32, st->x16, st->hn,
                    st->ids, meta, ctx->flags_dev};
      {
        ProfScope ps(ctx, "dedup_append");
        hipLaunchKernelGGL(k_append, dim3((unsigned)nB), dim3(256), 0, ctx->stream, aa);
        LAM_HIP(hipGetLastError());
      }
      if (want_max) {
        hipLaunchKernelGGL(k_maxcos, dim3((unsigned)((nB + 3) / 4)), dim3(256), 0, ctx->stream, nB, maxcos, G,
                           kept_words, max_cos + c0, ctx->flags_dev);
        LAM_HIP(hipGetLastError());
      }
    }
    LAM_TRY(read_flags(ctx));
    const DevFlags f = *ctx->flags_host;
    LAM_CHECK(f.nonfinite == 0, LAM_EINVAL, "input holds NaN or Inf (%u rows)", f.nonfinite);
    LAM_CHECK(f.out_of_range == 0, LAM_EINVAL, "input has coordinates with |x| >= 256 (%u rows)", f.out_of_range);
    if (f.pair_overflow & 1u) {
      ctx->pair_cap = std::max<uint32_t>(ctx->pair_cap * 2u, f.pairs_needed + (f.pairs_needed >> 2));
      continue;
    }
    if (f.pair_overflow & 2u) {
      careful = true;
      continue;
    }
    double dh2 = 0.0;
    memcpy(&dh2, &f.dhat2_bits, 8);
    const double dh_call = std::sqrt(dh2);
    st->size = m_before + f.n_kept;
    st->n_seen += n;
    st->delta_hat_run = std::max(st->delta_hat_run, dh_call);
    if (stats) {
      stats->n_in = n;
      stats->n_kept = f.n_kept;
      stats->n_dropped = n - f.n_kept;
      stats->store_size = st->size;
      stats->n_ambiguous_pairs = f.n_pairs;
      stats->n_exact_escalations = f.n_escalate;
      stats->delta_hat_call = dh_call;
      stats->delta_hat_run = st->delta_hat_run;
    }
    return LAM_OK;
  }
  set_error("ingest did not converge (ambiguous-pair list kept overflowing)");
  return LAM_EDEVICE;
}

}  // namespace lam
