// Per-block fixed-length codec of the retained store's Q_eps codes (Section
// 2.2, L2 "error-bounded byte compression"; Section "Composite reduction":
// the reductions of deduplication and of the codec multiply).  Applied to the
// codes themselves, so decoding gives back exactly the Q_eps reconstruction and
// the score bound eps * ||q||_1 is unchanged.
//
// Format.  A block is 32 consecutive codes of a row.  Codes map to unsigned
// values by zigzag (u = 2q for q >= 0, -2q - 1 for q < 0); a block is stored
// with the bit width w of its largest u (0 for an all-zero block) as w 32-bit
// words in bit-plane order: bit j of word t is bit t of code j.  Per block one
// width byte; per row one 64-bit word offset (row_off[r], rows + 1 entries);
// blocks of a row and rows follow each other.
//
// On a 64-lane wave the two 32-lane halves hold two blocks with one code per
// lane: a block's bit planes are ballots of the lanes' bits (encode), and a
// lane rebuilds its code from the block's w planes (decode).
#include <algorithm>
#include <cmath>

#include "lam_internal.h"

namespace lam {
namespace {

__device__ __forceinline__ uint32_t zigzag(int32_t q) { return ((uint32_t)q << 1) ^ (uint32_t)(q >> 31); }
__device__ __forceinline__ int32_t unzigzag(uint32_t u) { return (int32_t)(u >> 1) ^ -(int32_t)(u & 1u); }

// A round of a row: up to kPairs pairs of blocks, the two 32-lane halves of
// the wave taking one block each with one code per lane (lane j of half h
// holds code j of block k0 + 2 i + h in round slot i).  A round's loads are
// all issued before any is used; consecutive lanes read consecutive fields,
// so a half reads its block's b words in one or two requests.
constexpr int kPairs = 16;

// A buffer resource over the words [base, base + words): loads past the end
// read as zero.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t words_rsrc(const uint32_t* base, uint32_t words) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<uint32_t*>(base), (short)0, (int)(words * 4u), 0x00020000);
}

// Code i of a row's b-bit stream (rs over the row): both words that may hold
// the field are loaded without a branch (the second past the row's end reads
// as zero and is shifted out), so a round's loads issue back to back.
__device__ __forceinline__ int32_t code_rs(__amdgpu_buffer_rsrc_t rs, int b, int i) {
  const uint32_t bit = (uint32_t)i * (uint32_t)b;
  const uint32_t w = bit >> 5, off = bit & 31u;
  const uint32_t lo = (uint32_t)__builtin_amdgcn_raw_buffer_load_b32(rs, w * 4u, 0, 0);
  const uint32_t hi = (uint32_t)__builtin_amdgcn_raw_buffer_load_b32(rs, w * 4u + 4u, 0, 0);
  const uint32_t u = __builtin_amdgcn_alignbit(hi, lo, off);   // bits [off, off + 32) of hi:lo
  return (int32_t)(u << (32 - b)) >> (32 - b);
}

__device__ __forceinline__ void load_round(const uint32_t* __restrict__ codes, int b, int64_t r, int D, int nb,
                                           int k0, uint32_t (&u)[kPairs]) {
  const int lane = threadIdx.x & 63, half = lane >> 5, j = lane & 31;
  const uint32_t row_words = (uint32_t)(D / 32) * (uint32_t)b;
  const __amdgpu_buffer_rsrc_t rs = words_rsrc(codes + r * (int64_t)row_words, row_words);
#pragma unroll
  for (int i = 0; i < kPairs; ++i) {
    const int kb = k0 + 2 * i + half;
    u[i] = kb < nb ? zigzag(code_rs(rs, b, kb * 32 + j)) : 0u;
  }
}

// Pass 1: one wave per row: block widths and the row's word count.  The bit
// length of a block's largest zigzag code is that of the OR of its codes:
// the highest bit t whose ballot over the half is not empty (b ballots per
// pair of blocks, all zigzag codes being below 2^b).
__global__ __launch_bounds__(256) void k_blk_widths(const uint32_t* __restrict__ codes, int b, int64_t rows, int D,
                                                    uint8_t* __restrict__ widths, uint32_t* __restrict__ row_words) {
  const int lane = threadIdx.x & 63, half = lane >> 5, j = lane & 31;
  const int64_t r = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (r >= rows) return;
  const int nb = D / 32;
  uint32_t total = 0;
  for (int k0 = 0; k0 < nb; k0 += 2 * kPairs) {
    uint32_t u[kPairs];
    load_round(codes, b, r, D, nb, k0, u);
#pragma unroll
    for (int i = 0; i < kPairs; ++i) {
      uint32_t w0 = 0, w1 = 0;
      for (int t = 0; t < b; ++t) {
        const unsigned long long m = __ballot((u[i] >> t) & 1u);
        w0 = (uint32_t)m ? (uint32_t)t + 1u : w0;
        w1 = (uint32_t)(m >> 32) ? (uint32_t)t + 1u : w1;
      }
      const uint32_t w = half ? w1 : w0;
      const int kb = k0 + 2 * i + half;
      if (j == 0 && kb < nb) {
        widths[r * nb + kb] = (uint8_t)w;
        total += w;
      }
    }
  }
  total = (uint32_t)__shfl((int)total, 0) + (uint32_t)__shfl((int)total, 32);
  if (lane == 0) row_words[r] = total;
}

// Exclusive scan of row word counts into row offsets (three small kernels:
// per-chunk scans, a scan of the chunk totals, and the add).
constexpr int kScanThreads = 1024;
constexpr int kScanPer = 4;
constexpr int kScanChunk = kScanThreads * kScanPer;

__device__ __forceinline__ uint64_t block_exclusive_scan(uint64_t v, uint64_t* warp_tot, uint64_t* total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  unsigned long long x = v;
  for (int o = 1; o < 64; o <<= 1) {
    const unsigned long long t = __shfl_up(x, o);
    if (lane >= o) x += t;
  }
  if (lane == 63) warp_tot[wave] = x;
  __syncthreads();
  if (threadIdx.x == 0) {
    uint64_t acc = 0;
    for (int w = 0; w < kScanThreads / 64; ++w) {
      const uint64_t t = warp_tot[w];
      warp_tot[w] = acc;
      acc += t;
    }
    *total = acc;
  }
  __syncthreads();
  return warp_tot[wave] + x - v;
}

__global__ __launch_bounds__(kScanThreads) void k_scan_chunks(const uint32_t* __restrict__ in, int64_t n,
                                                              uint64_t* __restrict__ out, uint64_t* __restrict__ sums) {
  __shared__ uint64_t wt[kScanThreads / 64];
  __shared__ uint64_t tot;
  const int64_t base = (int64_t)blockIdx.x * kScanChunk + (int64_t)threadIdx.x * kScanPer;
  uint32_t v[kScanPer];
  uint64_t s = 0;
#pragma unroll
  for (int i = 0; i < kScanPer; ++i) {
    v[i] = base + i < n ? in[base + i] : 0u;
    s += v[i];
  }
  uint64_t x = block_exclusive_scan(s, wt, &tot);
#pragma unroll
  for (int i = 0; i < kScanPer; ++i) {
    if (base + i < n) out[base + i] = x;
    x += v[i];
  }
  if (threadIdx.x == 0) sums[blockIdx.x] = tot;
}

__global__ __launch_bounds__(kScanThreads) void k_scan_sums(uint64_t* __restrict__ sums, int nchunks,
                                                            uint64_t* __restrict__ grand) {
  __shared__ uint64_t wt[kScanThreads / 64];
  __shared__ uint64_t tot;
  // nchunks <= kScanChunk: four per thread, as above
  const int base = threadIdx.x * kScanPer;
  uint64_t v[kScanPer];
  uint64_t s = 0;
#pragma unroll
  for (int i = 0; i < kScanPer; ++i) {
    v[i] = base + i < nchunks ? sums[base + i] : 0u;
    s += v[i];
  }
  uint64_t x = block_exclusive_scan(s, wt, &tot);
#pragma unroll
  for (int i = 0; i < kScanPer; ++i) {
    if (base + i < nchunks) sums[base + i] = x;
    x += v[i];
  }
  if (threadIdx.x == 0) *grand = tot;
}

__global__ void k_scan_add(uint64_t* __restrict__ out, int64_t n, const uint64_t* __restrict__ sums) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) out[i] += sums[i / kScanChunk];
}

// Prefix of the widths of a row's blocks below block k, for the lanes of one
// wave (lane l holds blocks l, l + 64, ... in turn); returns this lane's
// exclusive prefix for block `k` and carries the running total across rounds.
__device__ __forceinline__ uint32_t width_prefix(uint32_t w, uint32_t& carry) {
  const int lane = threadIdx.x & 63;
  uint32_t x = w;
  for (int o = 1; o < 64; o <<= 1) {
    const uint32_t t = __shfl_up(x, o);
    if (lane >= o) x += t;
  }
  const uint32_t ex = carry + x - w;
  carry += __shfl(x, 63);
  return ex;
}

// The word offsets within row r of its blocks k0 + l (lane l, l < 64) and
// their widths; carry: the words of the blocks before k0.
__device__ __forceinline__ void row_offsets(const uint8_t* __restrict__ widths, int64_t r, int nb, int k0,
                                            uint32_t& carry, uint32_t& wl, uint32_t& pre) {
  const int lane = threadIdx.x & 63;
  const int kl = k0 + lane;
  wl = kl < nb ? widths[r * nb + kl] : 0u;
  pre = width_prefix(wl, carry);
}

// Pass 2: one wave per row; per round of block pairs the codes are loaded
// first, then each bit plane of a block is a ballot over its half.
__global__ __launch_bounds__(256) void k_blk_pack(const uint32_t* __restrict__ codes, int b, int64_t rows, int D,
                                                  const uint8_t* __restrict__ widths,
                                                  const uint64_t* __restrict__ row_off, uint32_t* __restrict__ data) {
  const int lane = threadIdx.x & 63, half = lane >> 5, j = lane & 31;
  const int64_t r = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (r >= rows) return;
  const int nb = D / 32;
  const uint64_t roff = row_off[r];
  uint32_t carry = 0, wl = 0, pre = 0;
  for (int k0 = 0; k0 < nb; k0 += 2 * kPairs) {
    uint32_t u[kPairs];
    load_round(codes, b, r, D, nb, k0, u);
    if (k0 % 64 == 0) row_offsets(widths, r, nb, k0, carry, wl, pre);
#pragma unroll
    for (int i = 0; i < kPairs; ++i) {
      const int kb = k0 + 2 * i + half;
      const int src = (kb - (k0 & ~63)) & 63;
      const uint32_t w = (uint32_t)__shfl((int)wl, src);
      const uint32_t p = (uint32_t)__shfl((int)pre, src);
      const uint32_t wmax = max((uint32_t)__shfl((int)w, 0), (uint32_t)__shfl((int)w, 32));
      uint32_t mine = 0;
      for (uint32_t t = 0; t < wmax; ++t) {
        const unsigned long long m = __ballot((u[i] >> t) & 1u);
        const uint32_t plane = half ? (uint32_t)(m >> 32) : (uint32_t)m;
        mine = ((uint32_t)j == t) ? plane : mine;
      }
      if (kb < nb && (uint32_t)j < w) data[roff + p + j] = mine;
    }
  }
}

// One wave per row: decode every block, either to float32 x_hat =
// float32(float64(q * s)) (xhat != NULL) or back to the b-bit stream (codes_out
// != NULL; a block's 32 codes are exactly b words).  Per round the lanes j < w
// of each half load plane j of their block (every plane once), and a lane
// rebuilds its code from the planes by shuffles.
__global__ __launch_bounds__(256) void k_blk_decode(const uint8_t* __restrict__ widths,
                                                    const uint64_t* __restrict__ row_off,
                                                    const uint32_t* __restrict__ data, int64_t rows, int D, double s,
                                                    float* __restrict__ xhat, int b, uint32_t* __restrict__ codes_out) {
  const int lane = threadIdx.x & 63, half = lane >> 5, j = lane & 31;
  const int64_t r = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (r >= rows) return;
  const int nb = D / 32;
  const uint64_t roff = row_off[r];
  const __amdgpu_buffer_rsrc_t rs = words_rsrc(data + roff, (uint32_t)(row_off[r + 1] - roff));
  const uint32_t mask = b >= 32 ? 0xffffffffu : ((1u << b) - 1u);
  uint32_t carry = 0, wl = 0, pre = 0;
  for (int k0 = 0; k0 < nb; k0 += 2 * kPairs) {
    if (k0 % 64 == 0) row_offsets(widths, r, nb, k0, carry, wl, pre);
    uint32_t w[kPairs], pl[kPairs];
#pragma unroll
    for (int i = 0; i < kPairs; ++i) {
      const int kb = k0 + 2 * i + half;
      const int src = (kb - (k0 & ~63)) & 63;
      const uint32_t ws = (uint32_t)__shfl((int)wl, src);
      const uint32_t p = (uint32_t)__shfl((int)pre, src);
      w[i] = kb < nb ? ws : 0u;
      // plane j of this half's block (lanes past the width: an offset past the row, read as zero)
      pl[i] = (uint32_t)__builtin_amdgcn_raw_buffer_load_b32(rs, (uint32_t)j < w[i] ? (p + j) * 4u : 0xfffffff0u, 0, 0);
    }
#pragma unroll
    for (int i = 0; i < kPairs; ++i) {
      const int kb = k0 + 2 * i + half;
      const uint32_t wmax = max((uint32_t)__shfl((int)w[i], 0), (uint32_t)__shfl((int)w[i], 32));
      uint32_t u = 0;
      for (uint32_t t = 0; t < wmax; ++t) {
        const uint32_t plane = (uint32_t)__shfl((int)pl[i], (half << 5) | (int)t);   // (zero past the width)
        u |= ((plane >> j) & 1u) << t;
      }
      const int32_t q = unzigzag(u);
      const int64_t e = r * D + (int64_t)kb * 32 + j;
      if (xhat) {
        if (kb < nb) xhat[e] = (float)((double)q * s);
      } else {
        // word j of the block's b-bit stream holds bits [32 j, 32 j + 32): the
        // fields of codes c0 .. c0 + ceil(32 / b), c0 = 32 j / b (a loop of the
        // same length on every lane, so every shuffle has all lanes)
        const uint32_t f = (uint32_t)q & mask;
        const int c0 = (32 * j) / b;
        const int steps = (32 + b - 1) / b + 1;
        uint32_t word = 0;
        for (int i2 = 0; i2 < steps; ++i2) {
          const int c = c0 + i2;
          const uint32_t fc = (uint32_t)__shfl((int)f, (half << 5) | (c & 31));
          const int bit = c * b - j * 32;   // field start relative to word j
          if (c < 32 && bit > -b && bit < 32) word |= bit >= 0 ? (fc << bit) : (fc >> -bit);
        }
        if (kb < nb && j < b) codes_out[(r * (int64_t)D + (int64_t)kb * 32) * b / 32 + j] = word;
      }
    }
  }
}

}  // namespace

lam_status block_encode(lam_ctx* ctx, lam_store* st, lam_block_stats* out) {
  const int D = st->dim;
  const int nb = D / 32;
  const int64_t m = st->size;
  const int b = st->q.bits;
  const int64_t nchunks = (m + kScanChunk - 1) / kScanChunk;
  LAM_CHECK(nchunks <= kScanChunk, LAM_EINVAL, "store too large for the block codec's scan");
  if (!st->blk_w) {
    LAM_HIP(hipMalloc(&st->blk_w, (size_t)st->capacity * nb));
    LAM_HIP(hipMalloc(&st->blk_row_off, (size_t)(st->capacity + 1) * 8));
  }
  LAM_TRY(ctx->scratch[kScratchBlocks].ensure((size_t)m * 4 + (size_t)(nchunks + 1) * 8 + 64));
  uint32_t* row_words = ctx->scratch[kScratchBlocks].as<uint32_t>();
  uint64_t* sums = reinterpret_cast<uint64_t*>(ctx->scratch[kScratchBlocks].as<char>() + (((size_t)m * 4 + 7) & ~7ull));
  const unsigned rows_grid = (unsigned)((m + 3) / 4);
  {
    ProfScope ps(ctx, "store_block_encode");
    if (m > 0) {
      hipLaunchKernelGGL(k_blk_widths, dim3(rows_grid), dim3(256), 0, ctx->stream, st->codes, b, m, D, st->blk_w,
                         row_words);
      LAM_HIP(hipGetLastError());
      hipLaunchKernelGGL(k_scan_chunks, dim3((unsigned)nchunks), dim3(kScanThreads), 0, ctx->stream, row_words, m,
                         st->blk_row_off, sums);
      hipLaunchKernelGGL(k_scan_sums, dim3(1), dim3(kScanThreads), 0, ctx->stream, sums, (int)nchunks,
                         st->blk_row_off + m);
      hipLaunchKernelGGL(k_scan_add, dim3((unsigned)((m + 255) / 256)), dim3(256), 0, ctx->stream, st->blk_row_off,
                         m, sums);
      LAM_HIP(hipGetLastError());
    }
  }
  uint64_t words = 0;
  if (m > 0) LAM_HIP(hipMemcpyAsync(&words, st->blk_row_off + m, 8, hipMemcpyDeviceToHost, ctx->stream));
  LAM_HIP(hipStreamSynchronize(ctx->stream));
  if (words * 4 > st->blk_cap) {
    if (st->blk_data) LAM_HIP(hipFree(st->blk_data));
    st->blk_data = nullptr;
    st->blk_cap = 0;
    LAM_HIP(hipMalloc(&st->blk_data, std::max<uint64_t>(words * 4, 4)));
    st->blk_cap = std::max<uint64_t>(words * 4, 4);
  }
  if (m > 0) {
    ProfScope ps(ctx, "store_block_pack");
    hipLaunchKernelGGL(k_blk_pack, dim3(rows_grid), dim3(256), 0, ctx->stream, st->codes, b, m, D, st->blk_w,
                       st->blk_row_off, st->blk_data);
    LAM_HIP(hipGetLastError());
  }
  st->blk_rows = m;
  st->blk_words = words;
  if (out) {
    lam_block_stats s{};
    s.rows = m;
    s.blocks = m * nb;
    s.data_bytes = words * 4;
    s.meta_bytes = (uint64_t)m * nb + (uint64_t)(m + 1) * 8;
    s.total_bytes = s.data_bytes + s.meta_bytes;
    const double ncodes = (double)m * D;
    s.bits_per_code = ncodes > 0 ? 8.0 * (double)s.total_bytes / ncodes : 0.0;
    s.plain_bits = b;
    s.codec_ratio = s.bits_per_code > 0 ? 32.0 / s.bits_per_code : 0.0;
    s.composite_ratio = s.total_bytes > 0 ? (double)st->n_seen * D * 4.0 / (double)s.total_bytes : 0.0;
    *out = s;
  }
  return LAM_OK;
}

lam_status block_decode(lam_ctx* ctx, const lam_store* st, float* xhat, uint32_t* codes_out) {
  const int64_t m = st->blk_rows;
  if (m <= 0) return LAM_OK;
  ProfScope ps(ctx, xhat ? "store_block_decode" : "store_block_expand");
  hipLaunchKernelGGL(k_blk_decode, dim3((unsigned)((m + 3) / 4)), dim3(256), 0, ctx->stream, st->blk_w,
                     st->blk_row_off, st->blk_data, m, st->dim, st->q.step, xhat, st->q.bits, codes_out);
  LAM_HIP(hipGetLastError());
  return LAM_OK;
}

}  // namespace lam
