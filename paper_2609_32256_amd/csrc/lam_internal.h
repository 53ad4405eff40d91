// Internal declarations of liblam: context, store, scratch arena, error state
// and the kernel launchers.  Not part of the ABI.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>
#include <string>
#include <vector>

#include "exact.h"
#include "lam.h"

namespace lam {

// ------------------------------------------------------------------ errors
void set_error(const char* fmt, ...);

struct Status {
  lam_status s;
};

#define LAM_HIP(call)                                                            \
  do {                                                                           \
    hipError_t e_ = (call);                                                      \
    if (e_ != hipSuccess) {                                                      \
      ::lam::set_error("%s failed: %s (%s:%d)", #call, hipGetErrorString(e_),    \
                       __FILE__, __LINE__);                                      \
      return LAM_EDEVICE;                                                        \
    }                                                                            \
  } while (0)

#define LAM_CHECK(cond, status, ...)                                             \
  do {                                                                           \
    if (!(cond)) {                                                               \
      ::lam::set_error(__VA_ARGS__);                                             \
      return (status);                                                           \
    }                                                                            \
  } while (0)

#define LAM_TRY(expr)                                                            \
  do {                                                                           \
    lam_status s_ = (expr);                                                      \
    if (s_ != LAM_OK) return s_;                                                 \
  } while (0)

// ------------------------------------------------------------------ device buffer
// Context scratch slots: 0-6 ingest (dedup.hip), 7-11 scoring (score.hip),
// then the ones below.
constexpr int kScratchCeilingRep = 12;   // representatives of the ceiling passes (not returned)
constexpr int kScratchCertify = 13;      // top-(k+1) lists of the certified scoring
constexpr int kScratchBlocks = 14;       // block codec: row word counts and scan sums
constexpr int kScratchExpand = 15;       // block codec: codes expanded back to the b-bit stream for scoring
constexpr int kScratchLsh = 16;          // banded candidates: chunk keys and the chunk's own index
constexpr int kScratchWideCodes = 17;    // scoring: wide codes in their split 12-bit form
constexpr int kScratchWideQueries = 18;  // scoring: queries in the split form [2^11 q, q]
constexpr int kScratchSlots = 19;

struct DevBuf {
  void* p = nullptr;
  size_t bytes = 0;
  lam_status ensure(size_t need);   // grows (never shrinks); contents not kept
  void release();
  template <class T> T* as() const { return static_cast<T*>(p); }
};

// Device-side status words written by kernels and read back at the end of a
// synchronous call.  Pinned host mirror for the readback.
struct DevFlags {
  uint32_t nonfinite;      // NaN/Inf seen in an input
  uint32_t out_of_range;   // |x| > declared absmax, or |x| >= 255.9375 for the screen
  uint32_t absmax_bits;    // max |x| as float bits (measured absmax)
  uint32_t pair_overflow;  // bit 0: ambiguous-pair list overflowed
  uint32_t n_pairs;        // ambiguous pairs found
  uint32_t n_escalate;     // pairs decided on exact integers
  uint32_t n_kept;         // arrivals retained by this ingest
  uint32_t pairs_needed;   // pair-list capacity that would have sufficed
  unsigned long long dhat2_bits;  // max merged d^2 (binary64 bits, non-negative)
  unsigned long long n_cand;      // candidate pairs of a banded store
  unsigned long long margin_inv;  // ~bits of the smallest |d^2 - delta^2| the exact test saw (0: none)
};

// ------------------------------------------------------------------ profiling
struct ProfRec {
  const char* name;
  hipEvent_t a, b;
};

}  // namespace lam

struct lam_ctx {
  int device = 0;
  hipStream_t stream = nullptr;
  lam::DevFlags* flags_dev = nullptr;   // device status words
  lam::DevFlags* flags_host = nullptr;  // pinned, coherent mirror
  lam::DevFlags* flags_host_dev = nullptr;  // its device-side address (kernels write it directly)
  bool flags_zero = false;              // flags_dev known to hold zeros
  // scratch arena, grown on demand
  lam::DevBuf scratch[lam::kScratchSlots];
  // profiling
  uint32_t pair_cap = 1u << 20;         // ambiguous-pair list capacity (grows on overflow)
  int screen_tile = 0;                  // LAM_SCREEN_TILE_*
  bool profiling = false;
  std::string prof_only;                // empty: every kernel
  std::vector<lam::ProfRec> prof;
  std::vector<hipEvent_t> event_pool;
};

struct lam_store {
  lam_ctx* ctx = nullptr;
  int32_t dim = 0;
  double tau = 0.0;
  double d2 = 0.0;          // delta^2 = 2 - 2 tau (binary64)
  int64_t capacity = 0;
  // banded candidates (Algorithm "admit" with a band index); lsh_r == 0: every
  // retained row is a candidate (the MFMA screen)
  int32_t lsh_r = 0;                 // band width (coordinates per band)
  int32_t lsh_nb = 0;                // bands per row
  double lsh_eps = 0.0;              // Q_eps step of the band codes
  uint64_t lsh_slots = 0;            // index slots (a power of two)
  unsigned long long* lsh_key = nullptr;   // slot key (0 = empty)
  int32_t* lsh_head = nullptr;       // slot -> newest entry (entry = store position * nb + band)
  int32_t* lsh_next = nullptr;       // entry -> older entry with the same key, -1 at the end
  unsigned long long* lsh_rowkey = nullptr;  // band keys of retained rows (position * nb + band)
  int64_t size = 0;           // exact when !pending
  int64_t n_seen = 0;         // exact when !pending
  double delta_hat_run = 0.0; // exact when !pending
  bool pending = false;       // ingest calls ran without waiting; the device bookkeeping holds the truth
  int64_t size_ub = 0;        // upper bound of the size while pending
  hipStream_t last_stream = nullptr;  // stream of the last call that did not wait
  lam::Big6 thr{};            // floor((2 - 2 tau) * 2^298), the exact predicate's right side
  // retained rows (capacity rows each)
  float* x32 = nullptr;       // float32 rows
  _Float16* x16 = nullptr;    // float16 rows scaled by 2^8 (screen operand)
  float* hn = nullptr;        // ||x||^2 / 2 (float32, rounded to nearest)
  float* et = nullptr;        // per-row term of the screen's error bound (float32, rounded up)
  int64_t* ids = nullptr;     // global ids
  float* stat_dev = nullptr;  // device bookkeeping block (retained-row count)
  void* meta_host = nullptr;  // pinned host copy of that block, made when settling
  bool meta_reset = false;    // cleared: the next ingest's first kernel zeroes the block
  uint32_t hn_max = 0;        // max of hn over the coded rows (float bits), set with the codes
  // the device bookkeeping's maxima over the retained rows, as last read by the host
  bool maxima_known = false;  // false until read again after calls that may have changed them
  uint32_t absmax_bits = 0;   // max |x| (float bits)
  uint32_t hnmax_bits = 0;    // max ||x||^2 / 2 (float bits)
  // codes
  uint32_t* codes = nullptr;
  uint64_t codes_cap = 0;
  int64_t coded_rows = 0;     // rows covered by the current codes
  // per-block codec of the codes (blockcodec.hip); valid when blk_rows == coded_rows
  uint8_t* blk_w = nullptr;          // widths, capacity x dim/32
  uint64_t* blk_row_off = nullptr;   // word offset of each row, capacity + 1
  uint32_t* blk_data = nullptr;      // bit planes
  uint64_t blk_cap = 0;              // bytes allocated for blk_data
  uint64_t blk_words = 0;
  int64_t blk_rows = -1;             // rows encoded, -1 when none or stale
  lam_qparams q{};
};

namespace lam {

// profiling helpers (no-ops unless ctx->profiling)
lam_status prof_begin(lam_ctx* ctx, const char* name, size_t* slot);
lam_status prof_end(lam_ctx* ctx, size_t slot);
// events for hipExtLaunchKernel (null unless this kernel is profiled)
lam_status prof_launch_events(lam_ctx* ctx, const char* name, hipEvent_t* start, hipEvent_t* stop);

struct ProfScope {
  lam_ctx* ctx;
  size_t slot = (size_t)-1;
  lam_status st = LAM_OK;
  ProfScope(lam_ctx* c, const char* name, bool on = true) : ctx(c) {
    if (on) st = prof_begin(ctx, name, &slot);
  }
  ~ProfScope() { if (slot != (size_t)-1) prof_end(ctx, slot); }
};

// status words: cleared by a kernel, read back with a stream synchronisation
lam_status clear_flags(lam_ctx* ctx);
lam_status read_flags(lam_ctx* ctx);

// ------------------------------------------------------------------ Q_eps (qeps.hip)
lam_status qeps_plan_host(double eps, float absmax, int mode, int64_t n, lam_qparams* out);
lam_status launch_absmax(lam_ctx* ctx, const float* x, int64_t n, uint32_t* absmax_bits_dev,
                         const char* prof_name = "qeps_absmax");
lam_status launch_encode(lam_ctx* ctx, const float* x, int64_t n, const lam_qparams& p,
                         uint32_t* codes, uint32_t* viol_dev, const char* prof_name = "qeps_encode");
lam_status launch_decode(lam_ctx* ctx, const uint32_t* codes, const lam_qparams& p, float* xhat,
                         const char* prof_name = "qeps_decode");

// ------------------------------------------------------------------ dedup (dedup.hip)
lam_status dedup_ingest(lam_ctx* ctx, lam_store* st, const float* x, int64_t n, int64_t* rep,
                        float* max_cos, lam_ingest_stats* stats);
lam_status store_alloc(lam_store* st);
lam_status store_maxima(lam_store* st);   // settles the store and makes absmax_bits / hnmax_bits current
void store_free(lam_store* st);

// ------------------------------------------------------------------ scoring (score.hip)
// codes: the b-bit code stream to score (NULL: the store's own)
lam_status score_topk(lam_ctx* ctx, const lam_store* st, const float* q, int64_t nq, int32_t k,
                      float* scores, int64_t* ids, float* bound, const uint32_t* codes = nullptr);
// score_topk with every scratch buffer carved from the file-scope device
// array of score.hip (no allocation); noalloc_setup must have run on the
// device (lam_ctx_create does).
lam_status score_topk_noalloc(lam_ctx* ctx, const lam_store* st, const float* q, int64_t nq, int32_t k,
                              float* scores, int64_t* ids, float* bound);
lam_status noalloc_setup(int device);

// ------------------------------------------------------------------ bandwidth anchor (triad.hip)
lam_status launch_triad(lam_ctx* ctx, const float* a, const float* b, float* c, int64_t n, float s);
lam_status score_certify(lam_ctx* ctx, const lam_store* st, const float* q, int64_t nq, int32_t k, float* scores,
                         int64_t* ids, float* bound, uint8_t* certified, float* margin);
lam_status block_encode(lam_ctx* ctx, lam_store* st, lam_block_stats* out);
// decode the blocks to float32 (xhat) or back to the b-bit code stream (codes_out)
lam_status block_decode(lam_ctx* ctx, const lam_store* st, float* xhat, uint32_t* codes_out);

// Empties the band index of a store and puts back the entries of its first
// keep_rows rows (no-op for a store without a band index).
lam_status lsh_reset(lam_ctx* ctx, lam_store* st, int64_t keep_rows);

// Waits for ingest calls that did not wait, copies the device bookkeeping into
// the host fields and reports (once) invalid input those calls met.
lam_status store_settle(lam_store* st);
// Largest ||x||^2 / 2 over the store's rows, for the scoring error bound
// (score.hip); enqueued by lam_store_quantize.

}  // namespace lam
