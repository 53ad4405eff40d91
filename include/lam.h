/*
 * lam.h -- C ABI of liblam, the MI355X (gfx950) hot path of LAM, the lossy
 * agent memory of "LAM: A Lossy Agent Memory Framework With a Retrieval-Score
 * Error Bound".
 *
 * Three operations, each as the paper states it:
 *   1. Q_eps, the error-bounded quantizer of Section 2.2 ("Three layers", L1):
 *      q = round(x / 2 eps) per coordinate, so |x - q*2eps| <= eps.
 *   2. The epsilon error-bounded near-duplicate test of Section 2.3,
 *      Algorithm "admit": arrivals, in order, are dropped iff a retained record
 *      lies within l2 distance delta = sqrt(2 - 2 tau) (Eq. identity,
 *      Section 2.1); the representative is the lowest-indexed such record
 *      (Appendix "Representative selection"); the measured bound delta_hat is
 *      reported (Appendix "The measured bound").
 *   3. Retrieval scoring of queries against the quantized retained store,
 *      dequantized on the fly, with top-k and the per-query bound
 *      eps * ||q||_1 on |q.x - q.x_hat| (Appendix "Rank invariance, in full").
 * and, around them, the paper's further mechanisms: candidates from a band
 * index over Q_eps codes (lam_store_create_banded), the removal ceiling and
 * entropy bracket from greedy at delta and 2 delta (lam_removal_ceiling), the
 * rank-invariance certificate (lam_score_topk_certified) and a per-block
 * fixed-length codec of the store's codes (lam_store_block_*,
 * lam_score_topk_blocks).
 *
 * Conventions for every call:
 *   - Pointers named *_dev are device pointers on the context's device; the
 *     caller owns them.  Pointers without the suffix are host memory.  The
 *     library keeps no caller pointer after a call returns.
 *   - Device work is enqueued on the context's stream, in call order.  Calls
 *     that fill a host struct (marked "synchronous") wait for that stream
 *     before returning; the others return once the work is enqueued.
 *   - Every call returns a lam_status.  On LAM_EINVAL / LAM_ERANGE /
 *     LAM_ECAPACITY / LAM_ESTATE detected on the host nothing is enqueued and
 *     no output is written.  When the device detects the error (non-finite
 *     input, |x| above a declared absmax) the call returns that status, the
 *     store is left as it was, and the contents of caller output buffers are
 *     unspecified.  LAM_EDEVICE reports a HIP runtime error; the context
 *     should then be destroyed.
 *   - lam_last_error() returns a thread-local message for the last non-OK
 *     status of the calling thread.
 *   - One context per host thread; a store must not be used by two calls at
 *     once.  Calls that overlap on one device through different contexts are
 *     independent (each context owns its scratch memory).
 */
#ifndef LAM_H
#define LAM_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define LAM_ABI_VERSION 1

typedef enum lam_status {
  LAM_OK = 0,
  LAM_EINVAL = 1,     /* bad argument, or non-finite / out-of-range input data  */
  LAM_ERANGE = 2,     /* |x| above the declared absmax, or code range >= 2^31   */
  LAM_ENOMEM = 3,     /* device or host allocation failed                       */
  LAM_ECAPACITY = 4,  /* the store cannot take the batch                        */
  LAM_EDEVICE = 5,    /* HIP runtime error                                      */
  LAM_ESTATE = 6      /* call not valid in the object's state                   */
} lam_status;

int lam_abi_version(void);
const char* lam_status_name(lam_status s);
const char* lam_last_error(void);

/* ------------------------------------------------------------------ context */
typedef struct lam_ctx lam_ctx;

/* device: HIP device ordinal.  hip_stream: a hipStream_t on that device, or
 * NULL for the null stream.  The stream is borrowed, not owned. */
lam_status lam_ctx_create(int device, void* hip_stream, lam_ctx** out);
void lam_ctx_destroy(lam_ctx* ctx);
lam_status lam_ctx_synchronize(lam_ctx* ctx);

/* Per-kernel timing with HIP events recorded on the context's stream around
 * each launch of the named kernels while enabled.  read() is synchronous and
 * returns the summed elapsed milliseconds and launch count of one kernel name
 * (0 / 0 if never launched).  For benchmarks; off by default. */
lam_status lam_ctx_profile(lam_ctx* ctx, int enable);
/* Restricts the timing to the launches of the kernel names in a
 * comma-separated list (NULL or "": every kernel), so that a timed run carries
 * only those kernels' events.  The list is copied. */
lam_status lam_ctx_profile_only(lam_ctx* ctx, const char* kernel);
lam_status lam_ctx_profile_reset(lam_ctx* ctx);
lam_status lam_ctx_profile_read(lam_ctx* ctx, const char* kernel, double* total_ms, int64_t* launches);

/* Tile of the similarity screen (Algorithm "admit": the store and in-chunk
 * screens of lam_dedup_ingest on an unbanded store).  Two MFMA tilings
 * compute the same decisions: 128 x 128 tiles (two workgroups per CU), and,
 * at D = 768 and 1,024, 256 x 256 tiles (one workgroup per CU, half the
 * operand loads per flop), faster for launches of many tiles and slower for
 * small ones.  policy: LAM_SCREEN_TILE_AUTO (default: the large tile for a
 * launch of at least 768 large tiles), LAM_SCREEN_TILE_SMALL or
 * LAM_SCREEN_TILE_LARGE (every launch, where the dimension allows it).  A
 * tuning and testing setting of the context; LAM_EINVAL for another value. */
enum { LAM_SCREEN_TILE_AUTO = 0, LAM_SCREEN_TILE_SMALL = 1, LAM_SCREEN_TILE_LARGE = 2 };
lam_status lam_ctx_set_screen_tile(lam_ctx* ctx, int policy);

/* ------------------------------------------------------------------ Q_eps   */
/* Section 2.2 (L1): Q_eps(x) = round(x / 2eps), with round half to even of the
 * exact real quotient of the float32 x by the binary64 step s = 2*eps.  Codes
 * are two's-complement integers of width b, element i occupying bits
 * [i*b, (i+1)*b) of a little-endian stream of uint32 words, least significant
 * bit first; unused bits of the last word are zero. */
enum { LAM_PACK_BITS = 0,   /* b = max(1, ceil(log2(2M + 1)))            */
       LAM_PACK_BYTES = 1   /* b = smallest of 8, 16, 32 that holds +-M  */ };

typedef struct lam_qparams {
  double eps;           /* error budget; |x - code*step| <= eps on exact reals */
  double step;          /* s = 2 * eps                                          */
  float absmax;         /* A, declared or measured                              */
  int32_t bits;         /* b                                                    */
  int32_t mode;         /* LAM_PACK_BITS or LAM_PACK_BYTES                      */
  int32_t max_code;     /* M = Q_eps(A) < 2^31                                  */
  int64_t n;            /* number of codes                                      */
  uint64_t code_bytes;  /* 4 * ceil(n * b / 32)                                 */
} lam_qparams;

/* Host only: the width plan for n values bounded by absmax.
 * EINVAL: eps not finite or outside [2^-60, 2^20], absmax not finite or < 0,
 * n < 0, bad mode.  ERANGE: M >= 2^31. */
lam_status lam_qeps_plan(double eps, float absmax, int mode, int64_t n, lam_qparams* out);

/* Encode n float32 values.  absmax > 0 declares A (every |x| must be <= A,
 * else ERANGE); absmax <= 0 measures A = max|x| on the device first (one extra
 * read of x).  codes_dev receives code_bytes bytes and needs at least that
 * capacity (EINVAL otherwise).  x_dev must be 4-byte aligned; codes_dev
 * 4-byte aligned.  Synchronous (fills *out).  EINVAL also for NaN/Inf in x. */
lam_status lam_quantize(lam_ctx* ctx, const float* x_dev, int64_t n, double eps, float absmax,
                        int mode, uint32_t* codes_dev, uint64_t codes_cap_bytes, lam_qparams* out);

/* lam_quantize for pipelines that do not wait: returns once the encode is
 * queued on the context's stream, with *out planned from the declared
 * absmax (> 0, required; EINVAL otherwise).  Instead of a status, the encode
 * adds, in stream order, a positive count to status_dev[0] if any element is
 * NaN or Inf and to status_dev[1] if any |x| > absmax (Inf included): two
 * uint32 in device memory that the caller owns and clears (the counts are of
 * the device threads that met such elements).  The codes are valid when
 * neither count grew.  Argument errors (EINVAL, ERANGE for a code range
 * beyond 2^31) are returned at once, before anything is queued. */
lam_status lam_quantize_async(lam_ctx* ctx, const float* x_dev, int64_t n, double eps, float absmax, int mode,
                              uint32_t* codes_dev, uint64_t codes_cap_bytes, uint32_t* status_dev,
                              lam_qparams* out);

/* Decode p->n codes: x_hat = float32(float64(code * step)) (round to binary64,
 * then to binary32; the bound holds on the exact code*step).  Asynchronous. */
lam_status lam_dequantize(lam_ctx* ctx, const uint32_t* codes_dev, const lam_qparams* p, float* xhat_dev);

/* ------------------------------------------------------------------ store   */
/* The retained set R of Algorithm "admit": float32 rows of the kept
 * arrivals in arrival order, with their global ids (0-based arrival ordinals
 * counted over every ingest call on the store).  Library-owned device memory,
 * sized for `capacity` rows at creation.  dim must be a positive multiple of
 * 32 (at most 4096); tau in (-1, 1]; the merge radius is delta^2 = 2 - 2 tau. */
typedef struct lam_store lam_store;

lam_status lam_store_create(lam_ctx* ctx, int32_t dim, double tau, int64_t capacity, lam_store** out);

/* A store whose ingest takes its candidates from a band index over Q_eps codes
 * (Section 2.2, the candidate layer L1; Appendix "Band width and quantizer
 * step") instead of screening every retained row.  Each row's codes at step
 * eps_band (code = round-half-even of the exact x / (2 eps_band), as
 * lam_quantize) are cut into dim / band_width bands of band_width consecutive
 * coordinates; a retained row is a candidate of an arrival when the codes of
 * at least one band are equal in both (a 64-bit digest only finds equal bands;
 * the codes are compared before a pair counts).  Every candidate is decided by
 * the exact merge predicate and the lowest-indexed candidate within delta is
 * the representative; an arrival with none is kept and its bands enter the
 * index.  So rep is that of Algorithm "admit" with the retained set cut down
 * to the candidates; a coarse enough step (every code 0) gives exhaustive
 * greedy.  The index holds retained rows only.  Library-owned device memory
 * grows by about 28 bytes per (row of capacity, band).
 * band_width must divide dim; eps_band in [2^-23, 2^40];
 * capacity * (dim / band_width) < 2^31.  On such a store lam_dedup_ingest
 * rejects max_cos_dev (EINVAL), and n_ambiguous_pairs counts candidate pairs:
 * the arrival against retained rows of earlier chunks (a chunk is 4,096
 * arrivals of a call), plus pairs of arrivals j < i within one chunk with an
 * equal band, whether or not j is later kept. */
lam_status lam_store_create_banded(lam_ctx* ctx, int32_t dim, double tau, int64_t capacity, double eps_band,
                                   int32_t band_width, lam_store** out);
void lam_store_destroy(lam_store* store);

typedef struct lam_store_info {
  int64_t size;          /* retained rows                                       */
  int64_t capacity;
  int64_t n_seen;        /* arrivals ingested so far (next global id)           */
  int32_t dim;
  int32_t quantized;     /* 1 once lam_store_quantize has run on every row      */
  double tau;
  double delta_hat_run;  /* max substitution distance over all calls            */
  lam_qparams q;         /* valid when quantized                                */
} lam_store_info;

/* Synchronous: waits for ingest calls that did not wait (see lam_dedup_ingest)
 * and returns EINVAL, once, if any of them met invalid input.  The wait is for
 * the stream of the last such call, so it also covers work queued on that
 * stream after the call. */
lam_status lam_store_get_info(const lam_store* store, lam_store_info* out);

/* Empty the store (size, n_seen, delta_hat and codes reset; memory kept), as
 * if newly created.  Asynchronous; drops the pending error report of earlier
 * calls that did not wait. */
lam_status lam_store_clear(lam_ctx* ctx, lam_store* store);

typedef struct lam_ingest_stats {
  int64_t n_in;                 /* arrivals in this call                        */
  int64_t n_kept;
  int64_t n_dropped;
  int64_t store_size;           /* retained rows after the call                 */
  int64_t n_ambiguous_pairs;    /* pairs whose screened distance lay within the
                                   screen's error bound of delta^2 and were
                                   decided by the exact binary64 test           */
  int64_t n_exact_escalations;  /* pairs within binary64 rounding distance of
                                   delta^2, decided on exact integers (device)  */
  double delta_hat_call;        /* max ||x_i - x_rep|| over this call's merges  */
  double delta_hat_run;         /* same over the store's lifetime               */
  double min_margin_d2;         /* smallest |d^2 - delta^2| (binary64) among the
                                   pairs the exact test decided in this call;
                                   +inf when it decided none (every pair was
                                   then at least the screen's bound away)       */
} lam_ingest_stats;

/* Algorithm "admit" over x_dev (n rows of dim float32, row-major, expected
 * unit-normalised; used exactly as given).  For each arrival i, in order:
 * rep_dev[i] = global id of the lowest-indexed retained row y with
 * sum_d (x_i,d - y_d)^2 <= 2 - 2 tau (exact reals, inclusive), which drops i;
 * or -1, and i is appended to the store with global id n_seen + i.
 * max_cos_dev (optional, NULL to skip): max over rows retained at i's arrival
 * of the dot product x_i . y in the screen's precision (|error| <= 1.1e-3 for
 * unit rows), -inf if none.
 *
 * With stats (host struct) the call waits for the device and fills it; errors
 * are returned by the call itself.  With stats == NULL the call returns as soon
 * as its kernels are queued on the context's stream (rep and max_cos are
 * written in stream order) whenever the library can guarantee that no host
 * step is needed: the ambiguous-pair list can hold every pair the call's
 * chunks could produce (n (size + n) entries, at most 2^26) and the store has
 * room even if every earlier row was kept.  Otherwise it waits as above.  An
 * asynchronous call whose input turns out invalid leaves the store unchanged,
 * writes no outputs, and is reported (EINVAL, once for all such calls) by the
 * next call on the store that waits: lam_store_get_info, lam_store_quantize,
 * lam_store_dequantize, lam_store_export, lam_score_topk or an ingest with
 * stats; later calls are decided as if it had not happened.
 * EINVAL: n < 0, NaN/Inf or |x| >= 255.9375 (= 2^8 - 2^-4, above which the
 * screen's float16 operand 2^8 x would overflow) in a coordinate (store
 * unchanged).
 * ECAPACITY: size + n > capacity (checked before any work; a call that does
 * not wait checks an upper bound of the size and waits if that bound is over). */
lam_status lam_dedup_ingest(lam_ctx* ctx, lam_store* store, const float* x_dev, int64_t n,
                            int64_t* rep_dev, float* max_cos_dev, lam_ingest_stats* stats);

/* Q_eps over every retained row (the store's codec, Algorithm "admit",
 * "store the compressed embedding"); rows start on word boundaries (dim is a
 * multiple of 32).  Same absmax semantics as lam_quantize: a declared absmax
 * below the store's largest |x| (kept exactly by the appends) is ERANGE,
 * decided on the host before any code is written, and leaves the store
 * unquantized.  Waits for ingest calls that did not wait (as
 * lam_store_get_info), then returns with the encode queued (fills *out; the
 * rows were checked at ingest, so the encode cannot fail on the data).
 * Rows retained later are not coded until this is called again. */
lam_status lam_store_quantize(lam_ctx* ctx, lam_store* store, double eps, float absmax, int mode,
                              lam_qparams* out);

/* Decode the store's codes into xhat_dev (size x dim float32, row-major):
 * x_hat = float32(float64(code * step)), the reconstruction the scores use.
 * ESTATE if the store is not quantized.  Asynchronous. */
lam_status lam_store_dequantize(lam_ctx* ctx, const lam_store* store, float* xhat_dev);

/* Copy the retained ids (size int64) and, if codes_dev is not NULL and the
 * store is quantized, the packed codes (q.code_bytes bytes) out.  Async. */
lam_status lam_store_export(lam_ctx* ctx, const lam_store* store, int64_t* ids_dev,
                            uint32_t* codes_dev, uint64_t codes_cap_bytes);

/* Score nq float32 queries (row-major, dim each) against the quantized store:
 * score(j, y) = step * sum_d q_j,d * code_y,d, i.e. q_j . x_hat_y with the
 * exact dequantized row (|error| <= 1e-5 for unit rows: float32 accumulation
 * of the query's fp16 hi and lo parts, or, for the rows of a large store that
 * reach a query's top-k, a binary64 sum rounded once; the ranking is the one
 * these scores give).  Per query the k best by (score desc, id asc) go to scores_dev and
 * ids_dev (nq x k, row-major), padded with (-inf, -1) past the store size.
 * bound_dev (optional): eps * ||q_j||_1 rounded up to float32.
 * 1 <= k <= 64.  Codes of up to 12 bits are multiplied as exact float16
 * values; codes of 13 to 22 bits are scored in a split form, each code c as
 * the two 12-bit parts c >> 11 and c & 2047 against the query scaled by 2^11
 * and the query itself (the same scores; twice the matrix work, 3 dim bytes
 * per stored row and 8 dim bytes per query of context scratch; a query with
 * |q| * 2^11 beyond float32 range counts as holding Inf).  ESTATE if the
 * store is not quantized (or has rows added since), or if its codes are wider
 * than 22 bits (quantize with a larger eps: 22 bits hold absmax / (2 eps) <
 * 2,097,151.5).  A query row holding NaN/Inf gets (NaN, -1) in all k slots
 * and a NaN bound instead of an error status.  Asynchronous. */
lam_status lam_score_topk(lam_ctx* ctx, const lam_store* store, const float* q_dev, int64_t nq,
                          int32_t k, float* scores_dev, int64_t* ids_dev, float* bound_dev);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid allocation):
 * lam_score_topk with every scratch buffer taken from a fixed 32 MiB array
 * that each device holds from the library's load until the process ends (set
 * up by lam_ctx_create); the call itself allocates nothing.  Results equal
 * lam_score_topk's.  Limits: nq <= 256 (EINVAL beyond); codes of at most 12
 * bits (ESTATE for wider ones, whose split form needs scratch in proportion
 * to the store).  The store must be
 * quantized and settled: ESTATE while ingest calls that did not wait are in
 * flight (lam_store_get_info settles them) -- settling can need the host.
 * Every call on one device shares that device's array: calls that overlap on
 * one device (through any contexts or streams) race and give undefined
 * results; calls in one stream's order are safe.  No profiling events are
 * recorded.  Asynchronous. */
lam_status lam_score_topk_noalloc(lam_ctx* ctx, const lam_store* store, const float* q_dev, int64_t nq,
                                  int32_t k, float* scores_dev, int64_t* ids_dev, float* bound_dev);

/* Top-k with the rank-invariance certificate (Appendix "Rank invariance, in
 * full"): as lam_score_topk (1 <= k <= 63), plus per query certified_dev[j] = 1
 * when the float32 margin m_j = s_k - s_{k+1} between ranks k and k+1 exceeds
 *   2 (beta_j + ||q_j||_2 delta_hat + e_j),
 * beta_j = eps ||q_j||_1, delta_hat the store's measured bound, and e_j =
 * kappa ||q_j||_1 (A + eps) a bound on the float32 score's error (A the store's
 * absmax, kappa = 1.01 (2^-22 + gamma_2D + 2^-23)).  A flag implies that the
 * exact margin exceeds 2 (beta_j + ||q_j||_2 delta_hat), so no record crosses
 * the rank-k boundary when every score moves by the substitution and
 * quantization bounds.  A store with at most k rows certifies every valid
 * query; a NaN/Inf query row is never certified.  margin_dev (optional): m_j
 * (+inf past the store size, NaN for an invalid query).  Asynchronous. */
lam_status lam_score_topk_certified(lam_ctx* ctx, const lam_store* store, const float* q_dev, int64_t nq,
                                    int32_t k, float* scores_dev, int64_t* ids_dev, float* bound_dev,
                                    uint8_t* certified_dev, float* margin_dev);

/* ------------------------------------------------------------------ block codec */

typedef struct lam_block_stats {
  int64_t rows;             /* retained rows encoded                                 */
  int64_t blocks;           /* rows x dim / 32                                       */
  uint64_t data_bytes;      /* bit-plane words                                       */
  uint64_t meta_bytes;      /* one width byte per block + (rows + 1) 64-bit offsets   */
  uint64_t total_bytes;
  double bits_per_code;     /* 8 total_bytes / (rows x dim)                          */
  int32_t plain_bits;       /* b of the fixed-width codes                            */
  int32_t pad;
  double codec_ratio;       /* 32 / bits_per_code: float32 rows over encoded rows     */
  double composite_ratio;   /* n_seen x dim x 4 / total_bytes: deduplication x codec  */
} lam_block_stats;

/* Section 2.2 (L2) and Section "Composite reduction": encode the store's Q_eps
 * codes in blocks of 32 codes of a row: zigzag values (u = 2q, or -2q - 1 for
 * q < 0), each block with the bit width w of its largest u (0 if all zero) as w
 * 32-bit bit planes (bit j of word t = bit t of code j), one width byte per
 * block and a 64-bit word offset per row.  Lossless on the codes, so the
 * reconstruction and the score bound are those of Q_eps.  Requires a store
 * quantized after its last ingest (ESTATE otherwise); an encoding lasts until
 * the store is re-quantized or cleared.  Synchronous (fills out). */
lam_status lam_store_block_encode(lam_ctx* ctx, lam_store* store, lam_block_stats* out);

/* Decode the block encoding to x_hat (size x dim float32), bit for bit the
 * values lam_store_dequantize gives.  ESTATE without a current encoding.
 * Asynchronous. */
lam_status lam_store_block_decode(lam_ctx* ctx, const lam_store* store, float* xhat_dev);

/* Copy the encoding out: widths (size x dim/32 bytes), row offsets (size + 1
 * uint64 word offsets; the last is the total word count) and the bit-plane
 * words (data_cap_bytes must hold them).  NULL pointers are skipped.  Async. */
lam_status lam_store_block_export(lam_ctx* ctx, const lam_store* store, uint8_t* widths_dev, uint64_t* row_off_dev,
                                  uint32_t* data_dev, uint64_t data_cap_bytes);

/* lam_score_topk over the block encoding: the blocks are expanded to the
 * fixed-width code stream in context scratch (one pass) and scored by the same
 * fused kernel, so the results equal lam_score_topk's.  ESTATE without a current
 * encoding.  Asynchronous. */
lam_status lam_score_topk_blocks(lam_ctx* ctx, const lam_store* store, const float* q_dev, int64_t nq, int32_t k,
                                 float* scores_dev, int64_t* ids_dev, float* bound_dev);

/* ------------------------------------------------------------------ removal ceiling */

typedef struct lam_ceiling_stats {
  int64_t n;               /* arrivals                                               */
  int64_t kept;            /* |R(delta)|: greedy at tau                               */
  int64_t kept_2delta;     /* |R(2 delta)|: greedy at tau' = 4 tau - 3                */
  double tau, tau_2delta;
  double removal;          /* attained: 1 - kept / n                                  */
  double ceiling;          /* 1 - kept_2delta / n, an upper bound on the removal of
                              any delta-bounded compactor of this stream             */
  double frac_of_ceiling;  /* removal / ceiling (0 when the ceiling is 0)             */
  double bits_lo, bits_hi; /* log2 kept_2delta <= H_delta(S) <= log2 kept             */
  double delta_hat, delta_hat_2delta;   /* measured bounds of the two passes          */
} lam_ceiling_stats;

/* Theorem "removal ceiling" and Corollary "measured bracket": greedy
 * first-occurrence over x_dev (n rows of dim float32, arrival order, the same
 * input contract as lam_dedup_ingest) at radius delta = sqrt(2 - 2 tau) and at
 * radius 2 delta (threshold 4 tau - 3, exact in binary64), in batches of
 * `batch`, on two temporary stores of capacity n that the call frees.
 * Synchronous.  EINVAL: tau outside (1/2, 1], n < 1, batch < 1, or invalid rows
 * (as lam_dedup_ingest); ENOMEM if the two stores do not fit. */
lam_status lam_removal_ceiling(lam_ctx* ctx, const float* x_dev, int64_t n, int32_t dim, double tau,
                               int64_t batch, lam_ceiling_stats* out);

/* ------------------------------------------------------------------ bandwidth anchor */

/* The triad c = a + s * b over n float32 values (a_dev, b_dev, c_dev
 * 16-byte aligned device arrays; 12 bytes moved per element): the streaming
 * bandwidth the paper measures on its platform so that every bandwidth figure
 * is stated against a measured ceiling as well as the published one
 * (Appendix "Measured hardware constants", Table "anchors", 3 x 512 MB).
 * Timed under the kernel name "triad" when profiling.  EINVAL: n < 0, NULL or
 * misaligned arrays.  Asynchronous. */
lam_status lam_triad(lam_ctx* ctx, const float* a_dev, const float* b_dev, float* c_dev, int64_t n, float s);

#ifdef __cplusplus
}
#endif
#endif /* LAM_H */
