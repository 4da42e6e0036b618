/*
 * hill.h -- C ABI of libhill: the per-decode-step token-importance path of
 * HillInfer (arxiv 2602.18750) on AMD Instinct MI355X (gfx950).
 *
 * One decode step of one layer, for a batch of sequences that each own a
 * KV cache (Sec. 2.1, "KV Cache Mechanism"):
 *
 *   score      l[b,h,j] = q[b,h,:] . K[b,kv(h),j,:]           (Sec. 4.4, Eq. 1)
 *              ATTN: w = softmax_j(sm_scale * l)  (Eq. 1 weights)
 *              RAW:  w = l                        (Sec. 4.4 simplification)
 *              S[b,r,j] += sum_{h in heads(r)} w[b,h,j]         (Sec. 4.1)
 *   select     idx[b,r,:] = the k largest S[b,r,:], ascending token order,
 *              ties to the lower token index    (Sec. 3.1 top-alpha; Sec. 4.2)
 *   attention  out[b,h,:] = softmax over I of sm_scale * q.K_j, times V_j,
 *              I = idx[b,r(h),:]                 (Eq. 1 over the selection;
 *                                                 Sec. 4.1 workflow step 6)
 *
 * kv(h) = h / G with G = n_q_heads / n_kv_heads (contiguous GQA groups; MHA is
 * G = 1, MQA is n_kv_heads = 1).  Granularity: HILL_SEL_TOKEN keeps one
 * importance row and one index set per sequence (R = 1, summed over all query
 * heads); HILL_SEL_KVHEAD keeps one per (sequence, KV head) (R = n_kv_heads,
 * summed over that head's G query heads); r(h) = 0 or kv(h) respectively.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * Memory.  Every data pointer is a DEVICE pointer owned by the caller; the
 *   library never allocates, frees or synchronises.  Scratch memory is the
 *   caller's workspace `ws` of at least hill_workspace_bytes() bytes, 16-byte
 *   aligned; its contents on entry are irrelevant and on return undefined.
 * Streams.  `stream` is a hipStream_t (NULL = the default stream).  All work
 *   is enqueued on it in order and the call returns without waiting.
 * Layouts.  q: fp16/bf16 [B, Hq, D] with strides (q_stride_b, q_stride_h),
 *   D contiguous.  K, V: fp16/bf16 [B, Hkv, Ncap, D] with strides
 *   (*_stride_b, *_stride_h, *_stride_n), D contiguous, only the first
 *   n_tokens rows read.  S: fp32 [B, R, >= n_tokens] with strides
 *   (s_stride_b, s_stride_r), token index contiguous.  idx: int32
 *   [B, R, k_sel] contiguous.  out: fp32 [B, Hq, D] contiguous.  Strides are
 *   in elements.
 * Alignment.  q, K, V, S, out and ws base addresses 16-byte aligned; q, K, V
 *   strides multiples of 8 elements; S strides multiples of 4 elements.
 * Supported.  head_dim == 128; dtype fp16 or bf16; n_q_heads % n_kv_heads
 *   == 0, n_q_heads <= 256, n_q_heads / n_kv_heads <= 128; 1 <= k_sel <=
 *   n_tokens; n_tokens <= 2097152; k_stride_n and v_stride_n below 2^31
 *   elements.
 * Errors.  All arguments are checked on the host before anything is
 *   enqueued; on any error nothing is enqueued and no output is written.
 *   HILL_ERR_INVALID_ARG: null/misaligned pointer, bad shape, stride or k_sel.
 *   HILL_ERR_UNSUPPORTED: a valid but unimplemented head_dim, dtype, head
 *                         count, context length or token stride.
 *   HILL_ERR_WORKSPACE:   ws too small.
 *   HILL_ERR_HIP:         a kernel launch failed (enqueued work before it in
 *                         the same call may still run).
 *   Device-side faults surface at the caller's next synchronisation.
 *   hill_last_error() returns a message for the calling thread's last error.
 * Determinism.  No floating-point atomics: results are bitwise reproducible
 *   for identical inputs and shapes.
 * Inputs containing Inf/NaN are outside the contract; they never cause an
 *   out-of-bounds access (NaN importance ranks below every number).
 */
#ifndef HILL_H
#define HILL_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define HILL_ABI_VERSION 6

/* The library exports these entry points only (built with hidden visibility). */
#define HILL_API __attribute__((visibility("default")))

typedef enum hill_status {
    HILL_OK = 0,
    HILL_ERR_INVALID_ARG = 1,
    HILL_ERR_UNSUPPORTED = 2,
    HILL_ERR_WORKSPACE = 3,
    HILL_ERR_HIP = 4
} hill_status;

typedef enum hill_dtype { HILL_F16 = 0, HILL_BF16 = 1 } hill_dtype;

/* ATTN: column sums of softmax(sm_scale * q.K^T) (Sec. 4.1 importance metric).
 * RAW: column sums of the raw q.K^T (Sec. 4.4 simplification; no scale). */
typedef enum hill_score_mode { HILL_SCORE_ATTN = 0, HILL_SCORE_RAW = 1 } hill_score_mode;

typedef enum hill_granularity { HILL_SEL_TOKEN = 0, HILL_SEL_KVHEAD = 1 } hill_granularity;

/* Problem descriptor.  Set struct_size = sizeof(hill_desc). */
typedef struct hill_desc {
    uint32_t struct_size;
    int32_t batch;        /* B  >= 1 */
    int32_t n_q_heads;    /* Hq >= 1 */
    int32_t n_kv_heads;   /* Hkv >= 1, divides Hq */
    int32_t head_dim;     /* D == 128 */
    int32_t n_tokens;     /* n >= 1: cached tokens scored this step */
    int32_t dtype;        /* hill_dtype of q, K, V */
    int32_t score_mode;   /* hill_score_mode */
    int32_t granularity;  /* hill_granularity */
    float sm_scale;       /* softmax scale; 0 selects 1/sqrt(head_dim) */
    int64_t q_stride_b, q_stride_h;
    int64_t k_stride_b, k_stride_h, k_stride_n;
    int64_t v_stride_b, v_stride_h, v_stride_n;
    int64_t s_stride_b, s_stride_r;
    /* Selection pinning (optional; 0 and 0 give the plain top-k).  The first
     * min(n_sink, n) tokens and the last min(n_recent, n) tokens are always
     * selected (attention sinks and the recent window, Sec. 4.2's temporal
     * locality and hit-rate stability); the rest of the budget takes the
     * largest S among the other tokens, ties to the lower index.  hill_topk,
     * hill_step and hill_step_sketch require k_sel >= the number of pinned
     * tokens. */
    int32_t n_sink;       /* >= 0 */
    int32_t n_recent;     /* >= 0 */
} hill_desc;

/* ABI version of the loaded library (HILL_ABI_VERSION it was built with). */
HILL_API int hill_abi_version(void);

/* Static description of a status code. */
HILL_API const char* hill_status_str(int status);

/* Message describing the calling thread's most recent failed call (empty
 * string if none).  Valid until the next libhill call on this thread. */
HILL_API const char* hill_last_error(void);

/* Workspace bytes that hill_score / hill_topk / hill_gather_attn / hill_step
 * need for this descriptor and token budget (the maximum over the four).
 * Pure host function; writes *bytes.  k_sel is only used by the attention
 * and select parts and may be any value in [1, n_tokens]. */
HILL_API hill_status hill_workspace_bytes(const hill_desc* d, int32_t k_sel, size_t* bytes);

/* Importance scoring (Sec. 4.1 metric; Sec. 4.4 raw variant):
 * S[b,r,j] += sum_{h in heads(r)} w[b,h,j] for every j < n_tokens.
 * q, k: inputs.  s: in/out, the caller's cumulative importance (zero it
 * before the first step and for newly appended tokens). */
HILL_API hill_status hill_score(const hill_desc* d, const void* q, const void* k, float* s,
                       void* ws, size_t ws_bytes, void* stream);

/* Top-k selection (Sec. 3.1 top-alpha; Sec. 4.2 global top-alpha indices):
 * for each row (b, r), the k_sel tokens with the largest S, ties broken toward
 * the lower token index, NaN below every number, -0.0 equal to +0.0.
 * idx_out: [B, R, k_sel] int32, ascending within a row.
 * val_out: nullable; if given, [B, R, k_sel] fp32 with S at those tokens. */
HILL_API hill_status hill_topk(const hill_desc* d, const float* s, int32_t k_sel,
                      int32_t* idx_out, float* val_out,
                      void* ws, size_t ws_bytes, void* stream);

/* Sparse decode attention over the selected tokens (Eq. 1 restricted to I,
 * softmax renormalised over I).  idx: [B, R, k_sel] int32, each row k_sel
 * distinct indices in [0, n_tokens) in any order (not checked on device: an
 * out-of-range index is clamped into [0, n_tokens), so it never reads out of
 * bounds, and the result is then unspecified).  out: [B, Hq, D] fp32. */
HILL_API hill_status hill_gather_attn(const hill_desc* d, const void* q, const void* k, const void* v,
                             const int32_t* idx, int32_t k_sel, float* out,
                             void* ws, size_t ws_bytes, void* stream);

/* One full decode step in the paper's order (Sec. 4.1 workflow, steps 5-6):
 * update S with this query, select k_sel tokens on the updated S, attend over
 * them.  Equivalent to hill_score, hill_topk (val_out = NULL) and
 * hill_gather_attn in sequence, with fewer launches. */
HILL_API hill_status hill_step(const hill_desc* d, const void* q, const void* k, const void* v,
                      float* s, int32_t k_sel, int32_t* idx_out, float* out,
                      void* ws, size_t ws_bytes, void* stream);

/* Kernel timestamps for profiling a decode step.  A step runs as a chain of
 * kernel launches on the caller's stream; each launch belongs to one stage:
 *
 *   HILL_STAGE_SCAN     streams the keys: q.K^T of every cached token (ATTN:
 *                       logits and per-256-token softmax partials; RAW with
 *                       one row per KV head: added straight into S)
 *   HILL_STAGE_STATS    ATTN only, for rows longer than 32768 tokens or calls
 *                       whose update would re-read more than 128 MiB of
 *                       softmax partials (e.g. 32 sequences of 32768
 *                       tokens): the softmax normaliser of every head
 *   HILL_STAGE_UPDATE   S += the step's weights, and the selection's first
 *                       radix digit histogram (RAW per-KV-head rows: only
 *                       the histogram; a streamed step with a valid bound:
 *                       the candidate list and its class counts instead)
 *   HILL_STAGE_REFINE   the threshold's first-digit bin and the second-digit
 *                       histogram (hill_step, and reset steps of the
 *                       streamed selection)
 *   HILL_STAGE_SELECT   the exact threshold, each chunk's selected tokens and
 *                       the attention partials over them
 *   HILL_STAGE_MERGE    the partials merged into the output, the ordered
 *                       index list written
 *
 * Each non-NULL start[i] / stop[i] is a caller-created hipEvent_t
 * (hipEventCreate, timing enabled) that stage i's launch stamps when it
 * starts / ends: the kernels are launched with hipExtLaunchKernel's start and
 * stop events, so no extra work is enqueued, and elapsed times between them
 * are GPU execution times.  Events of stages a call does not run are left
 * untouched. */
enum {
    HILL_STAGE_SCAN = 0,
    HILL_STAGE_STATS = 1,
    HILL_STAGE_UPDATE = 2,
    HILL_STAGE_REFINE = 3,
    HILL_STAGE_SELECT = 4,
    HILL_STAGE_MERGE = 5,
    HILL_STAGES = 6
};

typedef struct hill_step_events {
    void* start[HILL_STAGES];
    void* stop[HILL_STAGES];
} hill_step_events;

/* hill_step with kernel timestamps (ev may be NULL: then identical to hill_step).
 * Same arguments, validation and results as hill_step. */
HILL_API hill_status hill_step_profiled(const hill_desc* d, const void* q, const void* k, const void* v,
                               float* s, int32_t k_sel, int32_t* idx_out, float* out,
                               void* ws, size_t ws_bytes, void* stream, const hill_step_events* ev);

/* Streamed selection (Sec. 4.2 HIE: scores streamed as (token, score) blocks
 * and merged against a running threshold): hill_step with the selection's
 * refine pass replaced.  With ATTN scores S only grows from step to step, so
 * the previous step's threshold is a lower bound on this one; the update
 * lists every token whose first radix digit reaches that bound, grouped by
 * that digit (the bound's bin, the next three, or above), and the selection
 * resolves the exact threshold from the counts of those groups, a
 * second-digit histogram of the four bins and the list.  Results are
 * identical to hill_step.
 *
 * state: uint32 [B, R, 8], 16-byte aligned, caller-owned, one per S buffer;
 * zero it at the start of a sequence.  Each call reads the bound and writes
 * the next one.  The bound is used only while it holds: the same pins,
 * n_tokens not smaller than at the previous call (growing only without pins),
 * and k_sel at most the number of tokens whose first radix digit reached the
 * previous threshold's (usually k_sel plus a few hundred, so a budget that
 * grows with the context keeps it); otherwise, and on the first call, every
 * workgroup of the selection walks the whole row instead, which is exact but
 * slow on long rows.  If S is changed outside these calls the results stay
 * exact: when fewer than k_sel keys then reach the bound's first digit, the
 * selection counts that digit again over the whole row (slow); a reset step
 * after such a change avoids the walk.
 *
 * flags: 0, or HILL_STREAM_RESET: this call selects through the refine pass
 * exactly as hill_step does (no bound read, no candidate list) and writes a
 * fresh bound from its threshold.  Use it for the first steps of a sequence
 * (while S is young it can double from one step to the next, so the previous
 * threshold bounds the next one only loosely) and after S was changed
 * outside these calls; results are the same either way.  ATTN score mode
 * only (HILL_ERR_UNSUPPORTED otherwise).  ev: as hill_step_profiled (without
 * HILL_STREAM_RESET the REFINE stage does not run). */
#define HILL_STREAM_RESET 1u
HILL_API hill_status hill_step_streamed(const hill_desc* d, const void* q, const void* k, const void* v, float* s,
                               uint32_t* state, uint32_t flags, int32_t k_sel, int32_t* idx_out, float* out,
                               void* ws, size_t ws_bytes, void* stream, const hill_step_events* ev);

/* hill_step without a workspace argument, for callers that cannot allocate
 * device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc).  The scratch is a fixed device buffer of
 * HILL_NOALLOC_SCRATCH_BYTES that the library holds on each GPU it runs on
 * until the process ends (looked up on a device's first call, never
 * allocated by the call).  A step whose hill_workspace_bytes() exceeds it is
 * rejected with HILL_ERR_WORKSPACE before anything is enqueued (a 32K-token
 * GQA 32/8 step of batch 1 needs about 6 MB).  Every call on one GPU shares
 * that GPU's buffer, whose contents the previous call left: calls ordered on
 * one stream are fine, but calls that overlap in time on one GPU (other
 * streams or threads) race and give undefined results.  Otherwise the same
 * arguments, validation and results as hill_step. */
#define HILL_NOALLOC_SCRATCH_BYTES (32u << 20)
HILL_API hill_status hill_step_noalloc(const hill_desc* d, const void* q, const void* k, const void* v,
                              float* s, int32_t k_sel, int32_t* idx_out, float* out, void* stream);

/* Asymmetric-precision scoring (Sec. 4.4: the evaluation runs on int8 or
 * int4 casts of the keys and an int8 cast of the query, attention on the
 * original 16-bit K and V).
 *
 * The sketch of a key row (sequence b, KV head g, token j) is 128 codes plus
 * one exponent e (int8): with qmax = 127 (bits 8) or 7 (bits 4), e is the
 * smallest integer with max|K[b,g,j,:]| * 2^-e <= qmax, clamped to
 * [-128, 127] (-128 for an all-zero row), and code i = K[b,g,j,i] * 2^-e
 * rounded to nearest, ties to even, clamped to [-qmax, qmax].
 * Layouts: codes [B, Hkv, cap, 128] int8 (bits 8) or [B, Hkv, cap, 64] bytes
 * (bits 4: each group of 8 codes c0..c7 is one 4-byte word whose byte i is
 * (c_i + 8) | (c_{i+4} + 8) << 4), contiguous, 16-byte aligned; k_exp
 * [B, Hkv, cap] int8 contiguous, 4-byte aligned; cap >= n_tokens, cap a
 * multiple of 4.  The query is cast to int8 the same way per head inside the
 * scan.  The score of token j for head h is (sum_i q8[h,i] * code[j,i]) *
 * 2^(e_q + e_k), exact up to one fp32 rounding; weights, S, selection and
 * attention are as in hill_score / hill_step. */

/* Writes the sketch (bits 8 or 4) of key rows [token_begin, token_end) of
 * every (b, g): run it over the whole cache once, then for each appended
 * token. */
HILL_API hill_status hill_sketch_keys(const hill_desc* d, const void* k, int8_t* k8, int8_t* k_exp, int64_t cap, int32_t bits,
                             int32_t token_begin, int32_t token_end, void* stream);

/* hill_score on the sketch (no 16-bit keys read). */
HILL_API hill_status hill_score_sketch(const hill_desc* d, const void* q, const int8_t* k8, const int8_t* k_exp,
                              int64_t cap, int32_t bits, float* s, void* ws, size_t ws_bytes, void* stream);

/* hill_step whose scoring reads the sketch; selection and attention as in
 * hill_step (attention reads the 16-bit K and V of the selected tokens).
 * state: NULL, or the streamed selection's state (see hill_step_streamed;
 * ATTN only), then the selection runs streamed; flags as there (0 when
 * state is NULL).  ev may be NULL (see hill_step_profiled). */
HILL_API hill_status hill_step_sketch(const hill_desc* d, const void* q, const void* k, const void* v,
                             const int8_t* k8, const int8_t* k_exp, int64_t cap, int32_t bits, float* s,
                             uint32_t* state, uint32_t flags, int32_t k_sel, int32_t* idx_out, float* out,
                             void* ws, size_t ws_bytes, void* stream, const hill_step_events* ev);

/* Bidirectional KV Cache Pools (Sec. 4.2, HKM / BKP): the per-token hit-rate
 * table and the hot/cold pool policy, run once after each decoding step (the
 * paper's background maintenance pass).  On one GPU both pools live in HBM;
 * the call returns which tokens move between them, for a caller that keeps
 * the cold pool in a slower tier.
 *
 * Per importance row (b, r) over its first N = n_tokens tokens:
 *  1. hits[j] += 1 (saturating at 65535) for every j of this step's
 *     selected set idx[b, r, 0..k_sel);
 *  2. the most recent min(n_recent, N) tokens are hot (temporal pinning);
 *  3. the other min(capacity, N) - min(n_recent, N) hot slots go to the
 *     remaining tokens with the most hits; a token hot before the call wins a
 *     tie in hits, then the lower index wins (frequency tracking: a cold
 *     token is promoted only when it strictly exceeds the lowest-ranked hot
 *     token, which is then demoted);
 *  4. promote[b, r, :] lists the tokens that became hot and demote[b, r, :]
 *     those that became cold, each ascending; counts[b, r, 0..1] are their
 *     numbers (which may exceed list_cap: only the first list_cap entries of
 *     each list are written).
 * Positions at and beyond N are neither read nor written. */
typedef struct hill_bkp_desc {
    uint32_t struct_size;    /* sizeof(hill_bkp_desc) */
    int32_t batch;           /* B >= 1 */
    int32_t rows;            /* R >= 1 importance rows per sequence (1 in token mode, n_kv_heads in KV-head mode);
                                B * R <= 65535 */
    int32_t n_tokens;        /* N, 1 <= N <= 2097152 */
    int32_t n_recent;        /* >= 0: recent tokens pinned hot */
    int32_t capacity;        /* >= n_recent: hot pool size in tokens */
    int64_t stride_b;        /* elements between sequences of hits and hot (>= R * stride_r when B > 1) */
    int64_t stride_r;        /* elements between rows of hits and hot (>= N) */
} hill_bkp_desc;

/* Workspace bytes for hill_bkp_update (a pure function of the descriptor). */
HILL_API hill_status hill_bkp_workspace_bytes(const hill_bkp_desc* d, size_t* bytes);

/* One BKP pass.  idx: int32 [B, R, k_sel] (the layout of hill_step's
 * idx_out), indices unique within a row; entries outside [0, N) are skipped;
 * k_sel in [0, N] (idx may be NULL when 0).  hits: uint16 [B, R, >= N] and
 * hot: uint8 [B, R, >= N] (1 = hot, 0 = cold; bit 0 is read, 0 or 1 is
 * written), both with the descriptor's strides, caller-owned, zero at the
 * start of a sequence.  promote, demote: int32 [B, R, list_cap]; counts:
 * int32 [B, R, 2].  All device pointers, asynchronous on `stream`. */
HILL_API hill_status hill_bkp_update(const hill_bkp_desc* d, const int32_t* idx, int32_t k_sel, uint16_t* hits,
                            uint8_t* hot, int32_t* promote, int32_t* demote, int32_t list_cap, int32_t* counts,
                            void* ws, size_t ws_bytes, void* stream);

/* Tiered KV cache: the hot and cold pools of Sec. 4.2 (BKP) as two memory
 * tiers of one node -- the hot pool's K/V rows in HBM, the cold pool's in
 * host memory that the GPU reads and writes in place (pinned, allocated with
 * hipHostMalloc) -- with each token's row in exactly one of them.  Scoring
 * reads a key sketch of every token kept in HBM (the low-precision
 * evaluation the paper runs beside its cold pool, Sec. 4.4); the attention
 * gathers the selected tokens' rows from whichever pool holds them; after a
 * step, hill_bkp_update decides the pools and hill_tier_apply moves the rows.
 *
 * Layouts.  Hot pool: K_hot, V_hot [B, Hkv, capacity, D] 16-bit rows by slot,
 * both with the strides below (D contiguous).  Cold pool: K_cold, V_cold
 * [B, Hkv, >= n_cap, D] rows by token position, with the hill_desc's k / v
 * strides.  loc: int32 [B, R, n_cap] contiguous, 16-byte aligned: the slot
 * that holds the token's row in the hot pool, or -1 (cold pool).  R = 1 in
 * token mode (all KV heads of a token share its slot and move together) or
 * n_kv_heads in KV-head mode (one slot table per KV head).  A pool that
 * starts empty has loc = -1 everywhere and every row in the cold pool. */
typedef struct hill_tier_desc {
    uint32_t struct_size;   /* sizeof(hill_tier_desc) */
    int32_t capacity;       /* hot-pool slots per row (b, r), >= 1 */
    int32_t n_cap;          /* tokens per row of loc: >= n_tokens, a multiple of 4 */
    int32_t reserved;       /* 0 */
    int64_t hot_stride_b, hot_stride_h, hot_stride_n;   /* K_hot and V_hot strides in elements */
} hill_tier_desc;

/* One row migration after a BKP pass (Sec. 4.2 BKP (3)): promote / demote /
 * counts are hill_bkp_update's lists for this context (d->n_tokens tokens,
 * rows = R, capacity = the pool's), list_cap the lists' row length, at least
 * min(capacity, n_tokens) so that no list is cut.  The i-th demoted token's
 * row moves from its slot to the cold pool and the i-th promoted token's row
 * from the cold pool into that slot; promoted tokens beyond the demoted ones
 * take the slots never used before, from min(capacity, n_prev) on, where
 * n_prev is the context of the previous pass over this pool (0 for an empty
 * pool): the pool then holds min(capacity, n_tokens) rows in slots 0 .. that
 * number - 1.  loc is updated.  A row whose lists do not fit that (cut lists,
 * a pass over another context, a token out of place) is left as it was and
 * sets bit 0 or 1 of *status (device int32, caller-cleared; nothing else
 * writes it).  k_hot, v_hot, k_cold, v_cold: 16-byte aligned; the cold pool
 * may be host memory.  Asynchronous on stream. */
HILL_API hill_status hill_tier_apply(const hill_desc* d, const hill_tier_desc* t, void* k_hot, void* v_hot,
                            void* k_cold, void* v_cold, int32_t* loc, const int32_t* promote,
                            const int32_t* demote, int32_t list_cap, const int32_t* counts, int32_t n_prev,
                            int32_t* status, void* stream);

/* hill_step_sketch over a tiered cache: S, the selection and the outputs are
 * those of hill_step_sketch on a cache holding every row (the same values,
 * read from whichever pool holds them); d's k / v strides describe the cold
 * pool.  state, flags and ev as for hill_step_sketch. */
HILL_API hill_status hill_step_tiered(const hill_desc* d, const hill_tier_desc* t, const void* q, const void* k_hot,
                             const void* v_hot, const void* k_cold, const void* v_cold, const int32_t* loc,
                             const int8_t* k8, const int8_t* k_exp, int64_t cap, int32_t bits, float* s,
                             uint32_t* state, uint32_t flags, int32_t k_sel, int32_t* idx_out, float* out,
                             void* ws, size_t ws_bytes, void* stream, const hill_step_events* ev);

/* Adaptive Prefetch-based Pipeline (Sec. 4.3, Eqs. 2-4): the split of the KV
 * bytes M scored per step between a hot pool (subscript c) and a cold pool
 * (subscript s) whose scorers run in parallel, so that both paths, scoring
 * plus moving the retained fraction, take the same time:
 *     T_c = M_c / f_c + alpha_c * M_c / b_c  =  M_s / f_s + alpha_s * M_s / b_s = T_s,
 * M_c + M_s = M, M_c <= m0.  With alpha_c = alpha_s = alpha this is Eq. 2 and
 * beta = M_c / M_s is Eq. 4; separate values are the skew correction the
 * paper applies to alpha (the hot pool holds more of the retained tokens).
 * Host-only; no GPU work.  All rates in bytes per second, sizes in bytes. */
typedef struct hill_app_params {
    double f_c, f_s;            /* scoring throughput of each pool's evaluator, > 0 */
    double b_c, b_s;            /* bandwidth moving each pool's retained KV to the attention device, > 0 */
    double alpha_c, alpha_s;    /* retained fraction of each pool, in [0, 1] */
    double m;                   /* M > 0: KV bytes scored per step */
    double m0;                  /* bound on M_c (> 0), or <= 0 for none */
} hill_app_params;

typedef struct hill_app_plan {
    double beta;                /* M_c / M_s (infinite when M_s == 0) */
    double m_c, m_s;            /* the split */
    double t_c, t_s;            /* the two path times of Eq. 2, seconds */
    int32_t capped;             /* 1 if M_c was limited to m0 */
} hill_app_plan;

/* Fills *plan; HILL_ERR_INVALID_ARG for non-finite or out-of-range inputs. */
HILL_API hill_status hill_app_balance(const hill_app_params* p, hill_app_plan* plan);

#ifdef __cplusplus
}
#endif

#endif /* HILL_H */
