// Internal interface between the C-ABI host layer (hill_api.cpp) and the
// kernel translation units.  Not installed; not part of the ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace hill {

constexpr int kHeadDim = 128;      // D supported by every kernel
constexpr int kScoreTile = 32;     // tokens per scoring wave-tile
constexpr int kUnitTiles = 8;      // wave-tiles per scoring workgroup unit (softmax partial granularity)
constexpr int kMaxGroup = 128;     // query heads per KV head supported
constexpr int kUpdThreads = 512;   // threads per importance-update workgroup (two waves per SIMD)
constexpr int kStatLoads = 8;      // softmax partials per thread when the update reduces them itself
constexpr int kHistBits = 12;      // first radix digit of the selection keys
constexpr int kHistBins = 1 << kHistBits;
constexpr int kCoarseBins = 64;    // each 12-bit digit histogram also counts its top 6 bits
constexpr int kHistRow = kHistBins + kCoarseBins;   // words per histogram row: fine, then coarse
constexpr int kUpdChunk = 128;     // tokens per importance-update workgroup (two per lane)
constexpr int kHistChunk = 2048;   // tokens per standalone histogram workgroup
constexpr int kSelChunk = 512;     // tokens per selection chunk (256 threads x 2)

enum ScoreOut : int {
    kOutLogits = 0,    // ATTN: logits [B,Hq,n] + per-tile softmax partials
    kOutRawS = 1,      // RAW, one row per KV head: add head-group sums into S
    kOutRawGroups = 2  // RAW, token rows with Hkv > 1: head-group sums [B,Hkv,n]
};

struct ScoreArgs {
    const uint16_t* q;
    const uint16_t* k;
    int64_t q_sb, q_sh;
    int64_t k_sb, k_sh, k_sn;
    int B, Hq, Hkv, G, n, ntiles;
    int npart;               // workgroup units per (b, g): ceil(ntiles / kUnitTiles) rounded up to even
    int64_t ld;              // row stride of the logits buffer (n rounded up to 4)
    float s2;                // sm_scale * log2(e): logits are kept in the exp2 domain
    float* logits;           // kOutLogits: [B,Hq,ld]; kOutRawGroups: [B,Hkv,ld]
    float2* part;            // kOutLogits: [B,Hq,npart] (max, sum exp2) per unit of kUnitTiles tiles
    float* s;                // kOutRawS: importance rows
    int64_t s_sb, s_sr;
    uint32_t* zero_ptr;      // nullable: words to clear for a later kernel
    int64_t zero_words;
    const int8_t* k8;        // nullable: key sketch scored instead of k: int8 codes [B,Hkv,cap,128]
                             //   (kbits 8) or packed int4 codes [B,Hkv,cap,64] bytes (kbits 4)
    const int8_t* k_exp;     //   its per-row exponents [B,Hkv,cap]
    int64_t cap;             //   tokens per (b, g) in the sketch, a multiple of 4
    int kbits;               //   8 or 4
    int nt_logits;           // logits written with non-temporal stores (short launches, see kNtLogitsMaxKeyBytes)
};

// A scan reading at most this many key bytes writes its logits with non-temporal stores: in such a short
// launch the end-of-kernel write-back of logits left dirty in L2 delays the next kernel by ~2 us (32K tokens,
// B = 1: -0.8 us per layer-step); longer launches evict and write them back while they run, and there the
// non-temporal stores cost more read bandwidth than they save (256 MiB - 4 GiB of keys: 1-3 % slower).
constexpr int64_t kNtLogitsMaxKeyBytes = 96ll << 20;

// int8 key sketch: codes and one power-of-two exponent per key row
struct SketchArgs {
    const uint16_t* k;
    int64_t k_sb, k_sh, k_sn;
    int B, Hkv, t0, t1;
    int64_t cap;
    int8_t* k8;              // int8 codes [.., 128] or packed int4 codes [.., 64] bytes
    int8_t* k_exp;
    int bits;                // 8 or 4
};

struct UpdateArgs {
    const float* logits;     // ATTN: [B,Hq,ld]; RAW: group sums [B,Hkv,ld]
    int64_t ld;
    const float2* stats;     // ATTN: [B,Hq] (max, 1/sum) in the exp2 domain, or null: then
    const float2* part;      //   the kernel reduces the [B,Hq,npart] unit partials itself
    int npart;
    int tph;                 // update_attn: threads per head in the reduction (kUpdThreads / heads per row)
    float inv_tph;           //   and 1 / tph
    float* s;
    int64_t s_sb, s_sr;
    int B, Hq, Hkv, G, R, n;
    float s2;
    uint32_t* hist;          // nullable: [B*R, kHistRow] first-digit counts (fine, coarse); with a
                             // streamed bound only keys in the bound's bin or above are counted
    int pin_lo, pin_hi;      // tokens outside [pin_lo, pin_hi) count with the largest key (lo == hi: all)
    // streamed selection (nullable prev): candidates above the previous step's threshold
    const uint4* prev;       // [B*R, 2] caller's state (see StreamState)
    uint2* spairs;           // [B*R, n] (key, token) of every token whose first digit >= the bound's:
                             //   update block u's at u * kUpdChunk
    uint32_t* scount;        // [B*R, nup, kSlotWords] per update block: pairs per class, then the bound
                             //   (nup = ceil(n / kUpdChunk); see kSlotWords)
    uint32_t* hist2;         // [kStreamBins, B*R, kHistRow] second-digit counts of the keys in first-digit
                             //   bin d0 + w (w = 0: the selection's usual second-digit histogram)
    int k;                   // this step's budget
};

// Per-row state of the streamed selection, caller-owned between steps, two
// uint4: (threshold key, keys whose first digit reached the threshold's, n,
// valid) and (sink tokens, recent tokens, 0, 0).  The threshold's first digit
// bounds the next step's from below while S only grows (ATTN weights), the
// next budget is at most that count, n does not shrink and the pins stay.
constexpr int kStreamStateWords = 8;
// First-digit bins above the bound (the bound's included) whose second digits
// the update counts: the threshold rarely moves further in one step.
constexpr int kStreamBins = 4;

struct AttnArgs {
    const uint16_t* q;
    const uint16_t* k;
    const uint16_t* v;
    int64_t q_sb, q_sh;
    int64_t k_sb, k_sh, k_sn;
    int64_t v_sb, v_sh, v_sn;
    const int32_t* idx;      // [B, R, ksel]
    int B, Hq, Hkv, G, R, n, ksel, nsplit, per_split;
    int kv_per_wg;           // fused select+attend, token rows: KV heads per workgroup (divides Hkv)
    float s2;
    const float* logits;     // fused select+attend: the scan's q.k logits [B,Hq,ld] of these keys, or NULL
    int64_t ld;
    float* part_o;           // [B,Hq,nsplit,D]
    float2* part_ml;         // [B,Hq,nsplit] (max, sum) in the exp2 domain
    float* out;              // [B,Hq,D]
    // tiered cache (nullable loc): k and v above are the cold pool (rows by token), these the hot pool
    // (rows by slot); loc [B, R, loc_sr] holds each token's slot or -1
    const int32_t* loc;
    int64_t loc_sr;
    const uint16_t* k_hot;
    const uint16_t* v_hot;
    int64_t hk_sb, hk_sh, hk_sn, hv_sb, hv_sh, hv_sn;
    int cap;                 // hot-pool slots per row
};

// Row migration of a BKP pass between the hot pool (HBM slots) and the cold
// pool (rows by token, host memory): see hill_tier_apply.
struct TierArgs {
    uint16_t* k_hot;
    uint16_t* v_hot;
    uint16_t* k_cold;
    uint16_t* v_cold;
    int64_t hk_sb, hk_sh, hk_sn, hv_sb, hv_sh, hv_sn;    // hot pool strides
    int64_t ck_sb, ck_sh, ck_sn, cv_sb, cv_sh, cv_sn;    // cold pool strides
    int32_t* loc;             // [B, R, loc_sr]
    int64_t loc_sr;
    const int32_t* promote;   // [B, R, list_cap]
    const int32_t* demote;
    const int32_t* counts;    // [B, R, 2] (promotions, demotions)
    int list_cap;
    int R, Hkv, n, cap;
    int used_prev, used_now;  // slots in use before and after the pass: min(cap, n_prev), min(cap, n)
    int32_t* status;          // set to 1 when a row's counts do not fit (that row is left as it was)
};


// Exact top-k over 512-token chunks of each importance row (rows = B*R).
// Counts and lists live in the workspace.
struct RefineArgs {
    const float* s;
    int64_t s_sb, s_sr;
    int R, n, k, nchunks;
    const uint32_t* hist1;   // [rows, kHistRow] first-digit counts (bits 31..20; coarse: bits 31..26)
    uint32_t* hist2;         // [rows, kHistRow] second-digit counts (bits 19..8; coarse: bits 19..14), zeroed before
    uint32_t* cand_key;      // [rows, n] keys inside the first-digit bin, chunk c at offset c*kSelChunk
    uint32_t* cand_n;        // [rows, nchunks]
    uint4* state;            // [rows] (first-digit bin, keys still needed from it, keys in it, 0)
    int32_t* sel_list;       // [rows, n] each chunk's selected tokens in order, chunk c at c*kSelChunk
    uint32_t* sel_n;         // [rows, nchunks]
    int pin_lo, pin_hi;      // tokens outside [pin_lo, pin_hi) are always selected (lo == hi: all)
    // streamed selection: the update's candidate pairs replace the refine pass
    const uint2* spairs;     // [rows, n] update block u's pairs at u * kUpdChunk
    const uint32_t* scount;  // [rows, nup, kSlotWords] per update block: pairs per class, then the bound
    // hist2 continues as [kStreamBins, rows, kHistRow]: second digits of first-digit bins d0 + w
    uint4* state_out;        // [rows, 2] this step's threshold bound, for the next step (streamed
                             // selection; a reset step writes it from the refine pass), or NULL
};

// Splits of the selected set per (sequence, KV head) for the attention pass.
// A pure function of the shape so that workspace sizing needs no device query.
inline int attn_splits(int64_t b_hkv, int ksel, int* per_split)
{
    const int64_t target_wgs = 512;   // about two workgroups per CU
    const int min_tokens = 64;
    int64_t s = (target_wgs + b_hkv - 1) / b_hkv;
    int64_t cap = (ksel + min_tokens - 1) / min_tokens;
    if (s > cap) s = cap;
    if (s < 1) s = 1;
    int p = (int)((ksel + s - 1) / s);
    *per_split = p;
    return (ksel + p - 1) / p;   // every split non-empty; at most target_wgs
}
constexpr int kMaxSplits = 512;

// KV heads per fused select+attend workgroup for token rows: the largest
// power of two dividing Hkv that still leaves about eight workgroups per CU,
// so that large batches stop repeating the chunk's selection per KV head.
inline int emit_kv_per_wg(int B, int Hkv, int nchunks, int R)
{
    if (R != 1) return 1;
    const int64_t target = 2048;
    int h = 1;
    while (h * 2 <= Hkv && Hkv % (h * 2) == 0 && (int64_t)B * nchunks * (Hkv / (h * 2)) >= target) h *= 2;
    return h;
}
// Streamed selection: the pairs of an update block are grouped in kPairClasses
// classes (the kStreamBins window bins, then every key above the window).  The
// block's slot of kSlotWords words holds the class counts (words 0-4) and the
// bound the update used (word 5: the previous threshold's first digit |
// 0x80000000 if the bound held, else 0; the same in every block of a row), so
// that the selection reads both with one pair of 16-byte loads.
constexpr int kPairClasses = kStreamBins + 1;
constexpr int kSlotWords = 8;
constexpr int kSlotBound = 5;
static_assert(kPairClasses == kSlotBound && kSlotBound < kSlotWords, "class counts, then the bound");
constexpr int kMaxSlots = 4096;   // partial slots merged per head (splits or chunks)

// Optional start/stop timestamps of one launch (hipExtLaunchKernel events).
struct Stamp {
    hipEvent_t start = nullptr;
    hipEvent_t stop = nullptr;
};

// Fixed device scratch of hill_step_noalloc (noalloc.hip): a file-scope device
// array of kStaticScratchBytes per GPU; *ptr receives the current device's copy
// (its address looked up once per device, then cached).
constexpr size_t kStaticScratchBytes = (size_t)32 << 20;
hipError_t static_scratch(void** ptr);

hipError_t launch_fill_zero(uint32_t* p, int64_t words, hipStream_t st);
hipError_t launch_tier_apply(const TierArgs& a, int rows, hipStream_t st, Stamp ts = {});
hipError_t launch_sketch_keys(const SketchArgs& a, int dtype, hipStream_t st);
// Bidirectional KV cache pools (bkp.hip).
struct BkpArgs {
    const int32_t* idx;       // [rows, k]
    int k;
    uint16_t* hits;           // [B, R, >= n] strided
    uint8_t* hot;             // same strides as hits
    int64_t sb, sr;
    int R, n, w, f;           // w = min(n_recent, n); f = frequency slots
    int pos_shift;            // (n - 1) >> pos_shift < 128: the rank value's position bins
    float* v;                 // [rows, ld] rank values for the selection
    int64_t ld;
    uint32_t* zero;           // histogram region cleared by bkp_hits
    int64_t zero_words;
    uint32_t* hist1;          // [rows, kHistRow] first-digit counts of v
    const int32_t* sel_list;  // [rows, n] chosen tokens per 512-token chunk (topk emit)
    const uint32_t* sel_n;    // [rows, nchunks]
    int nchunks;
    uint2* chunk_moves;       // [rows, nchunks] (promotions, demotions) per chunk
    int32_t* promote;         // [rows, list_cap]
    int32_t* demote;
    int list_cap;
    int32_t* counts;          // [rows, 2]
    __host__ __device__ int64_t off(int row) const { return (int64_t)(row / R) * sb + (int64_t)(row % R) * sr; }
};
hipError_t launch_bkp_hits(const BkpArgs& a, int rows, hipStream_t st);
hipError_t launch_bkp_rank(const BkpArgs& a, int rows, hipStream_t st);
hipError_t launch_bkp_lists(const BkpArgs& a, int rows, hipStream_t st);
hipError_t launch_score_tiles(const ScoreArgs& a, int dtype, ScoreOut out, int ncu, hipStream_t st, Stamp ts = {});
hipError_t launch_softmax_stats(const float2* part, float2* stats, int bh, int npart, hipStream_t st,
                                Stamp ts = {});
// Whether update_attn reduces the softmax partials itself (no separate
// softmax_stats launch): every thread then loads at most kStatLoads of them,
// and every update workgroup re-reads its row's partials. The extra launch
// costs about 4 us; the re-reads it saves cost about 0.05 us per MiB (8 x 32K
// tokens, 64 MiB: about 3 us; 32 x 32K, 256 MiB: about 12.5 us), so calls
// re-reading more than kStatRereadMax bytes take the separate launch.
constexpr int64_t kStatRereadMax = 128ll << 20;
inline bool update_reduces_stats(int nheads_per_row, int npart, int64_t update_blocks)
{
    if (nheads_per_row < 1 || nheads_per_row > 256) return false;
    const int tph = kUpdThreads / nheads_per_row;
    return (int64_t)npart <= (int64_t)kStatLoads * tph &&
           update_blocks * npart * nheads_per_row * (int64_t)sizeof(float2) <= kStatRereadMax;
}
hipError_t launch_update_attn(const UpdateArgs& a, hipStream_t st, Stamp ts = {});
hipError_t launch_update_raw_groups(const UpdateArgs& a, hipStream_t st, Stamp ts = {});
hipError_t launch_topk_hist(const float* s, int64_t s_sb, int64_t s_sr, int B, int R, int n, int pin_lo,
                            int pin_hi, uint32_t* hist, hipStream_t st, Stamp ts = {});
hipError_t launch_topk_refine(const RefineArgs& a, int rows, hipStream_t st, Stamp ts = {});
// Selects per chunk and writes the ordered indices (and values, if val).
hipError_t launch_topk_emit_indices(const RefineArgs& r, int rows, int32_t* idx, float* val, hipStream_t st,
                                    Stamp ts = {});
// Streamed selection + attention: the exact threshold from the first-digit
// histogram and the update's candidate pairs (no refine pass), then as
// launch_topk_emit_attn; writes the next step's bound to r.state_out.
hipError_t launch_topk_emit_attn_stream(const RefineArgs& r, const AttnArgs& at, int dtype, hipStream_t st,
                                        Stamp ts = {});
// Selects per chunk only: chunk c's tokens in order in r.sel_list, their count in r.sel_n.
hipError_t launch_topk_emit_lists(const RefineArgs& r, int rows, hipStream_t st);
// Selects per chunk and attends over each chunk's selected tokens: one
// partial per (query head, chunk) in at.part_o / at.part_ml ([B*Hq, nchunks]
// slots).  launch_merge_write then merges the partials into at.out and
// writes the ordered indices.
hipError_t launch_topk_emit_attn(const RefineArgs& r, const AttnArgs& at, int dtype, hipStream_t st, Stamp ts = {});
hipError_t launch_merge_write(const RefineArgs& r, const AttnArgs& at, int32_t* idx, int rows, hipStream_t st,
                              Stamp ts = {});
hipError_t launch_attn_split(const AttnArgs& a, int dtype, hipStream_t st);
hipError_t launch_attn_combine(const AttnArgs& a, hipStream_t st, Stamp ts = {});

}  // namespace hill
