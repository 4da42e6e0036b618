// C-ABI host layer of libhill: argument validation, workspace layout and
// kernel orchestration.  Every check runs before the first HIP call, so an
// invalid call enqueues nothing and touches no output.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <string>

#include "hill.h"
#include "hill_internal.h"

using namespace hill;

namespace {

thread_local std::string g_last_error;

hill_status fail(hill_status st, const char* fmt, ...)
{
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof(buf), fmt, ap);
    va_end(ap);
    g_last_error = buf;
    return st;
}

// Shape facts derived from a validated descriptor.
struct Shape {
    int B, Hq, Hkv, G, D, n, R, ntiles, npart;
    int64_t ld;
    int dtype, mode, gran;
    float scale;
    int pin_lo, pin_hi;   // tokens outside [pin_lo, pin_hi) are always selected (lo == hi: all of them)
    int pinned;           // how many tokens that is
};

// Workspace regions, in this order, each 256-byte aligned:
//   logits   ATTN [B,Hq,ld] fp32 | RAW token rows with Hkv > 1: [B,Hkv,ld] fp32 (ld = n rounded up to 4)
//   part     ATTN [B,Hq,npart] float2 (per 256-token unit);  stats ATTN [B,Hq] float2
//   zeroed   hist1 [rows,4096+64] | hist2 [rows,4096+64] (u32 fine + coarse bins) | hist2x [3,rows,4096+64] (the
//            streamed selection's further second-digit windows, hist2 continued) -- cleared by the first kernel of
//            every call that accumulates into them
//   scount [rows,ceil(n/kUpdChunk),8] u32 | spairs [rows,n] uint2 (key, token) (streamed selection only)
//   cand_key [rows,n] u32 | cand_n [rows,nchunks] u32 | state [rows] uint4
//   sel_list [rows,n] i32 | sel_n [rows,nchunks] u32
//   slots: attention partials [B,Hq,nslots,D] fp32 and [B,Hq,nslots] float2, nslots =
//          max(nchunks, splits of the standalone attention)
// Only the last region depends on k_sel.
struct Layout {
    size_t logits, part, stats;
    size_t zero, hist1, hist2, hist2x;
    int64_t zero_words, zero_words_stream;   // the streamed selection also clears hist2x
    size_t cand_key, cand_n, state, sel_list, sel_n;
    size_t scount, spairs;   // streamed selection: pair counts and bound per update block, pairs
    size_t slot_o, slot_ml;
    size_t end_score, end_topk, end_all;
    int nchunks, nsplit, per_split, nslots;
};

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

Layout layout_for(const Shape& s, int ksel)
{
    Layout L{};
    size_t off = 0;
    const bool attn = s.mode == HILL_SCORE_ATTN;
    const bool raw_groups = !attn && s.gran == HILL_SEL_TOKEN && s.Hkv > 1;
    const size_t rows = (size_t)s.B * s.R;
    L.logits = off;
    if (attn) off += align256((size_t)s.B * s.Hq * s.ld * sizeof(float));
    else if (raw_groups) off += align256((size_t)s.B * s.Hkv * s.ld * sizeof(float));
    L.part = off;
    if (attn) off += align256((size_t)s.B * s.Hq * s.npart * sizeof(float2));
    L.stats = off;
    if (attn) off += align256((size_t)s.B * s.Hq * sizeof(float2));
    L.end_score = off;
    L.zero = off;
    L.hist1 = off;
    L.hist2 = L.hist1 + rows * kHistRow * sizeof(uint32_t);
    L.hist2x = L.hist2 + rows * kHistRow * sizeof(uint32_t);
    L.zero_words = (int64_t)((L.hist2x - L.zero) / sizeof(uint32_t));
    // the streamed selection's regions exist for ATTN scores only (the only mode it runs in)
    const size_t zero_end = L.hist2x + (attn ? rows * (kStreamBins - 1) * kHistRow * sizeof(uint32_t) : 0);
    L.zero_words_stream = (int64_t)((zero_end - L.zero) / sizeof(uint32_t));
    off = align256(zero_end);
    L.scount = off;
    if (attn) off += align256(rows * (size_t)((s.n + kUpdChunk - 1) / kUpdChunk) * kSlotWords * sizeof(uint32_t));
    L.spairs = off;
    if (attn) off += align256(rows * (size_t)s.n * sizeof(uint2));
    L.nchunks = (s.n + kSelChunk - 1) / kSelChunk;
    L.cand_key = off;
    off += align256(rows * (size_t)s.n * sizeof(uint32_t));
    L.cand_n = off;
    off += align256(rows * L.nchunks * sizeof(uint32_t));
    L.state = off;
    off += align256(rows * sizeof(uint4));
    L.sel_list = off;
    off += align256(rows * (size_t)s.n * sizeof(int32_t));
    L.sel_n = off;
    off += align256(rows * L.nchunks * sizeof(uint32_t));
    L.end_topk = off;
    L.nsplit = attn_splits((int64_t)s.B * s.Hkv, ksel, &L.per_split);
    L.nslots = L.nsplit > L.nchunks ? L.nsplit : L.nchunks;
    L.slot_o = off;
    off += align256((size_t)s.B * s.Hq * L.nslots * kHeadDim * sizeof(float));
    L.slot_ml = off;
    off += align256((size_t)s.B * s.Hq * L.nslots * sizeof(float2));
    L.end_all = off;
    return L;
}

bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

hill_status check_desc(const hill_desc* d, Shape* s, bool uses_s = true)
{
    if (!d) return fail(HILL_ERR_INVALID_ARG, "descriptor is NULL");
    if (d->struct_size != sizeof(hill_desc))
        return fail(HILL_ERR_INVALID_ARG, "struct_size %u != sizeof(hill_desc) %zu", d->struct_size,
                    sizeof(hill_desc));
    if (d->batch < 1 || d->n_q_heads < 1 || d->n_kv_heads < 1 || d->n_tokens < 1 || d->head_dim < 1)
        return fail(HILL_ERR_INVALID_ARG, "batch, heads, head_dim and n_tokens must be >= 1");
    if (d->n_q_heads % d->n_kv_heads)
        return fail(HILL_ERR_INVALID_ARG, "n_q_heads %d is not a multiple of n_kv_heads %d", d->n_q_heads,
                    d->n_kv_heads);
    if (d->n_q_heads > 256 || d->n_q_heads / d->n_kv_heads > kMaxGroup)
        return fail(HILL_ERR_UNSUPPORTED, "more than 256 query heads or %d query heads per KV head", kMaxGroup);
    if (d->dtype != HILL_F16 && d->dtype != HILL_BF16)
        return fail(HILL_ERR_UNSUPPORTED, "dtype %d is not fp16 (0) or bf16 (1)", d->dtype);
    if (d->score_mode != HILL_SCORE_ATTN && d->score_mode != HILL_SCORE_RAW)
        return fail(HILL_ERR_INVALID_ARG, "score_mode %d is not ATTN (0) or RAW (1)", d->score_mode);
    if (d->granularity != HILL_SEL_TOKEN && d->granularity != HILL_SEL_KVHEAD)
        return fail(HILL_ERR_INVALID_ARG, "granularity %d is not TOKEN (0) or KVHEAD (1)", d->granularity);
    if (d->head_dim != kHeadDim)
        return fail(HILL_ERR_UNSUPPORTED, "head_dim %d is not supported (only 128)", d->head_dim);
    if ((int64_t)d->n_tokens > (int64_t)kMaxSlots * kSelChunk)
        return fail(HILL_ERR_UNSUPPORTED, "n_tokens %d exceeds the supported %d", d->n_tokens, kMaxSlots * kSelChunk);
    if (!std::isfinite(d->sm_scale)) return fail(HILL_ERR_INVALID_ARG, "sm_scale is not finite");
    if (d->n_sink < 0 || d->n_recent < 0)
        return fail(HILL_ERR_INVALID_ARG, "n_sink (%d) and n_recent (%d) must be >= 0", d->n_sink, d->n_recent);
    const int64_t D = d->head_dim;
    const int64_t strides16[] = {d->q_stride_b, d->q_stride_h, d->k_stride_b, d->k_stride_h,
                                 d->k_stride_n, d->v_stride_b, d->v_stride_h, d->v_stride_n};
    for (int64_t st : strides16)
        if (st < 0 || st % 8)
            return fail(HILL_ERR_INVALID_ARG, "q/K/V strides must be non-negative multiples of 8 elements");
    if (d->q_stride_h < D && d->n_q_heads > 1) return fail(HILL_ERR_INVALID_ARG, "q_stride_h < head_dim");
    if (d->k_stride_n < D || d->v_stride_n < D)
        return fail(HILL_ERR_INVALID_ARG, "k_stride_n / v_stride_n < head_dim");
    if (d->k_stride_n > INT32_MAX || d->v_stride_n > INT32_MAX)
        return fail(HILL_ERR_UNSUPPORTED, "k_stride_n / v_stride_n above 2^31 - 1 elements");
    const int R = d->granularity == HILL_SEL_TOKEN ? 1 : d->n_kv_heads;
    if (uses_s) {
        if (d->s_stride_r < d->n_tokens || d->s_stride_r % 4)
            return fail(HILL_ERR_INVALID_ARG, "s_stride_r must be >= n_tokens and a multiple of 4");
        if (d->s_stride_b % 4 || (d->batch > 1 && d->s_stride_b < (int64_t)R * d->s_stride_r))
            return fail(HILL_ERR_INVALID_ARG, "s_stride_b must be a multiple of 4 and >= R * s_stride_r");
    }
    s->B = d->batch;
    s->Hq = d->n_q_heads;
    s->Hkv = d->n_kv_heads;
    s->G = d->n_q_heads / d->n_kv_heads;
    s->D = d->head_dim;
    s->n = d->n_tokens;
    s->R = R;
    s->ntiles = (d->n_tokens + kScoreTile - 1) / kScoreTile;
    s->npart = ((s->ntiles + kUnitTiles - 1) / kUnitTiles + 1) / 2 * 2;   // even: the update reads pairs
    s->ld = ((int64_t)d->n_tokens + 3) / 4 * 4;
    s->dtype = d->dtype;
    s->mode = d->score_mode;
    s->gran = d->granularity;
    s->scale = d->sm_scale != 0.0f ? d->sm_scale : 1.0f / std::sqrt((float)d->head_dim);
    s->pin_lo = d->n_sink < d->n_tokens ? d->n_sink : d->n_tokens;
    s->pin_hi = d->n_tokens - (d->n_recent < d->n_tokens ? d->n_recent : d->n_tokens);
    if (s->pin_hi <= s->pin_lo) s->pin_lo = s->pin_hi = 0;   // the windows cover the row: all pinned
    s->pinned = s->pin_lo + (d->n_tokens - s->pin_hi);
    if (s->pin_lo == s->pin_hi) s->pinned = d->n_tokens;
    return HILL_OK;
}

hill_status check_ptr(const void* p, const char* name)
{
    if (!p) return fail(HILL_ERR_INVALID_ARG, "%s is NULL", name);
    if (!aligned16(p)) return fail(HILL_ERR_INVALID_ARG, "%s is not 16-byte aligned", name);
    return HILL_OK;
}

hill_status check_ksel(const Shape& s, int32_t ksel)
{
    if (ksel < 1 || ksel > s.n) return fail(HILL_ERR_INVALID_ARG, "k_sel %d not in [1, n_tokens=%d]", ksel, s.n);
    return HILL_OK;
}

// Selections must have room for every pinned token.
hill_status check_pins(const Shape& s, int32_t ksel)
{
    if (ksel < s.pinned)
        return fail(HILL_ERR_INVALID_ARG, "k_sel %d is smaller than the %d pinned tokens (n_sink, n_recent)", ksel,
                    s.pinned);
    return HILL_OK;
}

hill_status check_ws(const void* ws, size_t ws_bytes, size_t need)
{
    if (ws_bytes < need)
        return fail(HILL_ERR_WORKSPACE, "workspace of %zu bytes is smaller than the %zu needed", ws_bytes, need);
    if (need && !ws) return fail(HILL_ERR_INVALID_ARG, "workspace is NULL");
    if (need && !aligned16(ws)) return fail(HILL_ERR_INVALID_ARG, "workspace is not 16-byte aligned");
    return HILL_OK;
}

#define HILL_TRY(expr)                            \
    do {                                          \
        hill_status st_ = (expr);                 \
        if (st_ != HILL_OK) return st_;           \
    } while (0)

#define HIP_TRY(expr)                                                                              \
    do {                                                                                           \
        hipError_t e_ = (expr);                                                                    \
        if (e_ != hipSuccess) return fail(HILL_ERR_HIP, "%s: %s", #expr, hipGetErrorString(e_)); \
    } while (0)

// Compute units of the current device, cached per device.
int device_cus()
{
    static int cache[64] = {0};
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
    int v = __atomic_load_n(&cache[dev], __ATOMIC_RELAXED);
    if (v > 0) return v;
    if (hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || v <= 0) v = 256;
    __atomic_store_n(&cache[dev], v, __ATOMIC_RELAXED);
    return v;
}

// The start / stop events of one stage of a step (include/hill.h).
Stamp stage(const hill_step_events& ev, int i)
{
    return Stamp{static_cast<hipEvent_t>(ev.start[i]), static_cast<hipEvent_t>(ev.stop[i])};
}

template <typename T>
T* at(void* ws, size_t off)
{
    return reinterpret_cast<T*>(static_cast<char*>(ws) + off);
}

// Optional int8 / int4 key sketch scored in place of the 16-bit keys.
struct Sketch {
    const int8_t* k8 = nullptr;
    const int8_t* k_exp = nullptr;
    int64_t cap = 0;
    int bits = 8;
};

hill_status check_sketch(const Shape& s, const int8_t* k8, const int8_t* k_exp, int64_t cap, int bits)
{
    if (!k8 || !k_exp) return fail(HILL_ERR_INVALID_ARG, "sketch codes or exponents are NULL");
    if (bits != 8 && bits != 4) return fail(HILL_ERR_INVALID_ARG, "sketch bits %d is not 8 or 4", bits);
    if ((uintptr_t)k8 & 15u) return fail(HILL_ERR_INVALID_ARG, "sketch codes are not 16-byte aligned");
    if ((uintptr_t)k_exp & 3u) return fail(HILL_ERR_INVALID_ARG, "sketch exponents are not 4-byte aligned");
    if (cap < s.n || cap % 4) return fail(HILL_ERR_INVALID_ARG, "sketch capacity %lld must be >= n_tokens and a multiple of 4",
                                          (long long)cap);
    return HILL_OK;
}

// Scoring; if `hist` is given the first selection digit is counted as a side
// effect (hill_step) and the counts are cleared by the first kernel.
hill_status run_score(const hill_desc* d, const Shape& s, const Layout& L, const void* q, const void* k,
                      const Sketch& sk, float* sacc, void* ws, bool with_hist, hipStream_t st,
                      const hill_step_events& ev, const uint4* stream_prev = nullptr, int ksel = 0)
{
    const Stamp scan = stage(ev, HILL_STAGE_SCAN);
    const Stamp upd = stage(ev, HILL_STAGE_UPDATE);
    uint32_t* hist = with_hist ? at<uint32_t>(ws, L.hist1) : nullptr;
    ScoreArgs a{};
    a.q = static_cast<const uint16_t*>(q);
    a.k = static_cast<const uint16_t*>(k);
    a.q_sb = d->q_stride_b;
    a.q_sh = d->q_stride_h;
    a.k_sb = d->k_stride_b;
    a.k_sh = d->k_stride_h;
    a.k_sn = d->k_stride_n;
    a.B = s.B;
    a.Hq = s.Hq;
    a.Hkv = s.Hkv;
    a.G = s.G;
    a.n = s.n;
    a.ntiles = s.ntiles;
    a.npart = s.npart;
    a.ld = s.ld;
    a.s2 = s.scale * 1.4426950408889634f;
    a.s = sacc;
    a.s_sb = d->s_stride_b;
    a.s_sr = d->s_stride_r;
    a.zero_ptr = with_hist ? at<uint32_t>(ws, L.zero) : nullptr;
    a.zero_words = with_hist ? (stream_prev ? L.zero_words_stream : L.zero_words) : 0;
    a.k8 = sk.k8;
    a.k_exp = sk.k_exp;
    a.cap = sk.cap;
    a.kbits = sk.bits;
    {   // bytes of keys (or sketch codes) this scan reads
        const int64_t row_bytes = sk.k8 ? (sk.bits == 4 ? 64 : 128) : (int64_t)kHeadDim * 2;
        a.nt_logits = (int64_t)s.B * s.Hkv * s.n * row_bytes <= kNtLogitsMaxKeyBytes;
    }
    const int ncu = device_cus();

    UpdateArgs u{};
    u.s = sacc;
    u.s_sb = d->s_stride_b;
    u.s_sr = d->s_stride_r;
    u.B = s.B;
    u.Hq = s.Hq;
    u.Hkv = s.Hkv;
    u.G = s.G;
    u.R = s.R;
    u.n = s.n;
    u.ld = s.ld;
    u.s2 = a.s2;
    u.hist = hist;
    u.pin_lo = s.pin_lo;
    u.pin_hi = s.pin_hi;
    if (stream_prev) {   // streamed selection (ATTN only): candidate pairs above the previous threshold
        u.prev = stream_prev;
        u.spairs = at<uint2>(ws, L.spairs);
        u.scount = at<uint32_t>(ws, L.scount);
        u.hist2 = at<uint32_t>(ws, L.hist2);
        u.k = ksel;
    }

    if (s.mode == HILL_SCORE_ATTN) {
        a.logits = at<float>(ws, L.logits);
        a.part = at<float2>(ws, L.part);
        HIP_TRY(launch_score_tiles(a, s.dtype, kOutLogits, ncu, st, scan));
        u.logits = a.logits;
        u.part = a.part;
        u.npart = s.npart;
        u.tph = kUpdThreads / (s.R == 1 ? s.Hq : s.G);   // heads per row <= 256 (validated)
        u.inv_tph = 1.0f / (float)u.tph;
        u.stats = nullptr;
        const int64_t update_blocks = (int64_t)s.B * s.R * ((s.n + kUpdChunk - 1) / kUpdChunk);
        if (!update_reduces_stats(s.R == 1 ? s.Hq : s.G, s.npart, update_blocks)) {
            float2* stats = at<float2>(ws, L.stats);
            HIP_TRY(launch_softmax_stats(a.part, stats, s.B * s.Hq, s.npart, st, stage(ev, HILL_STAGE_STATS)));
            u.stats = stats;
        }
        HIP_TRY(launch_update_attn(u, st, upd));
    } else if (s.R == s.Hkv) {
        // one row per KV head (or a single KV head): the scan adds straight into S
        HIP_TRY(launch_score_tiles(a, s.dtype, kOutRawS, ncu, st, scan));
        if (with_hist)
            HIP_TRY(launch_topk_hist(sacc, d->s_stride_b, d->s_stride_r, s.B, s.R, s.n, s.pin_lo, s.pin_hi, hist, st,
                                     upd));
    } else {
        a.logits = at<float>(ws, L.logits);
        HIP_TRY(launch_score_tiles(a, s.dtype, kOutRawGroups, ncu, st, scan));
        u.logits = a.logits;
        HIP_TRY(launch_update_raw_groups(u, st, upd));
    }
    return HILL_OK;
}

RefineArgs refine_args(const hill_desc* d, const Shape& s, const Layout& L, const float* sacc, int32_t ksel, void* ws)
{
    RefineArgs r{};
    r.s = sacc;
    r.s_sb = d->s_stride_b;
    r.s_sr = d->s_stride_r;
    r.R = s.R;
    r.n = s.n;
    r.k = ksel;
    r.nchunks = L.nchunks;
    r.hist1 = at<uint32_t>(ws, L.hist1);
    r.hist2 = at<uint32_t>(ws, L.hist2);
    r.cand_key = at<uint32_t>(ws, L.cand_key);
    r.cand_n = at<uint32_t>(ws, L.cand_n);
    r.state = at<uint4>(ws, L.state);
    r.sel_list = at<int32_t>(ws, L.sel_list);
    r.sel_n = at<uint32_t>(ws, L.sel_n);
    r.pin_lo = s.pin_lo;
    r.pin_hi = s.pin_hi;
    r.spairs = at<uint2>(ws, L.spairs);
    r.scount = at<uint32_t>(ws, L.scount);
    return r;
}

// Standalone selection: clear the counters, count the first digit, refine, emit.
hill_status run_select(const hill_desc* d, const Shape& s, const Layout& L, const float* sacc, int32_t ksel,
                       int32_t* idx, float* val, void* ws, hipStream_t st)
{
    const RefineArgs r = refine_args(d, s, L, sacc, ksel, ws);
    HIP_TRY(launch_fill_zero(at<uint32_t>(ws, L.zero), L.zero_words, st));
    HIP_TRY(launch_topk_hist(sacc, d->s_stride_b, d->s_stride_r, s.B, s.R, s.n, s.pin_lo, s.pin_hi,
                             at<uint32_t>(ws, L.hist1), st));
    HIP_TRY(launch_topk_refine(r, s.B * s.R, st));
    HIP_TRY(launch_topk_emit_indices(r, s.B * s.R, idx, val, st));
    return HILL_OK;
}

AttnArgs attn_args(const hill_desc* d, const Shape& s, const Layout& L, const void* q, const void* k, const void* v,
                   const int32_t* idx, int32_t ksel, float* out, void* ws)
{
    AttnArgs a{};
    a.q = static_cast<const uint16_t*>(q);
    a.k = static_cast<const uint16_t*>(k);
    a.v = static_cast<const uint16_t*>(v);
    a.q_sb = d->q_stride_b;
    a.q_sh = d->q_stride_h;
    a.k_sb = d->k_stride_b;
    a.k_sh = d->k_stride_h;
    a.k_sn = d->k_stride_n;
    a.v_sb = d->v_stride_b;
    a.v_sh = d->v_stride_h;
    a.v_sn = d->v_stride_n;
    a.idx = idx;
    a.B = s.B;
    a.Hq = s.Hq;
    a.Hkv = s.Hkv;
    a.G = s.G;
    a.R = s.R;
    a.n = s.n;
    a.ksel = ksel;
    a.nsplit = L.nsplit;
    a.per_split = L.per_split;
    a.kv_per_wg = emit_kv_per_wg(s.B, s.Hkv, L.nchunks, s.R);
    a.s2 = s.scale * 1.4426950408889634f;
    a.part_o = at<float>(ws, L.slot_o);
    a.part_ml = at<float2>(ws, L.slot_ml);
    a.out = out;
    return a;
}

hill_status run_attn(const hill_desc* d, const Shape& s, const Layout& L, const void* q, const void* k, const void* v,
                     const int32_t* idx, int32_t ksel, float* out, void* ws, hipStream_t st)
{
    const AttnArgs a = attn_args(d, s, L, q, k, v, idx, ksel, out, ws);
    HIP_TRY(launch_attn_split(a, s.dtype, st));
    HIP_TRY(launch_attn_combine(a, st));
    return HILL_OK;
}

// One decode step: score (16-bit keys or the sketch), refine the threshold,
// then emit the indices and attend over each chunk's picks in the same kernel.
// Optional tiered cache of a decode step: the hot pool and the slot table
// (the step's k and v are then the cold pool).
struct Tier {
    const hill_tier_desc* t = nullptr;
    const void* k_hot = nullptr;
    const void* v_hot = nullptr;
    const int32_t* loc = nullptr;
};

// The cold pool may be host memory: it must be memory the GPU can reach (pinned host memory from
// hipHostMalloc, or device memory); pageable host memory is refused here instead of faulting on the device.
hill_status check_reachable(const void* p, const char* name)
{
    hipPointerAttribute_t at{};
    if (hipPointerGetAttributes(&at, p) != hipSuccess) {
        (void)hipGetLastError();   // clear the query's error
        return fail(HILL_ERR_INVALID_ARG, "%s is not memory the GPU can reach (pinned host or device memory)", name);
    }
    if (at.type != hipMemoryTypeHost && at.type != hipMemoryTypeDevice && at.type != hipMemoryTypeManaged)
        return fail(HILL_ERR_INVALID_ARG, "%s is not memory the GPU can reach (pinned host or device memory)", name);
    if (at.type == hipMemoryTypeHost && at.devicePointer != p)
        return fail(HILL_ERR_UNSUPPORTED, "%s: pinned host memory whose device address differs from its host address", name);
    return HILL_OK;
}

hill_status check_tier(const Shape& s, const hill_tier_desc* t)
{
    if (!t) return fail(HILL_ERR_INVALID_ARG, "tier descriptor is NULL");
    if (t->struct_size != sizeof(hill_tier_desc))
        return fail(HILL_ERR_INVALID_ARG, "struct_size %u != sizeof(hill_tier_desc) %zu", t->struct_size,
                    sizeof(hill_tier_desc));
    if (t->capacity < 1) return fail(HILL_ERR_INVALID_ARG, "capacity %d < 1", t->capacity);
    if (t->n_cap < s.n || t->n_cap % 4)
        return fail(HILL_ERR_INVALID_ARG, "n_cap %d must be >= n_tokens (%d) and a multiple of 4", t->n_cap, s.n);
    if (t->reserved != 0) return fail(HILL_ERR_INVALID_ARG, "reserved must be 0");
    const int64_t st[] = {t->hot_stride_b, t->hot_stride_h, t->hot_stride_n};
    for (int64_t x : st)
        if (x < 0 || x % 8) return fail(HILL_ERR_INVALID_ARG, "hot-pool strides must be non-negative multiples of 8");
    if (t->hot_stride_n < s.D) return fail(HILL_ERR_INVALID_ARG, "hot_stride_n < head_dim");
    if (t->hot_stride_n > INT32_MAX) return fail(HILL_ERR_UNSUPPORTED, "hot_stride_n above 2^31 - 1 elements");
    return HILL_OK;
}

// Every argument of a decode step except the workspace.
hill_status check_step(const hill_desc* d, const void* q, const void* k, const void* v, const Sketch& sk,
                       const float* s_acc, int32_t k_sel, const int32_t* idx_out, const float* out, Shape* s)
{
    HILL_TRY(check_desc(d, s));
    HILL_TRY(check_ksel(*s, k_sel));
    HILL_TRY(check_pins(*s, k_sel));
    HILL_TRY(check_ptr(q, "q"));
    HILL_TRY(check_ptr(k, "k"));
    HILL_TRY(check_ptr(v, "v"));
    if (sk.k8) HILL_TRY(check_sketch(*s, sk.k8, sk.k_exp, sk.cap, sk.bits));
    HILL_TRY(check_ptr(s_acc, "s"));
    HILL_TRY(check_ptr(out, "out"));
    if (!idx_out) return fail(HILL_ERR_INVALID_ARG, "idx_out is NULL");
    if ((uintptr_t)idx_out & 3u) return fail(HILL_ERR_INVALID_ARG, "idx_out is not 4-byte aligned");
    return HILL_OK;
}

hill_status run_step(const hill_desc* d, const void* q, const void* k, const void* v, const Sketch& sk, float* s_acc,
                     int32_t k_sel, int32_t* idx_out, float* out, void* ws, size_t ws_bytes, void* stream,
                     const hill_step_events* ev, uint32_t* stream_state = nullptr, bool stream_reset = false,
                     const Tier& tier = Tier{})
{
    Shape s;
    HILL_TRY(check_step(d, q, k, v, sk, s_acc, k_sel, idx_out, out, &s));
    if (tier.t) {
        HILL_TRY(check_tier(s, tier.t));
        HILL_TRY(check_ptr(tier.k_hot, "k_hot"));
        HILL_TRY(check_ptr(tier.v_hot, "v_hot"));
        HILL_TRY(check_ptr(tier.loc, "loc"));
        if (!sk.k8) return fail(HILL_ERR_INVALID_ARG, "a tiered step scores on the key sketch");
        HILL_TRY(check_reachable(k, "k_cold"));
        HILL_TRY(check_reachable(v, "v_cold"));
    }
    const Layout L = layout_for(s, k_sel);
    HILL_TRY(check_ws(ws, ws_bytes, L.end_all));
    hipStream_t st = static_cast<hipStream_t>(stream);
    const hill_step_events none{};
    const hill_step_events& e = ev ? *ev : none;
    uint4* state4 = reinterpret_cast<uint4*>(stream_state);
    // a reset step selects through the refine pass and only writes the bound
    HILL_TRY(run_score(d, s, L, q, k, sk, s_acc, ws, true, st, e, stream_reset ? nullptr : state4, k_sel));
    RefineArgs r = refine_args(d, s, L, s_acc, k_sel, ws);
    AttnArgs a = attn_args(d, s, L, q, k, v, idx_out, k_sel, out, ws);
    if (s.mode == HILL_SCORE_ATTN && !sk.k8) {   // the scan's logits are those of the 16-bit keys: reused
        a.logits = at<float>(ws, L.logits);
        a.ld = s.ld;
    }
    if (tier.t) {   // K and V rows through the slot table: the hot pool, else the cold pool (k, v)
        a.loc = tier.loc;
        a.loc_sr = tier.t->n_cap;
        a.k_hot = static_cast<const uint16_t*>(tier.k_hot);
        a.v_hot = static_cast<const uint16_t*>(tier.v_hot);
        a.hk_sb = a.hv_sb = tier.t->hot_stride_b;
        a.hk_sh = a.hv_sh = tier.t->hot_stride_h;
        a.hk_sn = a.hv_sn = tier.t->hot_stride_n;
        a.cap = tier.t->capacity;
    }
    if (state4 && !stream_reset) {   // no refine pass
        r.state_out = state4;
        HIP_TRY(launch_topk_emit_attn_stream(r, a, s.dtype, st, stage(e, HILL_STAGE_SELECT)));
    } else {
        r.state_out = state4;   // NULL, or a reset step's fresh bound
        HIP_TRY(launch_topk_refine(r, s.B * s.R, st, stage(e, HILL_STAGE_REFINE)));
        HIP_TRY(launch_topk_emit_attn(r, a, s.dtype, st, stage(e, HILL_STAGE_SELECT)));
    }
    HIP_TRY(launch_merge_write(r, a, idx_out, s.B * s.R, st, stage(e, HILL_STAGE_MERGE)));
    return HILL_OK;
}

}  // namespace

extern "C" {

int hill_abi_version(void) { return HILL_ABI_VERSION; }

const char* hill_status_str(int status)
{
    switch (status) {
    case HILL_OK: return "HILL_OK";
    case HILL_ERR_INVALID_ARG: return "HILL_ERR_INVALID_ARG";
    case HILL_ERR_UNSUPPORTED: return "HILL_ERR_UNSUPPORTED";
    case HILL_ERR_WORKSPACE: return "HILL_ERR_WORKSPACE";
    case HILL_ERR_HIP: return "HILL_ERR_HIP";
    default: return "HILL_ERR_UNKNOWN";
    }
}

const char* hill_last_error(void) { return g_last_error.c_str(); }

hill_status hill_workspace_bytes(const hill_desc* d, int32_t k_sel, size_t* bytes)
{
    Shape s;
    HILL_TRY(check_desc(d, &s, false));
    HILL_TRY(check_ksel(s, k_sel));
    if (!bytes) return fail(HILL_ERR_INVALID_ARG, "bytes is NULL");
    *bytes = layout_for(s, k_sel).end_all;
    return HILL_OK;
}

hill_status hill_score(const hill_desc* d, const void* q, const void* k, float* s_acc, void* ws, size_t ws_bytes,
                       void* stream)
{
    Shape s;
    HILL_TRY(check_desc(d, &s));
    HILL_TRY(check_ptr(q, "q"));
    HILL_TRY(check_ptr(k, "k"));
    HILL_TRY(check_ptr(s_acc, "s"));
    const Layout L = layout_for(s, 1);
    HILL_TRY(check_ws(ws, ws_bytes, L.end_score));
    return run_score(d, s, L, q, k, Sketch{}, s_acc, ws, false, static_cast<hipStream_t>(stream), hill_step_events{});
}

hill_status hill_sketch_keys(const hill_desc* d, const void* k, int8_t* k8, int8_t* k_exp, int64_t cap, int32_t bits,
                             int32_t token_begin, int32_t token_end, void* stream)
{
    Shape s;
    HILL_TRY(check_desc(d, &s, false));
    HILL_TRY(check_ptr(k, "k"));
    HILL_TRY(check_sketch(s, k8, k_exp, cap, bits));
    if (token_begin < 0 || token_begin > token_end || token_end > s.n)
        return fail(HILL_ERR_INVALID_ARG, "token range [%d, %d) not inside [0, n_tokens=%d)", token_begin, token_end, s.n);
    SketchArgs a{};
    a.k = static_cast<const uint16_t*>(k);
    a.k_sb = d->k_stride_b;
    a.k_sh = d->k_stride_h;
    a.k_sn = d->k_stride_n;
    a.B = s.B;
    a.Hkv = s.Hkv;
    a.t0 = token_begin;
    a.t1 = token_end;
    a.cap = cap;
    a.k8 = k8;
    a.k_exp = k_exp;
    a.bits = bits;
    HIP_TRY(launch_sketch_keys(a, s.dtype, static_cast<hipStream_t>(stream)));
    return HILL_OK;
}

// ---------------------------------------------------------------- BKP pools --

struct BkpLayout {
    size_t v, zero, hist1, hist2, cand_key, cand_n, state, sel_list, sel_n, moves, end;
    int64_t zero_words, ld;
    int nchunks;
};

BkpLayout bkp_layout(const hill_bkp_desc* d)
{
    BkpLayout L{};
    const size_t rows = (size_t)d->batch * d->rows;
    const size_t n = (size_t)d->n_tokens;
    L.ld = ((int64_t)n + 3) / 4 * 4;
    L.nchunks = (int)((n + kSelChunk - 1) / kSelChunk);
    size_t off = 0;
    L.v = off;
    off += align256(rows * (size_t)L.ld * sizeof(float));
    L.zero = L.hist1 = off;
    L.hist2 = L.hist1 + rows * kHistRow * sizeof(uint32_t);
    const size_t zero_end = L.hist2 + rows * kHistRow * sizeof(uint32_t);
    L.zero_words = (int64_t)((zero_end - L.zero) / sizeof(uint32_t));
    off = align256(zero_end);
    L.cand_key = off;
    off += align256(rows * n * sizeof(uint32_t));
    L.cand_n = off;
    off += align256(rows * L.nchunks * sizeof(uint32_t));
    L.state = off;
    off += align256(rows * sizeof(uint4));
    L.sel_list = off;
    off += align256(rows * n * sizeof(int32_t));
    L.sel_n = off;
    off += align256(rows * L.nchunks * sizeof(uint32_t));
    L.moves = off;
    off += align256(rows * L.nchunks * sizeof(uint2));
    L.end = off;
    return L;
}

hill_status check_bkp(const hill_bkp_desc* d)
{
    if (!d) return fail(HILL_ERR_INVALID_ARG, "descriptor is NULL");
    if (d->struct_size != sizeof(hill_bkp_desc))
        return fail(HILL_ERR_INVALID_ARG, "struct_size %u != sizeof(hill_bkp_desc) %zu", d->struct_size,
                    sizeof(hill_bkp_desc));
    if (d->batch < 1 || d->rows < 1 || d->n_tokens < 1)
        return fail(HILL_ERR_INVALID_ARG, "batch, rows and n_tokens must be >= 1");
    if ((int64_t)d->batch * d->rows > 65535)
        return fail(HILL_ERR_UNSUPPORTED, "batch * rows %lld exceeds 65535", (long long)d->batch * d->rows);
    if ((int64_t)d->n_tokens > (int64_t)kMaxSlots * kSelChunk)
        return fail(HILL_ERR_UNSUPPORTED, "n_tokens %d exceeds the supported %d", d->n_tokens, kMaxSlots * kSelChunk);
    if (d->n_recent < 0 || d->capacity < d->n_recent)
        return fail(HILL_ERR_INVALID_ARG, "need 0 <= n_recent (%d) <= capacity (%d)", d->n_recent, d->capacity);
    if (d->stride_r < d->n_tokens) return fail(HILL_ERR_INVALID_ARG, "stride_r must be >= n_tokens");
    if (d->batch > 1 && d->stride_b < (int64_t)d->rows * d->stride_r)
        return fail(HILL_ERR_INVALID_ARG, "stride_b must be >= rows * stride_r");
    return HILL_OK;
}

hill_status hill_bkp_workspace_bytes(const hill_bkp_desc* d, size_t* bytes)
{
    HILL_TRY(check_bkp(d));
    if (!bytes) return fail(HILL_ERR_INVALID_ARG, "bytes is NULL");
    *bytes = bkp_layout(d).end;
    return HILL_OK;
}

hill_status hill_bkp_update(const hill_bkp_desc* d, const int32_t* idx, int32_t k_sel, uint16_t* hits, uint8_t* hot,
                            int32_t* promote, int32_t* demote, int32_t list_cap, int32_t* counts, void* ws,
                            size_t ws_bytes, void* stream)
{
    HILL_TRY(check_bkp(d));
    if (k_sel < 0 || k_sel > d->n_tokens)
        return fail(HILL_ERR_INVALID_ARG, "k_sel %d not in [0, n_tokens=%d]", k_sel, d->n_tokens);
    if (k_sel > 0 && (!idx || ((uintptr_t)idx & 3u)))
        return fail(HILL_ERR_INVALID_ARG, "idx is NULL or not 4-byte aligned");
    if (!hits || ((uintptr_t)hits & 1u)) return fail(HILL_ERR_INVALID_ARG, "hits is NULL or not 2-byte aligned");
    if (!hot) return fail(HILL_ERR_INVALID_ARG, "hot is NULL");
    if (list_cap < 0) return fail(HILL_ERR_INVALID_ARG, "list_cap %d < 0", list_cap);
    if (list_cap > 0 && (!promote || !demote || ((uintptr_t)promote & 3u) || ((uintptr_t)demote & 3u)))
        return fail(HILL_ERR_INVALID_ARG, "promote / demote NULL or not 4-byte aligned");
    if (!counts || ((uintptr_t)counts & 3u)) return fail(HILL_ERR_INVALID_ARG, "counts is NULL or not 4-byte aligned");
    const BkpLayout L = bkp_layout(d);
    HILL_TRY(check_ws(ws, ws_bytes, L.end));
    hipStream_t st = static_cast<hipStream_t>(stream);
    const int rows = d->batch * d->rows;
    const int n = d->n_tokens;
    BkpArgs a{};
    a.idx = idx;
    a.k = k_sel;
    a.hits = hits;
    a.hot = hot;
    a.sb = d->stride_b;
    a.sr = d->stride_r;
    a.R = d->rows;
    a.n = n;
    a.w = d->n_recent < n ? d->n_recent : n;
    a.f = (d->capacity < n ? d->capacity : n) - a.w;
    a.pos_shift = 0;
    while (((n - 1) >> a.pos_shift) >= 128) ++a.pos_shift;
    a.v = at<float>(ws, L.v);
    a.ld = L.ld;
    a.zero = at<uint32_t>(ws, L.zero);
    a.zero_words = L.zero_words;
    a.hist1 = at<uint32_t>(ws, L.hist1);
    a.sel_list = at<int32_t>(ws, L.sel_list);
    a.sel_n = at<uint32_t>(ws, L.sel_n);
    a.nchunks = L.nchunks;
    a.chunk_moves = at<uint2>(ws, L.moves);
    a.promote = promote;
    a.demote = demote;
    a.list_cap = list_cap;
    a.counts = counts;
    HIP_TRY(launch_bkp_hits(a, rows, st));
    if (a.f > 0) {   // frequency slots: the exact top-f of the rank values, ties to the lower index
        HIP_TRY(launch_bkp_rank(a, rows, st));
        RefineArgs r{};
        r.s = a.v;
        r.s_sb = (int64_t)d->rows * L.ld;
        r.s_sr = L.ld;
        r.R = d->rows;
        r.n = n;
        r.k = a.f;
        r.nchunks = L.nchunks;
        r.hist1 = at<uint32_t>(ws, L.hist1);
        r.hist2 = at<uint32_t>(ws, L.hist2);
        r.cand_key = at<uint32_t>(ws, L.cand_key);
        r.cand_n = at<uint32_t>(ws, L.cand_n);
        r.state = at<uint4>(ws, L.state);
        r.sel_list = at<int32_t>(ws, L.sel_list);
        r.sel_n = at<uint32_t>(ws, L.sel_n);
        r.pin_lo = 0;
        r.pin_hi = n;
        HIP_TRY(launch_topk_refine(r, rows, st));
        HIP_TRY(launch_topk_emit_lists(r, rows, st));
    }
    HIP_TRY(launch_bkp_lists(a, rows, st));
    return HILL_OK;
}

hill_status hill_app_balance(const hill_app_params* p, hill_app_plan* plan)
{
    if (!p || !plan) return fail(HILL_ERR_INVALID_ARG, "params or plan is NULL");
    const double rates[] = {p->f_c, p->f_s, p->b_c, p->b_s, p->m};
    for (double x : rates)
        if (!std::isfinite(x) || x <= 0.0)
            return fail(HILL_ERR_INVALID_ARG, "throughputs, bandwidths and m must be finite and > 0");
    if (!std::isfinite(p->alpha_c) || !std::isfinite(p->alpha_s) || p->alpha_c < 0.0 || p->alpha_c > 1.0 ||
        p->alpha_s < 0.0 || p->alpha_s > 1.0)
        return fail(HILL_ERR_INVALID_ARG, "alpha_c and alpha_s must lie in [0, 1]");
    if (!std::isfinite(p->m0)) return fail(HILL_ERR_INVALID_ARG, "m0 is not finite");
    // seconds per byte along each path (Eq. 2): scoring plus moving the retained part
    const double a_c = 1.0 / p->f_c + p->alpha_c / p->b_c;
    const double a_s = 1.0 / p->f_s + p->alpha_s / p->b_s;
    hill_app_plan r{};
    r.m_c = p->m * a_s / (a_c + a_s);   // a_c * M_c == a_s * (M - M_c)
    if (p->m0 > 0.0 && r.m_c > p->m0) {
        r.m_c = p->m0;
        r.capped = 1;
    }
    r.m_s = p->m - r.m_c;
    r.beta = r.m_s > 0.0 ? r.m_c / r.m_s : HUGE_VAL;
    r.t_c = a_c * r.m_c;
    r.t_s = a_s * r.m_s;
    *plan = r;
    return HILL_OK;
}

hill_status hill_score_sketch(const hill_desc* d, const void* q, const int8_t* k8, const int8_t* k_exp, int64_t cap,
                              int32_t bits, float* s_acc, void* ws, size_t ws_bytes, void* stream)
{
    Shape s;
    HILL_TRY(check_desc(d, &s));
    HILL_TRY(check_ptr(q, "q"));
    HILL_TRY(check_sketch(s, k8, k_exp, cap, bits));
    HILL_TRY(check_ptr(s_acc, "s"));
    const Layout L = layout_for(s, 1);
    HILL_TRY(check_ws(ws, ws_bytes, L.end_score));
    return run_score(d, s, L, q, nullptr, Sketch{k8, k_exp, cap, bits}, s_acc, ws, false, static_cast<hipStream_t>(stream),
                     hill_step_events{});
}

hill_status hill_topk(const hill_desc* d, const float* s_acc, int32_t k_sel, int32_t* idx_out, float* val_out,
                      void* ws, size_t ws_bytes, void* stream)
{
    Shape s;
    HILL_TRY(check_desc(d, &s));
    HILL_TRY(check_ksel(s, k_sel));
    HILL_TRY(check_pins(s, k_sel));
    HILL_TRY(check_ptr(s_acc, "s"));
    if (!idx_out) return fail(HILL_ERR_INVALID_ARG, "idx_out is NULL");
    if ((uintptr_t)idx_out & 3u) return fail(HILL_ERR_INVALID_ARG, "idx_out is not 4-byte aligned");
    if (val_out && ((uintptr_t)val_out & 3u)) return fail(HILL_ERR_INVALID_ARG, "val_out is not 4-byte aligned");
    const Layout L = layout_for(s, k_sel);
    HILL_TRY(check_ws(ws, ws_bytes, L.end_topk));
    return run_select(d, s, L, s_acc, k_sel, idx_out, val_out, ws, static_cast<hipStream_t>(stream));
}

hill_status hill_gather_attn(const hill_desc* d, const void* q, const void* k, const void* v, const int32_t* idx,
                             int32_t k_sel, float* out, void* ws, size_t ws_bytes, void* stream)
{
    Shape s;
    HILL_TRY(check_desc(d, &s, false));
    HILL_TRY(check_ksel(s, k_sel));
    HILL_TRY(check_ptr(q, "q"));
    HILL_TRY(check_ptr(k, "k"));
    HILL_TRY(check_ptr(v, "v"));
    HILL_TRY(check_ptr(out, "out"));
    if (!idx) return fail(HILL_ERR_INVALID_ARG, "idx is NULL");
    if ((uintptr_t)idx & 3u) return fail(HILL_ERR_INVALID_ARG, "idx is not 4-byte aligned");
    const Layout L = layout_for(s, k_sel);
    HILL_TRY(check_ws(ws, ws_bytes, L.end_all));
    return run_attn(d, s, L, q, k, v, idx, k_sel, out, ws, static_cast<hipStream_t>(stream));
}

hill_status hill_step(const hill_desc* d, const void* q, const void* k, const void* v, float* s_acc, int32_t k_sel,
                      int32_t* idx_out, float* out, void* ws, size_t ws_bytes, void* stream)
{
    return hill_step_profiled(d, q, k, v, s_acc, k_sel, idx_out, out, ws, ws_bytes, stream, nullptr);
}

hill_status hill_step_profiled(const hill_desc* d, const void* q, const void* k, const void* v, float* s_acc,
                               int32_t k_sel, int32_t* idx_out, float* out, void* ws, size_t ws_bytes, void* stream,
                               const hill_step_events* ev)
{
    return run_step(d, q, k, v, Sketch{}, s_acc, k_sel, idx_out, out, ws, ws_bytes, stream, ev);
}

hill_status hill_step_noalloc(const hill_desc* d, const void* q, const void* k, const void* v, float* s_acc,
                              int32_t k_sel, int32_t* idx_out, float* out, void* stream)
{
    Shape s;
    HILL_TRY(check_step(d, q, k, v, Sketch{}, s_acc, k_sel, idx_out, out, &s));
    const size_t need = layout_for(s, k_sel).end_all;
    if (need > kStaticScratchBytes)
        return fail(HILL_ERR_WORKSPACE, "this step needs %zu bytes of scratch, more than the %zu of the fixed device buffer",
                    need, (size_t)kStaticScratchBytes);
    void* ws = nullptr;
    const hipError_t e = static_scratch(&ws);
    if (e != hipSuccess) return fail(HILL_ERR_HIP, "fixed device scratch: %s", hipGetErrorString(e));
    return run_step(d, q, k, v, Sketch{}, s_acc, k_sel, idx_out, out, ws, kStaticScratchBytes, stream, nullptr);
}

static hill_status check_stream_flags(const uint32_t* state, uint32_t flags)
{
    if (flags & ~HILL_STREAM_RESET) return fail(HILL_ERR_INVALID_ARG, "unknown streamed-selection flags 0x%x", flags);
    if (flags && !state) return fail(HILL_ERR_INVALID_ARG, "streamed-selection flags without a state");
    return HILL_OK;
}

hill_status hill_step_streamed(const hill_desc* d, const void* q, const void* k, const void* v, float* s_acc,
                               uint32_t* state, uint32_t flags, int32_t k_sel, int32_t* idx_out, float* out, void* ws,
                               size_t ws_bytes, void* stream, const hill_step_events* ev)
{
    if (!d) return fail(HILL_ERR_INVALID_ARG, "descriptor is NULL");
    if (d->score_mode != HILL_SCORE_ATTN)
        return fail(HILL_ERR_UNSUPPORTED, "streamed selection needs ATTN scores (S must only grow)");
    if (!state || ((uintptr_t)state & 15u)) return fail(HILL_ERR_INVALID_ARG, "state is NULL or not 16-byte aligned");
    HILL_TRY(check_stream_flags(state, flags));
    return run_step(d, q, k, v, Sketch{}, s_acc, k_sel, idx_out, out, ws, ws_bytes, stream, ev, state,
                    (flags & HILL_STREAM_RESET) != 0);
}

hill_status hill_step_sketch(const hill_desc* d, const void* q, const void* k, const void* v, const int8_t* k8,
                             const int8_t* k_exp, int64_t cap, int32_t bits, float* s_acc, uint32_t* state,
                             uint32_t flags, int32_t k_sel, int32_t* idx_out, float* out, void* ws, size_t ws_bytes,
                             void* stream, const hill_step_events* ev)
{
    if (!k8 || !k_exp) return fail(HILL_ERR_INVALID_ARG, "sketch codes or exponents are NULL");
    HILL_TRY(check_stream_flags(state, flags));
    if (state) {
        if (!d) return fail(HILL_ERR_INVALID_ARG, "descriptor is NULL");
        if (d->score_mode != HILL_SCORE_ATTN)
            return fail(HILL_ERR_UNSUPPORTED, "streamed selection needs ATTN scores (S must only grow)");
        if ((uintptr_t)state & 15u) return fail(HILL_ERR_INVALID_ARG, "state is not 16-byte aligned");
    }
    return run_step(d, q, k, v, Sketch{k8, k_exp, cap, bits}, s_acc, k_sel, idx_out, out, ws, ws_bytes, stream, ev,
                    state, (flags & HILL_STREAM_RESET) != 0);
}

hill_status hill_step_tiered(const hill_desc* d, const hill_tier_desc* t, const void* q, const void* k_hot,
                             const void* v_hot, const void* k_cold, const void* v_cold, const int32_t* loc,
                             const int8_t* k8, const int8_t* k_exp, int64_t cap, int32_t bits, float* s_acc,
                             uint32_t* state, uint32_t flags, int32_t k_sel, int32_t* idx_out, float* out, void* ws,
                             size_t ws_bytes, void* stream, const hill_step_events* ev)
{
    if (!t) return fail(HILL_ERR_INVALID_ARG, "tier descriptor is NULL");
    if (!k8 || !k_exp) return fail(HILL_ERR_INVALID_ARG, "sketch codes or exponents are NULL");
    HILL_TRY(check_stream_flags(state, flags));
    if (state) {
        if (!d) return fail(HILL_ERR_INVALID_ARG, "descriptor is NULL");
        if (d->score_mode != HILL_SCORE_ATTN)
            return fail(HILL_ERR_UNSUPPORTED, "streamed selection needs ATTN scores (S must only grow)");
        if ((uintptr_t)state & 15u) return fail(HILL_ERR_INVALID_ARG, "state is not 16-byte aligned");
    }
    if (loc && ((uintptr_t)loc & 15u)) return fail(HILL_ERR_INVALID_ARG, "loc is not 16-byte aligned");
    Tier tier;
    tier.t = t;
    tier.k_hot = k_hot;
    tier.v_hot = v_hot;
    tier.loc = loc;
    return run_step(d, q, k_cold, v_cold, Sketch{k8, k_exp, cap, bits}, s_acc, k_sel, idx_out, out, ws, ws_bytes,
                    stream, ev, state, (flags & HILL_STREAM_RESET) != 0, tier);
}

hill_status hill_tier_apply(const hill_desc* d, const hill_tier_desc* t, void* k_hot, void* v_hot, void* k_cold,
                            void* v_cold, int32_t* loc, const int32_t* promote, const int32_t* demote,
                            int32_t list_cap, const int32_t* counts, int32_t n_prev, int32_t* status, void* stream)
{
    Shape s;
    HILL_TRY(check_desc(d, &s, false));
    HILL_TRY(check_tier(s, t));
    HILL_TRY(check_ptr(k_hot, "k_hot"));
    HILL_TRY(check_ptr(v_hot, "v_hot"));
    HILL_TRY(check_ptr(k_cold, "k_cold"));
    HILL_TRY(check_ptr(v_cold, "v_cold"));
    HILL_TRY(check_ptr(loc, "loc"));
    if (list_cap < 1) return fail(HILL_ERR_INVALID_ARG, "list_cap %d < 1", list_cap);
    HILL_TRY(check_reachable(k_cold, "k_cold"));
    HILL_TRY(check_reachable(v_cold, "v_cold"));
    if (!promote || !demote || ((uintptr_t)promote & 3u) || ((uintptr_t)demote & 3u))
        return fail(HILL_ERR_INVALID_ARG, "promote / demote NULL or not 4-byte aligned");
    if (!counts || ((uintptr_t)counts & 3u)) return fail(HILL_ERR_INVALID_ARG, "counts is NULL or not 4-byte aligned");
    if (!status || ((uintptr_t)status & 3u)) return fail(HILL_ERR_INVALID_ARG, "status is NULL or not 4-byte aligned");
    if (n_prev < 0 || n_prev > s.n)
        return fail(HILL_ERR_INVALID_ARG, "n_prev %d not in [0, n_tokens=%d]", n_prev, s.n);
    if ((int64_t)s.B * s.R > 65535) return fail(HILL_ERR_UNSUPPORTED, "batch * rows above 65535");
    TierArgs a{};
    a.k_hot = static_cast<uint16_t*>(k_hot);
    a.v_hot = static_cast<uint16_t*>(v_hot);
    a.k_cold = static_cast<uint16_t*>(k_cold);
    a.v_cold = static_cast<uint16_t*>(v_cold);
    a.hk_sb = a.hv_sb = t->hot_stride_b;
    a.hk_sh = a.hv_sh = t->hot_stride_h;
    a.hk_sn = a.hv_sn = t->hot_stride_n;
    a.ck_sb = d->k_stride_b;
    a.ck_sh = d->k_stride_h;
    a.ck_sn = d->k_stride_n;
    a.cv_sb = d->v_stride_b;
    a.cv_sh = d->v_stride_h;
    a.cv_sn = d->v_stride_n;
    a.loc = loc;
    a.loc_sr = t->n_cap;
    a.promote = promote;
    a.demote = demote;
    a.counts = counts;
    a.list_cap = list_cap;
    a.R = s.R;
    a.Hkv = s.Hkv;
    a.n = s.n;
    a.cap = t->capacity;
    a.used_prev = n_prev < t->capacity ? n_prev : t->capacity;
    a.used_now = s.n < t->capacity ? s.n : t->capacity;
    a.status = status;
    HIP_TRY(launch_tier_apply(a, s.B * s.R, static_cast<hipStream_t>(stream)));
    return HILL_OK;
}

}  // extern "C"
