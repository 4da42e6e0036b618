// Importance update on gfx950 (Sec. 4.1 metric): the kernels that consume
// the scan's logits (score.hip).
//
//  softmax_stats reduces the scan's unit pairs to one (max, 1/sum) per head:
//                the softmax normaliser over all n tokens of Eq. 1.  Only for
//                rows longer than the update can reduce itself.
//  update_attn   turns logits into softmax weights and adds their sum over
//                the row's heads to the cumulative importance S, counts the
//                first radix digit of the new S for the selection and, for
//                the streamed selection (Sec. 4.2 HIE's running threshold),
//                lists the tokens at or above the previous threshold's bin.
//  update_raw_groups (RAW, token rows, Hkv > 1) adds the scan's per-group
//                sums of raw logits to S.
#include <hip/hip_ext.h>

#include "hill_device.h"
#include "hill_internal.h"

namespace hill {

namespace {

// One workgroup per (b, h): combine the unit pairs into (max, 1/sum), each
// thread over a fixed strided subset, then waves in a fixed order.  Used when
// the update cannot reduce them itself (long contexts).
__global__ __launch_bounds__(256) void softmax_stats_kernel(const float2* __restrict__ part,
                                                            float2* __restrict__ stats, int npart)
{
    __shared__ float red_m[4], red_z[4];
    const int bh = blockIdx.x;
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const float2* p = part + (int64_t)bh * npart;
    constexpr int kBatch = 8;
    float m = -INFINITY, z = 0.0f;
    for (int i0 = tid; i0 < npart; i0 += 256 * kBatch) {
        float2 v[kBatch];
#pragma unroll
        for (int u = 0; u < kBatch; ++u) {
            const int i = i0 + u * 256;
            v[u] = i < npart ? p[i] : make_float2(-INFINITY, 0.0f);
        }
#pragma unroll
        for (int u = 0; u < kBatch; ++u) {
            if (v[u].x == -INFINITY) continue;
            const float mn = fmaxf(m, v[u].x);
            z = z * exp2_ftz(m - mn) + v[u].y * exp2_ftz(v[u].x - mn);
            m = mn;
        }
    }
    const float mw = wave_max(m);
    z = m > -INFINITY ? z * exp2_ftz(m - mw) : 0.0f;
    z = wave_sum(z);
    if (lane == 0) {
        red_m[w] = mw;
        red_z[w] = z;
    }
    __syncthreads();
    if (tid == 0) {
        float M = red_m[0];
        for (int i = 1; i < 4; ++i) M = fmaxf(M, red_m[i]);
        float Z = 0.0f;
        for (int i = 0; i < 4; ++i) Z += red_m[i] > -INFINITY ? red_z[i] * exp2_ftz(red_m[i] - M) : 0.0f;
        stats[bh] = make_float2(M, 1.0f / Z);
    }
}

// First-digit histogram of the importance keys a workgroup writes (bits
// 31..20), counted in LDS without returning atomics, with a bitmap of the bins
// touched.  The flush adds the touched bins to the row's histogram one 64-bin
// window per instruction (a wave's lanes hold consecutive bins, so a hot
// window costs one request per cache line, not one per bin) and derives the
// coarse bins (bits 31..26: one window each) from the same loads, flushed
// together at the end.  NT: threads of the workgroup (256 or 512).
struct KeyHist {
    alignas(16) uint32_t bins[kHistBins];
    uint32_t mark[kHistBins / 32];
    uint32_t coarse[kCoarseBins];
};

template <int NT>
__device__ __forceinline__ void key_hist_clear(KeyHist& h)
{
    uint4* b4 = reinterpret_cast<uint4*>(h.bins);
    for (int i = threadIdx.x; i < kHistBins / 4; i += NT) b4[i] = make_uint4(0u, 0u, 0u, 0u);
    if (threadIdx.x < kHistBins / 32) h.mark[threadIdx.x] = 0u;
    if (threadIdx.x < kCoarseBins) h.coarse[threadIdx.x] = 0u;
}

__device__ __forceinline__ void count_key(KeyHist& h, uint32_t key)
{
    const uint32_t d = key >> (32 - kHistBits);
    atomicAdd(&h.bins[d], 1u);
    atomicOr(&h.mark[d >> 5], 1u << (d & 31));
}

// After a barrier; every thread calls it (it ends with a barrier of its own).
// Wave w of the NW = NT/64 waves owns windows w, w+NW, ...: lane l < 2*64/NW
// reads bitmap word l of them (window w + NW * (l / 2), half l % 2), one
// ballot names the touched windows, and the wave flushes only those.
// Integer atomics: order-independent.
template <int NT>
__device__ __forceinline__ void key_hist_flush(KeyHist& h, uint32_t* ghist)
{
    static_assert(kHistBins == 64 * kCoarseBins, "one coarse bin per 64-bin window");
    constexpr int NW = NT / 64, kWords = 2 * kCoarseBins / NW;
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const uint32_t mw = lane < kWords ? h.mark[2 * (w + NW * (lane >> 1)) + (lane & 1)] : 0u;
    uint64_t live = __ballot(mw != 0u);   // wave-uniform
    while (live) {
        const int i = __builtin_ctzll(live) >> 1;
        live &= ~(3ull << (2 * i));
        const int c = w + NW * i;
        const uint32_t v = h.bins[c * 64 + lane];
        if (v) atomicAdd(ghist + c * 64 + lane, v);
        const uint32_t tot = wave_sum_u32(v);
        if (lane == 0) h.coarse[c] = tot;
    }
    __syncthreads();
    if (threadIdx.x < kCoarseBins) {
        const uint32_t v = h.coarse[threadIdx.x];
        if (v) atomicAdd(ghist + kHistBins + threadIdx.x, v);
    }
}

constexpr int kHeadBatch = 4;   // float2 logits loads in flight per thread (update_attn)
constexpr int kRawBatch = 8;    // float2 group-sum loads in flight per thread (update_raw_groups)
constexpr int kUpdWaves = kUpdThreads / 64;
constexpr int kTokWaves = kUpdChunk / 64;   // waves whose threads finish a token (thread t < kUpdChunk)
static_assert(kUpdChunk % 64 == 0 && kTokWaves <= kUpdWaves, "whole waves of tokens");

// First-digit bound of the streamed selection for this row: the first digit
// of the previous step's threshold, while the keys at or above that bin then
// were at least this step's k (S only grows), the pins are the same and n did
// not shrink (n may only grow without pins); with 0x80000000 set.  Else 0
// (no bound: every token is a candidate).
// p0, p1: the row's two state words, loaded by the caller with its other
// loads (the test is branch-free, so nothing waits for them early).
__device__ __forceinline__ uint32_t stream_bound(const UpdateArgs& a, uint4 p0, uint4 p1)
{
    const bool nopins = (a.pin_lo == 0) & (a.pin_hi == a.n);
    const bool ok = (p0.w == 1u) & ((uint32_t)a.k <= p0.y) & ((uint32_t)a.n >= p0.z) &
                    (p1.x == (uint32_t)a.pin_lo) & (p1.y == (uint32_t)(a.n - a.pin_hi)) &
                    (((uint32_t)a.n == p0.z) | nopins);
    return ok ? (p0.x >> (32 - kHistBits)) | 0x80000000u : 0u;
}

// Streamed selection: the block's tokens whose first digit reaches the bound
// go to the block's slot of the row's (key, token) list, grouped by class --
// the key's window bin (the bound's first-digit bin or one of the next
// kStreamBins - 1) or, for every key above the window (and for every key when
// there is no bound), class kStreamBins -- with the counts of the classes.
// The selection sums those counts over the row's blocks to find the first
// digit of the k-th key (with a bound it lies in the window or above), and a
// walk for one first-digit bin reads one class only.  Keys in the window also
// count their second digit (fine bins, straight to memory: they spread over
// the window's 4 x 4096 bins; the threshold seldom moves further in one step).
// Two halves around the caller's barrier: stream_rank (class, rank within the
// class in the wave, wave counts into LDS) and stream_store (the pair at its
// slot position, the class counts).
struct StreamRank {
    bool cand;
    int cls;
    uint32_t rank;
};

__device__ __forceinline__ StreamRank stream_rank(const UpdateArgs& a, int row, int j, uint32_t key, uint32_t bnd,
                                                  uint32_t (*wcnt)[kTokWaves])
{
    const uint32_t d0 = bnd & (kHistBins - 1);
    const uint32_t dig = key >> (32 - kHistBits);
    StreamRank s;
    s.cand = j < a.n && dig >= d0;
    const uint32_t wdx = dig - d0;   // window bin of the key (valid when cand)
    const bool win = s.cand && (bnd >> 31) && wdx < (uint32_t)kStreamBins;
    s.cls = win ? (int)wdx : kStreamBins;
    const int64_t rows = (int64_t)a.B * a.R;
    if (win) atomicAdd(&a.hist2[((int64_t)wdx * rows + row) * kHistRow + ((key >> 8) & (kHistBins - 1))], 1u);
    // rank within the class: one ballot per class, wave counts through LDS
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const uint64_t below = (1ull << lane) - 1ull;
    s.rank = 0;
#pragma unroll
    for (int k = 0; k < kPairClasses; ++k) {
        const uint64_t m = __ballot(s.cand && s.cls == k);
        if (s.cand && s.cls == k) s.rank = (uint32_t)__popcll(m & below);
        if (lane == 0) wcnt[k][w] = (uint32_t)__popcll(m);
    }
    return s;
}

__device__ __forceinline__ uint32_t class_total(const uint32_t (*wcnt)[kTokWaves], int k)
{
    uint32_t t = 0u;
#pragma unroll
    for (int v = 0; v < kTokWaves; ++v) t += wcnt[k][v];
    return t;
}

__device__ __forceinline__ void stream_store(const UpdateArgs& a, int row, int j, uint32_t key, uint32_t bnd,
                                             const StreamRank& s, const uint32_t (*wcnt)[kTokWaves])
{
    const int w = threadIdx.x >> 6;
    if (s.cand) {
        uint32_t pos = s.rank;
        for (int k = 0; k < s.cls; ++k) pos += class_total(wcnt, k);
        for (int v = 0; v < w; ++v) pos += wcnt[s.cls][v];
        a.spairs[(int64_t)row * a.n + (int64_t)blockIdx.x * kUpdChunk + pos] = make_uint2(key, (uint32_t)j);
    }
    const int nup = (a.n + kUpdChunk - 1) / kUpdChunk;
    if (threadIdx.x == 0) {
        uint32_t c[kPairClasses];
#pragma unroll
        for (int k = 0; k < kPairClasses; ++k) c[k] = class_total(wcnt, k);
        uint4* slot = reinterpret_cast<uint4*>(a.scount + ((int64_t)row * nup + blockIdx.x) * kSlotWords);
        static_assert(kSlotWords == 8 && kPairClasses == 5, "two 16-byte words per slot");
        slot[0] = make_uint4(c[0], c[1], c[2], c[3]);
        slot[1] = make_uint4(c[4], bnd, 0u, 0u);
    }
}

// (max, 1/sum) of heads h0 .. h0+nh of sequence b into ms[]: copied from the
// stats kernel's output, or reduced here from the unit partials.  Thread t
// works for head t / tph (tph = kUpdThreads / nh threads per head) and holds
// the partial pairs t % tph, + tph, ... (at most kStatLoads partials); the
// head's maximum is taken first (DPP within a wave when tph is a power of two
// up to 64, else through LDS by one thread per head), then every pair's sum is
// scaled to it with one exp2 and the scaled sums are added the same way.  The
// partial loads are issued by load_head_parts() before the logits; every
// thread calls finish_head_stats(), which ends with a barrier.
struct HeadParts {
    float2 v[kStatLoads];
};

// Thread t's head among the heads of a row (tph threads each, set by the
// host with its reciprocal): t / tph as a float product, exact for t < 512 and
// tph <= 512 -- (t + 1/2) / tph lies at least 1/(2 tph) from an integer, far
// more than the product's rounding.
__device__ __forceinline__ int head_of_thread(const UpdateArgs& a, int t)
{
    return (int)(((float)t + 0.5f) * a.inv_tph);
}

// p: the row's first head's partials (uniform); hh, sub: this thread's head
// and its place among the head's threads.
__device__ __forceinline__ void load_head_parts(const UpdateArgs& a, const float2* p2, int hh, int sub, int nh,
                                                HeadParts& hp)
{
    const int tph = a.tph;
    const bool active = a.stats == nullptr && hh < nh;
    // npart is even and the rows 16-byte aligned: pairs of partials per load;
    // per-thread offsets in 32 bits (at most 256 heads x 2^20 partials)
    const int npair = a.npart / 2;
    const float4* p = reinterpret_cast<const float4*>(p2) + (uint32_t)((active ? hh : 0) * npair);
#pragma unroll
    for (int i = 0; i < kStatLoads / 2; ++i) {
        // consecutive lanes read consecutive pairs; unconditional (clamped)
        // loads, invalid ones replaced afterwards
        const int idx = sub + i * tph;
        const float4 v = p[(uint32_t)min(idx, npair - 1)];
        const bool ok = active && idx < npair;
        hp.v[2 * i] = ok ? make_float2(v.x, v.y) : make_float2(-INFINITY, 0.0f);
        hp.v[2 * i + 1] = ok ? make_float2(v.z, v.w) : make_float2(-INFINITY, 0.0f);
    }
}

// max (or, ADD, sum) over the aligned group of tph lanes (tph a power of two,
// 2..64); every lane of the group gets it.
template <bool ADD>
__device__ __forceinline__ float group_fold(float v, int tph)
{
    auto op = [](float x, float y) { return ADD ? x + y : fmaxf(x, y); };
    v = op(v, dpp<0xB1>(v));                         // lane ^ 1
    if (tph >= 4) v = op(v, dpp<0x4E>(v));           // lane ^ 2
    if (tph >= 8) v = op(v, dpp<0x141>(v));          // mirror within 8
    if (tph >= 16) v = op(v, dpp<0x140>(v));         // mirror within 16
    if (tph >= 32) v = op(v, __shfl_xor(v, 16, 64));
    if (tph >= 64) v = op(v, __shfl_xor(v, 32, 64));
    return v;
}

// red: kUpdThreads float2 of LDS; ms: the heads' (max, 1/sum)
__device__ __forceinline__ void finish_head_stats(const UpdateArgs& a, int b, int h0, int nh, int hh,
                                                  const HeadParts& hp, float2* red, float2* ms)
{
    const int t = threadIdx.x;
    if (a.stats) {
        if (t < nh) ms[t] = a.stats[(int64_t)b * a.Hq + h0 + t];
        __syncthreads();
        return;
    }
    float m = -INFINITY;
#pragma unroll
    for (int i = 0; i < kStatLoads; ++i) m = fmaxf(m, hp.v[i].x);
    const int tph = a.tph;
    const bool dpp_path = (tph & (tph - 1)) == 0 && tph >= 2 && tph <= 64;   // block-uniform
    if (dpp_path) {
        m = group_fold<false>(m, tph);   // every lane is active here; groups of tph lanes are aligned
    } else {
        red[t].x = m;
        __syncthreads();
        if (t < nh) {
            float M = -INFINITY;
            for (int i = 0; i < tph; ++i) M = fmaxf(M, red[t * tph + i].x);
            ms[t].x = M;
        }
        __syncthreads();
        m = hh < nh ? ms[hh].x : -INFINITY;
    }
    float z = 0.0f;
#pragma unroll
    for (int i = 0; i < kStatLoads; ++i) z += hp.v[i].x == -INFINITY ? 0.0f : hp.v[i].y * exp2_ftz(hp.v[i].x - m);
    if (dpp_path) {
        z = group_fold<true>(z, tph);
        if (t == hh * tph && hh < nh) ms[hh] = make_float2(m, 1.0f / z);
    } else {
        red[t].y = z;
        __syncthreads();
        if (t < nh) {
            float Z = 0.0f;
            for (int i = 0; i < tph; ++i) Z += red[t * tph + i].y;
            ms[t].y = 1.0f / Z;
        }
    }
    __syncthreads();
}

// S[b,r,j] += sum_{h in heads(r)} exp2(s2*l - max_h) / sum_h   (softmax weights).
// kUpdChunk = 128 tokens per workgroup of kUpdThreads = 512 threads (one
// workgroup per CU at a 32K-token row, two waves per SIMD to hide the
// latency of the short dependent chains): lane l of wave w loads tokens
// [2l, 2l+2) of heads w, w+8, ... as float2 (unconditional loads, heads
// clamped into the row's; heads past it weigh nothing); the eight wave
// partials are added in wave order, then thread t < 128 finishes token t.
// The head statistics come from the stats kernel or, for short rows, from the
// unit partials reduced here.  The first-digit histogram of the new keys
// (LDS, then the touched windows) is counted for the refine pass and for a
// streamed selection without a bound; with a bound the selection takes the
// first digit from the class counts of the pairs.
__global__ __launch_bounds__(kUpdThreads) void update_attn_kernel(UpdateArgs a)
{
    __shared__ float2 wsum[kUpdWaves][64];
    __shared__ KeyHist kh;
    __shared__ float2 red[kUpdThreads];
    __shared__ float2 ms[256];
    __shared__ uint32_t sc_wcnt[kPairClasses][kTokWaves];
    const int r = blockIdx.y, b = blockIdx.z;
    const int row = b * a.R + r;
    const int h0 = a.R == 1 ? 0 : r * a.G;
    const int nh = a.R == 1 ? a.Hq : a.G;
    const int tid = threadIdx.x, lane = tid & 63;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int hh = head_of_thread(a, tid);                // this thread's head in the statistics
    // Every load of the opening is issued before anything waits for one: the
    // softmax partials, this thread's old S, the first batch of logits and the
    // streamed selection's state (whose test runs only after the statistics).
    HeadParts hp;
    load_head_parts(a, a.part + ((int64_t)b * a.Hq + h0) * a.npart, hh, tid - hh * a.tph, nh, hp);
    const int j2 = blockIdx.x * kUpdChunk + 2 * lane;     // first of this lane's 2 tokens
    const int jc = min(j2, (int)(a.ld - 2));              // rows are padded to ld (multiple of 4)
    const float* lg = a.logits + ((int64_t)b * a.Hq + h0) * a.ld + jc;
    // thread tid < kUpdChunk finishes token j; the others hold no token
    const int j = tid < kUpdChunk ? blockIdx.x * kUpdChunk + tid : a.n;
    float* srow = a.s + (int64_t)b * a.s_sb + (int64_t)r * a.s_sr;
    const float s_ld = srow[min(j, a.n - 1)];             // unconditional: no branch around the load
    float2 x[kHeadBatch];
#pragma unroll
    for (int i = 0; i < kHeadBatch; ++i)
        x[i] = *reinterpret_cast<const float2*>(lg + (int64_t)min(w + kUpdWaves * i, nh - 1) * a.ld);
    uint4 p0 = make_uint4(0u, 0u, 0u, 0u), p1 = p0;
    if (a.prev) {
        p0 = a.prev[2 * row];
        p1 = a.prev[2 * row + 1];
    }
    __builtin_amdgcn_sched_barrier(0);
    if (a.hist) key_hist_clear<kUpdThreads>(kh);
    finish_head_stats(a, b, h0, nh, hh, hp, red, ms);
    const float s_old = j < a.n ? s_ld : 0.0f;
    const uint32_t bnd = a.prev ? stream_bound(a, p0, p1) : 0u;
    const bool do_hist = a.hist != nullptr && !(bnd >> 31);   // block-uniform
    float2 acc = make_float2(0.0f, 0.0f);
    for (int hb = w;;) {
        float2 st[kHeadBatch];   // every statistics read of the batch before the first use
#pragma unroll
        for (int i = 0; i < kHeadBatch; ++i) st[i] = ms[min(hb + kUpdWaves * i, nh - 1)];
#pragma unroll
        for (int i = 0; i < kHeadBatch; ++i) {
            const float e0 = exp2_ftz(a.s2 * x[i].x - st[i].x) * st[i].y;
            const float e1 = exp2_ftz(a.s2 * x[i].y - st[i].x) * st[i].y;
            const bool live = hb + kUpdWaves * i < nh;   // wave-uniform
            acc.x += live ? e0 : 0.0f;
            acc.y += live ? e1 : 0.0f;
        }
        hb += kUpdWaves * kHeadBatch;
        if (hb >= nh) break;
#pragma unroll
        for (int i = 0; i < kHeadBatch; ++i)
            x[i] = *reinterpret_cast<const float2*>(lg + (int64_t)min(hb + kUpdWaves * i, nh - 1) * a.ld);
    }
    wsum[w][lane] = acc;
    __syncthreads();
    const float* ws = reinterpret_cast<const float*>(&wsum[0][0]);
    uint32_t key = 0u;
    if (j < a.n) {
        float tot = ws[tid];
#pragma unroll
        for (int v = 1; v < kUpdWaves; ++v) tot += ws[v * 2 * 64 + tid];
        const float s_new = s_old + tot;
        srow[j] = s_new;
        key = select_key(s_new, j, a.pin_lo, a.pin_hi);
        if (do_hist) count_key(kh, key);
    }
    // the streamed selection's ranks and pairs: the token waves only (the others
    // would share SIMDs with them for nothing)
    StreamRank sr{};
    if (a.prev && w < kTokWaves) sr = stream_rank(a, row, j, key, bnd, sc_wcnt);   // wave-uniform
    __syncthreads();
    if (do_hist) key_hist_flush<kUpdThreads>(kh, a.hist + (int64_t)row * kHistRow);
    if (a.prev && w < kTokWaves) stream_store(a, row, j, key, bnd, sr, sc_wcnt);
}

// Token rows, RAW mode, Hkv > 1: S[b,0,j] += sum_g groupsum[b,g,j] (same layout).
__global__ __launch_bounds__(256) void update_raw_groups_kernel(UpdateArgs a)
{
    __shared__ float2 wsum[4][64];
    __shared__ KeyHist kh;
    const int b = blockIdx.y;
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const bool do_hist = a.hist != nullptr;
    if (do_hist) key_hist_clear<256>(kh);
    const int j2 = blockIdx.x * kUpdChunk + 2 * lane;
    const int jc = min(j2, (int)(a.ld - 2));
    const float* gs = a.logits + (int64_t)b * a.Hkv * a.ld + jc;
    const int j = tid < kUpdChunk ? blockIdx.x * kUpdChunk + tid : a.n;
    float* srow = a.s + (int64_t)b * a.s_sb;
    const float s_old = j < a.n ? srow[j] : 0.0f;
    float2 acc = make_float2(0.0f, 0.0f);
    for (int gb = w; gb < a.Hkv; gb += 4 * kRawBatch) {
        float2 x[kRawBatch];
#pragma unroll
        for (int i = 0; i < kRawBatch; ++i) {
            const int g = gb + 4 * i;
            x[i] = g < a.Hkv ? *reinterpret_cast<const float2*>(gs + (int64_t)g * a.ld) : make_float2(0.f, 0.f);
        }
#pragma unroll
        for (int i = 0; i < kRawBatch; ++i) {
            acc.x += x[i].x;
            acc.y += x[i].y;
        }
    }
    wsum[w][lane] = acc;
    __syncthreads();
    const float* ws = reinterpret_cast<const float*>(&wsum[0][0]);
    if (j < a.n) {
        const float tot = ((ws[tid] + ws[128 + tid]) + ws[256 + tid]) + ws[384 + tid];
        const float s_new = s_old + tot;
        srow[j] = s_new;
        if (do_hist) count_key(kh, select_key(s_new, j, a.pin_lo, a.pin_hi));
    }
    if (do_hist) {
        __syncthreads();
        key_hist_flush<256>(kh, a.hist + (int64_t)b * kHistRow);
    }
}

}  // namespace

hipError_t launch_softmax_stats(const float2* part, float2* stats, int bh, int npart, hipStream_t st, Stamp ts)
{
    hipExtLaunchKernelGGL(softmax_stats_kernel, dim3(bh), dim3(256), 0, st, ts.start, ts.stop, 0, part, stats, npart);
    return hipGetLastError();
}

hipError_t launch_update_attn(const UpdateArgs& a, hipStream_t st, Stamp ts)
{
    const int nh = a.R == 1 ? a.Hq : a.G;
    if (nh < 1 || a.tph != kUpdThreads / nh || a.B > 65535 || a.R > 65535) return hipErrorInvalidValue;
    dim3 grid((a.n + kUpdChunk - 1) / kUpdChunk, a.R, a.B);
    hipExtLaunchKernelGGL(update_attn_kernel, grid, dim3(kUpdThreads), 0, st, ts.start, ts.stop, 0, a);
    return hipGetLastError();
}

hipError_t launch_update_raw_groups(const UpdateArgs& a, hipStream_t st, Stamp ts)
{
    dim3 grid((a.n + kUpdChunk - 1) / kUpdChunk, a.B);
    hipExtLaunchKernelGGL(update_raw_groups_kernel, grid, dim3(256), 0, st, ts.start, ts.stop, 0, a);
    return hipGetLastError();
}

}  // namespace hill
