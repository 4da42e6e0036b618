// Exact top-k token selection on gfx950 (Sec. 3.1 top-alpha; Sec. 4.2 global
// top-alpha indices) as a radix select on order-preserving 32-bit keys, split
// over 512-token chunks of each importance row so that every step runs on
// many CUs -- the GPU form of the paper's chunked evaluation whose per-chunk
// results are merged into one global threshold (Sec. 4.2, HIE).
//
//  topk_hist    first-digit (bits 31..20) histogram of every row; in hill_step
//               the importance update counts it as it writes S.
//  topk_refine  per chunk: finds the first-digit bin holding the k-th key,
//               histograms the second digit (bits 19..8) of the chunk's keys
//               inside that bin and keeps those keys in a compact candidate
//               list.
//  topk_emit    per chunk: resolves the exact threshold key from the row's
//               second-digit histogram (and, when keys still tie on 24 bits,
//               the third digit from the candidate lists), marks the chunk's
//               selected tokens -- every key above the threshold plus, among
//               keys equal to it, the lowest token indices that fit the
//               budget -- and stores them in token order with their count.
//               With attention, the workgroup then attends over the chunk's
//               selected tokens for one or more KV heads (fused gather +
//               softmax over the list, attn_device.h; the logits are the
//               scan's own when it read the 16-bit keys, so only V rows are
//               gathered) and writes one partial per query head.  The
//               streamed variant takes the first two digits from the
//               update's histograms (the second from its window above the
//               previous step's threshold) and, when those do not settle the
//               threshold, walks the update's candidate pairs instead of
//               refine's lists; it writes the bound for the next step.
//  topk_write   places each chunk's list at its ascending-order offset (the
//               counts of the chunks before it) in the output; in hill_step
//               this runs inside merge_write, with the merge of the attention
//               partials.
//
// Every histogram is a 12-bit digit whose top 6 bits are also counted, so the
// bin of the k-th key is found in registers: every wave scans the 64 coarse
// bins (one per lane), and the wave that holds the 64 fine bins of the chosen
// coarse bin finishes.  Cross-chunk results always pass through a kernel
// boundary: on this multi-XCD part an agent-scope fence per workgroup (needed
// by a last-workgroup-done merge) costs far more than a launch.  The
// selection is exactly the k largest S with ties to the lower index: keys are
// integers, so no floating-point rounding takes part.
#include <hip/hip_ext.h>

#include "attn_device.h"

namespace hill {

namespace {

constexpr int kThreads = 256;
constexpr int kPerThread = kSelChunk / kThreads;   // 2 consecutive tokens per thread
static_assert(kPerThread == 2, "load_s_pair reads float2");
static_assert(kSelChunk == 16 * 32, "16 row groups of 32 tokens");

__global__ __launch_bounds__(256) void topk_hist_kernel(const float* __restrict__ s, int64_t s_sb, int64_t s_sr,
                                                        int R, int n, int pin_lo, int pin_hi,
                                                        uint32_t* __restrict__ hist)
{
    __shared__ uint32_t lds_hist[kHistRow];
    __shared__ uint32_t list[kHistRow];
    __shared__ uint32_t nlist;
    const int row = blockIdx.y;
    const int b = row / R, r = row % R;
    for (int i = threadIdx.x; i < kHistRow; i += 256) lds_hist[i] = 0u;
    if (threadIdx.x == 0) nlist = 0u;
    __syncthreads();
    const float* srow = s + (int64_t)b * s_sb + (int64_t)r * s_sr;
    constexpr int kPer = kHistChunk / 256;
#pragma unroll
    for (int i = 0; i < kPer; ++i) {
        const int j = blockIdx.x * kHistChunk + i * 256 + threadIdx.x;
        if (j < n) {
            const uint32_t kk = select_key(srow[j], j, pin_lo, pin_hi);
            hist_add(lds_hist, list, &nlist, kk >> (32 - kHistBits));
            hist_add(lds_hist, list, &nlist, kHistBins + (kk >> 26));
        }
    }
    __syncthreads();
    hist_flush(lds_hist, list, nlist, hist + (int64_t)row * kHistRow);
}

__device__ __forceinline__ const float* row_ptr(const RefineArgs& a, int row)
{
    const int b = row / a.R, r = row % a.R;
    return a.s + (int64_t)b * a.s_sb + (int64_t)r * a.s_sr;
}

// S of this thread's 2 consecutive tokens of chunk c: one unconditional
// 8-byte load (row bases 16-byte aligned, row strides a multiple of 4 floats
// and at least n, so the pair at an even index below n lies inside the row;
// a pair past the end reads the row's last pair, and keys_of marks it invalid).
// The keys are formed by keys_of() once every other load of the kernel's
// opening is in flight: a branch around the load would make the compiler
// wait for it before issuing anything else.
__device__ __forceinline__ float2 load_s_pair(const float* srow, int c, int n)
{
    const int j = c * kSelChunk + threadIdx.x * kPerThread;
    const int jl = j < n ? j : ((n - 1) & ~1);
    return *reinterpret_cast<const float2*>(srow + jl);
}

// Selection keys of the pair loaded by load_s_pair; tokens outside [lo, hi)
// are pinned, tokens at or past n are not valid (ok false, key 0).
__device__ __forceinline__ void keys_of(float2 x, int c, int n, int lo, int hi, uint32_t (&key)[kPerThread],
                                        bool (&ok)[kPerThread])
{
    const int j = c * kSelChunk + threadIdx.x * kPerThread;
    ok[0] = j < n;
    ok[1] = j + 1 < n;
    key[0] = ok[0] ? select_key(x.x, j, lo, hi) : 0u;
    key[1] = ok[1] ? select_key(x.y, j + 1, lo, hi) : 0u;
}

// A histogram row of one 12-bit digit, loaded so that thread t holds fine
// bins i*256 + t (i < 16) and every lane holds coarse bin `lane` (the bin's
// top 6 bits).  Fine bins 64*C .. 64*C+63 of coarse bin C then sit in
// register C/4 of wave C%4, one per lane.
struct DigitHist {
    uint32_t fine[kHistBins / kThreads];
    uint32_t coarse;
};

__device__ __forceinline__ void load_digit_hist(const uint32_t* h, DigitHist& d)
{
#pragma unroll
    for (int i = 0; i < kHistBins / kThreads; ++i) d.fine[i] = h[i * kThreads + threadIdx.x];
    d.coarse = h[kHistBins + (threadIdx.x & 63)];
}

// A 12-bit digit histogram row held in registers from the top: thread t holds
// bins [4096 - 16(t+1), 4096 - 16t) (four 16-byte loads), so the bin of the
// need-th largest key is found with one block scan of the threads' totals and
// a walk of one thread's 16 registers -- no coarse bins needed.
struct DigitBins {
    uint32_t v[kHistBins / kThreads];   // v[i] = bin base + i, base = 4096 - 16(t+1)
};

__device__ __forceinline__ void load_digit_bins(const uint32_t* h, DigitBins& d)
{
    static_assert(kHistBins / kThreads == 16, "16 bins per thread");
    const uint4* p = reinterpret_cast<const uint4*>(h + kHistBins - 16 * ((int)threadIdx.x + 1));
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        const uint4 x = p[q];
        d.v[4 * q] = x.x;
        d.v[4 * q + 1] = x.y;
        d.v[4 * q + 2] = x.z;
        d.v[4 * q + 3] = x.w;
    }
}

// res[0] = the bin holding the need-th largest key (1 <= need <= keys in the
// row), res[1] = keys still needed from it, res[2] = keys in it (all 0 if the
// row holds fewer than need keys).  Every thread calls it; the caller reads
// res after a barrier, and `scratch` (4 words) is not rewritten before it.
__device__ __forceinline__ void find_digit_bins(const DigitBins& d, uint32_t need, uint32_t* scratch, uint32_t* res)
{
    if (threadIdx.x == 0) {   // defined result even if the counts were inconsistent
        res[0] = 0u;
        res[1] = 0u;
        res[2] = 0u;
    }
    uint32_t local = 0u;
#pragma unroll
    for (int i = 0; i < kHistBins / kThreads; ++i) local += d.v[i];
    uint32_t total;
    const uint32_t before = block_excl_scan_1b(local, scratch, &total);   // keys in the bins above this thread's
    if (before < need && before + local >= need) {
        const uint32_t base = (uint32_t)(kHistBins - 16 * ((int)threadIdx.x + 1));
        uint32_t c = before, bin = base, left = 0u, in = 0u;
        bool found = false;
#pragma unroll
        for (int i = kHistBins / kThreads - 1; i >= 0; --i) {   // from the top bin of the range
            const bool hit = !found && c + d.v[i] >= need;
            bin = hit ? base + (uint32_t)i : bin;
            left = hit ? need - c : left;
            in = hit ? d.v[i] : in;
            found = found || hit;
            c += d.v[i];
        }
        res[0] = bin;
        res[1] = left;
        res[2] = in;
    }
}

// Streamed selection: this thread's share of the class counts of the row's
// update blocks, and the bound they were listed against.  The first slot
// (block t, clamped) is one pair of unconditional 16-byte loads issued with the
// kernel's other opening loads; blocks t + kThreads, ... (rows longer than
// kThreads update blocks) are added by add_class_counts after those.
__device__ __forceinline__ uint32_t load_class_counts(const RefineArgs& r, int row, uint32_t (&c)[kPairClasses])
{
    static_assert(kPairClasses == 5 && kSlotWords == 8 && kSlotBound == 5, "counts 0-3, then count 4 and the bound");
    const int nup = (r.n + kUpdChunk - 1) / kUpdChunk;
    const uint4* slot = reinterpret_cast<const uint4*>(r.scount + ((int64_t)row * nup + min((int)threadIdx.x, nup - 1)) *
                                                                       kSlotWords);
    const uint4 lo = slot[0], hi = slot[1];
    const bool ok = (int)threadIdx.x < nup;
    c[0] = ok ? lo.x : 0u;
    c[1] = ok ? lo.y : 0u;
    c[2] = ok ? lo.z : 0u;
    c[3] = ok ? lo.w : 0u;
    c[4] = ok ? hi.x : 0u;
    return hi.y;   // every block of the row wrote the same bound
}

__device__ __forceinline__ void add_class_counts(const RefineArgs& r, int row, uint32_t (&c)[kPairClasses])
{
    const int nup = (r.n + kUpdChunk - 1) / kUpdChunk;
    const uint32_t* base = r.scount + (int64_t)row * nup * kSlotWords;
    for (int u = threadIdx.x + kThreads; u < nup; u += kThreads) {
        const uint4 v = *reinterpret_cast<const uint4*>(base + (int64_t)u * kSlotWords);
        c[0] += v.x;
        c[1] += v.y;
        c[2] += v.z;
        c[3] += v.w;
        c[4] += base[(int64_t)u * kSlotWords + 4];
    }
}

// Block-wide sums of the class counts (every thread gets them); one barrier.
// packed (block-uniform): every thread holds one block's counts (at most
// kUpdChunk each) and the row at most kThreads blocks, so every sum stays
// below 2^16 and two counts share a word.
__device__ __forceinline__ void reduce_class_counts(uint32_t (&c)[kPairClasses], uint32_t (*red)[kThreads / 64],
                                                    bool packed)
{
    static_assert(kPairClasses == 5 && kThreads * kUpdChunk < 65536, "three packed sums");
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    if (packed) {
        const uint32_t v0 = wave_sum_u32(c[0] | (c[1] << 16));
        const uint32_t v1 = wave_sum_u32(c[2] | (c[3] << 16));
        const uint32_t v2 = wave_sum_u32(c[4]);
        if (lane == 0) {
            red[0][w] = v0;
            red[1][w] = v1;
            red[2][w] = v2;
        }
        __syncthreads();
        const uint32_t t0 = (red[0][0] + red[0][1]) + (red[0][2] + red[0][3]);
        const uint32_t t1 = (red[1][0] + red[1][1]) + (red[1][2] + red[1][3]);
        c[0] = t0 & 0xffffu;
        c[1] = t0 >> 16;
        c[2] = t1 & 0xffffu;
        c[3] = t1 >> 16;
        c[4] = (red[2][0] + red[2][1]) + (red[2][2] + red[2][3]);
        return;
    }
#pragma unroll
    for (int k = 0; k < kPairClasses; ++k) {
        const uint32_t v = wave_sum_u32(c[k]);
        if (lane == 0) red[k][w] = v;
    }
    __syncthreads();
#pragma unroll
    for (int k = 0; k < kPairClasses; ++k) c[k] = (red[k][0] + red[k][1]) + (red[k][2] + red[k][3]);
}

// The bin holding the need-th largest key of the row (1 <= need <= keys in
// the row): res[0] = bin, res[1] = keys still needed from it (need minus the
// keys in higher bins), res[2] = keys in it.  Every wave finds the coarse bin;
// the wave holding its fine bins finishes and publishes the result.  The
// caller reads res after a barrier.
__device__ __forceinline__ void find_digit(const DigitHist& d, uint32_t need, uint32_t* res)
{
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    int C;
    uint32_t above_c;
    wave_find_bin(d.coarse, need, C, above_c);
    if (w == (C & 3)) {
        uint32_t v = 0u;
#pragma unroll
        for (int i = 0; i < kHistBins / kThreads; ++i) v = i == (C >> 2) ? d.fine[i] : v;
        int L;
        uint32_t above_f;
        wave_find_bin(v, need - above_c, L, above_f);
        const uint32_t in_bin = __shfl(v, L, 64);
        if (lane == 0) {
            res[0] = (uint32_t)(64 * C + L);
            res[1] = need - above_c - above_f;
            res[2] = in_bin;
        }
    }
}

// Histogram of `nb` bins in LDS: the bin holding the need-th largest key,
// i.e. the largest d with count(bins >= d) >= need.  res[0] = d,
// res[1] = count(bins > d).  Every thread of the NT-thread block must call this.
template <int NT>
__device__ void find_bin(const uint32_t* hist, int nb, uint32_t need, uint32_t* scan_scratch, uint32_t* res)
{
    const int tid = threadIdx.x;
    if (tid == 0) {   // defined result even if the counts were inconsistent
        res[0] = 0u;
        res[1] = 0u;
    }
    const int per = nb >= NT ? nb / NT : 1;
    const int nt = nb / per;
    // thread t owns bins [nb - (t+1)*per, nb - t*per), visited from the top
    uint32_t local = 0;
    if (tid < nt)
        for (int i = 0; i < per; ++i) local += hist[nb - 1 - (tid * per + i)];
    uint32_t total;
    const uint32_t before = block_excl_scan<NT>(local, scan_scratch, &total);
    if (tid < nt && before < need && before + local >= need) {
        uint32_t c = before;
        for (int i = 0; i < per; ++i) {
            const int bin = nb - 1 - (tid * per + i);
            const uint32_t h = hist[bin];
            if (c + h >= need) {
                res[0] = (uint32_t)bin;
                res[1] = c;
                break;
            }
            c += h;
        }
    }
    __syncthreads();
}

__global__ __launch_bounds__(kThreads) void topk_refine_kernel(RefineArgs a)
{
    __shared__ uint32_t hist[kHistRow];
    __shared__ uint32_t list[2 * kSelChunk];
    __shared__ uint32_t res[3];
    __shared__ uint32_t n_cand, nlist;

    const int tid = threadIdx.x, lane = tid & 63;
    const int c = blockIdx.x, row = blockIdx.y;
    const float* srow = row_ptr(a, row);

    // the chunk's S and the row's first-digit histogram are loaded together
    const float2 sx = load_s_pair(srow, c, a.n);
    DigitHist h1;
    load_digit_hist(a.hist1 + (int64_t)row * kHistRow, h1);
    uint32_t key[kPerThread];
    bool ok[kPerThread];
    keys_of(sx, c, a.n, a.pin_lo, a.pin_hi, key, ok);
    for (int i = tid; i < kHistRow; i += kThreads) hist[i] = 0u;
    if (tid == 0) n_cand = nlist = 0u;
    // first digit: the bin of the k-th key
    find_digit(h1, (uint32_t)a.k, res);
    __syncthreads();
    const uint32_t b1 = res[0] & (kHistBins - 1);
    const uint32_t need1 = res[1];
    const uint32_t in1 = res[2];
    const bool refine = need1 < in1;
    if (c == 0 && tid == 0) a.state[row] = make_uint4(b1, need1, in1, 0u);

    // keys inside the bin are the candidates: their second digit is
    // histogrammed and they are appended (wave-compacted) to the chunk's
    // candidate list, whose order does not matter
    uint32_t* cand = a.cand_key + (int64_t)row * a.n + (int64_t)c * kSelChunk;
#pragma unroll
    for (int e = 0; e < kPerThread; ++e) {
        const bool is_c = ok[e] && (key[e] >> 20) == b1;
        if (is_c && refine) {
            hist_add(hist, list, &nlist, (key[e] >> 8) & (kHistBins - 1));
            hist_add(hist, list, &nlist, kHistBins + ((key[e] >> 14) & (kCoarseBins - 1)));
        }
        const uint64_t mask = __ballot(is_c);
        if (mask) {
            const int leader = __ffsll((unsigned long long)mask) - 1;
            uint32_t base = 0;
            if (lane == leader) base = atomicAdd(&n_cand, (uint32_t)__popcll(mask));
            base = __shfl(base, leader, 64);
            if (is_c) cand[base + __popcll(mask & ((1ull << lane) - 1ull))] = key[e];
        }
    }
    __syncthreads();
    if (refine) hist_flush(hist, list, nlist, a.hist2 + (int64_t)row * kHistRow);
    if (tid == 0) a.cand_n[(int64_t)row * a.nchunks + c] = n_cand;
}

// Calls f(key) for every candidate of chunks [c0, c1) of a row.  Groups of
// up to kThreads chunks are flattened with one block scan of their counts
// (offsets in `offs`, kThreads words of LDS) and a binary search per key, so
// all loads of a round are in flight together instead of one chunk after
// another.  Every thread of the block calls it.
template <typename F>
__device__ __forceinline__ void for_candidates(const RefineArgs& a, int row, int c0, int c1, uint32_t* offs,
                                               uint32_t* scratch, F f)
{
    constexpr int kU = 8;
    const uint32_t tid = threadIdx.x;
    const uint32_t* cn = a.cand_n + (int64_t)row * a.nchunks;
    const uint32_t* cl = a.cand_key + (int64_t)row * a.n;
    for (int g0 = c0; g0 < c1; g0 += kThreads) {
        const int ng = min(kThreads, c1 - g0);
        const uint32_t m = (int)tid < ng ? cn[g0 + tid] : 0u;
        uint32_t tot;
        const uint32_t o = block_excl_scan<kThreads>(m, scratch, &tot);
        offs[tid] = o;
        __syncthreads();
        for (uint32_t i0 = 0; i0 < tot; i0 += kThreads * kU) {
            uint32_t v[kU];
#pragma unroll
            for (int u = 0; u < kU; ++u) {
                const uint32_t i = i0 + u * kThreads + tid;
                v[u] = 0u;
                if (i < tot) {
                    int lo = 0, hi = ng - 1;   // the last chunk whose offset is <= i
                    while (lo < hi) {
                        const int mid = (lo + hi + 1) >> 1;
                        if (offs[mid] <= i) lo = mid; else hi = mid - 1;
                    }
                    v[u] = cl[(int64_t)(g0 + lo) * kSelChunk + (i - offs[lo])];
                }
            }
#pragma unroll
            for (int u = 0; u < kU; ++u)
                if (i0 + u * kThreads + tid < tot) f(v[u]);
        }
        __syncthreads();   // offs is rewritten by the next group
    }
}

// Streamed selection: calls f(key, token) for every (key, token) pair of
// class cls that the update listed for the row (fast: the class holds every
// key of the first-digit bin in question), or for every token of the row with
// its selection key (slow: the bound did not hold).  The pairs sit in
// per-update-block slots, grouped by class; groups of up to 256 slots are
// flattened with one block scan of the class counts (offsets in `offs`, the
// class's start in each slot in `starts`, 256 words of LDS each) and a binary
// search per pair, so all loads of a round are in flight together.  Every
// thread of the block calls it.
template <typename F>
__device__ __forceinline__ void for_row_pairs(const RefineArgs& r, int row, bool fast, int cls, uint32_t* offs,
                                              uint32_t* starts, uint32_t* scratch, F f)
{
    constexpr int kU = 8;
    const uint32_t tid = threadIdx.x;
    if (fast) {
        const int nup = (r.n + kUpdChunk - 1) / kUpdChunk;
        const uint32_t* cnt = r.scount + (int64_t)row * nup * kSlotWords;
        const uint2* pr = r.spairs + (int64_t)row * r.n;
        for (int g0 = 0; g0 < nup; g0 += kThreads) {
            const int ng = min(kThreads, nup - g0);
            uint32_t c = 0u, st = 0u;
            if ((int)tid < ng) {
                const uint32_t* cs = cnt + (int64_t)(g0 + tid) * kSlotWords;
                for (int k = 0; k < cls; ++k) st += cs[k];
                c = cs[cls];
            }
            uint32_t tot;
            const uint32_t o = block_excl_scan<kThreads>(c, scratch, &tot);
            offs[tid] = o;
            starts[tid] = st;
            __syncthreads();
            for (uint32_t i0 = 0; i0 < tot; i0 += kThreads * kU) {
                uint2 v[kU];
#pragma unroll
                for (int u = 0; u < kU; ++u) {
                    const uint32_t i = i0 + u * kThreads + tid;
                    v[u] = make_uint2(0u, 0u);
                    if (i < tot) {
                        int lo = 0, hi = ng - 1;   // the last slot whose offset is <= i
                        while (lo < hi) {
                            const int mid = (lo + hi + 1) >> 1;
                            if (offs[mid] <= i) lo = mid; else hi = mid - 1;
                        }
                        v[u] = pr[(int64_t)(g0 + lo) * kUpdChunk + starts[lo] + (i - offs[lo])];
                    }
                }
#pragma unroll
                for (int u = 0; u < kU; ++u)
                    if (i0 + u * kThreads + tid < tot) f(v[u].x, v[u].y);
            }
            __syncthreads();   // offs and starts are rewritten by the next group
        }
    } else {
        const float* srow = row_ptr(r, row);
        for (int j0 = 0; j0 < r.n; j0 += kThreads * kU) {
            float v[kU];
#pragma unroll
            for (int u = 0; u < kU; ++u) {
                const int j = j0 + u * kThreads + (int)tid;
                v[u] = j < r.n ? srow[j] : 0.0f;
            }
#pragma unroll
            for (int u = 0; u < kU; ++u) {
                const int j = j0 + u * kThreads + (int)tid;
                if (j < r.n) f(select_key(v[u], j, r.pin_lo, r.pin_hi), (uint32_t)j);
            }
        }
    }
}

// The scan's logits of heads h0 .. h0+GC of this thread's two tokens of
// chunk c (rows of ld floats, ld a multiple of 4; tokens past the row's end
// read the padded tail or an earlier pair and are never selected).
template <int GC>
__device__ __forceinline__ void load_chunk_logits(const AttnArgs& at, int b, int h0, int c, float2 (&lg)[GC])
{
    const int j = min(c * kSelChunk + (int)threadIdx.x * kPerThread, (int)at.ld - 2);
    const float* p = at.logits + ((int64_t)b * at.Hq + h0) * at.ld + j;
#pragma unroll
    for (int hh = 0; hh < GC; ++hh) lg[hh] = *reinterpret_cast<const float2*>(p + hh * at.ld);
}

// With LG the attention takes its logits from the scan (at.logits) instead
// of recomputing q.k from gathered K rows.  TIER: a tiered cache -- each
// selected token's K and V rows are read from the hot pool's slot that
// at.loc gives it, or from the cold pool (its row by position) when that is
// -1; the slots of the chunk's tokens are loaded with its S.
template <int DT, int GC, bool ATTN, bool STREAM = false, bool LG = false, bool TIER = false>
__global__ __launch_bounds__(kThreads) void topk_emit_kernel(RefineArgs r, AttnArgs at)
{
    static_assert(!TIER || (ATTN && !LG), "a tiered cache gathers K and V for the attention");
    __shared__ int32_t sloc[TIER ? kAttnBlock : 1];
    __shared__ uint32_t hist3[256];
    __shared__ typename std::conditional<STREAM, uint32_t[kHistBins], uint32_t[1]>::type hist2s;
    __shared__ uint32_t pair_offs[kThreads];   // also the chunk offsets of the candidate walks
    __shared__ typename std::conditional<STREAM, uint32_t[kThreads], uint32_t[1]>::type pair_starts;
    __shared__ uint32_t scan_scratch[kThreads / 64 + 1];
    __shared__ uint32_t red[kThreads / 64];
    __shared__ uint32_t res[3];
    __shared__ typename std::conditional<STREAM, uint32_t[kPairClasses][kThreads / 64], uint32_t[1][1]>::type cls_red;
    __shared__ AttnLds<ATTN ? GC : 1> sh;

    const int tid = threadIdx.x, lane = tid & 63;
    const int c = blockIdx.x;
    int row, b = 0, g = 0, ng = 1;
    if constexpr (ATTN) {
        // KV heads g .. g+ng-1 of sequence b (ng > 1 only for token rows)
        ng = at.kv_per_wg;
        const int groups = at.Hkv / ng;
        b = blockIdx.y / groups;
        g = (blockIdx.y % groups) * ng;
        row = r.R == 1 ? b : b * at.Hkv + g;
    } else {
        row = blockIdx.y;
    }
    // one workgroup per chunk stores the list (token rows: the one with KV head 0)
    const bool writer = !ATTN || r.R != 1 || g == 0;

    // independent loads first: queries, this chunk's keys, the row's state and
    // second-digit histogram
    uint4 qv[ATTN && !LG ? GC : 1];
    if constexpr (ATTN && !LG) load_queries<GC>(at, b, g, 0, qv);
    const float2 sx = load_s_pair(row_ptr(r, row), c, r.n);
    int2 lv = make_int2(-1, -1);   // TIER: the hot-pool slots of this thread's two tokens
    if constexpr (TIER) {
        const int j = c * kSelChunk + tid * kPerThread;
        lv = *reinterpret_cast<const int2*>(at.loc + (int64_t)row * at.loc_sr + (j < r.n ? j : ((r.n - 1) & ~1)));
    }
    float2 lgv[LG ? GC : 1];
    if constexpr (LG) load_chunk_logits<GC>(at, b, g * at.G, c, lgv);
    // exact threshold: (key >> shift) compared with prefix; `need` keys equal to it are taken
    uint32_t prefix, need;
    int shift;
    bool all_eq;
    bool fast = true;   // streamed: the update's pairs hold every key of the threshold's first-digit bin
    int pair_cls = kStreamBins;   // streamed: the class of the update's pairs that holds that bin
    if constexpr (STREAM) {
        // First digit of the k-th key.  With a valid bound (the one the update used) it lies in
        // the bound's bin or above: the update's class counts of the row's pairs, summed here
        // over its blocks, give the keys in each of the window's kStreamBins bins and above
        // it, and only a threshold above the window needs a first-digit histogram, counted
        // here from the above-window pairs.  If fewer than k pairs are there, S did not only
        // grow since the bound was written -- it was changed outside these calls -- and the
        // first digit is counted over the whole row, whose keys the later walks then read
        // directly (fast = false).  Without a bound the update counted the row's histogram.
        // The second digit of a threshold in the window comes from the update's histogram of
        // that bin (the bound's own bin is loaded up front), the third (and ties) from the
        // keys of the threshold's bin in the pair list.
        uint32_t cnt[kPairClasses];
        const uint32_t bnd = load_class_counts(r, row, cnt);
        // the threshold mostly stays in the bound's bin or moves one bin up: both bins' counts
        // are loaded with the opening loads
        DigitBins h2, h2n;
        load_digit_bins(r.hist2 + (int64_t)row * kHistRow, h2);
        load_digit_bins(r.hist2 + ((int64_t)at.B * r.R + row) * kHistRow, h2n);   // [w][rows][bins]
        add_class_counts(r, row, cnt);
        reduce_class_counts(cnt, cls_red, (r.n + kUpdChunk - 1) / kUpdChunk <= kThreads);
        const uint32_t d0 = bnd & (kHistBins - 1);
        const bool bound = bnd >> 31;   // block-uniform
        uint32_t b1 = 0u, need1 = 0u, in1 = 0u;
        // first digit of the k-th key among the pairs of class cls (or the whole row when !fast)
        auto first_digit_from_pairs = [&](int cls) {
            uint32_t* h1s = hist2s;
            for (int i = tid; i < kHistBins; i += kThreads) h1s[i] = 0u;
            __syncthreads();
            for_row_pairs(r, row, fast, cls, pair_offs, pair_starts, scan_scratch,
                          [h1s](uint32_t kk, uint32_t) { atomicAdd(&h1s[kk >> 20], 1u); });
            __syncthreads();
            find_bin<kThreads>(h1s, kHistBins, (uint32_t)r.k, scan_scratch, res);
            b1 = res[0] & (kHistBins - 1);
            need1 = (uint32_t)r.k - res[1];
            in1 = h1s[b1];
            __syncthreads();   // res and the counts have been read before either is reused
        };
        if (!bound) {
            DigitBins h1;
            load_digit_bins(r.hist1 + (int64_t)row * kHistRow, h1);
            find_digit_bins(h1, (uint32_t)r.k, scan_scratch, res);
            __syncthreads();
            b1 = res[0] & (kHistBins - 1);
            need1 = res[1];
            in1 = res[2];
            __syncthreads();   // res has been read
        } else {
            uint32_t total = 0u;
#pragma unroll
            for (int k = 0; k < kPairClasses; ++k) total += cnt[k];
            fast = total >= (uint32_t)r.k;   // block-uniform
            if (!fast) {
                first_digit_from_pairs(kStreamBins);
            } else if (cnt[kStreamBins] >= (uint32_t)r.k) {
                first_digit_from_pairs(kStreamBins);   // above the window
            } else {
                uint32_t above = cnt[kStreamBins];
                int wsel = 0;
#pragma unroll
                for (int wd = kStreamBins - 1; wd >= 0; --wd) {
                    if (above + cnt[wd] >= (uint32_t)r.k) {
                        wsel = wd;
                        break;
                    }
                    above += cnt[wd];
                }
                b1 = d0 + (uint32_t)wsel;
                need1 = (uint32_t)r.k - above;
                in1 = cnt[wsel];
            }
        }
        pair_cls = (fast && bound && b1 - d0 < (uint32_t)kStreamBins) ? (int)(b1 - d0) : kStreamBins;
        prefix = b1;
        need = need1;
        shift = 20;
        all_eq = need1 == in1;
        if (!all_eq) {
            uint32_t b2, need2, in2;
            const uint32_t wdx = b1 - d0;
            if (bound && fast && wdx < (uint32_t)kStreamBins) {   // block-uniform
                if (wdx == 1) {
#pragma unroll
                    for (int i = 0; i < kHistBins / kThreads; ++i) h2.v[i] = h2n.v[i];
                } else if (wdx > 1) {   // the threshold moved further: that bin's counts
                    load_digit_bins(r.hist2 + ((int64_t)wdx * at.B * r.R + row) * kHistRow, h2);
                }
                find_digit_bins(h2, need1, scan_scratch, res);
                __syncthreads();
                b2 = res[0] & (kHistBins - 1);
                need2 = res[1];
                in2 = res[2];
            } else {
                uint32_t* h2s = hist2s;
                for (int i = tid; i < kHistBins; i += kThreads) h2s[i] = 0u;
                __syncthreads();
                // the threshold's bin lies above the window (or there is no bound): class kStreamBins
                for_row_pairs(r, row, fast, kStreamBins, pair_offs, pair_starts, scan_scratch,
                              [b1, h2s](uint32_t kk, uint32_t) {
                    if ((kk >> 20) == b1) atomicAdd(&h2s[(kk >> 8) & (kHistBins - 1)], 1u);
                });
                __syncthreads();
                find_bin<kThreads>(h2s, kHistBins, need1, scan_scratch, res);
                b2 = res[0] & (kHistBins - 1);
                need2 = need1 - res[1];
                in2 = h2s[b2];
            }
            prefix = (b1 << 12) | b2;
            shift = 8;
            need = need2;
            all_eq = need2 == in2;
            if (!all_eq) {   // third digit (bits 7..0)
                // needed only by workgroups holding a key of the threshold's 24-bit bin (and by the
                // one that writes the next step's bound): elsewhere the keys above that bin are
                // exactly the selected ones
                const uint32_t p2 = prefix;
                uint32_t kx[kPerThread];
                bool okx[kPerThread];
                keys_of(sx, c, r.n, r.pin_lo, r.pin_hi, kx, okx);
                bool mine = writer && c == 0;
#pragma unroll
                for (int e = 0; e < kPerThread; ++e) mine = mine || (okx[e] && (kx[e] >> 8) == p2);
                if (__syncthreads_or(mine)) {   // block-uniform
                    uint32_t* h3 = hist3;
                    for (int i = tid; i < 256; i += kThreads) h3[i] = 0u;
                    __syncthreads();
                    for_row_pairs(r, row, fast, pair_cls, pair_offs, pair_starts, scan_scratch,
                                  [p2, h3](uint32_t kk, uint32_t) {
                        if ((kk >> 8) == p2) atomicAdd(&h3[kk & 0xffu], 1u);
                    });
                    __syncthreads();
                    find_bin<kThreads>(h3, 256, need2, scan_scratch, res);
                    const uint32_t b3 = res[0] & 0xffu;
                    prefix = (p2 << 8) | b3;
                    shift = 0;
                    need = need2 - res[1];
                    all_eq = need == h3[b3];
                } else {
                    all_eq = true;   // no key of this chunk ties with the threshold at 24 bits
                }
            }
            __syncthreads();
        }
        if (writer && c == 0 && tid == 0) {
            // bound for the next step: the threshold's first-digit bin, with the number of keys in it or
            // above (S only grows, so any budget up to that number keeps its threshold in or above the bin)
            const uint32_t at_or_above = (uint32_t)r.k - need1 + in1;
            r.state_out[2 * row] = make_uint4(prefix << shift, at_or_above, (uint32_t)r.n, 1u);
            r.state_out[2 * row + 1] = make_uint4((uint32_t)r.pin_lo, (uint32_t)(r.n - r.pin_hi), 0u, 0u);
        }
    } else {
    const uint4 s1 = r.state[row];
    DigitHist h2;
    load_digit_hist(r.hist2 + (int64_t)row * kHistRow, h2);
    const uint32_t b1 = s1.x, need1 = s1.y, in1 = s1.z;
    if (r.state_out && writer && c == 0 && tid == 0) {   // a reset step of the streamed selection: its bound
        r.state_out[2 * row] = make_uint4(b1 << 20, (uint32_t)r.k - need1 + in1, (uint32_t)r.n, 1u);
        r.state_out[2 * row + 1] = make_uint4((uint32_t)r.pin_lo, (uint32_t)(r.n - r.pin_hi), 0u, 0u);
    }
    prefix = b1;
    need = need1;
    shift = 20;
    all_eq = need1 == in1;
    if (!all_eq) {
        find_digit(h2, need1, res);
        __syncthreads();
        const uint32_t b2 = res[0] & (kHistBins - 1);
        const uint32_t need2 = res[1];
        const uint32_t in2 = res[2];
        prefix = (b1 << 12) | b2;
        shift = 8;
        need = need2;
        all_eq = need2 == in2;
        if (!all_eq) {   // third digit (bits 7..0) from the candidate lists
            // only workgroups holding a key of the threshold's 24-bit bin need it (elsewhere the
            // keys above that bin are exactly the selected ones)
            const uint32_t p2 = prefix;
            uint32_t kx[kPerThread];
            bool okx[kPerThread];
            keys_of(sx, c, r.n, r.pin_lo, r.pin_hi, kx, okx);
            bool mine = false;
#pragma unroll
            for (int e = 0; e < kPerThread; ++e) mine = mine || (okx[e] && (kx[e] >> 8) == p2);
            if (__syncthreads_or(mine)) {   // block-uniform
                for (int i = tid; i < 256; i += kThreads) hist3[i] = 0u;
                __syncthreads();
                for_candidates(r, row, 0, r.nchunks, pair_offs, scan_scratch, [p2](uint32_t kk) {
                    if ((kk >> 8) == p2) atomicAdd(&hist3[kk & 0xffu], 1u);
                });
                __syncthreads();
                find_bin<kThreads>(hist3, 256, need2, scan_scratch, res);
                const uint32_t b3 = res[0] & 0xffu;
                prefix = (p2 << 8) | b3;
                shift = 0;
                need = need2 - res[1];
                all_eq = need == hist3[b3];
                __syncthreads();
            } else {
                all_eq = true;   // no key of this chunk ties with the threshold at 24 bits
            }
        }
    }
    }

    uint32_t key[kPerThread];
    bool ok[kPerThread];
    keys_of(sx, c, r.n, r.pin_lo, r.pin_hi, key, ok);
    bool gt[kPerThread], eq[kPerThread], sel[kPerThread];
    uint32_t neq = 0;
#pragma unroll
    for (int e = 0; e < kPerThread; ++e) {
        const uint32_t kd = key[e] >> shift;
        gt[e] = ok[e] && kd > prefix;
        eq[e] = ok[e] && kd == prefix;
        neq += eq[e];
    }
    if (all_eq) {
#pragma unroll
        for (int e = 0; e < kPerThread; ++e) sel[e] = gt[e] || eq[e];
    } else {
        // the budget cuts through keys equal to the threshold: rank them by
        // token index (equal keys in the chunks before, then in this chunk)
        uint32_t before_chunks = 0;
        const uint32_t pf = prefix;
        if constexpr (STREAM) {
            const uint32_t jlim = (uint32_t)c * kSelChunk;
            for_row_pairs(r, row, fast, pair_cls, pair_offs, pair_starts, scan_scratch,
                          [&before_chunks, pf, jlim](uint32_t kk, uint32_t j) {
                before_chunks += (kk == pf && j < jlim) ? 1u : 0u;
            });
        } else {
            for_candidates(r, row, 0, c, pair_offs, scan_scratch,
                           [&before_chunks, pf](uint32_t kk) { before_chunks += kk == pf; });
        }
        before_chunks = wave_sum_u32(before_chunks);
        if (lane == 0) red[tid >> 6] = before_chunks;
        __syncthreads();
        uint32_t eq_rank = 0;
        for (int i = 0; i < kThreads / 64; ++i) eq_rank += red[i];
        uint32_t tot;
        eq_rank += block_excl_scan<kThreads>(neq, scan_scratch, &tot);
#pragma unroll
        for (int e = 0; e < kPerThread; ++e) {
            sel[e] = gt[e] || (eq[e] && eq_rank < need);
            eq_rank += eq[e];
        }
    }

    // the chunk's selected tokens in token order, and their count
    const uint32_t nsel = (uint32_t)sel[0] + (uint32_t)sel[1];
    uint32_t tot;
    const uint32_t pos = block_excl_scan_1b(nsel, scan_scratch, &tot);
    const int j0 = c * kSelChunk + tid * kPerThread;
    int32_t* list = r.sel_list + (int64_t)row * r.n + (int64_t)c * kSelChunk;
    if constexpr (ATTN) {
        // attention of the group's heads over the chunk's selected tokens
        // (one partial per head in slot c), then the list is stored
        AttnAcc<GC> acc;
        attn_begin<GC>(acc, sh);
        uint32_t p = pos;
#pragma unroll
        for (int e = 0; e < kPerThread; ++e) {
            if (sel[e]) {
                sh.tok[p] = j0 + e;
                if constexpr (TIER) sloc[p] = e == 0 ? lv.x : lv.y;
                if constexpr (LG) {
#pragma unroll
                    for (int hh = 0; hh < GC; ++hh) sh.p[p][hh] = at.s2 * (e == 0 ? lgv[hh].x : lgv[hh].y);
                }
                ++p;
            }
        }
        __syncthreads();
        // the first head chunk with the queries (or logits) loaded at the start
        if (tot) {
            if constexpr (LG) attn_block_logits<DT, GC>(at, b, g, (int)tot, acc, sh);
            else attn_block<DT, GC, TIER>(at, b, g, qv, (int)tot, acc, sh, sloc);
        }
        attn_finish<GC>(at, b, g, 0, acc, c, r.nchunks, sh);
        for (int i = 1; i < ng * (at.G / GC); ++i) {   // further head chunks and KV heads
            const int gg = g + i / (at.G / GC), hc = (i % (at.G / GC)) * GC;
            AttnAcc<GC> acc2;
            attn_begin<GC>(acc2, sh);
            if constexpr (LG) {   // the list's logits of these heads
                const float* lp = at.logits + ((int64_t)b * at.Hq + gg * at.G + hc) * at.ld;
                for (uint32_t t = tid; t < tot; t += kThreads) {
                    const int j = sh.tok[t];
#pragma unroll
                    for (int hh = 0; hh < GC; ++hh) sh.p[t][hh] = at.s2 * lp[hh * at.ld + j];
                }
                __syncthreads();
                if (tot) attn_block_logits<DT, GC>(at, b, gg, (int)tot, acc2, sh);
            } else {
                load_queries<GC>(at, b, gg, hc, qv);
                if (tot) attn_block<DT, GC, TIER>(at, b, gg, qv, (int)tot, acc2, sh, sloc);
            }
            attn_finish<GC>(at, b, gg, hc, acc2, c, r.nchunks, sh);
        }
        if (writer) {
            for (uint32_t i = tid; i < tot; i += kThreads) list[i] = sh.tok[i];
            if (tid == 0) r.sel_n[(int64_t)row * r.nchunks + c] = tot;
        }
    } else {
        uint32_t p = pos;
#pragma unroll
        for (int e = 0; e < kPerThread; ++e)
            if (sel[e]) list[p++] = j0 + e;
        if (tid == 0) r.sel_n[(int64_t)row * r.nchunks + c] = tot;
    }
}

// Copies the list of chunk c of a row to the output at its ascending-order
// offset (the selected counts of the chunks before it).  Every load is issued
// before the first wait: the counts before c, this chunk's count and its list
// entries (two per thread, at most kSelChunk; positions past the chunk's
// tokens are clamped into it and never stored).
__device__ __forceinline__ void write_chunk(const RefineArgs& r, int row, int c, int32_t* idx, float* val,
                                            uint32_t* red)
{
    const int tid = threadIdx.x, lane = tid & 63;
    const uint32_t* sn = r.sel_n + (int64_t)row * r.nchunks;
    const int32_t* list = r.sel_list + (int64_t)row * r.n + (int64_t)c * kSelChunk;
    const int last = min(kSelChunk, r.n - c * kSelChunk) - 1;   // the chunk's last slot
    const int32_t e0 = list[min(tid, last)];
    const int32_t e1 = list[min(tid + kThreads, last)];
    const uint32_t m = sn[c];
    uint32_t before = 0;
    for (int cc = tid; cc < c; cc += kThreads) before += sn[cc];
    before = wave_sum_u32(before);
    if (lane == 0) red[tid >> 6] = before;
    __syncthreads();
    uint32_t base = 0;
    for (int i = 0; i < kThreads / 64; ++i) base += red[i];
    const float* srow = row_ptr(r, row);
    static_assert(kSelChunk == 2 * kThreads, "two list entries per thread");
#pragma unroll
    for (int e = 0; e < 2; ++e) {
        const uint32_t i = (uint32_t)(tid + e * kThreads);
        const uint32_t p = base + i;
        if (i < m && p < (uint32_t)r.k) {
            const int32_t j = e == 0 ? e0 : e1;
            idx[(int64_t)row * r.k + p] = j;
            if (val) val[(int64_t)row * r.k + p] = srow[j];
        }
    }
}

__global__ __launch_bounds__(kThreads) void topk_write_kernel(RefineArgs r, int32_t* idx, float* val)
{
    __shared__ uint32_t red[kThreads / 64];
    write_chunk(r, blockIdx.y, blockIdx.x, idx, val, red);
}

// hill_step's last kernel: workgroups [0, B*Hq*kMergeSlices) merge the chunk
// partials of one slice of kHeadDim / kMergeSlices output dimensions of one
// query head each (a slice's loads are one 128-byte line per slot; more,
// shorter workgroups finish sooner than one per head); the rest copy one
// chunk list each into the index output.
constexpr int kMergeSlices = 4;

__global__ __launch_bounds__(kThreads) void merge_write_kernel(RefineArgs r, AttnArgs at, int32_t* idx)
{
    constexpr int DS = kHeadDim / kMergeSlices;
    __shared__ float red[kThreads / 64 + kThreads / DS];
    __shared__ float osum[kThreads];
    __shared__ uint32_t ured[kThreads / 64];
    const int nmerge = at.B * at.Hq * kMergeSlices;
    if ((int)blockIdx.x < nmerge) {
        const int bh = blockIdx.x / kMergeSlices, sl = blockIdx.x % kMergeSlices;
        merge_head<kThreads, DS>(at, bh / at.Hq, bh % at.Hq, sl * DS, r.nchunks, red, osum);
    } else {
        const int t = blockIdx.x - nmerge;
        write_chunk(r, t / r.nchunks, t % r.nchunks, idx, nullptr, ured);
    }
}

template <int DT, int GC, bool STREAM, bool LG, bool TIER>
void emit_attn_launch(const RefineArgs& r, const AttnArgs& at, hipStream_t st, Stamp ts)
{
    dim3 grid(r.nchunks, at.B * (at.Hkv / at.kv_per_wg));
    hipExtLaunchKernelGGL((topk_emit_kernel<DT, GC, true, STREAM, LG, TIER>), grid, dim3(kThreads), 0, st, ts.start,
                          ts.stop, 0, r, at);
}

template <int DT, bool STREAM, bool LG, bool TIER = false>
void emit_attn_gc(const RefineArgs& r, const AttnArgs& at, hipStream_t st, Stamp ts)
{
    const int gc = (at.G % 8 == 0) ? 8 : (at.G % 4 == 0) ? 4 : (at.G % 2 == 0) ? 2 : 1;
    switch (gc) {
    case 8: emit_attn_launch<DT, 8, STREAM, LG, TIER>(r, at, st, ts); break;
    case 4: emit_attn_launch<DT, 4, STREAM, LG, TIER>(r, at, st, ts); break;
    case 2: emit_attn_launch<DT, 2, STREAM, LG, TIER>(r, at, st, ts); break;
    default: emit_attn_launch<DT, 1, STREAM, LG, TIER>(r, at, st, ts); break;
    }
}

template <bool STREAM>
hipError_t emit_attn_any(const RefineArgs& r, const AttnArgs& at, int dtype, hipStream_t st, Stamp ts)
{
    if (dtype == 1) {
        if (at.loc) emit_attn_gc<1, STREAM, false, true>(r, at, st, ts);
        else if (at.logits) emit_attn_gc<1, STREAM, true>(r, at, st, ts);
        else emit_attn_gc<1, STREAM, false>(r, at, st, ts);
    } else {
        if (at.loc) emit_attn_gc<0, STREAM, false, true>(r, at, st, ts);
        else if (at.logits) emit_attn_gc<0, STREAM, true>(r, at, st, ts);
        else emit_attn_gc<0, STREAM, false>(r, at, st, ts);
    }
    return hipGetLastError();
}

}  // namespace

hipError_t launch_topk_hist(const float* s, int64_t s_sb, int64_t s_sr, int B, int R, int n, int pin_lo, int pin_hi,
                            uint32_t* hist, hipStream_t st, Stamp ts)
{
    dim3 grid((n + kHistChunk - 1) / kHistChunk, B * R);
    hipExtLaunchKernelGGL(topk_hist_kernel, grid, dim3(256), 0, st, ts.start, ts.stop, 0, s, s_sb, s_sr, R, n, pin_lo,
                          pin_hi, hist);
    return hipGetLastError();
}

hipError_t launch_topk_refine(const RefineArgs& a, int rows, hipStream_t st, Stamp ts)
{
    dim3 grid(a.nchunks, rows);
    hipExtLaunchKernelGGL(topk_refine_kernel, grid, dim3(kThreads), 0, st, ts.start, ts.stop, 0, a);
    return hipGetLastError();
}

hipError_t launch_topk_emit_indices(const RefineArgs& r, int rows, int32_t* idx, float* val, hipStream_t st, Stamp ts)
{
    dim3 grid(r.nchunks, rows);
    hipExtLaunchKernelGGL((topk_emit_kernel<0, 1, false>), grid, dim3(kThreads), 0, st, ts.start, nullptr, 0, r,
                          AttnArgs{});
    hipExtLaunchKernelGGL(topk_write_kernel, grid, dim3(kThreads), 0, st, nullptr, ts.stop, 0, r, idx, val);
    return hipGetLastError();
}

hipError_t launch_topk_emit_lists(const RefineArgs& r, int rows, hipStream_t st)
{
    hipLaunchKernelGGL((topk_emit_kernel<0, 1, false>), dim3(r.nchunks, rows), dim3(kThreads), 0, st, r, AttnArgs{});
    return hipGetLastError();
}

hipError_t launch_topk_emit_attn_stream(const RefineArgs& r, const AttnArgs& at, int dtype, hipStream_t st, Stamp ts)
{
    return emit_attn_any<true>(r, at, dtype, st, ts);
}

hipError_t launch_topk_emit_attn(const RefineArgs& r, const AttnArgs& at, int dtype, hipStream_t st, Stamp ts)
{
    return emit_attn_any<false>(r, at, dtype, st, ts);
}

hipError_t launch_merge_write(const RefineArgs& r, const AttnArgs& at, int32_t* idx, int rows, hipStream_t st,
                              Stamp ts)
{
    const int blocks = at.B * at.Hq * kMergeSlices + rows * r.nchunks;
    hipExtLaunchKernelGGL(merge_write_kernel, dim3(blocks), dim3(kThreads), 0, st, ts.start, ts.stop, 0, r, at, idx);
    return hipGetLastError();
}

}  // namespace hill
