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
            z = z * exp2f(m - mn) + v[u].y * exp2f(v[u].x - mn);
            m = mn;
        }
    }
    const float mw = wave_max(m);
    z = m > -INFINITY ? z * exp2f(m - mw) : 0.0f;
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
        for (int i = 0; i < 4; ++i) Z += red_m[i] > -INFINITY ? red_z[i] * exp2f(red_m[i] - M) : 0.0f;
        stats[bh] = make_float2(M, 1.0f / Z);
    }
}

// First-digit histogram of the importance keys a workgroup writes (bits
// 31..20, and the coarse bins of bits 31..26), merged sparsely.
struct KeyHist {
    uint32_t bins[kHistRow];
    uint32_t list[2 * kUpdChunk];
    uint32_t nlist;
};

__device__ __forceinline__ void key_hist_clear(KeyHist& h)
{
    for (int i = threadIdx.x; i < kHistRow; i += 256) h.bins[i] = 0u;
    if (threadIdx.x == 0) h.nlist = 0u;
}

__device__ __forceinline__ void count_key(KeyHist& h, uint32_t key)
{
    hist_add(h.bins, h.list, &h.nlist, key >> (32 - kHistBits));
    hist_add(h.bins, h.list, &h.nlist, kHistBins + (key >> 26));
}

constexpr int kHeadBatch = 8;   // float4 logits loads in flight per thread

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
// there is no bound), class kStreamBins -- with the counts of the classes, so
// that a walk for one first-digit bin reads one class only.  Keys in the
// window also count their second digit (the threshold seldom moves further
// in one step).
static_assert(kStreamBins * kCoarseBins == 256, "one window coarse bin per update thread");

__device__ __forceinline__ void stream_candidates(const UpdateArgs& a, int row, int j, uint32_t key, uint32_t bnd,
                                                  uint32_t (*wcnt)[4], uint32_t* coarse)
{
    const uint32_t d0 = bnd & (kHistBins - 1);
    const uint32_t dig = key >> (32 - kHistBits);
    const bool cand = j < a.n && dig >= d0;
    const uint32_t wdx = dig - d0;   // window bin of the key (valid when cand)
    const bool win = cand && (bnd >> 31) && wdx < (uint32_t)kStreamBins;
    const int cls = win ? (int)wdx : kStreamBins;
    const int64_t rows = (int64_t)a.B * a.R;
    if (win) {   // fine bins spread out: straight to memory; the few coarse bins are summed in LDS first
        atomicAdd(&a.hist2[((int64_t)wdx * rows + row) * kHistRow + ((key >> 8) & (kHistBins - 1))], 1u);
        atomicAdd(&coarse[wdx * kCoarseBins + ((key >> 14) & (kCoarseBins - 1))], 1u);
    }
    // rank within the class: one ballot per class, wave counts through LDS
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const uint64_t below = (1ull << lane) - 1ull;
    uint32_t rank = 0;
#pragma unroll
    for (int k = 0; k < kPairClasses; ++k) {
        const uint64_t m = __ballot(cand && cls == k);
        if (cand && cls == k) rank = (uint32_t)__popcll(m & below);
        if (lane == 0) wcnt[k][w] = (uint32_t)__popcll(m);
    }
    __syncthreads();   // also completes `coarse`
    if (bnd >> 31) {
        const int i = threadIdx.x;   // kStreamBins * kCoarseBins == 256 bins, one per thread
        const uint32_t c = coarse[i];
        if (c) atomicAdd(&a.hist2[((int64_t)(i / kCoarseBins) * rows + row) * kHistRow + kHistBins + i % kCoarseBins], c);
    }
    if (cand) {
        uint32_t pos = rank;
        for (int k = 0; k < cls; ++k) pos += (wcnt[k][0] + wcnt[k][1]) + (wcnt[k][2] + wcnt[k][3]);
        for (int v = 0; v < w; ++v) pos += wcnt[cls][v];
        a.spairs[(int64_t)row * a.n + (int64_t)blockIdx.x * kUpdChunk + pos] = make_uint2(key, (uint32_t)j);
    }
    const int nup = (a.n + kUpdChunk - 1) / kUpdChunk;
    if (threadIdx.x < kPairClasses) {
        const int k = threadIdx.x;
        a.scount[((int64_t)row * nup + blockIdx.x) * kSlotWords + k] = (wcnt[k][0] + wcnt[k][1]) + (wcnt[k][2] + wcnt[k][3]);
    }
    if (threadIdx.x == 0 && blockIdx.x == 0) a.d0[row] = bnd;
}

// (max, 1/sum) of heads h0 .. h0+nh of sequence b into ms[]: copied from the
// stats kernel's output, or reduced here from the unit partials.  Thread t
// works for head t / tph (tph = 256 / nh threads per head) and folds the
// partial pairs t % tph, + tph, ... (at most kStatLoads partials); the tph
// results of a
// head are then folded across lanes (DPP within a wave when tph is a power of
// two up to 64, else in order through LDS).  The partial loads
// are issued by load_head_parts() before the logits; every thread calls
// finish_head_stats(), which ends with a barrier.
struct HeadParts {
    float2 v[kStatLoads];
};

__device__ __forceinline__ void load_head_parts(const UpdateArgs& a, int b, int h0, int nh, HeadParts& hp)
{
    const int tph = nh <= 256 ? 256 / nh : 1;
    const int t = threadIdx.x, hh = t / tph, sub = t % tph;
    const bool active = a.stats == nullptr && hh < nh;
    // npart is even and the rows 16-byte aligned: pairs of partials per load
    const float4* p = reinterpret_cast<const float4*>(a.part + ((int64_t)b * a.Hq + h0 + (active ? hh : 0)) * a.npart);
    const int npair = a.npart / 2;
#pragma unroll
    for (int i = 0; i < kStatLoads / 2; ++i) {
        // consecutive lanes read consecutive pairs; unconditional (clamped)
        // loads, invalid ones replaced afterwards
        const int idx = sub + i * tph;
        const float4 v = p[min(idx, npair - 1)];
        const bool ok = active && idx < npair;
        hp.v[2 * i] = ok ? make_float2(v.x, v.y) : make_float2(-INFINITY, 0.0f);
        hp.v[2 * i + 1] = ok ? make_float2(v.z, v.w) : make_float2(-INFINITY, 0.0f);
    }
}

// (m, z) of two disjoint sets of exp2 terms merged (z relative to m).
__device__ __forceinline__ void merge_mz(float& m, float& z, float mo, float zo)
{
    const float M = fmaxf(m, mo);
    const float a = m == -INFINITY ? 0.0f : z * exp2f(m - M);
    const float c = mo == -INFINITY ? 0.0f : zo * exp2f(mo - M);
    m = M;
    z = a + c;
}

template <int CTRL>
__device__ __forceinline__ void merge_mz_dpp(float& m, float& z)
{
    const float mo = dpp<CTRL>(m), zo = dpp<CTRL>(z);
    merge_mz(m, z, mo, zo);
}

__device__ __forceinline__ void finish_head_stats(const UpdateArgs& a, int b, int h0, int nh, const HeadParts& hp,
                                                  float2* red, float2* ms)
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
    float z = 0.0f;
#pragma unroll
    for (int i = 0; i < kStatLoads; ++i) z += hp.v[i].x == -INFINITY ? 0.0f : hp.v[i].y * exp2f(hp.v[i].x - m);
    const int tph = 256 / nh;
    if ((tph & (tph - 1)) == 0 && tph >= 2 && tph <= 64) {
        // every lane is active here; groups of tph lanes are aligned
        merge_mz_dpp<0xB1>(m, z);                      // lane ^ 1
        if (tph >= 4) merge_mz_dpp<0x4E>(m, z);        // lane ^ 2
        if (tph >= 8) merge_mz_dpp<0x141>(m, z);       // mirror within 8
        if (tph >= 16) merge_mz_dpp<0x140>(m, z);      // mirror within 16
        if (tph >= 32) merge_mz(m, z, __shfl_xor(m, 16, 64), __shfl_xor(z, 16, 64));
        if (tph >= 64) merge_mz(m, z, __shfl_xor(m, 32, 64), __shfl_xor(z, 32, 64));
        if (t % tph == 0 && t / tph < nh) ms[t / tph] = make_float2(m, 1.0f / z);
    } else {
        red[t] = make_float2(m, z);
        __syncthreads();
        if (t < nh) {
            float M = -INFINITY, Z = 0.0f;
            for (int i = 0; i < tph; ++i) merge_mz(M, Z, red[t * tph + i].x, red[t * tph + i].y);
            ms[t] = make_float2(M, 1.0f / Z);
        }
    }
    __syncthreads();
}

// S[b,r,j] += sum_{h in heads(r)} exp2(s2*l - max_h) / sum_h   (softmax weights).
// kUpdChunk = 256 tokens per workgroup: lane l of wave w loads tokens
// [4l, 4l+4) of heads w, w+4, ... as float4; the four wave partials are added
// in wave order, then each thread finishes one token and counts its first
// selection digit in an LDS histogram.  The head statistics come from the
// stats kernel or, for short rows, from the unit partials reduced here.
__global__ __launch_bounds__(256) void update_attn_kernel(UpdateArgs a)
{
    __shared__ float4 wsum[4][64];
    __shared__ KeyHist kh;
    __shared__ float2 red[256];
    __shared__ float2 ms[256];
    __shared__ uint32_t sc_wcnt[kPairClasses][4];
    const int row = blockIdx.y;          // b * R + r
    const int b = row / a.R, r = row % a.R;
    const int h0 = a.R == 1 ? 0 : r * a.G;
    const int nh = a.R == 1 ? a.Hq : a.G;
    const int tid = threadIdx.x, lane = tid & 63;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
    const bool do_hist = a.hist != nullptr;
    // Every load of the opening is issued before anything waits for one: the
    // softmax partials, this thread's old S, the first batch of logits and the
    // streamed selection's state (whose test runs only after the statistics).
    HeadParts hp;
    load_head_parts(a, b, h0, nh, hp);
    const int j4 = blockIdx.x * kUpdChunk + 4 * lane;     // first of this lane's 4 tokens
    const int jc = min(j4, (int)(a.ld - 4));              // rows are padded to ld (multiple of 4)
    const float* lg = a.logits + ((int64_t)b * a.Hq + h0) * a.ld + jc;
    const int j = blockIdx.x * kUpdChunk + tid;
    float* srow = a.s + (int64_t)b * a.s_sb + (int64_t)r * a.s_sr;
    const float s_ld = srow[min(j, a.n - 1)];             // unconditional: no branch around the load
    float4 x[kHeadBatch];
#pragma unroll
    for (int i = 0; i < kHeadBatch; ++i) {
        const int h = w + 4 * i;
        x[i] = h < nh ? *reinterpret_cast<const float4*>(lg + (int64_t)h * a.ld) : make_float4(0.f, 0.f, 0.f, 0.f);
    }
    uint4 p0 = make_uint4(0u, 0u, 0u, 0u), p1 = p0;
    if (a.prev) {
        p0 = a.prev[2 * row];
        p1 = a.prev[2 * row + 1];
    }
    __builtin_amdgcn_sched_barrier(0);
    if (do_hist) key_hist_clear(kh);
    finish_head_stats(a, b, h0, nh, hp, red, ms);
    const float s_old = j < a.n ? s_ld : 0.0f;
    const uint32_t bnd = a.prev ? stream_bound(a, p0, p1) : 0u;
    const uint32_t hist_lo = (bnd >> 31) ? (bnd & (kHistBins - 1)) : 0u;
    float4 acc = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
    for (int hb = w;;) {
#pragma unroll
        for (int i = 0; i < kHeadBatch; ++i) {
            const int h = hb + 4 * i;
            if (h < nh) {
                const float2 st = ms[h];
                acc.x += exp2f(a.s2 * x[i].x - st.x) * st.y;
                acc.y += exp2f(a.s2 * x[i].y - st.x) * st.y;
                acc.z += exp2f(a.s2 * x[i].z - st.x) * st.y;
                acc.w += exp2f(a.s2 * x[i].w - st.x) * st.y;
            }
        }
        hb += 4 * kHeadBatch;
        if (hb >= nh) break;
#pragma unroll
        for (int i = 0; i < kHeadBatch; ++i) {
            const int h = hb + 4 * i;
            x[i] = h < nh ? *reinterpret_cast<const float4*>(lg + (int64_t)h * a.ld) : make_float4(0.f, 0.f, 0.f, 0.f);
        }
    }
    // streamed selection: the window's coarse bins reuse red[] (its last reader,
    // finish_head_stats, ended with a barrier); the barrier below orders the clear
    uint32_t* sc_coarse = reinterpret_cast<uint32_t*>(red);
    static_assert(sizeof(red) >= kStreamBins * kCoarseBins * sizeof(uint32_t), "coarse window fits in red[]");
    if (a.prev) sc_coarse[tid] = 0u;
    wsum[w][lane] = acc;
    __syncthreads();
    const float* ws = reinterpret_cast<const float*>(&wsum[0][0]);
    uint32_t key = 0u;
    if (j < a.n) {
        const float tot = ((ws[tid] + ws[256 + tid]) + ws[512 + tid]) + ws[768 + tid];
        const float s_new = s_old + tot;
        srow[j] = s_new;
        key = select_key(s_new, j, a.pin_lo, a.pin_hi);
        // with a streamed bound the k-th key lies in the bound's first-digit bin
        // or above, so only those bins are counted (most keys lie below it)
        if (do_hist && (key >> (32 - kHistBits)) >= hist_lo) count_key(kh, key);
    }
    if (do_hist) {
        __syncthreads();
        hist_flush(kh.bins, kh.list, kh.nlist, a.hist + (int64_t)row * kHistRow);
    }
    if (a.prev) stream_candidates(a, row, j, key, bnd, sc_wcnt, sc_coarse);   // block-uniform
}

// Token rows, RAW mode, Hkv > 1: S[b,0,j] += sum_g groupsum[b,g,j] (same layout).
__global__ __launch_bounds__(256) void update_raw_groups_kernel(UpdateArgs a)
{
    __shared__ float4 wsum[4][64];
    __shared__ KeyHist kh;
    const int b = blockIdx.y;
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const bool do_hist = a.hist != nullptr;
    if (do_hist) key_hist_clear(kh);
    const int j4 = blockIdx.x * kUpdChunk + 4 * lane;
    const int jc = min(j4, (int)(a.ld - 4));
    const float* gs = a.logits + (int64_t)b * a.Hkv * a.ld + jc;
    const int j = blockIdx.x * kUpdChunk + tid;
    float* srow = a.s + (int64_t)b * a.s_sb;
    const float s_old = j < a.n ? srow[j] : 0.0f;
    float4 acc = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
    for (int gb = w; gb < a.Hkv; gb += 4 * kHeadBatch) {
        float4 x[kHeadBatch];
#pragma unroll
        for (int i = 0; i < kHeadBatch; ++i) {
            const int g = gb + 4 * i;
            x[i] = g < a.Hkv ? *reinterpret_cast<const float4*>(gs + (int64_t)g * a.ld) : make_float4(0.f, 0.f, 0.f, 0.f);
        }
#pragma unroll
        for (int i = 0; i < kHeadBatch; ++i) {
            acc.x += x[i].x;
            acc.y += x[i].y;
            acc.z += x[i].z;
            acc.w += x[i].w;
        }
    }
    wsum[w][lane] = acc;
    __syncthreads();
    const float* ws = reinterpret_cast<const float*>(&wsum[0][0]);
    if (j < a.n) {
        const float tot = ((ws[tid] + ws[256 + tid]) + ws[512 + tid]) + ws[768 + tid];
        const float s_new = s_old + tot;
        srow[j] = s_new;
        if (do_hist) count_key(kh, select_key(s_new, j, a.pin_lo, a.pin_hi));
    }
    if (do_hist) {
        __syncthreads();
        hist_flush(kh.bins, kh.list, kh.nlist, a.hist + (int64_t)b * kHistRow);
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
    dim3 grid((a.n + kUpdChunk - 1) / kUpdChunk, a.B * a.R);
    hipExtLaunchKernelGGL(update_attn_kernel, grid, dim3(256), 0, st, ts.start, ts.stop, 0, a);
    return hipGetLastError();
}

hipError_t launch_update_raw_groups(const UpdateArgs& a, hipStream_t st, Stamp ts)
{
    dim3 grid((a.n + kUpdChunk - 1) / kUpdChunk, a.B);
    hipExtLaunchKernelGGL(update_raw_groups_kernel, grid, dim3(256), 0, st, ts.start, ts.stop, 0, a);
    return hipGetLastError();
}

}  // namespace hill
