// Top-k token selection on gfx950 (Sec. 3.1 top-alpha; Sec. 4.2 global
// top-alpha indices) as an exact radix select on order-preserving 32-bit keys.
//
//  topk_hist     many workgroups per row count the first 12-bit digit of the
//                keys (also fused into the importance update).
//  topk_select   one 1024-thread workgroup per row.  Each thread holds a
//                contiguous 32-key segment of the row in registers (32768
//                keys per chunk, loaded with coalesced reads and transposed
//                through LDS; rows up to that length are read once).  The
//                threshold key is found digit by digit (12 + 12 + 8 bits;
//                later digits only count keys that still tie on the earlier
//                ones), then every key above it plus the lowest-index keys
//                equal to it are written in ascending token order, placed by
//                one block-wide scan of (greater, equal) counts per chunk.
//
// The result is exactly the k largest S with ties to the lower index: the
// keys are integers, so no floating-point rounding is involved.
#include <hip/hip_ext.h>

#include "hill_device.h"
#include "hill_internal.h"

namespace hill {

namespace {

constexpr int kSelThreads = 1024;
constexpr int kSelPer = 32;                         // keys per thread per chunk
constexpr int kSelChunk = kSelThreads * kSelPer;    // 32768 keys

__global__ __launch_bounds__(256) void topk_hist_kernel(const float* __restrict__ s, int64_t s_sb, int64_t s_sr,
                                                        int R, int n, uint32_t* __restrict__ hist)
{
    __shared__ uint32_t lds_hist[kHistBins];
    const int row = blockIdx.y;
    const int b = row / R, r = row % R;
    for (int i = threadIdx.x; i < kHistBins; i += 256) lds_hist[i] = 0u;
    __syncthreads();
    const float* srow = s + (int64_t)b * s_sb + (int64_t)r * s_sr;
    constexpr int kPer = kHistChunk / 256;
#pragma unroll
    for (int i = 0; i < kPer; ++i) {
        const int j = blockIdx.x * kHistChunk + i * 256 + threadIdx.x;
        if (j < n) atomicAdd(&lds_hist[order_key(srow[j]) >> (32 - kHistBits)], 1u);
    }
    __syncthreads();
    uint32_t* gh = hist + (int64_t)row * kHistBins;
    for (int i = threadIdx.x; i < kHistBins; i += 256) {
        const uint32_t c = lds_hist[i];
        if (c) atomicAdd(gh + i, c);
    }
}

constexpr int kSelPitch = kSelPer + 1;             // LDS words per thread segment (bank-conflict free)

// Stage chunk c of the row through LDS: coalesced 16-byte global loads, then
// each thread takes its contiguous segment of tokens [c*kSelChunk + 32*tid, +32)
// as order keys.  Returns how many of those tokens are inside the row.
// Row bases are 16-byte aligned.  Every thread of the block must call this.
__device__ __forceinline__ int load_segment(const float* srow, int c, int n, uint32_t* stage,
                                            uint32_t (&key)[kSelPer])
{
    const int tid = threadIdx.x;
    const int c0 = c * kSelChunk;
#pragma unroll
    for (int i = 0; i < kSelPer / 4; ++i) {
        const int pl = 4 * (i * kSelThreads + tid);     // position within the chunk
        const int p = c0 + pl;
        uint32_t k4[4];
        if (p + 3 < n) {
            const float4 x = *reinterpret_cast<const float4*>(srow + p);
            k4[0] = order_key(x.x);
            k4[1] = order_key(x.y);
            k4[2] = order_key(x.z);
            k4[3] = order_key(x.w);
        } else {
#pragma unroll
            for (int e = 0; e < 4; ++e) k4[e] = p + e < n ? order_key(srow[p + e]) : 0u;
        }
        uint32_t* dst = stage + (pl / kSelPer) * kSelPitch + (pl % kSelPer);
#pragma unroll
        for (int e = 0; e < 4; ++e) dst[e] = k4[e];
    }
    __syncthreads();
#pragma unroll
    for (int i = 0; i < kSelPer; ++i) key[i] = stage[tid * kSelPitch + i];
    __syncthreads();
    return min(max(n - (c0 + tid * kSelPer), 0), kSelPer);
}

// Given a histogram of `nb` bins (nb in {256, 4096}) in LDS, find the bin
// holding the need-th largest key: the largest d with count(bins >= d) >= need.
// Writes the bin and count(bins > d) to res[0], res[1].
__device__ void find_bin(const uint32_t* hist, int nb, uint32_t need, uint32_t* scan_scratch, uint32_t* res)
{
    const int tid = threadIdx.x;
    if (tid == 0) {   // defined result even if the counts were inconsistent
        res[0] = 0u;
        res[1] = 0u;
    }
    const int per = nb / kSelThreads > 0 ? nb / kSelThreads : 1;
    const int nthreads = nb / per;
    // thread t owns bins [nb - (t+1)*per, nb - t*per), visited from the top
    uint32_t local = 0;
    if (tid < nthreads)
        for (int i = 0; i < per; ++i) local += hist[nb - 1 - (tid * per + i)];
    uint32_t total;
    const uint32_t before = block_excl_scan<kSelThreads>(local, scan_scratch, &total);
    if (tid < nthreads && before < need && before + local >= need) {
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

__global__ __launch_bounds__(kSelThreads) void topk_select_kernel(SelectArgs a)
{
    __shared__ uint32_t stage[kSelThreads * kSelPitch];
    __shared__ uint32_t hist[kHistBins];
    __shared__ uint32_t scan_scratch[kSelThreads / 64 + 1];
    __shared__ uint2 scan2_scratch[kSelThreads / 64 + 1];
    __shared__ uint32_t res[2];

    const int tid = threadIdx.x;
    const int row = blockIdx.x;
    const int b = row / a.R, r = row % a.R;
    const float* srow = a.s + (int64_t)b * a.s_sb + (int64_t)r * a.s_sr;
    const int n = a.n;
    const int nchunks = (n + kSelChunk - 1) / kSelChunk;

    uint32_t key[kSelPer];
    int valid = 0;
    if (nchunks == 1) valid = load_segment(srow, 0, n, stage, key);

    // digit 1 (bits 31..20): counts come from the multi-workgroup histogram
    const uint32_t* gh = a.hist + (int64_t)row * kHistBins;
    for (int i = tid; i < kHistBins; i += kSelThreads) hist[i] = gh[i];
    __syncthreads();
    uint32_t need = (uint32_t)a.k;
    find_bin(hist, kHistBins, need, scan_scratch, res);
    uint32_t prefix = res[0] & (kHistBins - 1);
    int shift = 20;
    need -= res[1];
    uint32_t in_bin = hist[prefix];

    // digits 2 (bits 19..8) and 3 (bits 7..0), only while the threshold bin is split
    for (int pass = 0; pass < 2 && need < in_bin; ++pass) {
        const int nb = pass == 0 ? kHistBins : 256;
        const int next_shift = pass == 0 ? 8 : 0;
        __syncthreads();
        for (int i = tid; i < nb; i += kSelThreads) hist[i] = 0u;
        __syncthreads();
        for (int c = 0; c < nchunks; ++c) {
            if (nchunks > 1) valid = load_segment(srow, c, n, stage, key);
#pragma unroll
            for (int i = 0; i < kSelPer; ++i)
                if (i < valid && (key[i] >> shift) == prefix)
                    atomicAdd(&hist[(key[i] >> next_shift) & (uint32_t)(nb - 1)], 1u);
        }
        __syncthreads();
        find_bin(hist, nb, need, scan_scratch, res);
        const uint32_t d = res[0] & (uint32_t)(nb - 1);
        need -= res[1];
        in_bin = hist[d];
        prefix = (prefix << (shift - next_shift)) | d;
        shift = next_shift;
    }
    // Selection rule: (key >> shift) > prefix, or == prefix and among the
    // first `need` such keys in token order.

    int32_t* out_idx = a.idx + (int64_t)row * a.k;
    float* out_val = a.val ? a.val + (int64_t)row * a.k : nullptr;
    uint32_t carry_gt = 0, carry_eq = 0;
    for (int c = 0; c < nchunks; ++c) {
        if (nchunks > 1) valid = load_segment(srow, c, n, stage, key);
        uint32_t gtm = 0u, eqm = 0u;   // bit i: token 32*tid + i is above / at the threshold
#pragma unroll
        for (int i = 0; i < kSelPer; ++i) {
            const uint32_t kd = key[i] >> shift;
            gtm |= (i < valid && kd > prefix) ? (1u << i) : 0u;
            eqm |= (i < valid && kd == prefix) ? (1u << i) : 0u;
        }
        uint2 total;
        const uint2 before = block_excl_scan2<kSelThreads>(
            make_uint2((uint32_t)__builtin_popcount(gtm), (uint32_t)__builtin_popcount(eqm)), scan2_scratch, &total);
        const int j0 = c * kSelChunk + tid * kSelPer;
        for (uint32_t m = gtm | eqm; m; m &= m - 1u) {
            const int i = __builtin_ctz(m);
            const uint32_t below = (1u << i) - 1u;
            const uint32_t gt_b = carry_gt + before.x + (uint32_t)__builtin_popcount(gtm & below);
            const uint32_t eq_b = carry_eq + before.y + (uint32_t)__builtin_popcount(eqm & below);
            if (((gtm >> i) & 1u) || eq_b < need) {
                const uint32_t pos = gt_b + (eq_b < need ? eq_b : need);
                if (pos < (uint32_t)a.k) {
                    out_idx[pos] = j0 + i;
                    if (out_val) out_val[pos] = srow[j0 + i];
                }
            }
        }
        carry_gt += total.x;
        carry_eq += total.y;
    }
}

}  // namespace

hipError_t launch_topk_hist(const float* s, int64_t s_sb, int64_t s_sr, int B, int R, int n, uint32_t* hist,
                            hipStream_t st, Stamp ts)
{
    dim3 grid((n + kHistChunk - 1) / kHistChunk, B * R);
    hipExtLaunchKernelGGL(topk_hist_kernel, grid, dim3(256), 0, st, ts.start, ts.stop, 0, s, s_sb, s_sr, R, n, hist);
    return hipGetLastError();
}

hipError_t launch_topk_select(const SelectArgs& a, int rows, hipStream_t st, Stamp ts)
{
    hipExtLaunchKernelGGL(topk_select_kernel, dim3(rows), dim3(kSelThreads), 0, st, ts.start, ts.stop, 0, a);
    return hipGetLastError();
}

}  // namespace hill
