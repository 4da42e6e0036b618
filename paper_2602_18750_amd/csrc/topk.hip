// Top-k token selection on gfx950 (Sec. 3.1 top-alpha; Sec. 4.2 global
// top-alpha indices) as an exact radix select on order-preserving 32-bit keys.
//
//  topk_hist     many workgroups per row count the first 12-bit digit of the
//                keys (also fused into the importance update).
//  topk_select   one 1024-thread workgroup per row: finds the threshold key
//                digit by digit (12 + 12 + 8 bits; later digits only look at
//                keys that still tie on the earlier ones), then emits every
//                key above the threshold plus the lowest-index keys equal to
//                it, in ascending token order, with one ordered block scan
//                per 4096-key tile.
//
// The result is exactly the k largest S with ties to the lower index: the
// keys are integers, so no floating-point rounding is involved.
#include "hill_device.h"
#include "hill_internal.h"

namespace hill {

namespace {

constexpr int kSelThreads = 1024;
constexpr int kSelTile = kSelThreads * 4;

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

// Reads 4 consecutive keys starting at j (j a multiple of 4); keys past n are
// reported invalid.  The row base is 16-byte aligned.
__device__ __forceinline__ void load4(const float* srow, int j, int n, float v[4], bool ok[4])
{
    if (j + 3 < n) {
        const float4 x = *reinterpret_cast<const float4*>(srow + j);
        v[0] = x.x; v[1] = x.y; v[2] = x.z; v[3] = x.w;
        ok[0] = ok[1] = ok[2] = ok[3] = true;
    } else {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            ok[e] = j + e < n;
            v[e] = ok[e] ? srow[j + e] : 0.0f;
        }
    }
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
    __shared__ uint32_t hist[kHistBins];
    __shared__ uint32_t scan_scratch[kSelThreads / 64 + 1];
    __shared__ uint32_t res[2];

    const int tid = threadIdx.x;
    const int row = blockIdx.x;
    const int b = row / a.R, r = row % a.R;
    const float* srow = a.s + (int64_t)b * a.s_sb + (int64_t)r * a.s_sr;
    const int n = a.n;

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
        for (int base = 0; base < n; base += kSelTile) {
            float v[4];
            bool ok[4];
            load4(srow, base + tid * 4, n, v, ok);
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const uint32_t key = order_key(v[e]);
                if (ok[e] && (key >> shift) == prefix)
                    atomicAdd(&hist[(key >> next_shift) & (uint32_t)(nb - 1)], 1u);
            }
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
    for (int base = 0; base < n; base += kSelTile) {
        const int j = base + tid * 4;
        float v[4];
        bool ok[4];
        load4(srow, j, n, v, ok);
        uint32_t gt_mask = 0, eq_mask = 0;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const uint32_t key = order_key(v[e]) >> shift;
            if (ok[e] && key > prefix) gt_mask |= 1u << e;
            if (ok[e] && key == prefix) eq_mask |= 1u << e;
        }
        const uint32_t packed = ((uint32_t)__builtin_popcount(gt_mask) << 16) | (uint32_t)__builtin_popcount(eq_mask);
        uint32_t total;
        const uint32_t before = block_excl_scan<kSelThreads>(packed, scan_scratch, &total);
        uint32_t gt_b = carry_gt + (before >> 16);
        uint32_t eq_b = carry_eq + (before & 0xffffu);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const bool is_gt = (gt_mask >> e) & 1u;
            const bool is_eq = (eq_mask >> e) & 1u;
            if (is_gt || (is_eq && eq_b < need)) {
                const uint32_t pos = gt_b + (eq_b < need ? eq_b : need);
                if (pos < (uint32_t)a.k) {
                    out_idx[pos] = j + e;
                    if (out_val) out_val[pos] = v[e];
                }
            }
            gt_b += is_gt;
            eq_b += is_eq;
        }
        carry_gt += total >> 16;
        carry_eq += total & 0xffffu;
    }
}

}  // namespace

hipError_t launch_topk_hist(const float* s, int64_t s_sb, int64_t s_sr, int B, int R, int n, uint32_t* hist,
                            hipStream_t st)
{
    dim3 grid((n + kHistChunk - 1) / kHistChunk, B * R);
    hipLaunchKernelGGL(topk_hist_kernel, grid, dim3(256), 0, st, s, s_sb, s_sr, R, n, hist);
    return hipGetLastError();
}

hipError_t launch_topk_select(const SelectArgs& a, int rows, hipStream_t st)
{
    hipLaunchKernelGGL(topk_select_kernel, dim3(rows), dim3(kSelThreads), 0, st, a);
    return hipGetLastError();
}

}  // namespace hill
