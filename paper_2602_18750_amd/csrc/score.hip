// Importance scoring on gfx950.
//
//  score_tiles   streams every cached key row once and forms the raw logits
//                q.K^T of all query heads that share it (GQA group)
//                (Sec. 4.4 raw inner product; Eq. 1).  ATTN keeps the logits
//                and a per-tile (max, sum of exp2) pair per head; RAW sums
//                each head group per token.
//  softmax_stats reduces the tile pairs to one (max, 1/sum) per head: the
//                softmax normaliser over all n tokens of Eq. 1.
//  update_*      turns logits into weights and adds their per-row column sum
//                to the cumulative importance S (Sec. 4.1 metric), and counts
//                the first radix digit of the new S for the selection.
//
// Key rows are 256 bytes (D = 128 x 16 bit).  A group of 16 lanes reads one
// row with 16-byte loads, so a wave reads 4 contiguous rows (1 KiB) per load;
// each lane keeps 8 rows in flight.  Partial dot products are combined with
// four DPP adds inside the 16-lane group.
#include "hill_device.h"
#include "hill_internal.h"

namespace hill {

namespace {

constexpr int kRowsPerLane = kScoreTile / 16;  // 8 key rows in flight per lane
constexpr float kLog2e = 1.4426950408889634f;

__global__ __launch_bounds__(256) void fill_zero_kernel(uint32_t* p, int64_t words)
{
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < words;
         i += (int64_t)gridDim.x * blockDim.x)
        p[i] = 0u;
}

template <int DT, int GC, int OUT>
__global__ __launch_bounds__(256) void score_tiles_kernel(ScoreArgs a)
{
    __shared__ float tile_logit[OUT == kOutLogits ? GC : 1][kScoreTile];

    const int tid = threadIdx.x;
    const int rg = tid >> 4;    // row group: which of the 16 rows of a load slot
    const int l16 = tid & 15;   // 16-byte column within the row

    if (a.zero_ptr) {
        for (int64_t i = (int64_t)blockIdx.x * 256 + tid; i < a.zero_words; i += (int64_t)gridDim.x * 256)
            a.zero_ptr[i] = 0u;
    }

    const int total = a.B * a.Hkv * a.ntiles;
    for (int t = blockIdx.x; t < total; t += gridDim.x) {
        const int tile = t % a.ntiles;
        const int bg = t / a.ntiles;
        const int g = bg % a.Hkv;
        const int b = bg / a.Hkv;
        const int j0 = tile * kScoreTile;
        const uint16_t* kb = a.k + (int64_t)b * a.k_sb + (int64_t)g * a.k_sh + l16 * 8;

        uint4 kr[kRowsPerLane];
#pragma unroll
        for (int u = 0; u < kRowsPerLane; ++u) {
            const int j = j0 + u * 16 + rg;
            if (j < a.n)
                kr[u] = load_stream16(kb + (int64_t)j * a.k_sn);
            else
                kr[u] = make_uint4(0u, 0u, 0u, 0u);
        }

        float rawsum[kRowsPerLane];
#pragma unroll
        for (int u = 0; u < kRowsPerLane; ++u) rawsum[u] = 0.0f;

        for (int hc = 0; hc < a.G; hc += GC) {
            uint4 qv[GC];
#pragma unroll
            for (int hh = 0; hh < GC; ++hh) {
                const int h = g * a.G + hc + hh;
                qv[hh] = *reinterpret_cast<const uint4*>(a.q + (int64_t)b * a.q_sb + (int64_t)h * a.q_sh + l16 * 8);
            }
#pragma unroll
            for (int u = 0; u < kRowsPerLane; ++u) {
#pragma unroll
                for (int hh = 0; hh < GC; ++hh) {
                    float d = sum16(dot8<DT>(kr[u], qv[hh]));
                    if constexpr (OUT == kOutLogits) {
                        if (l16 == hh) tile_logit[hh][u * 16 + rg] = d;
                    } else {
                        rawsum[u] += d;
                    }
                }
            }
            if constexpr (OUT == kOutLogits) {
                __syncthreads();
                // coalesced logits store: GC rows of kScoreTile floats
                for (int e = tid; e < GC * kScoreTile; e += 256) {
                    const int hh = e / kScoreTile, c = e % kScoreTile;
                    const int j = j0 + c;
                    if (j < a.n) {
                        const int h = g * a.G + hc + hh;
                        a.logits[((int64_t)b * a.Hq + h) * a.n + j] = tile_logit[hh][c];
                    }
                }
                // per-tile softmax partials in the exp2 domain: one wave per head
                const int w = tid >> 6, lane = tid & 63;
                for (int hh = w; hh < GC; hh += 4) {
                    const int c0 = lane, c1 = lane + 64;
                    const bool v0 = j0 + c0 < a.n, v1 = j0 + c1 < a.n;
                    const float x0 = v0 ? a.s2 * tile_logit[hh][c0] : -INFINITY;
                    const float x1 = v1 ? a.s2 * tile_logit[hh][c1] : -INFINITY;
                    const float m = wave_max(fmaxf(x0, x1));
                    float z = (v0 ? exp2f(x0 - m) : 0.0f) + (v1 ? exp2f(x1 - m) : 0.0f);
                    z = wave_sum(z);
                    if (lane == 0) {
                        const int h = g * a.G + hc + hh;
                        a.part[((int64_t)b * a.Hq + h) * a.ntiles + tile] = make_float2(m, z);
                    }
                }
                __syncthreads();
            }
        }

        if constexpr (OUT != kOutLogits) {
            if (l16 == 0) {
#pragma unroll
                for (int u = 0; u < kRowsPerLane; ++u) {
                    const int j = j0 + u * 16 + rg;
                    if (j < a.n) {
                        if constexpr (OUT == kOutRawS)
                            a.s[(int64_t)b * a.s_sb + (int64_t)g * a.s_sr + j] += rawsum[u];
                        else
                            a.logits[((int64_t)b * a.Hkv + g) * a.n + j] = rawsum[u];
                    }
                }
            }
        }
    }
}

// One wave per (b, h): combine the tile pairs into (max, 1/sum) in a fixed order.
__global__ __launch_bounds__(256) void softmax_stats_kernel(const float2* __restrict__ part,
                                                            float2* __restrict__ stats, int bh_total, int ntiles)
{
    const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
    const int bh = blockIdx.x * 4 + w;
    if (bh >= bh_total) return;
    const float2* p = part + (int64_t)bh * ntiles;
    float m = -INFINITY;
    for (int i = lane; i < ntiles; i += 64) m = fmaxf(m, p[i].x);
    m = wave_max(m);
    float z = 0.0f;
    for (int i = lane; i < ntiles; i += 64) {
        const float2 pi = p[i];
        z += pi.y * exp2f(pi.x - m);
    }
    z = wave_sum(z);
    if (lane == 0) stats[bh] = make_float2(m, 1.0f / z);
}

// Local histogram of the first radix digit of the new S values, merged into
// the row's global histogram (integer atomics: order-independent result).
__device__ __forceinline__ void hist_flush(uint32_t* lds_hist, uint32_t* ghist)
{
    __syncthreads();
    for (int i = threadIdx.x; i < kHistBins; i += blockDim.x) {
        const uint32_t c = lds_hist[i];
        if (c) atomicAdd(ghist + i, c);
    }
}

// S[b,r,j] += sum_{h in heads(r)} exp2(s2*l - max_h) / sum_h   (softmax weights)
__global__ __launch_bounds__(256) void update_attn_kernel(UpdateArgs a)
{
    __shared__ uint32_t lds_hist[kHistBins];
    const int row = blockIdx.y;          // b * R + r
    const int b = row / a.R, r = row % a.R;
    const int h0 = a.R == 1 ? 0 : r * a.G;
    const int nh = a.R == 1 ? a.Hq : a.G;
    const bool do_hist = a.hist != nullptr;
    if (do_hist) {
        for (int i = threadIdx.x; i < kHistBins; i += 256) lds_hist[i] = 0u;
        __syncthreads();
    }
    float* srow = a.s + (int64_t)b * a.s_sb + (int64_t)r * a.s_sr;
    const float* lg = a.logits + ((int64_t)b * a.Hq + h0) * a.n;
    const float2* st = a.stats + (int64_t)b * a.Hq + h0;
    constexpr int kPer = kUpdChunk / 256;
#pragma unroll
    for (int i = 0; i < kPer; ++i) {
        const int j = blockIdx.x * kUpdChunk + i * 256 + threadIdx.x;
        if (j < a.n) {
            float acc = 0.0f;
            for (int h = 0; h < nh; ++h) {
                const float2 ms = st[h];
                acc += exp2f(a.s2 * lg[(int64_t)h * a.n + j] - ms.x) * ms.y;
            }
            const float s_new = srow[j] + acc;
            srow[j] = s_new;
            if (do_hist) atomicAdd(&lds_hist[order_key(s_new) >> (32 - kHistBits)], 1u);
        }
    }
    if (do_hist) hist_flush(lds_hist, a.hist + (int64_t)row * kHistBins);
}

// Token rows, RAW mode, Hkv > 1: S[b,0,j] += sum_g groupsum[b,g,j].
__global__ __launch_bounds__(256) void update_raw_groups_kernel(UpdateArgs a)
{
    __shared__ uint32_t lds_hist[kHistBins];
    const int b = blockIdx.y;
    const bool do_hist = a.hist != nullptr;
    if (do_hist) {
        for (int i = threadIdx.x; i < kHistBins; i += 256) lds_hist[i] = 0u;
        __syncthreads();
    }
    float* srow = a.s + (int64_t)b * a.s_sb;
    const float* gs = a.logits + (int64_t)b * a.Hkv * a.n;
    constexpr int kPer = kUpdChunk / 256;
#pragma unroll
    for (int i = 0; i < kPer; ++i) {
        const int j = blockIdx.x * kUpdChunk + i * 256 + threadIdx.x;
        if (j < a.n) {
            float acc = 0.0f;
            for (int g = 0; g < a.Hkv; ++g) acc += gs[(int64_t)g * a.n + j];
            const float s_new = srow[j] + acc;
            srow[j] = s_new;
            if (do_hist) atomicAdd(&lds_hist[order_key(s_new) >> (32 - kHistBits)], 1u);
        }
    }
    if (do_hist) hist_flush(lds_hist, a.hist + (int64_t)b * kHistBins);
}

template <int DT, int OUT>
hipError_t launch_score_gc(const ScoreArgs& a, int gc, dim3 grid, hipStream_t st)
{
    switch (gc) {
    case 8: hipLaunchKernelGGL((score_tiles_kernel<DT, 8, OUT>), grid, dim3(256), 0, st, a); break;
    case 4: hipLaunchKernelGGL((score_tiles_kernel<DT, 4, OUT>), grid, dim3(256), 0, st, a); break;
    case 2: hipLaunchKernelGGL((score_tiles_kernel<DT, 2, OUT>), grid, dim3(256), 0, st, a); break;
    default: hipLaunchKernelGGL((score_tiles_kernel<DT, 1, OUT>), grid, dim3(256), 0, st, a); break;
    }
    return hipGetLastError();
}

template <int DT>
hipError_t launch_score_dt(const ScoreArgs& a, ScoreOut out, int gc, dim3 grid, hipStream_t st)
{
    switch (out) {
    case kOutLogits: return launch_score_gc<DT, kOutLogits>(a, gc, grid, st);
    case kOutRawS: return launch_score_gc<DT, kOutRawS>(a, gc, grid, st);
    default: return launch_score_gc<DT, kOutRawGroups>(a, gc, grid, st);
    }
}

}  // namespace

hipError_t launch_fill_zero(uint32_t* p, int64_t words, hipStream_t st)
{
    if (words <= 0) return hipSuccess;
    int64_t blocks = (words + 255) / 256;
    if (blocks > 1024) blocks = 1024;
    hipLaunchKernelGGL(fill_zero_kernel, dim3((unsigned)blocks), dim3(256), 0, st, p, words);
    return hipGetLastError();
}

hipError_t launch_score_tiles(const ScoreArgs& a, int dtype, ScoreOut out, int grid_cap, hipStream_t st)
{
    // heads per pass over the key registers: the largest of 8, 4, 2, 1 dividing G
    const int gc = (a.G % 8 == 0) ? 8 : (a.G % 4 == 0) ? 4 : (a.G % 2 == 0) ? 2 : 1;
    int64_t total = (int64_t)a.B * a.Hkv * a.ntiles;
    int64_t grid = total < grid_cap ? total : grid_cap;
    if (grid < 1) grid = 1;
    if (dtype == 1) return launch_score_dt<1>(a, out, gc, dim3((unsigned)grid), st);
    return launch_score_dt<0>(a, out, gc, dim3((unsigned)grid), st);
}

hipError_t launch_softmax_stats(const float2* part, float2* stats, int bh, int ntiles, hipStream_t st)
{
    hipLaunchKernelGGL(softmax_stats_kernel, dim3((bh + 3) / 4), dim3(256), 0, st, part, stats, bh, ntiles);
    return hipGetLastError();
}

hipError_t launch_update_attn(const UpdateArgs& a, hipStream_t st)
{
    dim3 grid((a.n + kUpdChunk - 1) / kUpdChunk, a.B * a.R);
    hipLaunchKernelGGL(update_attn_kernel, grid, dim3(256), 0, st, a);
    return hipGetLastError();
}

hipError_t launch_update_raw_groups(const UpdateArgs& a, hipStream_t st)
{
    dim3 grid((a.n + kUpdChunk - 1) / kUpdChunk, a.B);
    hipLaunchKernelGGL(update_raw_groups_kernel, grid, dim3(256), 0, st, a);
    return hipGetLastError();
}

}  // namespace hill
