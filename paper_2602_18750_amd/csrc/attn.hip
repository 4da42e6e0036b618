// Sparse decode attention over the selected tokens on gfx950 (Eq. 1
// restricted to the selected set I, softmax renormalised over I; Sec. 4.1
// workflow step 6: only the selected tokens' original 16-bit K and V are
// read).
//
//  attn_split    one workgroup per (sequence, KV head, split of I).  The
//                selected K and V rows are gathered in place from the cache
//                (no copy) and each row is read once for all G query heads
//                of the group.  A 16-lane group handles one token at a time
//                with an online softmax (running max, sum, and 8 of the 128
//                output dims per lane); the 16 groups are merged in LDS.
//  attn_combine  merges the split partials of each query head.
//
// Softmax arithmetic runs in the exp2 domain (scale pre-multiplied by log2 e).
#include <hip/hip_ext.h>

#include "hill_device.h"
#include "hill_internal.h"

namespace hill {

namespace {

constexpr int kTokBatch = 4;  // tokens per 16-lane group whose rows are loaded together

template <int DT, int GC>
__global__ __launch_bounds__(256) void attn_split_kernel(AttnArgs a)
{
    __shared__ float sm[16][GC];
    __shared__ float sl[16][GC];
    __shared__ float so[16][GC][kHeadDim];

    const int tid = threadIdx.x;
    const int rg = tid >> 4, l16 = tid & 15;
    const int split = blockIdx.x;
    const int bg = blockIdx.y;
    const int b = bg / a.Hkv, g = bg % a.Hkv;
    const int r = a.R == 1 ? 0 : g;
    const int32_t* I = a.idx + ((int64_t)b * a.R + r) * a.ksel;
    const int t0 = split * a.per_split;
    const int t1 = min(t0 + a.per_split, a.ksel);
    const uint16_t* kb = a.k + (int64_t)b * a.k_sb + (int64_t)g * a.k_sh + l16 * 8;
    const uint16_t* vb = a.v + (int64_t)b * a.v_sb + (int64_t)g * a.v_sh + l16 * 8;

    for (int hc = 0; hc < a.G; hc += GC) {
        uint4 qv[GC];
#pragma unroll
        for (int hh = 0; hh < GC; ++hh) {
            const int h = g * a.G + hc + hh;
            qv[hh] = *reinterpret_cast<const uint4*>(a.q + (int64_t)b * a.q_sb + (int64_t)h * a.q_sh + l16 * 8);
        }
        float m[GC], l[GC], o[GC][8];
#pragma unroll
        for (int hh = 0; hh < GC; ++hh) {
            m[hh] = -INFINITY;
            l[hh] = 0.0f;
#pragma unroll
            for (int i = 0; i < 8; ++i) o[hh][i] = 0.0f;
        }

        for (int tb = t0 + rg; tb < t1; tb += 16 * kTokBatch) {
            // indices first (clamped into the split, so every load is in bounds),
            // then every K and V row of the batch, then the arithmetic
            int jj[kTokBatch];
#pragma unroll
            for (int u = 0; u < kTokBatch; ++u) jj[u] = I[min(tb + u * 16, t1 - 1)];
            uint4 kr[kTokBatch], vr[kTokBatch];
#pragma unroll
            for (int u = 0; u < kTokBatch; ++u) {
                // clamped: an out-of-range index reads a valid row instead of faulting
                const int64_t j = min(max(jj[u], 0), a.n - 1);
                kr[u] = *reinterpret_cast<const uint4*>(kb + j * a.k_sn);
                vr[u] = *reinterpret_cast<const uint4*>(vb + j * a.v_sn);
            }
#pragma unroll
            for (int u = 0; u < kTokBatch; ++u) {
                if (tb + u * 16 >= t1) break;   // uniform within the 16-lane group
                float vf[8];
                widen2<DT>(vr[u].x, vf[0], vf[1]);
                widen2<DT>(vr[u].y, vf[2], vf[3]);
                widen2<DT>(vr[u].z, vf[4], vf[5]);
                widen2<DT>(vr[u].w, vf[6], vf[7]);
#pragma unroll
                for (int hh = 0; hh < GC; ++hh) {
                    const float x = a.s2 * sum16(dot8<DT>(kr[u], qv[hh]));
                    const float mn = fmaxf(m[hh], x);
                    const float sc = exp2f(m[hh] - mn);
                    const float p = exp2f(x - mn);
                    l[hh] = l[hh] * sc + p;
#pragma unroll
                    for (int i = 0; i < 8; ++i) o[hh][i] = o[hh][i] * sc + p * vf[i];
                    m[hh] = mn;
                }
            }
        }

#pragma unroll
        for (int hh = 0; hh < GC; ++hh) {
#pragma unroll
            for (int i = 0; i < 8; ++i) so[rg][hh][l16 * 8 + i] = o[hh][i];
            if (l16 == 0) {
                sm[rg][hh] = m[hh];
                sl[rg][hh] = l[hh];
            }
        }
        __syncthreads();
        for (int e = tid; e < GC * kHeadDim; e += 256) {
            const int hh = e / kHeadDim, d = e % kHeadDim;
            float mx = -INFINITY;
#pragma unroll
            for (int q = 0; q < 16; ++q) mx = fmaxf(mx, sm[q][hh]);
            float accl = 0.0f, acco = 0.0f;
#pragma unroll
            for (int q = 0; q < 16; ++q) {
                const float w = sl[q][hh] > 0.0f ? exp2f(sm[q][hh] - mx) : 0.0f;
                accl += w * sl[q][hh];
                acco += w * so[q][hh][d];
            }
            const int h = g * a.G + hc + hh;
            const int64_t pi = ((int64_t)b * a.Hq + h) * a.nsplit + split;
            a.part_o[pi * kHeadDim + d] = acco;
            if (d == 0) a.part_ml[pi] = make_float2(mx, accl);
        }
        __syncthreads();
    }
}

// out[b,h,:] = sum_s e^{m_s - M} o_s / sum_s e^{m_s - M} l_s.  The split
// weights are formed once in LDS; each thread then accumulates one output
// dimension over the splits with several loads in flight.
__global__ __launch_bounds__(kHeadDim) void attn_combine_kernel(AttnArgs a)
{
    __shared__ float wsplit[kMaxSplits];
    __shared__ float red[kHeadDim / 64];
    const int bh = blockIdx.x;
    const int d = threadIdx.x;
    const int lane = d & 63, w = d >> 6;
    const float2* ml = a.part_ml + (int64_t)bh * a.nsplit;
    float mx = -INFINITY;
    for (int s = d; s < a.nsplit; s += kHeadDim) mx = fmaxf(mx, ml[s].x);
    mx = wave_max(mx);
    if (lane == 0) red[w] = mx;
    __syncthreads();
    mx = red[0];
#pragma unroll
    for (int i = 1; i < kHeadDim / 64; ++i) mx = fmaxf(mx, red[i]);
    __syncthreads();
    float lsum = 0.0f;
    for (int s = d; s < a.nsplit; s += kHeadDim) {
        const float2 v = ml[s];
        const float ws = exp2f(v.x - mx);
        wsplit[s] = ws;
        lsum += ws * v.y;
    }
    lsum = wave_sum(lsum);
    if (lane == 0) red[w] = lsum;
    __syncthreads();
    float L = 0.0f;
#pragma unroll
    for (int i = 0; i < kHeadDim / 64; ++i) L += red[i];
    const float* po = a.part_o + (int64_t)bh * a.nsplit * kHeadDim + d;
    float O = 0.0f;
    int s = 0;
    for (; s + 8 <= a.nsplit; s += 8) {
        float x[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) x[i] = po[(int64_t)(s + i) * kHeadDim];
#pragma unroll
        for (int i = 0; i < 8; ++i) O += wsplit[s + i] * x[i];
    }
    for (; s < a.nsplit; ++s) O += wsplit[s] * po[(int64_t)s * kHeadDim];
    a.out[(int64_t)bh * kHeadDim + d] = O / L;
}

template <int DT>
hipError_t launch_attn_dt(const AttnArgs& a, dim3 grid, hipStream_t st)
{
    const int gc = (a.G % 8 == 0) ? 8 : (a.G % 4 == 0) ? 4 : (a.G % 2 == 0) ? 2 : 1;
    switch (gc) {
    case 8: hipLaunchKernelGGL((attn_split_kernel<DT, 8>), grid, dim3(256), 0, st, a); break;
    case 4: hipLaunchKernelGGL((attn_split_kernel<DT, 4>), grid, dim3(256), 0, st, a); break;
    case 2: hipLaunchKernelGGL((attn_split_kernel<DT, 2>), grid, dim3(256), 0, st, a); break;
    default: hipLaunchKernelGGL((attn_split_kernel<DT, 1>), grid, dim3(256), 0, st, a); break;
    }
    return hipGetLastError();
}

}  // namespace

hipError_t launch_attn_split(const AttnArgs& a, int dtype, hipStream_t st)
{
    dim3 grid(a.nsplit, a.B * a.Hkv);
    if (dtype == 1) return launch_attn_dt<1>(a, grid, st);
    return launch_attn_dt<0>(a, grid, st);
}

hipError_t launch_attn_combine(const AttnArgs& a, hipStream_t st, Stamp ts)
{
    hipExtLaunchKernelGGL(attn_combine_kernel, dim3(a.B * a.Hq), dim3(kHeadDim), 0, st, ts.start, ts.stop, 0, a);
    return hipGetLastError();
}

}  // namespace hill
