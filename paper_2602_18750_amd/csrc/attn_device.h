// Device building blocks of the sparse decode attention (Eq. 1 restricted to
// the selected set, softmax renormalised over it; Sec. 4.1 workflow step 6),
// shared by the standalone split-K kernel and the fused select+attend kernel.
//
// A 256-thread workgroup handles one (sequence b, KV head g) and GC query
// heads of its group over a list of selected tokens.  Sixteen 16-lane row
// groups each take every 16th token of the list: lane l16 loads elements
// [8*l16, 8*l16+8) of the token's K and V rows (16-byte loads, read in place
// from the cache), the dot products are summed by four DPP adds, and each
// row group keeps an online softmax (running max m, sum l, and 8 of the 128
// output dims per lane) per head.  The 16 row groups are then merged in LDS
// and one partial (m, l, o[D]) per head is written to a slot of the partial
// buffer; partials of all slots are merged by merge_head().
#pragma once

#include "hill_device.h"
#include "hill_internal.h"

namespace hill {

constexpr int kTokBatch = 4;   // tokens per row group whose rows are loaded together

template <int GC>
struct AttnLds {
    float m[16][GC];
    float l[16][GC];
    float o[16][GC][kHeadDim];
};

// This lane's 8 query elements of heads g*G+hc .. +GC.
template <int GC>
__device__ __forceinline__ void load_queries(const AttnArgs& a, int b, int g, int hc, uint4 (&qv)[GC])
{
    const int l16 = threadIdx.x & 15;
#pragma unroll
    for (int hh = 0; hh < GC; ++hh) {
        const int h = g * a.G + hc + hh;
        qv[hh] = *reinterpret_cast<const uint4*>(a.q + (int64_t)b * a.q_sb + (int64_t)h * a.q_sh + l16 * 8);
    }
}

// Merges the 16 row groups' online-softmax states (m, l, o) in LDS and writes
// one partial (m, l, o[D]) per head to slot `slot` of `nslots`.
template <int GC>
__device__ __forceinline__ void merge_row_groups(const AttnArgs& a, int b, int g, int hc, const float (&m)[GC],
                                                 const float (&l)[GC], const float (&o)[GC][8], int slot, int nslots,
                                                 AttnLds<GC>& sh)
{
    const int tid = threadIdx.x;
    const int rg = tid >> 4, l16 = tid & 15;
#pragma unroll
    for (int hh = 0; hh < GC; ++hh) {
#pragma unroll
        for (int i = 0; i < 8; ++i) sh.o[rg][hh][l16 * 8 + i] = o[hh][i];
        if (l16 == 0) {
            sh.m[rg][hh] = m[hh];
            sh.l[rg][hh] = l[hh];
        }
    }
    __syncthreads();
    for (int e = tid; e < GC * kHeadDim; e += 256) {
        const int hh = e / kHeadDim, d = e % kHeadDim;
        float mx = -INFINITY;
#pragma unroll
        for (int q = 0; q < 16; ++q) mx = fmaxf(mx, sh.m[q][hh]);
        float accl = 0.0f, acco = 0.0f;
#pragma unroll
        for (int q = 0; q < 16; ++q) {
            const float w = sh.l[q][hh] > 0.0f ? exp2f(sh.m[q][hh] - mx) : 0.0f;
            accl += w * sh.l[q][hh];
            acco += w * sh.o[q][hh][d];
        }
        const int h = g * a.G + hc + hh;
        const int64_t pi = ((int64_t)b * a.Hq + h) * nslots + slot;
        a.part_o[pi * kHeadDim + d] = acco;
        if (d == 0) a.part_ml[pi] = make_float2(mx, accl);
    }
    __syncthreads();
}


// One token's K and V row (this lane's 8 elements) folded into the online
// softmax state of each head.
template <int DT, int GC>
__device__ __forceinline__ void fold_token(const AttnArgs& a, const uint4 (&qv)[GC], const uint4& kr, const uint4& vr,
                                           float (&m)[GC], float (&l)[GC], float (&o)[GC][8])
{
    float vf[8];
    widen2<DT>(vr.x, vf[0], vf[1]);
    widen2<DT>(vr.y, vf[2], vf[3]);
    widen2<DT>(vr.z, vf[4], vf[5]);
    widen2<DT>(vr.w, vf[6], vf[7]);
#pragma unroll
    for (int hh = 0; hh < GC; ++hh) {
        const float x = a.s2 * sum16(dot8<DT>(kr, qv[hh]));
        const float mn = fmaxf(m[hh], x);
        const float sc = exp2f(m[hh] - mn);
        const float p = exp2f(x - mn);
        l[hh] = l[hh] * sc + p;
#pragma unroll
        for (int i = 0; i < 8; ++i) o[hh][i] = o[hh][i] * sc + p * vf[i];
        m[hh] = mn;
    }
}

// Partial attention where every row group attends over its own tokens:
// bit i of `mask` selects token jbase + i (mask and jbase uniform within the
// 16-lane group).  Rows are loaded kTokBatch at a time.
template <int DT, int GC>
__device__ __forceinline__ void attend_masked(const AttnArgs& a, int b, int g, int hc, const uint4 (&qv)[GC], int jbase,
                                              uint32_t mask, int slot, int nslots, AttnLds<GC>& sh)
{
    const int l16 = threadIdx.x & 15;
    const uint16_t* kb = a.k + (int64_t)b * a.k_sb + (int64_t)g * a.k_sh + l16 * 8;
    const uint16_t* vb = a.v + (int64_t)b * a.v_sb + (int64_t)g * a.v_sh + l16 * 8;
    float m[GC], l[GC], o[GC][8];
#pragma unroll
    for (int hh = 0; hh < GC; ++hh) {
        m[hh] = -INFINITY;
        l[hh] = 0.0f;
#pragma unroll
        for (int i = 0; i < 8; ++i) o[hh][i] = 0.0f;
    }
    while (mask) {
        int jj[kTokBatch];
        int cnt = 0;
#pragma unroll
        for (int u = 0; u < kTokBatch; ++u) {
            jj[u] = jbase + (mask ? __builtin_ctz(mask) : 0);
            cnt += mask ? 1 : 0;
            mask &= mask - 1u;
        }
        uint4 kr[kTokBatch], vr[kTokBatch];
#pragma unroll
        for (int u = 0; u < kTokBatch; ++u) {
            // clamped: an out-of-range index reads a valid row instead of faulting
            const int64_t j = min(max(jj[u], 0), a.n - 1);
            kr[u] = *reinterpret_cast<const uint4*>(kb + j * a.k_sn);
            vr[u] = *reinterpret_cast<const uint4*>(vb + j * a.v_sn);
        }
#pragma unroll
        for (int u = 0; u < kTokBatch; ++u)
            if (u < cnt) fold_token<DT, GC>(a, qv, kr[u], vr[u], m, l, o);
    }
    merge_row_groups<GC>(a, b, g, hc, m, l, o, slot, nslots, sh);
}

// Partial attention of heads g*G+hc .. +GC (queries qv from load_queries) over
// list entries [t0, t1), written to slot `slot` of `nslots`.  idx_at(t)
// returns the token index of entry t.  Every thread of the workgroup must
// call this.
template <int DT, int GC, typename IdxAt>
__device__ __forceinline__ void attend_partial(const AttnArgs& a, int b, int g, int hc, const uint4 (&qv)[GC], int t0,
                                               int t1, IdxAt idx_at, int slot, int nslots, AttnLds<GC>& sh)
{
    const int tid = threadIdx.x;
    const int rg = tid >> 4, l16 = tid & 15;
    const uint16_t* kb = a.k + (int64_t)b * a.k_sb + (int64_t)g * a.k_sh + l16 * 8;
    const uint16_t* vb = a.v + (int64_t)b * a.v_sb + (int64_t)g * a.v_sh + l16 * 8;

    float m[GC], l[GC], o[GC][8];
#pragma unroll
    for (int hh = 0; hh < GC; ++hh) {
        m[hh] = -INFINITY;
        l[hh] = 0.0f;
#pragma unroll
        for (int i = 0; i < 8; ++i) o[hh][i] = 0.0f;
    }

    for (int tb = t0 + rg; tb < t1; tb += 16 * kTokBatch) {
        // indices first (clamped into the list, so every load is in bounds),
        // then every K and V row of the batch, then the arithmetic
        int jj[kTokBatch];
#pragma unroll
        for (int u = 0; u < kTokBatch; ++u) jj[u] = idx_at(min(tb + u * 16, t1 - 1));
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
            fold_token<DT, GC>(a, qv, kr[u], vr[u], m, l, o);
        }
    }

    merge_row_groups<GC>(a, b, g, hc, m, l, o, slot, nslots, sh);
}

// out[b,h,:] = sum_s e^{m_s - M} o_s / sum_s e^{m_s - M} l_s over the nslots
// partials of head h (empty slots have l = 0 and weigh 0).  The slot weights
// are formed once in LDS (wsl holds nslots floats); thread t then sums output
// dimension t % D over every (blockDim/D)-th slot with eight loads in flight,
// and the slot groups are added in order.  red holds blockDim/64 + 1 floats,
// osum blockDim floats.  Called by one workgroup of NT threads per (b, h).
template <int NT>
__device__ __forceinline__ void merge_head(const AttnArgs& a, int b, int h, int nslots, float* wsl, float* red,
                                           float* osum)
{
    constexpr int NW = NT / 64, NG = NT / kHeadDim;
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const int d = tid % kHeadDim, grp = tid / kHeadDim;
    const int64_t bh = (int64_t)b * a.Hq + h;
    const float2* ml = a.part_ml + bh * nslots;
    float mx = -INFINITY;
    for (int s = tid; s < nslots; s += NT) {
        const float2 v = ml[s];
        mx = fmaxf(mx, v.y > 0.0f ? v.x : -INFINITY);
    }
    mx = wave_max(mx);
    if (lane == 0) red[w] = mx;
    __syncthreads();
    mx = red[0];
#pragma unroll
    for (int i = 1; i < NW; ++i) mx = fmaxf(mx, red[i]);
    __syncthreads();
    float lsum = 0.0f;
    for (int s = tid; s < nslots; s += NT) {
        const float2 v = ml[s];
        const float ws = v.y > 0.0f ? exp2f(v.x - mx) : 0.0f;
        wsl[s] = ws;
        lsum += ws * v.y;
    }
    lsum = wave_sum(lsum);
    if (lane == 0) red[w] = lsum;
    __syncthreads();
    float L = 0.0f;
#pragma unroll
    for (int i = 0; i < NW; ++i) L += red[i];
    const float* po = a.part_o + bh * nslots * kHeadDim + d;
    float O = 0.0f;
    int s = grp;
    for (; s + 8 * NG <= nslots; s += 8 * NG) {
        float x[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) x[i] = po[(int64_t)(s + i * NG) * kHeadDim];
#pragma unroll
        for (int i = 0; i < 8; ++i) O += wsl[s + i * NG] * x[i];
    }
    for (; s < nslots; s += NG) O += wsl[s] * po[(int64_t)s * kHeadDim];
    osum[tid] = O;
    __syncthreads();
    if (grp == 0) {
        float t = osum[d];
#pragma unroll
        for (int q = 1; q < NG; ++q) t += osum[q * kHeadDim + d];
        a.out[bh * kHeadDim + d] = t / L;
    }
}

}  // namespace hill
