// Device building blocks of the sparse decode attention (Eq. 1 restricted to
// the selected set, softmax renormalised over it; Sec. 4.1 workflow step 6),
// shared by the standalone split-K kernel and the fused select+attend kernel.
//
// A 256-thread workgroup handles one (sequence b, KV head g) and GC query
// heads of its group over a list of selected tokens, in blocks of at most
// kAttnBlock list entries held in LDS:
//   A  logits: sixteen 16-lane row groups take every 16th entry; lane l16
//      loads elements [8*l16, 8*l16+8) of the token's K row (16-byte loads,
//      read in place from the cache) and four DPP adds finish each dot
//      product.  The logits of the block go to LDS.
//   B  softmax: one wave per head takes the block maximum, folds it into the
//      head's running maximum and turns the logits into exp2 weights (one
//      exp2 per head and token) and their sum.
//   C  values: wave w takes entries w, w+4, ...; lane l reads elements
//      (2l, 2l+1) of the V row (one 4-byte load per lane: a whole 256-byte
//      row per wave instruction) and accumulates weight * V for every head.
//      The V loads of the first batch are issued before phase A.
// When the scan's logits of the same keys are at hand (the fused step over
// the 16-bit cache), the caller puts them in LDS with the list and phase A
// is skipped: only V rows are read (attn_block_logits).
// The four waves' outputs are added in LDS at the end, and one partial
// (m, l, o[D]) per head is written to a slot of the partial buffer; partials
// of all slots are merged by merge_head().
#pragma once

#include "hill_device.h"
#include "hill_internal.h"

namespace hill {

constexpr int kAttnBlock = 512;   // list entries per LDS block
constexpr int kKBatch = 4;        // K rows per row group per batch (64 entries)
constexpr int kVBatch = 16;       // V rows per wave per batch (64 entries)
// Zero weights after a block's last entry: a wave's batch of eight entries
// reaches at most 30 entries past the block's count, which then weigh 0
// without a per-entry test.
constexpr int kWeightPad = 32;

template <int GC>
struct AttnLds {
    int32_t tok[kAttnBlock];          // token index of each entry of the block
    float p[kAttnBlock + kWeightPad][GC];   // logits, then exp2 weights (0 past the block's entries)
    float mrun[GC], lrun[GC], alpha[GC];
    float o[4][GC][kHeadDim];         // per-wave outputs, added at the end
};

// This lane's 8 query elements of heads g*G+hc .. +GC (16-lane row layout).
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

// Running state of one workgroup's attention: this lane's two output
// elements (2*lane, 2*lane+1) per head, summed over its wave's entries.
template <int GC>
struct AttnAcc {
    float o[GC][2];
};

template <int GC>
__device__ __forceinline__ void attn_begin(AttnAcc<GC>& acc, AttnLds<GC>& sh)
{
#pragma unroll
    for (int hh = 0; hh < GC; ++hh) acc.o[hh][0] = acc.o[hh][1] = 0.0f;
    if (threadIdx.x < GC) {
        sh.mrun[threadIdx.x] = -INFINITY;
        sh.lrun[threadIdx.x] = 0.0f;
    }
}

// Row offset of token j (clamped into [0, n) so that a bad index reads a
// valid row instead of faulting; lists hold valid tokens).  Row strides are
// below 2^31 elements (checked on the host): one 32x32->64-bit multiply.
__device__ __forceinline__ uint64_t row_off(int j, int n, int64_t stride)
{
    j = min(max(j, 0), n - 1);
    return (uint64_t)(uint32_t)j * (uint32_t)stride;
}

// Where list entry t's row lies: the cache row of its token, or, in a tiered
// cache (TIER), the hot pool's slot sloc[t] when that is >= 0 and the cold
// pool's row of the token otherwise (sloc: the entries' slots in LDS).  cold
// and hot are the row bases of this lane's slice for the (b, KV head).
struct RowSrc {
    const uint16_t* cold;
    const uint16_t* hot;
    int64_t cold_sn, hot_sn;
    int n, cap;
    const int32_t* sloc;
};

template <bool TIER>
__device__ __forceinline__ const uint16_t* entry_row(const RowSrc& r, const int32_t* tok, int t)
{
    if constexpr (TIER) {
        const int s = r.sloc[t];
        const bool hot = s >= 0;
        return hot ? r.hot + row_off(s, r.cap, r.hot_sn) : r.cold + row_off(tok[t], r.n, r.cold_sn);
    }
    return r.cold + row_off(tok[t], r.n, r.cold_sn);
}

// K rows of entries t0, t0+16, ... (kKBatch of them) for this lane's
// 16-byte slice; entries past cnt are clamped to the last one (their logits
// are not stored).  Unconditional loads keep the wait counters exact.
template <bool TIER = false>
__device__ __forceinline__ void load_k_rows(const RowSrc& kr_src, const int32_t* tok, int t0, int cnt,
                                            uint4 (&kr)[kKBatch])
{
#pragma unroll
    for (int u = 0; u < kKBatch; ++u) {
        const int t = min(t0 + 16 * u, cnt - 1);
        kr[u] = *reinterpret_cast<const uint4*>(entry_row<TIER>(kr_src, tok, t));
    }
}

// V element pairs of entries t0, t0+4, ... (kVBatch of them); entries past
// cnt are clamped to the last one (they weigh 0).
template <bool TIER = false>
__device__ __forceinline__ void load_v_rows(const RowSrc& vr_src, const int32_t* tok, int t0, int cnt,
                                            uint32_t (&vr)[kVBatch])
{
#pragma unroll
    for (int i = 0; i < kVBatch; ++i) {
        const int t = min(t0 + 4 * i, cnt - 1);
        vr[i] = *reinterpret_cast<const uint32_t*>(entry_row<TIER>(vr_src, tok, t));
    }
}

// The K (lane offset 8 * l16 elements) and V (lane offset 2 * lane) row
// sources of (b, g): the cache, or the two pools of a tiered cache with the
// block's slots in sloc.
__device__ __forceinline__ RowSrc k_src(const AttnArgs& a, int b, int g, const int32_t* sloc)
{
    const int l16 = threadIdx.x & 15;
    RowSrc r;
    r.cold = a.k + (int64_t)b * a.k_sb + (int64_t)g * a.k_sh + l16 * 8;
    r.cold_sn = a.k_sn;
    r.n = a.n;
    r.hot = a.loc ? a.k_hot + (int64_t)b * a.hk_sb + (int64_t)g * a.hk_sh + l16 * 8 : r.cold;
    r.hot_sn = a.hk_sn;
    r.cap = a.cap;
    r.sloc = sloc;
    return r;
}

__device__ __forceinline__ RowSrc v_src(const AttnArgs& a, int b, int g, const int32_t* sloc)
{
    const int lane = threadIdx.x & 63;
    RowSrc r;
    r.cold = a.v + (int64_t)b * a.v_sb + (int64_t)g * a.v_sh + 2 * lane;
    r.cold_sn = a.v_sn;
    r.n = a.n;
    r.hot = a.loc ? a.v_hot + (int64_t)b * a.hv_sb + (int64_t)g * a.hv_sh + 2 * lane : r.cold;
    r.hot_sn = a.hv_sn;
    r.cap = a.cap;
    r.sloc = sloc;
    return r;
}

// Logits of entries t0, t0+16, ... into sh.p (lane l16 == hh of the row group
// writes head hh).  nu (wave-uniform) bounds the batches that hold an entry
// of any row group of the wave; entries past cnt are not stored.
template <int DT, int GC>
__device__ __forceinline__ void logits_rows(const AttnArgs& a, const uint4 (&qv)[GC], const uint4 (&kr)[kKBatch], int t0,
                                            int cnt, int nu, float (*p)[GC])
{
    const int l16 = threadIdx.x & 15;
#pragma unroll
    for (int u = 0; u < kKBatch; ++u) {
        if (u >= nu) break;
        const int t = t0 + 16 * u;
        float mine = 0.0f;   // lane l16 == hh keeps head hh's dot product
#pragma unroll
        for (int hh = 0; hh < GC; ++hh) {
            const float d = sum16(dot8<DT>(kr[u], qv[hh]));
            mine = l16 == hh ? d : mine;
        }
        if (l16 < GC && t < cnt) p[t][l16] = a.s2 * mine;
    }
}

// weight * V of this wave's entries idx0 .. idx0+N-1 (entry w + 4*idx) into
// the accumulators; entries at or past nmine lie past the block's count,
// where softmax_block left zero weights (their V registers hold a clamped,
// valid row).
template <int DT, int GC>
__device__ __forceinline__ void values_rows(const uint32_t (&vr)[kVBatch], int w, int idx0, int nmine, int cnt,
                                            const float (*p)[GC], AttnAcc<GC>& acc)
{
#pragma unroll
    for (int c0 = 0; c0 < kVBatch; c0 += 8) {
        if (idx0 + c0 >= nmine) break;   // wave-uniform
#pragma unroll
        for (int i = c0; i < c0 + 8; ++i) {
            const int idx = idx0 + i;
            const int tc = w + 4 * idx;   // < cnt + kWeightPad
            float v0, v1;
            widen2<DT>(vr[i], v0, v1);
            float pw[GC];
            if constexpr (GC % 4 == 0) {
#pragma unroll
                for (int h4 = 0; h4 < GC; h4 += 4) {
                    const float4 x = *reinterpret_cast<const float4*>(&p[tc][h4]);
                    pw[h4] = x.x;
                    pw[h4 + 1] = x.y;
                    pw[h4 + 2] = x.z;
                    pw[h4 + 3] = x.w;
                }
            } else {
#pragma unroll
                for (int hh = 0; hh < GC; ++hh) pw[hh] = p[tc][hh];
            }
#pragma unroll
            for (int hh = 0; hh < GC; ++hh) {
                acc.o[hh][0] += pw[hh] * v0;
                acc.o[hh][1] += pw[hh] * v1;
            }
        }
    }
}

// Softmax step of a block of cnt entries whose logits are in sh.p: per head
// (one wave each), block maximum -> running maximum, exp2 weights in place
// and their sum; ends with a barrier.
template <int GC>
__device__ __forceinline__ void softmax_block(int cnt, AttnLds<GC>& sh)
{
    const int lane = threadIdx.x & 63;
    const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    for (int hh = w; hh < GC; hh += 4) {
        float mx = -INFINITY;
        for (int t = lane; t < cnt; t += 64) mx = fmaxf(mx, sh.p[t][hh]);
        mx = wave_max(mx);
        const float m_old = sh.mrun[hh];
        const float m_new = fmaxf(m_old, mx);
        float ls = 0.0f;
        for (int t = lane; t < cnt; t += 64) {
            const float e = exp2_ftz(sh.p[t][hh] - m_new);
            sh.p[t][hh] = e;
            ls += e;
        }
        ls = wave_sum(ls);
        if (lane < kWeightPad) sh.p[cnt + lane][hh] = 0.0f;   // entries past the block weigh 0
        if (lane == 0) {
            const float al = m_old == -INFINITY ? 0.0f : exp2_ftz(m_old - m_new);
            sh.alpha[hh] = al;
            sh.lrun[hh] = sh.lrun[hh] * al + ls;
            sh.mrun[hh] = m_new;
        }
    }
    __syncthreads();
}

// weight * V over this wave's entries w, w+4, ... of the block: the first 16
// (and, when `two`, 32) from the rows already loaded, the rest loaded here.
template <int DT, int GC, bool TIER = false>
__device__ __forceinline__ void values_block(const RowSrc& vs, int w, int cnt, int nmine, bool two,
                                             const uint32_t (&vr)[kVBatch], const uint32_t (&vr2)[kVBatch],
                                             AttnAcc<GC>& acc, AttnLds<GC>& sh)
{
#pragma unroll
    for (int hh = 0; hh < GC; ++hh) {
        const float al = sh.alpha[hh];
        acc.o[hh][0] *= al;
        acc.o[hh][1] *= al;
    }
    values_rows<DT, GC>(vr, w, 0, nmine, cnt, sh.p, acc);
    if (two) values_rows<DT, GC>(vr2, w, kVBatch, nmine, cnt, sh.p, acc);
    for (int i0 = 2 * kVBatch; i0 < nmine; i0 += kVBatch) {   // lists longer than 128
        uint32_t vx[kVBatch];
        load_v_rows<TIER>(vs, sh.tok, w + 4 * i0, cnt, vx);
        values_rows<DT, GC>(vx, w, i0, nmine, cnt, sh.p, acc);
    }
}

// Folds list entries [0, cnt) of sh.tok (1 <= cnt <= kAttnBlock, written and
// made visible by a barrier before the call) into the running state.  Every
// thread of the workgroup must call this.  The K rows are issued before the
// V rows, so that the logits wait for K only; every loop bound is
// wave-uniform.  TIER: a tiered cache, the entries' hot-pool slots in sloc
// (written with sh.tok).
template <int DT, int GC, bool TIER = false>
__device__ __forceinline__ void attn_block(const AttnArgs& a, int b, int g, const uint4 (&qv)[GC], int cnt,
                                           AttnAcc<GC>& acc, AttnLds<GC>& sh, const int32_t* sloc = nullptr)
{
    const int tid = threadIdx.x;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);   // wave-uniform: scalar control flow
    const int rg = tid >> 4;
    const RowSrc ks = k_src(a, b, g, sloc);
    const RowSrc vs = v_src(a, b, g, sloc);

    // A: logits of every entry, into sh.p.  Up to 128 entries take one round
    // trip: the K rows of entries < 64 (and < 128 when the list is longer),
    // then the V rows of this wave's first 16 (and 32) entries.
    const int nmine = cnt > w ? (cnt - w + 3) / 4 : 0;   // this wave's entries w, w+4, ...
    const bool two = cnt > 16 * kKBatch;                 // block-uniform
    uint4 kr[kKBatch], kr2[kKBatch];
    load_k_rows<TIER>(ks, sh.tok, rg, cnt, kr);
    if (two) load_k_rows<TIER>(ks, sh.tok, rg + 16 * kKBatch, cnt, kr2);
    __builtin_amdgcn_sched_barrier(0);   // keep the K loads ahead of the V loads in the queue
    uint32_t vr[kVBatch], vr2[kVBatch];
    load_v_rows<TIER>(vs, sh.tok, w, cnt, vr);
    if (two) load_v_rows<TIER>(vs, sh.tok, w + 4 * kVBatch, cnt, vr2);
    logits_rows<DT, GC>(a, qv, kr, rg, cnt, (cnt - 4 * w + 15) / 16, sh.p);
    if (two) logits_rows<DT, GC>(a, qv, kr2, rg + 16 * kKBatch, cnt, (cnt - 16 * kKBatch - 4 * w + 15) / 16, sh.p);
    for (int base = 32 * kKBatch; base < cnt; base += 16 * kKBatch) {   // lists longer than 128
        uint4 kx[kKBatch];
        load_k_rows<TIER>(ks, sh.tok, base + rg, cnt, kx);
        logits_rows<DT, GC>(a, qv, kx, base + rg, cnt, (cnt - base - 4 * w + 15) / 16, sh.p);
    }
    __syncthreads();

    softmax_block<GC>(cnt, sh);
    values_block<DT, GC, TIER>(vs, w, cnt, nmine, two, vr, vr2, acc, sh);
}

// attn_block with the logits already in sh.p (scaled by s2, written with
// sh.tok before the barrier that precedes the call, after attn_begin): only
// the V rows are read, and their loads are in flight during the softmax.
template <int DT, int GC>
__device__ __forceinline__ void attn_block_logits(const AttnArgs& a, int b, int g, int cnt, AttnAcc<GC>& acc,
                                                  AttnLds<GC>& sh)
{
    const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const RowSrc vs = v_src(a, b, g, nullptr);
    const int nmine = cnt > w ? (cnt - w + 3) / 4 : 0;
    const bool two = cnt > 4 * kVBatch;   // block-uniform
    uint32_t vr[kVBatch], vr2[kVBatch];
    load_v_rows(vs, sh.tok, w, cnt, vr);
    if (two) load_v_rows(vs, sh.tok, w + 4 * kVBatch, cnt, vr2);
    softmax_block<GC>(cnt, sh);
    values_block<DT, GC>(vs, w, cnt, nmine, two, vr, vr2, acc, sh);
}

// Adds the four waves' outputs and writes the partial (m, l, o[D]) of heads
// g*G+hc .. +GC to slot `slot` of `nslots`.  An empty list gives m = -inf,
// l = 0, o = 0 (weight 0 in the merge).  Every thread must call this.
template <int GC>
__device__ __forceinline__ void attn_finish(const AttnArgs& a, int b, int g, int hc, const AttnAcc<GC>& acc, int slot,
                                            int nslots, AttnLds<GC>& sh)
{
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
#pragma unroll
    for (int hh = 0; hh < GC; ++hh)
        *reinterpret_cast<float2*>(&sh.o[w][hh][2 * lane]) = make_float2(acc.o[hh][0], acc.o[hh][1]);
    __syncthreads();
    for (int e = tid; e < GC * kHeadDim; e += 256) {
        const int hh = e / kHeadDim, d = e % kHeadDim;
        const float o = ((sh.o[0][hh][d] + sh.o[1][hh][d]) + sh.o[2][hh][d]) + sh.o[3][hh][d];
        const int64_t pi = ((int64_t)b * a.Hq + g * a.G + hc + hh) * nslots + slot;
        a.part_o[pi * kHeadDim + d] = o;
        if (d == 0) a.part_ml[pi] = make_float2(sh.mrun[hh], sh.lrun[hh]);
    }
    __syncthreads();
}

// out[b,h,d0:d0+DS] = sum_s e^{m_s - M} o_s / sum_s e^{m_s - M} l_s over the
// nslots partials of head h (empty slots have l = 0 and weigh 0), for one
// slice of DS output dimensions.  Thread t takes dimension d0 + t % DS of
// every (NT/DS)-th slot, starting at slot t / DS: it loads those slots' o and
// (m, l) at once, and after one block-wide maximum adds both its weighted o
// and its weighted l; the groups' sums are then added in order.  red holds
// NT/64 + NT/DS floats, osum NT floats.  One workgroup of NT threads per
// (b, h, slice); every slice forms the same (M, L).
template <int NT, int DS = kHeadDim>
__device__ __forceinline__ void merge_head(const AttnArgs& a, int b, int h, int d0, int nslots, float* red,
                                           float* osum)
{
    static_assert(NT % DS == 0 && kHeadDim % DS == 0, "slices tile the head and the workgroup");
    constexpr int NW = NT / 64, NG = NT / DS, kPre = NG >= 8 ? 16 : 32;
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const int d = tid % DS, grp = tid / DS;
    const int64_t bh = (int64_t)b * a.Hq + h;
    const float2* ml = a.part_ml + bh * nslots;
    const float* po = a.part_o + bh * nslots * kHeadDim + d0 + d;

    // this thread's first kPre slots: o and (m, l) in flight together
    float x[kPre];
    float2 v[kPre];
#pragma unroll
    for (int i = 0; i < kPre; ++i) {
        const int s = grp + i * NG;
        x[i] = s < nslots ? po[(int64_t)s * kHeadDim] : 0.0f;
        v[i] = s < nslots ? ml[s] : make_float2(-INFINITY, 0.0f);
    }
    float mx = -INFINITY;
#pragma unroll
    for (int i = 0; i < kPre; ++i) mx = fmaxf(mx, v[i].y > 0.0f ? v[i].x : -INFINITY);
    for (int s = grp + kPre * NG; s < nslots; s += NG) {
        const float2 u = ml[s];
        mx = fmaxf(mx, u.y > 0.0f ? u.x : -INFINITY);
    }
    mx = wave_max(mx);
    if (lane == 0) red[w] = mx;
    __syncthreads();
    mx = red[0];
#pragma unroll
    for (int i = 1; i < NW; ++i) mx = fmaxf(mx, red[i]);
    float O = 0.0f, L = 0.0f;
#pragma unroll
    for (int i = 0; i < kPre; ++i) {
        const float ws = v[i].y > 0.0f ? exp2_ftz(v[i].x - mx) : 0.0f;
        O += ws * x[i];
        L += ws * v[i].y;
    }
    for (int s0 = grp + kPre * NG; s0 < nslots; s0 += kPre * NG) {
#pragma unroll
        for (int i = 0; i < kPre; ++i) {
            const int s = s0 + i * NG;
            x[i] = s < nslots ? po[(int64_t)s * kHeadDim] : 0.0f;
            v[i] = s < nslots ? ml[s] : make_float2(-INFINITY, 0.0f);
        }
#pragma unroll
        for (int i = 0; i < kPre; ++i) {
            const float ws = v[i].y > 0.0f ? exp2_ftz(v[i].x - mx) : 0.0f;
            O += ws * x[i];
            L += ws * v[i].y;
        }
    }
    osum[tid] = O;
    if (d == 0) red[NW + grp] = L;
    __syncthreads();
    if (grp == 0) {
        float t = osum[d], l = red[NW];
#pragma unroll
        for (int q = 1; q < NG; ++q) {
            t += osum[q * DS + d];
            l += red[NW + q];
        }
        a.out[bh * kHeadDim + d0 + d] = t / l;
    }
}

}  // namespace hill
