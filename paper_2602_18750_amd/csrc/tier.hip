// Row migration between the hot pool (HBM) and the cold pool (host memory)
// that a BKP pass decides (Sec. 4.2 BKP (3): promoted tokens move up, demoted
// tokens move down; the pools are exclusive, each token's K/V row lives in
// exactly one of them).
//
//  tier_apply   one workgroup per (list position i, row (b, r)), looping over
//               i: the i-th demoted token's row goes from its slot to the
//               cold pool and the i-th promoted token's row from the cold
//               pool into that slot; promoted tokens beyond the demoted ones
//               take the slots never used before (from used_prev on).  Each
//               row copy is 256 bytes, sixteen lanes x 16 bytes; a workgroup
//               reads every row it moves before it writes any, so a slot
//               that changes hands is read before it is overwritten.  Rows of
//               different list positions touch different slots and tokens.
#include <hip/hip_ext.h>

#include "hill_device.h"
#include "hill_internal.h"

namespace hill {

namespace {

constexpr int kTierWgs = 64;   // workgroups per row; each loops over list positions

__global__ __launch_bounds__(256) void tier_apply_kernel(TierArgs a)
{
    const int row = blockIdx.y;   // b * R + r
    const int b = row / a.R, r = row % a.R;
    const int np = a.counts[2 * row], nd = a.counts[2 * row + 1];
    // the pass must leave the pool min(cap, n) full: anything else (lists cut at list_cap, a pass
    // over a context other than the one the pool holds) leaves the row alone and raises status
    if (np - nd != a.used_now - a.used_prev || np > a.list_cap || nd > a.list_cap || np < 0 || nd < 0) {
        if (blockIdx.x == 0 && threadIdx.x == 0) atomicOr(a.status, 1);
        return;
    }
    const int heads = a.R == 1 ? a.Hkv : 1;   // token rows move every KV head's row
    const int g0 = a.R == 1 ? 0 : r;
    const int rg = threadIdx.x >> 4, l16 = threadIdx.x & 15;   // 16 row groups of 16 lanes
    int32_t* locrow = a.loc + (int64_t)row * a.loc_sr;
    const int npos = np > nd ? np : nd;
    for (int i = blockIdx.x; i < npos; i += gridDim.x) {
        int tok_d = i < nd ? a.demote[(int64_t)row * a.list_cap + i] : -1;
        int tok_p = i < np ? a.promote[(int64_t)row * a.list_cap + i] : -1;
        if (tok_d >= a.n) tok_d = -1;
        if (tok_p >= a.n) tok_p = -1;
        const int slot_d = tok_d >= 0 ? locrow[tok_d] : -1;
        const int slot_p = i < nd ? slot_d : a.used_prev + (i - nd);
        // a token out of range, a demoted token without a slot or a promoted one with a slot already:
        // the move is skipped and status raised (the lists did not come from a pass over this pool)
        const bool ok_d = i >= nd || (tok_d >= 0 && slot_d >= 0 && slot_d < a.cap);
        const bool ok_p = i >= np || (tok_p >= 0 && slot_p >= 0 && slot_p < a.cap && locrow[tok_p] < 0);
        if (!(ok_d && ok_p)) {
            if (threadIdx.x == 0) atomicOr(a.status, 2);
            tok_d = -1;
            tok_p = -1;
        }
        // row copies of this list position: per KV head, K then V, down (hot -> cold) then up (cold -> hot)
        const int jobs = heads * 4;
        for (int j0 = 0; j0 < jobs; j0 += 16) {
            const int job = j0 + rg;
            const bool act = job < jobs;
            const int g = g0 + (act ? job >> 2 : 0);
            const bool is_v = (job >> 1) & 1;
            const bool up = job & 1;
            const bool live = act && (up ? tok_p >= 0 : tok_d >= 0);
            const uint16_t* src = nullptr;
            uint16_t* dst = nullptr;
            if (live) {
                const int64_t hot_off = (int64_t)b * (is_v ? a.hv_sb : a.hk_sb) + (int64_t)g * (is_v ? a.hv_sh : a.hk_sh);
                const int64_t cold_off = (int64_t)b * (is_v ? a.cv_sb : a.ck_sb) + (int64_t)g * (is_v ? a.cv_sh : a.ck_sh);
                uint16_t* hot = (is_v ? a.v_hot : a.k_hot) + hot_off;
                uint16_t* cold = (is_v ? a.v_cold : a.k_cold) + cold_off;
                const int64_t hsn = is_v ? a.hv_sn : a.hk_sn, csn = is_v ? a.cv_sn : a.ck_sn;
                if (up) {
                    src = cold + (int64_t)tok_p * csn;
                    dst = hot + (int64_t)slot_p * hsn;
                } else {
                    src = hot + (int64_t)slot_d * hsn;
                    dst = cold + (int64_t)tok_d * csn;
                }
            }
            const uint4 v = live ? *reinterpret_cast<const uint4*>(src + 8 * l16) : make_uint4(0u, 0u, 0u, 0u);
            __syncthreads();   // every read of this round is done before any write
            if (live) *reinterpret_cast<uint4*>(dst + 8 * l16) = v;
        }
        if (threadIdx.x == 0) {
            if (tok_d >= 0) locrow[tok_d] = -1;
            if (tok_p >= 0) locrow[tok_p] = slot_p;
        }
    }
}

}  // namespace

hipError_t launch_tier_apply(const TierArgs& a, int rows, hipStream_t st, Stamp ts)
{
    const int x = a.list_cap < kTierWgs ? (a.list_cap < 1 ? 1 : a.list_cap) : kTierWgs;
    hipExtLaunchKernelGGL(tier_apply_kernel, dim3(x, rows), dim3(256), 0, st, ts.start, ts.stop, 0, a);
    return hipGetLastError();
}

}  // namespace hill
