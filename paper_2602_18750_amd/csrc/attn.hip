// Standalone sparse decode attention over a caller-given index set (Eq. 1
// restricted to the selected set I, softmax renormalised over I; Sec. 4.1
// workflow step 6: only the selected tokens' original 16-bit K and V rows are
// read, in place).  hill_step does not use these two kernels: its attention
// is fused into the selection's emit kernel (topk.hip).
//
//  attn_split    one workgroup per (sequence, KV head, split of I); each K
//                and V row is read once for all G query heads of the group.
//  attn_combine  merges the split partials of each query head.
#include <hip/hip_ext.h>

#include "attn_device.h"

namespace hill {

namespace {

template <int DT, int GC>
__global__ __launch_bounds__(256) void attn_split_kernel(AttnArgs a)
{
    __shared__ AttnLds<GC> sh;
    const int split = blockIdx.x;
    const int b = blockIdx.y / a.Hkv, g = blockIdx.y % a.Hkv;
    const int r = a.R == 1 ? 0 : g;
    const int32_t* I = a.idx + ((int64_t)b * a.R + r) * a.ksel;
    const int t0 = split * a.per_split;
    const int t1 = min(t0 + a.per_split, a.ksel);
    for (int hc = 0; hc < a.G; hc += GC) {
        uint4 qv[GC];
        load_queries<GC>(a, b, g, hc, qv);
        AttnAcc<GC> acc;
        attn_begin<GC>(acc, sh);
        for (int tb = t0; tb < t1; tb += kAttnBlock) {
            const int cnt = min(kAttnBlock, t1 - tb);
            __syncthreads();   // the previous block's list reads are done
            for (int i = threadIdx.x; i < cnt; i += 256) sh.tok[i] = I[tb + i];
            __syncthreads();
            attn_block<DT, GC>(a, b, g, qv, cnt, acc, sh);
        }
        attn_finish<GC>(a, b, g, hc, acc, split, a.nsplit, sh);
    }
}

__global__ __launch_bounds__(kHeadDim) void attn_combine_kernel(AttnArgs a)
{
    __shared__ float red[kHeadDim / 64 + 1];
    __shared__ float osum[kHeadDim];
    merge_head<kHeadDim>(a, blockIdx.x / a.Hq, blockIdx.x % a.Hq, 0, a.nsplit, red, osum);
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
