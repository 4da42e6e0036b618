// Scoring sketch of the key cache (Sec. 4.4 asymmetric precision: the
// evaluation runs in low precision while attention keeps the 16-bit K and V).
//
//  sketch_keys  casts key rows [t0, t1) of every (sequence, KV head) to int8
//               (BITS 8) or int4 (BITS 4) codes with one power-of-two
//               exponent per row: the smallest e with max|x| * 2^-e <= qmax
//               (127 or 7), codes x * 2^-e rounded to nearest (ties to even).
//               Every operation is exact, so the sketch does not depend on
//               the order of evaluation.  In a decode loop it runs once per
//               appended token; the scan then reads 128 + 1 (int8) or 64 + 1
//               (int4) bytes per key row instead of 256.
//
// Layout: 16 lanes per row, lane l16 reads elements [8*l16, 8*l16+8) with one
// 16-byte load and writes their 8 codes with one 8-byte store (int8) or one
// 4-byte word (int4: byte i = (code i + 8) | (code i+4 + 8) << 4); a wave
// covers 4 rows, a workgroup 16.
#include <hip/hip_ext.h>

#include "hill_device.h"
#include "hill_internal.h"

namespace hill {

namespace {

template <int DT, int BITS>
__global__ __launch_bounds__(256) void sketch_keys_kernel(SketchArgs a)
{
    const int rows_per_bg = a.t1 - a.t0;
    const int64_t r = (int64_t)blockIdx.x * 16 + (threadIdx.x >> 4);   // row index over (b, g, token)
    const int l16 = threadIdx.x & 15;
    const int64_t total = (int64_t)a.B * a.Hkv * rows_per_bg;
    const bool valid = r < total;
    const int64_t rr = valid ? r : 0;
    const int64_t bg = rr / rows_per_bg;
    const int j = a.t0 + (int)(rr % rows_per_bg);
    const int b = (int)(bg / a.Hkv), g = (int)(bg % a.Hkv);
    // every lane of the wave takes part in the row maximum (clamped rows are not stored)
    const uint4 w = *reinterpret_cast<const uint4*>(a.k + (int64_t)b * a.k_sb + (int64_t)g * a.k_sh +
                                                    (int64_t)j * a.k_sn + l16 * 8);
    const uint32_t pw[4] = {w.x, w.y, w.z, w.w};
    float x[8];
    float amax = 0.0f;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        widen2<DT>(pw[i], x[2 * i], x[2 * i + 1]);
        amax = fmaxf(amax, fmaxf(fabsf(x[2 * i]), fabsf(x[2 * i + 1])));
    }
    constexpr int kQmax = BITS == 8 ? 127 : 7;
    const int e = sketch_exponent<kQmax>(max16(amax));
    if constexpr (BITS == 8) {
        uint32_t lo = 0u, hi = 0u;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            lo |= ((uint32_t)sketch_code<kQmax>(x[i], e) & 0xffu) << (8 * i);
            hi |= ((uint32_t)sketch_code<kQmax>(x[4 + i], e) & 0xffu) << (8 * i);
        }
        if (valid) {
            const int64_t row = bg * a.cap + j;
            *reinterpret_cast<uint2*>(a.k8 + row * kHeadDim + l16 * 8) = make_uint2(lo, hi);
            if (l16 == 0) a.k_exp[row] = (int8_t)e;
        }
    } else {
        uint32_t word = 0u;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const uint32_t lo = (uint32_t)(sketch_code<kQmax>(x[i], e) + 8);
            const uint32_t hi = (uint32_t)(sketch_code<kQmax>(x[4 + i], e) + 8);
            word |= (lo | (hi << 4)) << (8 * i);
        }
        if (valid) {
            const int64_t row = bg * a.cap + j;
            *reinterpret_cast<uint32_t*>(a.k8 + row * (kHeadDim / 2) + l16 * 4) = word;
            if (l16 == 0) a.k_exp[row] = (int8_t)e;
        }
    }
}

}  // namespace

hipError_t launch_sketch_keys(const SketchArgs& a, int dtype, hipStream_t st)
{
    const int64_t rows = (int64_t)a.B * a.Hkv * (a.t1 - a.t0);
    if (rows <= 0) return hipSuccess;
    const int64_t blocks = (rows + 15) / 16;
    const dim3 grid((unsigned)blocks);
    if (a.bits == 4) {
        if (dtype == 1) hipLaunchKernelGGL((sketch_keys_kernel<1, 4>), grid, dim3(256), 0, st, a);
        else hipLaunchKernelGGL((sketch_keys_kernel<0, 4>), grid, dim3(256), 0, st, a);
    } else {
        if (dtype == 1) hipLaunchKernelGGL((sketch_keys_kernel<1, 8>), grid, dim3(256), 0, st, a);
        else hipLaunchKernelGGL((sketch_keys_kernel<0, 8>), grid, dim3(256), 0, st, a);
    }
    return hipGetLastError();
}

}  // namespace hill
