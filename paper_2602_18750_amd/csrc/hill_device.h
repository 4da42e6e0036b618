// Device helpers for the gfx950 kernels: 16-bit dot products, 16-lane DPP
// reductions, wave reductions/scans and the order-preserving key map used
// by the selection.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace hill {

typedef _Float16 half2_t __attribute__((ext_vector_type(2)));
typedef __bf16 bf162_t __attribute__((ext_vector_type(2)));

typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

// 16-byte load that bypasses cache retention (streamed once per step).
__device__ __forceinline__ uint4 load_stream16(const void* p)
{
    const u32x4_t v = __builtin_nontemporal_load(reinterpret_cast<const u32x4_t*>(p));
    return make_uint4(v.x, v.y, v.z, v.w);
}

// 16-byte non-temporal store: the logits of a short scan go to memory as they
// are written instead of staying dirty in L2 until the kernel's end, where
// their write-back delayed the next launch.
__device__ __forceinline__ void store_stream16(float* p, float4 v)
{
    typedef float f32x4_t __attribute__((ext_vector_type(4)));
    const f32x4_t x = {v.x, v.y, v.z, v.w};
    __builtin_nontemporal_store(x, reinterpret_cast<f32x4_t*>(p));
}

// 2^x on the transcendental unit alone (v_exp_f32, about 1 ulp), without the
// range scaling that keeps results below 2^-126 denormal: those come out as
// zero.  Every caller exponentiates relative to a maximum (softmax weights,
// rescaled partial sums), so such a term is below 2^-126 of the sum it joins.
__device__ __forceinline__ float exp2_ftz(float x)
{
    return __builtin_amdgcn_exp2f(x);
}

// 8-byte non-temporal load (streamed int4 key codes).
__device__ __forceinline__ uint2 load_stream8(const void* p)
{
    typedef uint32_t u32x2_t __attribute__((ext_vector_type(2)));
    const u32x2_t v = __builtin_nontemporal_load(reinterpret_cast<const u32x2_t*>(p));
    return make_uint2(v.x, v.y);
}

// fp32 += a.lo*b.lo + a.hi*b.hi over packed 16-bit pairs (v_dot2c_f32_{f16,bf16}).
template <int DT>
__device__ __forceinline__ float dot2(uint32_t a, uint32_t b, float c);

template <>
__device__ __forceinline__ float dot2<0>(uint32_t a, uint32_t b, float c)
{
    return __builtin_amdgcn_fdot2(__builtin_bit_cast(half2_t, a), __builtin_bit_cast(half2_t, b), c, false);
}

template <>
__device__ __forceinline__ float dot2<1>(uint32_t a, uint32_t b, float c)
{
    return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf162_t, a), __builtin_bit_cast(bf162_t, b),
                                           c, false);
}

// Dot product of 8 packed 16-bit elements (one 16-byte load each side).
template <int DT>
__device__ __forceinline__ float dot8(const uint4& k, const uint4& q)
{
    float acc = dot2<DT>(k.x, q.x, 0.0f);
    acc = dot2<DT>(k.y, q.y, acc);
    acc = dot2<DT>(k.z, q.z, acc);
    acc = dot2<DT>(k.w, q.w, acc);
    return acc;
}

// Widen a packed pair to two floats.
template <int DT>
__device__ __forceinline__ void widen2(uint32_t x, float& lo, float& hi);

template <>
__device__ __forceinline__ void widen2<0>(uint32_t x, float& lo, float& hi)
{
    half2_t h = __builtin_bit_cast(half2_t, x);
    lo = (float)h[0];
    hi = (float)h[1];
}

template <>
__device__ __forceinline__ void widen2<1>(uint32_t x, float& lo, float& hi)
{
    lo = __uint_as_float(x << 16);
    hi = __uint_as_float(x & 0xffff0000u);
}

template <int CTRL>
__device__ __forceinline__ float dpp(float v)
{
    return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), CTRL, 0xF, 0xF,
                                                                  false));
}

// Sum over each aligned group of 8 lanes; every lane of the group gets the sum.
// quad_perm[1,0,3,2], quad_perm[2,3,0,1], row_half_mirror.
__device__ __forceinline__ float sum8(float v)
{
    v += dpp<0xB1>(v);
    v += dpp<0x4E>(v);
    v += dpp<0x141>(v);
    return v;
}

// Integer sum over each aligned group of 8 lanes (exact); every lane of the
// group gets the sum.
__device__ __forceinline__ int isum8(int v)
{
    v += __builtin_amdgcn_update_dpp(0, v, 0xB1, 0xF, 0xF, false);
    v += __builtin_amdgcn_update_dpp(0, v, 0x4E, 0xF, 0xF, false);
    v += __builtin_amdgcn_update_dpp(0, v, 0x141, 0xF, 0xF, false);
    return v;
}

// Max over each aligned group of 8 / 16 lanes; every lane of the group gets it.
__device__ __forceinline__ float max8(float v)
{
    v = fmaxf(v, dpp<0xB1>(v));
    v = fmaxf(v, dpp<0x4E>(v));
    v = fmaxf(v, dpp<0x141>(v));
    return v;
}

__device__ __forceinline__ float max16(float v)
{
    v = max8(v);
    return fmaxf(v, dpp<0x140>(v));
}

// Exponent of a scoring sketch with codes in [-QMAX, QMAX] (127: int8, 7:
// int4) of a row whose largest magnitude is amax: the smallest e with
// amax * 2^-e <= QMAX, clamped to [-128, 127] (-128 for an all-zero row).
// frexp is exact; QMAX / (QMAX + 1) is exact in fp32.
template <int QMAX>
__device__ __forceinline__ int sketch_exponent(float amax)
{
    static_assert(QMAX == 127 || QMAX == 7, "int8 or int4 codes");
    constexpr int kLg = QMAX == 127 ? 7 : 3;   // QMAX + 1 = 2^kLg
    if (!(amax > 0.0f)) return -128;
    int E;
    const float m = frexpf(amax, &E);   // amax = m * 2^E, m in [0.5, 1)
    const int e = m <= (float)QMAX / (float)(QMAX + 1) ? E - kLg : E - kLg + 1;
    return e < -128 ? -128 : (e > 127 ? 127 : e);
}

// Code of x under exponent e: x * 2^-e (exact) rounded to nearest, ties to
// even, clamped to [-QMAX, QMAX].
template <int QMAX>
__device__ __forceinline__ int sketch_code(float x, int e)
{
    const float r = rintf(ldexpf(x, -e));
    return (int)fminf(fmaxf(r, -(float)QMAX), (float)QMAX);
}

// Sum over each aligned group of 16 lanes; every lane of the group gets the sum.
// quad_perm[1,0,3,2], quad_perm[2,3,0,1], row_half_mirror, row_mirror.
__device__ __forceinline__ float sum16(float v)
{
    v += dpp<0xB1>(v);
    v += dpp<0x4E>(v);
    v += dpp<0x141>(v);
    v += dpp<0x140>(v);
    return v;
}

__device__ __forceinline__ float readlane_f(float v, int lane)
{
    return __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), lane));
}

// Max over the 64 lanes of a wave (every lane active): a 16-lane DPP
// reduction, then the four row results read as scalars.
__device__ __forceinline__ float wave_max(float v)
{
    v = fmaxf(v, dpp<0xB1>(v));
    v = fmaxf(v, dpp<0x4E>(v));
    v = fmaxf(v, dpp<0x141>(v));
    v = fmaxf(v, dpp<0x140>(v));
    return fmaxf(fmaxf(readlane_f(v, 0), readlane_f(v, 16)), fmaxf(readlane_f(v, 32), readlane_f(v, 48)));
}

// Sum over the 64 lanes of a wave (every lane active), in a fixed order.
__device__ __forceinline__ float wave_sum(float v)
{
    v = sum16(v);
    return (readlane_f(v, 0) + readlane_f(v, 16)) + (readlane_f(v, 32) + readlane_f(v, 48));
}

template <int CTRL, int ROW_MASK>
__device__ __forceinline__ uint32_t dpp_u32(uint32_t v)
{
    // lanes that the control does not write (masked rows, shifted-in lanes) read 0
    return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, CTRL, ROW_MASK, 0xF, false);
}

// Inclusive prefix sum over the 64 lanes of a wave, all in DPP: shifts by
// 1, 2, 4, 8 within each 16-lane row (row_shr), then the last lane of row 0
// added to row 1 and of row 2 to row 3 (row_bcast:15), then the last lane of
// row 1 added to rows 2 and 3 (row_bcast:31).
__device__ __forceinline__ uint32_t wave_incl_scan(uint32_t v)
{
    v += dpp_u32<0x111, 0xF>(v);   // row_shr:1
    v += dpp_u32<0x112, 0xF>(v);   // row_shr:2
    v += dpp_u32<0x114, 0xF>(v);   // row_shr:4
    v += dpp_u32<0x118, 0xF>(v);   // row_shr:8
    v += dpp_u32<0x142, 0xA>(v);   // row_bcast:15 into rows 1 and 3
    v += dpp_u32<0x143, 0xC>(v);   // row_bcast:31 into rows 2 and 3
    return v;
}

// Sum over the 64 lanes of a wave (every lane active), as a scalar.
__device__ __forceinline__ uint32_t wave_sum_u32(uint32_t v)
{
    return (uint32_t)__builtin_amdgcn_readlane((int)wave_incl_scan(v), 63);
}

// 64 histogram bins held one per lane (lane l: count of bin l; higher bins
// hold larger keys).  Finds the bin L holding the need-th largest key
// (need >= 1) and the number of keys in the bins above L.  Wave-uniform
// results; L = 0 if the bins hold fewer than need keys.
__device__ __forceinline__ void wave_find_bin(uint32_t cnt, uint32_t need, int& L, uint32_t& above)
{
    const uint32_t incl = wave_incl_scan(cnt);
    const uint32_t total = __shfl(incl, 63, 64);
    const uint32_t suffix = total - incl + cnt;   // keys in bins >= this lane's
    const uint64_t m = __ballot(suffix >= need);  // lanes 0 .. L
    L = m ? 63 - __clzll((long long)m) : 0;
    above = __shfl(suffix - cnt, L, 64);
}

// Exclusive prefix sum over a 256-thread block with a single barrier.  The
// four wave totals stay in scratch[0..3], which must not be rewritten before
// the next barrier.
__device__ __forceinline__ uint32_t block_excl_scan_1b(uint32_t v, uint32_t* scratch, uint32_t* total)
{
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const uint32_t inc = wave_incl_scan(v);
    if (lane == 63) scratch[w] = inc;
    __syncthreads();
    uint32_t base = 0, tot = 0;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const uint32_t s = scratch[i];
        base += i < w ? s : 0u;
        tot += s;
    }
    *total = tot;
    return base + inc - v;
}

// Exclusive prefix sum over a block of NT threads (NT a multiple of 64, <= 1024).
// `scratch` holds at least NT/64 + 1 words of LDS.  Returns the block total in *total.
template <int NT>
__device__ __forceinline__ uint32_t block_excl_scan(uint32_t v, uint32_t* scratch, uint32_t* total)
{
    constexpr int NW = NT / 64;
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    uint32_t inc = wave_incl_scan(v);
    if (lane == 63) scratch[w] = inc;
    __syncthreads();
    if (w == 0) {
        uint32_t x = lane < NW ? scratch[lane] : 0u;
        uint32_t xi = wave_incl_scan(x);
        if (lane < NW) scratch[lane] = xi - x;
        if (lane == NW - 1) scratch[NW] = xi;
    }
    __syncthreads();
    uint32_t r = scratch[w] + inc - v;
    *total = scratch[NW];
    __syncthreads();
    return r;
}

// Exclusive prefix sums of two counters at once over a block of NT threads.
// `scratch` holds at least NT/64 + 1 uint2 of LDS.
template <int NT>
__device__ __forceinline__ uint2 block_excl_scan2(uint2 v, uint2* scratch, uint2* total)
{
    constexpr int NW = NT / 64;
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    uint2 inc = v;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
        const uint32_t tx = __shfl_up(inc.x, o, 64);
        const uint32_t ty = __shfl_up(inc.y, o, 64);
        if (lane >= o) {
            inc.x += tx;
            inc.y += ty;
        }
    }
    if (lane == 63) scratch[w] = inc;
    __syncthreads();
    if (w == 0) {
        uint2 x = lane < NW ? scratch[lane] : make_uint2(0u, 0u);
        uint2 xi = x;
#pragma unroll
        for (int o = 1; o < 64; o <<= 1) {
            const uint32_t tx = __shfl_up(xi.x, o, 64);
            const uint32_t ty = __shfl_up(xi.y, o, 64);
            if (lane >= o) {
                xi.x += tx;
                xi.y += ty;
            }
        }
        if (lane < NW) scratch[lane] = make_uint2(xi.x - x.x, xi.y - x.y);
        if (lane == NW - 1) scratch[NW] = xi;
    }
    __syncthreads();
    const uint2 base = scratch[w];
    *total = scratch[NW];
    __syncthreads();
    return make_uint2(base.x + inc.x - v.x, base.y + inc.y - v.y);
}

// Workgroup histogram in LDS that also lists the bins it touched, so that
// only those are added to the global histogram.  `bins` starts zeroed and
// *nlist at 0; `list` holds at least as many entries as distinct bins can
// be touched.
__device__ __forceinline__ void hist_add(uint32_t* bins, uint32_t* list, uint32_t* nlist, uint32_t bin)
{
    if (atomicAdd(&bins[bin], 1u) == 0u) list[atomicAdd(nlist, 1u)] = bin;
}

// Adds the touched bins to the global histogram (one integer atomic each:
// order-independent).  Called by every thread after a barrier.
__device__ __forceinline__ void hist_flush(const uint32_t* bins, const uint32_t* list, uint32_t nlist, uint32_t* ghist)
{
    for (uint32_t i = threadIdx.x; i < nlist; i += blockDim.x) {
        const uint32_t b = list[i];
        atomicAdd(ghist + b, bins[b]);
    }
}

// Order-preserving map of fp32 to uint32: larger float -> larger key.
// -0.0 is folded onto +0.0; every NaN maps to 0, below -inf.
__device__ __forceinline__ uint32_t order_key(float f)
{
    if (f != f) return 0u;
    uint32_t u = __float_as_uint(f);
    if (u == 0x80000000u) u = 0u;
    return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// Selection key of token j: pinned tokens (outside [lo, hi), with 0 <= lo <=
// hi; lo == hi pins all) take the largest key, which no float reaches (+inf
// maps to 0xFF800000, NaN to 0).
__device__ __forceinline__ uint32_t select_key(float f, int j, int lo, int hi)
{
    return (uint32_t)(j - lo) >= (uint32_t)(hi - lo) ? 0xFFFFFFFFu : order_key(f);
}

}  // namespace hill
