// Bidirectional KV Cache Pools (Sec. 4.2, HKM / BKP) on gfx950: the per-token
// hit-rate table and the hot/cold pool policy, one pass after each decoding
// step.
//
//  bkp_hits   one hit for every token of the step's selected set (2-byte
//             counters, saturating; indices are unique within a row, so each
//             counter has one writer)
//  bkp_rank   per token the value the frequency slots are chosen by:
//             2 * hits + (hot before the call), -1 inside the recent window;
//             small integers, exact in fp32, so the library's exact top-k
//             (ties to the lower index) picks the slots
//  bkp_mark   flags the chosen tokens (bit 1 of the pool byte)
//  bkp_lists  one workgroup per row: the new pool (window or chosen), the
//             promotions and demotions compacted in token order
#include "hill_device.h"
#include "hill_internal.h"

namespace hill {

namespace {

__global__ __launch_bounds__(256) void bkp_hits_kernel(BkpArgs a)
{
    const int row = blockIdx.y;
    const int i = blockIdx.x * 256 + threadIdx.x;
    if (i >= a.k) return;
    const int j = a.idx[(int64_t)row * a.k + i];
    if ((unsigned)j >= (unsigned)a.n) return;
    uint16_t* h = a.hits + a.off(row) + j;
    const uint16_t x = *h;
    if (x != 0xffffu) *h = (uint16_t)(x + 1u);
}

__global__ __launch_bounds__(256) void bkp_rank_kernel(BkpArgs a)
{
    const int row = blockIdx.y;
    const int j = blockIdx.x * 256 + threadIdx.x;
    if (j >= a.n) return;
    const int64_t o = a.off(row) + j;
    const uint8_t hv = a.hot[o];
    const uint32_t old = hv & 1u;
    if (hv != old) a.hot[o] = (uint8_t)old;   // only bit 0 carries state between calls
    a.v[(int64_t)row * a.ld + j] = j >= a.n - a.w ? -1.0f : (float)(2u * a.hits[o] + old);
}

__global__ __launch_bounds__(256) void bkp_mark_kernel(BkpArgs a)
{
    const int row = blockIdx.y;
    const int i = blockIdx.x * 256 + threadIdx.x;
    if (i >= a.f) return;
    const int j = a.flist[(int64_t)row * a.f + i];
    uint8_t* p = a.hot + a.off(row) + j;
    *p = (uint8_t)(*p | 2u);
}

constexpr int kListPerThread = 4;

__global__ __launch_bounds__(256) void bkp_lists_kernel(BkpArgs a)
{
    __shared__ uint2 scratch[256 / 64 + 1];
    const int row = blockIdx.x;
    uint8_t* hot = a.hot + a.off(row);
    int32_t* pro = a.promote + (int64_t)row * a.list_cap;
    int32_t* dem = a.demote + (int64_t)row * a.list_cap;
    const int first_recent = a.n - a.w;
    uint32_t base_p = 0, base_d = 0;
    for (int j0 = 0; j0 < a.n; j0 += 256 * kListPerThread) {   // block-uniform trip count
        const int jt = j0 + kListPerThread * threadIdx.x;
        uint32_t nv = 0, moves = 0;   // per token u: bit u = hot now; bits 2u, 2u+1 = promoted, demoted
        uint2 c = make_uint2(0u, 0u);
#pragma unroll
        for (int u = 0; u < kListPerThread; ++u) {
            const int j = jt + u;
            if (j >= a.n) continue;
            const uint32_t h = hot[j];
            const uint32_t was = h & 1u;
            const uint32_t now = (j >= first_recent || (h & 2u)) ? 1u : 0u;
            nv |= now << u;
            if (now && !was) {
                moves |= 1u << (2 * u);
                ++c.x;
            } else if (was && !now) {
                moves |= 2u << (2 * u);
                ++c.y;
            }
        }
        uint2 tot;
        uint2 off = block_excl_scan2<256>(c, scratch, &tot);
#pragma unroll
        for (int u = 0; u < kListPerThread; ++u) {
            const int j = jt + u;
            if (j >= a.n) continue;
            hot[j] = (uint8_t)((nv >> u) & 1u);
            if ((moves >> (2 * u)) & 1u) {
                const uint32_t p = base_p + off.x++;
                if (p < (uint32_t)a.list_cap) pro[p] = j;
            } else if ((moves >> (2 * u)) & 2u) {
                const uint32_t p = base_d + off.y++;
                if (p < (uint32_t)a.list_cap) dem[p] = j;
            }
        }
        base_p += tot.x;
        base_d += tot.y;
    }
    if (threadIdx.x == 0) {
        a.counts[2 * (int64_t)row] = (int32_t)base_p;
        a.counts[2 * (int64_t)row + 1] = (int32_t)base_d;
    }
}

}  // namespace

hipError_t launch_bkp_hits(const BkpArgs& a, int rows, hipStream_t st)
{
    if (a.k < 1) return hipSuccess;
    hipLaunchKernelGGL(bkp_hits_kernel, dim3((a.k + 255) / 256, rows), dim3(256), 0, st, a);
    return hipGetLastError();
}

hipError_t launch_bkp_rank(const BkpArgs& a, int rows, hipStream_t st)
{
    hipLaunchKernelGGL(bkp_rank_kernel, dim3((a.n + 255) / 256, rows), dim3(256), 0, st, a);
    return hipGetLastError();
}

hipError_t launch_bkp_mark(const BkpArgs& a, int rows, hipStream_t st)
{
    if (a.f < 1) return hipSuccess;
    hipLaunchKernelGGL(bkp_mark_kernel, dim3((a.f + 255) / 256, rows), dim3(256), 0, st, a);
    return hipGetLastError();
}

hipError_t launch_bkp_lists(const BkpArgs& a, int rows, hipStream_t st)
{
    hipLaunchKernelGGL(bkp_lists_kernel, dim3(rows), dim3(256), 0, st, a);
    return hipGetLastError();
}

}  // namespace hill
