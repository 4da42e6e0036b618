// Bidirectional KV Cache Pools (Sec. 4.2, HKM / BKP) on gfx950: the per-token
// hit-rate table and the hot/cold pool policy, one pass after each decoding
// step.  Six launches, each parallel over the row's tokens:
//
//  bkp_hits    one hit for every token of the step's selected set (2-byte
//              counters, saturating; indices are unique within a row, so each
//              counter has one writer); also clears the selection histograms
//  bkp_rank    per token the value the frequency slots are chosen by:
//              2 * hits + (hot before the call), then a position bin, -1
//              inside the recent window (integers, exact in fp32), and the
//              first-digit histogram of those values for the library's exact
//              top-k (ties to the lower index)
//  refine, emit (topk.hip) the chosen tokens, listed per 512-token chunk
//  bkp_count   per chunk: how many tokens become hot / cold
//  bkp_write   per chunk: the new pool bytes, and the promotions and
//              demotions written in token order after the earlier chunks'
#include "hill_device.h"
#include "hill_internal.h"

namespace hill {

namespace {

static_assert(kSelChunk == 512, "one chunk is 256 threads x 2 tokens");

__global__ __launch_bounds__(256) void bkp_hits_kernel(BkpArgs a)
{
    const int64_t nblocks = (int64_t)gridDim.x * gridDim.y;
    const int64_t bid = (int64_t)blockIdx.y * gridDim.x + blockIdx.x;
    for (int64_t i = bid * 256 + threadIdx.x; i < a.zero_words; i += nblocks * 256) a.zero[i] = 0u;
    const int row = blockIdx.y;
    const int i = blockIdx.x * 256 + threadIdx.x;
    if (i >= a.k) return;
    const int j = a.idx[(int64_t)row * a.k + i];
    if ((unsigned)j >= (unsigned)a.n) return;
    uint16_t* h = a.hits + a.off(row) + j;
    const uint16_t x = *h;
    if (x != 0xffffu) *h = (uint16_t)(x + 1u);
}

constexpr int kRankChunk = 512;   // tokens per rank workgroup
// Position bins folded into the rank value below the (hits, incumbency) part:
// lower token index, larger value.  The order is the one the exact top-k's
// lower-index tie rule gives anyway, but tokens with equal hits no longer tie
// across the whole row (which would send the selection down its slow path);
// (2 * 65535 + 1) * 128 + 127 < 2^24 keeps every value exact in fp32.
constexpr uint32_t kPosBins = 128;

__global__ __launch_bounds__(256) void bkp_rank_kernel(BkpArgs a)
{
    __shared__ uint32_t bins[kHistRow];
    __shared__ uint32_t list[kHistRow];
    __shared__ uint32_t nlist;
    const int row = blockIdx.y;
    for (int i = threadIdx.x; i < kHistRow; i += 256) bins[i] = 0u;
    if (threadIdx.x == 0) nlist = 0u;
    const int64_t o = a.off(row);
    float* v = a.v + (int64_t)row * a.ld;
    uint32_t kk[kRankChunk / 256];
    bool in[kRankChunk / 256];
#pragma unroll
    for (int u = 0; u < kRankChunk / 256; ++u) {
        const int j = blockIdx.x * kRankChunk + u * 256 + threadIdx.x;
        in[u] = j < a.n;
        if (in[u]) {
            const uint32_t old = a.hot[o + j] & 1u;   // only bit 0 carries state between calls
            const uint32_t pos = kPosBins - 1u - ((uint32_t)j >> a.pos_shift);
            const float x = j >= a.n - a.w ? -1.0f : (float)((2u * a.hits[o + j] + old) * kPosBins + pos);
            v[j] = x;
            kk[u] = order_key(x);
        }
    }
    __syncthreads();
#pragma unroll
    for (int u = 0; u < kRankChunk / 256; ++u) {
        if (in[u]) {
            hist_add(bins, list, &nlist, kk[u] >> (32 - kHistBits));
            hist_add(bins, list, &nlist, kHistBins + (kk[u] >> 26));
        }
    }
    __syncthreads();
    hist_flush(bins, list, nlist, a.hist1 + (int64_t)row * kHistRow);
}

// Hot-now bits of this thread's two tokens of chunk c, from the chunk's
// chosen list (when there are frequency slots) and the recent window.
__device__ __forceinline__ uint32_t chunk_flags(const BkpArgs& a, int row, int c, uint32_t* chosen,
                                                uint32_t (&now)[2], uint32_t (&was)[2], int (&j)[2])
{
    if (threadIdx.x < kSelChunk / 32) chosen[threadIdx.x] = 0u;
    __syncthreads();
    if (a.f > 0) {
        const uint32_t cnt = a.sel_n[(int64_t)row * a.nchunks + c];
        const int32_t* sl = a.sel_list + (int64_t)row * a.n + (int64_t)c * kSelChunk;
        for (uint32_t i = threadIdx.x; i < cnt; i += 256) {
            const int t = sl[i] - c * kSelChunk;
            atomicOr(&chosen[t >> 5], 1u << (t & 31));
        }
    }
    __syncthreads();
    const uint8_t* hot = a.hot + a.off(row);
    uint32_t moves = 0;
#pragma unroll
    for (int e = 0; e < 2; ++e) {
        j[e] = c * kSelChunk + 2 * threadIdx.x + e;
        was[e] = now[e] = 0u;
        if (j[e] < a.n) {
            const int t = j[e] - c * kSelChunk;
            was[e] = hot[j[e]] & 1u;
            now[e] = (j[e] >= a.n - a.w || ((chosen[t >> 5] >> (t & 31)) & 1u)) ? 1u : 0u;
            moves |= (now[e] && !was[e] ? 1u : 0u) << (2 * e);
            moves |= (was[e] && !now[e] ? 2u : 0u) << (2 * e);
        }
    }
    return moves;
}

__global__ __launch_bounds__(256) void bkp_count_kernel(BkpArgs a)
{
    __shared__ uint32_t chosen[kSelChunk / 32];
    __shared__ uint2 scratch[256 / 64 + 1];
    const int c = blockIdx.x, row = blockIdx.y;
    uint32_t now[2], was[2];
    int j[2];
    const uint32_t m = chunk_flags(a, row, c, chosen, now, was, j);
    uint2 v = make_uint2(((m >> 0) & 1u) + ((m >> 2) & 1u), ((m >> 1) & 1u) + ((m >> 3) & 1u));
    uint2 tot;
    block_excl_scan2<256>(v, scratch, &tot);
    if (threadIdx.x == 0) a.chunk_moves[(int64_t)row * a.nchunks + c] = tot;
}

__global__ __launch_bounds__(256) void bkp_write_kernel(BkpArgs a)
{
    __shared__ uint32_t chosen[kSelChunk / 32];
    __shared__ uint2 scratch[256 / 64 + 1];
    __shared__ uint2 base_s;
    const int c = blockIdx.x, row = blockIdx.y;
    // moves of the earlier chunks (and, in chunk 0, of all chunks for the counts)
    const uint2* cm = a.chunk_moves + (int64_t)row * a.nchunks;
    const int upto = c == 0 ? a.nchunks : c;
    uint2 s = make_uint2(0u, 0u);
    for (int i = threadIdx.x; i < upto; i += 256) {
        const uint2 x = cm[i];
        s.x += x.x;
        s.y += x.y;
    }
    uint2 all;
    block_excl_scan2<256>(s, scratch, &all);
    if (threadIdx.x == 0) {
        base_s = c == 0 ? make_uint2(0u, 0u) : all;
        if (c == 0) {
            a.counts[2 * (int64_t)row] = (int32_t)all.x;
            a.counts[2 * (int64_t)row + 1] = (int32_t)all.y;
        }
    }
    uint32_t now[2], was[2];
    int j[2];
    const uint32_t m = chunk_flags(a, row, c, chosen, now, was, j);   // its barriers also publish base_s
    uint2 v = make_uint2(((m >> 0) & 1u) + ((m >> 2) & 1u), ((m >> 1) & 1u) + ((m >> 3) & 1u));
    uint2 tot;
    uint2 off = block_excl_scan2<256>(v, scratch, &tot);
    const uint2 base = base_s;
    uint8_t* hot = a.hot + a.off(row);
    int32_t* pro = a.promote + (int64_t)row * a.list_cap;
    int32_t* dem = a.demote + (int64_t)row * a.list_cap;
#pragma unroll
    for (int e = 0; e < 2; ++e) {
        if (j[e] >= a.n) continue;
        hot[j[e]] = (uint8_t)now[e];   // 0 or 1, whatever else the byte held
        if ((m >> (2 * e)) & 1u) {
            const uint32_t p = base.x + off.x++;
            if (p < (uint32_t)a.list_cap) pro[p] = j[e];
        } else if ((m >> (2 * e)) & 2u) {
            const uint32_t p = base.y + off.y++;
            if (p < (uint32_t)a.list_cap) dem[p] = j[e];
        }
    }
}

}  // namespace

hipError_t launch_bkp_hits(const BkpArgs& a, int rows, hipStream_t st)
{
    const int gx = a.k > 0 ? (a.k + 255) / 256 : 1;   // launched even without hits: it clears the histograms
    hipLaunchKernelGGL(bkp_hits_kernel, dim3(gx, rows), dim3(256), 0, st, a);
    return hipGetLastError();
}

hipError_t launch_bkp_rank(const BkpArgs& a, int rows, hipStream_t st)
{
    hipLaunchKernelGGL(bkp_rank_kernel, dim3((a.n + kRankChunk - 1) / kRankChunk, rows), dim3(256), 0, st, a);
    return hipGetLastError();
}

hipError_t launch_bkp_lists(const BkpArgs& a, int rows, hipStream_t st)
{
    hipLaunchKernelGGL(bkp_count_kernel, dim3(a.nchunks, rows), dim3(256), 0, st, a);
    hipLaunchKernelGGL(bkp_write_kernel, dim3(a.nchunks, rows), dim3(256), 0, st, a);
    return hipGetLastError();
}

}  // namespace hill
