// Importance scoring on gfx950.
//
//  score_tiles   streams every cached key row once and forms the raw logits
//                q.K^T of all query heads that share it (GQA group)
//                (Sec. 4.4 raw inner product; Eq. 1).  ATTN keeps the logits
//                and, per 256-token unit, a (max, sum of exp2) pair per head;
//                RAW sums each head group per token.
//
// The importance update that consumes the logits is in update.hip.
//
// score_tiles layout.  A key row is 256 bytes (D = 128 x 16 bit).  Eight
// lanes share a row: lane l8 reads elements [8*l8, 8*l8+8) with one 16-byte
// load and [64+8*l8, 64+8*l8+8) with a second, so each load instruction of a
// wave covers whole 128-byte lines of 8 rows.  A wave-tile is 32 consecutive
// tokens of one (sequence, KV head): row group rg (lanes 8*rg .. 8*rg+7) owns
// tokens j0 + 4*rg .. j0 + 4*rg + 3.  A workgroup unit is 8 wave-tiles (256
// tokens; each wave takes two); the tiles' pairs are merged in LDS into one
// pair per head.  Queries stay in registers while (b, g) stays the same.
// Latency is hidden by occupancy (four workgroups per CU) rather than by
// double-buffering, which costs more registers than it returns.  Partial dot
// products are combined by three DPP adds.  ATTN logits with G >= 4 heads per
// KV head take the dots on the matrix cores instead (KeysF16Mfma: the same
// tiles, units and whole-line loads, a different lane-to-element map).
#include <hip/hip_ext.h>

#include <type_traits>

#include "hill_device.h"
#include "hill_internal.h"

namespace hill {

namespace {

constexpr int kRowsPerLane = kScoreTile / 8;   // 4 rows per row group

__global__ __launch_bounds__(256) void fill_zero_kernel(uint32_t* p, int64_t words)
{
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < words;
         i += (int64_t)gridDim.x * blockDim.x)
        p[i] = 0u;
}

struct TileCoord {
    int b, g, tile, j0;
};

__device__ __forceinline__ TileCoord coord(const ScoreArgs& a, int t)
{
    TileCoord c;
    c.tile = t % a.ntiles;
    const int bg = t / a.ntiles;
    c.g = bg % a.Hkv;
    c.b = bg / a.Hkv;
    c.j0 = c.tile * kScoreTile;
    return c;
}

// Key sources of the scan.  Each provides: load(a, c, rg, l8) -- issue the
// tile's key loads of this lane; query(a, c, hc, l8) -- make the queries of
// heads hc .. hc+GC of group (c.b, c.g) ready (kept while the group stays the
// same); dot(a, u, hh, l8) -- the raw logit q_hh . K_row of this lane's row u,
// complete in every lane of the 8-lane row group.

// 16-bit keys: lane l8 holds elements [8*l8, 8*l8+8) and [64+8*l8, 64+8*l8+8)
// of each of its 4 rows (two 16-byte non-temporal loads per row).
template <int DT, int GC>
struct KeysF16 {
    // tiles whose loads are in flight together: two where the queries take few
    // registers (G <= 2 heads per pass keeps 4 workgroups per CU), else one
    static constexpr int kSlots = GC <= 2 ? 2 : 1;
    static constexpr bool kGroupQuery = false;
    static constexpr bool kIntDot = false;
    static constexpr bool kMfmaSplit = false;
    uint4 kr[kSlots][2 * kRowsPerLane];
    uint4 qa[GC], qb[GC];
    int q_tag = -1;

    template <int SLOT>
    __device__ __forceinline__ void load(const ScoreArgs& a, const TileCoord& c, int rg, int l8)
    {
        const uint16_t* kb = a.k + (int64_t)c.b * a.k_sb + (int64_t)c.g * a.k_sh + l8 * 8;
#pragma unroll
        for (int u = 0; u < kRowsPerLane; ++u) {
            const int j = c.j0 + rg * kRowsPerLane + u;
            if (j < a.n) {
                const uint16_t* row = kb + (int64_t)j * a.k_sn;
                kr[SLOT][2 * u] = load_stream16(row);
                kr[SLOT][2 * u + 1] = load_stream16(row + 64);
            } else {
                kr[SLOT][2 * u] = make_uint4(0u, 0u, 0u, 0u);
                kr[SLOT][2 * u + 1] = make_uint4(0u, 0u, 0u, 0u);
            }
        }
    }

    __device__ __forceinline__ void query(const ScoreArgs& a, const TileCoord& c, int hc, int l8)
    {
        const int tag = (c.b * a.Hkv + c.g) * a.G + hc;
        if (tag == q_tag) return;
#pragma unroll
        for (int hh = 0; hh < GC; ++hh) {
            const uint16_t* qr = a.q + (int64_t)c.b * a.q_sb + (int64_t)(c.g * a.G + hc + hh) * a.q_sh + l8 * 8;
            qa[hh] = *reinterpret_cast<const uint4*>(qr);
            qb[hh] = *reinterpret_cast<const uint4*>(qr + 64);
        }
        q_tag = tag;
    }

    template <int SLOT>
    __device__ __forceinline__ float dot(const ScoreArgs&, int u, int hh, int) const
    {
        float d = dot8<DT>(kr[SLOT][2 * u], qa[hh]);
        d += dot8<DT>(kr[SLOT][2 * u + 1], qb[hh]);
        return sum8(d);
    }
};

// Key sketch (Sec. 4.4 asymmetric precision), BITS = 8 or 4: lane l8 holds
// codes [16*l8, 16*l8+16) of each of its 4 rows (one 16-byte load per row for
// int8, one 8-byte load for int4) and the rows' exponents.  An int4 row packs
// each group of 8 codes into one word: byte i holds code i + 8 in its low
// nibble and code i+4 + 8 in its high nibble, so two masks give four int8
// lanes in element order, and the +8 offset is taken off as 8 * (sum of the
// query codes).  The queries of the group are cast to int8 (power-of-two
// scale per head, round to nearest even) once per workgroup when the group
// changes: wave w casts heads w, w+4, ... into LDS (group_query), and every
// wave reads its slices from there (query).  The dot product is exact in
// int32 (|sum| < 2^24) and scaled by 2^(e_q + e_k).
struct QueryLds {
    int8_t q8[kMaxGroup][kHeadDim];
    int eq[kMaxGroup];
};

// The queries of a key-sketch scan: cast once per (b, g) into LDS.
template <int DT>
struct SketchQuery {
    QueryLds* ql = nullptr;
    int q_tag = -1;

    // The raw query words of the group's first heads (wave w: heads w and
    // w + 4, lane l: elements 2l, 2l+1), fetched before the key loads so that
    // the cast waits only for them.
    static constexpr int kQPre = 2;
    uint32_t qpre[kQPre];

    __device__ __forceinline__ const uint32_t* qword(const ScoreArgs& a, int b, int g, int h, int lane) const
    {
        return reinterpret_cast<const uint32_t*>(a.q + (int64_t)b * a.q_sb + (int64_t)(g * a.G + h) * a.q_sh +
                                                 2 * lane);
    }

    __device__ __forceinline__ void group_query_fetch(const ScoreArgs& a, int b, int g, int w, int lane)
    {
#pragma unroll
        for (int i = 0; i < kQPre; ++i) {
            const int h = w + 4 * i;
            qpre[i] = h < a.G ? *qword(a, b, g, h, lane) : 0u;
        }
    }

    __device__ __forceinline__ void cast_head(uint32_t word, int h, int lane)
    {
        float x0, x1;
        widen2<DT>(word, x0, x1);
        const int e = sketch_exponent<127>(wave_max(fmaxf(fabsf(x0), fabsf(x1))));
        const uint32_t c2 =
            ((uint32_t)sketch_code<127>(x0, e) & 0xffu) | (((uint32_t)sketch_code<127>(x1, e) & 0xffu) << 8);
        *reinterpret_cast<uint16_t*>(&ql->q8[h][2 * lane]) = (uint16_t)c2;
        if (lane == 0) ql->eq[h] = e;
    }

    // Casts the G queries of group (b, g) into ql; wave w takes heads w, w+4, ...
    // (the first kQPre of them from group_query_fetch).  Called by every wave;
    // the caller orders it with a barrier before the reads.
    __device__ __forceinline__ void group_query(const ScoreArgs& a, int b, int g, int w, int lane)
    {
#pragma unroll
        for (int i = 0; i < kQPre; ++i)
            if (w + 4 * i < a.G) cast_head(qpre[i], w + 4 * i, lane);
        for (int h = w + 4 * kQPre; h < a.G; h += 4) cast_head(*qword(a, b, g, h, lane), h, lane);
        q_tag = -1;
    }

};

template <int DT, int GC, int BITS>
struct KeysSketch : SketchQuery<DT> {
    static_assert(BITS == 8 || BITS == 4, "int8 or int4 key codes");
    static constexpr int kSlots = 2;   // a wave's two tiles of a unit are loaded together
    static constexpr bool kGroupQuery = true;
    static constexpr bool kIntDot = true;   // idot + scale: one conversion per row for the lane's head
    static constexpr bool kMfmaSplit = false;
    static constexpr int kRowBytes = kHeadDim * BITS / 8;
    using Codes = typename std::conditional<BITS == 8, uint4, uint2>::type;
    using SketchQuery<DT>::ql;
    using SketchQuery<DT>::q_tag;
    Codes kr[kSlots][kRowsPerLane];
    uint32_t ek4[kSlots];   // exponents of the 4 rows, one byte each
    uint4 q8[GC];
    int eq[GC];
    int qbias[GC];          // int4: 8 * (sum of this lane's 16 query codes)
    int eq_lane = 0;        // exponent of this lane's head (lane l8 < GC holds head l8 of the chunk)

    template <int SLOT>
    __device__ __forceinline__ void load(const ScoreArgs& a, const TileCoord& c, int rg, int l8)
    {
        const int64_t bg = (int64_t)c.b * a.Hkv + c.g;
        const int jr = c.j0 + rg * kRowsPerLane;
        const int8_t* kb = a.k8 + bg * a.cap * kRowBytes + l8 * (kRowBytes / 8);
#pragma unroll
        for (int u = 0; u < kRowsPerLane; ++u) {
            const int j = jr + u;
            if constexpr (BITS == 8) {
                kr[SLOT][u] = j < a.n ? load_stream16(kb + (int64_t)j * kRowBytes) : make_uint4(0u, 0u, 0u, 0u);
            } else {
                kr[SLOT][u] = j < a.n ? load_stream8(kb + (int64_t)j * kRowBytes) : make_uint2(0u, 0u);
            }
        }
        // jr is a multiple of 4 and cap too: the 4 exponents are one aligned word inside the row
        ek4[SLOT] = jr < a.n ? *reinterpret_cast<const uint32_t*>(a.k_exp + bg * a.cap + jr) : 0u;
    }

    __device__ __forceinline__ void query(const ScoreArgs& a, const TileCoord& c, int hc, int l8)
    {
        const int tag = (c.b * a.Hkv + c.g) * a.G + hc;
        if (tag == q_tag) return;
#pragma unroll
        for (int hh = 0; hh < GC; ++hh) {
            q8[hh] = *reinterpret_cast<const uint4*>(&ql->q8[hc + hh][16 * l8]);
            eq[hh] = ql->eq[hc + hh];
            if constexpr (BITS == 4) {
                const int ones = 0x01010101;
                int sq = __builtin_amdgcn_sdot4((int)q8[hh].x, ones, 0, false);
                sq = __builtin_amdgcn_sdot4((int)q8[hh].y, ones, sq, false);
                sq = __builtin_amdgcn_sdot4((int)q8[hh].z, ones, sq, false);
                sq = __builtin_amdgcn_sdot4((int)q8[hh].w, ones, sq, false);
                qbias[hh] = 8 * sq;
            }
        }
        eq_lane = ql->eq[hc + (l8 < GC ? l8 : 0)];   // from LDS: a register-array pick would be indexed
        q_tag = tag;
    }

    // Exact integer q . k of row u for head hh, complete in every lane of the row group.
    template <int SLOT>
    __device__ __forceinline__ int idot(int u, int hh) const
    {
        int d;
        if constexpr (BITS == 8) {
            const uint4 k = kr[SLOT][u];
            d = __builtin_amdgcn_sdot4((int)k.x, (int)q8[hh].x, 0, false);
            d = __builtin_amdgcn_sdot4((int)k.y, (int)q8[hh].y, d, false);
            d = __builtin_amdgcn_sdot4((int)k.z, (int)q8[hh].z, d, false);
            d = __builtin_amdgcn_sdot4((int)k.w, (int)q8[hh].w, d, false);
        } else {
            // codes + 8 in [1, 15]: low nibbles are elements 0..3 of a group, high nibbles 4..7
            const uint2 k = kr[SLOT][u];
            const uint32_t m = 0x0F0F0F0Fu;
            d = __builtin_amdgcn_sdot4((int)(k.x & m), (int)q8[hh].x, -qbias[hh], false);
            d = __builtin_amdgcn_sdot4((int)((k.x >> 4) & m), (int)q8[hh].y, d, false);
            d = __builtin_amdgcn_sdot4((int)(k.y & m), (int)q8[hh].z, d, false);
            d = __builtin_amdgcn_sdot4((int)((k.y >> 4) & m), (int)q8[hh].w, d, false);
        }
        return isum8(d);
    }

    // The logit of an integer dot of row u for this lane's head: d * 2^(e_q + e_k), exact.
    template <int SLOT>
    __device__ __forceinline__ float scale(int d, int u) const
    {
        const int ek = (int)(int8_t)(ek4[SLOT] >> (8 * u));
        return ldexpf((float)d, eq_lane + ek);
    }

    template <int SLOT>
    __device__ __forceinline__ float dot(const ScoreArgs&, int u, int hh, int) const
    {
        const int ek = (int)(int8_t)(ek4[SLOT] >> (8 * u));
        return ldexpf((float)idot<SLOT>(u, hh), eq[hh] + ek);
    }
};

typedef int i32x4_t __attribute__((ext_vector_type(4)));

// 16-bit keys on the matrix cores (ATTN logits, G >= 4): the dot products as
// v_mfma_f32_16x16x32_{bf16,f16}, D[row][col] = sum_k A[row][k] B[k][col].
// A row of the 16-row operand is half a key row: row 4q + 2u + p of group gr
// (gr = 0..3) holds the 16-byte chunks of parity p (chunks 2m + p of the 16 in
// the 256-byte row) of token 8q + 4u + gr of the tile; lane l (row l % 16,
// quarter c = l / 16) loads chunk 8s + 2c + p for line s = 0, 1 (one MFMA per
// line).  The 8 lanes of a token thus read its whole 128-byte line s in one
// load instruction.  Column 2h + p' of the query operand holds the parity-p'
// chunks of head hc + h (8 heads per pass, zero beyond G), in the same order,
// so D[(t, p)][(h, p)] is the parity-p half of q_h . K_t and the two halves
// sit in neighbouring lanes (columns 2h, 2h + 1) of the same output row pair.
// One DPP add joins them: even lanes finish token 8q + gr, odd lanes token
// 8q + 4 + gr (q = l / 16), so over the four groups a lane holds 4
// consecutive tokens of its head and stores them as one float4.
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef _Float16 f16x8_t __attribute__((ext_vector_type(8)));

template <int DT>
__device__ __forceinline__ f32x4_t mfma16(const uint4& a, const uint4& b, f32x4_t acc)
{
    if constexpr (DT == 1)
        return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, a),
                                                       __builtin_bit_cast(bf16x8_t, b), acc, 0, 0, 0);
    else
        return __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(f16x8_t, a), __builtin_bit_cast(f16x8_t, b),
                                                      acc, 0, 0, 0);
}

constexpr int kMfmaHeads = 8;   // heads per pass of KeysF16Mfma (two columns each)

template <int DT>
struct KeysF16Mfma {
    static constexpr int kSlots = 1;
    static constexpr bool kGroupQuery = false;
    static constexpr bool kIntDot = false;
    static constexpr bool kMfmaSplit = true;
    uint4 kr[kSlots][8];   // [tile][2 * group + line]: the lane's 16-byte chunk
    uint4 qb[2];           // query operand per line (column l % 16)
    int q_tag = -1;

    template <int SLOT>
    __device__ __forceinline__ void load(const ScoreArgs& a, const TileCoord& c, int rg, int l8)
    {
        const int lane = rg * 8 + l8;
        const int i = lane & 15, q = i >> 2, u = (i >> 1) & 1, p = i & 1;
        const uint16_t* kb = a.k + (int64_t)c.b * a.k_sb + (int64_t)c.g * a.k_sh + (2 * (lane >> 4) + p) * 8;
#pragma unroll
        for (int gr = 0; gr < 4; ++gr) {
            const int j = c.j0 + 8 * q + 4 * u + gr;
            const uint16_t* row = kb + (int64_t)j * a.k_sn;
#pragma unroll
            for (int s = 0; s < 2; ++s)
                kr[SLOT][2 * gr + s] = j < a.n ? load_stream16(row + 64 * s) : make_uint4(0u, 0u, 0u, 0u);
        }
    }

    // Query operand of heads hc .. hc+7: column 2h + p' of lane l = l % 16 holds
    // the chunks 8s + 2c + p' (c = l / 16) of head hc + h, zero beyond G.
    __device__ __forceinline__ void mquery(const ScoreArgs& a, const TileCoord& c, int hc, int lane)
    {
        const int tag = (c.b * a.Hkv + c.g) * a.G + hc;
        if (tag == q_tag) return;
        const int col = lane & 15, h = hc + (col >> 1);
        const int e0 = (2 * (lane >> 4) + (col & 1)) * 8;
        const uint16_t* qr = a.q + (int64_t)c.b * a.q_sb + (int64_t)(c.g * a.G + min(h, a.G - 1)) * a.q_sh + e0;
#pragma unroll
        for (int s = 0; s < 2; ++s)
            qb[s] = h < a.G ? *reinterpret_cast<const uint4*>(qr + 64 * s) : make_uint4(0u, 0u, 0u, 0u);
        q_tag = tag;
    }

    // Raw logits of this lane's 4 tokens (see above) for head hc + (l % 16) / 2.
    template <int SLOT>
    __device__ __forceinline__ void dots(int lane, float (&out)[4]) const
    {
        const bool odd = lane & 1;
#pragma unroll
        for (int gr = 0; gr < 4; ++gr) {
            f32x4_t acc = {0.0f, 0.0f, 0.0f, 0.0f};
            acc = mfma16<DT>(kr[SLOT][2 * gr], qb[0], acc);
            acc = mfma16<DT>(kr[SLOT][2 * gr + 1], qb[1], acc);
            // even lane (p' = 0): its row pair u = 0 half + the odd neighbour's;
            // odd lane (p' = 1): its u = 1 half + the even neighbour's
            const float own = odd ? acc[3] : acc[0];
            const float send = odd ? acc[1] : acc[2];
            out[gr] = own + dpp<0xB1>(send);
        }
    }
};

// Int8 key sketch on the matrix cores (ATTN logits, G >= 4), in the split-row
// layout of KeysF16Mfma: row 4q + 2u + p of group gr holds the 16-byte chunks
// 2c + p (c = 0..3) of token 8q + 4u + gr's 128-byte code row, so one load
// instruction reads 8 whole rows, and each lane's 16 bytes feed two
// v_mfma_i32_16x16x32_i8 (its low and high 8 codes).  The integer halves are
// joined by one DPP add and scaled by 2^(e_q + e_k) as on the vector units:
// the logits are the same exact values.
template <int DT>
struct KeysSketchMfma8 : SketchQuery<DT> {
    static constexpr int kSlots = 2;
    static constexpr bool kGroupQuery = true;
    static constexpr bool kIntDot = true;
    static constexpr bool kMfmaSplit = true;
    using SketchQuery<DT>::ql;
    using SketchQuery<DT>::q_tag;
    uint4 kr[kSlots][4];       // [tile][group]: the lane's 16 code bytes
    uint32_t ek4[kSlots];      // exponents of the lane's 4 output tokens
    uint64_t qb[2];            // query operand of the two MFMAs (column l % 16)
    int eq_lane = 0;           // exponent of the lane's head

    template <int SLOT>
    __device__ __forceinline__ void load(const ScoreArgs& a, const TileCoord& c, int rg, int l8)
    {
        const int lane = rg * 8 + l8;
        const int i = lane & 15, q = i >> 2, u = (i >> 1) & 1, p = i & 1;
        const int64_t bg = (int64_t)c.b * a.Hkv + c.g;
        const int8_t* kb = a.k8 + bg * a.cap * kHeadDim + (2 * (lane >> 4) + p) * 16;
#pragma unroll
        for (int gr = 0; gr < 4; ++gr) {
            const int j = c.j0 + 8 * q + 4 * u + gr;
            kr[SLOT][gr] = j < a.n ? load_stream16(kb + (int64_t)j * kHeadDim) : make_uint4(0u, 0u, 0u, 0u);
        }
        // the output tokens start at a multiple of 4 and cap is one too: one aligned word
        const int jt = c.j0 + 8 * (lane >> 4) + 4 * (lane & 1);
        ek4[SLOT] = jt < a.n ? *reinterpret_cast<const uint32_t*>(a.k_exp + bg * a.cap + jt) : 0u;
    }

    // Query operand of heads hc .. hc+7 (column 2h + p': the codes of chunk
    // 2c + p' of head hc + h, zero beyond G) and the lane's head exponent.
    __device__ __forceinline__ void mquery(const ScoreArgs& a, const TileCoord& c, int hc, int lane)
    {
        const int tag = (c.b * a.Hkv + c.g) * a.G + hc;
        if (tag == q_tag) return;
        const int col = lane & 15, h = hc + (col >> 1);
        uint4 x = make_uint4(0u, 0u, 0u, 0u);
        eq_lane = 0;
        if (h < a.G) {
            x = *reinterpret_cast<const uint4*>(&ql->q8[h][(2 * (lane >> 4) + (col & 1)) * 16]);
            eq_lane = ql->eq[h];
        }
        qb[0] = (uint64_t)x.x | ((uint64_t)x.y << 32);
        qb[1] = (uint64_t)x.z | ((uint64_t)x.w << 32);
        q_tag = tag;
    }

    template <int SLOT>
    __device__ __forceinline__ void dots(int lane, float (&out)[4]) const
    {
        const bool odd = lane & 1;
#pragma unroll
        for (int gr = 0; gr < 4; ++gr) {
            const uint4 k = kr[SLOT][gr];
            i32x4_t acc = {0, 0, 0, 0};
            acc = __builtin_amdgcn_mfma_i32_16x16x32_i8((long)((uint64_t)k.x | ((uint64_t)k.y << 32)), (long)qb[0],
                                                        acc, 0, 0, 0);
            acc = __builtin_amdgcn_mfma_i32_16x16x32_i8((long)((uint64_t)k.z | ((uint64_t)k.w << 32)), (long)qb[1],
                                                        acc, 0, 0, 0);
            const int own = odd ? acc[3] : acc[0];
            const int send = odd ? acc[1] : acc[2];
            const int d = own + __builtin_amdgcn_update_dpp(0, send, 0xB1, 0xF, 0xF, false);
            const int ek = (int)(int8_t)(ek4[SLOT] >> (8 * gr));
            out[gr] = ldexpf((float)d, eq_lane + ek);
        }
    }
};

// Int4 key sketch on the matrix cores (ATTN logits, G >= 4), split-row layout.
// A 64-byte code row packs each group of 8 codes into one word (byte i holds
// code i + 8 in its low nibble and code i+4 + 8 in its high nibble), so two
// masks turn a word into 8 int8 operands in element order.  Row 4q + 2u + p of
// group gr's 16-row operand holds the 16-byte chunks p and p + 2 of token
// 8q + 2gr + u, lane quarter c its 8 bytes at 16p + 8(c & 1) + 32(c >> 1): one
// load instruction reads 8 whole rows, i.e. the 4 whole 128-byte lines of 4
// token pairs.  Column 2h + p' of the query operand holds head hc + h's codes
// in the same order, and each column's accumulator starts at -8 times the sum
// of those codes (the +8 of the key codes).  One DPP add joins a token's two
// halves (even lanes: token 8q + 2gr, odd lanes 8q + 2gr + 1); one DPP
// exchange of two sums per group then leaves 4 consecutive tokens per lane
// (even lanes 8q .. +3, odd lanes 8q + 4 .. +7), scaled by 2^(e_q + e_k) as on
// the vector units: the same exact logits.
template <int DT>
struct KeysSketchMfma4 : SketchQuery<DT> {
    static constexpr int kSlots = 2;
    static constexpr bool kGroupQuery = true;
    static constexpr bool kIntDot = true;
    static constexpr bool kMfmaSplit = true;
    static constexpr int kRowBytes = kHeadDim / 2;
    using SketchQuery<DT>::ql;
    using SketchQuery<DT>::q_tag;
    uint2 kr[kSlots][4];       // [tile][group]: the lane's 8 code bytes (two words)
    uint32_t ek4[kSlots];      // exponents of the lane's 4 output tokens
    uint64_t qb[2];            // query operand of the two MFMAs (column l % 16)
    int eq_lane = 0;           // exponent of the lane's head
    int bias = 0;              // 8 * (sum of the column's 64 query codes)

    template <int SLOT>
    __device__ __forceinline__ void load(const ScoreArgs& a, const TileCoord& c, int rg, int l8)
    {
        const int lane = rg * 8 + l8;
        const int i = lane & 15, q = i >> 2, u = (i >> 1) & 1, p = i & 1, qc = lane >> 4;
        const int64_t bg = (int64_t)c.b * a.Hkv + c.g;
        const int8_t* kb = a.k8 + bg * a.cap * kRowBytes + 16 * p + 8 * (qc & 1) + 32 * (qc >> 1);
#pragma unroll
        for (int gr = 0; gr < 4; ++gr) {
            const int j = c.j0 + 8 * q + 2 * gr + u;
            kr[SLOT][gr] = j < a.n ? load_stream8(kb + (int64_t)j * kRowBytes) : make_uint2(0u, 0u);
        }
        // the output tokens start at a multiple of 4 and cap is one too: one aligned word
        const int jt = c.j0 + 8 * qc + 4 * (lane & 1);
        ek4[SLOT] = jt < a.n ? *reinterpret_cast<const uint32_t*>(a.k_exp + bg * a.cap + jt) : 0u;
    }

    __device__ __forceinline__ void mquery(const ScoreArgs& a, const TileCoord& c, int hc, int lane)
    {
        const int tag = (c.b * a.Hkv + c.g) * a.G + hc;
        if (tag == q_tag) return;
        const int col = lane & 15, h = hc + (col >> 1), qc = lane >> 4;
        uint4 x = make_uint4(0u, 0u, 0u, 0u);
        eq_lane = 0;
        if (h < a.G) {
            // codes of the lane's key bytes: 2 per byte, at 2 * (16p' + 8(c & 1) + 32(c >> 1))
            x = *reinterpret_cast<const uint4*>(&ql->q8[h][32 * (col & 1) + 16 * (qc & 1) + 64 * (qc >> 1)]);
            eq_lane = ql->eq[h];
        }
        qb[0] = (uint64_t)x.x | ((uint64_t)x.y << 32);
        qb[1] = (uint64_t)x.z | ((uint64_t)x.w << 32);
        const int ones = 0x01010101;
        int sq = __builtin_amdgcn_sdot4((int)x.x, ones, 0, false);
        sq = __builtin_amdgcn_sdot4((int)x.y, ones, sq, false);
        sq = __builtin_amdgcn_sdot4((int)x.z, ones, sq, false);
        sq = __builtin_amdgcn_sdot4((int)x.w, ones, sq, false);
        sq += __shfl_xor(sq, 16, 64);
        sq += __shfl_xor(sq, 32, 64);
        bias = 8 * sq;
        q_tag = tag;
    }

    template <int SLOT>
    __device__ __forceinline__ void dots(int lane, float (&out)[4]) const
    {
        const bool odd = lane & 1;
        const uint32_t m = 0x0F0F0F0Fu;
        int v[4];
#pragma unroll
        for (int gr = 0; gr < 4; ++gr) {
            const uint2 k = kr[SLOT][gr];
            i32x4_t acc = {-bias, -bias, -bias, -bias};
            acc = __builtin_amdgcn_mfma_i32_16x16x32_i8(
                (long)((uint64_t)(k.x & m) | ((uint64_t)((k.x >> 4) & m) << 32)), (long)qb[0], acc, 0, 0, 0);
            acc = __builtin_amdgcn_mfma_i32_16x16x32_i8(
                (long)((uint64_t)(k.y & m) | ((uint64_t)((k.y >> 4) & m) << 32)), (long)qb[1], acc, 0, 0, 0);
            const int own = odd ? acc[3] : acc[0];
            const int send = odd ? acc[1] : acc[2];
            v[gr] = own + __builtin_amdgcn_update_dpp(0, send, 0xB1, 0xF, 0xF, false);
        }
        // even lanes hold tokens 0, 2, 4, 6 of the lane's 8 (q = l / 16), odd lanes 1, 3, 5, 7
        const int ra = __builtin_amdgcn_update_dpp(0, odd ? v[0] : v[2], 0xB1, 0xF, 0xF, false);
        const int rb = __builtin_amdgcn_update_dpp(0, odd ? v[1] : v[3], 0xB1, 0xF, 0xF, false);
        const int d[4] = {odd ? ra : v[0], odd ? v[2] : ra, odd ? rb : v[1], odd ? v[3] : rb};
#pragma unroll
        for (int t = 0; t < 4; ++t) {
            const int ek = (int)(int8_t)(ek4[SLOT] >> (8 * t));
            out[t] = ldexpf((float)d[t], eq_lane + ek);
        }
    }
};

// One wave-tile of KeysF16Mfma (ATTN): lane l holds head hc + (l % 16) / 2
// for tokens j0 + 8*(l/16) + 4*(l & 1) .. +3; the head's 32 tokens sit in
// lanes l ^ 1, l ^ 16, l ^ 32.
template <int SLOT, typename Keys>
__device__ __forceinline__ void compute_tile_mfma16(const ScoreArgs& a, const TileCoord& c, int lane, Keys& ks,
                                                    float2* tile_part)
{
    const int jt = c.j0 + 8 * (lane >> 4) + 4 * (lane & 1);   // this lane's first token
    for (int hc = 0; hc < a.G; hc += kMfmaHeads) {
        ks.mquery(a, c, hc, lane);
        const int h = hc + ((lane & 15) >> 1);
        float mine[4], x[4];
        ks.template dots<SLOT>(lane, mine);
        float m = -INFINITY;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            x[i] = jt + i < a.n ? a.s2 * mine[i] : -INFINITY;
            m = fmaxf(m, x[i]);
        }
        if (h < a.G) {
            float* lrow = a.logits + ((int64_t)c.b * a.Hq + c.g * a.G + h) * a.ld + jt;
            if (jt + 4 <= a.n) {
                const float4 v4 = make_float4(mine[0], mine[1], mine[2], mine[3]);
                if (a.nt_logits) store_stream16(lrow, v4);
                else *reinterpret_cast<float4*>(lrow) = v4;
            } else {
#pragma unroll
                for (int i = 0; i < 4; ++i)
                    if (jt + i < a.n) lrow[i] = mine[i];
            }
        }
        m = fmaxf(m, dpp<0xB1>(m));
        m = fmaxf(m, __shfl_xor(m, 16, 64));
        m = fmaxf(m, __shfl_xor(m, 32, 64));
        float z = 0.0f;
#pragma unroll
        for (int i = 0; i < 4; ++i) z += jt + i < a.n ? exp2_ftz(x[i] - m) : 0.0f;
        z += dpp<0xB1>(z);
        z += __shfl_xor(z, 16, 64);
        z += __shfl_xor(z, 32, 64);
        if (lane < 16 && !(lane & 1) && h < a.G) tile_part[h] = make_float2(m, z);
    }
}

template <int GC, int OUT, int SLOT, typename Keys>
__device__ __forceinline__ void compute_tile(const ScoreArgs& a, const TileCoord& c, int rg, int l8, Keys& ks,
                                             float2* tile_part)
{
    const int jr = c.j0 + rg * kRowsPerLane;   // first token of this row group
    float rawsum[kRowsPerLane];
#pragma unroll
    for (int u = 0; u < kRowsPerLane; ++u) rawsum[u] = 0.0f;

    for (int hc = 0; hc < a.G; hc += GC) {
        ks.query(a, c, hc, l8);
        float mine[kRowsPerLane];   // lane l8 == hh keeps head hh's logits
        if constexpr (OUT == kOutLogits && Keys::kIntDot) {
            // integer dots: each lane keeps its own head's sum and scales only that one
#pragma unroll
            for (int u = 0; u < kRowsPerLane; ++u) {
                int mi = 0;
#pragma unroll
                for (int hh = 0; hh < GC; ++hh) {
                    const int d = ks.template idot<SLOT>(u, hh);
                    mi = (l8 == hh) ? d : mi;
                }
                mine[u] = ks.template scale<SLOT>(mi, u);
            }
        } else {
#pragma unroll
            for (int u = 0; u < kRowsPerLane; ++u) {
                mine[u] = 0.0f;
#pragma unroll
                for (int hh = 0; hh < GC; ++hh) {
                    const float d = ks.template dot<SLOT>(a, u, hh, l8);
                    if constexpr (OUT == kOutLogits)
                        mine[u] = (l8 == hh) ? d : mine[u];
                    else
                        rawsum[u] += d;
                }
            }
        }
        if constexpr (OUT == kOutLogits) {
            const int h = c.g * a.G + hc + l8;   // valid for l8 < GC
            float* lrow = a.logits + ((int64_t)c.b * a.Hq + h) * a.ld + jr;
            float x[kRowsPerLane];
            float m = -INFINITY;
#pragma unroll
            for (int u = 0; u < kRowsPerLane; ++u) {
                x[u] = jr + u < a.n ? a.s2 * mine[u] : -INFINITY;
                m = fmaxf(m, x[u]);
            }
            if (l8 < GC) {
                if (jr + kRowsPerLane <= a.n) {
                    const float4 v4 = make_float4(mine[0], mine[1], mine[2], mine[3]);
                    if (a.nt_logits) store_stream16(lrow, v4);
                    else *reinterpret_cast<float4*>(lrow) = v4;
                } else {
#pragma unroll
                    for (int u = 0; u < kRowsPerLane; ++u)
                        if (jr + u < a.n) lrow[u] = mine[u];
                }
            }
            // tile max and sum of exp2 over the 8 row groups (lanes l8 + 8*rg)
            m = fmaxf(m, __shfl_xor(m, 8, 64));
            m = fmaxf(m, __shfl_xor(m, 16, 64));
            m = fmaxf(m, __shfl_xor(m, 32, 64));
            float z = 0.0f;
#pragma unroll
            for (int u = 0; u < kRowsPerLane; ++u) z += jr + u < a.n ? exp2_ftz(x[u] - m) : 0.0f;
            z += __shfl_xor(z, 8, 64);
            z += __shfl_xor(z, 16, 64);
            z += __shfl_xor(z, 32, 64);
            if (rg == 0 && l8 < GC) tile_part[hc + l8] = make_float2(m, z);
        }
    }

    if constexpr (OUT != kOutLogits) {
        if (l8 == 0 && jr < a.n) {
            float* dst = OUT == kOutRawS ? a.s + (int64_t)c.b * a.s_sb + (int64_t)c.g * a.s_sr + jr
                                         : a.logits + ((int64_t)c.b * a.Hkv + c.g) * a.ld + jr;
            if (jr + kRowsPerLane <= a.n) {
                float4 v = make_float4(rawsum[0], rawsum[1], rawsum[2], rawsum[3]);
                if constexpr (OUT == kOutRawS) {
                    const float4 o = *reinterpret_cast<const float4*>(dst);
                    v.x += o.x; v.y += o.y; v.z += o.z; v.w += o.w;
                }
                *reinterpret_cast<float4*>(dst) = v;
            } else {
#pragma unroll
                for (int u = 0; u < kRowsPerLane; ++u)
                    if (jr + u < a.n) dst[u] = (OUT == kOutRawS ? dst[u] : 0.0f) + rawsum[u];
            }
        }
    }
}

// Merges the unit's tile pairs of every head of the group into the unit's
// pair (tile order), by threads 0 .. G-1.
__device__ __forceinline__ void merge_unit(const ScoreArgs& a, int bg, int unit, const float2 (*tp)[kMaxGroup])
{
    const int h = threadIdx.x;
    if (h >= a.G) return;
    float m = -INFINITY;
#pragma unroll
    for (int i = 0; i < kUnitTiles; ++i) m = fmaxf(m, tp[i][h].x);
    float z = 0.0f;
#pragma unroll
    for (int i = 0; i < kUnitTiles; ++i)
        z += tp[i][h].x == -INFINITY ? 0.0f : tp[i][h].y * exp2_ftz(tp[i][h].x - m);
    const int b = bg / a.Hkv, g = bg % a.Hkv;
    a.part[((int64_t)b * a.Hq + g * a.G + h) * a.npart + unit] = make_float2(m, z);
}

// Work unit: kUnitTiles consecutive wave-tiles of one (b, g); wave w takes
// tiles w, w+4, ... of the unit.  Each workgroup walks a contiguous range of
// units.  Keys = KeysF16 (16-bit cache) or KeysSketch (int8 / int4 sketch).
template <int GC, int OUT, typename Keys>
__global__ __launch_bounds__(256) void score_tiles_kernel(ScoreArgs a)
{
    __shared__ float2 tile_part[kUnitTiles][kMaxGroup];   // ATTN: per tile of the unit, per head of the group
    __shared__ typename std::conditional<Keys::kGroupQuery, QueryLds, int>::type qlds;
    const int lane = threadIdx.x & 63;
    const int wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int rg = lane >> 3;
    const int l8 = lane & 7;

    if (a.zero_ptr) {
        for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < a.zero_words; i += (int64_t)gridDim.x * 256)
            a.zero_ptr[i] = 0u;
    }

    const int total = a.B * a.Hkv * a.npart;
    const int per = (total + gridDim.x - 1) / gridDim.x;
    int u = blockIdx.x * per;
    const int u_end = min(u + per, total);

    static_assert(kUnitTiles == 8, "each wave takes two tiles of a unit");
    // one tile in flight per wave: the next unit's first tile is requested
    // before this unit's merge, so its barriers overlap that load
    constexpr bool kAhead = !Keys::kGroupQuery && Keys::kSlots == 1;
    bool ahead = false;
    Keys ks;
    int cur_bg = -1;
    for (; u < u_end; ++u) {
        const int bg = u / a.npart, unit = u % a.npart;
        const int i0 = wv, i1 = wv + 4;   // this wave's tiles of the unit
        const int t0 = unit * kUnitTiles + i0, t1 = unit * kUnitTiles + i1;
        const TileCoord c0 = coord(a, bg * a.ntiles + min(t0, a.ntiles - 1));
        const TileCoord c1 = coord(a, bg * a.ntiles + min(t1, a.ntiles - 1));
        if constexpr (Keys::kGroupQuery) {
            // query words first, then both tiles' keys (clamped coordinates: no
            // branch between them), then the cast, which waits only for the query
            const bool fresh = bg != cur_bg;   // workgroup-uniform
            if (fresh) {
                if (cur_bg >= 0 && OUT != kOutLogits) __syncthreads();   // earlier reads of the casts are done
                ks.group_query_fetch(a, bg / a.Hkv, bg % a.Hkv, wv, lane);
            }
            ks.template load<0>(a, c0, rg, l8);
            ks.template load<1>(a, c1, rg, l8);
            if (fresh) {
                ks.ql = &qlds;
                ks.group_query(a, bg / a.Hkv, bg % a.Hkv, wv, lane);
                __syncthreads();
                cur_bg = bg;
            }
        } else {
            if (t0 < a.ntiles && !ahead) ks.template load<0>(a, c0, rg, l8);
            if constexpr (Keys::kSlots == 2) {   // both tiles in flight at once
                if (t1 < a.ntiles) ks.template load<1>(a, c1, rg, l8);
            }
        }
        if (t0 < a.ntiles) {
            if constexpr (Keys::kMfmaSplit) compute_tile_mfma16<0>(a, c0, rg * 8 + l8, ks, tile_part[i0]);
            else compute_tile<GC, OUT, 0>(a, c0, rg, l8, ks, tile_part[i0]);
        } else if constexpr (OUT == kOutLogits) {
            for (int h = lane; h < a.G; h += 64) tile_part[i0][h] = make_float2(-INFINITY, 0.0f);
        }
        if (t1 < a.ntiles) {
            if constexpr (Keys::kSlots == 1) ks.template load<0>(a, c1, rg, l8);
            if constexpr (Keys::kMfmaSplit)
                compute_tile_mfma16<Keys::kSlots - 1>(a, c1, rg * 8 + l8, ks, tile_part[i1]);
            else compute_tile<GC, OUT, Keys::kSlots - 1>(a, c1, rg, l8, ks, tile_part[i1]);
        } else if constexpr (OUT == kOutLogits) {
            for (int h = lane; h < a.G; h += 64) tile_part[i1][h] = make_float2(-INFINITY, 0.0f);
        }
        if constexpr (kAhead) {
            ahead = u + 1 < u_end;   // workgroup-uniform
            if (ahead) {
                const int un = u + 1, tn = (un % a.npart) * kUnitTiles + i0;
                if (tn < a.ntiles) ks.template load<0>(a, coord(a, (un / a.npart) * a.ntiles + tn), rg, l8);
            }
        }

        if constexpr (OUT == kOutLogits) {
            __syncthreads();
            merge_unit(a, bg, unit, tile_part);
            __syncthreads();
        }
    }
}

// Workgroups of `kernel` that stay resident on one CU (queried once per instantiation).
template <typename K>
int resident_per_cu(K kernel)
{
    static const int v = [kernel] {
        int nb = 0;
        if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&nb, kernel, 256, 0) != hipSuccess || nb < 1) nb = 1;
        return nb;
    }();
    return v;
}

// Persistent grid: every workgroup resident at once, each with at least one unit.
template <int DT, int GC, int OUT>
hipError_t launch_score_inst(const ScoreArgs& a, int ncu, hipStream_t st, Stamp ts)
{
    const int64_t total = (int64_t)a.B * a.Hkv * a.npart;
    if constexpr (OUT == kOutLogits) {
        // int4 sketch, ATTN logits, G >= 4: integer dots on the matrix cores (with fewer heads per
        // key the vector units' dot chains are short and faster)
        if (a.k8 && a.kbits == 4 && a.G >= 4) {
            auto kernel = score_tiles_kernel<1, OUT, KeysSketchMfma4<DT>>;
            const int64_t cap = (int64_t)ncu * resident_per_cu(kernel);
            const int64_t grid = total < cap ? (total < 1 ? 1 : total) : cap;
            hipExtLaunchKernelGGL(kernel, dim3((unsigned)grid), dim3(256), 0, st, ts.start, ts.stop, 0, a);
            return hipGetLastError();
        }
        if (a.k8 && a.kbits == 8 && a.G >= 4) {
            auto kernel = score_tiles_kernel<1, OUT, KeysSketchMfma8<DT>>;
            const int64_t cap = (int64_t)ncu * resident_per_cu(kernel);
            const int64_t grid = total < cap ? (total < 1 ? 1 : total) : cap;
            hipExtLaunchKernelGGL(kernel, dim3((unsigned)grid), dim3(256), 0, st, ts.start, ts.stop, 0, a);
            return hipGetLastError();
        }
        // 16-bit keys, G >= 4: the dots on the matrix cores as well
        if (!a.k8 && a.G >= 4) {
            auto kernel = score_tiles_kernel<1, OUT, KeysF16Mfma<DT>>;
            const int64_t cap = (int64_t)ncu * resident_per_cu(kernel);
            const int64_t grid = total < cap ? (total < 1 ? 1 : total) : cap;
            hipExtLaunchKernelGGL(kernel, dim3((unsigned)grid), dim3(256), 0, st, ts.start, ts.stop, 0, a);
            return hipGetLastError();
        }
    }
    if (a.k8 && a.kbits == 4) {
        auto kernel = score_tiles_kernel<GC, OUT, KeysSketch<DT, GC, 4>>;
        const int64_t cap = (int64_t)ncu * resident_per_cu(kernel);
        const int64_t grid = total < cap ? (total < 1 ? 1 : total) : cap;
        hipExtLaunchKernelGGL(kernel, dim3((unsigned)grid), dim3(256), 0, st, ts.start, ts.stop, 0, a);
    } else if (a.k8) {
        auto kernel = score_tiles_kernel<GC, OUT, KeysSketch<DT, GC, 8>>;
        const int64_t cap = (int64_t)ncu * resident_per_cu(kernel);
        const int64_t grid = total < cap ? (total < 1 ? 1 : total) : cap;
        hipExtLaunchKernelGGL(kernel, dim3((unsigned)grid), dim3(256), 0, st, ts.start, ts.stop, 0, a);
    } else {
        auto kernel = score_tiles_kernel<GC, OUT, KeysF16<DT, GC>>;
        const int64_t cap = (int64_t)ncu * resident_per_cu(kernel);
        const int64_t grid = total < cap ? (total < 1 ? 1 : total) : cap;
        hipExtLaunchKernelGGL(kernel, dim3((unsigned)grid), dim3(256), 0, st, ts.start, ts.stop, 0, a);
    }
    return hipGetLastError();
}

template <int DT, int OUT>
hipError_t launch_score_gc(const ScoreArgs& a, int gc, int ncu, hipStream_t st, Stamp ts)
{
    switch (gc) {
    case 8: return launch_score_inst<DT, 8, OUT>(a, ncu, st, ts);
    case 4: return launch_score_inst<DT, 4, OUT>(a, ncu, st, ts);
    case 2: return launch_score_inst<DT, 2, OUT>(a, ncu, st, ts);
    default: return launch_score_inst<DT, 1, OUT>(a, ncu, st, ts);
    }
}

template <int DT>
hipError_t launch_score_dt(const ScoreArgs& a, ScoreOut out, int gc, int ncu, hipStream_t st, Stamp ts)
{
    switch (out) {
    case kOutLogits: return launch_score_gc<DT, kOutLogits>(a, gc, ncu, st, ts);
    case kOutRawS: return launch_score_gc<DT, kOutRawS>(a, gc, ncu, st, ts);
    default: return launch_score_gc<DT, kOutRawGroups>(a, gc, ncu, st, ts);
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

hipError_t launch_score_tiles(const ScoreArgs& a, int dtype, ScoreOut out, int ncu, hipStream_t st, Stamp ts)
{
    // heads per pass over the key registers: the largest of 8, 4, 2, 1 dividing G
    const int gc = (a.G % 8 == 0) ? 8 : (a.G % 4 == 0) ? 4 : (a.G % 2 == 0) ? 2 : 1;
    if (dtype == 1) return launch_score_dt<1>(a, out, gc, ncu, st, ts);
    return launch_score_dt<0>(a, out, gc, ncu, st, ts);
}

}  // namespace hill
