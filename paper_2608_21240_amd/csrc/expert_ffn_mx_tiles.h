// MXFP4 tile code of the grouped expert FFN (the HIT tiles of expert_ffn_mx.hip and of the
// decode layer's launches in layer_decode.hip): the weight-format description, the
// contraction layout and the buffer loads are documented in expert_ffn_mx.hip.  Everything
// here has internal linkage; each kernel source compiles its own copy.
#pragma once

#include "expert_ffn_tiles.h"

namespace spice {
namespace {


typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));

// Bytes of one pool slot: an MXFP4 blob of [2I][d] (W13) or [d][I] (W2).
__device__ __forceinline__ size_t expert_w13_bytes_dev(const FfnArgs& a) {
    const size_t n = (size_t)2 * a.I * a.d;
    return n / 2 + n / 32;
}
__device__ __forceinline__ size_t expert_w2_bytes_dev(const FfnArgs& a) {
    const size_t n = (size_t)a.I * a.d;
    return n / 2 + n / 32;
}

// E8M0 block scale -> fp32 2^(s - 127): the exponent field for s >= 1, the subnormal
// 2^-127 for s = 0, NaN for s = 255; the conversion applies it exactly.
__device__ __forceinline__ float e8m0(uint32_t s) {
    return s == 255u ? __uint_as_float(0x7FC00000u) : s == 0u ? __uint_as_float(0x00400000u) : __uint_as_float(s << 23);
}

// 32 E2M1 codes (16 bytes) times the block scale -> 32 bf16 as four MFMA A operands:
// op[k] holds elements 8k .. 8k+7 (bytes 4k .. 4k+3, low nibble first).
__device__ __forceinline__ void mx_decode(u32x4_t raw, float scale, u32x4_t (&op)[4]) {
    const uint32_t w[4] = {raw.x, raw.y, raw.z, raw.w};
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        const bf16x2_t p0 = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(w[k], scale, 0);
        const bf16x2_t p1 = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(w[k], scale, 1);
        const bf16x2_t p2 = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(w[k], scale, 2);
        const bf16x2_t p3 = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(w[k], scale, 3);
        op[k] = u32x4_t{__builtin_bit_cast(uint32_t, p0), __builtin_bit_cast(uint32_t, p1),
                        __builtin_bit_cast(uint32_t, p2), __builtin_bit_cast(uint32_t, p3)};
    }
}

// Raw buffer resources (base, size; unstrided): a load whose lane offset lies past the
// size reads zero, which covers the rows past the end of a matrix and the lanes past
// the end of a row in a partial group.  Offsets that differ per lane live in VGPRs; a
// group's offset, which is uniform, goes in the scalar offset.
typedef __amdgpu_buffer_rsrc_t rsrc_t;
constexpr int kRawBufferWord3 = 0x00020000;     // gfx9 raw buffer: 32-bit data format
constexpr uint32_t kOutOfRange = 0x80000000u;   // a lane offset past every buffer here

__device__ __forceinline__ rsrc_t raw_buffer(const void* p, size_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), 0, (int)bytes, kRawBufferWord3);
}

constexpr int kMxUpR = 2;      // 16-row tiles of W1 (and of W3) per up tile
constexpr int kMxDownR = 4;    // 16-row tiles of W2 per down tile
constexpr int kMxDepth = 2;    // groups in flight per wave
constexpr int kMxMaxNb = SPICE_MXFP4_MAX_K / 32;  // E8M0 scales per row, at most
// A tile's block scales sit in LDS: [matrix][16 R rows][nb], filled once per tile by
// coalesced 16-byte loads (a quarter of a byte per weight element would otherwise cost
// one byte load per row stream and group).
constexpr int kMxScaleBytes = std::max(2 * kMxUpR, kMxDownR) * 16 * kMxMaxNb + 16;

// The operands of one MX tile: NM matrices (W1 and W3 for up, W2 for down) of NR row
// tiles each, so NA = NM NR row streams, and one token row per lane (16 tokens).  Lane
// (m, quad) of stream (mat, r) reads row 16 r + m of the tile in matrix mat: codes at
// vc[r] + 64 g for group g, its scale from LDS; its token row at vt + 256 g.
template <int NM, int NR>
struct MxTile {
    rsrc_t codes[NM], tok;
    uint32_t vc[NR], vt;
    int nb;
    const uint8_t* sc;  // LDS scales of the tile
};

// One group in flight: the codes of its NA row streams and its 4 token chunks.
template <int NA>
struct MxSlot {
    u32x4_t a[NA], b[4];
};

template <int NM, int NR>
__device__ __forceinline__ void mx_issue_w(const MxTile<NM, NR>& o, int g, bool ok, MxSlot<NM * NR>& sl) {
#pragma unroll
    for (int mm = 0; mm < NM; ++mm)
#pragma unroll
        for (int r = 0; r < NR; ++r) {
            const uint32_t vc = ok ? o.vc[r] : kOutOfRange;
            sl.a[mm * NR + r] =
                __builtin_bit_cast(u32x4_t, __builtin_amdgcn_raw_buffer_load_b128(o.codes[mm], vc, g * 64, 0));
        }
}

template <int NM, int NR>
__device__ __forceinline__ void mx_issue_t(const MxTile<NM, NR>& o, int g, bool ok, MxSlot<NM * NR>& sl) {
    const uint32_t vt = ok ? o.vt : kOutOfRange;
#pragma unroll
    for (int u = 0; u < 4; ++u)
        sl.b[u] = __builtin_bit_cast(u32x4_t, __builtin_amdgcn_raw_buffer_load_b128(o.tok, vt + 16 * u, g * 256, 0));
}

// The MFMAs of group g; ok = false for a lane whose block lies past the row end (its
// codes read zero; its scale is taken as 1 so that no stale byte can make a NaN).
template <int NM, int NR>
__device__ __forceinline__ void mx_use(const MxTile<NM, NR>& o, int g, bool ok, const MxSlot<NM * NR>& sl,
                                       f32x4_t (&acc)[NM * NR]) {
    const int lane = threadIdx.x & 63, m = lane & 15, quad = lane >> 4;
#pragma unroll
    for (int mm = 0; mm < NM; ++mm)
#pragma unroll
        for (int r = 0; r < NR; ++r) {
            const int i = mm * NR + r;
            const uint32_t sb = ok ? o.sc[(mm * 16 * NR + 16 * r + m) * o.nb + 4 * g + quad] : 127u;
            u32x4_t op[4];
            mx_decode(sl.a[i], e8m0(sb), op);
#pragma unroll
            for (int u = 0; u < 4; ++u) acc[i] = Tr<SPICE_BF16>::mma(op[u], sl.b[u], acc[i]);
            __builtin_amdgcn_sched_barrier(0);  // one stream's decoded operands live at a time
        }
}

// Whole groups of 4 MX blocks are dealt to the waves (w uniform); the last wave also
// takes the partial group.
struct MxGroups {
    int g0, g1;
    __device__ MxGroups(int nb, int w) {
        const int ngr = nb / 4;
        g0 = w * ngr / kWaves;
        g1 = (w + 1) * ngr / kWaves;
    }
};

// The codes, then (once the token row is known) the token chunks of the wave's first
// kMxDepth groups.  Every load is issued, a group past the wave's share reading zeros,
// so that no branch stands between a load and the wait for it.
template <int NM, int NR>
__device__ __forceinline__ void mx_prologue_w(const MxTile<NM, NR>& o, const MxGroups& wg,
                                              MxSlot<NM * NR> (&ring)[kMxDepth]) {
#pragma unroll
    for (int d = 0; d < kMxDepth; ++d) mx_issue_w(o, wg.g0 + d, wg.g0 + d < wg.g1, ring[d]);
}
template <int NM, int NR>
__device__ __forceinline__ void mx_prologue_t(const MxTile<NM, NR>& o, const MxGroups& wg,
                                              MxSlot<NM * NR> (&ring)[kMxDepth]) {
#pragma unroll
    for (int d = 0; d < kMxDepth; ++d) mx_issue_t(o, wg.g0 + d, wg.g0 + d < wg.g1, ring[d]);
}

// This wave's share of the tile's product over K = 32 nb; ring holds the wave's first
// kMxDepth groups (mx_prologue_w, mx_prologue_t).  Each group's MFMAs are followed by
// the loads of the group kMxDepth ahead into the same slot, issued unconditionally (past
// the wave's share they read zeros), so each wait leaves the later groups in flight.
template <int NM, int NR>
__device__ __forceinline__ void mx_wave_product(const MxTile<NM, NR>& o, const MxGroups& wg, int w,
                                                MxSlot<NM * NR> (&ring)[kMxDepth], f32x4_t (&acc)[NM * NR]) {
    constexpr int NA = NM * NR, D = kMxDepth;
#pragma unroll
    for (int i = 0; i < NA; ++i) acc[i] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    for (int g = wg.g0; g < wg.g1; g += D) {
#pragma unroll
        for (int d = 0; d < D; ++d) {
            if (g + d < wg.g1) mx_use(o, g + d, true, ring[d], acc);
            const int gn = g + d + D;
            mx_issue_w(o, gn, gn < wg.g1, ring[d]);
            mx_issue_t(o, gn, gn < wg.g1, ring[d]);
        }
    }
    if (w == kWaves - 1 && o.nb % 4) {  // the partial group: lanes past the row end read zeros
        const int ngr = o.nb / 4;
        const bool ok = 4 * ngr + (int)((threadIdx.x & 63) >> 4) < o.nb;
        mx_issue_w(o, ngr, ok, ring[0]);
        mx_issue_t(o, ngr, ok, ring[0]);
        mx_use(o, ngr, ok, ring[0], acc);
    }
}

// Coalesced loads of a tile's scale rows, issued first: 16 R rows of nb bytes from row
// row0 of each of the NM matrices, whose scale blocks follow each other (mat_rows rows
// apart) in the buffer sc; rows past the buffer, and chunks past the tile, read zero.
// mx_scale_store puts them in LDS once they have arrived.
constexpr int kMxScaleChunks = (std::max(2 * kMxUpR, kMxDownR) * kMxMaxNb + kThreads - 1) / kThreads;  // per thread
template <int NM, int NR>
__device__ __forceinline__ void mx_scale_load(rsrc_t sc, int mat_rows, int row0, int nb, u32x4_t (&v)[kMxScaleChunks]) {
    const int per_mat = NR * nb;  // 16-byte chunks of one matrix's rows (16 NR nb bytes)
#pragma unroll
    for (int i = 0; i < kMxScaleChunks; ++i) {
        const int c = threadIdx.x + kThreads * i;
        const int mm = c / per_mat, cc = c % per_mat;
        const uint32_t off = c < NM * per_mat ? (uint32_t)((mm * mat_rows + row0) * nb + cc * 16) : kOutOfRange;
        v[i] = __builtin_bit_cast(u32x4_t, __builtin_amdgcn_raw_buffer_load_b128(sc, off, 0, 0));
    }
}

template <int NM, int NR>
__device__ __forceinline__ void mx_scale_store(uint8_t* lds, int nb, const u32x4_t (&v)[kMxScaleChunks]) {
#pragma unroll
    for (int i = 0; i < kMxScaleChunks; ++i) {
        const int c = threadIdx.x + kThreads * i;
        if (c < NM * NR * nb) *reinterpret_cast<u32x4_t*>(lds + c * 16) = v[i];
    }
}

// ---------------------------------------------------------------------------
// up: 16 R W1 rows and the same 16 R W3 rows of a HIT expert in MXFP4.  An MXFP4 row
// carries a quarter of the bytes of a bf16 row, so a tile takes R times the rows of a bf16
// up tile: the token loads of a group are shared by 2 R weight loads.
// ---------------------------------------------------------------------------
template <int R>
struct MxUpLds {
    f32x4_t red[kWaves][2 * R][64];
    alignas(16) uint8_t sc[kMxScaleBytes];
};
template <int R>
struct MxDownLds {
    f32x4_t red[kWaves][R][64];
    alignas(16) uint8_t sc[kMxScaleBytes];
};

// Up tile rt of a HIT group: ids = the group's slot ids in bucket order (the global perm
// from the group's start, or a list in LDS).
template <int R>
__device__ void mx_up_tile(const FfnArgs& a, const Group& g, int rt, const int32_t* ids, MxUpLds<R>& lds) {
    const int lane = threadIdx.x & 63;
    const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int m = lane & 15, quad = lane >> 4;
    const int K = a.d, nb = K / 32;
    const size_t rb = K / 2;  // code bytes of a row
    // the group is the same in every lane: say so, so that the buffer resources live in SGPRs
    const int slot = __builtin_amdgcn_readfirstlane(g.slot);
    const char* blob = static_cast<const char*>(a.w13_pool) + (size_t)slot * expert_w13_bytes_dev(a);
    const char* scb = blob + (size_t)2 * a.I * rb;
    const int row0 = rt * 16 * R;
    const int start = g.start, n = g.n;
    u32x4_t scv[kMxScaleChunks];
    mx_scale_load<2, R>(raw_buffer(scb, (size_t)2 * a.I * nb), a.I, row0, nb, scv);
    MxTile<2, R> o;
    o.codes[0] = raw_buffer(blob, (size_t)a.I * rb);
    o.codes[1] = raw_buffer(blob + (size_t)a.I * rb, (size_t)a.I * rb);
    o.tok = raw_buffer(a.x, (size_t)a.T * a.d * 2);
    o.nb = nb;
    o.sc = lds.sc;
#pragma unroll
    for (int r = 0; r < R; ++r)  // rows past the end of the matrix read zeros; their outputs are dropped
        o.vc[r] = (uint32_t)((row0 + 16 * r + m) * rb + quad * 16);
    const MxGroups wg(nb, w);
    const int TK = a.T * a.K;
    for (int g0 = 0; g0 < n; g0 += 16) {  // passes of 16 tokens: ids, then codes, then token rows
        const int pid = ids[min(g0 + m, n - 1)];
        MxSlot<2 * R> ring[kMxDepth];
        mx_prologue_w(o, wg, ring);
        const bool bad = pid < 0 || pid >= TK;
        o.vt = (uint32_t)((bad ? 0 : pid / a.K) * a.d * 2 + quad * 64);
        mx_prologue_t(o, wg, ring);
        if (bad) atomicOr(&a.ctrl[kWordFlags], (uint32_t)SPICE_FLAG_BAD_INDEX);
        if (g0 == 0) {
            mx_scale_store<2, R>(lds.sc, nb, scv);
            __syncthreads();
        }
        f32x4_t acc[2 * R];
        mx_wave_product<2, R>(o, wg, w, ring, acc);
#pragma unroll
        for (int i = 0; i < 2 * R; ++i) lds.red[w][i][lane] = acc[i];
        __syncthreads();
        for (int rr = w; rr < R; rr += kWaves) {  // wave w finalises row tiles w, w + 4, ...
            f32x4_t sg = lds.red[0][rr][lane], su = lds.red[0][R + rr][lane];
#pragma unroll
            for (int ww = 1; ww < kWaves; ++ww) {
                sg += lds.red[ww][rr][lane];
                su += lds.red[ww][R + rr][lane];
            }
            const int gi = g0 + m;
            const int orow = row0 + rr * 16 + quad * 4;
            if (gi < n && orow < a.I) {
                f32x4_t h;
                h.x = silu(sg.x) * su.x;
                h.y = silu(sg.y) * su.y;
                h.z = silu(sg.z) * su.z;
                h.w = silu(sg.w) * su.w;
                Tr<SPICE_BF16>::store4(a.h, (size_t)(start + gi) * a.ldh + orow, h);
            }
        }
        __syncthreads();
    }
}

// ---------------------------------------------------------------------------
// down: 16 R W2 rows of a HIT expert in MXFP4, K = I
// ---------------------------------------------------------------------------
template <int R>
__device__ void mx_down_tile(const FfnArgs& a, const Group& g, int rt, MxDownLds<R>& lds) {
    const int lane = threadIdx.x & 63;
    const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int m = lane & 15, quad = lane >> 4;
    const int K = a.I, nb = K / 32;
    const size_t rb = K / 2;
    const int slot = __builtin_amdgcn_readfirstlane(g.slot);
    const char* blob = static_cast<const char*>(a.w2_pool) + (size_t)slot * expert_w2_bytes_dev(a);
    const int dim0 = rt * 16 * R;
    const int start = g.start, n = g.n;
    u32x4_t scv[kMxScaleChunks];
    mx_scale_load<1, R>(raw_buffer(blob + (size_t)a.d * rb, (size_t)a.d * nb), a.d, dim0, nb, scv);
    MxTile<1, R> o;
    o.codes[0] = raw_buffer(blob, (size_t)a.d * rb);
    o.tok = raw_buffer(a.h, (size_t)a.T * a.K * a.ldh * 2);
    o.nb = nb;
    o.sc = lds.sc;
#pragma unroll
    for (int r = 0; r < R; ++r)  // rows past d read zeros; their outputs are dropped
        o.vc[r] = (uint32_t)((dim0 + 16 * r + m) * rb + quad * 16);
    const MxGroups wg(nb, w);
    for (int g0 = 0; g0 < n; g0 += 16) {  // passes of 16 tokens
        MxSlot<R> ring[kMxDepth];
        mx_prologue_w(o, wg, ring);
        o.vt = (uint32_t)((start + min(g0 + m, n - 1)) * a.ldh * 2 + quad * 64);
        mx_prologue_t(o, wg, ring);
        if (g0 == 0) {
            mx_scale_store<1, R>(lds.sc, nb, scv);
            __syncthreads();
        }
        f32x4_t acc[R];
        mx_wave_product<1, R>(o, wg, w, ring, acc);
#pragma unroll
        for (int i = 0; i < R; ++i) lds.red[w][i][lane] = acc[i];
        __syncthreads();
        for (int rr = w; rr < R; rr += kWaves) {
            f32x4_t s = lds.red[0][rr][lane];
#pragma unroll
            for (int ww = 1; ww < kWaves; ++ww) s += lds.red[ww][rr][lane];
            const int gi = g0 + m;
            const int dim = dim0 + rr * 16 + quad * 4;
            if (gi < n && dim < a.d) *reinterpret_cast<f32x4_t*>(a.y_slots + (size_t)(start + gi) * a.d + dim) = s;
        }
        __syncthreads();
    }
}

}  // namespace
}  // namespace spice
