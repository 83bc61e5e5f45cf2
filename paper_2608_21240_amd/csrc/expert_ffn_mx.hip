// Grouped expert FFN with MXFP4 routed experts: the quantised-weight variant of the
// grouped SwiGLU FFN (Eq. 6; Sec. 2.1, 4.2), with the shared block and the LoRE
// correction (Eq. 9) unchanged in bf16.
//
// Pool slots hold OCP MXFP4 blobs (FP4 E2M1 codes, two per byte, then one E8M0 scale per
// 32 elements of a row).  HIT tiles decode their weights in registers with the gfx950
// scaled conversion v_cvt_scalef32_pk_bf16_fp4 (two codes and the block scale -> two
// bf16, exact) and feed the same bf16 MFMA as the bf16 path; the shared-block and LoRE
// tiles run the bf16 tile code of expert_ffn_tiles.h.  Two launches, as in
// expert_ffn.hip; one block (4 waves) per tile, in the same tile order.
//
// Contraction layout of a HIT tile: an MFMA step takes 8 consecutive k per lane, and the
// k order only has to agree between the two operands.  Lane (m, q) of group j takes the
// whole MX block b = 4j + q (32 elements, one 16-byte load and one scale byte) and uses it
// for the 4 steps of the group: step u gets elements 8u .. 8u+7 of the block, and the
// token operand of lane (n, q) reads the same 8 k of its token row.  So a group covers
// 128 consecutive k, the weight bytes of a wave are one 16-byte load per row stream and
// group, and two groups are in flight.  Whole groups are dealt to the 4 waves; a last
// partial group (K/32 not a multiple of 4) goes to the last wave with the lanes past the
// row end reading nothing.
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

// E8M0 block scale -> fp32 2^(s - 127) (s = 255 is NaN); the conversion applies it exactly.
__device__ __forceinline__ float e8m0(uint32_t s) {
    return s == 255u ? __uint_as_float(0x7FC00000u) : __uint_as_float(s << 23);
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

// Per-lane pointers of NA weight row streams (elements and scales of the lane's row) and
// NB token rows (bf16, at the lane's column).
template <int NA, int NB>
struct MxOps {
    const char* el[NA];  // row's E2M1 bytes
    const uint8_t* sc[NA];  // row's E8M0 scales
    const char* tok[NB];  // token row (bf16 elements)
};

// One group's loads: per row stream the 16 bytes and the scale of block b, per token tile
// the 4 chunks of 8 bf16 that the group's steps use.  ok: this lane's block is in range.
template <int NA, int NB>
__device__ __forceinline__ void mx_load(const MxOps<NA, NB>& o, int b, bool ok, u32x4_t (&ar)[NA], uint32_t (&as)[NA],
                                        u32x4_t (&bv)[NB][4]) {
    const u32x4_t zero = {0u, 0u, 0u, 0u};
#pragma unroll
    for (int i = 0; i < NA; ++i) {
        ar[i] = ok ? *reinterpret_cast<const u32x4_t*>(o.el[i] + (size_t)b * 16) : zero;
        as[i] = ok ? o.sc[i][b] : 127u;
    }
#pragma unroll
    for (int j = 0; j < NB; ++j)
#pragma unroll
        for (int u = 0; u < 4; ++u)
            bv[j][u] = ok ? *reinterpret_cast<const u32x4_t*>(o.tok[j] + ((size_t)b * 32 + 8 * u) * 2) : zero;
}

template <int NA, int NB>
__device__ __forceinline__ void mx_comp(const u32x4_t (&ar)[NA], const uint32_t (&as)[NA], const u32x4_t (&bv)[NB][4],
                                        f32x4_t (&acc)[NA][NB]) {
#pragma unroll
    for (int i = 0; i < NA; ++i) {
        u32x4_t op[4];
        mx_decode(ar[i], e8m0(as[i]), op);
#pragma unroll
        for (int u = 0; u < 4; ++u)
#pragma unroll
            for (int j = 0; j < NB; ++j) acc[i][j] = Tr<SPICE_BF16>::mma(op[u], bv[j][u], acc[i][j]);
    }
}

// This wave's share of a (NA row streams) x (NB token tiles) product over K = 32 nb
// elements: whole groups [g0, g1) with two in flight, then (last wave) the partial group.
template <int NA, int NB>
__device__ __forceinline__ void mx_wave_product(const MxOps<NA, NB>& o, int nb, int w, int quad,
                                                f32x4_t (&acc)[NA][NB]) {
#pragma unroll
    for (int i = 0; i < NA; ++i)
#pragma unroll
        for (int j = 0; j < NB; ++j) acc[i][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    const int ngr = nb / 4;  // whole groups
    const int g0 = w * ngr / kWaves, g1 = (w + 1) * ngr / kWaves;
    u32x4_t a0[NA], a1[NA], b0[NB][4], b1[NB][4];
    uint32_t s0[NA], s1[NA];
    if (g1 > g0) {
        mx_load<NA, NB>(o, 4 * g0 + quad, true, a0, s0, b0);
        int g = g0;
        for (; g + 2 < g1; g += 2) {
            mx_load<NA, NB>(o, 4 * (g + 1) + quad, true, a1, s1, b1);
            __builtin_amdgcn_sched_barrier(0);
            mx_comp<NA, NB>(a0, s0, b0, acc);
            mx_load<NA, NB>(o, 4 * (g + 2) + quad, true, a0, s0, b0);
            __builtin_amdgcn_sched_barrier(0);
            mx_comp<NA, NB>(a1, s1, b1, acc);
        }
        if (g + 1 < g1) {
            mx_load<NA, NB>(o, 4 * (g + 1) + quad, true, a1, s1, b1);
            __builtin_amdgcn_sched_barrier(0);
            mx_comp<NA, NB>(a0, s0, b0, acc);
            mx_comp<NA, NB>(a1, s1, b1, acc);
        } else {
            mx_comp<NA, NB>(a0, s0, b0, acc);
        }
    }
    if (w == kWaves - 1 && nb % 4) {  // the partial group: lanes past the row end add zero
        const int b = 4 * ngr + quad;
        mx_load<NA, NB>(o, b, b < nb, a0, s0, b0);
        mx_comp<NA, NB>(a0, s0, b0, acc);
    }
}

// ---------------------------------------------------------------------------
// up: 16 W1 rows and the same 16 W3 rows of a HIT expert in MXFP4
// ---------------------------------------------------------------------------
__device__ void mx_up_tile(const FfnArgs& a, const Group& g, const Tile& tile,
                           f32x4_t (&red)[kWaves][kTokTiles][2][64]) {
    constexpr int es = 2;
    const int lane = threadIdx.x & 63;
    const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int m = lane & 15, quad = lane >> 4;
    const int rows = 2 * a.I, K = a.d, nb = K / 32;
    const char* blob = static_cast<const char*>(a.w13_pool) + (size_t)g.slot * expert_w13_bytes_dev(a);
    const uint8_t* scales = reinterpret_cast<const uint8_t*>(blob) + (size_t)rows * (K / 2);
    // rows past the end of the matrix read its last row; their outputs are dropped
    const int row = min(tile.rt * 16 + m, a.I - 1);
    const int start = g.start, n = g.n;
    for (int g0 = 0; g0 < n; g0 += 16 * kTokTiles) {
        const int ntt = min(kTokTiles, (n - g0 + 15) / 16);
        const int gi0 = min(g0 + m, n - 1), gi1 = min(g0 + 16 + m, n - 1);
        if (ntt == 1) {
            MxOps<2, 1> o;
            o.el[0] = blob + (size_t)row * (K / 2);
            o.el[1] = blob + (size_t)(a.I + row) * (K / 2);
            o.sc[0] = scales + (size_t)row * nb;
            o.sc[1] = scales + (size_t)(a.I + row) * nb;
            int t0, t1;
            token_ids<1>(a, start + gi0, start + gi1, t0, t1);
            o.tok[0] = static_cast<const char*>(a.x) + (size_t)t0 * a.d * es;
            f32x4_t acc[2][1];
            mx_wave_product<2, 1>(o, nb, w, quad, acc);
            red[w][0][0][lane] = acc[0][0];
            red[w][0][1][lane] = acc[1][0];
        } else {
            MxOps<2, 2> o;
            o.el[0] = blob + (size_t)row * (K / 2);
            o.el[1] = blob + (size_t)(a.I + row) * (K / 2);
            o.sc[0] = scales + (size_t)row * nb;
            o.sc[1] = scales + (size_t)(a.I + row) * nb;
            int t0, t1;
            token_ids<2>(a, start + gi0, start + gi1, t0, t1);
            o.tok[0] = static_cast<const char*>(a.x) + (size_t)t0 * a.d * es;
            o.tok[1] = static_cast<const char*>(a.x) + (size_t)t1 * a.d * es;
            f32x4_t acc[2][2];
            mx_wave_product<2, 2>(o, nb, w, quad, acc);
#pragma unroll
            for (int j = 0; j < 2; ++j) { red[w][j][0][lane] = acc[0][j]; red[w][j][1][lane] = acc[1][j]; }
        }
        __syncthreads();
        if (w < ntt) {
            const int tt = w;
            f32x4_t sg = red[0][tt][0][lane], su = red[0][tt][1][lane];
#pragma unroll
            for (int ww = 1; ww < kWaves; ++ww) {
                sg += red[ww][tt][0][lane];
                su += red[ww][tt][1][lane];
            }
            const int gi = g0 + tt * 16 + m;
            const int orow = tile.rt * 16 + quad * 4;
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
// down: kDownRows x 16 W2 rows of a HIT expert in MXFP4, K = I
// ---------------------------------------------------------------------------
__device__ void mx_down_tile(const FfnArgs& a, const Group& g, const Tile& tile,
                             f32x4_t (&red)[kWaves][kDownRows][kTokTiles][64]) {
    constexpr int es = 2;
    const int lane = threadIdx.x & 63;
    const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int m = lane & 15, quad = lane >> 4;
    const int rows = a.d, K = a.I, nb = K / 32;
    const char* blob = static_cast<const char*>(a.w2_pool) + (size_t)g.slot * expert_w2_bytes_dev(a);
    const uint8_t* scales = reinterpret_cast<const uint8_t*>(blob) + (size_t)rows * (K / 2);
    const int dim0 = tile.rt * 16 * kDownRows;
    const int start = g.start, n = g.n;
    int r[kDownRows];
#pragma unroll
    for (int rr = 0; rr < kDownRows; ++rr) r[rr] = min(dim0 + rr * 16 + m, a.d - 1);  // tail rows: dropped
    for (int g0 = 0; g0 < n; g0 += 16 * kTokTiles) {
        const int ntt = min(kTokTiles, (n - g0 + 15) / 16);
        const char* hb0 = static_cast<const char*>(a.h) + (size_t)(start + min(g0 + m, n - 1)) * a.ldh * es;
        const char* hb1 = static_cast<const char*>(a.h) + (size_t)(start + min(g0 + 16 + m, n - 1)) * a.ldh * es;
        if (ntt == 1) {
            MxOps<kDownRows, 1> o;
#pragma unroll
            for (int rr = 0; rr < kDownRows; ++rr) {
                o.el[rr] = blob + (size_t)r[rr] * (K / 2);
                o.sc[rr] = scales + (size_t)r[rr] * nb;
            }
            o.tok[0] = hb0;
            f32x4_t acc[kDownRows][1];
            mx_wave_product<kDownRows, 1>(o, nb, w, quad, acc);
#pragma unroll
            for (int rr = 0; rr < kDownRows; ++rr) red[w][rr][0][lane] = acc[rr][0];
        } else {
            MxOps<kDownRows, 2> o;
#pragma unroll
            for (int rr = 0; rr < kDownRows; ++rr) {
                o.el[rr] = blob + (size_t)r[rr] * (K / 2);
                o.sc[rr] = scales + (size_t)r[rr] * nb;
            }
            o.tok[0] = hb0;
            o.tok[1] = hb1;
            f32x4_t acc[kDownRows][2];
            mx_wave_product<kDownRows, 2>(o, nb, w, quad, acc);
#pragma unroll
            for (int rr = 0; rr < kDownRows; ++rr)
#pragma unroll
                for (int j = 0; j < 2; ++j) red[w][rr][j][lane] = acc[rr][j];
        }
        __syncthreads();
        const int rr = w % kDownRows, tt = w / kDownRows;  // wave w finalises (row tile, token tile) w
        if (tt < ntt) {
            f32x4_t s = red[0][rr][tt][lane];
#pragma unroll
            for (int ww = 1; ww < kWaves; ++ww) s += red[ww][rr][tt][lane];
            const int gi = g0 + tt * 16 + m;
            const int dim = dim0 + rr * 16 + quad * 4;
            if (gi < n && dim < a.d) *reinterpret_cast<f32x4_t*>(a.y_slots + (size_t)(start + gi) * a.d + dim) = s;
        }
        __syncthreads();
    }
}

__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(3))) void ffn_up_mx_kernel(FfnArgs a,
                                                                                                       Grid gr) {
    __shared__ f32x4_t red[kWaves][kTokTiles][2][64];
    Tile tile;
    if (!gr.decode(blockIdx.x, tile)) return;
    Group g{0, 0, a.T, -1};
    if (tile.kind != kKindShared &&
        !find_group(a, tile.kind == kKindHit ? SPICE_CLASS_HIT : SPICE_CLASS_LORE, tile.ordinal, g))
        return;
    if (tile.kind == kKindHit) mx_up_tile(a, g, tile, red);
    else up_tile<SPICE_BF16>(a, g, tile, red);
}

__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(3))) void ffn_down_mx_kernel(FfnArgs a,
                                                                                                         Grid gr) {
    __shared__ f32x4_t red[kWaves][kDownRows][kTokTiles][64];
    Tile tile;
    if (!gr.decode(blockIdx.x, tile)) return;
    Group g{0, 0, a.T, -1};
    if (tile.kind != kKindShared &&
        !find_group(a, tile.kind == kKindHit ? SPICE_CLASS_HIT : SPICE_CLASS_LORE, tile.ordinal, g))
        return;
    if (tile.kind == kKindLore)
        lore_down_tile<SPICE_BF16>(a, g.e, g.start, g.n, tile.rt, reinterpret_cast<float*>(&red[0][0][0][0]));
    else if (tile.kind == kKindHit)
        mx_down_tile(a, g, tile, red);
    else
        down_tile<SPICE_BF16>(a, g, tile, red);
}

}  // namespace

hipError_t launch_expert_ffn_mx(const FfnArgs& a, hipStream_t s) {
    if (a.dtype != SPICE_BF16) return hipErrorInvalidValue;
    const bool hit = (a.groups & kDoHit) != 0;
    const bool shared = (a.groups & kDoShared) != 0 && a.Is > 0;
    const bool lore = (a.groups & kDoLore) != 0 && a.r > 0;
    const int slots = a.T * a.K;
    Grid up{0, 1, 0, 0, 1}, dn{0, 1, 0, 0, 1};
    if (hit) {
        up.nhit = dn.nhit = std::min(std::min(a.N, a.C), slots);
        up.thit = (a.I + 15) / 16;
        dn.thit = (a.d + 16 * kDownRows - 1) / (16 * kDownRows);
    }
    if (shared) {
        up.tsh = (a.Is + 15) / 16;
        dn.tsh = (a.d + 16 * kDownRows - 1) / (16 * kDownRows);
    }
    if (lore) {
        up.nlore = dn.nlore = std::min(a.N, slots);
        up.tlore = (a.r + 15) / 16;
        dn.tlore = (a.d + kLoreRows - 1) / kLoreRows;
    }
    const long long nup = (long long)up.nhit * up.thit + up.tsh + (long long)up.nlore * up.tlore;
    const long long ndn = (long long)dn.nhit * dn.thit + dn.tsh + (long long)dn.nlore * dn.tlore;
    if (nup == 0) return hipSuccess;
    hipLaunchKernelGGL(ffn_up_mx_kernel, dim3((unsigned)nup), dim3(kThreads), 0, s, a, up);
    hipLaunchKernelGGL(ffn_down_mx_kernel, dim3((unsigned)ndn), dim3(kThreads), 0, s, a, dn);
    return hipGetLastError();
}

}  // namespace spice
