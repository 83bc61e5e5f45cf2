// Tile code of the grouped expert FFN shared by its kernels (expert_ffn.hip: the
// grouped HIT / shared / LoRE launches; expert_ffn_fetched.hip: the fetched-expert
// launches).  Everything here has internal linkage: each kernel source compiles its
// own copy, so a kernel added in one source leaves the other's code untouched.
#pragma once

#include <hip/hip_runtime.h>

#include <algorithm>

#include "spice_internal.h"
#include "tile_index.h"

namespace spice {
namespace {

constexpr int kThreads = 256;
constexpr int kWaves = 4;

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

template <int DT>
struct Tr;

template <>
struct Tr<SPICE_BF16> {
    static constexpr int kStep = 32;  // contraction elements per MFMA step
    static constexpr int kLaneK = 8;  // elements each lane loads per step (16 bytes)
    __device__ __forceinline__ static u32x4_t load(const void* base, size_t elem) {
        return *reinterpret_cast<const u32x4_t*>(static_cast<const uint16_t*>(base) + elem);
    }
    __device__ __forceinline__ static f32x4_t mma(u32x4_t a, u32x4_t b, f32x4_t c) {
        return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, a),
                                                       __builtin_bit_cast(bf16x8_t, b), c, 0, 0, 0);
    }
    // store 4 consecutive values of a row of the intermediate (bf16, round to nearest even)
    __device__ __forceinline__ static void store4(void* base, size_t elem, f32x4_t v);
};

template <>
struct Tr<SPICE_F32> {
    static constexpr int kStep = 16;
    static constexpr int kLaneK = 4;
    __device__ __forceinline__ static u32x4_t load(const void* base, size_t elem) {
        return *reinterpret_cast<const u32x4_t*>(static_cast<const float*>(base) + elem);
    }
    // four 16x16x4 steps; step j uses element j of every lane's 4-element chunk
    __device__ __forceinline__ static f32x4_t mma(u32x4_t a, u32x4_t b, f32x4_t c) {
        c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.x), __uint_as_float(b.x), c, 0, 0, 0);
        c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.y), __uint_as_float(b.y), c, 0, 0, 0);
        c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.z), __uint_as_float(b.z), c, 0, 0, 0);
        c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.w), __uint_as_float(b.w), c, 0, 0, 0);
        return c;
    }
    __device__ __forceinline__ static void store4(void* base, size_t elem, f32x4_t v) {
        *reinterpret_cast<f32x4_t*>(static_cast<float*>(base) + elem) = v;
    }
};

__device__ __forceinline__ uint32_t f32_to_bf16_rne(float f) {
    const uint32_t u = __float_as_uint(f);
    if ((u & 0x7FFFFFFFu) > 0x7F800000u) return 0x7FC0u;  // NaN stays NaN
    return (u + 0x7FFFu + ((u >> 16) & 1u)) >> 16;
}

__device__ __forceinline__ void Tr<SPICE_BF16>::store4(void* base, size_t elem, f32x4_t v) {
    uint2 p;
    p.x = f32_to_bf16_rne(v.x) | (f32_to_bf16_rne(v.y) << 16);
    p.y = f32_to_bf16_rne(v.z) | (f32_to_bf16_rne(v.w) << 16);
    *reinterpret_cast<uint2*>(static_cast<uint16_t*>(base) + elem) = p;
}

__device__ __forceinline__ float silu(float u) { return u / (1.0f + __expf(-u)); }

// The j-th expert (ascending id) whose bucket of class c is non-empty; for HIT
// buckets its pool slot is fetched in the same round trip as the offsets.
__device__ __attribute__((unused)) bool find_group(const FfnArgs& a, int c, int j, Group& g) {
    const int lane = threadIdx.x & 63;
    const int32_t* off = a.offsets + c * (a.N + 1);
    const unsigned long long lt = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
    int seen = 0;
    for (int base = 0; base < a.N; base += 64) {
        const int e = base + lane;
        Group mine_g{e, 0, 0, -1};
        if (e < a.N) mine_g = bucket_of(off, e, c, c == SPICE_CLASS_HIT ? a.resident_slot[e] : -1);
        const unsigned long long m = __ballot(mine_g.n > 0);
        const int cnt = __popcll(m);
        if (j < seen + cnt) {
            const bool mine = mine_g.n > 0 && __popcll(m & lt) == j - seen;
            const int src = __ffsll((long long)__ballot(mine)) - 1;
            g.e = base + src;
            g.start = __shfl(mine_g.start, src);
            g.n = __shfl(mine_g.n, src);
            g.slot = __shfl(mine_g.slot, src);
            if (!group_in_range(a, c, g)) {
                const bool slot_bad = c == SPICE_CLASS_HIT && g.start >= 0 && g.n >= 0 && g.start + g.n <= a.T * a.K;
                if (lane == 0)
                    atomicOr(&a.ctrl[kWordFlags], (uint32_t)(slot_bad ? SPICE_FLAG_BAD_SLOT : SPICE_FLAG_BAD_INDEX));
                return false;
            }
            return true;
        }
        seen += cnt;
    }
    return false;
}

// ---------------------------------------------------------------------------
// MFMA main loop shared by both launches.
//   a[i]: per-lane pointer to weight row (tile row m = lane & 15) at the lane's k offset
//   b[j]: per-lane pointer to the token row (column m) at the lane's k offset
// The contraction is cut into whole groups of U full steps, dealt to the 4 waves; the
// last wave also does the steps left over.  The wave index is read as a uniform value,
// so the loop bounds live in scalar registers and the group loop has no divergent
// branches: its loads are unconditional and in order, and the wait before each MFMA
// leaves the next group's loads in flight (two groups per wave).
// ---------------------------------------------------------------------------

// Steps per load group: 4 with three operand streams (two weight tiles and one token tile,
// or one and two), 2 with four; two groups are in flight, which fits 3 waves per SIMD.
#define SPICE_GROUP_STEPS(NA, NB) (((NA) + (NB) <= 3) ? 4 : 2)

// Loads of the U steps [sg, sg + U) of one group: unconditional, at immediate offsets
// from one address per operand stream.
template <int DT, int NA, int NB>
__device__ __forceinline__ void mma_load(const char* const (&a)[NA], const char* const (&b)[NB], int sg,
                                         u32x4_t (&av)[NA][SPICE_GROUP_STEPS(NA, NB)],
                                         u32x4_t (&bv)[NB][SPICE_GROUP_STEPS(NA, NB)]) {
    constexpr int U = SPICE_GROUP_STEPS(NA, NB);
    const size_t off = (size_t)sg * kStepBytes;
    // weight loads first: they depend only on the expert's pool slot, while the token
    // rows wait for the bucket's token ids
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
        for (int i = 0; i < NA; ++i) av[i][u] = *reinterpret_cast<const u32x4_t*>(a[i] + off + u * kStepBytes);
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
        for (int j = 0; j < NB; ++j) bv[j][u] = *reinterpret_cast<const u32x4_t*>(b[j] + off + u * kStepBytes);
}

template <int DT, int NA, int NB>
__device__ __forceinline__ void mma_comp(const u32x4_t (&av)[NA][SPICE_GROUP_STEPS(NA, NB)],
                                         const u32x4_t (&bv)[NB][SPICE_GROUP_STEPS(NA, NB)],
                                         f32x4_t (&acc)[NA][NB]) {
    constexpr int U = SPICE_GROUP_STEPS(NA, NB);
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
        for (int j = 0; j < NB; ++j)
#pragma unroll
            for (int i = 0; i < NA; ++i) acc[i][j] = Tr<DT>::mma(av[i][u], bv[j][u], acc[i][j]);
}

// ng whole groups starting at step s0 (uniform), two groups in flight: the loads of
// group g+1 go out before the MFMAs of group g.  The steady-state body loads
// unconditionally, so the wait before each MFMA leaves the next group's loads pending.
template <int DT, int NA, int NB>
__device__ __forceinline__ void mma_groups(const char* const (&a)[NA], const char* const (&b)[NB], int s0, int ng,
                                           f32x4_t (&acc)[NA][NB], u32x4_t (&a0)[NA][SPICE_GROUP_STEPS(NA, NB)]) {
    constexpr int U = SPICE_GROUP_STEPS(NA, NB);
    if (ng <= 0) return;
    u32x4_t b0[NB][U], a1[NA][U], b1[NB][U];
    {  // a0 already holds the weights of group 0 (mma_first_a); its token rows now
        const size_t off = (size_t)s0 * kStepBytes;
#pragma unroll
        for (int u = 0; u < U; ++u)
#pragma unroll
            for (int j = 0; j < NB; ++j) b0[j][u] = *reinterpret_cast<const u32x4_t*>(b[j] + off + u * kStepBytes);
    }
    int g = 0;
    for (; g + 2 < ng; g += 2) {
        mma_load<DT, NA, NB>(a, b, s0 + (g + 1) * U, a1, b1);
        __builtin_amdgcn_sched_barrier(0);
        mma_comp<DT, NA, NB>(a0, b0, acc);
        mma_load<DT, NA, NB>(a, b, s0 + (g + 2) * U, a0, b0);
        __builtin_amdgcn_sched_barrier(0);
        mma_comp<DT, NA, NB>(a1, b1, acc);
    }
    if (g + 1 < ng) {
        mma_load<DT, NA, NB>(a, b, s0 + (g + 1) * U, a1, b1);
        __builtin_amdgcn_sched_barrier(0);
        mma_comp<DT, NA, NB>(a0, b0, acc);
        mma_comp<DT, NA, NB>(a1, b1, acc);
    } else {
        mma_comp<DT, NA, NB>(a0, b0, acc);
    }
}

// Single full steps [ks0, ks1) (the few left over after the whole groups).
template <int DT, int NA, int NB>
__device__ __forceinline__ void mma_singles(const char* const (&a)[NA], const char* const (&b)[NB], int ks0, int ks1,
                                            f32x4_t (&acc)[NA][NB]) {
    for (int ks = ks0; ks < ks1; ++ks) {
        const size_t off = (size_t)ks * kStepBytes;
        u32x4_t av[NA], bv[NB];
#pragma unroll
        for (int i = 0; i < NA; ++i) av[i] = *reinterpret_cast<const u32x4_t*>(a[i] + off);
#pragma unroll
        for (int j = 0; j < NB; ++j) bv[j] = *reinterpret_cast<const u32x4_t*>(b[j] + off);
#pragma unroll
        for (int j = 0; j < NB; ++j)
#pragma unroll
            for (int i = 0; i < NA; ++i) acc[i][j] = Tr<DT>::mma(av[i], bv[j], acc[i][j]);
    }
}

// The one partial contraction step (kdim not a multiple of the step): lanes whose
// 16-byte chunk lies beyond kdim contribute zero.
template <int DT, int NA, int NB>
__device__ __forceinline__ void mma_tail(const char* const (&a)[NA], const char* const (&b)[NB], int ks, bool lane_in,
                                         f32x4_t (&acc)[NA][NB]) {
    const size_t off = (size_t)ks * kStepBytes;
    const u32x4_t zero = {0u, 0u, 0u, 0u};
    u32x4_t av[NA], bv[NB];
#pragma unroll
    for (int i = 0; i < NA; ++i) av[i] = lane_in ? *reinterpret_cast<const u32x4_t*>(a[i] + off) : zero;
#pragma unroll
    for (int j = 0; j < NB; ++j) bv[j] = lane_in ? *reinterpret_cast<const u32x4_t*>(b[j] + off) : zero;
#pragma unroll
    for (int j = 0; j < NB; ++j)
#pragma unroll
        for (int i = 0; i < NA; ++i) acc[i][j] = Tr<DT>::mma(av[i], bv[j], acc[i][j]);
}

// The whole groups of U full steps of kdim are dealt to the waves (w uniform); the
// last wave also takes the full steps left over and the partial step, if any.
template <int DT, int NA, int NB>
struct WaveGroups {
    int g0, g1;
    __device__ WaveGroups(int kdim, int w) {
        const int ngr = (kdim / Tr<DT>::kStep) / SPICE_GROUP_STEPS(NA, NB);
        g0 = w * ngr / kWaves;
        g1 = (w + 1) * ngr / kWaves;
    }
};

// Weight loads of this wave's first group, issued before the token rows are known.
template <int DT, int NA, int NB>
__device__ __forceinline__ void mma_first_a(const char* const (&a)[NA], int kdim, int w,
                                            u32x4_t (&a0)[NA][SPICE_GROUP_STEPS(NA, NB)]) {
    constexpr int U = SPICE_GROUP_STEPS(NA, NB);
    const WaveGroups<DT, NA, NB> wg(kdim, w);
    if (wg.g1 > wg.g0) {
        const size_t off = (size_t)wg.g0 * U * kStepBytes;
#pragma unroll
        for (int u = 0; u < U; ++u)
#pragma unroll
            for (int i = 0; i < NA; ++i) a0[i][u] = *reinterpret_cast<const u32x4_t*>(a[i] + off + u * kStepBytes);
    }
}

// One wave's share of a (NA row streams) x (NB token tiles) product over kdim; a0 holds
// the weights of the wave's first group (mma_first_a).
template <int DT, int NA, int NB>
__device__ __forceinline__ void wave_product(const char* const (&a)[NA], const char* const (&b)[NB], int kdim, int w,
                                             int quad, f32x4_t (&acc)[NA][NB],
                                             u32x4_t (&a0)[NA][SPICE_GROUP_STEPS(NA, NB)]) {
    constexpr int kStep = Tr<DT>::kStep;
    constexpr int U = SPICE_GROUP_STEPS(NA, NB);
#pragma unroll
    for (int i = 0; i < NA; ++i)
#pragma unroll
        for (int j = 0; j < NB; ++j) acc[i][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    const WaveGroups<DT, NA, NB> wg(kdim, w);
    mma_groups<DT, NA, NB>(a, b, wg.g0 * U, wg.g1 - wg.g0, acc, a0);
    if (w == kWaves - 1) {
        const int nfull = kdim / kStep;
        mma_singles<DT, NA, NB>(a, b, (nfull / U) * U, nfull, acc);
        if (nfull * kStep < kdim)  // the partial step
            mma_tail<DT, NA, NB>(a, b, nfull, nfull * kStep + quad * Tr<DT>::kLaneK < kdim, acc);
    }
}

// ---------------------------------------------------------------------------
// up: gate/up SwiGLU rows (HIT, shared) or A_e rows (LORE)
// ---------------------------------------------------------------------------
// Token ids of bucket entries i0 and i1 (i1 only with two token tiles), from the bucket's
// slot ids (global perm or an LDS list): both loads go out before either is checked.
// Garbage gives token 0 and a flag.
template <int NB>
__device__ __forceinline__ void token_ids(const FfnArgs& a, const int32_t* ids, int i0, int i1, int& t0, int& t1) {
    const int s0 = ids[i0];
    const int s1 = (NB == 2) ? ids[i1] : 0;
    __builtin_amdgcn_sched_barrier(0);  // both loads out before the first wait
    const int TK = a.T * a.K;
    const bool bad0 = s0 < 0 || s0 >= TK, bad1 = (NB == 2) && (s1 < 0 || s1 >= TK);
    if (bad0 || bad1) atomicOr(&a.ctrl[kWordFlags], (uint32_t)SPICE_FLAG_BAD_INDEX);
    t0 = bad0 ? 0 : s0 / a.K;
    t1 = (NB == 2 && !bad1) ? s1 / a.K : 0;
}

// One token group of an up tile: the weight loads of the first group go out, then the
// token ids are read (ids != nullptr: a bucket; nullptr: tokens 0..T-1 in order) and the
// product runs.
template <int DT, int NB, bool kUp>
__device__ __forceinline__ void up_pass(const FfnArgs& a, const char* gate, const char* up, const int32_t* ids, int gi0,
                                        int gi1, size_t kb, int w, int quad, f32x4_t (&red)[kWaves][kTokTiles][2][64],
                                        int lane) {
    constexpr int es = (DT == SPICE_BF16) ? 2 : 4;
    constexpr int NA = kUp ? 2 : 1;
    constexpr int U = SPICE_GROUP_STEPS(NA, NB);
    const char* p[NA];
    p[0] = gate;
    if constexpr (NA == 2) p[1] = up;
    u32x4_t a0[NA][U];
    mma_first_a<DT, NA, NB>(p, a.d, w, a0);
    __builtin_amdgcn_sched_barrier(0);
    int t0 = gi0, t1 = gi1;
    if (ids) token_ids<NB>(a, ids, gi0, gi1, t0, t1);
    const char* xn[NB];
    xn[0] = static_cast<const char*>(a.x) + (size_t)t0 * a.d * es + kb;
    if constexpr (NB == 2) xn[1] = static_cast<const char*>(a.x) + (size_t)t1 * a.d * es + kb;
    f32x4_t acc[NA][NB];
    wave_product<DT, NA, NB>(p, xn, a.d, w, quad, acc, a0);
#pragma unroll
    for (int j = 0; j < NB; ++j) {
        red[w][j][0][lane] = acc[0][j];
        if constexpr (kUp) red[w][j][1][lane] = acc[NA - 1][j];
    }
}

// Up tile rt of one group, the kind fixed at compile time (so is the weight base: no tile
// chooses it at run time).  KIND = kKindHit: 16 W1 rows and the same 16 W3 rows of the
// group's pool slot, H = silu(X W1^T) * (X W3^T) to a.h at the bucket positions;
// kKindShared: the same of the shared block for tokens 0..T-1, to a.hs; kKindLore: 16 rows
// of A_e, U = X A_e^T to a.u at the bucket positions.  ids: the group's slot ids in bucket
// order (its start is g.start), unused for kKindShared.
template <int DT, int KIND>
__device__ void up_tile(const FfnArgs& a, const Group& g, int rt, const int32_t* ids,
                        f32x4_t (&red)[kWaves][kTokTiles][2][64]) {
    using T_ = Tr<DT>;
    constexpr int es = (DT == SPICE_BF16) ? 2 : 4;
    constexpr bool kUp = KIND != kKindLore;
    const int lane = threadIdx.x & 63;
    const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);  // wave index, uniform
    const void* wbase = up_weights<KIND>(a);
    const UpBlock ub = up_block<KIND>(a, g);
    const int nrows = ub.nrows;
    int start, n;
    tile_entries<KIND>(a, g, start, n);
    if constexpr (KIND == kKindShared) ids = nullptr;
    const int m = lane & 15;  // A row / B column owned by this lane
    const int quad = lane >> 4;
    const int row = tile_row(rt, kTileRows, m, nrows);
    const size_t kb = (size_t)quad * T_::kLaneK * es;  // lane's byte offset inside a step
    const char* gate = static_cast<const char*>(wbase) + (ub.gate_row0 + row) * (size_t)a.d * es + kb;
    const char* up = static_cast<const char*>(wbase) + (ub.up_row0 + row) * (size_t)a.d * es + kb;

    for (int g0 = 0; g0 < n; g0 += 16 * kTokTiles) {
        const int ntt = min(kTokTiles, (n - g0 + 15) / 16);
        const int gi0 = tile_entry(g0, 0, m, n), gi1 = tile_entry(g0, 1, m, n);
        if (ntt == 1) up_pass<DT, 1, kUp>(a, gate, up, ids, gi0, gi1, kb, w, quad, red, lane);
        else up_pass<DT, 2, kUp>(a, gate, up, ids, gi0, gi1, kb, w, quad, red, lane);
        __syncthreads();
        if (w < ntt) {
            const int tt = w;
            f32x4_t sg = red[0][tt][0][lane];
#pragma unroll
            for (int ww = 1; ww < kWaves; ++ww) sg += red[ww][tt][0][lane];
            const int gi = g0 + tt * 16 + m;  // output column = token of lane m
            const int orow = rt * 16 + quad * 4;
            if constexpr (KIND == kKindLore) {
                if (gi < n && orow < nrows) *reinterpret_cast<f32x4_t*>(a.u + up_out_elem<KIND>(a, start, gi, orow)) = sg;
            } else {
                f32x4_t su = red[0][tt][1][lane];
#pragma unroll
                for (int ww = 1; ww < kWaves; ++ww) su += red[ww][tt][1][lane];
                if (gi < n && orow < nrows) {
                    f32x4_t h;
                    h.x = silu(sg.x) * su.x;
                    h.y = silu(sg.y) * su.y;
                    h.z = silu(sg.z) * su.z;
                    h.w = silu(sg.w) * su.w;
                    T_::store4(KIND == kKindHit ? a.h : a.hs, up_out_elem<KIND>(a, start, gi, orow), h);
                }
            }
        }
        __syncthreads();
    }
}

// A tile of any kind (the kind read at run time selects one of the instantiations).
template <int DT>
__device__ __forceinline__ void up_tile_kind(const FfnArgs& a, const Group& g, const Tile& tile,
                                             f32x4_t (&red)[kWaves][kTokTiles][2][64]) {
    if (tile.kind == kKindHit) up_tile<DT, kKindHit>(a, g, tile.rt, a.perm + g.start, red);
    else if (tile.kind == kKindShared) up_tile<DT, kKindShared>(a, g, tile.rt, nullptr, red);
    else up_tile<DT, kKindLore>(a, g, tile.rt, a.perm + g.start, red);
}

// ---------------------------------------------------------------------------
// down: W2 rows (HIT, shared) with the MFMA path, B_e rows (LORE) on vector ALUs
// ---------------------------------------------------------------------------
// B_e rows of a LoRE tile, one row per thread, on vector ALUs (the rank is too small for
// MFMA): delta[t][row] = sum_q B[row][q] U[t][q].  Each pass over kLoreChunk ranks issues
// the row's B loads first, then stages U for up to kLoreTok tokens in LDS.
template <int DT>
__device__ void lore_down_tile(const FfnArgs& a, int expert, int start, int n, int rt, float* s_u) {
    constexpr int L = Tr<DT>::kLaneK;  // elements per 16-byte load
    constexpr int kLoreChunk = 64;
    constexpr int NL = kLoreChunk / L;
    constexpr int kUPer = kLoreTok * kLoreChunk / kThreads;  // U values staged per thread
    const int tid = threadIdx.x;
    const int row = rt * kLoreRows + tid;
    const bool row_ok = row < a.d;
    const size_t brow = lore_b_elem(a, expert, row_ok ? row : 0, 0);
    const u32x4_t zero = {0u, 0u, 0u, 0u};
    for (int g0 = 0; g0 < n; g0 += kLoreTok) {
        const int nt = min(kLoreTok, n - g0);
        float acc[kLoreTok];
#pragma unroll
        for (int j = 0; j < kLoreTok; ++j) acc[j] = 0.f;
        for (int q0 = 0; q0 < a.r; q0 += kLoreChunk) {
            const int nq = min(kLoreChunk, a.r - q0);
            u32x4_t raw[NL];
#pragma unroll
            for (int i = 0; i < NL; ++i) raw[i] = (i * L < nq) ? Tr<DT>::load(a.lore_B, brow + q0 + i * L) : zero;
            float uv[kUPer];
#pragma unroll
            for (int i = 0; i < kUPer; ++i) {
                const int idx = tid + i * kThreads, j = idx / kLoreChunk, q = idx - j * kLoreChunk;
                uv[i] = (j < nt && q < nq) ? a.u[lore_u_elem(a, start, g0 + j, q0 + q)] : 0.f;
            }
#pragma unroll
            for (int i = 0; i < kUPer; ++i) s_u[tid + i * kThreads] = uv[i];
            __syncthreads();
            if (row_ok) {
#pragma unroll
                for (int i = 0; i < NL; ++i) {
                    if (i * L < nq) {
                        float bv[L];
                        if constexpr (DT == SPICE_BF16) {
                            const uint32_t wv[4] = {raw[i].x, raw[i].y, raw[i].z, raw[i].w};
#pragma unroll
                            for (int k = 0; k < 4; ++k) {
                                bv[2 * k] = __uint_as_float(wv[k] << 16);
                                bv[2 * k + 1] = __uint_as_float(wv[k] & 0xFFFF0000u);
                            }
                        } else {
                            bv[0] = __uint_as_float(raw[i].x); bv[1] = __uint_as_float(raw[i].y);
                            bv[2] = __uint_as_float(raw[i].z); bv[3] = __uint_as_float(raw[i].w);
                        }
#pragma unroll
                        for (int j = 0; j < kLoreTok; ++j) {
                            if (j < nt) {
#pragma unroll
                                for (int qq = 0; qq < L; ++qq) acc[j] += bv[qq] * s_u[j * kLoreChunk + i * L + qq];
                            }
                        }
                    }
                }
            }
            __syncthreads();
        }
        if (row_ok) {
#pragma unroll
            for (int j = 0; j < kLoreTok; ++j)
                if (j < nt) a.y_slots[lore_y_elem(a, start, g0 + j, row)] = acc[j];
        }
    }
}

template <int DT, int NA, int NB>
__device__ __forceinline__ void down_pass(const char* const (&a)[NA], const char* const (&hb)[NB], int kdim,
                                          int w, int quad, f32x4_t (&red)[kWaves][kDownRows][kTokTiles][64], int lane) {
    u32x4_t a0[NA][SPICE_GROUP_STEPS(NA, NB)];
    mma_first_a<DT, NA, NB>(a, kdim, w, a0);
    f32x4_t acc[NA][NB];
    wave_product<DT, NA, NB>(a, hb, kdim, w, quad, acc, a0);
#pragma unroll
    for (int rr = 0; rr < NA; ++rr)
#pragma unroll
        for (int j = 0; j < NB; ++j) red[w][rr][j][lane] = acc[rr][j];
}

// Down tile rt (R x 16 rows of W2, R = 1 or 2) of one group, the kind fixed at compile time:
// kKindHit reads H at the bucket positions and writes y_slots there; kKindShared reads the
// shared intermediate for tokens 0..T-1 and writes y_shared (times sgate[t] when set).
template <int DT, int KIND, int R = kDownRows>
__device__ void down_tile(const FfnArgs& a, const Group& g, int rt, f32x4_t (&red)[kWaves][kDownRows][kTokTiles][64]) {
    static_assert(KIND == kKindHit || KIND == kKindShared, "down tiles are HIT or shared");
    static_assert(R == 1 || R == kDownRows, "16 or 32 rows per down tile");
    using T_ = Tr<DT>;
    constexpr int es = (DT == SPICE_BF16) ? 2 : 4;
    const int lane = threadIdx.x & 63;
    const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);  // wave index, uniform
    const void* wbase = down_weights<KIND>(a);
    const void* hbase = down_inputs<KIND>(a);
    const DownBlock db = down_block<KIND>(a, g);
    const int kdim = db.kdim;
    int start, n;
    tile_entries<KIND>(a, g, start, n);
    const int m = lane & 15, quad = lane >> 4;
    const int dim0 = rt * kTileRows * R;
    const size_t kb = (size_t)quad * T_::kLaneK * es;
    const char* const aw[kDownRows] = {
        // tail rows read the last row; their outputs are dropped
        static_cast<const char*>(wbase) + (db.row0 + tile_row(rt, kTileRows * R, m, a.d)) * (size_t)kdim * es + kb,
        static_cast<const char*>(wbase) + (db.row0 + tile_row(rt, kTileRows * R, kTileRows + m, a.d)) * (size_t)kdim * es + kb};
    const char* const a1[1] = {aw[0]};
    for (int g0 = 0; g0 < n; g0 += 16 * kTokTiles) {
        const int ntt = min(kTokTiles, (n - g0 + 15) / 16);
        const char* const hb[kTokTiles] = {
            static_cast<const char*>(hbase) + (size_t)(start + tile_entry(g0, 0, m, n)) * db.ld * es + kb,
            static_cast<const char*>(hbase) + (size_t)(start + tile_entry(g0, 1, m, n)) * db.ld * es + kb};
        const char* const h1[1] = {hb[0]};
        if constexpr (R == 1) {
            if (ntt == 1) down_pass<DT, 1, 1>(a1, h1, kdim, w, quad, red, lane);
            else down_pass<DT, 1, 2>(a1, hb, kdim, w, quad, red, lane);
        } else {
            if (ntt == 1) down_pass<DT, kDownRows, 1>(aw, h1, kdim, w, quad, red, lane);
            else down_pass<DT, kDownRows, 2>(aw, hb, kdim, w, quad, red, lane);
        }
        __syncthreads();
        // wave w finalises (row tile, token tile) pair w
        const int rr = w % R, tt = w / R;
        if (tt < ntt) {
            f32x4_t s = red[0][rr][tt][lane];
#pragma unroll
            for (int ww = 1; ww < kWaves; ++ww) s += red[ww][rr][tt][lane];
            const int gi = g0 + tt * 16 + m;
            const int dim = dim0 + rr * 16 + quad * 4;
            if (gi < n && dim < a.d) {
                if constexpr (KIND == kKindShared) {
                    if (a.sgate) s *= a.sgate[gi];  // gated shared block
                    *reinterpret_cast<f32x4_t*>(a.y_shared + down_out_elem<KIND>(a, start, gi, dim)) = s;
                } else {
                    *reinterpret_cast<f32x4_t*>(a.y_slots + down_out_elem<KIND>(a, start, gi, dim)) = s;
                }
            }
        }
        __syncthreads();
    }
}

}  // namespace
}  // namespace spice
