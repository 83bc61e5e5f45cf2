// Grouped expert FFN for the resident (HIT) experts and the shared block (Eq. 6;
// Sec. 2.1, 4.2), and the LoRE correction B_e (A_e x) of low-confidence misses (Eq. 9).
//
// Two launches:
//   up   : per 16-row tile of W1/W3 (or of A_e): H = silu(X W1^T) * (X W3^T)
//          (or U = X A_e^T); X = the tokens of the expert's bucket.
//   down : per 32-row tile of W2: Y = H W2^T; per 256-row tile of B_e: delta = U B_e^T.
// A block (4 waves) owns one tile; its waves split the contraction dimension and
// add their partial MFMA accumulators through LDS.  The weight tile is the MFMA
// A operand (16 rows x 32 k per bf16 step, one 16-byte load per lane), the
// tokens are the B operand (16 columns, zero-padded), fp32 accumulation.
// Blocks map to (expert ordinal, row tile); the expert ordinal is resolved on
// the device from the bucket offsets, so no host synchronisation is needed and
// blocks beyond the live experts exit at once.
#include <hip/hip_runtime.h>

#include "spice_internal.h"

namespace spice {
namespace {

constexpr int kThreads = 256;
constexpr int kWaves = 4;
constexpr int kTokTiles = 2;        // token tiles of 16 per pass
constexpr int kDownRows = 2;        // 16-row tiles per down block
constexpr int kLoreRows = 256;      // B_e rows per LoRE block (one per thread)
constexpr int kLoreTok = 16;        // tokens per LoRE pass

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

template <int DT>
struct Tr;

template <>
struct Tr<SPICE_BF16> {
    static constexpr int kStep = 32;   // contraction elements per MFMA step
    static constexpr int kLaneK = 8;   // elements each lane loads per step (16 bytes)
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

struct Group {
    int e, start, n;
};

// The j-th expert (ascending id) whose bucket of class c is non-empty.
__device__ bool find_group(const FfnArgs& a, int c, int j, Group& g) {
    const int lane = threadIdx.x & 63;
    const int32_t* off = a.offsets + c * (a.N + 1);
    const unsigned long long lt = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
    int seen = 0;
    for (int base = 0; base < a.N; base += 64) {
        const int e = base + lane;
        int st = 0, n = 0;
        if (e < a.N) { st = off[e]; n = off[e + 1] - st; }
        const unsigned long long m = __ballot(n > 0);
        const int cnt = __popcll(m);
        if (j < seen + cnt) {
            const bool mine = n > 0 && __popcll(m & lt) == j - seen;
            const int src = __ffsll((long long)__ballot(mine)) - 1;
            g.e = base + src;
            g.start = __shfl(st, src);
            g.n = __shfl(n, src);
            if (g.start < 0 || g.n < 0 || g.start + g.n > a.T * a.K) {
                if (lane == 0) atomicOr(&a.ctrl[kWordFlags], (uint32_t)SPICE_FLAG_BAD_INDEX);
                return false;
            }
            return true;
        }
        seen += cnt;
    }
    return false;
}

// Token of bucket position pos (or -1, flagged, if perm holds garbage).
__device__ __forceinline__ int token_of(const FfnArgs& a, int pos) {
    const int s = a.perm[pos];
    if (s < 0 || s >= a.T * a.K) {
        atomicOr(&a.ctrl[kWordFlags], (uint32_t)SPICE_FLAG_BAD_INDEX);
        return -1;
    }
    return s / a.K;
}

enum : int { kKindHit = 0, kKindShared = 1, kKindLore = 2 };

// Decode a block index into (kind, group, row tile).  Segments in order: HIT
// experts x row tiles, the shared block's row tiles, LORE experts x row tiles.
struct Tile {
    int kind, ordinal, rt;
};
__device__ __forceinline__ bool decode_tile(int b, int nhit, int thit, int tsh, int nlore, int tlore, Tile& t) {
    if (b < nhit * thit) { t = {kKindHit, b / thit, b % thit}; return true; }
    b -= nhit * thit;
    if (b < tsh) { t = {kKindShared, 0, b}; return true; }
    b -= tsh;
    if (b < nlore * tlore) { t = {kKindLore, b / tlore, b % tlore}; return true; }
    return false;
}

struct UpGrid {
    int nhit, thit, tsh, nlore, tlore;
};

// ---------------------------------------------------------------------------
// up: gate/up SwiGLU rows (HIT, shared) or A_e rows (LORE)
// ---------------------------------------------------------------------------
template <int DT>
__global__ __launch_bounds__(kThreads) void ffn_up_kernel(FfnArgs a, UpGrid gr) {
    __shared__ f32x4_t red[kWaves][kTokTiles][2][64];
    using T_ = Tr<DT>;
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    Tile tile;
    if (!decode_tile(blockIdx.x, gr.nhit, gr.thit, gr.tsh, gr.nlore, gr.tlore, tile)) return;

    Group g{0, 0, a.T};
    const void* wbase;
    size_t gate_row0, up_row0;
    int nrows;
    bool has_up = true;
    if (tile.kind == kKindHit) {
        if (!find_group(a, SPICE_CLASS_HIT, tile.ordinal, g)) return;
        const int slot = a.resident_slot[g.e];
        if (slot < 0 || slot >= a.C) {
            if (threadIdx.x == 0) atomicOr(&a.ctrl[kWordFlags], (uint32_t)SPICE_FLAG_BAD_SLOT);
            return;
        }
        wbase = a.w13_pool;
        nrows = a.I;
        gate_row0 = (size_t)slot * 2 * a.I + (size_t)tile.rt * 16;
        up_row0 = gate_row0 + a.I;
    } else if (tile.kind == kKindShared) {
        wbase = a.w13s;
        nrows = a.Is;
        gate_row0 = (size_t)tile.rt * 16;
        up_row0 = gate_row0 + a.Is;
    } else {
        if (!find_group(a, SPICE_CLASS_LORE, tile.ordinal, g)) return;
        wbase = a.lore_A;
        nrows = a.r;
        gate_row0 = (size_t)g.e * a.r + (size_t)tile.rt * 16;
        up_row0 = 0;
        has_up = false;
    }

    const int m = lane & 15;              // A row / B column owned by this lane
    const int quad = lane >> 4;           // which k sub-chunk, and which 4 output rows
    const bool row_ok = tile.rt * 16 + m < nrows;
    const size_t a_gate = (gate_row0 + m) * (size_t)a.d;
    const size_t a_up = (up_row0 + m) * (size_t)a.d;
    const int koff = quad * T_::kLaneK;
    const int nks = (a.d + T_::kStep - 1) / T_::kStep;
    const int ks0 = w * nks / kWaves, ks1 = (w + 1) * nks / kWaves;
    const u32x4_t zero = {0u, 0u, 0u, 0u};

    for (int g0 = 0; g0 < g.n; g0 += 16 * kTokTiles) {
        const int ntt = min(kTokTiles, (g.n - g0 + 15) / 16);
        size_t xoff[kTokTiles];
        bool xok[kTokTiles];
#pragma unroll
        for (int tt = 0; tt < kTokTiles; ++tt) {
            const int gi = g0 + tt * 16 + m;
            int t = -1;
            if (tt < ntt && gi < g.n) t = (tile.kind == kKindShared) ? gi : token_of(a, g.start + gi);
            xok[tt] = t >= 0;
            xoff[tt] = (size_t)(t >= 0 ? t : 0) * a.d;
        }
        f32x4_t acc[2][kTokTiles];
#pragma unroll
        for (int tt = 0; tt < kTokTiles; ++tt) acc[0][tt] = acc[1][tt] = f32x4_t{0.f, 0.f, 0.f, 0.f};

#pragma unroll 2
        for (int ks = ks0; ks < ks1; ++ks) {
            const int k = ks * T_::kStep + koff;
            const bool kin = k < a.d;
            const u32x4_t ag = (row_ok && kin) ? T_::load(wbase, a_gate + k) : zero;
            const u32x4_t au = (has_up && row_ok && kin) ? T_::load(wbase, a_up + k) : zero;
#pragma unroll
            for (int tt = 0; tt < kTokTiles; ++tt) {
                if (tt < ntt) {
                    const u32x4_t b = (xok[tt] && kin) ? T_::load(a.x, xoff[tt] + k) : zero;
                    acc[0][tt] = T_::mma(ag, b, acc[0][tt]);
                    if (has_up) acc[1][tt] = T_::mma(au, b, acc[1][tt]);
                }
            }
        }

#pragma unroll
        for (int tt = 0; tt < kTokTiles; ++tt) {
            red[w][tt][0][lane] = acc[0][tt];
            red[w][tt][1][lane] = acc[1][tt];
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
            const int gi = g0 + tt * 16 + m;   // output column = token of lane m
            const int row = tile.rt * 16 + quad * 4;
            if (gi < g.n && row < nrows) {
                if (tile.kind == kKindLore) {
                    *reinterpret_cast<f32x4_t*>(a.u + (size_t)(g.start + gi) * a.r + row) = sg;
                } else {
                    f32x4_t h;
                    h.x = silu(sg.x) * su.x;
                    h.y = silu(sg.y) * su.y;
                    h.z = silu(sg.z) * su.z;
                    h.w = silu(sg.w) * su.w;
                    if (tile.kind == kKindHit)
                        T_::store4(a.h, (size_t)(g.start + gi) * a.I + row, h);
                    else
                        T_::store4(a.hs, (size_t)gi * a.Is + row, h);
                }
            }
        }
        __syncthreads();
    }
}

// ---------------------------------------------------------------------------
// down: W2 rows (HIT, shared) with the MFMA path, B_e rows (LORE) on vector ALUs
// ---------------------------------------------------------------------------
template <int DT>
__device__ void lore_down_tile(const FfnArgs& a, const Group& g, int rt, float* s_u) {
    const int tid = threadIdx.x;
    const int row = rt * kLoreRows + tid;
    const bool row_ok = row < a.d;
    const size_t brow = ((size_t)g.e * a.d + (row_ok ? row : 0)) * (size_t)a.r;
    for (int g0 = 0; g0 < g.n; g0 += kLoreTok) {
        const int nt = min(kLoreTok, g.n - g0);
        for (int i = tid; i < nt * a.r; i += kThreads) {
            const int j = i / a.r, q = i - j * a.r;
            s_u[j * a.r + q] = a.u[(size_t)(g.start + g0 + j) * a.r + q];
        }
        __syncthreads();
        float acc[kLoreTok];
#pragma unroll
        for (int j = 0; j < kLoreTok; ++j) acc[j] = 0.f;
        if (row_ok) {
            for (int q = 0; q < a.r; q += Tr<DT>::kLaneK) {
                const u32x4_t raw = Tr<DT>::load(a.lore_B, brow + q);
                float bv[8];
                if (DT == SPICE_BF16) {
                    const uint32_t wv[4] = {raw.x, raw.y, raw.z, raw.w};
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        bv[2 * i] = __uint_as_float(wv[i] << 16);
                        bv[2 * i + 1] = __uint_as_float(wv[i] & 0xFFFF0000u);
                    }
                } else {
                    bv[0] = __uint_as_float(raw.x); bv[1] = __uint_as_float(raw.y);
                    bv[2] = __uint_as_float(raw.z); bv[3] = __uint_as_float(raw.w);
                }
#pragma unroll
                for (int j = 0; j < kLoreTok; ++j) {
                    if (j < nt) {
#pragma unroll
                        for (int qq = 0; qq < Tr<DT>::kLaneK; ++qq) acc[j] += bv[qq] * s_u[j * a.r + q + qq];
                    }
                }
            }
#pragma unroll
            for (int j = 0; j < kLoreTok; ++j)
                if (j < nt) a.y_slots[(size_t)(g.start + g0 + j) * a.d + row] = acc[j];
        }
        __syncthreads();
    }
}

template <int DT>
__global__ __launch_bounds__(kThreads) void ffn_down_kernel(FfnArgs a, UpGrid gr) {
    __shared__ f32x4_t red[kWaves][kDownRows][kTokTiles][64];
    using T_ = Tr<DT>;
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    Tile tile;
    if (!decode_tile(blockIdx.x, gr.nhit, gr.thit, gr.tsh, gr.nlore, gr.tlore, tile)) return;

    Group g{0, 0, a.T};
    if (tile.kind == kKindLore) {
        if (!find_group(a, SPICE_CLASS_LORE, tile.ordinal, g)) return;
        lore_down_tile<DT>(a, g, tile.rt, reinterpret_cast<float*>(&red[0][0][0][0]));
        return;
    }
    const void* wbase;
    const void* hbase;
    int kdim;
    size_t row0;
    if (tile.kind == kKindHit) {
        if (!find_group(a, SPICE_CLASS_HIT, tile.ordinal, g)) return;
        const int slot = a.resident_slot[g.e];
        if (slot < 0 || slot >= a.C) {
            if (threadIdx.x == 0) atomicOr(&a.ctrl[kWordFlags], (uint32_t)SPICE_FLAG_BAD_SLOT);
            return;
        }
        wbase = a.w2_pool;
        hbase = a.h;
        kdim = a.I;
        row0 = (size_t)slot * a.d;
    } else {
        wbase = a.w2s;
        hbase = a.hs;
        kdim = a.Is;
        row0 = 0;
    }

    const int m = lane & 15, quad = lane >> 4;
    const int dim0 = tile.rt * 16 * kDownRows;
    size_t aoff[kDownRows];
    bool aok[kDownRows];
#pragma unroll
    for (int rr = 0; rr < kDownRows; ++rr) {
        const int dim = dim0 + rr * 16 + m;
        aok[rr] = dim < a.d;
        aoff[rr] = (row0 + (aok[rr] ? dim : 0)) * (size_t)kdim;
    }
    const int koff = quad * T_::kLaneK;
    const int nks = (kdim + T_::kStep - 1) / T_::kStep;
    const int ks0 = w * nks / kWaves, ks1 = (w + 1) * nks / kWaves;
    const u32x4_t zero = {0u, 0u, 0u, 0u};

    for (int g0 = 0; g0 < g.n; g0 += 16 * kTokTiles) {
        const int ntt = min(kTokTiles, (g.n - g0 + 15) / 16);
        size_t hoff[kTokTiles];
        bool hok[kTokTiles];
#pragma unroll
        for (int tt = 0; tt < kTokTiles; ++tt) {
            const int gi = g0 + tt * 16 + m;
            hok[tt] = tt < ntt && gi < g.n;
            const size_t hrow = (tile.kind == kKindShared) ? (size_t)gi : (size_t)(g.start + gi);
            hoff[tt] = (hok[tt] ? hrow : 0) * (size_t)kdim;
        }
        f32x4_t acc[kDownRows][kTokTiles];
#pragma unroll
        for (int rr = 0; rr < kDownRows; ++rr)
#pragma unroll
            for (int tt = 0; tt < kTokTiles; ++tt) acc[rr][tt] = f32x4_t{0.f, 0.f, 0.f, 0.f};

#pragma unroll 2
        for (int ks = ks0; ks < ks1; ++ks) {
            const int k = ks * T_::kStep + koff;
            const bool kin = k < kdim;
            u32x4_t av[kDownRows];
#pragma unroll
            for (int rr = 0; rr < kDownRows; ++rr) av[rr] = (aok[rr] && kin) ? T_::load(wbase, aoff[rr] + k) : zero;
#pragma unroll
            for (int tt = 0; tt < kTokTiles; ++tt) {
                if (tt < ntt) {
                    const u32x4_t b = (hok[tt] && kin) ? T_::load(hbase, hoff[tt] + k) : zero;
#pragma unroll
                    for (int rr = 0; rr < kDownRows; ++rr) acc[rr][tt] = T_::mma(av[rr], b, acc[rr][tt]);
                }
            }
        }

#pragma unroll
        for (int rr = 0; rr < kDownRows; ++rr)
#pragma unroll
            for (int tt = 0; tt < kTokTiles; ++tt) red[w][rr][tt][lane] = acc[rr][tt];
        __syncthreads();
        // wave w finalises (row tile, token tile) pair w
        const int rr = w % kDownRows, tt = w / kDownRows;
        if (tt < ntt) {
            f32x4_t s = red[0][rr][tt][lane];
#pragma unroll
            for (int ww = 1; ww < kWaves; ++ww) s += red[ww][rr][tt][lane];
            const int gi = g0 + tt * 16 + m;
            const int dim = dim0 + rr * 16 + quad * 4;
            if (gi < g.n && dim < a.d) {
                float* dst = (tile.kind == kKindShared) ? a.y_shared + (size_t)gi * a.d
                                                        : a.y_slots + (size_t)(g.start + gi) * a.d;
                *reinterpret_cast<f32x4_t*>(dst + dim) = s;
            }
        }
        __syncthreads();
    }
}

}  // namespace

hipError_t launch_expert_ffn(const FfnArgs& a, hipStream_t s) {
    const int slots = a.T * a.K;
    const bool hit = (a.groups & kDoHit) != 0;
    const bool shared = (a.groups & kDoShared) != 0 && a.Is > 0;
    const bool lore = (a.groups & kDoLore) != 0 && a.r > 0;
    UpGrid up{0, 1, 0, 0, 1}, dn{0, 1, 0, 0, 1};
    if (hit) {
        up.nhit = dn.nhit = min(min(a.N, a.C), slots);
        up.thit = (a.I + 15) / 16;
        dn.thit = (a.d + 16 * kDownRows - 1) / (16 * kDownRows);
    }
    if (shared) {
        up.tsh = (a.Is + 15) / 16;
        dn.tsh = (a.d + 16 * kDownRows - 1) / (16 * kDownRows);
    }
    if (lore) {
        up.nlore = dn.nlore = min(a.N, slots);
        up.tlore = (a.r + 15) / 16;
        dn.tlore = (a.d + kLoreRows - 1) / kLoreRows;
    }
    const long long nup = (long long)up.nhit * up.thit + up.tsh + (long long)up.nlore * up.tlore;
    const long long ndn = (long long)dn.nhit * dn.thit + dn.tsh + (long long)dn.nlore * dn.tlore;
    if (nup == 0) return hipSuccess;
    if (a.dtype == SPICE_BF16) {
        hipLaunchKernelGGL(ffn_up_kernel<SPICE_BF16>, dim3((unsigned)nup), dim3(kThreads), 0, s, a, up);
        hipLaunchKernelGGL(ffn_down_kernel<SPICE_BF16>, dim3((unsigned)ndn), dim3(kThreads), 0, s, a, dn);
    } else {
        hipLaunchKernelGGL(ffn_up_kernel<SPICE_F32>, dim3((unsigned)nup), dim3(kThreads), 0, s, a, up);
        hipLaunchKernelGGL(ffn_down_kernel<SPICE_F32>, dim3((unsigned)ndn), dim3(kThreads), 0, s, a, dn);
    }
    return hipGetLastError();
}

}  // namespace spice
