// Grouped expert GEMMs for large token counts (prefill): the SwiGLU FFN of Eq. 6
// over every HIT expert's bucket and over all tokens for the shared block
// (Sec. 2.1, 4.2), as dense MFMA contractions.  bf16 operands, fp32 accumulation.
//
//   up   : H[pos][f] = silu(sum_k W1[f][k] x[k]) * (sum_k W3[f][k] x[k])   (bf16 out)
//   down : Y[pos][j] = sum_k W2[j][k] H[pos][k]                            (fp32 out)
//
// Block tile: 128 weight rows x 128 tokens x 64 k, 4 waves of 64 x 64.  For `up`
// the 128 weight rows are 64 W1 rows and the same 64 W3 rows, so each wave holds
// the gate and up sums of its 32 features and applies SwiGLU in registers.  The
// weight tile is the MFMA A operand and the token tile the B operand
// (v_mfma_f32_16x16x32_bf16): a lane ends with 4 consecutive features of one
// token, stored with one 8- (bf16) or 16-byte (fp32) write.
// Both tiles are staged through LDS, double buffered, rows padded to 144 bytes so
// that the 16 rows read by a fragment load land on disjoint bank groups.  Token
// rows of an expert are gathered through perm once per tile.
// Tiles: the shared block first, then the HIT experts in id order; inside a group
// the token tiles of one weight tile are consecutive (the weight tile is then
// served from L2), and consecutive tiles are kept on one XCD.
#include <hip/hip_runtime.h>

#include <algorithm>

#include "spice_internal.h"

namespace spice {
namespace {

constexpr int kThreads = 256;
constexpr int kBM = 128;            // weight rows per tile
constexpr int kBT = 128;            // tokens per tile
constexpr int kBK = 64;             // contraction per stage
constexpr int kRowBytes = kBK * 2;  // 128 bytes of a staged row
constexpr int kLdsRow = kRowBytes + 16;
constexpr int kTileLds = kBM * kLdsRow;       // one operand tile of one stage
constexpr int kStageLds = 2 * kTileLds;       // weights + tokens
constexpr int kChunks = kBM * kRowBytes / 16 / kThreads;  // 16-byte chunks per thread per operand tile
static_assert(kBM == kBT, "both operand tiles are staged with one layout");

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

__device__ __forceinline__ uint32_t bf16_rne(float f) {
    const uint32_t u = __float_as_uint(f);
    if ((u & 0x7FFFFFFFu) > 0x7F800000u) return 0x7FC0u;
    return (u + 0x7FFFu + ((u >> 16) & 1u)) >> 16;
}

__device__ __forceinline__ float silu(float u) { return u / (1.0f + __expf(-u)); }

// Logical tile of block b when the hardware deals blocks to the 8 XCDs round robin:
// each XCD gets one contiguous range of logical tiles (a bijection on [0, G)).
__device__ __forceinline__ int xcd_tile(int b, int G) {
    const int x = b & 7, per = G >> 3, rem = G & 7;
    const int first = x < rem ? x * (per + 1) : rem * (per + 1) + (x - rem) * per;
    return first + (b >> 3);
}

struct TileJob {
    const uint16_t* w;    // weight matrix of the group (rows of W13 or W2)
    const uint16_t* act;  // activations: x (up) or H / Hs (down)
    int kdim;             // contraction length
    int wrow0;            // first weight row of this tile (up: W1 row; W3 row = wrow0 + up_off)
    int up_off;           // up: row distance from W1 to W3 inside w
    int tok0, ntok;       // tile's first bucket position / token count of the group
    int start;            // group's first bucket position (HIT) or 0 (shared)
    bool gather;          // activation rows via perm (up of a HIT expert)
    int feat0;            // first output feature of the tile
    bool shared;
};

// Resolve logical tile L of a launch.  Returns false for tiles past the live work.
template <bool kUp>
__device__ bool resolve(const GemmArgs& a, int L, TileJob& j, int* s_scan) {
    const int lane = threadIdx.x & 63;
    const int nt_sh = kUp ? a.Is / 64 : a.d / kBM;  // weight tiles of the shared block
    const int nt_e = kUp ? a.I / 64 : a.d / kBM;    // weight tiles of a routed expert
    const int mt_sh = (a.T + kBT - 1) / kBT;
    const int tiles_sh = a.Is > 0 ? nt_sh * mt_sh : 0;
    if (L < tiles_sh) {
        const int n = L / mt_sh, m = L - n * mt_sh;
        j.w = kUp ? a.w13s : a.w2s;
        j.act = kUp ? a.x : a.hs;
        j.kdim = kUp ? a.d : a.Is;
        j.wrow0 = kUp ? n * 64 : n * kBM;
        j.up_off = a.Is;
        j.tok0 = m * kBT;
        j.ntok = a.T;
        j.start = 0;
        j.gather = false;
        j.feat0 = j.wrow0;
        j.shared = true;
        return true;
    }
    L -= tiles_sh;
    // HIT experts: tiles_e = ceil(n_e / kBT) * nt_e, in expert id order (one wave scans)
    if (threadIdx.x < 64) {
        int base = 0, found = -1;
        for (int e0 = 0; e0 < a.N && found < 0; e0 += 64) {
            const int e = e0 + lane;
            int st = 0, n = 0;
            if (e < a.N) {
                st = a.offsets[e];
                n = a.offsets[e + 1] - st;
            }
            const int tiles = n > 0 ? ((n + kBT - 1) / kBT) * nt_e : 0;
            int incl = tiles;
#pragma unroll
            for (int o = 1; o < 64; o <<= 1) {
                const int up = __shfl_up(incl, o);
                if (lane >= o) incl += up;
            }
            const int excl = base + incl - tiles;
            const bool mine = tiles > 0 && L >= excl && L < excl + tiles;
            const unsigned long long bal = __ballot(mine);
            if (bal) {
                const int src = __ffsll((long long)bal) - 1;
                if (lane == src) {
                    s_scan[0] = e;
                    s_scan[1] = st;
                    s_scan[2] = n;
                    s_scan[3] = L - excl;
                }
                found = 1;
            }
            base += __shfl(incl, 63);
        }
        if (lane == 0 && found < 0) s_scan[0] = -1;
    }
    __syncthreads();
    const int e = s_scan[0];
    if (e < 0) return false;
    const int st = s_scan[1], n = s_scan[2], t = s_scan[3];
    if (st < 0 || n <= 0 || st + n > a.T * a.K) {
        if (threadIdx.x == 0) atomicOr(&a.ctrl[kWordFlags], (uint32_t)SPICE_FLAG_BAD_INDEX);
        return false;
    }
    const int slot = a.resident_slot[e];
    if (slot < 0 || slot >= a.C) {
        if (threadIdx.x == 0) atomicOr(&a.ctrl[kWordFlags], (uint32_t)SPICE_FLAG_BAD_SLOT);
        return false;
    }
    const int mt = (n + kBT - 1) / kBT;
    const int nn = t / mt, m = t - nn * mt;
    if (kUp) {
        j.w = a.w13_pool + (size_t)slot * 2 * a.I * a.d;
        j.act = a.x;
        j.kdim = a.d;
        j.wrow0 = nn * 64;
        j.up_off = a.I;
    } else {
        j.w = a.w2_pool + (size_t)slot * a.d * a.I;
        j.act = a.h;
        j.kdim = a.I;
        j.wrow0 = nn * kBM;
        j.up_off = 0;
    }
    j.tok0 = m * kBT;
    j.ntok = n;
    j.start = st;
    j.gather = kUp;
    j.feat0 = j.wrow0;
    j.shared = false;
    return true;
}

template <bool kUp>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(2))) void expert_gemm_kernel(GemmArgs a) {
    extern __shared__ __align__(16) unsigned char s_lds[];
    __shared__ int s_scan[4];
    TileJob j;
    if (!resolve<kUp>(a, xcd_tile(blockIdx.x, gridDim.x), j, s_scan)) return;

    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const int wf = w & 1, wt = w >> 1;  // wave's feature half and token half of the tile
    const int m = lane & 15, quad = lane >> 4;

    // This thread's staging chunks: rows r_i = tid / 8 + 32 i, 16-byte column c = tid % 8.
    const int c16 = tid & 7;
    const uint16_t* wsrc[kChunks];
    const uint16_t* xsrc[kChunks];
#pragma unroll
    for (int i = 0; i < kChunks; ++i) {
        const int r = (tid >> 3) + 32 * i;
        int wr;
        if (kUp) wr = r < 64 ? j.wrow0 + r : j.wrow0 + j.up_off + (r - 64);
        else wr = j.wrow0 + r;
        wsrc[i] = j.w + (size_t)wr * j.kdim + c16 * 8;
        // token rows past the group's end read its last row; their outputs are dropped
        const int pos = min(j.tok0 + r, j.ntok - 1);
        int row;
        if (j.shared) {
            row = pos;
        } else if (j.gather) {
            const int s = a.perm[j.start + pos];
            if (s < 0 || s >= a.T * a.K) {
                atomicOr(&a.ctrl[kWordFlags], (uint32_t)SPICE_FLAG_BAD_INDEX);
                row = 0;
            } else {
                row = s / a.K;
            }
        } else {
            row = j.start + pos;
        }
        xsrc[i] = j.act + (size_t)row * j.kdim + c16 * 8;
    }

    f32x4_t acc[4][4];
#pragma unroll
    for (int s = 0; s < 4; ++s)
#pragma unroll
        for (int t = 0; t < 4; ++t) acc[s][t] = f32x4_t{0.f, 0.f, 0.f, 0.f};

    u32x4_t wreg[kChunks], xreg[kChunks];
    auto load_stage = [&](int kt) {
        const size_t off = (size_t)kt * kBK;
#pragma unroll
        for (int i = 0; i < kChunks; ++i) {
            wreg[i] = *reinterpret_cast<const u32x4_t*>(wsrc[i] + off);
            xreg[i] = *reinterpret_cast<const u32x4_t*>(xsrc[i] + off);
        }
    };
    auto store_stage = [&](int buf) {
        unsigned char* wl = s_lds + buf * kStageLds;
        unsigned char* xl = wl + kTileLds;
#pragma unroll
        for (int i = 0; i < kChunks; ++i) {
            const int r = (tid >> 3) + 32 * i;
            *reinterpret_cast<u32x4_t*>(wl + r * kLdsRow + c16 * 16) = wreg[i];
            *reinterpret_cast<u32x4_t*>(xl + r * kLdsRow + c16 * 16) = xreg[i];
        }
    };

    // Fragment rows of this wave: weights (A) and tokens (B).  For `up` the wave's
    // feature sub-tiles are W1 rows wf*32 + {0, 16} and the W3 rows 64 + the same.
    int frow[4], trow[4];
#pragma unroll
    for (int s = 0; s < 4; ++s) {
        frow[s] = kUp ? ((s < 2 ? 0 : 64) + wf * 32 + (s & 1) * 16 + m) : (wf * 64 + s * 16 + m);
        trow[s] = wt * 64 + s * 16 + m;
    }

    const int nk = j.kdim / kBK;
    load_stage(0);
    store_stage(0);
    __syncthreads();
    for (int kt = 0; kt < nk; ++kt) {
        const int buf = kt & 1;
        if (kt + 1 < nk) load_stage(kt + 1);
        const unsigned char* wl = s_lds + buf * kStageLds;
        const unsigned char* xl = wl + kTileLds;
#pragma unroll
        for (int ks = 0; ks < kBK / 32; ++ks) {
            const int kb = (ks * 32 + quad * 8) * 2;
            u32x4_t af[4], bf[4];
#pragma unroll
            for (int s = 0; s < 4; ++s) {
                af[s] = *reinterpret_cast<const u32x4_t*>(wl + frow[s] * kLdsRow + kb);
                bf[s] = *reinterpret_cast<const u32x4_t*>(xl + trow[s] * kLdsRow + kb);
            }
#pragma unroll
            for (int s = 0; s < 4; ++s)
#pragma unroll
                for (int t = 0; t < 4; ++t)
                    acc[s][t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, af[s]),
                                                                        __builtin_bit_cast(bf16x8_t, bf[t]),
                                                                        acc[s][t], 0, 0, 0);
        }
        if (kt + 1 < nk) store_stage(buf ^ 1);
        __syncthreads();
    }

    // Epilogue: lane holds features 4*quad .. +3 of sub-tile s for token m of sub-tile t.
#pragma unroll
    for (int t = 0; t < 4; ++t) {
        const int pos = j.tok0 + wt * 64 + t * 16 + m;
        if (pos >= j.ntok) continue;
        if (kUp) {
#pragma unroll
            for (int s = 0; s < 2; ++s) {
                const f32x4_t g = acc[s][t], u = acc[s + 2][t];
                const int f = j.feat0 + wf * 32 + s * 16 + quad * 4;
                uint2 p;
                p.x = bf16_rne(silu(g.x) * u.x) | (bf16_rne(silu(g.y) * u.y) << 16);
                p.y = bf16_rne(silu(g.z) * u.z) | (bf16_rne(silu(g.w) * u.w) << 16);
                uint16_t* dst = j.shared ? a.hs + (size_t)pos * a.Is : a.h + (size_t)(j.start + pos) * a.I;
                *reinterpret_cast<uint2*>(dst + f) = p;
            }
        } else {
#pragma unroll
            for (int s = 0; s < 4; ++s) {
                const int f = j.feat0 + wf * 64 + s * 16 + quad * 4;
                float* dst = j.shared ? a.y_shared + (size_t)pos * a.d : a.y_slots + (size_t)(j.start + pos) * a.d;
                *reinterpret_cast<f32x4_t*>(dst + f) = acc[s][t];
            }
        }
    }
}

}  // namespace

bool expert_gemm_applies(const FfnArgs& a) {
    if (a.dtype != SPICE_BF16 || a.T < kGemmMinTokens || a.d % kBM || a.d % kBK || a.I % 64 || a.Is % 64)
        return false;
    // the double-buffered tiles need more LDS than the 64 KiB every AMD GPU offers
    static int lds_per_block[64] = {0};
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return false;
    if (lds_per_block[dev] == 0) {
        int v = 0;
        if (hipDeviceGetAttribute(&v, hipDeviceAttributeMaxSharedMemoryPerBlock, dev) != hipSuccess) return false;
        lds_per_block[dev] = v;
    }
    return lds_per_block[dev] >= 2 * kStageLds;
}

hipError_t launch_expert_gemm(const FfnArgs& f, bool hit, bool shared, hipStream_t s) {
    GemmArgs a{};
    a.T = f.T; a.d = f.d; a.N = f.N; a.K = f.K; a.C = f.C; a.I = f.I; a.Is = shared ? f.Is : 0;
    a.x = static_cast<const uint16_t*>(f.x);
    a.perm = f.perm;
    a.offsets = f.offsets;  // the HIT class comes first
    a.resident_slot = f.resident_slot;
    a.w13_pool = static_cast<const uint16_t*>(f.w13_pool);
    a.w2_pool = static_cast<const uint16_t*>(f.w2_pool);
    a.w13s = static_cast<const uint16_t*>(f.w13s);
    a.w2s = static_cast<const uint16_t*>(f.w2s);
    a.h = static_cast<uint16_t*>(f.h);
    a.hs = static_cast<uint16_t*>(f.hs);
    a.y_slots = f.y_slots;
    a.y_shared = f.y_shared;
    a.ctrl = f.ctrl;
    if (!hit) a.N = 0;  // no expert tiles
    // upper bound of the tile count: sum_e ceil(n_e / kBT) <= T*K / kBT + min(N, C)
    const long long mt_hit = hit ? (long long)a.T * a.K / kBT + std::min(a.N, a.C) : 0;
    const long long mt_sh = (a.T + kBT - 1) / kBT;
    const long long up_tiles = (a.Is > 0 ? mt_sh * (a.Is / 64) : 0) + mt_hit * (a.I / 64);
    const long long dn_tiles = (a.Is > 0 ? mt_sh * (a.d / kBM) : 0) + mt_hit * (a.d / kBM);
    if (up_tiles == 0) return hipSuccess;
    if (up_tiles > 0x7FFFFFFFll || dn_tiles > 0x7FFFFFFFll) return hipErrorInvalidValue;
    const size_t lds = 2 * kStageLds;
    hipLaunchKernelGGL(expert_gemm_kernel<true>, dim3((unsigned)up_tiles), dim3(kThreads), lds, s, a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(expert_gemm_kernel<false>, dim3((unsigned)dn_tiles), dim3(kThreads), lds, s, a);
    return hipGetLastError();
}

}  // namespace spice
