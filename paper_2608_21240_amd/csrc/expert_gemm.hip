// Grouped expert GEMMs for large token counts (prefill): the SwiGLU FFN of Eq. 6
// over every HIT expert's bucket and over all tokens for the shared block
// (Sec. 2.1, 4.2), as dense MFMA contractions.  bf16 operands, fp32 accumulation.
//
//   up   : H[pos][f] = silu(sum_k W1[f][k] x[k]) * (sum_k W3[f][k] x[k])   (bf16 out)
//   down : Y[pos][j] = sum_k W2[j][k] H[pos][k]                            (fp32 out)
//
// Block tile: 256 weight rows x 256 tokens, 64 k per stage, 8 waves of 128 weight rows x
// 64 tokens (LDS traffic is 43 flop per byte read).  For `up` the 256 weight rows are 128
// W1 rows and the same 128 W3 rows, so each wave holds the gate and up sums of its 64
// features and applies SwiGLU in registers.  The weight tile is the MFMA A operand and
// the token tile the B operand (v_mfma_f32_16x16x32_bf16): a lane ends with 4 consecutive
// features of one token, stored with one 8- (bf16) or 16-byte (fp32) write.  A wave's
// token sub-tiles are interleaved with the other waves' (rows 64 t + 16 wt), so the ragged
// last tile of an expert spreads over the SIMDs and sub-tiles without a live token issue
// no MFMA.
// Both tiles are staged through LDS (two stages, 128 KiB: one block per CU) in
// 128-byte rows whose 16-byte chunks are XOR-swizzled by row (chunk c of row r at
// c ^ ((r >> 1) & 7)), so fragment reads are free of bank conflicts.  The global loads of
// the next stage go straight to LDS (global_load_lds_dwordx4, no staging registers), issued
// before the MFMAs of the current one by waves 0-3 only.  Token rows of an expert are
// gathered through perm once per tile.
// Tiles: the shared block first, then the HIT experts in id order; inside a group
// the token tiles of one weight tile are consecutive (the weight tile is then
// served from L2), and consecutive tiles are kept on one XCD.
#include <hip/hip_runtime.h>

#include <algorithm>

#include "spice_internal.h"

namespace spice {
namespace {

constexpr int kWaveT = 64;                     // tokens per wave (a wave holds 128 features x kWaveT)
constexpr int kThreads = 64 * 2 * (256 / kWaveT);  // 2 (features) x 256 / kWaveT (tokens) waves
constexpr int kBM = 256;                       // weight rows per tile
constexpr int kBT = 256;                       // tokens per tile
constexpr int kBK = 64;                        // contraction per stage (32 or 64)
constexpr int kWavesPerEU = kWaveT == 128 ? 1 : 2;  // waves per SIMD the register budget targets
constexpr int kTS = kWaveT / 16;               // token sub-tiles per wave
constexpr int kTStride = 16 * (kBT / kWaveT);  // tile rows between a wave's token sub-tiles
constexpr int kXcdBlocks = 32;                 // blocks one XCD runs at a time (32 CUs, 1 block each)
constexpr int kRowBytes = kBK * 2;             // bytes of a staged row
constexpr int kCPR = kBK / 8;                  // 16-byte chunks per staged row
constexpr int kWTile = kBM * kRowBytes;        // weight tile of one stage
constexpr int kStageLds = (kBM + kBT) * kRowBytes;
constexpr int kLoaders = kThreads / 2;         // waves 0-3 issue every global load, one per SIMD
constexpr int kRowStep = kLoaders / kCPR;      // staging rows between a loader's chunks
constexpr int kWChunks = kBM * kCPR / kLoaders;  // 16-byte weight chunks per loader per stage
constexpr int kXChunks = kBT * kCPR / kLoaders;  // 16-byte token chunks per loader per stage
constexpr int kUpFeat = kBM / 2;               // features of an up tile (W1 rows = W3 rows)
static_assert(kBK == 32 || kBK == 64, "a stage is one or two MFMA k-steps");

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

__device__ __forceinline__ uint32_t bf16_rne(float f) {
    const uint32_t u = __float_as_uint(f);
    if ((u & 0x7FFFFFFFu) > 0x7F800000u) return 0x7FC0u;
    return (u + 0x7FFFu + ((u >> 16) & 1u)) >> 16;
}

__device__ __forceinline__ float silu(float u) { return u / (1.0f + __expf(-u)); }

// Logical tile of block b.  The hardware deals blocks to the 8 XCDs round robin
// (block b to XCD b % 8).  Here every round of 8 x 32 blocks gives each XCD 32
// consecutive logical tiles (neighbouring tiles share operands in that XCD's L2),
// and the rounds alternate over all XCDs so that long tiles at the front of the
// order spread over the whole chip.  A final partial round keeps block order; the
// map is a bijection on [0, G).
__device__ __forceinline__ int xcd_tile(int b, int G) {
    constexpr int kRound = 8 * kXcdBlocks;
    if (b >= (G / kRound) * kRound) return b;
    const int x = b & 7, slot = b >> 3;
    return (slot / kXcdBlocks) * kRound + x * kXcdBlocks + slot % kXcdBlocks;
}

struct TileJob {
    const uint16_t* w;    // weight matrix of the group (rows of W13 or W2)
    const uint16_t* act;  // activations: x (up) or H / Hs (down)
    int kdim;             // contraction length
    int ld;               // row stride (elements) of the activations inside one stage
    uint32_t kst;         // elements between consecutive stages of one activation row
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
    const int nt_sh = kUp ? a.Is / kUpFeat : a.d / kBM;  // weight tiles of the shared block
    const int nt_e = kUp ? a.I / kUpFeat : a.d / kBM;    // weight tiles of a routed expert
    const int mt_sh = (a.T + kBT - 1) / kBT;
    const int tiles_sh = a.Is > 0 ? nt_sh * mt_sh : 0;
    if (L < tiles_sh) {
        // groups of sn weight tiles x sm token tiles (about one XCD's worth of blocks)
        // run together and share their operand tiles in that XCD's L2
        const int sn = kUp ? a.super_up[0] : a.super_dn[0], sm = kUp ? a.super_up[1] : a.super_dn[1];
        const int g = L / (sn * sm), in = L - g * (sn * sm);
        const int mg = mt_sh / sm;
        const int n = (g / mg) * sn + in / sm;
        const int m = (g % mg) * sm + in % sm;
        j.w = kUp ? a.w13s : a.w2s;
        j.act = kUp ? a.x : a.hs;
        j.kdim = kUp ? a.d : a.Is;
        j.ld = kUp ? a.d : kBK;
        j.kst = kUp ? kBK : (uint32_t)a.T * kBK;
        j.wrow0 = kUp ? n * kUpFeat : n * kBM;
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
        j.ld = a.d;
        j.kst = kBK;
        j.wrow0 = nn * kUpFeat;
        j.up_off = a.I;
    } else {
        j.w = a.w2_pool + (size_t)slot * a.d * a.I;
        j.act = a.h;
        j.kdim = a.I;
        j.ld = kBK;
        j.kst = (uint32_t)a.T * a.K * kBK;
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

// Byte offset of 16-byte chunk c of staged row r inside an operand tile.
// XOR swizzle of the 16-byte chunks of a staged row.  Measured on gfx950 with the
// LDS bank-conflict counter: 128-byte rows swizzled by (r >> 1) & 7 read 16 rows x 4
// chunks per ds_read_b128 and write 8 chunks per row without conflicts, where padded
// rows, 64-byte rows and unswizzled rows do not.
__device__ __forceinline__ uint32_t lds_off(int r, int c) {
    const int sw = kBK == 64 ? ((r >> 1) & 7) : ((r >> 2) & 3);
    return (uint32_t)(r * kRowBytes + ((c ^ sw) << 4));
}

// 16 bytes from this lane's global address to LDS byte lds + 16 * lane, for an lds address
// uniform over the wave (global_load_lds_dwordx4; counted by vmcnt, not lgkmcnt).  Device
// pass only: the host pass of a kernel naming this target builtin would lose its launch stub.
__device__ __forceinline__ void load_lds16(const void* g, void* lds) {
#if defined(__HIP_DEVICE_COMPILE__)
    __builtin_amdgcn_global_load_lds(g, lds, 16, 0, 0);
#endif
}

template <bool kUp>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(kWavesPerEU))) void expert_gemm_kernel(
    GemmArgs a) {
    extern __shared__ __align__(16) unsigned char s_lds[];
    __shared__ int s_scan[4];
    TileJob j;
    if (!resolve<kUp>(a, xcd_tile(blockIdx.x, gridDim.x), j, s_scan)) return;

    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    // wave's feature half and token lane group: token sub-tile t of the wave holds the tile's
    // rows kTStride t + 16 wt .. + 15, so a ragged last tile spreads over the SIMDs
    const int wf = w & 1, wt = __builtin_amdgcn_readfirstlane(w >> 1);
    const int m = lane & 15, quad = lane >> 4;

    // Staging: waves 0-3 (one per SIMD) issue all of a stage's loads, so waves 4-7 never wait
    // behind a queue of loads and keep their SIMD's MFMAs going at the start of a stage.  A
    // wave's direct load (global_load_lds_dwordx4) writes 64 x 16 bytes to consecutive LDS:
    // 8 staged rows of 8 chunks.  Lane l fills LDS chunk l % 8 of row r0 = tid / kCPR (+
    // kRowStep i), which holds the row's chunk (l % 8) ^ swizzle(row), so that is the chunk
    // it fetches.  Weight rows step by a constant, so one 32-bit element offset (from the
    // group's uniform base pointer) and uniform deltas address them; token rows are gathered.
    const int r0 = (tid % kLoaders) / kCPR;
    const bool loader = tid < kLoaders;
    static_assert(kRowStep % 16 == 0 && kUpFeat % kRowStep == 0, "staging rows keep their swizzle");
    static_assert(kThreads % 64 == 0 && 64 % kCPR == 0, "a wave stages whole rows");
    const int c16 = (int)((uint32_t)(lds_off(r0, tid % kCPR) % kRowBytes) >> 4);  // the chunk landing at this lane's slot
    const uint32_t woff0 = (uint32_t)(j.wrow0 + r0) * (uint32_t)j.kdim + c16 * 8;
    auto wrow_delta = [&](int i) -> uint32_t {  // rows between chunk 0 and chunk i (uniform)
        const int r = kRowStep * i;
        if (kUp && r >= kUpFeat) return (uint32_t)(j.up_off + r - kUpFeat) * (uint32_t)j.kdim;
        return (uint32_t)r * (uint32_t)j.kdim;
    };
    // element offsets of a loader's token rows, kept in LDS (each loader reads back only its
    // own) rather than in registers, which the accumulators and fragments fill
    __shared__ uint32_t s_xoff[kXChunks][kLoaders];
    if (loader) {
#pragma unroll
        for (int i = 0; i < kXChunks; ++i) {
            // token rows past the group's end read its last row; their outputs are dropped
            const int pos = min(j.tok0 + r0 + kRowStep * i, j.ntok - 1);
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
            s_xoff[i][tid] = (uint32_t)row * (uint32_t)j.ld + c16 * 8;
        }
    }
    const uint16_t* __restrict__ wbase = j.w;
    const uint16_t* __restrict__ xbase = j.act;

    f32x4_t acc[8][kTS];
#pragma unroll
    for (int s = 0; s < 8; ++s)
#pragma unroll
        for (int t = 0; t < kTS; ++t) acc[s][t] = f32x4_t{0.f, 0.f, 0.f, 0.f};

    // LDS addresses.  The swizzle of row r depends on (r >> 1) & 7, which steps of 16
    // rows leave unchanged, so every sub-tile / staging chunk is a constant offset from
    // one base.  Fragments of k-step 0; with kBK = 64, k-step 1 reads chunk c ^ 4, i.e.
    // the address with bit 6 flipped.  Weights (A): for `up` the wave's feature
    // sub-tiles 0..3 are W1 rows wf*64 + 16 s and 4..7 the W3 rows kUpFeat + the same.
    const uint32_t fbase = lds_off(kUp ? wf * 64 + m : wf * 128 + m, quad);
    const uint32_t tbase = kWTile + lds_off(wt * 16 + m, quad);
    // token sub-tiles of this wave with a live row; the others issue no MFMA
    const int nlive = min(kTS, max(0, (j.ntok - j.tok0 - 16 * wt + kTStride - 1) / kTStride));
    auto frag_row = [](int s) { return kUp ? (s & 3) * 16 + (s >> 2) * kUpFeat : s * 16; };

    const int nk = j.kdim / kBK;
    // Stage kt goes straight from global memory into LDS buffer buf: chunk i of this loader
    // lane lands in its wave's 1 KiB run of the chunk's rows (lane l at byte 16 l).
    auto load = [&](int buf, int kt) {  // loaders only
        if (!loader) return;
        const uint32_t o = (uint32_t)kt * kBK, ox = (uint32_t)kt * j.kst;
        unsigned char* run = s_lds + buf * kStageLds + (w & 3) * 64 * 16;
#pragma unroll
        for (int i = 0; i < kWChunks; ++i)
            load_lds16(wbase + woff0 + wrow_delta(i) + o, run + i * kRowStep * kRowBytes);
#pragma unroll
        for (int i = 0; i < kXChunks; ++i)
            load_lds16(xbase + s_xoff[i][tid] + ox, run + kWTile + i * kRowStep * kRowBytes);
    };
    auto compute = [&](int buf) {
        const unsigned char* base = s_lds + buf * kStageLds;
        // the fragments of both k-steps are requested before the first MFMA, so the LDS
        // latency is paid once per stage
        u32x4_t bfr[kBK / 32][kTS], afr[kBK / 32][8];
#pragma unroll
        for (int ks = 0; ks < kBK / 32; ++ks) {
            const uint32_t kx = ks ? 64u : 0u;
#pragma unroll
            for (int t = 0; t < kTS; ++t)
                bfr[ks][t] = *reinterpret_cast<const u32x4_t*>(base + ((tbase + t * kTStride * kRowBytes) ^ kx));
#pragma unroll
            for (int s = 0; s < 8; ++s)
                afr[ks][s] = *reinterpret_cast<const u32x4_t*>(base + ((fbase + frag_row(s) * kRowBytes) ^ kx));
        }
        __builtin_amdgcn_sched_barrier(0);
        __builtin_amdgcn_s_setprio(1);  // favour the wave that is issuing MFMAs
#pragma unroll
        for (int ks = 0; ks < kBK / 32; ++ks)
#pragma unroll
            for (int t = 0; t < kTS; ++t) {
                if (t >= nlive) continue;  // no live token in this sub-tile
#pragma unroll
                for (int s = 0; s < 8; ++s)
                    acc[s][t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, afr[ks][s]),
                                                                        __builtin_bit_cast(bf16x8_t, bfr[ks][t]),
                                                                        acc[s][t], 0, 0, 0);
            }
        __builtin_amdgcn_s_setprio(0);
        __builtin_amdgcn_sched_barrier(0);
    };

    // The loads of stage kt + 1 run under the MFMAs of stage kt; its LDS buffer was last
    // read in stage kt - 1, which every wave finished before the previous barrier.
    load(0, 0);
    for (int kt = 0; kt < nk; ++kt) {
        __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0): this wave's direct loads have landed
        __syncthreads();
        if (kt + 1 < nk) load((kt + 1) & 1, kt + 1);
        compute(kt & 1);
    }

    // Epilogue: lane holds features 4*quad .. +3 of sub-tile s for token m of sub-tile t.
#pragma unroll
    for (int t = 0; t < kTS; ++t) {
        const int pos = j.tok0 + t * kTStride + wt * 16 + m;
        if (pos >= j.ntok) continue;
        if (kUp) {
            // intermediates are k-blocked: element (row, f) at ((f / kBK) * rows + row) * kBK + f % kBK,
            // so a down-projection stage reads its token rows as one contiguous block
            uint16_t* dst = j.shared ? a.hs + (size_t)pos * kBK : a.h + (size_t)(j.start + pos) * kBK;
            const size_t fstride = (size_t)(j.shared ? a.T : a.T * a.K) * kBK;
#pragma unroll
            for (int s = 0; s < 4; ++s) {
                const f32x4_t g = acc[s][t], u = acc[s + 4][t];
                const int f = j.feat0 + wf * 64 + s * 16 + quad * 4;
                uint2 p;
                p.x = bf16_rne(silu(g.x) * u.x) | (bf16_rne(silu(g.y) * u.y) << 16);
                p.y = bf16_rne(silu(g.z) * u.z) | (bf16_rne(silu(g.w) * u.w) << 16);
                *reinterpret_cast<uint2*>(dst + (size_t)(f / kBK) * fstride + (f % kBK)) = p;
            }
        } else {
            float* dst = j.shared ? a.y_shared + (size_t)pos * a.d : a.y_slots + (size_t)(j.start + pos) * a.d;
            const float gs = (j.shared && a.sgate) ? a.sgate[pos] : 1.0f;  // gated shared block
#pragma unroll
            for (int s = 0; s < 8; ++s) {
                const int f = j.feat0 + wf * 128 + s * 16 + quad * 4;
                *reinterpret_cast<f32x4_t*>(dst + f) = acc[s][t] * gs;
            }
        }
    }
}

// Super-tile of the shared block: sn weight tiles x sm token tiles with sn | nt and
// sm | mt, at most one XCD round of blocks, as square as possible (the bytes a group
// fetches per stage are proportional to sn + sm).
void super_shape(int mt, int nt, int* out) {
    int best_n = 1, best_m = 1, best_score = -1;
    for (int sm = 1; sm <= mt && sm <= kXcdBlocks; ++sm) {
        if (mt % sm) continue;
        for (int sn = 1; sn <= nt && sn * sm <= kXcdBlocks; ++sn) {
            if (nt % sn) continue;
            // more blocks per group first, then fewer distinct tiles per block
            const int score = sn * sm * 64 - (sn + sm);
            if (score > best_score) { best_score = score; best_n = sn; best_m = sm; }
        }
    }
    out[0] = best_n;
    out[1] = best_m;
}

}  // namespace

bool expert_gemm_applies(const FfnArgs& a) {
    if (a.dtype != SPICE_BF16 || a.T < kGemmMinTokens || a.d % kBM || a.d % kBK || a.I % kUpFeat ||
        a.Is % kUpFeat || a.I % kBK || a.Is % kBK)
        return false;
    // element offsets inside one operand are 32-bit
    const long long lim = 0x7FFFFFFFll;
    if ((long long)a.I * a.T * a.K > lim || (long long)a.Is * a.T > lim || (long long)a.d * a.T * a.K > lim ||
        2ll * a.I * a.d > lim || 2ll * a.Is * a.d > lim)
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
    a.ldh = f.ldh; a.ldhs = f.ldhs;
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
    a.sgate = f.sgate;
    a.ctrl = f.ctrl;
    if (!hit) a.N = 0;  // no expert tiles
    // upper bound of the tile count: sum_e ceil(n_e / kBT) <= T*K / kBT + min(N, C)
    const long long mt_hit = hit ? (long long)a.T * a.K / kBT + std::min(a.N, a.C) : 0;
    const long long mt_sh = (a.T + kBT - 1) / kBT;
    const long long up_tiles = (a.Is > 0 ? mt_sh * (a.Is / kUpFeat) : 0) + mt_hit * (a.I / kUpFeat);
    const long long dn_tiles = (a.Is > 0 ? mt_sh * (a.d / kBM) : 0) + mt_hit * (a.d / kBM);
    if (up_tiles == 0) return hipSuccess;
    if (up_tiles > 0x7FFFFFFFll || dn_tiles > 0x7FFFFFFFll) return hipErrorInvalidValue;
    if (a.Is > 0) {
        super_shape((int)mt_sh, a.Is / kUpFeat, a.super_up);
        super_shape((int)mt_sh, a.d / kBM, a.super_dn);
    }
    const size_t lds = 2 * kStageLds;
    hipLaunchKernelGGL(expert_gemm_kernel<true>, dim3((unsigned)up_tiles), dim3(kThreads), lds, s, a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(expert_gemm_kernel<false>, dim3((unsigned)dn_tiles), dim3(kThreads), lds, s, a);
    return hipGetLastError();
}

}  // namespace spice
