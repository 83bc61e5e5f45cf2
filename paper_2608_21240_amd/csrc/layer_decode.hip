// The GPU part of one decode layer call in three launches (Sec. 4.2 routing and
// classification, Eq. 6 expert FFN, Eq. 9 LoRE, Sec. 4.3 execution), arranged so that
// the work that does not depend on routing runs beside it:
//
//   A  route + shared up  : each token's router rows spread over a few blocks (fp64 logits,
//                           and the shared block's gate when it has one); the last of a
//                           token's blocks to finish takes its top-K, gates and classes (one
//                           arrival counter per token); beside them the shared block's up
//                           tiles, which need only x;
//   B  bucket + up        : block 0 sorts the slots by (class, expert), writes offsets /
//                           perm / inv_perm, the work lists and the CPU path's host copies;
//                           the shared block's down tiles; the LoRE and HIT up tiles, each of
//                           which finds its bucket from the routing itself (local bucketing)
//                           rather than waiting for block 0;
//   C  routed down        : LoRE and HIT down tiles, each reading its bucket from the work list.
//
// Only a token's routing blocks wait for each other (through the counter, never by
// spinning).  Up and down tiles are the grouped-FFN tile code (expert_ffn_tiles.h) with the
// tile kind fixed at compile time.
#include "expert_ffn_mx_tiles.h"
#include "expert_ffn_tiles.h"
#include "route_device.h"

namespace spice {
namespace {

// Largest T whose HIT down tiles take 16 rows instead of 32.
constexpr int kDownRows16MaxT = 8;

// Most slots T*K for which the up tiles bucket locally (4 per thread).
constexpr int kLocalPer = 4;
static_assert(kLayerMaxSlots == kLocalPer * kThreads, "local bucketing covers kLayerMaxSlots slots");

// LDS of a launch-B block, in ints: the bucketing block's tables, or an up tile's reduction
// buffer (and, for MXFP4 HIT tiles, their scale stage) plus the local bucketing tables.
constexpr int kMaxI(int a, int b) { return a > b ? a : b; }
constexpr int kRedInts = kWaves * kTokTiles * 2 * 64 * 4;  // f32x4_t red[kWaves][kTokTiles][2][64]
constexpr int kMxUpInts = (int)((sizeof(MxUpLds<kMxUpR>) + 15) / 16 * 4);
constexpr int kLocalInts = 3 * SPICE_MAX_EXPERTS + SPICE_MAX_EXPERTS + 2 * kLayerMaxSlots + 4;
constexpr int kBucketInts = (int)(bucket_lds_bytes(kThreads, SPICE_MAX_EXPERTS, kLayerMaxSlots) / sizeof(int));
template <bool kMx>
constexpr int up_region_ints() { return kMx ? kMaxI(kRedInts, kMxUpInts) : kRedInts; }
template <bool kMx>
constexpr int up_lds_ints() { return kMaxI(up_region_ints<kMx>() + kLocalInts, kBucketInts); }
// LDS of a launch-C block: a down tile's reduction buffer (and the MXFP4 scale stage).
constexpr int kDownF4 = kWaves * kDownRows * kTokTiles * 64;
template <bool kMx>
constexpr int down_lds_f4() { return kMx ? kMaxI(kDownF4, (int)((sizeof(MxDownLds<kMxDownR>) + 15) / 16)) : kDownF4; }

struct LayerGridA {
    int nroute, g_per_tok, tsh;
};
struct LayerGridB {
    int tsh_dn, nlore, tlore, nhit, thit;
};
struct LayerGridC {
    int nlore, tlore, nhit, thit, rows16;  // rows16: HIT down tiles of 16 rows (small T), else 32
};

__device__ __forceinline__ int wave_sum_int(int v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
    return v;
}

// The ordinal-th non-empty bucket of class c (ascending expert id), found by this block from
// the routing (topk_idx, slot_class) and resident_slot: its expert, pool slot (HIT), start
// and size, and its slot ids in ascending order in s_ids.  Keys and positions follow the
// bucketing block's rule (key = class * N + expert; start = slots with a smaller key; a slot
// with an impossible class or expert has no key), so they agree with its perm.  Returns
// false when the class has fewer non-empty buckets, or the pool slot is out of range.
__device__ bool local_group(const FfnArgs& f, const RouteArgs& r, int c, int ordinal, Group& g, int* lds,
                            int* s_ids) {
    const int N = f.N, S = f.T * f.K, NK = 3 * N;
    const int tid = threadIdx.x, lane = tid & 63;
    int* s_cnt = lds;          // [3N]
    int* s_res = s_cnt + NK;   // [N]
    int* s_key = s_res + N;    // [S]
    int* s_grp = s_key + S;    // [4]
    // one round trip: the keys of slots tid + 256 u and the resident slot of expert tid
    int key[kLocalPer];
#pragma unroll
    for (int u = 0; u < kLocalPer; ++u) {
        const int s = tid + kThreads * u;
        key[u] = -1;
        if (s < S) {
            const int cl = r.slot_class[s], e = r.topk_idx[s];
            if (cl <= SPICE_CLASS_EXACT && e >= 0 && e < N) key[u] = cl * N + e;
        }
    }
    const int res = tid < N ? f.resident_slot[tid] : -1;
    for (int i = tid; i < NK; i += kThreads) s_cnt[i] = 0;
    __syncthreads();
#pragma unroll
    for (int u = 0; u < kLocalPer; ++u) {
        const int s = tid + kThreads * u;
        if (s < S) {
            s_key[s] = key[u];
            if (key[u] >= 0) atomicAdd(&s_cnt[key[u]], 1);
        }
    }
    if (tid < N) s_res[tid] = res;
    __syncthreads();
    if (tid < 64) {
        const unsigned long long lt = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
        int seen = 0, ef = -1, nf = 0;
        for (int e0 = 0; e0 < N; e0 += 64) {
            const int e = e0 + lane;
            const int n = e < N ? s_cnt[c * N + e] : 0;
            const unsigned long long m = __ballot(n > 0);
            const int cnt = __popcll(m);
            if (ef < 0 && ordinal < seen + cnt) {  // uniform
                const bool mine = n > 0 && __popcll(m & lt) == ordinal - seen;
                const int src = __ffsll((long long)__ballot(mine)) - 1;
                ef = e0 + src;
                nf = __shfl(n, src);
            }
            seen += cnt;
        }
        if (ef >= 0) {
            const int target = c * N + ef;
            int part = 0;
            for (int k = lane; k < target; k += 64) part += s_cnt[k];
            const int start = wave_sum_int(part);
            int run = 0;
            for (int s0 = 0; s0 < S; s0 += 64) {
                const int s = s0 + lane;
                const bool mt = s < S && s_key[s] == target;
                const unsigned long long m = __ballot(mt);
                if (mt) s_ids[run + __popcll(m & lt)] = s;
                run += __popcll(m);
            }
            if (lane == 0) {
                s_grp[0] = ef;
                s_grp[1] = start;
                s_grp[2] = nf;
                s_grp[3] = c == SPICE_CLASS_HIT ? s_res[ef] : -1;
            }
        } else if (lane == 0) {
            s_grp[0] = -1;
        }
    }
    __syncthreads();
    g.e = s_grp[0];
    g.start = s_grp[1];
    g.n = s_grp[2];
    g.slot = s_grp[3];
    if (g.e < 0) return false;
    if (c == SPICE_CLASS_HIT && (g.slot < 0 || g.slot >= f.C)) {
        if (tid == 0) atomicOr(&f.ctrl[kWordFlags], (uint32_t)SPICE_FLAG_BAD_SLOT);
        return false;
    }
    return true;
}

// The j-th work record of class c, or false past the list's end (or for a record out of
// range, flagged).
__device__ bool work_group(const FfnArgs& f, const RouteArgs& r, int c, int j, Group& g) {
    const int cnt = r.wl_count[c];
    const int4 rec = *reinterpret_cast<const int4*>(r.worklist + 4 * (c * f.N + j));
    if (j >= cnt) return false;
    g.e = rec.x;
    g.slot = rec.y;
    g.start = rec.z;
    g.n = rec.w;
    const bool bad = g.e < 0 || g.e >= f.N || g.start < 0 || g.n <= 0 || g.start + g.n > f.T * f.K ||
                     (c == SPICE_CLASS_HIT && (g.slot < 0 || g.slot >= f.C));
    if (bad && threadIdx.x == 0) atomicOr(&f.ctrl[kWordFlags], (uint32_t)SPICE_FLAG_BAD_INDEX);
    return !bad;
}

template <int DT>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(3))) void layer_route_kernel(
    RouteArgs r, FfnArgs f, LayerGridA gr) {
    __shared__ __align__(16) f32x4_t red[kWaves][kTokTiles][2][64];
    __shared__ int s_flag;
    static_assert(sizeof(red) >= sizeof(TopkLds), "top-K scratch fits");
    const int b = blockIdx.x;
    if (b < gr.nroute) {
        const int t = b / gr.g_per_tok, g = b % gr.g_per_tok;
        constexpr int rows = kWaves * kRouteRowsPerWave;
        route_logits_rows<DT>(r, t, g * rows, min(r.N + (r.w_sg ? 1 : 0), (g + 1) * rows));
        if (!route_last_block(&r.ctrl[kWordTokCount + t * kTokCountStride], gr.g_per_tok, &s_flag)) return;
        block_topk<kThreads, true>(r, t, r.logits_ws + (size_t)t * r.N, *reinterpret_cast<TopkLds*>(&red[0][0][0][0]));
        return;
    }
    const Group g{0, 0, f.T, -1};
    up_tile<DT, kKindShared>(f, g, b - gr.nroute, nullptr, red);
}

template <int DT, bool kMx>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(3))) void layer_up_kernel(
    RouteArgs r, FfnArgs f, LayerGridB gr) {
    __shared__ __align__(16) int lds[up_lds_ints<kMx>()];
    int b = blockIdx.x;
    if (b == 0) {
        bucket_slots<kThreads, kLayerMaxSlots>(r, lds);
        if (r.hx || r.h_idx || r.h_w || r.h_cls || r.h_ready) mirror_host<kThreads>(r);
        return;
    }
    b -= 1;
    if (b < gr.tsh_dn) {
        const Group g{0, 0, f.T, -1};
        down_tile<DT, kKindShared, 1>(f, g, b, *reinterpret_cast<f32x4_t(*)[kWaves][kDownRows][kTokTiles][64]>(lds));
        return;
    }
    b -= gr.tsh_dn;
    auto& red = *reinterpret_cast<f32x4_t(*)[kWaves][kTokTiles][2][64]>(lds);
    int* s_ids = lds + up_region_ints<kMx>();
    int* s_loc = s_ids + kLayerMaxSlots;
    Group g;
    if (b < gr.nlore * gr.tlore) {
        if (!local_group(f, r, SPICE_CLASS_LORE, b / gr.tlore, g, s_loc, s_ids)) return;
        up_tile<DT, kKindLore>(f, g, b % gr.tlore, s_ids, red);
        return;
    }
    b -= gr.nlore * gr.tlore;
    if (b < gr.nhit * gr.thit) {
        if (!local_group(f, r, SPICE_CLASS_HIT, b / gr.thit, g, s_loc, s_ids)) return;
        if constexpr (kMx) mx_up_tile<kMxUpR>(f, g, b % gr.thit, s_ids, *reinterpret_cast<MxUpLds<kMxUpR>*>(lds));
        else up_tile<DT, kKindHit>(f, g, b % gr.thit, s_ids, red);
    }
}

template <int DT, bool kMx>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(3))) void layer_down_kernel(
    RouteArgs r, FfnArgs f, LayerGridC gr) {
    __shared__ f32x4_t lds[down_lds_f4<kMx>()];
    auto& red = *reinterpret_cast<f32x4_t(*)[kWaves][kDownRows][kTokTiles][64]>(lds);
    int b = blockIdx.x;
    Group g;
    if (b < gr.nlore * gr.tlore) {
        if (!work_group(f, r, SPICE_CLASS_LORE, b / gr.tlore, g)) return;
        lore_down_tile<DT>(f, g.e, g.start, g.n, b % gr.tlore, reinterpret_cast<float*>(&red[0][0][0][0]));
        return;
    }
    b -= gr.nlore * gr.tlore;
    if (b < gr.nhit * gr.thit) {
        if (!work_group(f, r, SPICE_CLASS_HIT, b / gr.thit, g)) return;
        if constexpr (kMx) mx_down_tile<kMxDownR>(f, g, b % gr.thit, *reinterpret_cast<MxDownLds<kMxDownR>*>(lds));
        else if (gr.rows16) down_tile<DT, kKindHit, 1>(f, g, b % gr.thit, red);
        else down_tile<DT, kKindHit>(f, g, b % gr.thit, red);
    }
}

}  // namespace

hipError_t launch_layer_decode(const RouteArgs& r, const FfnArgs& f, hipStream_t s) {
    const int S = f.T * f.K;
    const bool shared = f.Is > 0, lore = f.r > 0;
    const int gpt = route_blocks_per_token(r.N + (r.w_sg ? 1 : 0), kThreads);
    LayerGridA ga{f.T * gpt, gpt, shared ? (f.Is + 15) / 16 : 0};
    // the shared block's down tiles take 16 rows (twice as many, half as long: they would
    // otherwise be the longest tiles of the launch at small T); so do the HIT down tiles
    // while the batch is small (few experts, so too few tiles to fill the GPU)
    const bool mx = f.wfmt == SPICE_WFMT_MXFP4;
    if (mx && f.dtype != SPICE_BF16) return hipErrorInvalidValue;
    const bool rows16 = f.T <= kDownRows16MaxT;
    // HIT tiles: MXFP4 tiles are 2 x 16 W1/W3 rows (up) and 4 x 16 W2 rows (down)
    const int thit_up = mx ? (f.I + 16 * kMxUpR - 1) / (16 * kMxUpR) : (f.I + 15) / 16;
    const int thit_dn = mx ? (f.d + 16 * kMxDownR - 1) / (16 * kMxDownR)
                           : (rows16 ? (f.d + 15) / 16 : (f.d + 16 * kDownRows - 1) / (16 * kDownRows));
    LayerGridB gb{shared ? (f.d + 15) / 16 : 0, lore ? std::min(f.N, S) : 0, (f.r + 15) / 16,
                  f.C > 0 ? std::min(std::min(f.N, f.C), S) : 0, thit_up};
    LayerGridC gc{gb.nlore, (f.d + kLoreRows - 1) / kLoreRows, gb.nhit, thit_dn, (!mx && rows16) ? 1 : 0};
    const unsigned na = (unsigned)(ga.nroute + ga.tsh);
    const unsigned nb = (unsigned)(1 + gb.tsh_dn + gb.nlore * gb.tlore + gb.nhit * gb.thit);
    const unsigned nc = (unsigned)(gc.nlore * gc.tlore + gc.nhit * gc.thit);
    if (mx) {
        hipLaunchKernelGGL(layer_route_kernel<SPICE_BF16>, dim3(na), dim3(kThreads), 0, s, r, f, ga);
        hipLaunchKernelGGL((layer_up_kernel<SPICE_BF16, true>), dim3(nb), dim3(kThreads), 0, s, r, f, gb);
        if (nc) hipLaunchKernelGGL((layer_down_kernel<SPICE_BF16, true>), dim3(nc), dim3(kThreads), 0, s, r, f, gc);
    } else if (f.dtype == SPICE_BF16) {
        hipLaunchKernelGGL(layer_route_kernel<SPICE_BF16>, dim3(na), dim3(kThreads), 0, s, r, f, ga);
        hipLaunchKernelGGL((layer_up_kernel<SPICE_BF16, false>), dim3(nb), dim3(kThreads), 0, s, r, f, gb);
        if (nc) hipLaunchKernelGGL((layer_down_kernel<SPICE_BF16, false>), dim3(nc), dim3(kThreads), 0, s, r, f, gc);
    } else {
        hipLaunchKernelGGL(layer_route_kernel<SPICE_F32>, dim3(na), dim3(kThreads), 0, s, r, f, ga);
        hipLaunchKernelGGL((layer_up_kernel<SPICE_F32, false>), dim3(nb), dim3(kThreads), 0, s, r, f, gb);
        if (nc) hipLaunchKernelGGL((layer_down_kernel<SPICE_F32, false>), dim3(nc), dim3(kThreads), 0, s, r, f, gc);
    }
    return hipGetLastError();
}

}  // namespace spice
