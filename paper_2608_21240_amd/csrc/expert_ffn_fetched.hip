// Grouped SwiGLU FFN (Eq. 6) of the experts fetched for one call (M_fetch of Eq. 12;
// Sec. 4.3): exact misses whose weights the host copied into a small fetch pool.
//
// Two launches, one block (4 waves) per (fetch slot, row tile), with the tile code
// of the resident-expert FFN: fetch slot j serves the bucket (EXACT, fetch_expert[j])
// of the routing with the weights in slot j of the pool, writes its outputs to the
// bucket's rows of y_slots and relabels its slots EXACT -> EXACT_GPU so that the
// combine adds them like resident hits.
#include "expert_ffn_tiles.h"

namespace spice {
namespace {

__device__ bool find_fetched_group(const FfnArgs& a, const FetchArgs& f, int j, Group& g) {
    const int e = f.fetch_expert[j];
    if (e < 0) return false;  // unused slot
    if (e >= a.N) {
        if ((threadIdx.x & 63) == 0) atomicOr(&a.ctrl[kWordFlags], (uint32_t)SPICE_FLAG_BAD_INDEX);
        return false;
    }
    const int32_t* off = a.offsets + SPICE_CLASS_EXACT * (a.N + 1);
    const int st = off[e];
    const int n = off[e + 1] - st;
    if (st < 0 || n < 0 || st + n > a.T * a.K) {
        if ((threadIdx.x & 63) == 0) atomicOr(&a.ctrl[kWordFlags], (uint32_t)SPICE_FLAG_BAD_INDEX);
        return false;
    }
    g.e = e;
    g.start = st;
    g.n = n;
    g.slot = j;
    return n > 0;
}

template <int DT>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(3))) void ffn_up_fetched_kernel(
    FfnArgs a, FetchArgs f, int tiles) {
    __shared__ f32x4_t red[kWaves][kTokTiles][2][64];
    Tile tile;
    tile.kind = kKindHit;
    tile.ordinal = blockIdx.x / tiles;
    tile.rt = blockIdx.x % tiles;
    Group g;
    if (!find_fetched_group(a, f, tile.ordinal, g)) return;
    if (tile.rt == 0) {
        // the combine adds these slots like HIT slots from here on
        for (int i = threadIdx.x; i < g.n; i += kThreads) {
            const int s = a.perm[g.start + i];
            if (s >= 0 && s < a.T * a.K) f.slot_class[s] = SPICE_CLASS_EXACT_GPU;
        }
    }
    up_tile<DT, kKindHit>(a, g, tile.rt, a.perm + g.start, red);
}

template <int DT>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(3))) void ffn_down_fetched_kernel(
    FfnArgs a, FetchArgs f, int tiles) {
    __shared__ f32x4_t red[kWaves][kDownRows][kTokTiles][64];
    Tile tile;
    tile.kind = kKindHit;
    tile.ordinal = blockIdx.x / tiles;
    tile.rt = blockIdx.x % tiles;
    Group g;
    if (!find_fetched_group(a, f, tile.ordinal, g)) return;
    down_tile<DT, kKindHit>(a, g, tile.rt, red);
}

}  // namespace

hipError_t launch_expert_ffn_fetched(const FfnArgs& a, const FetchArgs& f, hipStream_t s) {
    if (f.n_slots <= 0) return hipSuccess;
    const int tup = (a.I + 15) / 16;
    const int tdn = (a.d + 16 * kDownRows - 1) / (16 * kDownRows);
    const unsigned nup = (unsigned)(f.n_slots * tup), ndn = (unsigned)(f.n_slots * tdn);
    if (a.dtype == SPICE_BF16) {
        hipLaunchKernelGGL(ffn_up_fetched_kernel<SPICE_BF16>, dim3(nup), dim3(kThreads), 0, s, a, f, tup);
        hipLaunchKernelGGL(ffn_down_fetched_kernel<SPICE_BF16>, dim3(ndn), dim3(kThreads), 0, s, a, f, tdn);
    } else {
        hipLaunchKernelGGL(ffn_up_fetched_kernel<SPICE_F32>, dim3(nup), dim3(kThreads), 0, s, a, f, tup);
        hipLaunchKernelGGL(ffn_down_fetched_kernel<SPICE_F32>, dim3(ndn), dim3(kThreads), 0, s, a, f, tdn);
    }
    return hipGetLastError();
}


}  // namespace spice
