// Grouped expert FFN for the resident (HIT) experts and the shared block (Eq. 6;
// Sec. 2.1, 4.2), and the LoRE correction B_e (A_e x) of low-confidence misses (Eq. 9).
//
// Two launches, one block (4 waves) per tile:
//   up   : 16-row tiles of W1/W3 (or of A_e): H = silu(X W1^T) * (X W3^T)  (or U = X A_e^T),
//          X = the tokens of the expert's bucket;
//   down : 32-row tiles of W2: Y = H W2^T;  256-row tiles of B_e: delta = U B_e^T.
// Blocks map to (expert ordinal, row tile): the shared block first, then LORE
// experts, then HIT experts (longest tiles first).  Each wave resolves its block's
// expert on the device from the bucket offsets (the pool slot comes in the same round trip), so no
// host synchronisation is needed and blocks beyond the live experts exit at once;
// the hardware dispatcher overlaps one block's set-up with the others' streaming.
// Within a tile the 4 waves split the contraction dimension and add their MFMA
// accumulators through LDS.  The weight tile is the MFMA A operand (16 rows x 32 k
// per bf16 step, one 16-byte load per lane), the tokens are the B operand (16
// columns; padding columns read a valid row and are dropped), fp32 accumulation.
// Pointer arrays handed to the inlined helpers are always named locals: passing
// brace-initialised temporaries by reference miscompiled one instantiation here.
#include "expert_ffn_tiles.h"

namespace spice {
namespace {

template <int DT>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(3))) void ffn_up_kernel(FfnArgs a, Grid gr) {
    __shared__ f32x4_t red[kWaves][kTokTiles][2][64];
    Tile tile;
    if (!gr.decode(blockIdx.x, tile)) return;
    Group g{0, 0, a.T, -1};
    if (tile.kind != kKindShared &&
        !find_group(a, tile.kind == kKindHit ? SPICE_CLASS_HIT : SPICE_CLASS_LORE, tile.ordinal, g))
        return;
    up_tile_kind<DT>(a, g, tile, red);
}

template <int DT>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(3))) void ffn_down_kernel(FfnArgs a, Grid gr) {
    __shared__ f32x4_t red[kWaves][kDownRows][kTokTiles][64];
    Tile tile;
    if (!gr.decode(blockIdx.x, tile)) return;
    Group g{0, 0, a.T, -1};
    if (tile.kind != kKindShared &&
        !find_group(a, tile.kind == kKindHit ? SPICE_CLASS_HIT : SPICE_CLASS_LORE, tile.ordinal, g))
        return;
    if (tile.kind == kKindLore)
        lore_down_tile<DT>(a, g.e, g.start, g.n, tile.rt, reinterpret_cast<float*>(&red[0][0][0][0]));
    else if (tile.kind == kKindHit)
        down_tile<DT, kKindHit>(a, g, tile.rt, red);
    else
        down_tile<DT, kKindShared>(a, g, tile.rt, red);
}

}  // namespace

hipError_t launch_expert_ffn(const FfnArgs& f, hipStream_t s) {
    FfnArgs a = f;
    if ((a.groups & (kDoHit | kDoShared)) && expert_gemm_applies(a)) {
        // many tokens: the HIT experts and the shared block as MFMA GEMMs; LoRE below
        const hipError_t e = launch_expert_gemm(a, (a.groups & kDoHit) != 0, (a.groups & kDoShared) != 0, s);
        if (e != hipSuccess) return e;
        a.groups &= kDoLore;
    }
    const bool hit = (a.groups & kDoHit) != 0;
    const bool shared = (a.groups & kDoShared) != 0 && a.Is > 0;
    const bool lore = (a.groups & kDoLore) != 0 && a.r > 0;
    Grid up, dn;
    ffn_grids(a, hit, shared, lore, up, dn);
    const long long nup = up.blocks(), ndn = dn.blocks();
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