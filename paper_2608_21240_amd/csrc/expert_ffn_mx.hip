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
// whole MX block b = 4j + q (32 elements: one 16-byte load) and uses it for the 4 steps of
// the group: step u gets elements 8u .. 8u+7 of the block, and the token operand of lane
// (n, q) reads the same 8 k of its token row.  So a group covers 128 consecutive k, and
// the weight bytes of a wave are one 16-byte load per row stream and group.  A tile takes
// 2 (up: W1 and W3) x 2 or 4 (down) row streams of 16 rows, so that one group's 4 token
// loads serve 4 weight loads; whole groups are dealt to the 4 waves, two in flight per
// wave; a last partial group (K/32 not a multiple of 4) goes to the last wave.
//
// Loads go through raw buffer resources: rows past the end of a matrix and lanes past the
// end of a row read zero, with no branch around any load, so that every wait leaves the
// next group in flight.  The block scales of a tile (one byte per row and block) are read
// once per tile with coalesced 16-byte loads into LDS rather than one byte load per
// stream and group.
#include "expert_ffn_mx_tiles.h"

namespace spice {
namespace {

// LDS of a block: whatever the tile it runs needs
constexpr size_t kUpLds = std::max(sizeof(MxUpLds<kMxUpR>), sizeof(f32x4_t) * kWaves * kTokTiles * 2 * 64);
constexpr size_t kDownLds = std::max(sizeof(MxDownLds<kMxDownR>), sizeof(f32x4_t) * kWaves * kDownRows * kTokTiles * 64);

__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(3))) void ffn_up_mx_kernel(FfnArgs a,
                                                                                                       Grid gr) {
    __shared__ f32x4_t lds[kUpLds / sizeof(f32x4_t)];
    Tile tile;
    if (!gr.decode(blockIdx.x, tile)) return;
    Group g{0, 0, a.T, -1};
    if (tile.kind != kKindShared &&
        !find_group(a, tile.kind == kKindHit ? SPICE_CLASS_HIT : SPICE_CLASS_LORE, tile.ordinal, g))
        return;
    auto& red = *reinterpret_cast<f32x4_t(*)[kWaves][kTokTiles][2][64]>(lds);
    if (tile.kind == kKindHit)
        mx_up_tile<kMxUpR>(a, g, tile.rt, a.perm + g.start, *reinterpret_cast<MxUpLds<kMxUpR>*>(lds));
    else if (tile.kind == kKindShared)
        up_tile<SPICE_BF16, kKindShared>(a, g, tile.rt, nullptr, red);
    else
        up_tile<SPICE_BF16, kKindLore>(a, g, tile.rt, a.perm + g.start, red);
}

__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(3))) void ffn_down_mx_kernel(FfnArgs a,
                                                                                                         Grid gr) {
    __shared__ f32x4_t lds[kDownLds / sizeof(f32x4_t)];
    Tile tile;
    if (!gr.decode(blockIdx.x, tile)) return;
    Group g{0, 0, a.T, -1};
    if (tile.kind != kKindShared &&
        !find_group(a, tile.kind == kKindHit ? SPICE_CLASS_HIT : SPICE_CLASS_LORE, tile.ordinal, g))
        return;
    if (tile.kind == kKindLore)
        lore_down_tile<SPICE_BF16>(a, g.e, g.start, g.n, tile.rt, reinterpret_cast<float*>(lds));
    else if (tile.kind == kKindHit)
        mx_down_tile<kMxDownR>(a, g, tile.rt, *reinterpret_cast<MxDownLds<kMxDownR>*>(lds));
    else
        down_tile<SPICE_BF16, kKindShared>(a, g, tile.rt,
                                           *reinterpret_cast<f32x4_t(*)[kWaves][kDownRows][kTokTiles][64]>(lds));
}

}  // namespace

hipError_t launch_expert_ffn_mx(const FfnArgs& a, hipStream_t s) {
    if (a.dtype != SPICE_BF16) return hipErrorInvalidValue;
    const bool hit = (a.groups & kDoHit) != 0;
    const bool shared = (a.groups & kDoShared) != 0 && a.Is > 0;
    const bool lore = (a.groups & kDoLore) != 0 && a.r > 0;
    Grid up, dn;
    ffn_grids(a, hit, shared, lore, up, dn);
    if (hit) {  // the MXFP4 HIT tiles are taller
        up.thit = (a.I + 16 * kMxUpR - 1) / (16 * kMxUpR);
        dn.thit = (a.d + 16 * kMxDownR - 1) / (16 * kMxDownR);
    }
    const long long nup = up.blocks(), ndn = dn.blocks();
    if (nup == 0) return hipSuccess;
    hipLaunchKernelGGL(ffn_up_mx_kernel, dim3((unsigned)nup), dim3(kThreads), 0, s, a, up);
    hipLaunchKernelGGL(ffn_down_mx_kernel, dim3((unsigned)ndn), dim3(kThreads), 0, s, a, dn);
    return hipGetLastError();
}

}  // namespace spice
