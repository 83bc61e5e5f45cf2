// Index arithmetic of the expert-FFN tiles, shared by the kernels (expert_ffn_tiles.h) and
// compiled as plain host C++ by the tile model of the test suite (tests/sanitize), which
// replays every tile's loads and stores against exactly-sized buffers under AddressSanitizer:
// the grid decode, the bucket of a group, the weight matrix each kind of tile streams (a
// compile-time choice: no tile picks a base pointer at run time), the clamped operand rows
// and token columns, and the output elements.  Nothing here touches memory.
#pragma once

#include <stddef.h>
#include <stdint.h>

#include "spice_internal.h"

#ifdef __HIPCC__
#define SPICE_HD __host__ __device__ __forceinline__
#else
#define SPICE_HD inline
#endif

namespace spice {

enum : int { kKindHit = 0, kKindShared = 1, kKindLore = 2 };

constexpr int kTileRows = 16;  // operand rows of one MFMA tile (weights) / token columns
constexpr int kTokTiles = 2;   // token tiles of 16 per pass
constexpr int kDownRows = 2;   // 16-row tiles per down tile of a routed expert (32 rows)
constexpr int kLoreRows = 256; // B_e rows per LoRE down tile (one per thread)
constexpr int kLoreTok = 16;   // tokens per LoRE down pass
constexpr int kStepBytes = 64; // bytes of one contraction step of one operand row (4 lanes x 16 B)

SPICE_HD int imin(int a, int b) { return a < b ? a : b; }

struct Tile {
    int kind, ordinal, rt;
};

struct Group {
    int e, start, n, slot;
};

// Block index -> tile of the grouped-FFN launches.  Segments, in dispatch order: shared-block
// row tiles (the longest tiles: all T tokens, and the longest contraction in the down pass),
// LORE experts x row tiles (short but latency-bound), HIT experts x row tiles.  Putting the
// long tiles first keeps them out of the launch's tail.  Expert counts are upper bounds;
// surplus blocks exit at once.
struct Grid {
    int nhit, thit, tsh, nlore, tlore;
    SPICE_HD bool decode(int b, Tile& t) const {
        if (b < 0) return false;
        if (b < tsh) { t = Tile{kKindShared, 0, b}; return true; }
        b -= tsh;
        if (b < nlore * tlore) { t = Tile{kKindLore, b / tlore, b % tlore}; return true; }
        b -= nlore * tlore;
        if (b < nhit * thit) { t = Tile{kKindHit, b / thit, b % thit}; return true; }
        return false;
    }
    SPICE_HD long long blocks() const { return (long long)tsh + (long long)nlore * tlore + (long long)nhit * thit; }
};

// The up and down grids of a grouped-FFN call (HIT experts, shared block, LoRE factors as
// requested by a.groups; hit, shared and lore say which are live).
SPICE_HD void ffn_grids(const FfnArgs& a, bool hit, bool shared, bool lore, Grid& up, Grid& dn) {
    const int slots = a.T * a.K;
    up = Grid{0, 1, 0, 0, 1};
    dn = Grid{0, 1, 0, 0, 1};
    if (hit) {
        up.nhit = dn.nhit = imin(imin(a.N, a.C), slots);
        up.thit = (a.I + kTileRows - 1) / kTileRows;
        dn.thit = (a.d + kTileRows * kDownRows - 1) / (kTileRows * kDownRows);
    }
    if (shared) {
        up.tsh = (a.Is + kTileRows - 1) / kTileRows;
        dn.tsh = (a.d + kTileRows * kDownRows - 1) / (kTileRows * kDownRows);
    }
    if (lore) {
        up.nlore = dn.nlore = imin(a.N, slots);
        up.tlore = (a.r + kTileRows - 1) / kTileRows;
        dn.tlore = (a.d + kLoreRows - 1) / kLoreRows;
    }
}

// Bucket (c, e) from the offsets: its start and size, and whether the group is usable
// (inside the T*K slots; for HIT, a pool slot in range).
SPICE_HD Group bucket_of(const int32_t* off_c, int e, int c, int32_t slot) {
    const int st = off_c[e];
    return Group{e, st, off_c[e + 1] - st, c == SPICE_CLASS_HIT ? slot : -1};
}
SPICE_HD bool group_in_range(const FfnArgs& a, int c, const Group& g) {
    if (g.start < 0 || g.n < 0 || g.start + g.n > a.T * a.K) return false;
    return c != SPICE_CLASS_HIT || (g.slot >= 0 && g.slot < a.C);
}

// ---- up tiles ------------------------------------------------------------------------
// The matrix an up tile of kind KIND streams: the pool's W1/W3 (HIT), the shared block's
// (shared) or the LoRE A factors (LORE).
template <int KIND>
SPICE_HD const void* up_weights(const FfnArgs& a) {
    if constexpr (KIND == kKindHit) return a.w13_pool;
    else if constexpr (KIND == kKindShared) return a.w13s;
    else return a.lore_A;
}
// The group's rows of that matrix: first gate row, first up row (= gate for LORE), count.
struct UpBlock {
    size_t gate_row0, up_row0;
    int nrows;
};
template <int KIND>
SPICE_HD UpBlock up_block(const FfnArgs& a, const Group& g) {
    if constexpr (KIND == kKindHit) {
        const size_t r0 = (size_t)g.slot * 2 * a.I;
        return UpBlock{r0, r0 + a.I, a.I};
    } else if constexpr (KIND == kKindShared) {
        return UpBlock{0, (size_t)a.Is, a.Is};
    } else {
        const size_t r0 = (size_t)g.e * a.r;
        return UpBlock{r0, r0, a.r};
    }
}
// The group's entries: HIT and LORE tiles read their bucket, shared tiles tokens 0..T-1.
template <int KIND>
SPICE_HD void tile_entries(const FfnArgs& a, const Group& g, int& start, int& n) {
    if constexpr (KIND == kKindShared) { start = 0; n = a.T; }
    else { start = g.start; n = g.n; }
}
// Operand row read for row m of row tile rt (tile_rows rows per tile); rows past the end
// read the last row, and their outputs are dropped.
SPICE_HD int tile_row(int rt, int tile_rows, int m, int nrows) { return imin(rt * tile_rows + m, nrows - 1); }
// Bucket entry of token column m of token tile tt in the pass at entry g0, clamped to the
// last entry (padding columns repeat it; their outputs are dropped).
SPICE_HD int tile_entry(int g0, int tt, int m, int n) { return imin(g0 + tt * kTileRows + m, n - 1); }
// Output element of entry gi, feature orow (the first of 4): H (HIT), the shared H, or U.
template <int KIND>
SPICE_HD size_t up_out_elem(const FfnArgs& a, int start, int gi, int orow) {
    if constexpr (KIND == kKindHit) return (size_t)(start + gi) * a.ldh + orow;
    else if constexpr (KIND == kKindShared) return (size_t)gi * a.ldhs + orow;
    else return (size_t)(start + gi) * a.r + orow;
}

// ---- down tiles ----------------------------------------------------------------------
template <int KIND>
SPICE_HD const void* down_weights(const FfnArgs& a) {
    static_assert(KIND == kKindHit || KIND == kKindShared, "down tiles are HIT or shared");
    if constexpr (KIND == kKindHit) return a.w2_pool;
    else return a.w2s;
}
template <int KIND>
SPICE_HD const void* down_inputs(const FfnArgs& a) {
    if constexpr (KIND == kKindHit) return a.h;
    else return a.hs;
}
// First W2 row of the group, contraction length, row stride of the intermediate.
struct DownBlock {
    size_t row0;
    int kdim, ld;
};
template <int KIND>
SPICE_HD DownBlock down_block(const FfnArgs& a, const Group& g) {
    if constexpr (KIND == kKindHit) return DownBlock{(size_t)g.slot * a.d, a.I, a.ldh};
    else return DownBlock{0, a.Is, a.ldhs};
}
// Output element of entry gi, feature dim (the first of 4): y_slots (HIT) or y_shared.
template <int KIND>
SPICE_HD size_t down_out_elem(const FfnArgs& a, int start, int gi, int dim) {
    if constexpr (KIND == kKindHit) return (size_t)(start + gi) * a.d + dim;
    else return (size_t)gi * a.d + dim;
}

// ---- LoRE down tiles (one B_e row per thread) ------------------------------------------
SPICE_HD size_t lore_b_elem(const FfnArgs& a, int e, int row, int q) { return ((size_t)e * a.d + row) * a.r + q; }
SPICE_HD size_t lore_u_elem(const FfnArgs& a, int start, int j, int q) { return (size_t)(start + j) * a.r + q; }
SPICE_HD size_t lore_y_elem(const FfnArgs& a, int start, int j, int row) { return (size_t)(start + j) * a.d + row; }

}  // namespace spice
