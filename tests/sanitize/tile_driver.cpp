// Host model of the expert-FFN tile indexing, built with -fsanitize=address,undefined by
// tests/test_sanitizers.py.  For each shape and batch it routes seeded tokens, buckets their
// slots (stable counting sort by (class, expert)), allocates every buffer a call reads or
// writes at exactly its size, and replays every block of the grouped-FFN launches (the grids
// of ffn_grids, the decode-layer variants with 16-row down tiles) through the index helpers
// the kernels use (tile_index.h): each 16-byte operand load of every lane and contraction step
// and each output store is performed on the host buffer it belongs to.  An access outside its
// buffer fails the explicit range check (and, past the allocation, AddressSanitizer).
// Prints the number of checked accesses and "ok".
#include <algorithm>
#include <cstdint>
#include <cstdio>
#include <cstring>
#include <vector>

#include "spice_internal.h"
#include "tile_index.h"

using namespace spice;

namespace {

int g_fail = 0;
long long g_access = 0;

struct Buf {
    const char* name;
    std::vector<uint8_t> v;
    const void* p() const { return v.data(); }
    void* p() { return v.data(); }
};

// One access of `bytes` at `ptr`, which must lie inside buffer b.
void touch(const Buf& b, const void* ptr, size_t bytes, bool write = false) {
    ++g_access;
    const uint8_t* q = static_cast<const uint8_t*>(ptr);
    const uint8_t* lo = b.v.data();
    if (q < lo || q + bytes > lo + b.v.size()) {
        if (g_fail < 20)
            std::fprintf(stderr, "%s access of %zu bytes at offset %lld outside [0, %zu)\n", b.name, bytes,
                         (long long)(q - lo), b.v.size());
        g_fail = 1;
        return;
    }
    uint8_t tmp[16];
    std::memcpy(tmp, q, bytes);  // a real read of the range (AddressSanitizer checks it)
    if (write) std::memcpy(const_cast<uint8_t*>(q), tmp, bytes);
}

uint64_t g_rng = 0xA4093822299F31D0ull;
double urand() {
    g_rng ^= g_rng >> 12; g_rng ^= g_rng << 25; g_rng ^= g_rng >> 27;
    return (double)((g_rng * 0x2545F4914F6CDD1Dull) >> 11) * (1.0 / 9007199254740992.0);
}

struct Case {
    FfnArgs a{};
    int es = 2, kstep = 32, klane = 8;
    Buf x{"x"}, w13{"w13_pool"}, w2{"w2_pool"}, w13s{"w13_shared"}, w2s{"w2_shared"}, la{"lore_A"}, lb{"lore_B"},
        h{"h"}, hs{"hs"}, u{"u"}, ys{"y_slots"}, ysh{"y_shared"}, sg{"sgate"}, perm{"perm"}, off{"offsets"},
        res{"resident_slot"};
    const Buf& by_ptr(const void* p) const {
        for (const Buf* b : {&w13, &w2, &w13s, &w2s, &la, &lb, &h, &hs})
            if (b->p() == p) return *b;
        std::fprintf(stderr, "unknown base pointer\n");
        g_fail = 1;
        return x;
    }
};

void alloc(Buf& b, size_t bytes) { b.v.assign(bytes, 0); }

// Route T tokens (K distinct experts each, Zipf-like skew), classify (R resident, LoRE below
// tau) and bucket the slots as the routing step does.
void make_case(Case& c, int d, int N, int K, int I, int Is, int r, int R, int T, int dtype) {
    FfnArgs& a = c.a;
    a.T = T; a.d = d; a.N = N; a.K = K; a.C = std::max(R, 1); a.I = I; a.Is = Is; a.r = r; a.dtype = dtype;
    a.ldh = I + kHPad; a.ldhs = Is + kHPad;
    c.es = dtype == SPICE_BF16 ? 2 : 4;
    c.kstep = dtype == SPICE_BF16 ? 32 : 16;
    c.klane = dtype == SPICE_BF16 ? 8 : 4;
    const int es = c.es, S = T * K;
    alloc(c.x, (size_t)T * d * es);
    alloc(c.w13, (size_t)a.C * 2 * I * d * es);
    alloc(c.w2, (size_t)a.C * d * I * es);
    alloc(c.w13s, (size_t)2 * Is * d * es);
    alloc(c.w2s, (size_t)d * Is * es);
    alloc(c.la, (size_t)N * r * d * es);
    alloc(c.lb, (size_t)N * d * r * es);
    alloc(c.h, (size_t)S * a.ldh * es);
    alloc(c.hs, (size_t)T * a.ldhs * es);
    alloc(c.u, (size_t)S * r * 4);
    alloc(c.ys, (size_t)S * d * 4);
    alloc(c.ysh, (size_t)T * d * 4);
    alloc(c.sg, (size_t)T * 4);
    alloc(c.perm, (size_t)S * 4);
    alloc(c.off, (size_t)3 * (N + 1) * 4);
    alloc(c.res, (size_t)N * 4);
    int32_t* rs = reinterpret_cast<int32_t*>(c.res.p());
    for (int e = 0; e < N; ++e) rs[e] = -1;
    for (int i = 0; i < R && i < N; ++i) rs[(i * 7) % N] = i;  // R resident experts in slots 0..R-1
    std::vector<int> key(S);
    for (int t = 0; t < T; ++t) {
        std::vector<int> pick;
        while ((int)pick.size() < K) {
            const int e = (int)(N * urand() * urand());  // skewed towards low ids
            if (std::find(pick.begin(), pick.end(), e) == pick.end()) pick.push_back(e);
        }
        for (int k = 0; k < K; ++k) {
            const int e = pick[k];
            const int cl = rs[e] >= 0 ? SPICE_CLASS_HIT : (urand() < 0.5 ? SPICE_CLASS_LORE : SPICE_CLASS_EXACT);
            key[t * K + k] = cl * N + e;
        }
    }
    std::vector<int> cnt(3 * N + 1, 0);
    for (int s = 0; s < S; ++s) ++cnt[key[s] + 1];
    for (int k = 0; k < 3 * N; ++k) cnt[k + 1] += cnt[k];
    int32_t* of = reinterpret_cast<int32_t*>(c.off.p());
    for (int cl = 0; cl < 3; ++cl) {
        for (int e = 0; e < N; ++e) of[cl * (N + 1) + e] = cnt[cl * N + e];
        of[cl * (N + 1) + N] = cnt[cl * N + N];
    }
    int32_t* pm = reinterpret_cast<int32_t*>(c.perm.p());
    std::vector<int> run(cnt.begin(), cnt.end() - 1);
    for (int s = 0; s < S; ++s) pm[run[key[s]]++] = s;
    a.x = c.x.p(); a.perm = pm; a.offsets = of; a.resident_slot = rs;
    a.w13_pool = c.w13.p(); a.w2_pool = c.w2.p(); a.w13s = c.w13s.p(); a.w2s = c.w2s.p();
    a.lore_A = c.la.p(); a.lore_B = c.lb.p();
    a.y_slots = reinterpret_cast<float*>(c.ys.p()); a.y_shared = reinterpret_cast<float*>(c.ysh.p());
    a.sgate = reinterpret_cast<const float*>(c.sg.p());
    a.h = c.h.p(); a.hs = c.hs.p(); a.u = reinterpret_cast<float*>(c.u.p());
}

// The j-th non-empty bucket of class cl in ascending expert order (the selection rule of the
// kernels' group lookup), through the same bucket_of / group_in_range.
bool host_group(const Case& c, int cl, int j, Group& g) {
    const FfnArgs& a = c.a;
    const int32_t* off = a.offsets + cl * (a.N + 1);
    int seen = 0;
    for (int e = 0; e < a.N; ++e) {
        const Group b = bucket_of(off, e, cl, cl == SPICE_CLASS_HIT ? a.resident_slot[e] : -1);
        if (b.n > 0 && seen++ == j) {
            g = b;
            return group_in_range(a, cl, g);
        }
    }
    return false;
}

// Contraction steps of one operand row at ptr (the lane's 16 bytes of every full step, and of
// the partial step if its chunk lies inside kdim).
void stream_row(const Case& c, const Buf& b, const char* ptr, int kdim, int quad) {
    const int nfull = kdim / c.kstep;
    for (int ks = 0; ks < nfull; ++ks) touch(b, ptr + (size_t)ks * kStepBytes, 16);
    if (nfull * c.kstep < kdim && nfull * c.kstep + quad * c.klane < kdim) touch(b, ptr + (size_t)nfull * kStepBytes, 16);
}

template <int KIND>
void up_tile_model(const Case& c, const Group& g, int rt) {
    const FfnArgs& a = c.a;
    const int es = c.es;
    const Buf& wb = c.by_ptr(up_weights<KIND>(a));
    const UpBlock ub = up_block<KIND>(a, g);
    int start, n;
    tile_entries<KIND>(a, g, start, n);
    for (int m = 0; m < 16; ++m)
        for (int quad = 0; quad < 4; ++quad) {
            const int row = tile_row(rt, kTileRows, m, ub.nrows);
            const size_t kb = (size_t)quad * c.klane * es;
            stream_row(c, wb, static_cast<const char*>(wb.p()) + (ub.gate_row0 + row) * (size_t)a.d * es + kb, a.d, quad);
            if (KIND != kKindLore)
                stream_row(c, wb, static_cast<const char*>(wb.p()) + (ub.up_row0 + row) * (size_t)a.d * es + kb, a.d,
                           quad);
            for (int g0 = 0; g0 < n; g0 += kTileRows * kTokTiles) {
                const int ntt = std::min(kTokTiles, (n - g0 + 15) / 16);
                for (int tt = 0; tt < ntt; ++tt) {
                    const int gi = tile_entry(g0, tt, m, n);
                    int tok = gi;
                    if (KIND != kKindShared) {
                        touch(c.perm, a.perm + g.start + gi, 4);
                        const int s = a.perm[g.start + gi];
                        tok = (s >= 0 && s < a.T * a.K) ? s / a.K : 0;
                    }
                    stream_row(c, c.x, static_cast<const char*>(a.x) + (size_t)tok * a.d * es + kb, a.d, quad);
                    const int go = g0 + tt * 16 + m, orow = rt * kTileRows + quad * 4;
                    if (go < n && orow < ub.nrows) {
                        const size_t el = up_out_elem<KIND>(a, start, go, orow);
                        if (KIND == kKindLore) touch(c.u, a.u + el, 16, true);
                        else touch(KIND == kKindHit ? c.h : c.hs,
                                   static_cast<const char*>(KIND == kKindHit ? a.h : a.hs) + el * es, 4 * es, true);
                    }
                }
            }
        }
}

template <int KIND>
void down_tile_model(const Case& c, const Group& g, int rt, int R) {
    const FfnArgs& a = c.a;
    const int es = c.es;
    const Buf& wb = c.by_ptr(down_weights<KIND>(a));
    const Buf& hb = c.by_ptr(down_inputs<KIND>(a));
    const DownBlock db = down_block<KIND>(a, g);
    int start, n;
    tile_entries<KIND>(a, g, start, n);
    for (int m = 0; m < 16; ++m)
        for (int quad = 0; quad < 4; ++quad) {
            const size_t kb = (size_t)quad * c.klane * es;
            for (int rr = 0; rr < R; ++rr) {
                const int row = tile_row(rt, kTileRows * R, rr * kTileRows + m, a.d);
                stream_row(c, wb, static_cast<const char*>(wb.p()) + (db.row0 + row) * (size_t)db.kdim * es + kb,
                           db.kdim, quad);
            }
            for (int g0 = 0; g0 < n; g0 += kTileRows * kTokTiles) {
                const int ntt = std::min(kTokTiles, (n - g0 + 15) / 16);
                for (int tt = 0; tt < ntt; ++tt) {
                    stream_row(c, hb,
                               static_cast<const char*>(hb.p()) + (size_t)(start + tile_entry(g0, tt, m, n)) * db.ld * es + kb,
                               db.kdim, quad);
                    for (int rr = 0; rr < R; ++rr) {
                        const int go = g0 + tt * 16 + m, dim = rt * kTileRows * R + rr * 16 + quad * 4;
                        if (go < n && dim < a.d) {
                            if (KIND == kKindShared) touch(c.sg, a.sgate + go, 4);
                            const size_t el = down_out_elem<KIND>(a, start, go, dim);
                            touch(KIND == kKindHit ? c.ys : c.ysh, (KIND == kKindHit ? a.y_slots : a.y_shared) + el, 16,
                                  true);
                        }
                    }
                }
            }
        }
}

void lore_down_model(const Case& c, const Group& g, int rt) {
    const FfnArgs& a = c.a;
    const int L = c.klane;
    for (int tid = 0; tid < 256; ++tid) {
        const int row = rt * kLoreRows + tid;
        const bool row_ok = row < a.d;
        const size_t brow = lore_b_elem(a, g.e, row_ok ? row : 0, 0);
        for (int g0 = 0; g0 < g.n; g0 += kLoreTok) {
            const int nt = std::min(kLoreTok, g.n - g0);
            for (int q0 = 0; q0 < a.r; q0 += 64) {
                const int nq = std::min(64, a.r - q0);
                for (int i = 0; i * L < nq; ++i)
                    touch(c.lb, static_cast<const char*>(a.lore_B) + (brow + q0 + i * L) * c.es, 16);
                for (int j = 0; j < nt; ++j)
                    for (int q = 0; q < nq; ++q) touch(c.u, a.u + lore_u_elem(a, g.start, g0 + j, q0 + q), 4);
            }
            if (row_ok)
                for (int j = 0; j < nt; ++j) touch(c.ys, a.y_slots + lore_y_elem(a, g.start, g0 + j, row), 4, true);
        }
    }
}

// Every block of the grouped-FFN launches; then the decode layer's variants (16-row HIT and
// shared down tiles).
void replay(const Case& c) {
    const FfnArgs& a = c.a;
    Grid up, dn;
    ffn_grids(a, a.C > 0, a.Is > 0, a.r > 0, up, dn);
    for (long long b = 0; b < up.blocks(); ++b) {
        Tile t;
        if (!up.decode((int)b, t)) { g_fail = 1; continue; }
        Group g{0, 0, a.T, -1};
        if (t.kind == kKindShared) { up_tile_model<kKindShared>(c, g, t.rt); continue; }
        if (!host_group(c, t.kind == kKindHit ? SPICE_CLASS_HIT : SPICE_CLASS_LORE, t.ordinal, g)) continue;
        if (t.kind == kKindHit) up_tile_model<kKindHit>(c, g, t.rt);
        else up_tile_model<kKindLore>(c, g, t.rt);
    }
    Tile none;
    if (up.decode((int)up.blocks(), none)) g_fail = 1;  // past the grid: no tile
    for (long long b = 0; b < dn.blocks(); ++b) {
        Tile t;
        if (!dn.decode((int)b, t)) { g_fail = 1; continue; }
        Group g{0, 0, a.T, -1};
        if (t.kind == kKindShared) { down_tile_model<kKindShared>(c, g, t.rt, kDownRows); continue; }
        if (!host_group(c, t.kind == kKindHit ? SPICE_CLASS_HIT : SPICE_CLASS_LORE, t.ordinal, g)) continue;
        if (t.kind == kKindHit) down_tile_model<kKindHit>(c, g, t.rt, kDownRows);
        else lore_down_model(c, g, t.rt);
    }
    // decode layer: shared and (small batches) HIT down tiles of 16 rows
    if (a.Is > 0)
        for (int rt = 0; rt < (a.d + 15) / 16; ++rt) down_tile_model<kKindShared>(c, Group{0, 0, a.T, -1}, rt, 1);
    for (int j = 0; j < std::min(std::min(a.N, a.C), a.T * a.K); ++j) {
        Group g;
        if (!host_group(c, SPICE_CLASS_HIT, j, g)) continue;
        for (int rt = 0; rt < (a.d + 15) / 16; ++rt) down_tile_model<kKindHit>(c, g, rt, 1);
    }
}

}  // namespace

int main() {
    struct S { int d, N, K, I, Is, r, R, T, dtype; };
    const S shapes[] = {
        {2048, 64, 6, 1408, 2816, 32, 32, 1, SPICE_BF16},  // DeepSeek-V2-Lite-shaped decode
        {2048, 64, 6, 1408, 2816, 32, 32, 8, SPICE_BF16},
        {2048, 64, 6, 1408, 2816, 32, 32, 32, SPICE_BF16},
        {200, 16, 4, 104, 168, 24, 6, 37, SPICE_BF16},     // ragged tails everywhere
        {196, 12, 3, 92, 100, 12, 4, 41, SPICE_F32},
        {200, 16, 4, 104, 168, 24, 16, 19, SPICE_BF16},    // all resident
        {200, 16, 4, 104, 168, 24, 0, 19, SPICE_BF16},     // none resident
        {256, 16, 4, 256, 384, 16, 5, 70, SPICE_BF16},
        {96, 8, 8, 40, 0, 8, 3, 9, SPICE_F32},             // K = N, no shared block
    };
    for (const S& s : shapes) {
        Case c;
        make_case(c, s.d, s.N, s.K, s.I, s.Is, s.r, s.R, s.T, s.dtype);
        replay(c);
    }
    std::printf("%lld accesses checked\n%s\n", g_access, g_fail ? "FAILED" : "ok");
    return g_fail;
}
