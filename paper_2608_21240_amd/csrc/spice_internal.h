// Internal declarations shared by the HIP kernels and the C-ABI layer of libspice_moe.
#pragma once

#include <hip/hip_runtime_api.h>
#include <stddef.h>
#include <stdint.h>

#include "spice_moe.h"

namespace spice {

// Workspace control region (32-bit words at the start of every workspace).
constexpr int kWordFlags = 0;       // device flags, SPICE_FLAG_* (atomic OR)
constexpr int kWordWorkCount = 16;  // [3] non-empty buckets per class (the work lists' lengths)
constexpr int kWordScanCount = 32;  // arrivals of the prefill bucket-scan blocks
constexpr int kWordRouteDone = 33;  // arrivals of the tokens' last routing blocks (decode routing call)
constexpr int kWordWorkList = 1024; // [3][N] int4 work records {expert, pool slot, start, n}
// [T] arrivals of a token's routing blocks (T <= kRouteTokenMaxT), each counter alone in a
// 128-byte line: the atomics of different tokens' blocks do not queue on one line
constexpr int kWordTokCount = 4096;
constexpr int kTokCountStride = 32;  // words between two tokens' counters
static_assert(kWordWorkList + 3 * SPICE_MAX_EXPERTS * 4 <= kWordTokCount, "work lists overlap the counters");

// Largest T whose routing spreads each token's router rows over a few blocks (larger T:
// the tiled logits kernel).
constexpr int kRouteTokenMaxT = 256;
static_assert((kWordTokCount + kRouteTokenMaxT * kTokCountStride) * 4 <= SPICE_WS_CONTROL_BYTES, "control region too small");
// [T*K] bucket keys (class * N + expert) of the decode routing call's slots, written through
// to the device-coherent level for the block that buckets them (top-K of 64 at most)
constexpr int kWordSlotKeys = 12288;
static_assert(kWordTokCount + kRouteTokenMaxT * kTokCountStride <= kWordSlotKeys, "slot keys overlap the counters");
static_assert((kWordSlotKeys + kRouteTokenMaxT * 64) * 4 <= SPICE_WS_CONTROL_BYTES, "control region too small");
// Most slots T*K of the fused decode-layer launches (layer_decode.hip); larger calls take
// the separate routing, FFN and combine launches.
constexpr int kLayerMaxSlots = 1024;

// Row padding (elements) of the SwiGLU intermediates in the workspace: row strides
// that are multiples of large powers of two put every row of a tile on the same
// HBM channel.
constexpr int kHPad = 64;

// Byte offsets of the workspace regions for one (cfg, T).
struct WsLayout {
    size_t logits;  // fp64 [T][N]
    size_t h;       // SwiGLU intermediate of routed slots [T*K][I + kHPad] (dtype)
    size_t hs;      // shared-block intermediate [T][I_s + kHPad] (dtype)
    size_t u;       // LoRE A x, fp32 [T*K][r]
    size_t sgate;   // output gate of the shared block, fp32 [T]
    size_t total;
};
WsLayout ws_layout(const spice_moe_cfg_t& c, int32_t T);

// Which expert groups a grouped-FFN launch covers.
enum : int { kDoHit = 1, kDoShared = 2, kDoLore = 4 };

struct RouteArgs {
    int32_t T, d, N, K, C, dtype, norm_topk, conf_mode;
    float tau;
    const void* x;
    const void* wg;
    const float* bias;
    const int32_t* resident_slot;
    const float* conf;
    double* logits_out;   // caller's, nullable
    double* logits_ws;    // workspace copy read by the top-K step
    int32_t* topk_idx;
    float* topk_w;
    uint8_t* slot_class;
    int32_t* offsets;
    int32_t* perm;
    int32_t* inv_perm;
    uint32_t* ctrl;       // workspace control words
    int32_t* worklist;    // [3][N][4] work records (control region)
    int32_t* wl_count;    // [3] their lengths (control region)
    const void* w_sg;     // nullable: the shared block's gate row [d]; sgate[t] = sigmoid(w_sg . x[t])
    float* sgate;         // [T], written when w_sg is set
    // device-visible addresses of the caller's pinned host copies (each nullable)
    void* hx;
    int32_t* h_idx;
    float* h_w;
    uint8_t* h_cls;
    int32_t* h_counts;
    uint32_t* h_ready;    // nullable: receives ready_value once every host copy has landed
    uint32_t ready_value;
};

// Bytes of one routed expert's W13 [2I][d] and W2 [d][I] in the cfg's weight format.
inline size_t expert_w13_bytes(const spice_moe_cfg_t& c) {
    const size_t n = (size_t)2 * c.inter * c.d;
    return c.wfmt == SPICE_WFMT_MXFP4 ? n / 2 + n / 32 : n * (c.dtype == SPICE_BF16 ? 2 : 4);
}
inline size_t expert_w2_bytes(const spice_moe_cfg_t& c) {
    const size_t n = (size_t)c.inter * c.d;
    return c.wfmt == SPICE_WFMT_MXFP4 ? n / 2 + n / 32 : n * (c.dtype == SPICE_BF16 ? 2 : 4);
}

struct FfnArgs {
    int32_t T, d, N, K, C, I, Is, r, dtype, groups;
    int32_t wfmt;  // SPICE_WFMT_*: the pools hold MXFP4 blobs when SPICE_WFMT_MXFP4
    int32_t ldh, ldhs;  // row strides (elements) of h and hs
    const void* x;
    const int32_t* perm;
    const int32_t* offsets;
    const int32_t* resident_slot;
    const void* w13_pool;
    const void* w2_pool;
    const void* w13s;
    const void* w2s;
    const void* lore_A;
    const void* lore_B;
    float* y_slots;
    float* y_shared;
    const float* sgate;  // nullable: y_shared[t] is scaled by sgate[t] (gated shared block)
    void* h;        // workspace [T*K][I]
    void* hs;       // workspace [T][I_s]
    float* u;       // workspace [T*K][r]
    uint32_t* ctrl;
};

// The fetched-expert FFN (M_fetch of Eq. 12): fetch slot j serves the bucket
// (EXACT, fetch_expert[j]) with the weights in slot j of the fetch pool (passed as
// the FfnArgs pools), and relabels that bucket's slots EXACT -> EXACT_GPU.
struct FetchArgs {
    const int32_t* fetch_expert;  // device [n_slots], -1 = unused slot
    uint8_t* slot_class;          // device [T*K]
    int32_t n_slots;
};

// One depth of the speculative-prefetch draft rollout (spec_draft.hip).
struct SpecArgs {
    int32_t T, d, K, dtype, delta, l_min, last, lore;
    float tau;
    const void* h_in;
    void* h_out;            // may equal h_in
    const int32_t* topk_idx;
    const float* topk_w;
    const int32_t* inv_perm;
    const float* y_slots;
    const float* y_shared;
    int32_t* halted;        // [T], in/out
    int32_t* pred_idx;      // [T][K]
    float* pred_prob;       // [T][K]
    float* conf;            // [T]
    uint32_t* ctrl;
    // device-visible addresses of the caller's pinned host copies (each nullable)
    int32_t* h_pred_idx;
    float* h_pred_prob;
    float* h_conf;
};

struct CombineArgs {
    int32_t T, d, K, dtype;
    const float* topk_w;
    const uint8_t* slot_class;
    const int32_t* inv_perm;
    const float* y_slots;
    const float* y_shared;
    const float* resid;
    void* out;
};

// Grouped MFMA GEMMs of the HIT experts and the shared block for large token
// counts (bf16; used by launch_expert_ffn when expert_gemm_applies).
constexpr int kGemmMinTokens = 256;

struct GemmArgs {
    int32_t T, d, N, K, C, I, Is;
    int32_t ldh, ldhs;
    int32_t super_up[2], super_dn[2];  // shared-block super-tile (weight tiles, token tiles)
    const uint16_t* x;
    const int32_t* perm;
    const int32_t* offsets;  // HIT class row of the bucket offsets
    const int32_t* resident_slot;
    const uint16_t* w13_pool;
    const uint16_t* w2_pool;
    const uint16_t* w13s;
    const uint16_t* w2s;
    uint16_t* h;
    uint16_t* hs;
    float* y_slots;
    float* y_shared;
    const float* sgate;  // nullable, as in FfnArgs
    uint32_t* ctrl;
};

bool expert_gemm_applies(const FfnArgs& a);
hipError_t launch_expert_gemm(const FfnArgs& a, bool hit, bool shared, hipStream_t s);

hipError_t launch_route_bucket(const RouteArgs& a, hipStream_t s);
// The fused decode layer (routing, bucketing, shared block, HIT and LoRE FFN) in three
// launches; bf16/fp32 or MXFP4 routed experts, T <= kRouteTokenMaxT, T*K <= kLayerMaxSlots.
hipError_t launch_layer_decode(const RouteArgs& r, const FfnArgs& f, hipStream_t s);
hipError_t launch_expert_ffn(const FfnArgs& a, hipStream_t s);
// The same launch with MXFP4 routed experts (expert_ffn_mx.hip).
hipError_t launch_expert_ffn_mx(const FfnArgs& a, hipStream_t s);
// sgate[t] = sigmoid(w_sg . x[t]) for T tokens (fp64 dot products), shared_gate.hip.
hipError_t launch_shared_gate(const void* x, const void* w_sg, int32_t T, int32_t d, int32_t dtype, float* sgate,
                              hipStream_t s);
hipError_t launch_expert_ffn_fetched(const FfnArgs& a, const FetchArgs& f, hipStream_t s);
hipError_t launch_combine(const CombineArgs& a, hipStream_t s);
hipError_t launch_spec_update(const SpecArgs& a, hipStream_t s);

// LoRE calibration fit (lore_fit.hip).
hipError_t launch_fit_setup(int32_t n, int32_t* perm, int32_t* offsets, int32_t* resident, hipStream_t s);
hipError_t launch_fit_residual(size_t count, float* y, const float* shared, hipStream_t s);
hipError_t launch_fit_gram(int32_t n, int32_t d, int dtype, const void* M, double* G, hipStream_t s);
hipError_t launch_fit_project(int32_t n, int32_t d, int32_t r, int dtype, const void* M, const double* C, float* out,
                              bool b_layout, hipStream_t s);
hipError_t launch_fill_u32(uint32_t* p, size_t words, uint32_t value, hipStream_t s);

}  // namespace spice
