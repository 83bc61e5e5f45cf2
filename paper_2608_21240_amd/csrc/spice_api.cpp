// C-ABI layer of libspice_moe: argument checks, workspace layout, kernel launches.
// Every entry point validates on the host before it touches HIP, returns a
// status and never throws across the ABI.
#include <algorithm>
#include <chrono>
#include <cmath>
#include <cstdint>
#include <cstring>
#include <exception>
#include <string>

#include "spice_internal.h"

namespace {

thread_local std::string g_last_error;

spice_status_t fail(spice_status_t st, const std::string& msg) {
    g_last_error = msg;
    return st;
}

spice_status_t hip_fail(hipError_t e, const char* where) {
    return fail(SPICE_ERR_HIP, std::string(where) + ": " + hipGetErrorString(e));
}

size_t align256(size_t n) { return (n + 255) & ~(size_t)255; }

size_t elem_size(const spice_moe_cfg_t& c) { return c.dtype == SPICE_BF16 ? 2 : 4; }

spice_status_t check_cfg(const spice_moe_cfg_t* c) {
    if (!c) return fail(SPICE_ERR_INVALID, "cfg is NULL");
    if (c->dtype != SPICE_F32 && c->dtype != SPICE_BF16)
        return fail(SPICE_ERR_UNSUPPORTED, "dtype must be SPICE_F32 or SPICE_BF16");
    if (c->d <= 0) return fail(SPICE_ERR_INVALID, "d must be positive");
    if (c->n_experts < 1) return fail(SPICE_ERR_INVALID, "n_experts must be >= 1");
    if (c->n_experts > SPICE_MAX_EXPERTS) return fail(SPICE_ERR_UNSUPPORTED, "n_experts above 256");
    if (c->top_k < 1 || c->top_k > c->n_experts) return fail(SPICE_ERR_INVALID, "top_k must be in [1, n_experts]");
    if (c->top_k > 64) return fail(SPICE_ERR_UNSUPPORTED, "top_k above 64");
    if (c->inter <= 0) return fail(SPICE_ERR_INVALID, "inter must be positive");
    if (c->shared_inter < 0) return fail(SPICE_ERR_INVALID, "shared_inter must be >= 0");
    if (c->lore_rank < 0) return fail(SPICE_ERR_INVALID, "lore_rank must be >= 0");
    if (c->lore_rank > SPICE_MAX_LORE_RANK) return fail(SPICE_ERR_UNSUPPORTED, "lore_rank above 256");
    if (c->n_slots < 0) return fail(SPICE_ERR_INVALID, "n_slots must be >= 0");
    if (c->norm_topk != 0 && c->norm_topk != 1) return fail(SPICE_ERR_INVALID, "norm_topk must be 0 or 1");
    if (c->conf_mode < SPICE_CONF_INPUT || c->conf_mode > SPICE_CONF_GATE_RENORM)
        return fail(SPICE_ERR_INVALID, "conf_mode must be a SPICE_CONF_* value");
    if (c->wfmt != SPICE_WFMT_DTYPE && c->wfmt != SPICE_WFMT_MXFP4)
        return fail(SPICE_ERR_INVALID, "wfmt must be SPICE_WFMT_DTYPE or SPICE_WFMT_MXFP4");
    if (c->wfmt == SPICE_WFMT_MXFP4 && c->dtype != SPICE_BF16)
        return fail(SPICE_ERR_UNSUPPORTED, "MXFP4 expert weights need dtype SPICE_BF16");
    if (c->wfmt == SPICE_WFMT_MXFP4 && (c->d % 32 || c->inter % 32))
        return fail(SPICE_ERR_UNSUPPORTED, "MXFP4 expert weights need d and inter multiples of 32");
    if (c->wfmt == SPICE_WFMT_MXFP4 && (c->d > SPICE_MXFP4_MAX_K || c->inter > SPICE_MXFP4_MAX_K))
        return fail(SPICE_ERR_UNSUPPORTED, "MXFP4 expert weights need d and inter at most SPICE_MXFP4_MAX_K");
    const int al = c->dtype == SPICE_BF16 ? 8 : 4;
    if (c->d % al || c->inter % al || c->shared_inter % al || c->lore_rank % al)
        return fail(SPICE_ERR_UNSUPPORTED, "d, inter, shared_inter and lore_rank must be multiples of " +
                                               std::to_string(al) + " (16-byte vector loads)");
    if ((int64_t)c->d * (c->dtype == SPICE_BF16 ? 2 : 4) > 16384)
        return fail(SPICE_ERR_UNSUPPORTED, "hidden rows above 16 KiB (d > 8192 bf16 / 4096 fp32)");
    const int64_t big = (int64_t)std::max({c->d, c->inter, c->shared_inter});
    if (big * SPICE_MAX_TOKENS * 64 > INT64_MAX / 8) return fail(SPICE_ERR_INVALID, "sizes overflow");
    return SPICE_OK;
}

spice_status_t check_tokens(const spice_moe_cfg_t& c, int32_t T) {
    if (T < 0) return fail(SPICE_ERR_INVALID, "T must be >= 0");
    if (T > SPICE_MAX_TOKENS) return fail(SPICE_ERR_UNSUPPORTED, "T above SPICE_MAX_TOKENS");
    if ((int64_t)T * c.top_k > INT32_MAX) return fail(SPICE_ERR_INVALID, "T*K overflows int32");
    return SPICE_OK;
}

spice_status_t check_ws(const spice_moe_cfg_t& c, int32_t T, const void* ws, size_t ws_bytes) {
    if (!ws) return fail(SPICE_ERR_INVALID, "workspace is NULL");
    const size_t need = spice::ws_layout(c, T).total;
    if (ws_bytes < need)
        return fail(SPICE_ERR_WORKSPACE, "workspace has " + std::to_string(ws_bytes) + " bytes, needs " +
                                             std::to_string(need));
    return SPICE_OK;
}

bool overlaps(const void* a, size_t an, const void* b, size_t bn) {
    if (!a || !b || an == 0 || bn == 0) return false;
    const uintptr_t a0 = (uintptr_t)a, b0 = (uintptr_t)b;
    return a0 < b0 + bn && b0 < a0 + an;
}

// Address a kernel may use for a caller buffer that must be pinned host memory
// (host_only) or either device or pinned host memory.  Pageable memory would make
// the kernel fault, so it is rejected here.
spice_status_t gpu_address(const void* p, bool host_only, const char* name, void** dev) {
    hipPointerAttribute_t at{};
    const hipError_t e = hipPointerGetAttributes(&at, p);
    if (e != hipSuccess) {
        (void)hipGetLastError();
        return fail(SPICE_ERR_INVALID, std::string(name) + ": not device or pinned host memory (" +
                                           hipGetErrorString(e) + ")");
    }
    if (at.type == hipMemoryTypeHost) {
        *dev = at.devicePointer ? at.devicePointer : const_cast<void*>(p);
        return SPICE_OK;
    }
    if (!host_only && (at.type == hipMemoryTypeDevice || at.type == hipMemoryTypeManaged)) {
        *dev = const_cast<void*>(p);
        return SPICE_OK;
    }
    return fail(SPICE_ERR_INVALID, std::string(name) + (host_only ? ": must be pinned host memory"
                                                                   : ": not device or pinned host memory"));
}

// Device-visible addresses of the caller's pinned host copies (each optional).
spice_status_t resolve_host_out(const spice_host_out_t* host_out, spice::RouteArgs& a) {
    if (!host_out) return SPICE_OK;
    spice_status_t st;
    void* d = nullptr;
    if (host_out->x) {
        if ((st = gpu_address(host_out->x, true, "host_out.x", &d)) != SPICE_OK) return st;
        a.hx = d;
    }
    if (host_out->topk_idx) {
        if ((st = gpu_address(host_out->topk_idx, true, "host_out.topk_idx", &d)) != SPICE_OK) return st;
        a.h_idx = static_cast<int32_t*>(d);
    }
    if (host_out->topk_w) {
        if ((st = gpu_address(host_out->topk_w, true, "host_out.topk_w", &d)) != SPICE_OK) return st;
        a.h_w = static_cast<float*>(d);
    }
    if (host_out->slot_class) {
        if ((st = gpu_address(host_out->slot_class, true, "host_out.slot_class", &d)) != SPICE_OK) return st;
        a.h_cls = static_cast<uint8_t*>(d);
    }
    if (host_out->class_counts) {
        if ((st = gpu_address(host_out->class_counts, true, "host_out.class_counts", &d)) != SPICE_OK) return st;
        a.h_counts = static_cast<int32_t*>(d);
    }
    if (host_out->ready) {
        if ((st = gpu_address(host_out->ready, true, "host_out.ready", &d)) != SPICE_OK) return st;
        a.h_ready = static_cast<uint32_t*>(d);
        a.ready_value = host_out->ready_value;
    }
    return SPICE_OK;
}

#define SPICE_REQUIRE(ptr, name) \
    if (!(ptr)) return fail(SPICE_ERR_INVALID, name " is NULL")

#define SPICE_TRY_BEGIN try {
#define SPICE_TRY_END                                                  \
    }                                                                  \
    catch (const std::exception& ex) {                                 \
        return fail(SPICE_ERR_INTERNAL, std::string("internal: ") + ex.what()); \
    }                                                                  \
    catch (...) {                                                      \
        return fail(SPICE_ERR_INTERNAL, "internal: unknown exception"); \
    }

}  // namespace

namespace spice {

WsLayout ws_layout(const spice_moe_cfg_t& c, int32_t T) {
    WsLayout L{};
    const size_t t = (size_t)std::max(T, 0), slots = t * (size_t)c.top_k, es = elem_size(c);
    size_t off = SPICE_WS_CONTROL_BYTES;
    L.logits = off; off += align256(t * (size_t)c.n_experts * sizeof(double));
    L.h = off;      off += align256(slots * ((size_t)c.inter + kHPad) * es);
    L.hs = off;     off += align256(t * ((size_t)c.shared_inter + kHPad) * es);
    L.u = off;      off += align256(slots * (size_t)c.lore_rank * sizeof(float));
    L.sgate = off;  off += align256(t * sizeof(float));
    L.total = off;
    return L;
}

}  // namespace spice

extern "C" {

size_t spice_workspace_bytes(const spice_moe_cfg_t* cfg, int32_t T) {
    if (check_cfg(cfg) != SPICE_OK || check_tokens(*cfg, T) != SPICE_OK) return 0;
    return spice::ws_layout(*cfg, T).total;
}

spice_status_t spice_workspace_init(void* ws, size_t ws_bytes, spice_stream_t stream) {
    SPICE_TRY_BEGIN
    SPICE_REQUIRE(ws, "workspace");
    if (ws_bytes < SPICE_WS_CONTROL_BYTES) return fail(SPICE_ERR_WORKSPACE, "workspace smaller than its control region");
    hipError_t e = spice::launch_fill_u32(static_cast<uint32_t*>(ws), SPICE_WS_CONTROL_BYTES / 4, 0u, stream);
    if (e != hipSuccess) return hip_fail(e, "spice_workspace_init");
    return SPICE_OK;
    SPICE_TRY_END
}

spice_status_t spice_workspace_flags(void* ws, size_t ws_bytes, uint32_t* flags, int32_t clear,
                                     spice_stream_t stream) {
    SPICE_TRY_BEGIN
    SPICE_REQUIRE(ws, "workspace");
    SPICE_REQUIRE(flags, "flags");
    if (ws_bytes < SPICE_WS_CONTROL_BYTES) return fail(SPICE_ERR_WORKSPACE, "workspace smaller than its control region");
    uint32_t* ctrl = static_cast<uint32_t*>(ws);
    hipError_t e = hipMemcpyAsync(flags, ctrl + spice::kWordFlags, sizeof(uint32_t), hipMemcpyDeviceToHost, stream);
    if (e == hipSuccess) e = hipStreamSynchronize(stream);
    if (e == hipSuccess && clear) e = spice::launch_fill_u32(ctrl + spice::kWordFlags, 1, 0u, stream);
    if (e != hipSuccess) return hip_fail(e, "spice_workspace_flags");
    return SPICE_OK;
    SPICE_TRY_END
}

}  // extern "C"

namespace {

// Checks of a routing call and its kernel arguments (no launch).  T == 0 is valid; the
// caller returns before launching.
spice_status_t prep_route(const spice_moe_cfg_t* cfg, int32_t T, const void* x, const void* w_gate,
                          const float* logit_bias, const int32_t* resident_slot, const float* conf, double* logits,
                          int32_t* topk_idx, float* topk_w, uint8_t* slot_class, int32_t* offsets, int32_t* perm,
                          int32_t* inv_perm, const spice_host_out_t* host_out, void* ws, size_t ws_bytes,
                          spice::RouteArgs& a) {
    spice_status_t st = check_cfg(cfg);
    if (st != SPICE_OK) return st;
    const spice_moe_cfg_t& c = *cfg;
    if ((st = check_tokens(c, T)) != SPICE_OK) return st;
    if (T == 0) return SPICE_OK;
    SPICE_REQUIRE(x, "x");
    SPICE_REQUIRE(w_gate, "w_gate");
    SPICE_REQUIRE(resident_slot, "resident_slot");
    if (c.conf_mode == SPICE_CONF_INPUT && !conf) return fail(SPICE_ERR_INVALID, "conf is NULL in SPICE_CONF_INPUT mode");
    SPICE_REQUIRE(topk_idx, "topk_idx");
    SPICE_REQUIRE(topk_w, "topk_w");
    SPICE_REQUIRE(slot_class, "slot_class");
    SPICE_REQUIRE(offsets, "offsets");
    SPICE_REQUIRE(perm, "perm");
    SPICE_REQUIRE(inv_perm, "inv_perm");
    if ((st = check_ws(c, T, ws, ws_bytes)) != SPICE_OK) return st;
    const spice::WsLayout L = spice::ws_layout(c, T);
    char* wsb = static_cast<char*>(ws);
    a = spice::RouteArgs{};
    a.T = T; a.d = c.d; a.N = c.n_experts; a.K = c.top_k; a.C = c.n_slots; a.dtype = c.dtype;
    a.norm_topk = c.norm_topk; a.conf_mode = c.conf_mode; a.tau = c.tau;
    a.x = x; a.wg = w_gate; a.bias = logit_bias; a.resident_slot = resident_slot; a.conf = conf;
    a.logits_out = logits; a.logits_ws = reinterpret_cast<double*>(wsb + L.logits);
    a.topk_idx = topk_idx; a.topk_w = topk_w; a.slot_class = slot_class;
    a.offsets = offsets; a.perm = perm; a.inv_perm = inv_perm;
    a.ctrl = reinterpret_cast<uint32_t*>(wsb);
    a.wl_count = reinterpret_cast<int32_t*>(wsb) + spice::kWordWorkCount;
    a.worklist = reinterpret_cast<int32_t*>(wsb) + spice::kWordWorkList;
    return resolve_host_out(host_out, a);
}

}  // namespace

extern "C" {

spice_status_t moe_route_bucket(const spice_moe_cfg_t* cfg, int32_t T, const void* x, const void* w_gate,
                                const float* logit_bias, const int32_t* resident_slot, const float* conf,
                                double* logits, int32_t* topk_idx, float* topk_w, uint8_t* slot_class,
                                int32_t* offsets, int32_t* perm, int32_t* inv_perm,
                                const spice_host_out_t* host_out, void* ws, size_t ws_bytes, spice_stream_t stream) {
    SPICE_TRY_BEGIN
    spice::RouteArgs a{};
    const spice_status_t st = prep_route(cfg, T, x, w_gate, logit_bias, resident_slot, conf, logits, topk_idx, topk_w,
                                         slot_class, offsets, perm, inv_perm, host_out, ws, ws_bytes, a);
    if (st != SPICE_OK || T == 0) return st;
    hipError_t e = spice::launch_route_bucket(a, stream);
    if (e != hipSuccess) return hip_fail(e, "moe_route_bucket");
    return SPICE_OK;
    SPICE_TRY_END
}

}  // extern "C"

namespace {

// Checks of a grouped-FFN call and its kernel arguments (no launch; T == 0 is valid).
spice_status_t prep_ffn(const spice_moe_cfg_t* cfg, int32_t T, const void* x, const int32_t* perm,
                        const int32_t* offsets, const int32_t* resident_slot, const void* w13_pool,
                        const void* w2_pool, const void* w13_shared, const void* w2_shared, const void* lore_A,
                        const void* lore_B, float* y_slots, float* y_shared, void* ws, size_t ws_bytes, int groups,
                        const char* name, spice::FfnArgs& a) {
    spice_status_t st = check_cfg(cfg);
    if (st != SPICE_OK) return st;
    const spice_moe_cfg_t& c = *cfg;
    if ((st = check_tokens(c, T)) != SPICE_OK) return st;
    if (T == 0) return SPICE_OK;
    SPICE_REQUIRE(x, "x");
    SPICE_REQUIRE(perm, "perm");
    SPICE_REQUIRE(offsets, "offsets");
    SPICE_REQUIRE(y_slots, "y_slots");
    if (groups & spice::kDoHit) {
        SPICE_REQUIRE(resident_slot, "resident_slot");
        if (c.n_slots > 0) {
            SPICE_REQUIRE(w13_pool, "w13_pool");
            SPICE_REQUIRE(w2_pool, "w2_pool");
        }
    }
    if ((groups & spice::kDoShared) && c.shared_inter > 0) {
        SPICE_REQUIRE(w13_shared, "w13_shared");
        SPICE_REQUIRE(w2_shared, "w2_shared");
        SPICE_REQUIRE(y_shared, "y_shared");
    }
    if ((groups & spice::kDoLore) && c.lore_rank > 0) {
        SPICE_REQUIRE(lore_A, "lore_A");
        SPICE_REQUIRE(lore_B, "lore_B");
    }
    if ((st = check_ws(c, T, ws, ws_bytes)) != SPICE_OK) return st;
    if (c.wfmt == SPICE_WFMT_MXFP4 && ((size_t)T * c.top_k * ((size_t)c.inter + spice::kHPad) * 2 >= (1ull << 31) ||
                                       (size_t)T * c.d * 2 >= (1ull << 31)))
        return fail(SPICE_ERR_UNSUPPORTED, std::string(name) + ": MXFP4 experts need x and H below 2 GiB");
    const size_t ysz = (size_t)T * c.top_k * c.d * sizeof(float);
    if (overlaps(y_slots, ysz, x, (size_t)T * c.d * elem_size(c)) ||
        overlaps(y_shared, (size_t)T * c.d * sizeof(float), x, (size_t)T * c.d * elem_size(c)) ||
        overlaps(y_slots, ysz, y_shared, (size_t)T * c.d * sizeof(float)))
        return fail(SPICE_ERR_INVALID, std::string(name) + ": outputs alias each other or x");
    const spice::WsLayout L = spice::ws_layout(c, T);
    char* wsb = static_cast<char*>(ws);
    a = spice::FfnArgs{};
    a.T = T; a.d = c.d; a.N = c.n_experts; a.K = c.top_k; a.C = c.n_slots; a.I = c.inter;
    a.Is = c.shared_inter; a.r = c.lore_rank; a.dtype = c.dtype; a.groups = groups;
    a.ldh = c.inter + spice::kHPad; a.ldhs = c.shared_inter + spice::kHPad;
    a.x = x; a.perm = perm; a.offsets = offsets; a.resident_slot = resident_slot;
    a.w13_pool = w13_pool; a.w2_pool = w2_pool; a.w13s = w13_shared; a.w2s = w2_shared;
    a.lore_A = lore_A; a.lore_B = lore_B; a.y_slots = y_slots; a.y_shared = y_shared;
    a.h = wsb + L.h; a.hs = wsb + L.hs; a.u = reinterpret_cast<float*>(wsb + L.u);
    a.ctrl = reinterpret_cast<uint32_t*>(wsb);
    a.wfmt = c.wfmt;
    return SPICE_OK;
}

// The grouped FFN's launches: the shared block's gate first when it has one, then the
// tiles (MXFP4 or dtype experts).
hipError_t launch_ffn(spice::FfnArgs& a, const void* w_shared_gate, void* ws, const spice_moe_cfg_t& c,
                      hipStream_t stream) {
    if (w_shared_gate && (a.groups & spice::kDoShared) && c.shared_inter > 0) {
        float* sg = reinterpret_cast<float*>(static_cast<char*>(ws) + spice::ws_layout(c, a.T).sgate);
        hipError_t e = spice::launch_shared_gate(a.x, w_shared_gate, a.T, c.d, c.dtype, sg, stream);
        if (e != hipSuccess) return e;
        a.sgate = sg;
    }
    return c.wfmt == SPICE_WFMT_MXFP4 ? spice::launch_expert_ffn_mx(a, stream) : spice::launch_expert_ffn(a, stream);
}

spice_status_t run_ffn(const spice_moe_cfg_t* cfg, int32_t T, const void* x, const int32_t* perm,
                       const int32_t* offsets, const int32_t* resident_slot, const void* w13_pool, const void* w2_pool,
                       const void* w13_shared, const void* w2_shared, const void* lore_A, const void* lore_B,
                       float* y_slots, float* y_shared, void* ws, size_t ws_bytes, spice_stream_t stream, int groups,
                       const char* name, const void* w_shared_gate = nullptr) {
    spice::FfnArgs a{};
    const spice_status_t st = prep_ffn(cfg, T, x, perm, offsets, resident_slot, w13_pool, w2_pool, w13_shared,
                                       w2_shared, lore_A, lore_B, y_slots, y_shared, ws, ws_bytes, groups, name, a);
    if (st != SPICE_OK || T == 0) return st;
    const hipError_t e = launch_ffn(a, w_shared_gate, ws, *cfg, stream);
    if (e != hipSuccess) return hip_fail(e, name);
    return SPICE_OK;
}

}  // namespace

extern "C" {

spice_status_t moe_expert_ffn_grouped(const spice_moe_cfg_t* cfg, int32_t T, const void* x, const int32_t* perm,
                                      const int32_t* offsets, const int32_t* resident_slot, const void* w13_pool,
                                      const void* w2_pool, const void* w13_shared, const void* w2_shared,
                                      const void* lore_A, const void* lore_B, float* y_slots, float* y_shared,
                                      void* ws, size_t ws_bytes, spice_stream_t stream) {
    SPICE_TRY_BEGIN
    int groups = spice::kDoHit | spice::kDoShared;
    if (lore_A && lore_B) groups |= spice::kDoLore;
    return run_ffn(cfg, T, x, perm, offsets, resident_slot, w13_pool, w2_pool, w13_shared, w2_shared, lore_A,
                   lore_B, y_slots, y_shared, ws, ws_bytes, stream, groups, "moe_expert_ffn_grouped");
    SPICE_TRY_END
}

spice_status_t moe_expert_ffn_grouped_gated(const spice_moe_cfg_t* cfg, int32_t T, const void* x,
                                            const int32_t* perm, const int32_t* offsets, const int32_t* resident_slot,
                                            const void* w13_pool, const void* w2_pool, const void* w13_shared,
                                            const void* w2_shared, const void* w_shared_gate, const void* lore_A,
                                            const void* lore_B, float* y_slots, float* y_shared, void* ws,
                                            size_t ws_bytes, spice_stream_t stream) {
    SPICE_TRY_BEGIN
    int groups = spice::kDoHit | spice::kDoShared;
    if (lore_A && lore_B) groups |= spice::kDoLore;
    if (cfg && cfg->shared_inter > 0 && !w_shared_gate)
        return fail(SPICE_ERR_INVALID, "moe_expert_ffn_grouped_gated: w_shared_gate is NULL");
    return run_ffn(cfg, T, x, perm, offsets, resident_slot, w13_pool, w2_pool, w13_shared, w2_shared, lore_A,
                   lore_B, y_slots, y_shared, ws, ws_bytes, stream, groups, "moe_expert_ffn_grouped_gated",
                   w_shared_gate);
    SPICE_TRY_END
}

spice_status_t lore_surrogate_apply(const spice_moe_cfg_t* cfg, int32_t T, const void* x, const int32_t* perm,
                                    const int32_t* offsets, const void* lore_A, const void* lore_B, float* y_slots,
                                    void* ws, size_t ws_bytes, spice_stream_t stream) {
    SPICE_TRY_BEGIN
    return run_ffn(cfg, T, x, perm, offsets, nullptr, nullptr, nullptr, nullptr, nullptr, lore_A, lore_B, y_slots,
                   nullptr, ws, ws_bytes, stream, spice::kDoLore, "lore_surrogate_apply");
    SPICE_TRY_END
}

spice_status_t moe_expert_ffn_fetched(const spice_moe_cfg_t* cfg, int32_t T, const void* x, const int32_t* perm,
                                      const int32_t* offsets, uint8_t* slot_class, const int32_t* fetch_expert,
                                      const void* w13_fetch, const void* w2_fetch, int32_t n_slots,
                                      float* y_slots, void* ws, size_t ws_bytes, spice_stream_t stream) {
    SPICE_TRY_BEGIN
    spice_status_t st = check_cfg(cfg);
    if (st != SPICE_OK) return st;
    const spice_moe_cfg_t& c = *cfg;
    if ((st = check_tokens(c, T)) != SPICE_OK) return st;
    if (n_slots < 1 || n_slots > c.n_experts)
        return fail(SPICE_ERR_INVALID, "moe_expert_ffn_fetched: n_slots must be in [1, n_experts]");
    if (c.wfmt != SPICE_WFMT_DTYPE)
        return fail(SPICE_ERR_UNSUPPORTED, "moe_expert_ffn_fetched: needs SPICE_WFMT_DTYPE expert weights");
    if (T == 0) return SPICE_OK;
    SPICE_REQUIRE(x, "x");
    SPICE_REQUIRE(perm, "perm");
    SPICE_REQUIRE(offsets, "offsets");
    SPICE_REQUIRE(slot_class, "slot_class");
    SPICE_REQUIRE(fetch_expert, "fetch_expert");
    SPICE_REQUIRE(w13_fetch, "w13_fetch");
    SPICE_REQUIRE(w2_fetch, "w2_fetch");
    SPICE_REQUIRE(y_slots, "y_slots");
    if ((st = check_ws(c, T, ws, ws_bytes)) != SPICE_OK) return st;
    if (overlaps(y_slots, (size_t)T * c.top_k * c.d * sizeof(float), x, (size_t)T * c.d * elem_size(c)))
        return fail(SPICE_ERR_INVALID, "moe_expert_ffn_fetched: y_slots aliases x");
    const spice::WsLayout L = spice::ws_layout(c, T);
    char* wsb = static_cast<char*>(ws);
    spice::FfnArgs a{};
    a.T = T; a.d = c.d; a.N = c.n_experts; a.K = c.top_k; a.C = n_slots; a.I = c.inter;
    a.Is = c.shared_inter; a.r = c.lore_rank; a.dtype = c.dtype; a.groups = spice::kDoHit;
    a.ldh = c.inter + spice::kHPad; a.ldhs = c.shared_inter + spice::kHPad;
    a.x = x; a.perm = perm; a.offsets = offsets; a.resident_slot = nullptr;
    a.w13_pool = w13_fetch; a.w2_pool = w2_fetch; a.y_slots = y_slots;
    a.h = wsb + L.h; a.hs = wsb + L.hs; a.u = reinterpret_cast<float*>(wsb + L.u);
    a.ctrl = reinterpret_cast<uint32_t*>(wsb);
    spice::FetchArgs f{};
    f.fetch_expert = fetch_expert; f.slot_class = slot_class; f.n_slots = n_slots;
    hipError_t e = spice::launch_expert_ffn_fetched(a, f, stream);
    if (e != hipSuccess) return hip_fail(e, "moe_expert_ffn_fetched");
    return SPICE_OK;
    SPICE_TRY_END
}

spice_status_t moe_spec_update(const spice_moe_cfg_t* cfg, int32_t T, int32_t depth, int32_t l_min, float tau,
                               int32_t last, const void* h_in, void* h_out, const int32_t* topk_idx,
                               const float* topk_w, const int32_t* inv_perm, const float* y_slots,
                               const float* y_shared, int32_t* halted, int32_t* pred_idx, float* pred_prob,
                               float* conf, const spice_spec_host_t* host_out, void* ws, size_t ws_bytes,
                               spice_stream_t stream) {
    SPICE_TRY_BEGIN
    spice_status_t st = check_cfg(cfg);
    if (st != SPICE_OK) return st;
    const spice_moe_cfg_t& c = *cfg;
    if ((st = check_tokens(c, T)) != SPICE_OK) return st;
    if (depth < 1) return fail(SPICE_ERR_INVALID, "moe_spec_update: depth must be >= 1");
    if (l_min < 0) return fail(SPICE_ERR_INVALID, "moe_spec_update: l_min must be >= 0");
    if (!(tau >= 0.f) || std::isinf(tau)) return fail(SPICE_ERR_INVALID, "moe_spec_update: tau must be finite and >= 0");
    if (T == 0) return SPICE_OK;
    SPICE_REQUIRE(h_in, "h_in");
    SPICE_REQUIRE(h_out, "h_out");
    SPICE_REQUIRE(topk_idx, "topk_idx");
    SPICE_REQUIRE(topk_w, "topk_w");
    SPICE_REQUIRE(inv_perm, "inv_perm");
    SPICE_REQUIRE(y_shared, "y_shared");
    if (c.lore_rank > 0) SPICE_REQUIRE(y_slots, "y_slots");
    SPICE_REQUIRE(halted, "halted");
    SPICE_REQUIRE(pred_idx, "pred_idx");
    SPICE_REQUIRE(pred_prob, "pred_prob");
    SPICE_REQUIRE(conf, "conf");
    if ((st = check_ws(c, T, ws, ws_bytes)) != SPICE_OK) return st;
    const size_t hb = (size_t)T * c.d * elem_size(c);
    if (h_out != h_in && overlaps(h_out, hb, h_in, hb))
        return fail(SPICE_ERR_INVALID, "moe_spec_update: h_out overlaps h_in without being it");
    spice::SpecArgs a{};
    a.T = T; a.d = c.d; a.K = c.top_k; a.dtype = c.dtype; a.delta = depth; a.l_min = l_min;
    a.last = last != 0; a.lore = c.lore_rank > 0; a.tau = tau;
    a.h_in = h_in; a.h_out = h_out; a.topk_idx = topk_idx; a.topk_w = topk_w; a.inv_perm = inv_perm;
    a.y_slots = y_slots; a.y_shared = y_shared; a.halted = halted; a.pred_idx = pred_idx;
    a.pred_prob = pred_prob; a.conf = conf; a.ctrl = static_cast<uint32_t*>(ws);
    if (host_out) {
        void* d = nullptr;
        if (host_out->pred_idx) {
            if ((st = gpu_address(host_out->pred_idx, true, "host_out.pred_idx", &d)) != SPICE_OK) return st;
            a.h_pred_idx = static_cast<int32_t*>(d);
        }
        if (host_out->pred_prob) {
            if ((st = gpu_address(host_out->pred_prob, true, "host_out.pred_prob", &d)) != SPICE_OK) return st;
            a.h_pred_prob = static_cast<float*>(d);
        }
        if (host_out->conf) {
            if ((st = gpu_address(host_out->conf, true, "host_out.conf", &d)) != SPICE_OK) return st;
            a.h_conf = static_cast<float*>(d);
        }
    }
    const hipError_t e = spice::launch_spec_update(a, stream);
    if (e != hipSuccess) return hip_fail(e, "moe_spec_update");
    return SPICE_OK;
    SPICE_TRY_END
}

}  // extern "C"

namespace {

// Checks of a combine call and its kernel arguments (no launch; T == 0 is valid).
spice_status_t prep_combine(const spice_moe_cfg_t* cfg, int32_t T, const float* topk_w, const uint8_t* slot_class,
                            const int32_t* inv_perm, const float* y_slots, const float* y_shared, const float* resid,
                            void* out, spice::CombineArgs& a) {
    spice_status_t st = check_cfg(cfg);
    if (st != SPICE_OK) return st;
    const spice_moe_cfg_t& c = *cfg;
    if ((st = check_tokens(c, T)) != SPICE_OK) return st;
    if (T == 0) return SPICE_OK;
    SPICE_REQUIRE(topk_w, "topk_w");
    SPICE_REQUIRE(slot_class, "slot_class");
    SPICE_REQUIRE(inv_perm, "inv_perm");
    SPICE_REQUIRE(y_slots, "y_slots");
    SPICE_REQUIRE(y_shared, "y_shared");
    SPICE_REQUIRE(out, "out");
    const size_t osz = (size_t)T * c.d * elem_size(c), fsz = (size_t)T * c.d * sizeof(float);
    if (overlaps(out, osz, y_slots, fsz * c.top_k) || overlaps(out, osz, y_shared, fsz) ||
        overlaps(out, osz, resid, fsz) || overlaps(out, osz, topk_w, (size_t)T * c.top_k * sizeof(float)))
        return fail(SPICE_ERR_INVALID, "moe_combine: out aliases an input");
    void* resid_dev = nullptr;
    if (resid && (st = gpu_address(resid, false, "moe_combine: resid", &resid_dev)) != SPICE_OK) return st;
    a = spice::CombineArgs{};
    a.T = T; a.d = c.d; a.K = c.top_k; a.dtype = c.dtype;
    a.topk_w = topk_w; a.slot_class = slot_class; a.inv_perm = inv_perm; a.y_slots = y_slots;
    a.y_shared = y_shared; a.resid = static_cast<const float*>(resid_dev); a.out = out;
    return SPICE_OK;
}

}  // namespace

extern "C" {

spice_status_t moe_combine(const spice_moe_cfg_t* cfg, int32_t T, const float* topk_w, const uint8_t* slot_class,
                           const int32_t* inv_perm, const float* y_slots, const float* y_shared, const float* resid,
                           void* out, spice_stream_t stream) {
    SPICE_TRY_BEGIN
    spice::CombineArgs a{};
    const spice_status_t st = prep_combine(cfg, T, topk_w, slot_class, inv_perm, y_slots, y_shared, resid, out, a);
    if (st != SPICE_OK || T == 0) return st;
    hipError_t e = spice::launch_combine(a, stream);
    if (e != hipSuccess) return hip_fail(e, "moe_combine");
    return SPICE_OK;
    SPICE_TRY_END
}

spice_status_t moe_layer_gpu(const spice_moe_cfg_t* cfg, int32_t T, const void* x, const void* w_gate,
                             const float* logit_bias, const int32_t* resident_slot, const float* conf,
                             const void* w13_pool, const void* w2_pool, const void* w13_shared, const void* w2_shared,
                             const void* w_shared_gate, const void* lore_A, const void* lore_B, double* logits,
                             int32_t* topk_idx, float* topk_w, uint8_t* slot_class, int32_t* offsets, int32_t* perm,
                             int32_t* inv_perm, float* y_slots, float* y_shared, const spice_host_out_t* host_out,
                             const float* resid, void* out, void* ws, size_t ws_bytes, spice_stream_t stream) {
    SPICE_TRY_BEGIN
    spice::RouteArgs r{};
    spice_status_t st = prep_route(cfg, T, x, w_gate, logit_bias, resident_slot, conf, logits, topk_idx, topk_w,
                                   slot_class, offsets, perm, inv_perm, host_out, ws, ws_bytes, r);
    if (st != SPICE_OK || T == 0) return st;
    const spice_moe_cfg_t& c = *cfg;
    int groups = spice::kDoHit | spice::kDoShared;
    if (lore_A && lore_B) groups |= spice::kDoLore;
    spice::FfnArgs f{};
    st = prep_ffn(cfg, T, x, perm, offsets, resident_slot, w13_pool, w2_pool, w13_shared, w2_shared, lore_A, lore_B,
                  y_slots, y_shared, ws, ws_bytes, groups, "moe_layer_gpu", f);
    if (st != SPICE_OK) return st;
    spice::CombineArgs cb{};
    if (out && (st = prep_combine(cfg, T, topk_w, slot_class, inv_perm, y_slots, y_shared, resid, out, cb)) != SPICE_OK)
        return st;
    const bool gated = w_shared_gate && c.shared_inter > 0;
    hipError_t e;
    if (T <= spice::kRouteTokenMaxT && T * c.top_k <= spice::kLayerMaxSlots &&
        (c.wfmt == SPICE_WFMT_MXFP4 || !spice::expert_gemm_applies(f))) {
        if (gated) {
            float* sg = reinterpret_cast<float*>(static_cast<char*>(ws) + spice::ws_layout(c, T).sgate);
            r.w_sg = w_shared_gate;
            r.sgate = sg;
            f.sgate = sg;
        }
        e = spice::launch_layer_decode(r, f, stream);
    } else {
        e = spice::launch_route_bucket(r, stream);
        if (e == hipSuccess) e = launch_ffn(f, gated ? w_shared_gate : nullptr, ws, c, stream);
    }
    if (e == hipSuccess && out) e = spice::launch_combine(cb, stream);
    if (e != hipSuccess) return hip_fail(e, "moe_layer_gpu");
    return SPICE_OK;
    SPICE_TRY_END
}

spice_status_t spice_wait_ready(const volatile uint32_t* ready, uint32_t value, int64_t timeout_us) {
    SPICE_TRY_BEGIN
    SPICE_REQUIRE(ready, "ready");
    const auto t0 = std::chrono::steady_clock::now();
    const int64_t limit = timeout_us > 0 ? timeout_us : 10000000;
    for (uint64_t i = 0;; ++i) {
        if (__atomic_load_n(ready, __ATOMIC_ACQUIRE) == value) return SPICE_OK;
        if ((i & 255) == 255) {
            const int64_t el =
                std::chrono::duration_cast<std::chrono::microseconds>(std::chrono::steady_clock::now() - t0).count();
            if (el > limit)
                return fail(SPICE_ERR_HIP, "spice_wait_ready: the ready word did not reach " + std::to_string(value) +
                                               " within " + std::to_string(limit) + " us");
        }
        __builtin_ia32_pause();
    }
    SPICE_TRY_END
}

const char* spice_status_string(spice_status_t s) {
    switch (s) {
        case SPICE_OK: return "SPICE_OK";
        case SPICE_ERR_INVALID: return "SPICE_ERR_INVALID";
        case SPICE_ERR_UNSUPPORTED: return "SPICE_ERR_UNSUPPORTED";
        case SPICE_ERR_HIP: return "SPICE_ERR_HIP";
        case SPICE_ERR_WORKSPACE: return "SPICE_ERR_WORKSPACE";
        case SPICE_ERR_INTERNAL: return "SPICE_ERR_INTERNAL";
    }
    return "unknown spice_status_t";
}

const char* spice_last_error(void) { return g_last_error.c_str(); }

}  // extern "C"

// Shared with host_exact.cpp, which has no HIP dependency of its own.
namespace spice {
spice_status_t set_error(spice_status_t st, const char* msg) { return fail(st, msg); }
spice_status_t validate(const spice_moe_cfg_t* cfg, int32_t T) {
    spice_status_t st = check_cfg(cfg);
    if (st == SPICE_OK) st = check_tokens(*cfg, T);
    return st;
}
}  // namespace spice
