// Per-layer GPU expert cache for a decode stack: the limited set of resident
// routed experts that the hit test of Sec. 4.2 consults (Sec. 1, 3: a small GPU
// holds only part of the experts), kept up to date with a least-recently-used
// policy, the cache baseline the paper evaluates against (Sec. 5).
//
// Host-side bookkeeping plus asynchronous host-to-pool copies.  The policy:
//   - an expert with a HIT slot in a layer call at step s is "used at s";
//   - the exact-miss experts of the call are admission candidates, more slots
//     first, then lower id; low-confidence misses are never admitted (they are
//     served by LoRE and need no transfer, Sec. 4.2);
//   - a candidate takes the slot whose expert was used longest ago (then the
//     lower expert id, an empty slot first), never a slot used at s;
//   - at most max_admit admissions per call (a bounded copy queue, Sec. 4.1).
// The admitted experts are still served on the CPU at step s and are resident
// for the layer's next call.
// Speculative admissions (moe_cache_prefetch, Sec. 4.1) put predicted experts of a
// future layer into that layer's least recently used slots that hold neither an
// expert used at s nor another predicted one, ahead of the layer's call.
//
// Every batch of copies for a layer re-stages the layer's whole slot table from one
// row of a small ring of pinned rows; batches of one layer are chained on the copy
// streams, so the last batch's event covers them all.
#include <hip/hip_runtime_api.h>

#include <algorithm>
#include <cstdint>
#include <cstring>
#include <exception>
#include <string>
#include <vector>

#include "spice_moe.h"
#include "spice_internal.h"

namespace spice {
spice_status_t set_error(spice_status_t st, const char* msg);
spice_status_t validate(const spice_moe_cfg_t* cfg, int32_t T);
}  // namespace spice

struct spice_cache {
    spice_moe_cfg_t cfg{};
    int32_t L = 0, N = 0, C = 0;
    size_t bytes13 = 0, bytes2 = 0;
    bool device = false;  // false: bookkeeping only (no pools, no copies)
    std::vector<const void*> w13_host, w2_host;  // [L*N]
    std::vector<void*> w13_pool, w2_pool;        // [L]
    std::vector<int32_t*> resident_dev;          // [L]
    std::vector<int32_t> slot_expert;            // [L*C], -1 = empty
    std::vector<int32_t> last_use;               // [L*C], -1 = never
    std::vector<hipEvent_t> used, ready;         // per layer: its last call's work; its last copies
    std::vector<uint8_t> pending;                // per layer: copies in flight
    std::vector<uint8_t> used_valid;             // per layer: `used` has been recorded
    static constexpr int kRing = 4;              // staging rows per layer
    int32_t* resident_stage = nullptr;           // pinned [L*kRing*N], sources of resident_slot updates
    std::vector<hipEvent_t> stage_ev;            // [L*kRing]: the row's copy has been read
    std::vector<uint8_t> stage_busy;             // [L*kRing]
    std::vector<int32_t> stage_next;             // [L]
};

namespace {

spice_status_t err(spice_status_t st, const std::string& m) { return spice::set_error(st, m.c_str()); }

spice_status_t hip_err(hipError_t e, const char* where) {
    return err(SPICE_ERR_HIP, std::string(where) + ": " + hipGetErrorString(e));
}

void release(spice_cache* c) {
    if (!c) return;
    for (hipEvent_t e : c->used)
        if (e) (void)hipEventDestroy(e);
    for (hipEvent_t e : c->ready)
        if (e) (void)hipEventDestroy(e);
    for (hipEvent_t e : c->stage_ev)
        if (e) (void)hipEventDestroy(e);
    if (c->resident_stage) (void)hipHostFree(c->resident_stage);
    delete c;
}

// Fill staging row r of layer l with the slot of every expert (-1 if absent).
int32_t* stage_resident(spice_cache* c, int32_t l, int32_t r) {
    int32_t* row = c->resident_stage + ((size_t)l * spice_cache::kRing + r) * c->N;
    std::fill(row, row + c->N, -1);
    const int32_t* se = &c->slot_expert[(size_t)l * c->C];
    for (int32_t s = 0; s < c->C; ++s)
        if (se[s] >= 0) row[se[s]] = s;
    return row;
}

struct Move {
    int32_t expert, slot, old;
};

// Queue the copies of one batch of moves of layer l (state already updated): after the
// layer's last call (its `used` event) and after the layer's previous batch, the
// weights into their slots, then the layer's slot table from a free staging row.
hipError_t queue_moves(spice_cache* c, int32_t l, const std::vector<Move>& moves, hipStream_t copy_stream) {
    const int32_t N = c->N;
    const int32_t r = c->stage_next[l];
    c->stage_next[l] = (r + 1) % spice_cache::kRing;
    const size_t ri = (size_t)l * spice_cache::kRing + r;
    hipError_t e = hipSuccess;
    if (c->stage_busy[ri]) e = hipEventSynchronize(c->stage_ev[ri]);  // the row's last copy has run
    c->stage_busy[ri] = 0;
    if (e == hipSuccess && c->used_valid[l]) e = hipStreamWaitEvent(copy_stream, c->used[l], 0);
    if (e == hipSuccess && c->pending[l]) e = hipStreamWaitEvent(copy_stream, c->ready[l], 0);
    for (size_t i = 0; i < moves.size() && e == hipSuccess; ++i) {
        const Move& m = moves[i];
        e = hipMemcpyAsync(static_cast<char*>(c->w13_pool[l]) + (size_t)m.slot * c->bytes13,
                           c->w13_host[(size_t)l * N + m.expert], c->bytes13, hipMemcpyHostToDevice, copy_stream);
        if (e == hipSuccess)
            e = hipMemcpyAsync(static_cast<char*>(c->w2_pool[l]) + (size_t)m.slot * c->bytes2,
                               c->w2_host[(size_t)l * N + m.expert], c->bytes2, hipMemcpyHostToDevice, copy_stream);
    }
    if (e == hipSuccess)
        e = hipMemcpyAsync(c->resident_dev[l], stage_resident(c, l, r), (size_t)N * 4, hipMemcpyHostToDevice,
                           copy_stream);
    if (e == hipSuccess) e = hipEventRecord(c->stage_ev[ri], copy_stream);
    if (e == hipSuccess) c->stage_busy[ri] = 1;
    if (e == hipSuccess) e = hipEventRecord(c->ready[l], copy_stream);
    if (e == hipSuccess) c->pending[l] = 1;
    return e;
}

}  // namespace

extern "C" {

spice_status_t moe_cache_create(const spice_moe_cfg_t* cfg, int32_t n_layers, const void* const* w13_host,
                                const void* const* w2_host, void* const* w13_pool, void* const* w2_pool,
                                int32_t* const* resident_slot, const int32_t* initial_experts, int32_t load,
                                spice_stream_t stream, spice_cache_t** out) {
    try {
        if (!out) return err(SPICE_ERR_INVALID, "moe_cache_create: out is NULL");
        *out = nullptr;
        spice_status_t st = spice::validate(cfg, 0);
        if (st != SPICE_OK) return st;
        if (n_layers < 1) return err(SPICE_ERR_INVALID, "moe_cache_create: n_layers must be >= 1");
        const int32_t N = cfg->n_experts, C = cfg->n_slots;
        if (C < 1 || C > N) return err(SPICE_ERR_INVALID, "moe_cache_create: n_slots must be in [1, n_experts]");
        if (!initial_experts) return err(SPICE_ERR_INVALID, "moe_cache_create: initial_experts is NULL");
        const bool device = w13_pool != nullptr;
        if (device && (!w2_pool || !resident_slot || !w13_host || !w2_host))
            return err(SPICE_ERR_INVALID, "moe_cache_create: pools given without w2_pool / resident_slot / host tables");
        if (!device && load)
            return err(SPICE_ERR_INVALID, "moe_cache_create: load needs pools");
        // initial contents: ids in range, each expert at most once per layer
        std::vector<uint8_t> seen((size_t)N);
        for (int32_t l = 0; l < n_layers; ++l) {
            std::fill(seen.begin(), seen.end(), 0);
            for (int32_t s = 0; s < C; ++s) {
                const int32_t e = initial_experts[(size_t)l * C + s];
                if (e < -1 || e >= N) return err(SPICE_ERR_INVALID, "moe_cache_create: initial expert id out of range");
                if (e >= 0 && seen[e]++) return err(SPICE_ERR_INVALID, "moe_cache_create: expert twice in one layer");
            }
        }
        spice_cache* c = new spice_cache;
        c->cfg = *cfg;
        c->L = n_layers;
        c->N = N;
        c->C = C;
        c->bytes13 = spice::expert_w13_bytes(*cfg);
        c->bytes2 = spice::expert_w2_bytes(*cfg);
        c->device = device;
        c->slot_expert.assign(initial_experts, initial_experts + (size_t)n_layers * C);
        c->last_use.assign((size_t)n_layers * C, -1);
        c->pending.assign((size_t)n_layers, 0);
        c->used_valid.assign((size_t)n_layers, 0);
        if (device) {
            const size_t ln = (size_t)n_layers * N;
            c->w13_host.assign(w13_host, w13_host + ln);
            c->w2_host.assign(w2_host, w2_host + ln);
            c->w13_pool.assign(w13_pool, w13_pool + n_layers);
            c->w2_pool.assign(w2_pool, w2_pool + n_layers);
            c->resident_dev.assign(resident_slot, resident_slot + n_layers);
            for (int32_t l = 0; l < n_layers; ++l)
                if (!c->w13_pool[l] || !c->w2_pool[l] || !c->resident_dev[l]) {
                    release(c);
                    return err(SPICE_ERR_INVALID, "moe_cache_create: a pool or resident_slot pointer is NULL");
                }
            hipError_t e = hipHostMalloc((void**)&c->resident_stage, ln * spice_cache::kRing * sizeof(int32_t),
                                         hipHostMallocDefault);
            if (e != hipSuccess) {
                c->resident_stage = nullptr;
                release(c);
                return hip_err(e, "moe_cache_create: hipHostMalloc");
            }
            c->used.assign((size_t)n_layers, nullptr);
            c->ready.assign((size_t)n_layers, nullptr);
            c->stage_ev.assign((size_t)n_layers * spice_cache::kRing, nullptr);
            c->stage_busy.assign((size_t)n_layers * spice_cache::kRing, 0);
            c->stage_next.assign((size_t)n_layers, 0);
            for (int32_t l = 0; l < n_layers && e == hipSuccess; ++l) {
                e = hipEventCreateWithFlags(&c->used[l], hipEventDisableTiming);
                if (e == hipSuccess) e = hipEventCreateWithFlags(&c->ready[l], hipEventDisableTiming);
            }
            for (size_t i = 0; i < c->stage_ev.size() && e == hipSuccess; ++i)
                e = hipEventCreateWithFlags(&c->stage_ev[i], hipEventDisableTiming);
            if (e != hipSuccess) {
                release(c);
                return hip_err(e, "moe_cache_create: hipEventCreate");
            }
            if (load) {
                for (int32_t l = 0; l < n_layers && e == hipSuccess; ++l) {
                    for (int32_t s = 0; s < C && e == hipSuccess; ++s) {
                        const int32_t x = c->slot_expert[(size_t)l * C + s];
                        if (x < 0) continue;
                        const void* h13 = c->w13_host[(size_t)l * N + x];
                        const void* h2 = c->w2_host[(size_t)l * N + x];
                        if (!h13 || !h2) {
                            (void)hipStreamSynchronize(stream);  // copies already queued read host memory
                            release(c);
                            return err(SPICE_ERR_INVALID, "moe_cache_create: host weights of an initial expert are NULL");
                        }
                        e = hipMemcpyAsync(static_cast<char*>(c->w13_pool[l]) + (size_t)s * c->bytes13, h13, c->bytes13,
                                           hipMemcpyHostToDevice, stream);
                        if (e == hipSuccess)
                            e = hipMemcpyAsync(static_cast<char*>(c->w2_pool[l]) + (size_t)s * c->bytes2, h2,
                                               c->bytes2, hipMemcpyHostToDevice, stream);
                    }
                    if (e == hipSuccess)  // row 0; the load waits for the stream before returning
                        e = hipMemcpyAsync(c->resident_dev[l], stage_resident(c, l, 0), (size_t)N * 4,
                                           hipMemcpyHostToDevice, stream);
                }
                if (e == hipSuccess) e = hipStreamSynchronize(stream);
                if (e != hipSuccess) {
                    (void)hipStreamSynchronize(stream);
                    release(c);
                    return hip_err(e, "moe_cache_create: initial load");
                }
            }
        }
        *out = c;
        return SPICE_OK;
    } catch (const std::exception& ex) {
        return err(SPICE_ERR_INTERNAL, std::string("moe_cache_create: ") + ex.what());
    } catch (...) {
        return err(SPICE_ERR_INTERNAL, "moe_cache_create: unknown exception");
    }
}

spice_status_t moe_cache_step(spice_cache_t* c, int32_t layer, int32_t step, int32_t T, const int32_t* topk_idx_host,
                              const uint8_t* slot_class_host, int32_t max_admit, spice_stream_t copy_stream,
                              spice_stream_t compute_stream, int32_t* n_admitted, int32_t* admitted,
                              int32_t* evicted) {
    try {
        if (!c) return err(SPICE_ERR_INVALID, "moe_cache_step: cache is NULL");
        if (!n_admitted) return err(SPICE_ERR_INVALID, "moe_cache_step: n_admitted is NULL");
        *n_admitted = 0;
        if (layer < 0 || layer >= c->L) return err(SPICE_ERR_INVALID, "moe_cache_step: layer out of range");
        if (step < 0) return err(SPICE_ERR_INVALID, "moe_cache_step: step must be >= 0");
        if (max_admit < 0) return err(SPICE_ERR_INVALID, "moe_cache_step: max_admit must be >= 0");
        spice_status_t st = spice::validate(&c->cfg, T);
        if (st != SPICE_OK) return st;
        if (max_admit > 0 && (!admitted || !evicted))
            return err(SPICE_ERR_INVALID, "moe_cache_step: admitted / evicted is NULL");
        if (T > 0 && (!topk_idx_host || !slot_class_host))
            return err(SPICE_ERR_INVALID, "moe_cache_step: routing arrays are NULL");
        const int32_t N = c->N, C = c->C;
        const size_t slots = (size_t)T * c->cfg.top_k;
        for (size_t i = 0; i < slots; ++i) {
            if (topk_idx_host[i] < 0 || topk_idx_host[i] >= N)
                return err(SPICE_ERR_INVALID, "moe_cache_step: expert id out of range");
            if (slot_class_host[i] > SPICE_CLASS_EXACT_GPU)
                return err(SPICE_ERR_INVALID, "moe_cache_step: slot class out of range");
        }
        int32_t* se = &c->slot_expert[(size_t)layer * C];
        int32_t* lu = &c->last_use[(size_t)layer * C];
        std::vector<int32_t> where((size_t)N, -1), wanted((size_t)N, 0);
        for (int32_t s = 0; s < C; ++s)
            if (se[s] >= 0) where[se[s]] = s;

        for (size_t i = 0; i < slots; ++i)  // an exact miss served on the GPU is still a miss
            if (slot_class_host[i] == SPICE_CLASS_EXACT || slot_class_host[i] == SPICE_CLASS_EXACT_GPU)
                ++wanted[topk_idx_host[i]];
        if (c->device)
            for (int32_t e = 0; e < N; ++e)
                if (wanted[e] > 0 && where[e] < 0 &&
                    (!c->w13_host[(size_t)layer * N + e] || !c->w2_host[(size_t)layer * N + e]))
                    return err(SPICE_ERR_INVALID, "moe_cache_step: host weights of an exact-miss expert are NULL");
        // nothing has changed so far; from here on the call succeeds or reports a HIP error
        for (size_t i = 0; i < slots; ++i)
            if (slot_class_host[i] == SPICE_CLASS_HIT && where[topk_idx_host[i]] >= 0)
                lu[where[topk_idx_host[i]]] = step;

        std::vector<Move> moves;
        while ((int32_t)moves.size() < max_admit) {
            // candidate: an EXACT expert not resident right now, most slots first, then lower id
            // (residency is re-read each time: an expert evicted here may become a candidate)
            int32_t e = -1;
            for (int32_t x = 0; x < N; ++x)
                if (wanted[x] > 0 && where[x] < 0 && (e < 0 || wanted[x] > wanted[e])) e = x;
            if (e < 0) break;
            int32_t v = -1;  // oldest use, then lower expert id (empty = -1 first); not used at `step`
            for (int32_t s = 0; s < C; ++s) {
                if (lu[s] == step) continue;
                if (v < 0 || lu[s] < lu[v] || (lu[s] == lu[v] && se[s] < se[v])) v = s;
            }
            if (v < 0) break;
            if (c->device && (!c->w13_host[(size_t)layer * N + e] || !c->w2_host[(size_t)layer * N + e]))
                break;  // only an expert evicted in this call can get here; its weights are not given
            moves.push_back({e, v, se[v]});
            if (se[v] >= 0) where[se[v]] = -1;
            se[v] = e;
            lu[v] = step;
            where[e] = v;
            wanted[e] = 0;
        }
        for (size_t i = 0; i < moves.size(); ++i) {
            admitted[i] = moves[i].expert;
            evicted[i] = moves[i].old;
        }
        *n_admitted = (int32_t)moves.size();
        if (!c->device) return SPICE_OK;

        // The call's work on the compute stream is the layer's last use of its pools
        // (marked on every call).  The evicted slots are not read by this call's kernels
        // (their experts were not used at `step`), but resident_slot is: the copies go
        // after that work.
        hipError_t e = hipEventRecord(c->used[layer], compute_stream);
        if (e == hipSuccess) c->used_valid[layer] = 1;
        if (e == hipSuccess && !moves.empty()) e = queue_moves(c, layer, moves, copy_stream);
        return e == hipSuccess ? SPICE_OK : hip_err(e, "moe_cache_step");
    } catch (const std::exception& ex) {
        return err(SPICE_ERR_INTERNAL, std::string("moe_cache_step: ") + ex.what());
    } catch (...) {
        return err(SPICE_ERR_INTERNAL, "moe_cache_step: unknown exception");
    }
}

spice_status_t moe_cache_prefetch(spice_cache_t* c, int32_t layer, int32_t step, int32_t n, const int32_t* experts,
                                  int32_t max_prefetch, spice_stream_t copy_stream, spice_stream_t compute_stream,
                                  int32_t* n_admitted, int32_t* admitted, int32_t* evicted) {
    try {
        if (!c) return err(SPICE_ERR_INVALID, "moe_cache_prefetch: cache is NULL");
        if (!n_admitted) return err(SPICE_ERR_INVALID, "moe_cache_prefetch: n_admitted is NULL");
        *n_admitted = 0;
        if (layer < 0 || layer >= c->L) return err(SPICE_ERR_INVALID, "moe_cache_prefetch: layer out of range");
        if (step < 0) return err(SPICE_ERR_INVALID, "moe_cache_prefetch: step must be >= 0");
        if (n < 0 || max_prefetch < 0) return err(SPICE_ERR_INVALID, "moe_cache_prefetch: n and max_prefetch must be >= 0");
        if (n > 0 && !experts) return err(SPICE_ERR_INVALID, "moe_cache_prefetch: experts is NULL");
        if (max_prefetch > 0 && (!admitted || !evicted))
            return err(SPICE_ERR_INVALID, "moe_cache_prefetch: admitted / evicted is NULL");
        const int32_t N = c->N, C = c->C;
        std::vector<uint8_t> listed((size_t)N, 0);
        for (int32_t i = 0; i < n; ++i) {
            if (experts[i] < 0 || experts[i] >= N) return err(SPICE_ERR_INVALID, "moe_cache_prefetch: expert id out of range");
            listed[experts[i]] = 1;
        }
        int32_t* se = &c->slot_expert[(size_t)layer * C];
        int32_t* lu = &c->last_use[(size_t)layer * C];
        std::vector<Move> moves;
        for (int32_t i = 0; i < n && (int32_t)moves.size() < max_prefetch; ++i) {
            const int32_t e = experts[i];
            if (std::find(se, se + C, e) != se + C) continue;  // already resident
            if (c->device && (!c->w13_host[(size_t)layer * N + e] || !c->w2_host[(size_t)layer * N + e]))
                continue;  // no host weights to copy from: not a prefetch candidate
            int32_t v = -1;  // oldest use, then lower expert id (empty first); not used at `step`, not listed
            for (int32_t s = 0; s < C; ++s) {
                if (lu[s] == step || (se[s] >= 0 && listed[se[s]])) continue;
                if (v < 0 || lu[s] < lu[v] || (lu[s] == lu[v] && se[s] < se[v])) v = s;
            }
            if (v < 0) break;
            moves.push_back({e, v, se[v]});
            se[v] = e;
            lu[v] = step;
        }
        for (size_t i = 0; i < moves.size(); ++i) {
            admitted[i] = moves[i].expert;
            evicted[i] = moves[i].old;
        }
        *n_admitted = (int32_t)moves.size();
        if (!c->device || moves.empty()) return SPICE_OK;
        // the copies wait for the layer's last call (moe_cache_step's mark), not for
        // whatever else the compute stream holds: a prefetch overlaps the current layer
        (void)compute_stream;
        const hipError_t e = queue_moves(c, layer, moves, copy_stream);
        return e == hipSuccess ? SPICE_OK : hip_err(e, "moe_cache_prefetch");
    } catch (const std::exception& ex) {
        return err(SPICE_ERR_INTERNAL, std::string("moe_cache_prefetch: ") + ex.what());
    } catch (...) {
        return err(SPICE_ERR_INTERNAL, "moe_cache_prefetch: unknown exception");
    }
}

spice_status_t moe_cache_wait(spice_cache_t* c, int32_t layer, spice_stream_t stream) {
    if (!c) return err(SPICE_ERR_INVALID, "moe_cache_wait: cache is NULL");
    if (layer < 0 || layer >= c->L) return err(SPICE_ERR_INVALID, "moe_cache_wait: layer out of range");
    if (!c->device || !c->pending[layer]) return SPICE_OK;
    const hipError_t e = hipStreamWaitEvent(stream, c->ready[layer], 0);
    return e == hipSuccess ? SPICE_OK : hip_err(e, "moe_cache_wait");
}

spice_status_t moe_cache_state(const spice_cache_t* c, int32_t layer, int32_t* slot_expert, int32_t* last_use) {
    if (!c) return err(SPICE_ERR_INVALID, "moe_cache_state: cache is NULL");
    if (layer < 0 || layer >= c->L) return err(SPICE_ERR_INVALID, "moe_cache_state: layer out of range");
    const size_t o = (size_t)layer * c->C;
    if (slot_expert) std::memcpy(slot_expert, &c->slot_expert[o], sizeof(int32_t) * c->C);
    if (last_use) std::memcpy(last_use, &c->last_use[o], sizeof(int32_t) * c->C);
    return SPICE_OK;
}

void moe_cache_destroy(spice_cache_t* c) {
    if (!c) return;
    if (c->device)
        for (size_t l = 0; l < c->pending.size(); ++l)
            if (c->pending[l]) (void)hipEventSynchronize(c->ready[l]);
    release(c);
}

}  // extern "C"
