// Exact-miss split M = M_fetch + M_cpu (Eq. 12; Sec. 4.3): choose which exact-miss
// experts to fetch over PCIe and run on the GPU while the CPU serves the rest, and
// copy the chosen experts into a fetch pool.
//
// The paper describes the scheduler only by what it compares (all-CPU service
// against candidate split plans, a per-layer cost table, a safety margin); the cost
// model here is this library's: both sides stream the expert's weights, the CPU
// also pays for its arithmetic, and the two sides run in parallel.
#include <hip/hip_runtime_api.h>

#include <algorithm>
#include <cstdint>
#include <exception>
#include <string>
#include <vector>

#include "spice_moe.h"

namespace spice {
spice_status_t set_error(spice_status_t st, const char* msg);
spice_status_t validate(const spice_moe_cfg_t* cfg, int32_t T);
}  // namespace spice

namespace {

spice_status_t err(spice_status_t st, const std::string& m) { return spice::set_error(st, m.c_str()); }

}  // namespace

extern "C" {

spice_status_t moe_split_plan(const spice_moe_cfg_t* cfg, int32_t T, const int32_t* topk_idx_host,
                              uint8_t* slot_class_host, const spice_split_cost_t* cost, int32_t max_fetch,
                              int32_t* fetch_experts, int32_t* n_fetch) {
    try {
        if (!n_fetch) return err(SPICE_ERR_INVALID, "moe_split_plan: n_fetch is NULL");
        *n_fetch = 0;
        spice_status_t st = spice::validate(cfg, T);
        if (st == SPICE_OK && cfg->wfmt != SPICE_WFMT_DTYPE)
            return err(SPICE_ERR_UNSUPPORTED, "moe_split_plan: the fetched-expert split needs SPICE_WFMT_DTYPE weights");
        if (st != SPICE_OK) return st;
        if (!cost) return err(SPICE_ERR_INVALID, "moe_split_plan: cost is NULL");
        if (max_fetch < 0) return err(SPICE_ERR_INVALID, "moe_split_plan: max_fetch must be >= 0");
        if (max_fetch > 0 && !fetch_experts) return err(SPICE_ERR_INVALID, "moe_split_plan: fetch_experts is NULL");
        if (!(cost->cpu_bytes_per_s > 0) || !(cost->cpu_flops_per_s > 0) || !(cost->pcie_bytes_per_s > 0) ||
            !(cost->gpu_fixed_s >= 0) || !(cost->margin >= 0 && cost->margin < 1))
            return err(SPICE_ERR_INVALID, "moe_split_plan: cost rates must be > 0, gpu_fixed_s >= 0, margin in [0, 1)");
        if (T == 0 || max_fetch == 0) return SPICE_OK;
        if (!topk_idx_host || !slot_class_host) return err(SPICE_ERR_INVALID, "moe_split_plan: routing arrays are NULL");
        const int N = cfg->n_experts;
        const size_t S = (size_t)T * cfg->top_k;
        std::vector<int> tokens((size_t)N, 0);
        for (size_t s = 0; s < S; ++s) {
            if (slot_class_host[s] > SPICE_CLASS_EXACT_GPU)
                return err(SPICE_ERR_INVALID, "moe_split_plan: slot class out of range");
            if (slot_class_host[s] != SPICE_CLASS_EXACT) continue;
            const int e = topk_idx_host[s];
            if (e < 0 || e >= N) return err(SPICE_ERR_INVALID, "moe_split_plan: expert id out of range");
            ++tokens[e];
        }
        const double es = cfg->dtype == SPICE_BF16 ? 2.0 : 4.0;
        const double bytes = 3.0 * cfg->inter * (double)cfg->d * es;
        const double flops_per_token = 6.0 * cfg->inter * (double)cfg->d;
        auto cpu_cost = [&](int e) {
            return bytes / cost->cpu_bytes_per_s + tokens[e] * flops_per_token / cost->cpu_flops_per_s;
        };
        std::vector<int> cand;
        double all_cpu = 0.0;
        for (int e = 0; e < N; ++e)
            if (tokens[e] > 0) {
                cand.push_back(e);
                all_cpu += cpu_cost(e);
            }
        // most expensive on the CPU first (more tokens), ties to the lower id
        std::stable_sort(cand.begin(), cand.end(), [&](int a, int b) { return tokens[a] > tokens[b]; });
        const int jmax = std::min((int)cand.size(), max_fetch);
        double cpu_left = all_cpu, fetch = cost->gpu_fixed_s, best = all_cpu;
        int best_j = 0;
        for (int j = 1; j <= jmax; ++j) {
            cpu_left -= cpu_cost(cand[j - 1]);
            fetch += bytes / cost->pcie_bytes_per_s;
            const double plan = std::max(cpu_left, fetch);
            if (plan < best) {
                best = plan;
                best_j = j;
            }
        }
        if (best_j == 0 || best >= (1.0 - cost->margin) * all_cpu) return SPICE_OK;  // all-CPU plan
        std::vector<uint8_t> chosen((size_t)N, 0);
        for (int j = 0; j < best_j; ++j) {
            fetch_experts[j] = cand[j];
            chosen[cand[j]] = 1;
        }
        for (size_t s = 0; s < S; ++s)
            if (slot_class_host[s] == SPICE_CLASS_EXACT && chosen[topk_idx_host[s]])
                slot_class_host[s] = SPICE_CLASS_EXACT_GPU;
        *n_fetch = best_j;
        return SPICE_OK;
    } catch (const std::exception& ex) {
        return err(SPICE_ERR_INTERNAL, std::string("moe_split_plan: ") + ex.what());
    } catch (...) {
        return err(SPICE_ERR_INTERNAL, "moe_split_plan: unknown exception");
    }
}

spice_status_t moe_fetch_experts(const spice_moe_cfg_t* cfg, int32_t n_fetch, const int32_t* experts,
                                 const void* const* w13_host, const void* const* w2_host, void* w13_fetch,
                                 void* w2_fetch, int32_t n_slots, int32_t* fetch_expert,
                                 int32_t* fetch_expert_stage, spice_stream_t copy_stream) {
    try {
        spice_status_t st = spice::validate(cfg, 0);
        if (st == SPICE_OK && cfg->wfmt != SPICE_WFMT_DTYPE)
            return err(SPICE_ERR_UNSUPPORTED, "moe_fetch_experts: the fetched-expert split needs SPICE_WFMT_DTYPE weights");
        if (st != SPICE_OK) return st;
        const int N = cfg->n_experts;
        if (n_slots < 1 || n_slots > N) return err(SPICE_ERR_INVALID, "moe_fetch_experts: n_slots must be in [1, N]");
        if (n_fetch < 0 || n_fetch > n_slots)
            return err(SPICE_ERR_INVALID, "moe_fetch_experts: n_fetch must be in [0, n_slots]");
        if (!fetch_expert || !fetch_expert_stage || !w13_fetch || !w2_fetch)
            return err(SPICE_ERR_INVALID, "moe_fetch_experts: a pool or table pointer is NULL");
        if (n_fetch > 0 && (!experts || !w13_host || !w2_host))
            return err(SPICE_ERR_INVALID, "moe_fetch_experts: experts or host tables are NULL");
        std::vector<uint8_t> seen((size_t)N, 0);
        for (int i = 0; i < n_fetch; ++i) {
            const int e = experts[i];
            if (e < 0 || e >= N) return err(SPICE_ERR_INVALID, "moe_fetch_experts: expert id out of range");
            if (seen[e]++) return err(SPICE_ERR_INVALID, "moe_fetch_experts: expert listed twice");
            if (!w13_host[e] || !w2_host[e]) return err(SPICE_ERR_INVALID, "moe_fetch_experts: host weights are NULL");
        }
        const size_t es = cfg->dtype == SPICE_BF16 ? 2 : 4;
        const size_t b13 = (size_t)2 * cfg->inter * cfg->d * es, b2 = (size_t)cfg->d * cfg->inter * es;
        hipError_t e = hipSuccess;
        for (int i = 0; i < n_fetch && e == hipSuccess; ++i) {
            e = hipMemcpyAsync(static_cast<char*>(w13_fetch) + (size_t)i * b13, w13_host[experts[i]], b13,
                               hipMemcpyHostToDevice, copy_stream);
            if (e == hipSuccess)
                e = hipMemcpyAsync(static_cast<char*>(w2_fetch) + (size_t)i * b2, w2_host[experts[i]], b2,
                                   hipMemcpyHostToDevice, copy_stream);
        }
        if (e == hipSuccess) {
            for (int i = 0; i < n_slots; ++i) fetch_expert_stage[i] = i < n_fetch ? experts[i] : -1;
            e = hipMemcpyAsync(fetch_expert, fetch_expert_stage, sizeof(int32_t) * n_slots, hipMemcpyHostToDevice,
                               copy_stream);
        }
        if (e != hipSuccess) return err(SPICE_ERR_HIP, std::string("moe_fetch_experts: ") + hipGetErrorString(e));
        return SPICE_OK;
    } catch (const std::exception& ex) {
        return err(SPICE_ERR_INTERNAL, std::string("moe_fetch_experts: ") + ex.what());
    } catch (...) {
        return err(SPICE_ERR_INTERNAL, "moe_fetch_experts: unknown exception");
    }
}

}  // extern "C"
