// Host side of speculative prefetching (Sec. 4.1): the minimum lookahead of Eq. 4 and
// the per-depth issue lists of the prefetch intents of Eq. 3.
#include <algorithm>
#include <cmath>
#include <cstdint>
#include <exception>
#include <string>
#include <vector>

#include "spice_moe.h"

namespace spice {
spice_status_t set_error(spice_status_t st, const char* msg);
spice_status_t validate(const spice_moe_cfg_t* cfg, int32_t T);
}  // namespace spice

extern "C" {

int32_t moe_prefetch_h_min(double P, double expert_bytes, double pcie_bytes_per_s, double t_attn_s, int32_t K,
                           double t_expert_s) {
    if (!(P >= 0) || !(expert_bytes >= 0) || !(t_attn_s >= 0) || !(t_expert_s >= 0) || K < 0) return -1;
    const double window = t_attn_s + (double)K * t_expert_s;
    if (!(window > 0) || !(pcie_bytes_per_s > 0)) return -1;
    const double h = std::ceil(P * expert_bytes / (pcie_bytes_per_s * window));
    return h > 2147483647.0 ? -1 : (int32_t)h;
}

spice_status_t moe_prefetch_queue(const spice_moe_cfg_t* cfg, int32_t T, int32_t n_depth,
                                  const int32_t* pred_idx_host, const float* pred_prob_host, int32_t max_per_depth,
                                  int32_t* experts, int32_t* counts) {
    try {
        spice_status_t st = spice::validate(cfg, T);
        if (st != SPICE_OK) return st;
        if (n_depth < 0 || max_per_depth < 0)
            return spice::set_error(SPICE_ERR_INVALID, "moe_prefetch_queue: n_depth and max_per_depth must be >= 0");
        if (n_depth == 0) return SPICE_OK;
        if (!counts) return spice::set_error(SPICE_ERR_INVALID, "moe_prefetch_queue: counts is NULL");
        if (max_per_depth > 0 && !experts)
            return spice::set_error(SPICE_ERR_INVALID, "moe_prefetch_queue: experts is NULL");
        if (T > 0 && (!pred_idx_host || !pred_prob_host))
            return spice::set_error(SPICE_ERR_INVALID, "moe_prefetch_queue: prediction arrays are NULL");
        const int32_t N = cfg->n_experts, K = cfg->top_k;
        const size_t per = (size_t)T * K;
        for (size_t i = 0; i < per * n_depth; ++i)
            if (pred_idx_host[i] < -1 || pred_idx_host[i] >= N)
                return spice::set_error(SPICE_ERR_INVALID, "moe_prefetch_queue: expert id out of range");
        std::vector<double> mass((size_t)N);
        std::vector<uint8_t> seen((size_t)N);
        std::vector<int32_t> order;
        for (int32_t dp = 0; dp < n_depth; ++dp) {
            std::fill(mass.begin(), mass.end(), 0.0);
            std::fill(seen.begin(), seen.end(), 0);
            const int32_t* pi = pred_idx_host + (size_t)dp * per;
            const float* pp = pred_prob_host + (size_t)dp * per;
            for (size_t i = 0; i < per; ++i)
                if (pi[i] >= 0) {
                    seen[pi[i]] = 1;
                    mass[pi[i]] += (double)pp[i];
                }
            order.clear();
            for (int32_t e = 0; e < N; ++e)
                if (seen[e]) order.push_back(e);
            std::stable_sort(order.begin(), order.end(), [&](int32_t a, int32_t b) { return mass[a] > mass[b]; });
            const int32_t n = std::min<int32_t>((int32_t)order.size(), max_per_depth);
            std::copy(order.begin(), order.begin() + n, experts + (size_t)dp * max_per_depth);
            counts[dp] = n;
        }
        return SPICE_OK;
    } catch (const std::exception& ex) {
        return spice::set_error(SPICE_ERR_INTERNAL, (std::string("moe_prefetch_queue: ") + ex.what()).c_str());
    } catch (...) {
        return spice::set_error(SPICE_ERR_INTERNAL, "moe_prefetch_queue: unknown exception");
    }
}

}  // extern "C"
