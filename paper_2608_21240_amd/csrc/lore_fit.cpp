// LoRE calibration fit (Sec. 4.2, Eq. 8-10) for one expert from n <= d calibration tokens.
//
// Eq. 10 asks for rank-r factors minimising sum_t || y_t - B A x_t ||^2 with
// y_t = E_e(x_t) - S(x_t).  With the tokens as columns, X (d x n) has full column rank
// when n <= d, so every target Y (d x n) is reachable by some map and the best rank-r
// map is the truncated SVD of Y carried back through X's pseudo-inverse:
//   Y = U S V^T,  B = U_r = Y V_r S_r^-1,  A = S_r V_r^T (X^T X)^-1 X^T,
//   loss = sum_{i > r} s_i^2.
// Everything n-dimensional is done on the host in fp64 from the two n x n Gram matrices
// X^T X and Y^T Y (computed on the GPU in fp64): Y^T Y = V S^2 V^T by Jacobi rotations
// (round-robin order), (X^T X) Z = V_r S_r by Cholesky.  The GPU computes E_e(x) and S(x) with the
// grouped-FFN kernels (a one-expert bucket of all n tokens), the residual, the Gram
// matrices and the final d x r products.
#include <hip/hip_runtime_api.h>

#include <algorithm>
#include <cmath>
#include <cstdint>
#include <exception>
#include <string>
#include <vector>

#include "spice_internal.h"
#include "spice_moe.h"

namespace spice {
spice_status_t set_error(spice_status_t st, const char* msg);
spice_status_t validate(const spice_moe_cfg_t* cfg, int32_t T);
}  // namespace spice

namespace {

constexpr int32_t kMaxFitTokens = 1024;

spice_status_t err(spice_status_t st, const std::string& m) { return spice::set_error(st, m.c_str()); }

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

// The one-expert cfg of the FFN launches inside the fit.
spice_moe_cfg_t one_expert(const spice_moe_cfg_t& c) {
    spice_moe_cfg_t o = c;
    o.n_experts = 1;
    o.top_k = 1;
    o.n_slots = 1;
    o.lore_rank = 0;
    return o;
}

struct FitLayout {
    size_t ffn_ws, perm, offsets, resident, y, ys, gx, gy, coef_a, coef_b, total;
};

FitLayout fit_layout(const spice_moe_cfg_t& c, int32_t n, int32_t r) {
    FitLayout L{};
    const spice_moe_cfg_t o = one_expert(c);
    size_t off = 0;
    L.ffn_ws = off;   off += align256(spice::ws_layout(o, n).total);
    L.perm = off;     off += align256((size_t)n * 4);
    L.offsets = off;  off += align256(6 * 4);
    L.resident = off; off += align256(4);
    L.y = off;        off += align256((size_t)n * c.d * 4);
    L.ys = off;       off += align256((size_t)n * c.d * 4);
    L.gx = off;       off += align256((size_t)n * n * 8);
    L.gy = off;       off += align256((size_t)n * n * 8);
    L.coef_a = off;   off += align256((size_t)n * r * 8);
    L.coef_b = off;   off += align256((size_t)n * r * 8);
    L.total = off;
    return L;
}

// Eigen-decomposition of the symmetric n x n matrix a (row-major, destroyed) by Jacobi
// rotations in round-robin order: each round rotates n/2 disjoint index pairs at once
// (every index meets every other once per sweep), applying all row rotations and then all
// column rotations row by row, so that every access runs along a row.
// a = V diag(w) V^T with the eigenvectors as the rows of vt (vt[k*n + i] = component i of
// vector k).
void jacobi_eigen(int n, std::vector<double>& a, std::vector<double>& w, std::vector<double>& vt) {
    vt.assign((size_t)n * n, 0.0);
    for (int i = 0; i < n; ++i) vt[(size_t)i * n + i] = 1.0;
    const int m = n + (n & 1);  // players of the tournament; index n is a bye when n is odd
    std::vector<int> player(m);
    for (int i = 0; i < m; ++i) player[i] = i;
    struct Rot {
        int p, q;
        double c, s;
    };
    std::vector<Rot> rots;
    rots.reserve(m / 2);
    auto rotate_rows = [&](double* base) {
        for (const Rot& r : rots) {
            double* rp = base + (size_t)r.p * n;
            double* rq = base + (size_t)r.q * n;
            for (int k = 0; k < n; ++k) {
                const double ap = rp[k], aq = rq[k];
                rp[k] = r.c * ap - r.s * aq;
                rq[k] = r.s * ap + r.c * aq;
            }
        }
    };
    for (int sweep = 0; sweep < 60; ++sweep) {
        double off = 0.0, diag = 0.0;
        for (int i = 0; i < n; ++i) {
            diag += a[(size_t)i * n + i] * a[(size_t)i * n + i];
            for (int j = i + 1; j < n; ++j) off += a[(size_t)i * n + j] * a[(size_t)i * n + j];
        }
        if (off == 0.0 || off <= 1e-30 * diag) break;
        for (int round = 0; round < m - 1; ++round) {
            rots.clear();
            for (int i = 0; i < m / 2; ++i) {
                int p = player[i], q = player[m - 1 - i];
                if (p > q) std::swap(p, q);
                if (q >= n) continue;
                const double apq = a[(size_t)p * n + q];
                if (apq == 0.0) continue;
                // the angle that zeroes a[p][q]: tan(2 theta) = 2 a_pq / (a_qq - a_pp)
                const double theta = (a[(size_t)q * n + q] - a[(size_t)p * n + p]) / (2.0 * apq);
                const double t = (theta >= 0 ? 1.0 : -1.0) / (std::fabs(theta) + std::sqrt(theta * theta + 1.0));
                const double c = 1.0 / std::sqrt(t * t + 1.0);
                rots.push_back({p, q, c, t * c});
            }
            rotate_rows(a.data());
            for (int k = 0; k < n; ++k) {  // the same rotations on the columns, row by row
                double* row = a.data() + (size_t)k * n;
                for (const Rot& r : rots) {
                    const double ap = row[r.p], aq = row[r.q];
                    row[r.p] = r.c * ap - r.s * aq;
                    row[r.q] = r.s * ap + r.c * aq;
                }
            }
            for (const Rot& r : rots) a[(size_t)r.p * n + r.q] = a[(size_t)r.q * n + r.p] = 0.0;
            rotate_rows(vt.data());
            // next round: the first player stays, the others move one place round the circle
            const int last = player[m - 1];
            for (int i = m - 1; i > 1; --i) player[i] = player[i - 1];
            player[1] = last;
        }
    }
    w.resize(n);
    for (int i = 0; i < n; ++i) w[i] = a[(size_t)i * n + i];
}

// Cholesky factor of the SPD n x n matrix g (row-major, lower factor in place); false if
// it is not positive definite.
bool cholesky(int n, std::vector<double>& g) {
    for (int j = 0; j < n; ++j) {
        double d = g[(size_t)j * n + j];
        for (int k = 0; k < j; ++k) d -= g[(size_t)j * n + k] * g[(size_t)j * n + k];
        if (!(d > 0.0)) return false;
        const double l = std::sqrt(d);
        g[(size_t)j * n + j] = l;
        for (int i = j + 1; i < n; ++i) {
            double s = g[(size_t)i * n + j];
            for (int k = 0; k < j; ++k) s -= g[(size_t)i * n + k] * g[(size_t)j * n + k];
            g[(size_t)i * n + j] = s / l;
        }
    }
    return true;
}

// Solve (L L^T) z = b in place for one right-hand side.
void cholesky_solve(int n, const std::vector<double>& l, double* b) {
    for (int i = 0; i < n; ++i) {
        double s = b[i];
        for (int k = 0; k < i; ++k) s -= l[(size_t)i * n + k] * b[k];
        b[i] = s / l[(size_t)i * n + i];
    }
    for (int i = n - 1; i >= 0; --i) {
        double s = b[i];
        for (int k = i + 1; k < n; ++k) s -= l[(size_t)k * n + i] * b[k];
        b[i] = s / l[(size_t)i * n + i];
    }
}

}  // namespace

extern "C" {

size_t spice_lore_fit_workspace_bytes(const spice_moe_cfg_t* cfg, int32_t n, int32_t r) {
    if (spice::validate(cfg, n) != SPICE_OK || n < 1 || n > kMaxFitTokens || r < 1) return 0;
    return fit_layout(*cfg, n, r).total;
}

spice_status_t moe_lore_fit(const spice_moe_cfg_t* cfg, int32_t n, int32_t r, const void* x, const void* w13,
                            const void* w2, const void* w13_shared, const void* w2_shared, float* A_out, float* B_out,
                            float* y_out, double* loss_out, void* ws, size_t ws_bytes, spice_stream_t stream) {
    try {
        spice_status_t st = spice::validate(cfg, n);
        if (st == SPICE_OK && cfg->wfmt != SPICE_WFMT_DTYPE)
            return spice::set_error(SPICE_ERR_UNSUPPORTED, "moe_lore_fit: needs SPICE_WFMT_DTYPE expert weights");
        if (st != SPICE_OK) return st;
        const spice_moe_cfg_t& c = *cfg;
        const int32_t d = c.d;
        if (n < 1) return err(SPICE_ERR_INVALID, "moe_lore_fit: n must be >= 1");
        if (n > d || n > kMaxFitTokens)
            return err(SPICE_ERR_UNSUPPORTED, "moe_lore_fit: n must be <= d and <= 1024 calibration tokens");
        if (r < 1 || r > d) return err(SPICE_ERR_INVALID, "moe_lore_fit: r must be in [1, d]");
        if (!x || !w13 || !w2 || !A_out || !B_out || !ws)
            return err(SPICE_ERR_INVALID, "moe_lore_fit: x, expert weights, outputs and workspace are required");
        if (c.shared_inter > 0 && (!w13_shared || !w2_shared))
            return err(SPICE_ERR_INVALID, "moe_lore_fit: shared-block weights are NULL");
        const FitLayout L = fit_layout(c, n, r);
        if (ws_bytes < L.total)
            return err(SPICE_ERR_WORKSPACE, "moe_lore_fit: workspace has " + std::to_string(ws_bytes) +
                                                " bytes, needs " + std::to_string(L.total));
        char* w = static_cast<char*>(ws);
        hipStream_t s = stream;
        const spice_moe_cfg_t o = one_expert(c);
        const spice::WsLayout FL = spice::ws_layout(o, n);
        char* fw = w + L.ffn_ws;
        float* y = reinterpret_cast<float*>(w + L.y);
        float* ys = reinterpret_cast<float*>(w + L.ys);
        double* gx = reinterpret_cast<double*>(w + L.gx);
        double* gy = reinterpret_cast<double*>(w + L.gy);

        // E_e(x) and S(x): the grouped FFN on a one-expert bucket of all n tokens
        hipError_t e = spice::launch_fill_u32(reinterpret_cast<uint32_t*>(fw), SPICE_WS_CONTROL_BYTES / 4, 0u, s);
        if (e == hipSuccess)  // S = 0 without a shared block
            e = spice::launch_fill_u32(reinterpret_cast<uint32_t*>(ys), (size_t)n * d, 0u, s);
        if (e == hipSuccess)
            e = spice::launch_fit_setup(n, reinterpret_cast<int32_t*>(w + L.perm),
                                        reinterpret_cast<int32_t*>(w + L.offsets),
                                        reinterpret_cast<int32_t*>(w + L.resident), s);
        if (e == hipSuccess) {
            spice::FfnArgs a{};
            a.T = n; a.d = d; a.N = 1; a.K = 1; a.C = 1; a.I = c.inter; a.Is = c.shared_inter; a.r = 0;
            a.dtype = c.dtype; a.groups = spice::kDoHit | spice::kDoShared;
            a.ldh = c.inter + spice::kHPad; a.ldhs = c.shared_inter + spice::kHPad;
            a.x = x; a.perm = reinterpret_cast<int32_t*>(w + L.perm);
            a.offsets = reinterpret_cast<int32_t*>(w + L.offsets);
            a.resident_slot = reinterpret_cast<int32_t*>(w + L.resident);
            a.w13_pool = w13; a.w2_pool = w2; a.w13s = w13_shared; a.w2s = w2_shared;
            a.y_slots = y; a.y_shared = ys;
            a.h = fw + FL.h; a.hs = fw + FL.hs; a.u = reinterpret_cast<float*>(fw + FL.u);
            a.ctrl = reinterpret_cast<uint32_t*>(fw);
            e = spice::launch_expert_ffn(a, s);
        }
        if (e == hipSuccess && c.shared_inter > 0) e = spice::launch_fit_residual((size_t)n * d, y, ys, s);
        if (e == hipSuccess) e = spice::launch_fit_gram(n, d, c.dtype, x, gx, s);
        if (e == hipSuccess) e = spice::launch_fit_gram(n, d, SPICE_F32, y, gy, s);
        std::vector<double> hx((size_t)n * n), hy((size_t)n * n);
        uint32_t flags = 0;
        if (e == hipSuccess) e = hipMemcpyAsync(hx.data(), gx, hx.size() * 8, hipMemcpyDeviceToHost, s);
        if (e == hipSuccess) e = hipMemcpyAsync(hy.data(), gy, hy.size() * 8, hipMemcpyDeviceToHost, s);
        if (e == hipSuccess) e = hipMemcpyAsync(&flags, fw, 4, hipMemcpyDeviceToHost, s);
        if (e == hipSuccess) e = hipStreamSynchronize(s);
        if (e != hipSuccess) return err(SPICE_ERR_HIP, std::string("moe_lore_fit: ") + hipGetErrorString(e));
        if (flags) return err(SPICE_ERR_INTERNAL, "moe_lore_fit: FFN device flags raised");

        // Y^T Y = V S^2 V^T; order by eigenvalue, largest first
        std::vector<double> ev, vec;
        jacobi_eigen(n, hy, ev, vec);
        std::vector<int> ord(n);
        for (int i = 0; i < n; ++i) ord[i] = i;
        std::stable_sort(ord.begin(), ord.end(), [&](int a_, int b_) { return ev[a_] > ev[b_]; });
        double loss = 0.0;
        for (int i = r; i < n; ++i) loss += std::max(ev[ord[i]], 0.0);
        if (loss_out) *loss_out = loss;
        if (!cholesky(n, hx))
            return err(SPICE_ERR_INVALID, "moe_lore_fit: the calibration tokens are linearly dependent");
        // coef_a = (X^T X)^-1 V_r S_r (n x r), coef_b = V_r S_r^-1 (n x r); directions beyond
        // n or with s = 0 give zero rows of A and columns of B
        const double s_max = std::sqrt(std::max(ev[ord[0]], 0.0));
        std::vector<double> ca((size_t)n * r, 0.0), cb((size_t)n * r, 0.0), col(n);
        for (int j = 0; j < std::min(r, n); ++j) {
            const double sj = std::sqrt(std::max(ev[ord[j]], 0.0));
            if (!(sj > 1e-12 * s_max)) continue;
            for (int i = 0; i < n; ++i) col[i] = vec[(size_t)n * ord[j] + i] * sj;
            for (int i = 0; i < n; ++i) cb[(size_t)i * r + j] = vec[(size_t)n * ord[j] + i] / sj;
            cholesky_solve(n, hx, col.data());
            for (int i = 0; i < n; ++i) ca[(size_t)i * r + j] = col[i];
        }
        double* da = reinterpret_cast<double*>(w + L.coef_a);
        double* db = reinterpret_cast<double*>(w + L.coef_b);
        e = hipMemcpyAsync(da, ca.data(), ca.size() * 8, hipMemcpyHostToDevice, s);
        if (e == hipSuccess) e = hipMemcpyAsync(db, cb.data(), cb.size() * 8, hipMemcpyHostToDevice, s);
        if (e == hipSuccess) e = spice::launch_fit_project(n, d, r, c.dtype, x, da, A_out, false, s);
        if (e == hipSuccess) e = spice::launch_fit_project(n, d, r, SPICE_F32, y, db, B_out, true, s);
        if (e == hipSuccess && y_out) e = hipMemcpyAsync(y_out, y, (size_t)n * d * 4, hipMemcpyDeviceToDevice, s);
        if (e == hipSuccess) e = hipStreamSynchronize(s);  // the host coefficient buffers are read by the copies
        if (e != hipSuccess) return err(SPICE_ERR_HIP, std::string("moe_lore_fit: ") + hipGetErrorString(e));
        return SPICE_OK;
    } catch (const std::exception& ex) {
        return err(SPICE_ERR_INTERNAL, std::string("moe_lore_fit: ") + ex.what());
    } catch (...) {
        return err(SPICE_ERR_INTERNAL, "moe_lore_fit: unknown exception");
    }
}

}  // extern "C"
