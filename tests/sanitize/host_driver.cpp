// Sanitizer driver for the host C++ of libspice_moe (built with -fsanitize=address,undefined
// by tests/test_sanitizers.py, the GPU launchers replaced by device_stubs.cpp, no GPU):
//   - the C ABI's argument validation (workspace sizes, NULL and out-of-range arguments, host
//     pointers where device memory is required) on every entry point;
//   - the exact CPU residual (moe_exact_residual_host): fp32, bf16 and MXFP4 weights, ragged
//     sizes, several thread counts (results identical across them, fp32/bf16 against a plain
//     double reference), EXACT_GPU slots skipped, error paths;
//   - the exact-miss split planner, the prefetch depth and queue;
//   - the expert cache in bookkeeping-only mode (no pools): LRU steps, speculative
//     admissions, state reads, rejected updates leaving the state unchanged;
//   - the bounded wait on the host ready word (time-out path).
// Prints "ok"; any failed check prints its line and the run exits non-zero.
#include <cmath>
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <vector>

#include "spice_moe.h"

static int g_fail = 0;
#define CHECK(c)                                                              \
    do {                                                                      \
        if (!(c)) {                                                           \
            std::fprintf(stderr, "check failed at line %d: %s\n", __LINE__, #c); \
            g_fail = 1;                                                       \
        }                                                                     \
    } while (0)

static uint64_t g_rng = 0x243F6A8885A308D3ull;
static double urand() {
    g_rng ^= g_rng >> 12; g_rng ^= g_rng << 25; g_rng ^= g_rng >> 27;
    return (double)((g_rng * 0x2545F4914F6CDD1Dull) >> 11) * (1.0 / 9007199254740992.0);
}
static uint16_t bf16_of(float f) {
    uint32_t u; std::memcpy(&u, &f, 4);
    return (uint16_t)((u + 0x7FFFu + ((u >> 16) & 1u)) >> 16);
}
static double widen(const void* p, int dtype, size_t i) {
    if (dtype == SPICE_BF16) {
        uint32_t u = (uint32_t)static_cast<const uint16_t*>(p)[i] << 16; float f; std::memcpy(&f, &u, 4); return f;
    }
    return static_cast<const float*>(p)[i];
}
static std::vector<uint8_t> tensor(size_t n, int dtype, double s) {
    std::vector<uint8_t> b(n * (dtype == SPICE_BF16 ? 2 : 4) + 1);
    for (size_t i = 0; i < n; ++i) {
        const float v = (float)((2.0 * urand() - 1.0) * s);
        if (dtype == SPICE_BF16) reinterpret_cast<uint16_t*>(b.data())[i] = bf16_of(v);
        else reinterpret_cast<float*>(b.data())[i] = v;
    }
    return b;
}
static std::vector<uint8_t> mx_blob(int rows, int K) {
    std::vector<uint8_t> b((size_t)rows * K / 2 + (size_t)rows * K / 32);
    const size_t ne = (size_t)rows * K / 2;
    for (size_t i = 0; i < b.size(); ++i) b[i] = i < ne ? (uint8_t)(urand() * 256) : (uint8_t)(120 + (int)(urand() * 4));
    return b;
}

static spice_moe_cfg_t cfg_of(int d, int N, int K, int I, int Is, int r, int C, int dtype, int wfmt = 0) {
    spice_moe_cfg_t c{};
    c.d = d; c.n_experts = N; c.top_k = K; c.inter = I; c.shared_inter = Is; c.lore_rank = r; c.n_slots = C;
    c.dtype = dtype; c.norm_topk = 0; c.conf_mode = SPICE_CONF_INPUT; c.tau = 0.5f; c.wfmt = wfmt;
    return c;
}

static void validation() {
    for (int s = -2; s <= 8; ++s) CHECK(spice_status_string((spice_status_t)s) != nullptr);
    CHECK(spice_last_error() != nullptr);
    const spice_moe_cfg_t ok = cfg_of(64, 8, 2, 32, 48, 8, 4, SPICE_BF16);
    CHECK(spice_workspace_bytes(&ok, 1) > SPICE_WS_CONTROL_BYTES);
    CHECK(spice_workspace_bytes(&ok, 0) >= SPICE_WS_CONTROL_BYTES);
    CHECK(spice_workspace_bytes(&ok, -1) == 0);
    CHECK(spice_workspace_bytes(&ok, SPICE_MAX_TOKENS + 1) == 0);
    CHECK(spice_workspace_bytes(nullptr, 4) == 0);
    // one bad field at a time
    const int bad_fields[][12] = {
        {0, 8, 2, 32, 48, 8, 4, SPICE_BF16, 0, 0, 0, 0},  {64, 0, 2, 32, 48, 8, 4, SPICE_BF16, 0, 0, 0, 0},
        {64, 300, 2, 32, 48, 8, 4, SPICE_BF16, 0, 0, 0, 0}, {64, 8, 9, 32, 48, 8, 4, SPICE_BF16, 0, 0, 0, 0},
        {64, 8, 0, 32, 48, 8, 4, SPICE_BF16, 0, 0, 0, 0},  {66, 8, 2, 32, 48, 8, 4, SPICE_BF16, 0, 0, 0, 0},
        {64, 8, 2, 30, 48, 8, 4, SPICE_BF16, 0, 0, 0, 0},  {64, 8, 2, 32, 48, 300, 4, SPICE_BF16, 0, 0, 0, 0},
        {64, 8, 2, 32, 48, -8, 4, SPICE_BF16, 0, 0, 0, 0}, {64, 8, 2, 32, 48, 8, 4, 7, 0, 0, 0, 0},
        {64, 8, 2, 32, 48, 8, 4, SPICE_F32, 0, 9, 0, 0},    {64, 8, 2, 32, 48, 8, 4, SPICE_F32, 2, 0, 0, 0},
        {100000, 8, 2, 32, 48, 8, 4, SPICE_BF16, 0, 0, 0, 0}, {64, 8, 2, 32, 48, 8, -1, SPICE_BF16, 0, 0, 0, 0}};
    for (const auto& f : bad_fields) {
        spice_moe_cfg_t c = cfg_of(f[0], f[1], f[2], f[3], f[4], f[5], f[6], f[7], f[8]);
        c.conf_mode = f[9];
        CHECK(spice_workspace_bytes(&c, 4) == 0);
    }
    // every device entry point rejects NULL or host memory before any launch
    std::vector<uint8_t> hostbuf(1 << 16);
    void* h = hostbuf.data();
    int32_t* ip = reinterpret_cast<int32_t*>(h);
    float* fp = reinterpret_cast<float*>(h);
    uint8_t* bp = reinterpret_cast<uint8_t*>(h);
    double* dp = reinterpret_cast<double*>(h);
    const size_t wsb = hostbuf.size();
    //                  cfg     T   x        w_gate bias     res conf     logits topk_idx w  cls offs perm inv host_out ws
    CHECK(moe_route_bucket(nullptr, 1, h, h, nullptr, ip, nullptr, dp, ip, fp, bp, ip, ip, ip, nullptr, h, wsb,
                           nullptr) != SPICE_OK);
    CHECK(moe_route_bucket(&ok, -3, h, h, nullptr, ip, nullptr, dp, ip, fp, bp, ip, ip, ip, nullptr, h, wsb,
                           nullptr) != SPICE_OK);
    CHECK(moe_route_bucket(&ok, 2, nullptr, h, nullptr, ip, nullptr, dp, ip, fp, bp, ip, ip, ip, nullptr, h, wsb,
                           nullptr) != SPICE_OK);
    CHECK(moe_route_bucket(&ok, 2, h, h, nullptr, ip, nullptr, dp, ip, fp, bp, ip, ip, ip, nullptr, h, 16,
                           nullptr) != SPICE_OK);
    CHECK(moe_route_bucket(&ok, 2, h, h, nullptr, ip, nullptr, dp, ip, fp, bp, ip, ip, ip, nullptr, h, wsb,
                           nullptr) != SPICE_OK);  // host memory where device memory is required
    CHECK(moe_expert_ffn_grouped(&ok, 2, nullptr, ip, ip, ip, h, h, h, h, nullptr, nullptr, fp, fp, h, wsb,
                                 nullptr) != SPICE_OK);
    CHECK(moe_expert_ffn_grouped(&ok, 2, h, ip, ip, ip, h, h, h, h, nullptr, nullptr, fp, fp, h, wsb, nullptr) !=
          SPICE_OK);
    CHECK(moe_combine(&ok, 2, nullptr, bp, ip, fp, fp, nullptr, h, nullptr) != SPICE_OK);
    CHECK(moe_combine(&ok, 2, fp, bp, ip, fp + 4096, fp + 8192, nullptr, h, nullptr) != SPICE_OK);
    CHECK(lore_surrogate_apply(&ok, 2, nullptr, ip, ip, h, h, fp, h, wsb, nullptr) != SPICE_OK);
    CHECK(moe_layer_gpu(&ok, 2, h, h, nullptr, ip, nullptr, h, h, h, h, nullptr, nullptr, nullptr, nullptr, ip, fp, bp,
                        ip, ip, ip, fp, fp, nullptr, nullptr, nullptr, nullptr, 0, nullptr) != SPICE_OK);
    CHECK(moe_layer_gpu(nullptr, 2, h, h, nullptr, ip, nullptr, h, h, h, h, nullptr, nullptr, nullptr, nullptr, ip,
                        fp, bp, ip, ip, ip, fp, fp, nullptr, nullptr, nullptr, h, wsb, nullptr) != SPICE_OK);
    CHECK(spice_workspace_init(nullptr, 0, nullptr) != SPICE_OK);
    CHECK(spice_workspace_init(h, 64, nullptr) != SPICE_OK);
    uint32_t flags = 0;
    CHECK(spice_workspace_flags(h, 64, &flags, 0, nullptr) != SPICE_OK);
    CHECK(spice_lore_fit_workspace_bytes(&ok, 0, 4) == 0);
    CHECK(spice_lore_fit_workspace_bytes(&ok, 16, 0) == 0);
    CHECK(spice_lore_fit_workspace_bytes(&ok, 16, 4) > 0);
    CHECK(moe_lore_fit(&ok, 16, 4, nullptr, h, h, h, h, fp, fp, nullptr, nullptr, h, wsb, nullptr) != SPICE_OK);
    CHECK(moe_lore_fit(&ok, 16, 4, h, h, h, h, h, fp, fp, nullptr, nullptr, h, wsb, nullptr) != SPICE_OK);
    // the host ready word: a value that never comes times out, one that is there returns at once
    volatile uint32_t ready = 5;
    CHECK(spice_wait_ready(&ready, 6, 2000) != SPICE_OK);
    CHECK(spice_wait_ready(&ready, 5, 2000) == SPICE_OK);
    CHECK(spice_wait_ready(nullptr, 5, 2000) != SPICE_OK);
}

// resid[t] = sum over EXACT slots of g * W2 (silu(W1 x) * (W3 x)), in double
static void exact_reference(const spice_moe_cfg_t& c, int T, const void* x, const int32_t* idx, const float* g,
                            const uint8_t* cls, const std::vector<std::vector<uint8_t>>& w13,
                            const std::vector<std::vector<uint8_t>>& w2, std::vector<double>& out) {
    const int d = c.d, I = c.inter, K = c.top_k;
    out.assign((size_t)T * d, 0.0);
    std::vector<double> h(I);
    for (int t = 0; t < T; ++t)
        for (int k = 0; k < K; ++k) {
            if (cls[t * K + k] != SPICE_CLASS_EXACT) continue;
            const int e = idx[t * K + k];
            for (int i = 0; i < I; ++i) {
                double a = 0, b = 0;
                for (int j = 0; j < d; ++j) {
                    const double xv = widen(x, c.dtype, (size_t)t * d + j);
                    a += widen(w13[e].data(), c.dtype, (size_t)i * d + j) * xv;
                    b += widen(w13[e].data(), c.dtype, (size_t)(I + i) * d + j) * xv;
                }
                h[i] = a / (1.0 + std::exp(-a)) * b;
            }
            for (int j = 0; j < d; ++j) {
                double y = 0;
                for (int i = 0; i < I; ++i) y += widen(w2[e].data(), c.dtype, (size_t)j * I + i) * h[i];
                out[(size_t)t * d + j] += g[t * K + k] * y;
            }
        }
}

static void exact_residual(int d, int N, int K, int I, int T, int dtype, int wfmt) {
    const spice_moe_cfg_t c = cfg_of(d, N, K, I, 16, 8, 2, dtype, wfmt);
    std::vector<uint8_t> x = tensor((size_t)T * d, dtype, 1.0);
    std::vector<int32_t> idx((size_t)T * K);
    std::vector<float> g((size_t)T * K);
    std::vector<uint8_t> cls((size_t)T * K);
    for (int t = 0; t < T; ++t)
        for (int k = 0; k < K; ++k) {
            idx[t * K + k] = (t * 3 + k * 5) % N;
            g[t * K + k] = (float)urand();
            const double u = urand();
            cls[t * K + k] = u < 0.6 ? SPICE_CLASS_EXACT : (u < 0.7 ? SPICE_CLASS_EXACT_GPU : (u < 0.85 ? 0 : 1));
        }
    std::vector<std::vector<uint8_t>> w13(N), w2(N);
    std::vector<const void*> t13(N, nullptr), t2(N, nullptr);
    std::vector<bool> needed(N, false);
    for (int s = 0; s < T * K; ++s)
        if (cls[s] == SPICE_CLASS_EXACT) needed[idx[s]] = true;
    for (int e = 0; e < N; ++e) {
        if (!needed[e]) continue;  // no EXACT slot: the table entry may stay NULL
        w13[e] = wfmt == SPICE_WFMT_MXFP4 ? mx_blob(2 * I, d) : tensor((size_t)2 * I * d, dtype, 0.1);
        w2[e] = wfmt == SPICE_WFMT_MXFP4 ? mx_blob(d, I) : tensor((size_t)d * I, dtype, 0.1);
        t13[e] = w13[e].data();
        t2[e] = w2[e].data();
    }
    std::vector<float> r1((size_t)T * d + 1), r3((size_t)T * d + 1), r0((size_t)T * d + 1);
    CHECK(moe_exact_residual_host(&c, T, x.data(), idx.data(), g.data(), cls.data(), t13.data(), t2.data(), r1.data(),
                                  1) == SPICE_OK);
    CHECK(moe_exact_residual_host(&c, T, x.data(), idx.data(), g.data(), cls.data(), t13.data(), t2.data(), r3.data(),
                                  3) == SPICE_OK);
    CHECK(moe_exact_residual_host(&c, T, x.data(), idx.data(), g.data(), cls.data(), t13.data(), t2.data(), r0.data(),
                                  0) == SPICE_OK);
    CHECK(std::memcmp(r1.data(), r3.data(), sizeof(float) * T * d) == 0);
    CHECK(std::memcmp(r1.data(), r0.data(), sizeof(float) * T * d) == 0);
    if (wfmt == SPICE_WFMT_DTYPE) {
        std::vector<double> ref;
        exact_reference(c, T, x.data(), idx.data(), g.data(), cls.data(), w13, w2, ref);
        double worst = 0;
        for (int t = 0; t < T; ++t) {
            double mx = 1e-30, err = 0;
            for (int j = 0; j < d; ++j) {
                mx = std::fmax(mx, std::fabs(ref[(size_t)t * d + j]));
                err = std::fmax(err, std::fabs(ref[(size_t)t * d + j] - r1[(size_t)t * d + j]));
            }
            worst = std::fmax(worst, err / mx);
        }
        CHECK(worst < 1e-4);
    }
    // error paths: a missing weight of an EXACT expert, NULL arguments, a bad class, a bad id
    for (int e = 0; e < N; ++e)
        if (needed[e]) {
            std::vector<const void*> miss = t13;
            miss[e] = nullptr;
            CHECK(moe_exact_residual_host(&c, T, x.data(), idx.data(), g.data(), cls.data(), miss.data(), t2.data(),
                                          r1.data(), 2) != SPICE_OK);
            break;
        }
    if (T > 0)  // (T = 0 is a no-op whatever the pointers)
        CHECK(moe_exact_residual_host(&c, T, nullptr, idx.data(), g.data(), cls.data(), t13.data(), t2.data(),
                                      r1.data(), 1) != SPICE_OK);
    CHECK(moe_exact_residual_host(&c, -1, x.data(), idx.data(), g.data(), cls.data(), t13.data(), t2.data(), r1.data(),
                                  1) != SPICE_OK);
    if (T > 0) {
        std::vector<int32_t> bad_idx = idx;
        bad_idx[0] = N;
        std::vector<uint8_t> bad_cls = cls;
        bad_cls[0] = SPICE_CLASS_EXACT;
        CHECK(moe_exact_residual_host(&c, T, x.data(), bad_idx.data(), g.data(), bad_cls.data(), t13.data(), t2.data(),
                                      r1.data(), 1) != SPICE_OK);
        bad_cls[0] = 9;
        CHECK(moe_exact_residual_host(&c, T, x.data(), idx.data(), g.data(), bad_cls.data(), t13.data(), t2.data(),
                                      r1.data(), 1) != SPICE_OK);
    }
}

static void split_and_prefetch() {
    const spice_moe_cfg_t c = cfg_of(64, 16, 4, 32, 48, 8, 6, SPICE_BF16);
    const int T = 9, K = 4;
    std::vector<int32_t> idx(T * K);
    std::vector<uint8_t> cls(T * K);
    for (int s = 0; s < T * K; ++s) { idx[s] = (s * 7) % 16; cls[s] = (uint8_t)(s % 3); }
    const spice_split_cost_t fetch_all{1e8, 1e12, 1e13, 0.0, 0.0}, fetch_none{1e13, 1e15, 1e6, 1.0, 0.05};
    for (int mf = 0; mf <= 16; mf += 4) {
        std::vector<int32_t> fe(mf + 1, -7);
        int32_t nf = -1;
        std::vector<uint8_t> cl = cls;
        CHECK(moe_split_plan(&c, T, idx.data(), cl.data(), &fetch_all, mf, fe.data(), &nf) == SPICE_OK);
        CHECK(nf >= 0 && nf <= mf);
        cl = cls;
        CHECK(moe_split_plan(&c, T, idx.data(), cl.data(), &fetch_none, mf, fe.data(), &nf) == SPICE_OK);
        CHECK(nf == 0);
    }
    int32_t nf = 0, fe[4];
    CHECK(moe_split_plan(&c, T, idx.data(), cls.data(), nullptr, 4, fe, &nf) != SPICE_OK);
    CHECK(moe_split_plan(&c, T, idx.data(), cls.data(), &fetch_all, -1, fe, &nf) != SPICE_OK);
    CHECK(moe_prefetch_h_min(4, 1e6, 1e9, 1e-3, 2, 1e-4) >= 1);
    CHECK(moe_prefetch_h_min(4, 1e6, 0.0, 1e-3, 2, 1e-4) == -1);
    CHECK(moe_prefetch_h_min(-1, 1e6, 1e9, 1e-3, 2, 1e-4) == -1);
    const int D = 3, M = 5;
    std::vector<int32_t> pidx(D * T * K);
    std::vector<float> pp(D * T * K);
    for (int i = 0; i < D * T * K; ++i) {
        pidx[i] = (i % 5 == 0) ? -1 : (i * 11) % 16;
        pp[i] = (float)urand();
    }
    std::vector<int32_t> ex(D * M), cnt(D);
    CHECK(moe_prefetch_queue(&c, T, D, pidx.data(), pp.data(), M, ex.data(), cnt.data()) == SPICE_OK);
    for (int d = 0; d < D; ++d) CHECK(cnt[d] >= 0 && cnt[d] <= M);
    pidx[3] = 99;
    CHECK(moe_prefetch_queue(&c, T, D, pidx.data(), pp.data(), M, ex.data(), cnt.data()) != SPICE_OK);
}

static void cache_bookkeeping() {
    const int L = 3, C = 4, N = 10, K = 3, T = 5;
    const spice_moe_cfg_t c = cfg_of(64, N, K, 32, 48, 8, C, SPICE_BF16);
    std::vector<int32_t> init = {0, 1, 2, -1, 5, 6, -1, -1, 9, 8, 7, 6};
    spice_cache_t* h = nullptr;
    CHECK(moe_cache_create(&c, L, nullptr, nullptr, nullptr, nullptr, nullptr, init.data(), 0, nullptr, &h) ==
          SPICE_OK);
    CHECK(h != nullptr);
    std::vector<int32_t> idx(T * K);
    std::vector<uint8_t> cls(T * K);
    int32_t adm[8], ev[8], na = 0;
    for (int step = 0; step < 12; ++step)
        for (int l = 0; l < L; ++l) {
            for (int s = 0; s < T * K; ++s) {
                idx[s] = (int32_t)(urand() * N);
                cls[s] = (uint8_t)(urand() * 3);
            }
            CHECK(moe_cache_step(h, l, step, T, idx.data(), cls.data(), 2, nullptr, nullptr, &na, adm, ev) ==
                  SPICE_OK);
            CHECK(na >= 0 && na <= 2);
            int32_t want[3] = {(step * 3) % N, (step * 7 + 1) % N, 4};
            CHECK(moe_cache_prefetch(h, l, step, 3, want, 2, nullptr, nullptr, &na, adm, ev) == SPICE_OK);
            std::vector<int32_t> se(C), lu(C);
            CHECK(moe_cache_state(h, l, se.data(), lu.data()) == SPICE_OK);
            for (int s = 0; s < C; ++s) CHECK(se[s] >= -1 && se[s] < N && lu[s] <= step);
        }
    // a rejected update leaves the state unchanged
    std::vector<int32_t> before(C), after(C);
    CHECK(moe_cache_state(h, 1, before.data(), nullptr) == SPICE_OK);
    idx[2] = N + 3;
    CHECK(moe_cache_step(h, 1, 99, T, idx.data(), cls.data(), 2, nullptr, nullptr, &na, adm, ev) != SPICE_OK);
    CHECK(moe_cache_state(h, 1, after.data(), nullptr) == SPICE_OK);
    CHECK(before == after);
    CHECK(moe_cache_step(h, L, 0, T, idx.data(), cls.data(), 2, nullptr, nullptr, &na, adm, ev) != SPICE_OK);
    CHECK(moe_cache_state(h, -1, after.data(), nullptr) != SPICE_OK);
    moe_cache_destroy(h);
    moe_cache_destroy(nullptr);
    // invalid initial states
    std::vector<int32_t> dup = {0, 0, 1, 2, 3, 4, 5, 6, 7, 8, 9, -1};
    CHECK(moe_cache_create(&c, L, nullptr, nullptr, nullptr, nullptr, nullptr, dup.data(), 0, nullptr, &h) !=
          SPICE_OK);
    CHECK(moe_cache_create(&c, L, nullptr, nullptr, nullptr, nullptr, nullptr, init.data(), 1, nullptr, &h) !=
          SPICE_OK);
    CHECK(moe_cache_create(&c, 0, nullptr, nullptr, nullptr, nullptr, nullptr, init.data(), 0, nullptr, &h) !=
          SPICE_OK);
}

int main() {
    validation();
    //             d    N   K  I   T   dtype       wfmt
    exact_residual(40, 6, 2, 24, 7, SPICE_F32, SPICE_WFMT_DTYPE);
    exact_residual(48, 9, 3, 40, 5, SPICE_BF16, SPICE_WFMT_DTYPE);
    exact_residual(24, 4, 4, 8, 3, SPICE_BF16, SPICE_WFMT_DTYPE);  // K = N
    exact_residual(64, 8, 2, 32, 6, SPICE_BF16, SPICE_WFMT_MXFP4);
    exact_residual(40, 6, 2, 24, 0, SPICE_F32, SPICE_WFMT_DTYPE);  // T = 0
    split_and_prefetch();
    cache_bookkeeping();
    std::printf(g_fail ? "FAILED\n" : "ok\n");
    return g_fail;
}
