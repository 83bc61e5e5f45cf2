/* Sanitizer driver for the oracle: every entry point of oracle/spice_oracle.c on small
 * seeded inputs (fp32, bf16 and MXFP4 weights; ragged sizes; T = 0; NaN confidences;
 * every class; the LRU and speculative-prefetch steps).  Built with
 * -fsanitize=address,undefined by tests/test_sanitizers.py; any out-of-bounds access,
 * use of freed memory, leak or undefined behaviour aborts the run.  Prints "ok". */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "spice_oracle.h"

static uint64_t rng = 0x9E3779B97F4A7C15ull;
static double urand(void) { /* xorshift64*, uniform in [0, 1) */
    rng ^= rng >> 12; rng ^= rng << 25; rng ^= rng >> 27;
    return (double)((rng * 0x2545F4914F6CDD1Dull) >> 11) * (1.0 / 9007199254740992.0);
}
static uint16_t to_bf16(float f) { uint32_t u; memcpy(&u, &f, 4); return (uint16_t)((u + 0x7FFFu + ((u >> 16) & 1u)) >> 16); }

/* n elements of dtype (0 fp32, 1 bf16) drawn from U(-s, s) */
static void* rand_tensor(size_t n, int dtype, double s) {
    void* p = malloc(n * (dtype == ORC_BF16 ? 2 : 4) + 1);
    for (size_t i = 0; i < n; ++i) {
        const float v = (float)((2.0 * urand() - 1.0) * s);
        if (dtype == ORC_BF16) ((uint16_t*)p)[i] = to_bf16(v); else ((float*)p)[i] = v;
    }
    return p;
}
/* an MXFP4 blob of a [rows][K] matrix: random codes, scales near 2^-3 */
static void* rand_mx(int rows, int K) {
    const size_t ne = (size_t)rows * K / 2, ns = (size_t)rows * K / 32;
    uint8_t* b = (uint8_t*)malloc(ne + ns);
    for (size_t i = 0; i < ne; ++i) b[i] = (uint8_t)(urand() * 256.0);
    for (size_t i = 0; i < ns; ++i) b[ne + i] = (uint8_t)(122 + (int)(urand() * 4.0));
    return b;
}

static int run_layer(int d, int N, int K, int I, int Is, int r, int dtype, int wfmt, int T, int conf_mode,
                     int norm, int nres) {
    orc_cfg_t c = {d, N, K, I, Is, r, dtype, norm, conf_mode, 0.5f, wfmt};
    const int wdt = wfmt == ORC_MXFP4 ? ORC_MXFP4 : dtype;
    void* x = rand_tensor((size_t)T * d, dtype, 1.0);
    void* wg = rand_tensor((size_t)N * d, dtype, 0.2);
    float* bias = (float*)rand_tensor(N, ORC_F32, 0.1);
    double* z = (double*)malloc(sizeof(double) * ((size_t)T * N + 1));
    double* za = (double*)malloc(sizeof(double) * ((size_t)T * N + 1));
    int32_t* idx = (int32_t*)malloc(sizeof(int32_t) * ((size_t)T * K + 1));
    double* g = (double*)malloc(sizeof(double) * ((size_t)T * K + 1));
    double* probs = (double*)malloc(sizeof(double) * ((size_t)T * N + 1));
    float* cin = (float*)malloc(sizeof(float) * ((size_t)T * K + 1));
    float* conf = (float*)malloc(sizeof(float) * ((size_t)T * K + 1));
    uint8_t* cls = (uint8_t*)malloc((size_t)T * K + 1);
    int32_t* res = (int32_t*)calloc(N, sizeof(int32_t));
    int32_t* off = (int32_t*)malloc(sizeof(int32_t) * 3 * (N + 1));
    int32_t* perm = (int32_t*)malloc(sizeof(int32_t) * ((size_t)T * K + 1));
    int32_t* inv = (int32_t*)malloc(sizeof(int32_t) * ((size_t)T * K + 1));
    int32_t counts[3];
    for (int i = 0; i < T * K; ++i) cin[i] = (i % 7 == 3) ? NAN : (float)urand();
    for (int e = 0; e < nres && e < N; ++e) res[(e * 5) % N] = 1;
    orc_router_logits(&c, T, x, wg, bias, z, za);
    orc_router_logits(&c, T, x, wg, NULL, z, NULL);
    orc_gates_topk(&c, T, z, idx, g, probs);
    orc_gates_topk(&c, T, z, idx, g, NULL);
    orc_confidence(&c, T, g, cin, conf);
    orc_classify(&c, T, idx, res, conf, cls);
    orc_bucket(&c, T, idx, cls, off, perm, inv, counts);
    orc_bucket(&c, T, idx, cls, off, perm, inv, NULL);

    /* per-expert weights: every expert (routed weights in wfmt), shared block, LoRE factors */
    void** w13 = (void**)calloc(N, sizeof(void*));
    void** w2 = (void**)calloc(N, sizeof(void*));
    void** la = (void**)calloc(N, sizeof(void*));
    void** lb = (void**)calloc(N, sizeof(void*));
    for (int e = 0; e < N; ++e) {
        w13[e] = wdt == ORC_MXFP4 ? rand_mx(2 * I, d) : rand_tensor((size_t)2 * I * d, dtype, 0.1);
        w2[e] = wdt == ORC_MXFP4 ? rand_mx(d, I) : rand_tensor((size_t)d * I, dtype, 0.1);
        /* rank 0: empty (but present) factors */
        la[e] = rand_tensor((size_t)r * d, dtype, 0.1);
        lb[e] = rand_tensor((size_t)d * r, dtype, 0.1);
    }
    void* w13s = Is > 0 ? rand_tensor((size_t)2 * Is * d, dtype, 0.1) : NULL;
    void* w2s = Is > 0 ? rand_tensor((size_t)d * Is, dtype, 0.1) : NULL;
    void* wsg = rand_tensor(d, dtype, 0.1);
    double* out = (double*)malloc(sizeof(double) * d);
    double* ys = (double*)malloc(sizeof(double) * d);
    double* ysl = (double*)malloc(sizeof(double) * (size_t)K * d);
    const size_t es = dtype == ORC_BF16 ? 2 : 4;
    int bad = 0;
    for (int t = 0; t < T; ++t) {
        const char* xr = (const char*)x + (size_t)t * d * es;
        bad |= orc_token_output(&c, xr, idx + (size_t)t * K, g + (size_t)t * K, cls + (size_t)t * K,
                                (const void* const*)w13, (const void* const*)w2, w13s, w2s,
                                (const void* const*)la, (const void* const*)lb, out, ys, ysl) != 0;
        bad |= orc_token_output_sg(&c, xr, idx + (size_t)t * K, g + (size_t)t * K, cls + (size_t)t * K,
                                   (const void* const*)w13, (const void* const*)w2, w13s, w2s, wsg,
                                   (const void* const*)la, (const void* const*)lb, out, NULL, NULL) != 0;
        (void)orc_shared_gate(d, dtype, xr, wsg);
    }
    double* resid = (double*)malloc(sizeof(double) * ((size_t)T * d + 1));
    bad |= orc_exact_residual(&c, T, x, idx, g, cls, (const void* const*)w13, (const void* const*)w2, resid) != 0;
    if (wdt == ORC_MXFP4) {
        double acc = 0.0;
        for (int rr = 0; rr < 2 * I; rr += 7)
            for (int cc = 0; cc < d; cc += 5) acc += orc_mxfp4_elem(w13[0], 2 * I, d, rr, cc);
        if (!isfinite(acc)) bad = 1;
    }
    /* a missing pointer is reported, not dereferenced */
    if (T > 0) {
        void** none = (void**)calloc(N, sizeof(void*));
        const int rc = orc_token_output(&c, x, idx, g, cls, (const void* const*)none, (const void* const*)none, w13s,
                                        w2s, (const void* const*)none, (const void* const*)none, out, NULL, NULL);
        if (rc != -1) bad = 1;
        free(none);
    }
    /* the LRU steps of the stack workload */
    const int C = N / 2 > 0 ? N / 2 : 1;
    int32_t* se = (int32_t*)malloc(sizeof(int32_t) * C);
    int32_t* lu = (int32_t*)malloc(sizeof(int32_t) * C);
    int32_t adm[8], ev[8];
    for (int s = 0; s < C; ++s) { se[s] = s; lu[s] = -1; }
    for (int step = 0; step < 4; ++step) {
        (void)orc_lru_step(N, C, se, lu, step, T, K, idx, cls, 8, adm, ev);
        int32_t want[3] = {N - 1, 0, N / 2};
        (void)orc_lru_prefetch(N, C, se, lu, step, 3, want, 2, adm, ev);
    }
    free(se); free(lu);
    /* one speculative rollout depth and its prefetch queue */
    if (r > 0 && Is > 0) {
        int32_t* halted = (int32_t*)calloc(T + 1, sizeof(int32_t));
        int32_t* pidx = (int32_t*)malloc(sizeof(int32_t) * ((size_t)2 * T * K + 1));
        double* pp = (double*)malloc(sizeof(double) * ((size_t)2 * T * K + 1));
        double* cf = (double*)malloc(sizeof(double) * (T + 1));
        void* h = rand_tensor((size_t)T * d, dtype, 1.0);
        for (int depth = 1; depth <= 2; ++depth)
            bad |= orc_spec_step(&c, T, depth, 1, 0.5, depth == 2, h, wg, bias, w13s, w2s, (const void* const*)la,
                                 (const void* const*)lb, halted, pidx + (size_t)(depth - 1) * T * K,
                                 pp + (size_t)(depth - 1) * T * K, cf, h) != 0;
        int32_t ex[2 * 4], cnt[2];
        orc_prefetch_queue(N, 2, T, K, pidx, pp, 4, ex, cnt);
        free(halted); free(pidx); free(pp); free(cf); free(h);
    }
    for (int e = 0; e < N; ++e) { free(w13[e]); free(w2[e]); free(la[e]); free(lb[e]); }
    free(w13); free(w2); free(la); free(lb); free(w13s); free(w2s); free(wsg);
    free(out); free(ys); free(ysl); free(resid);
    free(x); free(wg); free(bias); free(z); free(za); free(idx); free(g); free(probs); free(cin); free(conf);
    free(cls); free(res); free(off); free(perm); free(inv);
    return bad;
}

int main(void) {
    int bad = 0;
    /*          d   N   K   I   Is  r   dtype     wfmt       T   conf_mode             norm nres */
    bad |= run_layer(20, 6, 2, 12, 8, 4, ORC_F32, 0, 5, ORC_CONF_INPUT, 0, 2);
    bad |= run_layer(24, 9, 3, 10, 0, 0, ORC_BF16, 0, 7, ORC_CONF_GATE, 1, 3);
    bad |= run_layer(36, 12, 4, 20, 28, 8, ORC_BF16, 0, 11, ORC_CONF_GATE_RENORM, 0, 0);
    bad |= run_layer(64, 8, 2, 32, 16, 8, ORC_BF16, ORC_MXFP4, 6, ORC_CONF_INPUT, 0, 4);
    bad |= run_layer(16, 5, 5, 8, 8, 4, ORC_F32, 0, 3, ORC_CONF_GATE, 0, 5); /* K = N, all resident */
    bad |= run_layer(16, 4, 1, 8, 8, 4, ORC_F32, 0, 0, ORC_CONF_INPUT, 0, 1); /* T = 0 */
    double acc = 0.0;
    for (int i = -300; i <= 300; ++i) acc += orc_round_to(ORC_BF16, ldexp(1.0 + i / 1024.0, i / 8)) +
                                           orc_round_to(ORC_F32, i * 0.1);
    if (!isfinite(acc)) bad = 1;
    if (orc_h_min(4, 1e6, 0.0, 1e-3, 2, 1e-4) != -1) bad = 1;
    if (orc_h_min(4, 1e6, 1e9, 1e-3, 2, 1e-4) < 1) bad = 1;
    printf(bad ? "FAILED\n" : "ok\n");
    return bad;
}
