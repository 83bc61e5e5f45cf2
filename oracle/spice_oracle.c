/*
 * spice_oracle.c -- reference oracle (test infrastructure only; see spice_oracle.h).
 *
 * Plain loops in double precision, one step of the method per function, in the
 * order the paper states them:
 *   routing, Eq. 1 and Sec. 2.1            -> orc_router_logits, orc_gates_topk
 *   hit / low-confidence / exact rule, Sec. 4.2 and 4.3 -> orc_confidence, orc_classify
 *   grouping of slots by (class, expert)   -> orc_bucket
 *   expert FFN, Eq. 6; LoRE, Eq. 9         -> orc_swiglu, orc_lore_delta
 *   substitution, Eq. 7 / Eq. 11, and the gate-weighted aggregation of Sec. 2.1
 *                                          -> orc_token_output
 *   exact CPU path for M_cpu, Sec. 4.3     -> orc_exact_residual
 *   expert cache bookkeeping (LRU policy)  -> orc_lru_step
 *   speculative prefetching, Sec. 4.1 and Alg. 1:
 *     draft rollout depth (Eq. 2, 5; Alg. 1 steps 1-4) -> orc_spec_step
 *     minimum lookahead, Eq. 4             -> orc_h_min
 *     prefetch intents, Eq. 3              -> orc_prefetch_queue
 *     speculative cache admissions         -> orc_lru_prefetch
 */
#include "spice_oracle.h"

#include <math.h>
#include <stdlib.h>
#include <string.h>

/* Widen one stored element to double (exact for fp32 and bf16). */
static double elem(const void* p, int32_t dtype, size_t i) {
    if (dtype == ORC_BF16) {
        uint32_t bits = (uint32_t)((const uint16_t*)p)[i] << 16;
        float f;
        memcpy(&f, &bits, sizeof f);
        return (double)f;
    }
    return (double)((const float*)p)[i];
}

/* FP4 E2M1 code (OCP MX v1.0): sign bit 3, exponent bits 2..1 (bias 1), mantissa bit 0;
 * exponent 0 is subnormal (0 or 0.5).  Magnitudes 0, 0.5, 1, 1.5, 2, 3, 4, 6. */
static double e2m1(unsigned code) {
    const unsigned e = (code >> 1) & 3u, m = code & 1u;
    const double mag = (e == 0) ? 0.5 * m : ldexp(1.0 + 0.5 * m, (int)e - 1);
    return (code & 8u) ? -mag : mag;
}

double orc_mxfp4_elem(const void* blob, int32_t rows, int32_t K, int32_t r, int32_t c) {
    const uint8_t* b = (const uint8_t*)blob;
    const uint8_t byte = b[(size_t)r * (K / 2) + c / 2];
    const unsigned code = (c & 1) ? (byte >> 4) : (byte & 15u);
    const uint8_t s = b[(size_t)rows * (K / 2) + (size_t)r * (K / 32) + c / 32];
    if (s == 255) return NAN; /* E8M0 NaN */
    return ldexp(e2m1(code), (int)s - 127);
}

/* Weight (r, c) of a [rows][K] matrix in storage dtype (fp32, bf16 or an MXFP4 blob). */
static double welem(const void* p, int32_t dtype, int32_t rows, int32_t K, int32_t r, int32_t c) {
    if (dtype == ORC_MXFP4) return orc_mxfp4_elem(p, rows, K, r, c);
    return elem(p, dtype, (size_t)r * K + c);
}

/* Eq. 1: the router maps the hidden state to one logit per routed expert. */
void orc_router_logits(const orc_cfg_t* c, int32_t T, const void* x, const void* wg,
                       const float* bias, double* z, double* zabs) {
    const int32_t d = c->d, N = c->n_experts;
    for (int32_t t = 0; t < T; ++t) {
        for (int32_t e = 0; e < N; ++e) {
            double acc = 0.0, mag = 0.0;
            for (int32_t i = 0; i < d; ++i) {
                double p = elem(x, c->dtype, (size_t)t * d + i) * elem(wg, c->dtype, (size_t)e * d + i);
                acc += p;
                mag += fabs(p);
            }
            if (bias) acc += (double)bias[e];
            z[(size_t)t * N + e] = acc;
            if (zabs) zabs[(size_t)t * N + e] = mag;
        }
    }
}

/* Eq. 1 TopK with softmax gate scores (Sec. 2.1 weighting, Sec. 4.2 gate scores). */
void orc_gates_topk(const orc_cfg_t* c, int32_t T, const double* z, int32_t* idx, double* g,
                    double* probs) {
    const int32_t N = c->n_experts, K = c->top_k;
    double* p = (double*)malloc(sizeof(double) * (size_t)N);
    int32_t* taken = (int32_t*)malloc(sizeof(int32_t) * (size_t)N);
    for (int32_t t = 0; t < T; ++t) {
        const double* zt = z + (size_t)t * N;
        /* softmax over all N experts */
        double m = zt[0];
        for (int32_t e = 1; e < N; ++e)
            if (zt[e] > m) m = zt[e];
        double s = 0.0;
        for (int32_t e = 0; e < N; ++e) {
            p[e] = exp(zt[e] - m);
            s += p[e];
        }
        for (int32_t e = 0; e < N; ++e) p[e] /= s;
        if (probs)
            for (int32_t e = 0; e < N; ++e) probs[(size_t)t * N + e] = p[e];
        /* K rounds of "largest remaining logit"; a strict '>' while scanning ids
         * upward keeps the lower id on a tie. */
        for (int32_t e = 0; e < N; ++e) taken[e] = 0;
        double gsum = 0.0;
        for (int32_t k = 0; k < K; ++k) {
            int32_t best = -1;
            for (int32_t e = 0; e < N; ++e) {
                if (taken[e]) continue;
                if (best < 0 || zt[e] > zt[best]) best = e;
            }
            taken[best] = 1;
            idx[(size_t)t * K + k] = best;
            g[(size_t)t * K + k] = p[best];
            gsum += p[best];
        }
        if (c->norm_topk)
            for (int32_t k = 0; k < K; ++k) g[(size_t)t * K + k] /= gsum;
    }
    free(p);
    free(taken);
}

/* Sec. 4.2: a missing expert is judged by its routing confidence / estimated
 * contribution.  The confidence is the caller's, or the gate score. */
void orc_confidence(const orc_cfg_t* c, int32_t T, const double* g, const float* conf_in,
                    float* conf) {
    const int32_t K = c->top_k;
    for (int32_t t = 0; t < T; ++t) {
        double gsum = 0.0;
        for (int32_t k = 0; k < K; ++k) gsum += g[(size_t)t * K + k];
        for (int32_t k = 0; k < K; ++k) {
            size_t s = (size_t)t * K + k;
            if (c->conf_mode == ORC_CONF_INPUT)
                conf[s] = conf_in[s];
            else if (c->conf_mode == ORC_CONF_GATE)
                conf[s] = (float)g[s];
            else
                conf[s] = (float)(g[s] / gsum);
        }
    }
}

/* Sec. 4.2: resident (or prefetched) -> exact on the GPU; missing with low
 * confidence -> shared + LoRE; otherwise an exact miss (the set M of Sec. 4.3). */
void orc_classify(const orc_cfg_t* c, int32_t T, const int32_t* idx, const int32_t* resident,
                  const float* conf, uint8_t* cls) {
    const int32_t K = c->top_k;
    for (int32_t s = 0; s < T * K; ++s) {
        if (resident[idx[s]])
            cls[s] = ORC_HIT;
        else if (conf[s] < c->tau) /* false for NaN */
            cls[s] = ORC_LORE;
        else
            cls[s] = ORC_EXACT;
    }
}

void orc_bucket(const orc_cfg_t* c, int32_t T, const int32_t* idx, const uint8_t* cls,
                int32_t* offsets, int32_t* perm, int32_t* inv_perm, int32_t* counts) {
    const int32_t N = c->n_experts, S = T * c->top_k;
    int32_t* cnt = (int32_t*)calloc((size_t)3 * N, sizeof(int32_t));
    int32_t* fill = (int32_t*)calloc((size_t)3 * N, sizeof(int32_t));
    for (int32_t s = 0; s < S; ++s) cnt[cls[s] * N + idx[s]]++;
    int32_t run = 0;
    for (int32_t cl = 0; cl < 3; ++cl) {
        int32_t start = run;
        for (int32_t e = 0; e < N; ++e) {
            offsets[cl * (N + 1) + e] = run;
            run += cnt[cl * N + e];
        }
        offsets[cl * (N + 1) + N] = run;
        if (counts) counts[cl] = run - start;
    }
    for (int32_t s = 0; s < S; ++s) {
        int32_t key = cls[s] * N + idx[s];
        int32_t pos = offsets[cls[s] * (N + 1) + idx[s]] + fill[key]++;
        perm[pos] = s;
        inv_perm[s] = pos;
    }
    free(cnt);
    free(fill);
}

static double silu(double u) { return u / (1.0 + exp(-u)); }

/* Eq. 6: an expert is a SwiGLU FFN, y = W2 (silu(W1 x) * (W3 x)). */
void orc_swiglu(int32_t d, int32_t inter, int32_t dtype, const void* w13, const void* w2,
                const double* x, double* y) {
    double* h = (double*)malloc(sizeof(double) * (size_t)inter);
    for (int32_t i = 0; i < inter; ++i) {
        double a = 0.0, b = 0.0;
        for (int32_t j = 0; j < d; ++j) {
            a += welem(w13, dtype, 2 * inter, d, i, j) * x[j];
            b += welem(w13, dtype, 2 * inter, d, inter + i, j) * x[j];
        }
        h[i] = silu(a) * b;
    }
    for (int32_t j = 0; j < d; ++j) {
        double acc = 0.0;
        for (int32_t i = 0; i < inter; ++i) acc += welem(w2, dtype, d, inter, j, i) * h[i];
        y[j] = acc;
    }
    free(h);
}

/* Eq. 9: the LoRE correction is B_e (A_e h), with A_e [r][d] and B_e [d][r]. */
void orc_lore_delta(int32_t d, int32_t r, int32_t dtype, const void* A, const void* B,
                    const double* x, double* delta) {
    double* u = (double*)malloc(sizeof(double) * (size_t)(r > 0 ? r : 1));
    for (int32_t q = 0; q < r; ++q) {
        double acc = 0.0;
        for (int32_t j = 0; j < d; ++j) acc += elem(A, dtype, (size_t)q * d + j) * x[j];
        u[q] = acc;
    }
    for (int32_t j = 0; j < d; ++j) {
        double acc = 0.0;
        for (int32_t q = 0; q < r; ++q) acc += elem(B, dtype, (size_t)j * r + q) * u[q];
        delta[j] = acc;
    }
    free(u);
}

/* Gated shared block: S(x) = sigmoid(w_sg . x) SwiGLU_s(x), the shared expert with its
 * output gate (the Qwen2-style shared expert; the paper calls S the native shared expert). */
double orc_shared_gate(int32_t d, int32_t dtype, const void* x_row, const void* w_sg) {
    double z = 0.0;
    for (int32_t i = 0; i < d; ++i) z += elem(x_row, dtype, (size_t)i) * elem(w_sg, dtype, (size_t)i);
    return 1.0 / (1.0 + exp(-z));
}

int32_t orc_token_output(const orc_cfg_t* c, const void* x_row, const int32_t* idx_t,
                         const double* g_t, const uint8_t* cls_t,
                         const void* const* w13, const void* const* w2,
                         const void* w13s, const void* w2s,
                         const void* const* lA, const void* const* lB,
                         double* out, double* ys, double* yslot) {
    return orc_token_output_sg(c, x_row, idx_t, g_t, cls_t, w13, w2, w13s, w2s, NULL, lA, lB, out, ys, yslot);
}

int32_t orc_token_output_sg(const orc_cfg_t* c, const void* x_row, const int32_t* idx_t,
                            const double* g_t, const uint8_t* cls_t,
                            const void* const* w13, const void* const* w2,
                            const void* w13s, const void* w2s, const void* w_sg,
                            const void* const* lA, const void* const* lB,
                            double* out, double* ys, double* yslot) {
    const int32_t d = c->d, K = c->top_k;
    double* x = (double*)calloc((size_t)d, sizeof(double));
    double* s = (double*)calloc((size_t)d, sizeof(double));
    double* y = (double*)calloc((size_t)d, sizeof(double));
    int32_t rc = 0;
    for (int32_t j = 0; j < d; ++j) x[j] = elem(x_row, c->dtype, (size_t)j);

    /* the always-active shared block S(x) (Sec. 2.1), with its output gate if given */
    orc_swiglu(d, c->shared_inter, c->dtype, w13s, w2s, x, s);
    if (w_sg) {
        const double gs = orc_shared_gate(d, c->dtype, x_row, w_sg);
        for (int32_t j = 0; j < d; ++j) s[j] *= gs;
    }
    for (int32_t j = 0; j < d; ++j) out[j] = s[j];
    if (ys)
        for (int32_t j = 0; j < d; ++j) ys[j] = s[j];

    for (int32_t k = 0; k < K; ++k) {
        const int32_t e = idx_t[k];
        const double gk = g_t[k];
        if (cls_t[k] == ORC_LORE) {
            /* Eq. 11: the missing expert's output is replaced by S(x) + B_e A_e x */
            if (!lA[e] || !lB[e]) { rc = -1; break; }
            orc_lore_delta(d, c->lore_rank, c->dtype, lA[e], lB[e], x, y);
            for (int32_t j = 0; j < d; ++j) out[j] += gk * (s[j] + y[j]);
        } else {
            /* resident hit, or exact miss served with the same expert weights */
            if (!w13[e] || !w2[e]) { rc = -1; break; }
            orc_swiglu(d, c->inter, c->wfmt == ORC_MXFP4 ? ORC_MXFP4 : c->dtype, w13[e], w2[e], x, y);
            for (int32_t j = 0; j < d; ++j) out[j] += gk * y[j];
        }
        if (yslot)
            for (int32_t j = 0; j < d; ++j) yslot[(size_t)k * d + j] = y[j];
    }
    free(x);
    free(s);
    free(y);
    return rc;
}

int32_t orc_exact_residual(const orc_cfg_t* c, int32_t T, const void* x, const int32_t* idx,
                           const double* g, const uint8_t* cls, const void* const* w13,
                           const void* const* w2, double* resid) {
    const int32_t d = c->d, K = c->top_k;
    double* xr = (double*)malloc(sizeof(double) * (size_t)d);
    double* y = (double*)malloc(sizeof(double) * (size_t)d);
    int32_t rc = 0;
    for (int32_t t = 0; t < T && rc == 0; ++t) {
        for (int32_t j = 0; j < d; ++j) {
            xr[j] = elem(x, c->dtype, (size_t)t * d + j);
            resid[(size_t)t * d + j] = 0.0;
        }
        for (int32_t k = 0; k < K; ++k) {
            size_t s = (size_t)t * K + k;
            if (cls[s] != ORC_EXACT) continue;
            if (!w13[idx[s]] || !w2[idx[s]]) { rc = -1; break; }
            orc_swiglu(d, c->inter, c->wfmt == ORC_MXFP4 ? ORC_MXFP4 : c->dtype, w13[idx[s]], w2[idx[s]], xr, y);
            for (int32_t j = 0; j < d; ++j) resid[(size_t)t * d + j] += g[s] * y[j];
        }
    }
    free(xr);
    free(y);
    return rc;
}

int32_t orc_lru_step(int32_t n_experts, int32_t C, int32_t* slot_expert, int32_t* last_use,
                     int32_t step, int32_t T, int32_t K, const int32_t* idx, const uint8_t* cls,
                     int32_t max_admit, int32_t* admitted, int32_t* evicted) {
    int32_t* exact_count = (int32_t*)calloc((size_t)n_experts, sizeof(int32_t));
    int32_t* slot_of = (int32_t*)malloc(sizeof(int32_t) * (size_t)n_experts);
    for (int32_t e = 0; e < n_experts; ++e) slot_of[e] = -1;
    for (int32_t sl = 0; sl < C; ++sl)
        if (slot_expert[sl] >= 0) slot_of[slot_expert[sl]] = sl;

    /* touch the experts that were hit in this step */
    for (int32_t s = 0; s < T * K; ++s) {
        if (cls[s] == ORC_HIT && slot_of[idx[s]] >= 0) last_use[slot_of[idx[s]]] = step;
        if (cls[s] == ORC_EXACT) exact_count[idx[s]]++;
    }

    int32_t n_adm = 0;
    while (n_adm < max_admit) {
        /* next candidate: most tokens, then lowest id; never a LoRE-only miss */
        int32_t cand = -1;
        for (int32_t e = 0; e < n_experts; ++e) {
            if (exact_count[e] == 0 || slot_of[e] >= 0) continue;
            if (cand < 0 || exact_count[e] > exact_count[cand]) cand = e;
        }
        if (cand < 0) break;
        /* victim: least recently used slot not used in this step, ties by expert id
         * (an empty slot, expert -1, sorts first among equal last_use) */
        int32_t victim = -1;
        for (int32_t sl = 0; sl < C; ++sl) {
            if (last_use[sl] == step) continue;
            if (victim < 0 || last_use[sl] < last_use[victim] ||
                (last_use[sl] == last_use[victim] && slot_expert[sl] < slot_expert[victim]))
                victim = sl;
        }
        if (victim < 0) break;
        int32_t old = slot_expert[victim];
        if (old >= 0) slot_of[old] = -1;
        slot_expert[victim] = cand;
        slot_of[cand] = victim;
        last_use[victim] = step;
        exact_count[cand] = 0;
        admitted[n_adm] = cand;
        evicted[n_adm] = old;
        ++n_adm;
    }
    free(exact_count);
    free(slot_of);
    return n_adm;
}

/* ---- Speculative prefetching ------------------------------------------------------- */

double orc_round_to(int32_t dtype, double v) {
    if (dtype != ORC_BF16) return (double)(float)v;
    if (v == 0.0 || isnan(v) || isinf(v)) return v;
    /* bf16 keeps 8 significant bits: round v to a multiple of 2^(e-8), v = m 2^e, m in [0.5, 1) */
    int e;
    frexp(v, &e);
    if (e < -125) e = -125; /* subnormal range of the 8-bit exponent */
    const double ulp = ldexp(1.0, e - 8);
    return rint(v / ulp) * ulp; /* rint: to nearest, ties to even (default rounding mode) */
}

static void store_elem(void* p, int32_t dtype, size_t i, double v) {
    if (dtype == ORC_BF16) {
        float f = (float)orc_round_to(ORC_BF16, v); /* exact: a bf16 value is an fp32 value */
        uint32_t bits;
        memcpy(&bits, &f, sizeof bits);
        ((uint16_t*)p)[i] = (uint16_t)(bits >> 16);
    } else {
        ((float*)p)[i] = (float)v;
    }
}

int32_t orc_spec_step(const orc_cfg_t* c, int32_t T, int32_t delta, int32_t l_min, double tau, int32_t last,
                      const void* h_in, const void* wg, const float* bias, const void* w13s, const void* w2s,
                      const void* const* lA, const void* const* lB, int32_t* halted, int32_t* pred_idx,
                      double* pred_prob, double* conf, void* h_out) {
    const int32_t d = c->d, N = c->n_experts, K = c->top_k;
    orc_cfg_t raw = *c;
    raw.norm_topk = 0; /* pi is the router's own distribution */
    double* z = (double*)malloc(sizeof(double) * (size_t)N);
    int32_t* idx = (int32_t*)malloc(sizeof(int32_t) * (size_t)K);
    double* g = (double*)malloc(sizeof(double) * (size_t)K);
    double* h = (double*)malloc(sizeof(double) * (size_t)d);
    double* sh = (double*)malloc(sizeof(double) * (size_t)d);
    double* dl = (double*)malloc(sizeof(double) * (size_t)d);
    double* nh = (double*)malloc(sizeof(double) * (size_t)d);
    int32_t rc = 0;
    for (int32_t t = 0; t < T && rc == 0; ++t) {
        const size_t row = (size_t)t * d;
        for (int32_t i = 0; i < d; ++i) h[i] = elem(h_in, c->dtype, row + i);
        int32_t update = 0;
        if (halted[t]) {
            for (int32_t k = 0; k < K; ++k) {
                pred_idx[(size_t)t * K + k] = -1;
                pred_prob[(size_t)t * K + k] = 0.0;
            }
            conf[t] = NAN;
        } else {
            /* Step 1: the future layer's router on the draft state (Eq. 1, Eq. 2) */
            orc_router_logits(&raw, 1, (const char*)h_in + row * (c->dtype == ORC_BF16 ? 2 : 4), wg, bias, z, NULL);
            orc_gates_topk(&raw, 1, z, idx, g, NULL);
            /* Step 2: enqueue; Step 3: confidence (Eq. 5) and the halting test */
            double cf = 0.0;
            for (int32_t k = 0; k < K; ++k) {
                pred_idx[(size_t)t * K + k] = idx[k];
                pred_prob[(size_t)t * K + k] = g[k];
                cf += g[k];
            }
            conf[t] = cf;
            if (delta >= l_min && cf < tau) halted[t] = 1;
            else update = !last;
        }
        if (update) {
            /* Step 4: h <- Attn(h) + sum_k pi_k (S(h) + B_k A_k h), Attn = identity */
            orc_swiglu(d, c->shared_inter, c->dtype, w13s, w2s, h, sh);
            for (int32_t i = 0; i < d; ++i) nh[i] = h[i];
            for (int32_t k = 0; k < K; ++k) {
                for (int32_t i = 0; i < d; ++i) dl[i] = 0.0;
                if (c->lore_rank > 0) {
                    if (!lA[idx[k]] || !lB[idx[k]]) { rc = -1; break; }
                    orc_lore_delta(d, c->lore_rank, c->dtype, lA[idx[k]], lB[idx[k]], h, dl);
                }
                for (int32_t i = 0; i < d; ++i) nh[i] += g[k] * (sh[i] + dl[i]);
            }
            for (int32_t i = 0; i < d; ++i) store_elem(h_out, c->dtype, row + i, nh[i]);
        } else {
            for (int32_t i = 0; i < d; ++i) store_elem(h_out, c->dtype, row + i, h[i]);
        }
    }
    free(z); free(idx); free(g); free(h); free(sh); free(dl); free(nh);
    return rc;
}

int32_t orc_h_min(double P, double M_e, double B, double t_attn, int32_t K, double t_expert) {
    const double window = t_attn + (double)K * t_expert;
    if (!(window > 0.0) || !(B > 0.0)) return -1;
    return (int32_t)ceil(P * M_e / (B * window));
}

void orc_prefetch_queue(int32_t n_experts, int32_t n_depth, int32_t T, int32_t K, const int32_t* pred_idx,
                        const double* pred_prob, int32_t max_per_depth, int32_t* experts, int32_t* counts) {
    double* mass = (double*)malloc(sizeof(double) * (size_t)n_experts);
    int32_t* seen = (int32_t*)malloc(sizeof(int32_t) * (size_t)n_experts);
    for (int32_t dp = 0; dp < n_depth; ++dp) {
        for (int32_t e = 0; e < n_experts; ++e) { mass[e] = 0.0; seen[e] = 0; }
        /* Eq. 3: union of the enqueued sets of this depth, with their predicted mass */
        for (int32_t t = 0; t < T; ++t)
            for (int32_t k = 0; k < K; ++k) {
                const size_t i = ((size_t)dp * T + t) * K + k;
                if (pred_idx[i] < 0) continue;
                seen[pred_idx[i]] = 1;
                mass[pred_idx[i]] += pred_prob[i];
            }
        int32_t n = 0;
        while (n < max_per_depth) {
            int32_t best = -1;
            for (int32_t e = 0; e < n_experts; ++e)
                if (seen[e] && (best < 0 || mass[e] > mass[best])) best = e;
            if (best < 0) break;
            seen[best] = 0;
            experts[(size_t)dp * max_per_depth + n++] = best;
        }
        counts[dp] = n;
    }
    free(mass);
    free(seen);
}

int32_t orc_lru_prefetch(int32_t n_experts, int32_t C, int32_t* slot_expert, int32_t* last_use, int32_t step,
                         int32_t n, const int32_t* experts, int32_t max_prefetch, int32_t* admitted,
                         int32_t* evicted) {
    int32_t* listed = (int32_t*)calloc((size_t)n_experts, sizeof(int32_t));
    for (int32_t i = 0; i < n; ++i) listed[experts[i]] = 1;
    int32_t n_adm = 0;
    for (int32_t i = 0; i < n && n_adm < max_prefetch; ++i) {
        const int32_t e = experts[i];
        int32_t resident = 0;
        for (int32_t sl = 0; sl < C; ++sl)
            if (slot_expert[sl] == e) resident = 1;
        if (resident) continue;
        int32_t victim = -1;
        for (int32_t sl = 0; sl < C; ++sl) {
            if (last_use[sl] == step) continue;
            if (slot_expert[sl] >= 0 && listed[slot_expert[sl]]) continue;
            if (victim < 0 || last_use[sl] < last_use[victim] ||
                (last_use[sl] == last_use[victim] && slot_expert[sl] < slot_expert[victim]))
                victim = sl;
        }
        if (victim < 0) break;
        admitted[n_adm] = e;
        evicted[n_adm] = slot_expert[victim];
        ++n_adm;
        slot_expert[victim] = e;
        last_use[victim] = step;
    }
    free(listed);
    return n_adm;
}
