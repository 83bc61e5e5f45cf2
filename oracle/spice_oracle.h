/*
 * spice_oracle.h -- reference oracle for SPICE's per-layer MoE forward under a
 * partial GPU expert cache (arXiv 2608.21240, Sec. 2.1-2.2, 4.2, 4.3).
 *
 * TEST INFRASTRUCTURE ONLY.  This is a plain, slow CPU implementation in fp64
 * written from the paper to check the HIP library against.  It shares no code,
 * header, helper or table with the library; only tests, the package smoke
 * check and the benchmark's CPU-baseline leg may load it.
 *
 * Storage types: every tensor argument is either fp32 (dtype 0) or bf16 bits
 * stored as uint16 (dtype 1).  Each element is widened to double exactly and
 * all arithmetic is done in double.
 *
 * All matrices are row-major with Linear's [out][in] convention:
 *   router   Wg  [N][d]
 *   expert   W13 [2I][d]  (rows 0..I-1 = gate W1, rows I..2I-1 = up W3), W2 [d][I]
 *   shared   W13s[2Is][d], W2s[d][Is]
 *   LoRE     A   [r][d],  B [d][r]          (Eq. 9)
 * Slot id of token t's k-th routed choice = t*K + k.
 *
 * MXFP4 weights (routed experts when cfg.wfmt == ORC_MXFP4, OCP Microscaling formats v1.0):
 * a [rows][K] matrix (K a multiple of 32) is one byte blob: rows*K/2 bytes of FP4 E2M1
 * codes, row-major, element 2i in the low nibble of byte i and 2i+1 in the high nibble;
 * then rows*K/32 bytes of E8M0 block scales, row-major, one per 32 consecutive elements
 * of a row.  Element value = 2^(scale - 127) * e2m1(code).  W13 is [2I][d], W2 [d][I].
 * Parity pins: see tests/test_oracle_*.py.  No function here is unpinned.
 * Speculative prefetching (Alg. 1) uses an identity stand-in for the target layer's
 * attention: this oracle covers the MoE part of the draft update only.
 */
#ifndef SPICE_ORACLE_H
#define SPICE_ORACLE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum { ORC_F32 = 0, ORC_BF16 = 1, ORC_MXFP4 = 2 };
enum { ORC_HIT = 0, ORC_LORE = 1, ORC_EXACT = 2 };
enum { ORC_CONF_INPUT = 0, ORC_CONF_GATE = 1, ORC_CONF_GATE_RENORM = 2 };

typedef struct {
    int32_t d, n_experts, top_k, inter, shared_inter, lore_rank;
    int32_t dtype;     /* ORC_F32 / ORC_BF16 */
    int32_t norm_topk; /* 1: divide the K selected gates by their sum */
    int32_t conf_mode; /* ORC_CONF_* */
    float tau;         /* confidence threshold */
    int32_t wfmt;      /* routed experts' weight format: 0 = the cfg dtype, ORC_MXFP4 = MXFP4 blobs */
} orc_cfg_t;

/* Router logits z[t][e] = sum_i x[t][i] Wg[e][i] + bias[e] (Eq. 1).  zabs (nullable)
 * receives sum_i |x[t][i] Wg[e][i]|, the scale of the summation's rounding error. */
void orc_router_logits(const orc_cfg_t* c, int32_t T, const void* x, const void* wg,
                       const float* bias, double* z, double* zabs);

/* Softmax over all N experts and top-K by logit (descending, ties -> lower id):
 * idx[T][K], gate g[T][K] = softmax prob of the chosen expert (renormalised over
 * the K when norm_topk).  probs (nullable) receives the full softmax [T][N]. */
void orc_gates_topk(const orc_cfg_t* c, int32_t T, const double* z, int32_t* idx, double* g,
                    double* probs);

/* Per-slot confidence (fp32): caller's conf_in, the gate, or the renormalised gate. */
void orc_confidence(const orc_cfg_t* c, int32_t T, const double* g, const float* conf_in,
                    float* conf);

/* Slot class: HIT if the expert is resident, else LORE if conf < tau, else EXACT
 * (a NaN confidence is EXACT).  resident[e] != 0 means resident. */
void orc_classify(const orc_cfg_t* c, int32_t T, const int32_t* idx, const int32_t* resident,
                  const float* conf, uint8_t* cls);

/* Counting sort of slot ids by key (class, expert), stable in slot order.
 * offsets[3][N+1]: offsets[c][e] = first position of bucket (c, e); offsets[c][N] = end
 * of class c.  perm[pos] = slot, inv_perm[slot] = pos.  counts[3] (nullable) per class. */
void orc_bucket(const orc_cfg_t* c, int32_t T, const int32_t* idx, const uint8_t* cls,
                int32_t* offsets, int32_t* perm, int32_t* inv_perm, int32_t* counts);

/* One SwiGLU FFN on one token: y = W2 (silu(W1 x) * (W3 x)), x given in double.  dtype is
 * the weights' storage: ORC_F32, ORC_BF16 or ORC_MXFP4 (blobs as described above). */
void orc_swiglu(int32_t d, int32_t inter, int32_t dtype, const void* w13, const void* w2,
                const double* x, double* y);

/* LoRE correction delta = B (A x) for one token (Eq. 9). */
void orc_lore_delta(int32_t d, int32_t r, int32_t dtype, const void* A, const void* B,
                    const double* x, double* delta);

/* Layer output of one token t (Eq. 7 and Eq. 11 inside the gate-weighted sum of
 * Sec. 2.1):  out = S(x) + sum_{HIT,EXACT} g E_e(x) + sum_{LORE} g (S(x) + B_e A_e x).
 * w13/w2/lA/lB are per-expert pointer tables [N]; only experts this token needs
 * must be non-NULL.  ys (nullable) receives S(x); yslot (nullable, [K][d]) the
 * per-slot term (E_e(x) or B_e A_e x).  Returns 0, or -1 if a needed pointer is NULL. */
int32_t orc_token_output(const orc_cfg_t* c, const void* x_row, const int32_t* idx_t,
                         const double* g_t, const uint8_t* cls_t,
                         const void* const* w13, const void* const* w2,
                         const void* w13s, const void* w2s,
                         const void* const* lA, const void* const* lB,
                         double* out, double* ys, double* yslot);

/* The shared block's output gate sigmoid(sum_i x[i] w_sg[i]) for one token: the
 * Qwen2-style shared expert, whose output is scaled by this gate. */
double orc_shared_gate(int32_t d, int32_t dtype, const void* x_row, const void* w_sg);

/* orc_token_output with a gated shared block (w_sg [d], nullable): S(x) is
 * orc_shared_gate(x) SwiGLU_s(x), in the plain term and inside every LoRE slot's S(x) + B A x. */
int32_t orc_token_output_sg(const orc_cfg_t* c, const void* x_row, const int32_t* idx_t,
                            const double* g_t, const uint8_t* cls_t,
                            const void* const* w13, const void* const* w2,
                            const void* w13s, const void* w2s, const void* w_sg,
                            const void* const* lA, const void* const* lB,
                            double* out, double* ys, double* yslot);

/* One MXFP4 element (r, c) of a [rows][K] blob, widened to double (exact). */
double orc_mxfp4_elem(const void* blob, int32_t rows, int32_t K, int32_t r, int32_t c);

/* Exact residual of the CPU path (Sec. 4.3): resid[t] = sum_{k in EXACT(t)} g[t][k] E_e(x_t).
 * Returns 0, or -1 if a needed expert pointer is NULL. */
int32_t orc_exact_residual(const orc_cfg_t* c, int32_t T, const void* x, const int32_t* idx,
                           const double* g, const uint8_t* cls, const void* const* w13,
                           const void* const* w2, double* resid);

/* LRU expert-cache step for one layer at one decode step (the stack workload).
 * State: slot_expert[C] (expert in each slot), last_use[C] (step of last use, -1 unused).
 * HIT experts are touched; EXACT-miss experts are admission candidates ordered by
 * (token count desc, id asc); each takes the slot of the resident expert with the
 * smallest (last_use, expert id) not used in this step; at most max_admit.  LORE
 * misses are never admitted.  admitted[] / evicted[] receive up to max_admit ids.
 * Returns the number admitted. */
int32_t orc_lru_step(int32_t n_experts, int32_t C, int32_t* slot_expert, int32_t* last_use,
                     int32_t step, int32_t T, int32_t K, const int32_t* idx, const uint8_t* cls,
                     int32_t max_admit, int32_t* admitted, int32_t* evicted);

/* ---- Speculative prefetching (Sec. 4.1, Eq. 2-5, Alg. 1) ----------------------------- */

/* A value rounded to the storage dtype: nearest representable fp32 or bf16, ties to even
 * (bf16 rounding is done once, from the double, not through fp32). */
double orc_round_to(int32_t dtype, double v);

/* One depth delta (1-based) of the draft rollout of Alg. 1 for T tokens, each token on
 * its own.  Layer weights are those of layer l + delta: router wg[N][d] (+ bias[N] or
 * NULL), shared block w13s/w2s, LoRE tables lA/lB [N] (every routed expert non-NULL when
 * lore_rank > 0).  For a token still running (halted[t] == 0):
 *   pi = softmax of the router logits of h_in[t] (Eq. 1); S = TopK(pi) (Eq. 2, ties to the
 *   lower id); the prediction is enqueued: pred_idx[t][k] = S[k], pred_prob[t][k] = pi[S[k]];
 *   conf[t] = sum_k pi[S[k]] (Eq. 5);
 *   if delta >= l_min and conf[t] < tau: halted[t] = 1 (the prediction stays queued);
 *   else unless last: h_out[t] = round(h_in[t] + sum_k pi_k (S(h_in[t]) + B_k A_k h_in[t]))
 *   (the attention of the target layer is the identity here; Ẽ_k = S + B_k A_k, Eq. 11).
 * A token halted before this depth gets pred_idx -1, pred_prob 0 and conf NaN.  h_out of
 * a token not updated is h_in.  h_in and h_out are [T][d] in the cfg's dtype and may be
 * the same array.  Returns 0, or -1 if a needed LoRE pointer is NULL. */
int32_t orc_spec_step(const orc_cfg_t* c, int32_t T, int32_t delta, int32_t l_min, double tau, int32_t last,
                      const void* h_in, const void* wg, const float* bias, const void* w13s, const void* w2s,
                      const void* const* lA, const void* const* lB, int32_t* halted, int32_t* pred_idx,
                      double* pred_prob, double* conf, void* h_out);

/* Eq. 4: the least lookahead that hides the transfer of P experts of M_e bytes at
 * bandwidth B behind per-layer compute T_attn + K T_expert:
 * ceil(P M_e / (B (T_attn + K T_expert))).  Returns -1 if the compute window or B is not > 0. */
int32_t orc_h_min(double P, double M_e, double B, double t_attn, int32_t K, double t_expert);

/* Prefetch intents of one rollout (Eq. 3), per depth: the union over tokens of the
 * enqueued sets, in issue order: larger predicted mass sum_t pi first, ties to the lower
 * id; at most max_per_depth per depth.  pred_idx/pred_prob: [n_depth][T][K] as written
 * by orc_spec_step (-1 = nothing enqueued).  experts [n_depth][max_per_depth], counts [n_depth]. */
void orc_prefetch_queue(int32_t n_experts, int32_t n_depth, int32_t T, int32_t K, const int32_t* pred_idx,
                        const double* pred_prob, int32_t max_per_depth, int32_t* experts, int32_t* counts);

/* Speculative admissions into one layer's LRU cache at step `step`: the listed experts in
 * order, skipping resident ones, each into the slot of the resident expert with the
 * smallest (last_use, id) that was not used in this step and is not listed; the admitted
 * expert gets last_use = step.  At most max_prefetch; returns the number admitted. */
int32_t orc_lru_prefetch(int32_t n_experts, int32_t C, int32_t* slot_expert, int32_t* last_use, int32_t step,
                         int32_t n, const int32_t* experts, int32_t max_prefetch, int32_t* admitted,
                         int32_t* evicted);

#ifdef __cplusplus
}
#endif
#endif
