/*
 * spice_moe.h -- C ABI of the SPICE MoE-layer hot path for AMD Instinct MI355X (gfx950).
 *
 * The library computes one Mixture-of-Experts layer under a partial GPU expert
 * cache, as SPICE defines it (arXiv 2608.21240):
 *   1. router logits and top-K gating                    (Eq. 1; Sec. 2.1, 2.2)
 *   2. per-slot classification: resident hit, low-confidence miss (LoRE),
 *      exact miss; then bucketing of slots by (class, expert)   (Sec. 4.2, 4.3)
 *   3. grouped SwiGLU FFN of the resident experts plus the always-resident
 *      shared block                                       (Eq. 6; Sec. 2.1, 4.2)
 *   4. LoRE surrogate B_e A_e h for low-confidence misses (Eq. 7, 9, 11)
 *   5. exact CPU residual for exact misses, from host weights (Sec. 4.3, M_cpu)
 *   6. gate-weighted combine of all terms                 (Sec. 2.1; Eq. 11; Sec. 4.3 merge)
 *
 * Conventions for every entry point
 *   - Plain pointers.  "device" = memory the GPU reads/writes (hipMalloc or
 *     equivalent); "host" = CPU memory.  The caller owns every buffer, including
 *     the workspace; the library keeps no pointer after returning (except the
 *     cache handle, which borrows what it was created with until destroyed).
 *   - Row-major arrays.  Weight matrices use Linear's [out][in] layout.
 *     Expert ids are 0..N-1.  Slot id of token t's k-th choice = t*K + k.
 *   - dtype SPICE_F32: activations and weights are fp32.  dtype SPICE_BF16:
 *     activations and weights are bf16 (passed as raw 16-bit values); all
 *     accumulation is fp32 (router logits: fp64).
 *   - Device entry points check their arguments on the host, then enqueue
 *     kernels on `stream` and return; they never synchronise.  A bad value
 *     inside a device array (an out-of-range cache slot or expert id) never
 *     causes an out-of-bounds access: the kernels skip it and raise a flag
 *     in the workspace (read it with spice_workspace_flags).
 *   - Entry points never abort or throw; they return a negative status and
 *     leave a message for spice_last_error() (per thread).  T == 0 is a no-op
 *     that returns SPICE_OK.
 */
#ifndef SPICE_MOE_H
#define SPICE_MOE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Same type as hipStream_t; NULL selects the default stream. */
typedef struct ihipStream_t* spice_stream_t;

typedef enum {
    SPICE_OK = 0,
    SPICE_ERR_INVALID = -1,     /* a bad argument (NULL, out of range, overflow, aliasing) */
    SPICE_ERR_UNSUPPORTED = -2, /* valid but not handled: size alignment, dtype, N > 256 ... */
    SPICE_ERR_HIP = -3,         /* the HIP runtime reported an error (launch, copy, earlier fault) */
    SPICE_ERR_WORKSPACE = -4,   /* workspace smaller than spice_workspace_bytes() */
    SPICE_ERR_INTERNAL = -5
} spice_status_t;

enum { SPICE_F32 = 0, SPICE_BF16 = 1 };
/* Where the per-slot routing confidence comes from (Sec. 4.2 leaves it open):
 * the caller's array, the slot's gate score, or the gate renormalised over the K. */
enum { SPICE_CONF_INPUT = 0, SPICE_CONF_GATE = 1, SPICE_CONF_GATE_RENORM = 2 };
/* Slot classes (Sec. 4.2): resident or prefetched -> exact on the GPU; missing with
 * confidence < tau -> shared + LoRE; otherwise an exact miss served on the CPU.
 * SPICE_CLASS_EXACT_GPU marks an exact miss whose expert was fetched for this call and
 * computed on the GPU (M_fetch of Eq. 12); routing never produces it: moe_split_plan
 * (host copy) and moe_expert_ffn_fetched (device copy) relabel EXACT slots to it. */
enum { SPICE_CLASS_HIT = 0, SPICE_CLASS_LORE = 1, SPICE_CLASS_EXACT = 2, SPICE_CLASS_EXACT_GPU = 3 };

#define SPICE_MAX_EXPERTS 256
#define SPICE_MAX_TOKENS 65536
#define SPICE_MAX_LORE_RANK 256
/* The first SPICE_WS_CONTROL_BYTES of a workspace hold counters and flags.
 * They must be zero before the workspace is first used (spice_workspace_init,
 * or any zero fill); every completed call leaves the counters zero again. */
#define SPICE_WS_CONTROL_BYTES 131072

/* Device-side flags (bit mask) raised in the workspace by a kernel that met bad data. */
#define SPICE_FLAG_BAD_SLOT 1u   /* resident_slot[e] outside [-1, n_slots) */
#define SPICE_FLAG_BAD_INDEX 2u  /* perm / offsets / topk_idx value out of range */

typedef struct {
    int32_t d;            /* hidden size */
    int32_t n_experts;    /* N routed experts, 1..256 */
    int32_t top_k;        /* K, 1..N */
    int32_t inter;        /* I, routed SwiGLU intermediate size */
    int32_t shared_inter; /* I_s, intermediate of the shared block (all shared experts stacked) */
    int32_t lore_rank;    /* r of Eq. 9, 0..256 */
    int32_t n_slots;      /* C, slots of the GPU expert pool */
    int32_t dtype;        /* SPICE_F32 or SPICE_BF16 */
    int32_t norm_topk;    /* 1: renormalise the K selected gates to sum 1 */
    int32_t conf_mode;    /* SPICE_CONF_* */
    float tau;            /* confidence threshold: LoRE iff conf < tau (NaN conf -> exact) */
    int32_t wfmt;         /* routed experts' weight format: SPICE_WFMT_DTYPE or SPICE_WFMT_MXFP4 */
} spice_moe_cfg_t;

/* Weight formats of the routed experts (the pool slots and the host copies).
 * SPICE_WFMT_DTYPE: the cfg dtype, W13 [2I][d] and W2 [d][I] row-major.
 * SPICE_WFMT_MXFP4: OCP Microscaling MXFP4 (quantised expert weights; the paper runs one of
 *   its models with 5-bit weights of an unnamed layout).  A [rows][K] matrix is one byte
 *   blob: rows*K/2 bytes of FP4 E2M1 codes, row-major, element 2i in the low nibble of byte
 *   i and 2i+1 in the high one; then rows*K/32 bytes of E8M0 scales, row-major, one per 32
 *   consecutive elements of a row; element value = 2^(scale - 127) * e2m1(code).  A W13 blob
 *   holds [2I][d] (2I*d*17/32 bytes), a W2 blob [d][I] (d*I*17/32 bytes); a pool slot is one
 *   such blob.  Needs dtype SPICE_BF16 (activations, router, shared block and LoRE factors
 *   stay bf16), d and inter multiples of 32 and at most SPICE_MXFP4_MAX_K, and blobs below
 *   2 GiB.  The fetched-expert split (moe_split_plan,
 *   moe_fetch_experts, moe_expert_ffn_fetched) and moe_lore_fit return UNSUPPORTED for it;
 *   at any T the expert FFN runs on the streaming kernels, not the prefill GEMMs. */
enum { SPICE_WFMT_DTYPE = 0, SPICE_WFMT_MXFP4 = 2 };
#define SPICE_MXFP4_MAX_K 4096

/* Size alignment required: d, inter and shared_inter multiples of 8 (bf16) or 4 (fp32);
 * lore_rank a multiple of 8 (bf16) or 4 (fp32). */

/* Bytes of device workspace that a call with T tokens needs (every entry point below
 * accepts the same workspace).  Returns 0 for an invalid cfg or T. */
size_t spice_workspace_bytes(const spice_moe_cfg_t* cfg, int32_t T);

/* Zero the control region of a device workspace (a fill kernel on `stream`). */
spice_status_t spice_workspace_init(void* ws, size_t ws_bytes, spice_stream_t stream);

/* Copy the device flags of a workspace to *flags (synchronises `stream`); clear them if clear != 0. */
spice_status_t spice_workspace_flags(void* ws, size_t ws_bytes, uint32_t* flags, int32_t clear,
                                     spice_stream_t stream);

/*
 * Host copies written by moe_route_bucket (and moe_layer_gpu) for the exact CPU path
 * (Sec. 4.3: the hidden state and the routing decision of the exact misses go to the CPU).
 * Each pointer is pinned host memory that the GPU can write (hipHostMalloc, torch's
 * pin_memory), or NULL to skip that copy; pageable memory is rejected.  A kernel writes
 * them over PCIe; they are complete once the stream has passed the call, or, earlier,
 * once *ready holds ready_value: the kernel stores ready_value after every copy has
 * landed (spice_wait_ready waits for it on the host).  Use a new ready_value per call.
 */
typedef struct {
    void* x;               /* [T][d] dtype: the activations */
    int32_t* topk_idx;     /* [T][K] */
    float* topk_w;         /* [T][K] */
    uint8_t* slot_class;   /* [T][K] */
    int32_t* class_counts; /* [3]: slots per class (HIT, LORE, EXACT) */
    uint32_t* ready;       /* [1] or NULL: receives ready_value after the copies above */
    uint32_t ready_value;
} spice_host_out_t;

/* Wait on the host until *ready == value (a pinned word a kernel writes, e.g.
 * spice_host_out_t.ready).  Returns SPICE_ERR_HIP with a message if timeout_us passes
 * first (timeout_us <= 0: wait up to 10 s), INVALID for a NULL pointer. */
spice_status_t spice_wait_ready(const volatile uint32_t* ready, uint32_t value, int64_t timeout_us);

/*
 * Steps 1-2: router logits z = x Wg^T (+ bias), softmax over all N, top-K by logit
 * (descending, ties -> lower expert id; Eq. 1), gate g = softmax probability of the
 * chosen expert (Sec. 2.1 weighting), per-slot confidence and class (Sec. 4.2), and a
 * stable counting sort of slot ids by (class, expert).
 *   x             device [T][d]      activations (dtype)
 *   w_gate        device [N][d]      router weight (dtype)
 *   logit_bias    device [N] fp32    added to the logits, or NULL
 *   resident_slot device [N] int32   pool slot of expert e, or -1 when not resident
 *   conf          device [T][K] fp32 per-slot confidence; required iff conf_mode == INPUT
 *   logits        device [T][N] fp64 out, or NULL (logits are summed in fp64)
 *   topk_idx      device [T][K] int32 out
 *   topk_w        device [T][K] fp32 out, gate scores
 *   slot_class    device [T][K] uint8 out, SPICE_CLASS_*
 *   offsets       device [3][N+1] int32 out: offsets[c][e] = first position of bucket
 *                 (c, e) in perm; offsets[c][N] = end of class c (classes laid out
 *                 HIT, LORE, EXACT; inside a bucket slots keep ascending slot order)
 *   perm          device [T*K] int32 out: perm[pos] = slot id
 *   inv_perm      device [T*K] int32 out: inv_perm[slot] = pos
 *   host_out      host copies for the CPU path (see spice_host_out_t), or NULL
 * The workspace also receives the device work lists of the buckets (per class, the
 * non-empty buckets in ascending expert order with start and size), which the fused
 * layer path reads.  T <= 256 runs one block per token and one bucketing block; larger
 * T computes the logits as fp64 MFMA tiles.
 */
spice_status_t moe_route_bucket(const spice_moe_cfg_t* cfg, int32_t T, const void* x,
                                const void* w_gate, const float* logit_bias,
                                const int32_t* resident_slot, const float* conf, double* logits,
                                int32_t* topk_idx, float* topk_w, uint8_t* slot_class,
                                int32_t* offsets, int32_t* perm, int32_t* inv_perm,
                                const spice_host_out_t* host_out, void* ws, size_t ws_bytes,
                                spice_stream_t stream);

/*
 * Step 3: grouped SwiGLU FFN y = W2 (silu(W1 x) * (W3 x)) (Eq. 6) for every HIT slot,
 * grouped by expert, plus the shared block S(x) (Sec. 2.1, 4.2) for all T tokens.
 * When lore_A and lore_B are both non-NULL the LoRE corrections of step 4 are computed
 * in the same launches (the same result as calling lore_surrogate_apply).
 *   x, perm, offsets       as produced/consumed by moe_route_bucket
 *   resident_slot device [N] int32, as in moe_route_bucket
 *   w13_pool      device [C][2I][d]  rows 0..I-1 gate W1, rows I..2I-1 up W3 (dtype)
 *   w2_pool       device [C][d][I]   down projection (dtype)
 *   w13_shared    device [2I_s][d], w2_shared device [d][I_s]   (ignored if I_s == 0)
 *   lore_A, lore_B see lore_surrogate_apply, or NULL
 *   y_slots       device [T*K][d] fp32 out: row pos = expert output for slot perm[pos]
 *                 (HIT rows; LORE rows too when LoRE is fused; other rows untouched)
 *   y_shared      device [T][d] fp32 out: S(x_t)
 */
spice_status_t moe_expert_ffn_grouped(const spice_moe_cfg_t* cfg, int32_t T, const void* x,
                                      const int32_t* perm, const int32_t* offsets,
                                      const int32_t* resident_slot, const void* w13_pool,
                                      const void* w2_pool, const void* w13_shared,
                                      const void* w2_shared, const void* lore_A,
                                      const void* lore_B, float* y_slots, float* y_shared,
                                      void* ws, size_t ws_bytes, spice_stream_t stream);

/*
 * Step 3 with a gated shared block (the Qwen2-style shared expert, whose output carries a
 * sigmoid gate): as moe_expert_ffn_grouped, with
 *   S(x_t) = sigmoid(w_sg . x_t) SwiGLU_s(x_t),
 * the dot product taken in fp64.  S is the model's native shared expert of Sec. 4.2, so the
 * gated S is what y_shared holds and what moe_combine (and the draft update) use, in the
 * plain shared term and inside every LoRE slot's S(x) + B_e A_e x (Eq. 7 / 11).
 *   w_shared_gate  device [d] (dtype): the gate's weight row; required when shared_inter > 0
 * The gate values go to the workspace (its size covers them).  Errors: as
 * moe_expert_ffn_grouped, plus INVALID for a NULL w_shared_gate.
 */
spice_status_t moe_expert_ffn_grouped_gated(const spice_moe_cfg_t* cfg, int32_t T, const void* x,
                                            const int32_t* perm, const int32_t* offsets,
                                            const int32_t* resident_slot, const void* w13_pool,
                                            const void* w2_pool, const void* w13_shared,
                                            const void* w2_shared, const void* w_shared_gate,
                                            const void* lore_A, const void* lore_B, float* y_slots,
                                            float* y_shared, void* ws, size_t ws_bytes,
                                            spice_stream_t stream);

/*
 * Step 4: LoRE correction delta = B_e (A_e x) (Eq. 9) for every LORE slot, grouped by
 * expert.  The shared part S(x) of Eq. 11 is not recomputed: moe_combine adds it.
 *   lore_A  device [N][r][d] (dtype), lore_B device [N][d][r] (dtype): factors of every
 *           routed expert, always resident (Sec. 4.2)
 *   y_slots device [T*K][d] fp32 out: LORE rows receive delta; other rows untouched
 */
spice_status_t lore_surrogate_apply(const spice_moe_cfg_t* cfg, int32_t T, const void* x,
                                    const int32_t* perm, const int32_t* offsets,
                                    const void* lore_A, const void* lore_B, float* y_slots,
                                    void* ws, size_t ws_bytes, spice_stream_t stream);

/*
 * Step 6: out[t] = (1 + sum_{k in LORE(t)} g) S(x_t) + sum_{k in HIT(t) or EXACT_GPU(t)} g y
 *                  + sum_{k in LORE(t)} g delta + resid[t]
 * i.e. the gate-weighted sum of Sec. 2.1 with each LoRE slot's output replaced by
 * S(x) + B_e A_e x (Eq. 11) and the CPU outputs merged in (Sec. 4.3).
 *   topk_w, slot_class, inv_perm  device, from moe_route_bucket
 *   y_slots device [T*K][d] fp32, y_shared device [T][d] fp32
 *   resid   [T][d] fp32 exact-miss residual, or NULL (treated as zero): device memory,
 *           or pinned host memory (read over PCIe: the CPU result needs no separate copy)
 *   out     device [T][d] dtype out (bf16: round to nearest even); must not alias inputs
 */
spice_status_t moe_combine(const spice_moe_cfg_t* cfg, int32_t T, const float* topk_w,
                           const uint8_t* slot_class, const int32_t* inv_perm,
                           const float* y_slots, const float* y_shared, const float* resid,
                           void* out, spice_stream_t stream);

/*
 * Steps 1-4 (and 6 when out != NULL) of one layer call, enqueued on `stream` as one unit:
 * routing and bucketing (as moe_route_bucket), the grouped FFN of the HIT slots and the
 * shared block with the LoRE corrections fused (as moe_expert_ffn_grouped, or
 * moe_expert_ffn_grouped_gated when w_shared_gate != NULL), then, if out != NULL, the
 * combine with `resid` (as moe_combine).  Every output is the one those calls define.
 * The work that does not depend on routing is not ordered after it (Sec. 4.2: the shared
 * block S is always resident): for T <= 256 and T*K <= 1024 (routed experts in the cfg
 * dtype or in MXFP4; bf16 dtype experts only while the prefill GEMMs do not apply) the call is
 * three launches in which routing runs beside the shared block's up projection, the
 * shared block's down projection beside the routed up projections, and each routed tile
 * finds its bucket from the routing itself; otherwise the separate launches of those calls.
 * For the CPU path of Sec. 4.3, pass host_out (its ready word is stored as soon as the
 * copies have landed, before the FFN ends) and out = NULL, run moe_exact_residual_host on
 * the copies, then moe_combine.
 *   Arguments: as in moe_route_bucket, moe_expert_ffn_grouped(_gated) and moe_combine;
 *   lore_A / lore_B NULL: no LoRE rows (call lore_surrogate_apply separately);
 *   resid, out as in moe_combine (out NULL: no combine; resid is then ignored).
 * Errors: those of the calls it stands for.
 */
spice_status_t moe_layer_gpu(const spice_moe_cfg_t* cfg, int32_t T, const void* x, const void* w_gate,
                             const float* logit_bias, const int32_t* resident_slot, const float* conf,
                             const void* w13_pool, const void* w2_pool, const void* w13_shared,
                             const void* w2_shared, const void* w_shared_gate, const void* lore_A,
                             const void* lore_B, double* logits, int32_t* topk_idx, float* topk_w,
                             uint8_t* slot_class, int32_t* offsets, int32_t* perm, int32_t* inv_perm,
                             float* y_slots, float* y_shared, const spice_host_out_t* host_out,
                             const float* resid, void* out, void* ws, size_t ws_bytes,
                             spice_stream_t stream);

/*
 * moe_layer_gpu for callers that cannot allocate device memory: code under HIP graph
 * capture, tight serving loops, and harnesses that forbid hipMalloc.  The same launches and
 * outputs as moe_layer_gpu; instead of a caller's workspace it uses a static device array
 * of SPICE_NOALLOC_SCRATCH_BYTES that the library holds on each GPU it runs on until the
 * process ends (zero when loaded; its device address is looked up once per device).  The
 * call allocates nothing.  The caller still passes every input and output.
 *   Errors: those of moe_layer_gpu; UNSUPPORTED when spice_workspace_bytes(cfg, T) exceeds
 *   SPICE_NOALLOC_SCRATCH_BYTES.  Device flags raised by the kernels are not reported.
 * Every call on one GPU shares that GPU's array: calls that overlap on one GPU (different
 * streams, or host threads without ordering) race and must not be issued.
 */
#define SPICE_NOALLOC_SCRATCH_BYTES (32u << 20)
spice_status_t moe_layer_gpu_noalloc(const spice_moe_cfg_t* cfg, int32_t T, const void* x,
                                     const void* w_gate, const float* logit_bias,
                                     const int32_t* resident_slot, const float* conf,
                                     const void* w13_pool, const void* w2_pool,
                                     const void* w13_shared, const void* w2_shared,
                                     const void* w_shared_gate, const void* lore_A,
                                     const void* lore_B, double* logits, int32_t* topk_idx,
                                     float* topk_w, uint8_t* slot_class, int32_t* offsets,
                                     int32_t* perm, int32_t* inv_perm, float* y_slots,
                                     float* y_shared, const spice_host_out_t* host_out,
                                     const float* resid, void* out, spice_stream_t stream);

/*
 * Step 5, host side: resid[t] = sum_{k in EXACT(t)} g[t][k] E_e(x_t) computed on the
 * CPU from host-resident expert weights (M_cpu of Eq. 12; Sec. 4.3: exact, the same
 * weights, routing untouched).  Synchronous and reentrant; uses n_threads worker
 * threads (<= 0: one per online CPU).  The result does not depend on n_threads.
 *   x_host        host [T][d] (dtype)
 *   topk_idx_host host [T][K] int32, topk_w_host host [T][K] fp32,
 *   slot_class_host host [T][K] uint8 (only EXACT slots are computed; EXACT_GPU is skipped)
 *   w13_host      host table [N] of pointers to [2I][d] (dtype); entries of experts with
 *                 no EXACT slot may be NULL
 *   w2_host       host table [N] of pointers to [d][I] (dtype)
 *   resid_host    host [T][d] fp32 out (overwritten; zero rows for tokens with no exact slot)
 */
spice_status_t moe_exact_residual_host(const spice_moe_cfg_t* cfg, int32_t T, const void* x_host,
                                       const int32_t* topk_idx_host, const float* topk_w_host,
                                       const uint8_t* slot_class_host,
                                       const void* const* w13_host, const void* const* w2_host,
                                       float* resid_host, int32_t n_threads);

/*
 * Expert cache of a decode stack (the stack workload): per layer, the set of routed
 * experts resident in that layer's slot pool, which the hit test of Sec. 4.2 reads
 * through resident_slot.  The paper's GPU holds only part of the experts (Sec. 1, 3)
 * and compares against an LRU-managed cache (Sec. 5); this handle keeps each layer's
 * pool LRU-managed as follows.  After the layer's call at decode step s:
 *   1. experts of the call's HIT slots are marked used at s;
 *   2. experts of its EXACT slots that are not resident are candidates, more EXACT
 *      slots first, then lower id; LORE misses are never admitted (Sec. 4.2: they need
 *      no transfer);
 *   3. each candidate, at most max_admit per call (a bounded copy queue), takes the slot
 *      whose expert was used longest ago, ties to the lower expert id (an empty slot
 *      first), never a slot used at s; the new slot counts as used at s;
 *   4. the admitted weights are copied host -> pool on copy_stream, ordered after the
 *      work already queued on compute_stream, and the layer's device resident_slot is
 *      rewritten after them.
 * Admitted experts are still EXACT (served on the CPU) in step s; they are resident
 * for the layer's next call, which moe_cache_wait orders after the copies.
 * A handle is not thread-safe; one host thread drives it.
 */
typedef struct spice_cache spice_cache_t;

/*
 * Create a cache for n_layers layers of the same cfg, each with cfg->n_slots slots.
 *   w13_host, w2_host host tables [n_layers * N] of host pointers to expert e of layer l
 *                     at [l*N + e]: [2I][d] and [d][I] (dtype).  Pinned memory lets the
 *                     copies run asynchronously.  Entries may be NULL for experts that
 *                     are never admitted or loaded.
 *   w13_pool, w2_pool host tables [n_layers] of device pool bases ([C][2I][d], [C][d][I])
 *   resident_slot     host table [n_layers] of device int32 [N] arrays that the cache
 *                     keeps equal to its state (the moe_route_bucket / FFN input)
 *   initial_experts   host [n_layers][C] int32: expert in each slot (-1 = empty), each
 *                     expert at most once per layer; every slot starts "never used"
 *   load              1: copy the initial experts into the pools and write resident_slot
 *                     now, on `stream`, and wait for it; 0: the caller has done both
 *   out               receives the handle
 * With w13_pool == NULL the handle does the bookkeeping only: no pools, copies or HIP
 * calls (then w2_pool, resident_slot and the host tables are ignored and load must be 0).
 * The handle borrows every pointer in the tables until moe_cache_destroy.
 */
spice_status_t moe_cache_create(const spice_moe_cfg_t* cfg, int32_t n_layers, const void* const* w13_host,
                                const void* const* w2_host, void* const* w13_pool, void* const* w2_pool,
                                int32_t* const* resident_slot, const int32_t* initial_experts, int32_t load,
                                spice_stream_t stream, spice_cache_t** out);

/*
 * Update layer `layer` after its call at decode step `step` (rules 1-4 above).
 *   topk_idx_host, slot_class_host  host [T][K]: the call's routing (moe_route_bucket)
 *   max_admit          admissions allowed in this call (>= 0)
 *   copy_stream        stream of the host -> pool copies; compute_stream: stream of the
 *                      layer's kernels (the copies wait for its queued work, which this
 *                      call marks as the layer's last use on every call)
 *   n_admitted         out: number admitted
 *   admitted, evicted  host [max_admit] out: admitted experts in order, and the expert
 *                      each one replaced (-1 = the slot was empty)
 * Returns INVALID for out-of-range ids or classes, or a NULL host weight of an EXACT
 * expert; the state is then unchanged.
 */
spice_status_t moe_cache_step(spice_cache_t* cache, int32_t layer, int32_t step, int32_t T,
                              const int32_t* topk_idx_host, const uint8_t* slot_class_host, int32_t max_admit,
                              spice_stream_t copy_stream, spice_stream_t compute_stream, int32_t* n_admitted,
                              int32_t* admitted, int32_t* evicted);

/* Make `stream` wait for the layer's outstanding admissions (no-op if none).  Call it
 * before the layer's next moe_route_bucket. */
spice_status_t moe_cache_wait(spice_cache_t* cache, int32_t layer, spice_stream_t stream);

/* Host copy of a layer's state: slot_expert[C] and last_use[C] (-1 = never); either may be NULL. */
spice_status_t moe_cache_state(const spice_cache_t* cache, int32_t layer, int32_t* slot_expert, int32_t* last_use);

/* Wait for outstanding copies and free the handle (NULL is ignored). */
void moe_cache_destroy(spice_cache_t* cache);

/*
 * Exact-miss split M = M_fetch + M_cpu (Eq. 12; Sec. 4.3).  The paper's scheduler serves
 * every exact miss on the CPU unless fetching some of them over PCIe and running them
 * on the GPU, in parallel with the CPU, beats that plan by a safety margin.  It gives no
 * formula; this cost model is the library's own:
 *   CPU time of a set   = sum_e (expert_bytes / cpu_bytes_per_s + n_e * flops / cpu_flops_per_s)
 *   fetch time of a set = sum_e expert_bytes / pcie_bytes_per_s + gpu_fixed_s
 *   plan time           = max(CPU time of M_cpu, fetch time of M_fetch)
 * Candidates are taken in order of decreasing CPU cost (more tokens first, then lower
 * id); the plan with the smallest time is kept if it is below (1 - margin) times the
 * all-CPU time, otherwise nothing is fetched.
 */
typedef struct {
    double cpu_bytes_per_s;   /* host DRAM rate of the exact CPU path over expert weights */
    double cpu_flops_per_s;   /* its arithmetic rate (2 flops per multiply-add) */
    double pcie_bytes_per_s;  /* host -> GPU copy rate */
    double gpu_fixed_s;       /* fixed GPU-side cost of serving fetched experts (launches, FFN) */
    double margin;            /* fraction the split must save over all-CPU, e.g. 0.05 */
} spice_split_cost_t;

/*
 * Choose M_fetch from one call's routing (host copies, e.g. moe_route_bucket's host_out).
 *   slot_class_host host [T][K] in/out: EXACT slots of the chosen experts become EXACT_GPU
 *                   (so moe_exact_residual_host skips them)
 *   max_fetch       most experts to fetch (the fetch pool's slots)
 *   fetch_experts   host [max_fetch] out: chosen experts in order; n_fetch out: their count
 */
spice_status_t moe_split_plan(const spice_moe_cfg_t* cfg, int32_t T, const int32_t* topk_idx_host,
                              uint8_t* slot_class_host, const spice_split_cost_t* cost, int32_t max_fetch,
                              int32_t* fetch_experts, int32_t* n_fetch);

/*
 * Copy the chosen experts into a fetch pool on `copy_stream`: expert experts[i] into
 * slot i of w13_fetch [n_slots][2I][d] / w2_fetch [n_slots][d][I], and write
 * fetch_expert (device [n_slots] int32: expert id of each slot, -1 = unused) from the
 * caller's pinned staging row fetch_expert_stage (host [n_slots]).  The caller orders
 * its compute stream after `copy_stream` (an event) before moe_expert_ffn_fetched, and
 * leaves fetch_expert_stage and the pools alone until `copy_stream` has passed the call.
 *   w13_host, w2_host host tables [N] as in moe_exact_residual_host (pinned memory lets
 *                     the copies run asynchronously)
 */
spice_status_t moe_fetch_experts(const spice_moe_cfg_t* cfg, int32_t n_fetch, const int32_t* experts,
                                 const void* const* w13_host, const void* const* w2_host, void* w13_fetch,
                                 void* w2_fetch, int32_t n_slots, int32_t* fetch_expert,
                                 int32_t* fetch_expert_stage, spice_stream_t copy_stream);

/*
 * SwiGLU FFN (Eq. 6) of the fetched experts' EXACT slots on the GPU: for fetch slot j
 * with expert e = fetch_expert[j] >= 0, every slot of the bucket (EXACT, e) gets its
 * expert output in y_slots (row = bucket position) and its class becomes EXACT_GPU in
 * slot_class, so moe_combine adds it like a HIT slot.
 *   x, perm, offsets, slot_class  device, from moe_route_bucket (slot_class in/out)
 *   fetch_expert  device [n_slots] int32, from moe_fetch_experts
 *   w13_fetch, w2_fetch  device fetch pool
 *   y_slots       device [T*K][d] fp32 out (those rows only)
 */
spice_status_t moe_expert_ffn_fetched(const spice_moe_cfg_t* cfg, int32_t T, const void* x, const int32_t* perm,
                                      const int32_t* offsets, uint8_t* slot_class, const int32_t* fetch_expert,
                                      const void* w13_fetch, const void* w2_fetch, int32_t n_slots,
                                      float* y_slots, void* ws, size_t ws_bytes, spice_stream_t stream);

/*
 * Speculative prefetching (Sec. 4.1, Eq. 2-5, Alg. 1).  A draft rollout starts from the
 * current layer's input hidden state h0 [T][d] and runs depth delta = 1, 2, ... with the
 * weights of layer l + delta.  Each depth is three calls on one stream:
 *   1. moe_route_bucket on the draft state with the future layer's router, every expert
 *      absent (resident_slot all -1), conf all 0, cfg->conf_mode SPICE_CONF_INPUT,
 *      cfg->norm_topk 0 and cfg->tau > 0: every slot is then LoRE and topk_w holds the
 *      router's own probabilities pi;
 *   2. moe_expert_ffn_grouped with that layer's shared block and LoRE factors (no hits):
 *      y_shared = S(h), y_slots = B_k A_k h at each slot's bucket position;
 *   3. moe_spec_update below.
 * A token runs Alg. 1 on its own: it halts after the first depth >= l_min whose
 * confidence is below tau.  The target layer's attention is not part of this library:
 * the draft state moves by the MoE part only (an identity stand-in for Attn).
 */

/* Pinned host copies of one depth's predictions (each pointer may be NULL). */
typedef struct {
    int32_t* pred_idx;  /* [T][K] */
    float* pred_prob;   /* [T][K] */
    float* conf;        /* [T] */
} spice_spec_host_t;

/*
 * Steps 2-4 of Alg. 1 at depth `depth` (1-based) for every token t with halted[t] == 0:
 *   enqueue pred_idx[t][k] = topk_idx[t][k], pred_prob[t][k] = topk_w[t][k] (Eq. 2);
 *   conf[t] = sum_k topk_w[t][k] (Eq. 5, summed in fp64, stored fp32);
 *   if depth >= l_min and conf[t] < tau: halted[t] = 1;
 *   else, unless last != 0: h_out[t] = h_in[t] + sum_k pi_k (y_shared[t] + y_slots[inv_perm[t*K+k]])
 *   computed in fp32 and stored in the cfg's dtype (bf16: round to nearest even).
 * Tokens halted before this depth get pred_idx -1, pred_prob 0, conf NaN; tokens not
 * updated get h_out = h_in.
 *   h_in, h_out  device [T][d] (dtype); h_out may be h_in itself but not overlap it otherwise
 *   topk_idx, topk_w, inv_perm, y_slots, y_shared  device, from steps 1-2 of this depth
 *                (y_slots is not read when cfg->lore_rank is 0)
 *   halted       device [T] int32, in/out; zero it before depth 1
 *   pred_idx, pred_prob, conf  device [T][K], [T][K], [T] out
 *   host_out     nullable; pinned host copies written by the kernel (valid once the stream
 *                has passed the call)
 *   ws, ws_bytes the workspace of steps 1-2 (its flags word records an out-of-range inv_perm)
 */
spice_status_t moe_spec_update(const spice_moe_cfg_t* cfg, int32_t T, int32_t depth, int32_t l_min, float tau,
                               int32_t last, const void* h_in, void* h_out, const int32_t* topk_idx,
                               const float* topk_w, const int32_t* inv_perm, const float* y_slots,
                               const float* y_shared, int32_t* halted, int32_t* pred_idx, float* pred_prob,
                               float* conf, const spice_spec_host_t* host_out, void* ws, size_t ws_bytes,
                               spice_stream_t stream);

/*
 * Eq. 4: the least lookahead depth that hides the copies of P experts of expert_bytes
 * each at pcie_bytes_per_s behind per-layer compute t_attn_s + K * t_expert_s:
 * ceil(P * expert_bytes / (pcie_bytes_per_s * (t_attn_s + K * t_expert_s))).
 * Returns -1 if the compute window or the bandwidth is not > 0, or an argument is negative.
 */
int32_t moe_prefetch_h_min(double P, double expert_bytes, double pcie_bytes_per_s, double t_attn_s, int32_t K,
                           double t_expert_s);

/*
 * The prefetch intents of one rollout (Eq. 3) as per-depth issue lists: the union over
 * tokens of the experts enqueued at that depth, larger predicted mass sum_t pi first
 * (summed in fp64), ties to the lower id, at most max_per_depth each.
 *   pred_idx_host, pred_prob_host  host [n_depth][T][K] (-1 = nothing enqueued)
 *   experts      host [n_depth][max_per_depth] out;  counts  host [n_depth] out
 */
spice_status_t moe_prefetch_queue(const spice_moe_cfg_t* cfg, int32_t T, int32_t n_depth,
                                  const int32_t* pred_idx_host, const float* pred_prob_host, int32_t max_per_depth,
                                  int32_t* experts, int32_t* counts);

/*
 * Speculative admissions into layer `layer`'s cache at decode step `step` (the bounded
 * prefetch queue of Sec. 4.1): the n listed experts in order, skipping resident ones,
 * each into the slot of the resident expert with the smallest (last_use, id) that was
 * not used in this step and is not listed; the admitted expert gets last_use = step.
 * At most max_prefetch.  The copies wait for the layer's last call, as marked by its
 * last moe_cache_step (so every call of a layer must be followed by moe_cache_step for
 * it before a prefetch into it), and for the layer's earlier copies; they do not wait
 * for other work on the compute stream, so a prefetch into a future layer overlaps the
 * current one.  moe_cache_wait orders the layer's next call after them.  Experts whose
 * host weights are NULL are skipped.  compute_stream is not used.
 *   admitted, evicted  host [max_prefetch] out, n_admitted out
 */
spice_status_t moe_cache_prefetch(spice_cache_t* cache, int32_t layer, int32_t step, int32_t n,
                                  const int32_t* experts, int32_t max_prefetch, spice_stream_t copy_stream,
                                  spice_stream_t compute_stream, int32_t* n_admitted, int32_t* admitted,
                                  int32_t* evicted);

/*
 * LoRE calibration fit (Sec. 4.2, Eq. 8-10) of one expert from n calibration tokens:
 * the factors A [r][d], B [d][r] minimising sum_t || E_e(x_t) - S(x_t) - B A x_t ||^2.
 * With n <= d tokens of full rank every residual is reachable, so the minimiser is the
 * truncated SVD of the residual matrix carried back through the tokens' pseudo-inverse
 * (minimum-norm A); the loss is the sum of the squared singular values beyond the r-th,
 * and r >= n fits exactly (directions beyond n are zero rows of A / columns of B).
 * E_e and S run on the GPU (the grouped-FFN kernels), the n x n Gram matrices in fp64 on
 * the GPU, their eigen-decomposition and solve in fp64 on the host.  The call is
 * synchronous: it returns when A and B are written.
 *   n            calibration tokens, 1 <= n <= min(d, 1024)
 *   r            rank, 1 <= r <= d (the LoRE rank; it may differ from cfg->lore_rank)
 *   x            device [n][d] (dtype) calibration hidden states, linearly independent
 *   w13, w2      device weights of the expert: [2I][d], [d][I] (dtype)
 *   w13_shared, w2_shared  device shared block (ignored when cfg->shared_inter is 0)
 *   A_out, B_out device fp32 [r][d] and [d][r] out
 *   y_out        nullable device fp32 [n][d] out: the residual targets E_e(x) - S(x)
 *   loss_out     nullable host out: Eq. 10's minimum (fp64, from the residual spectrum)
 *   ws, ws_bytes workspace of spice_lore_fit_workspace_bytes(cfg, n, r) bytes
 * Returns UNSUPPORTED for n > min(d, 1024), INVALID for linearly dependent tokens.
 */
size_t spice_lore_fit_workspace_bytes(const spice_moe_cfg_t* cfg, int32_t n, int32_t r);
spice_status_t moe_lore_fit(const spice_moe_cfg_t* cfg, int32_t n, int32_t r, const void* x, const void* w13,
                            const void* w2, const void* w13_shared, const void* w2_shared, float* A_out, float* B_out,
                            float* y_out, double* loss_out, void* ws, size_t ws_bytes, spice_stream_t stream);

/* Text of a status code, and the last error message of the calling thread. */
const char* spice_status_string(spice_status_t status);
const char* spice_last_error(void);

#ifdef __cplusplus
}
#endif
#endif
