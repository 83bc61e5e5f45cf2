// Router logits, softmax top-K gating, per-slot classification and (class, expert)
// bucketing (Eq. 1; Sec. 2.1, 4.2, 4.3).  No block waits for another block.
//
// T <= kRouteTokenMaxT (decode), one launch (route_logits_kernel): a token's router rows
//   are spread over several blocks (one row per wave), each summing its logits in fp64; the
//   last of the token's blocks to finish (an arrival counter per token) takes the token's
//   top-K, gates, confidence and classes and publishes them, with the slots' bucket keys,
//   at the device-coherent level; the last of those blocks over all tokens (a second
//   arrival counter) sorts the T*K slots by (class, expert), writes the work lists and,
//   when asked, the CPU path's host copies and their ready word.
// Larger T (prefill), three launches:
//   1. route_prefill_kernel: per 16 tokens, the logits as fp64 MFMA tiles of 16 experts x
//      16 tokens (two waves per tile, each half the contraction), then the tokens' top-K,
//      gates and classes in the same block, and the block's histogram of bucket keys;
//   2. bucket_scan_kernel: a wave per bucket key turns its histogram row into each routing
//      block's running count within the key and the key's total; the last scan block to
//      finish turns the totals into each key's start (offsets, work lists, class counts);
//   3. bucket_scatter_kernel: per 16 tokens, the stable positions of their slots (perm,
//      inv_perm).  The last scan block also writes the host copies when asked.
//
// bf16 x bf16 and fp32 x fp32 products are exact in fp64, so on every path only the
// summation order of the logits differs from a plain loop.
#include <hip/hip_runtime.h>

#include "route_device.h"

namespace spice {
namespace {

constexpr int kLogitThreads = 256;   // routing logits: 4 waves, kRouteRowsPerWave router rows each
constexpr int kBucketCache = 1024;   // slots whose keys stay in LDS while the last block buckets them
// LDS of a decode routing block: the top-K scratch, then (in the last block) the bucketing tables
constexpr size_t kLogitLdsBytes = sizeof(TopkLds) > bucket_lds_bytes(kLogitThreads, SPICE_MAX_EXPERTS, kBucketCache)
                                      ? sizeof(TopkLds)
                                      : bucket_lds_bytes(kLogitThreads, SPICE_MAX_EXPERTS, kBucketCache);

typedef double f64x4_t __attribute__((ext_vector_type(4)));

template <int DT>
__global__ __launch_bounds__(kLogitThreads) void route_logits_kernel(RouteArgs a, int g_per_tok) {
    __shared__ __align__(16) int s_lds[kLogitLdsBytes / sizeof(int)];
    __shared__ int s_flag;
    const int t = blockIdx.x / g_per_tok, g = blockIdx.x % g_per_tok;
    const int rows = (kLogitThreads / 64) * kRouteRowsPerWave;
    const int n_rows = a.N + (a.w_sg ? 1 : 0);
    route_logits_rows<DT>(a, t, g * rows, min(n_rows, (g + 1) * rows));
    if (!route_last_block(&a.ctrl[kWordTokCount + t * kTokCountStride], g_per_tok, &s_flag)) return;
    block_topk<kLogitThreads, true, true>(a, t, a.logits_ws + (size_t)t * a.N, *reinterpret_cast<TopkLds*>(s_lds));
    // the published top-K outputs and keys of every token are at the device-coherent level
    // once every token's last block has counted itself here
    if (!route_last_block(&a.ctrl[kWordRouteDone], a.T, &s_flag)) return;
    bucket_slots<kLogitThreads, kBucketCache, true>(a, s_lds);
    if (a.hx || a.h_idx || a.h_w || a.h_cls || a.h_ready) mirror_host<kLogitThreads, true>(a);
}

constexpr int kPrefillThreads = 1024;  // 16 waves
constexpr int kGroupTiles = 2;          // expert tiles of 16 per routing wave
constexpr int kPrefillTok = 16;       // tokens per prefill routing block (one MFMA tile wide)
constexpr int kScanThreads = 1024;    // bucket_scan_kernel: a wave per key; the last block a thread per key
constexpr int kScanKeys = kScanThreads / 64;  // bucket keys per scan block
static_assert(3 * SPICE_MAX_EXPERTS <= kScanThreads, "a scan thread per bucket key");

// The prefill histogram table in the workspace's logits region (unused on this path: the
// top-K reads the logits from LDS): [3N][stride] counts (key-major, one column per routing
// block), then the [3N] key starts, then [3N] key totals (each row 4-aligned; the whole is
// under 1 byte per logit byte: (3N + 1) * (T / 16 + 4) + 3N ints against 8 T N bytes).
__host__ __device__ inline int prefill_hist_stride(int T) { return ((T + kPrefillTok - 1) / kPrefillTok + 3) & ~3; }

struct PrefillLds {
    // partial logits of the contraction parts: [parts][16 tokens][N], with parts x N <=
    // waves x 16 x kGroupTiles (parts = waves / groups, groups >= N / (16 kGroupTiles))
    double zp[kPrefillThreads / 64 * 16 * kGroupTiles * kPrefillTok];
    double z[kPrefillTok][SPICE_MAX_EXPERTS];  // logits
    unsigned long long key[kPrefillTok][SPICE_MAX_EXPERTS];  // their order-preserving keys
    int res[SPICE_MAX_EXPERTS];
    int pick[kPrefillTok][64];
    int hist[3 * SPICE_MAX_EXPERTS];
};

// The products of up to kGroupTiles expert tiles (16 experts each, from tile0) with 16 tokens over
// the contraction passes [p0, p1), with v_mfma_f64_16x16x4f64; each pass's x chunk is
// widened once for all the tiles.  A 16-byte load gives each lane 8 (bf16) or 4 (fp32)
// consecutive k of one row: lane (m = lane % 16, q = lane / 16) holds row m's elements
// q*V .. q*V + V-1 of a 4V-wide k chunk, and MFMA step u takes element u of every lane, so
// the 4 k of step u are {u, V + u, 2V + u, 3V + u} for both operands and each chunk's
// products are all summed once.  A pass is two chunks; the next pass's loads are in flight
// while one multiplies.  d is a multiple of V.
template <int DT>
__device__ __forceinline__ void prefill_group(const RouteArgs& a, const char* xr, int tile0, int ntg,
                                              int p0, int p1, int lane, f64x4_t (&out)[kGroupTiles]) {
    using E = RouteElem<DT>;
    constexpr int V = E::V, es = E::es;
    const int m = lane & 15, q = lane >> 4;
    const char* wr[kGroupTiles];
#pragma unroll
    for (int i = 0; i < kGroupTiles; ++i) {
        const int e = (tile0 + i) * 16 + m;
        wr[i] = static_cast<const char*>(a.wg) + (size_t)(i < ntg && e < a.N ? e : 0) * a.d * es;
    }
    f64x4_t acc[kGroupTiles][2] = {};
    // Loads are unconditional, from clamped addresses: rows past N and tokens past T read
    // row 0 / token 0 (finite values whose products land only in dropped outputs), and
    // chunks past d read chunk 0 of the row, whose x is zeroed where it is used.  A select
    // at the load would make every pass wait for the next pass's loads to land.
    auto load = [&](int p, uint4 (&xb)[2], uint4 (&wb)[kGroupTiles][2]) {
#pragma unroll
        for (int c = 0; c < 2; ++c) {
            const int k = p * 8 * V + c * 4 * V + q * V;
            const size_t kk = (size_t)(k < a.d ? k : 0) * es;
            xb[c] = *reinterpret_cast<const uint4*>(xr + kk);
#pragma unroll
            for (int i = 0; i < kGroupTiles; ++i) wb[i][c] = *reinterpret_cast<const uint4*>(wr[i] + kk);
        }
    };
    auto mul = [&](int p, const uint4 (&xb)[2], const uint4 (&wb)[kGroupTiles][2]) {
#pragma unroll
        for (int c = 0; c < 2; ++c) {
            const int k = p * 8 * V + c * 4 * V + q * V;
            const uint4 zero = {0u, 0u, 0u, 0u};
            double xd[V];
            E::widen(k < a.d ? xb[c] : zero, xd);
#pragma unroll
            for (int i = 0; i < kGroupTiles; ++i) {
                if (i < ntg) {  // uniform
                    double wd[V];
                    E::widen(wb[i][c], wd);
#pragma unroll
                    for (int u = 0; u < V; ++u)  // two accumulators per tile
                        acc[i][u & 1] = __builtin_amdgcn_mfma_f64_16x16x4f64(wd[u], xd[u], acc[i][u & 1], 0, 0, 0);
                }
            }
        }
    };
    if (p0 < p1) {
        uint4 xa[2], wa[kGroupTiles][2], xb[2], wb[kGroupTiles][2];
        load(p0, xa, wa);
        int p = p0;
        for (; p + 1 < p1; p += 2) {
            load(p + 1, xb, wb);
            mul(p, xa, wa);
            load(min(p + 2, p1 - 1), xa, wa);  // past the end: reloads the last pass, unused
            mul(p + 1, xb, wb);
        }
        if (p < p1) mul(p, xa, wa);
    }
#pragma unroll
    for (int i = 0; i < kGroupTiles; ++i) out[i] = acc[i][0] + acc[i][1];
}

// Prefill routing of tokens [16 b, 16 b + 16): logits, top-K, gates, classes, and the
// block's histogram of bucket keys (column b of the table).
template <int DT>
__global__ __launch_bounds__(kPrefillThreads) void route_prefill_kernel(RouteArgs a) {
    __shared__ PrefillLds L;
    constexpr int kNW = kPrefillThreads / 64;
    const int tid = threadIdx.x, lane = tid & 63, m = lane & 15, q = lane >> 4;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int N = a.N, K = a.K, NK = 3 * N;
    const int t0 = blockIdx.x * kPrefillTok;
    const int tok = t0 + m;
    const bool tok_ok = tok < a.T;
    const int es = RouteElem<DT>::es;
    const char* xr = static_cast<const char*>(a.x) + (size_t)(tok_ok ? tok : 0) * a.d * es;
    for (int e = tid; e < N; e += kPrefillThreads) L.res[e] = a.resident_slot[e];
    for (int k = tid; k < NK; k += kPrefillThreads) L.hist[k] = 0;

    // logits: the expert tiles in groups of kGroupTiles; wave w takes group w / parts and
    // contraction part w % parts (parts = waves / groups), leaving its partial logits in LDS;
    // then the parts are summed in order
    const int ntile = (N + 15) / 16, ngroups = (ntile + kGroupTiles - 1) / kGroupTiles, parts = kNW / ngroups;
    const int npass = (a.d + 8 * RouteElem<DT>::V - 1) / (8 * RouteElem<DT>::V);
    if (w < ngroups * parts) {
        const int g = w / parts, kp = w - g * parts;
        const int ntg = min(kGroupTiles, ntile - kGroupTiles * g);
        f64x4_t part[kGroupTiles];
        prefill_group<DT>(a, xr, kGroupTiles * g, ntg, kp * npass / parts, (kp + 1) * npass / parts, lane, part);
        // result layout of the f64 16x16x4 product: element v of lane (m, q) is expert
        // tile*16 + 4v + q for token t0 + m
#pragma unroll
        for (int i = 0; i < kGroupTiles; ++i)
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                const int ee = (kGroupTiles * g + i) * 16 + 4 * v + q;
                if (i < ntg && ee < N) L.zp[(kp * kPrefillTok + m) * N + ee] = part[i][v];
            }
    }
    __syncthreads();
    for (int i = tid; i < kPrefillTok * N; i += kPrefillThreads) {
        const int tt = i / N, ee = i - tt * N;
        double z = L.zp[tt * N + ee];
        for (int kp = 1; kp < parts; ++kp) z += L.zp[(kp * kPrefillTok + tt) * N + ee];
        z += a.bias ? (double)a.bias[ee] : 0.0;
        L.z[tt][ee] = z;
        L.key[tt][ee] = logit_key(z);
        if (a.logits_out && t0 + tt < a.T) a.logits_out[(size_t)(t0 + tt) * N + ee] = z;
    }
    __syncthreads();

    // top-K: wave w ranks tokens w, w + waves, ... (rank of e = experts with a larger logit,
    // or an equal one and a smaller id); then its wave takes the gates and classes
    constexpr int kJ = SPICE_MAX_EXPERTS / 64;
    static_assert(kPrefillTok % kNW == 0, "whole tokens per wave");
#pragma unroll
    for (int h = 0; h < kPrefillTok / kNW; ++h) {
        const int tt = w + h * kNW;
        const unsigned long long* kr = L.key[tt];
#pragma unroll
        for (int j = 0; j < kJ; ++j) {
            const int e = lane + 64 * j;
            if (64 * j < N) {  // uniform
                const unsigned long long ke = e < N ? kr[e] : 0ull;
                int r = 0;
#pragma unroll 8
                for (int ee = 0; ee < N; ++ee) {
                    const unsigned long long k2 = kr[ee];
                    r += (int)((k2 > ke) | ((k2 == ke) & (ee < e)));
                }
                if (e < N && r < K) L.pick[tt][r] = e;
            }
        }
    }
    __syncthreads();
    // then the block's histogram of bucket keys
#pragma unroll
    for (int h = 0; h < kPrefillTok / kNW; ++h) {
        const int tt = w + h * kNW, t = t0 + tt;
        if (t < a.T) {
            const float conf_in = (a.conf_mode == SPICE_CONF_INPUT && lane < K) ? a.conf[(size_t)t * K + lane] : 0.f;
            const int key = wave_topk_gates(a, t, L.z[tt], L.res, L.pick[tt], lane, conf_in);
            if (key >= 0) atomicAdd(&L.hist[key], 1);
        }
    }
    __syncthreads();
    // as column blockIdx.x of the table
    int* table = reinterpret_cast<int*>(a.logits_ws);
    const int stride = prefill_hist_stride(a.T);
    for (int k = tid; k < NK; k += kPrefillThreads) table[(size_t)k * stride + blockIdx.x] = L.hist[k];
}

// Each wave: one key's exclusive running count over the routing blocks (in place) and its
// total.  The last block to finish: the keys' starts (an exclusive scan over keys in order)
// to offsets, the table's start row and the work lists; the class counts; then the host
// copies when asked.
__global__ __launch_bounds__(kScanThreads) void bucket_scan_kernel(RouteArgs a) {
    __shared__ int s_tot[3 * SPICE_MAX_EXPERTS];
    __shared__ int s_start[3 * SPICE_MAX_EXPERTS];
    __shared__ int s_wsum[kScanThreads / 64];
    __shared__ int s_cls[3];
    __shared__ int s_res[SPICE_MAX_EXPERTS];
    __shared__ int s_flag;
    constexpr int kChunks = 4;  // 256-column spans whose loads one round trip carries
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const int N = a.N, NK = 3 * N;
    const int nblk = (a.T + kPrefillTok - 1) / kPrefillTok, stride = prefill_hist_stride(a.T);
    int* table = reinterpret_cast<int*>(a.logits_ws);
    int* totals = table + (size_t)(NK + 1) * stride;
    const int key = blockIdx.x * kScanKeys + w;
    if (key < NK) {
        // lane l holds columns 4l .. 4l+3 of each 256-column span, and a wave-wide inclusive
        // scan gives each column's exclusive running count
        int* row = table + (size_t)key * stride;
        int run = 0;
        for (int c0 = 0; c0 < stride; c0 += kChunks * 256) {
            int4 v[kChunks];
#pragma unroll
            for (int j = 0; j < kChunks; ++j) {
                const int col = c0 + 256 * j + 4 * lane;
                v[j] = col < stride ? *reinterpret_cast<const int4*>(row + col) : make_int4(0, 0, 0, 0);
            }
#pragma unroll
            for (int j = 0; j < kChunks; ++j) {
                const int col = c0 + 256 * j + 4 * lane;
                // columns past the last routing block hold garbage
                const int x0 = col < nblk ? v[j].x : 0, x1 = col + 1 < nblk ? v[j].y : 0;
                const int x2 = col + 2 < nblk ? v[j].z : 0, x3 = col + 3 < nblk ? v[j].w : 0;
                const int mine = x0 + x1 + x2 + x3;
                int incl = mine;
#pragma unroll
                for (int o = 1; o < 64; o <<= 1) {
                    const int up = __shfl_up(incl, o);
                    if (lane >= o) incl += up;
                }
                const int ex = run + incl - mine;
                if (col < stride)
                    *reinterpret_cast<int4*>(row + col) = make_int4(ex, ex + x0, ex + x0 + x1, ex + x0 + x1 + x2);
                run += __shfl(incl, 63);
            }
        }
        // written through to the device-coherent level for the last block (route_last_block)
        if (lane == 0) __hip_atomic_store(totals + key, run, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    if (!route_last_block(&a.ctrl[kWordScanCount], gridDim.x, &s_flag)) return;
    if (tid < 3) s_cls[tid] = 0;
    const int res = (a.worklist && tid < N) ? a.resident_slot[tid] : -1;  // for the HIT work list
    const int tot = tid < NK ? __hip_atomic_load(totals + tid, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) : 0;
    if (tid < NK) s_tot[tid] = tot;
    // exclusive scan of the totals over keys
    int incl = tot;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
        const int up = __shfl_up(incl, o);
        if (lane >= o) incl += up;
    }
    if (lane == 63) s_wsum[w] = incl;
    __syncthreads();
    int start = incl - tot;
    for (int ww = 0; ww < w; ++ww) start += s_wsum[ww];
    if (tid < NK) {
        s_start[tid] = start;
        table[(size_t)NK * stride + tid] = start;
        const int c = tid / N, e = tid - c * N;
        a.offsets[c * (N + 1) + e] = start;
        if (e == N - 1) a.offsets[c * (N + 1) + N] = start + tot;
        if (tot) atomicAdd(&s_cls[c], tot);
    }
    if (tid < N) s_res[tid] = res;
    __syncthreads();
    if (tid < 3 && a.h_counts) a.h_counts[tid] = s_cls[tid];
    // work lists: wave c (< 3) ranks the non-empty buckets of class c by expert id
    if (a.worklist && w < 3) {
        const int c = w;
        int seen = 0;
        const unsigned long long lt = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
        for (int e0 = 0; e0 < N; e0 += 64) {
            const int e = e0 + lane;
            const int n = e < N ? s_tot[c * N + e] : 0;
            const unsigned long long mk = __ballot(n > 0);
            if (n > 0) {
                int slot = -1;
                if (c == SPICE_CLASS_HIT) {
                    slot = s_res[e];
                    if (slot < 0 || slot >= a.C) slot = -1;  // routing flagged it already
                }
                *reinterpret_cast<int4*>(a.worklist + 4 * (c * N + seen + __popcll(mk & lt))) =
                    make_int4(e, slot, s_start[c * N + e], n);
            }
            seen += __popcll(mk);
        }
        if (lane == 0) a.wl_count[c] = seen;
    }
    if (a.hx || a.h_idx || a.h_w || a.h_cls || a.h_ready) {
        __syncthreads();
        mirror_host<kScanThreads>(a);
    }
}

// Stable positions of the slots of tokens [16 b, 16 b + 16), by one wave: slot s with key k
// goes to start[k] + (slots of key k in earlier blocks) + (earlier slots of key k here).
__global__ __launch_bounds__(64) void bucket_scatter_kernel(RouteArgs a) {
    __shared__ int s_run[3 * SPICE_MAX_EXPERTS];
    const int lane = threadIdx.x;
    const int N = a.N, NK = 3 * N, S = a.T * a.K;
    const int stride = prefill_hist_stride(a.T);
    const int* table = reinterpret_cast<const int*>(a.logits_ws);
    for (int k = lane; k < NK; k += 64) s_run[k] = 0;
    __syncthreads();
    const int s0 = blockIdx.x * kPrefillTok * a.K, s1 = min(a.T, (blockIdx.x + 1) * kPrefillTok) * a.K;
    const unsigned long long lt = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
    for (int c0 = s0; c0 < s1; c0 += 64) {  // chunks in slot order: ranks stay stable
        const int s = c0 + lane;
        const int key = s < s1 ? route_slot_key(a, s) : -1;
        const bool valid = key >= 0;
        const int base = valid ? table[(size_t)NK * stride + key] + table[(size_t)key * stride + blockIdx.x] : 0;
        unsigned long long match = __ballot(valid);
#pragma unroll
        for (int b = 0; b < 10; ++b) {
            const bool bit = (key >> b) & 1;
            const unsigned long long bb = __ballot(valid && bit);
            match &= bit ? bb : ~bb;
        }
        if (valid) {
            const int pos = base + s_run[key] + __popcll(match & lt);
            if (pos >= 0 && pos < S) {
                a.perm[pos] = s;
                a.inv_perm[s] = pos;
            } else {
                atomicOr(&a.ctrl[kWordFlags], (uint32_t)SPICE_FLAG_BAD_INDEX);
            }
        }
        __syncthreads();  // every lane has read s_run before the chunk's counts are added
        if (valid && (match >> lane) == 1ull) s_run[key] += __popcll(match);
        __syncthreads();
    }
}

}  // namespace

hipError_t launch_route_bucket(const RouteArgs& a, hipStream_t s) {
    if (a.T <= kRouteTokenMaxT) {
        const int g = route_blocks_per_token(a.N + (a.w_sg ? 1 : 0), kLogitThreads);
        const dim3 grid((unsigned)(a.T * g));
        if (a.dtype == SPICE_BF16)
            hipLaunchKernelGGL(route_logits_kernel<SPICE_BF16>, grid, dim3(kLogitThreads), 0, s, a, g);
        else
            hipLaunchKernelGGL(route_logits_kernel<SPICE_F32>, grid, dim3(kLogitThreads), 0, s, a, g);
    } else {
        const unsigned nb = (unsigned)((a.T + kPrefillTok - 1) / kPrefillTok);
        if (a.dtype == SPICE_BF16)
            hipLaunchKernelGGL(route_prefill_kernel<SPICE_BF16>, dim3(nb), dim3(kPrefillThreads), 0, s, a);
        else
            hipLaunchKernelGGL(route_prefill_kernel<SPICE_F32>, dim3(nb), dim3(kPrefillThreads), 0, s, a);
        hipLaunchKernelGGL(bucket_scan_kernel, dim3((unsigned)((3 * a.N + kScanKeys - 1) / kScanKeys)), dim3(kScanThreads),
                           0, s, a);
        hipLaunchKernelGGL(bucket_scatter_kernel, dim3(nb), dim3(64), 0, s, a);
    }
    return hipGetLastError();
}

}  // namespace spice
