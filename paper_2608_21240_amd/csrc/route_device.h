// Device code of the routing step (Eq. 1; Sec. 2.1, 4.2, 4.3) shared by the routing
// kernels (route_bucket.hip) and the fused decode-layer kernels (layer_decode.hip).
// Everything has internal linkage: each source that includes it compiles its own copy.
//
//   route_logits_rows : fp64 logits of one token against a range of router rows, by one
//                       block (a token's rows are spread over route_blocks_per_token blocks);
//   block_topk   : softmax over the N logits, the K largest (descending, the lower id wins
//                  ties), gate, confidence and class of each of the K slots, by one block;
//   bucket_slots : stable counting sort of the T*K slots by key (class, expert), the
//                  per-class work lists and the class counts, by one block;
//   mirror_host  : the CPU path's host copies and, after them, the ready word, by one block.
// No step waits for another block: there are no cross-block counters or fences.
#pragma once

#include <float.h>
#include <limits.h>

#include <hip/hip_runtime.h>

#include "spice_internal.h"

namespace spice {
namespace {

// 16-byte chunks of the activation / router rows, widened to double (exactly).
template <int DT>
struct RouteElem;

template <>
struct RouteElem<SPICE_BF16> {
    static constexpr int V = 8;  // elements per 16-byte chunk
    static constexpr int es = 2;
    __device__ __forceinline__ static void widen(const uint4& q, double (&v)[8]) {
        const uint32_t w[4] = {q.x, q.y, q.z, q.w};
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            v[2 * i] = (double)__uint_as_float(w[i] << 16);
            v[2 * i + 1] = (double)__uint_as_float(w[i] & 0xFFFF0000u);
        }
    }
};

template <>
struct RouteElem<SPICE_F32> {
    static constexpr int V = 4;
    static constexpr int es = 4;
    __device__ __forceinline__ static void widen(const uint4& q, double (&v)[4]) {
        v[0] = (double)__uint_as_float(q.x);
        v[1] = (double)__uint_as_float(q.y);
        v[2] = (double)__uint_as_float(q.z);
        v[3] = (double)__uint_as_float(q.w);
    }
};

// A 16-byte load from an address that is always valid, replaced by zeros when !ok: the load
// itself is unconditional, so it stays one vector load with no branch around it.
__device__ __forceinline__ uint4 load16_or_zero(const char* p, bool ok) {
    const uint4 v = *reinterpret_cast<const uint4*>(p);
    const uint4 zero = {0u, 0u, 0u, 0u};
    return ok ? v : zero;
}

// Sum over the wave; every lane returns lane 0's value, so the association order is fixed.
__device__ __forceinline__ double route_wave_sum(double v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
    return __shfl(v, 0);
}

// Rows per routing block: each wave owns kRouteRowsPerWave router rows of one token (one:
// the most blocks per token, so the shortest chain to the token's last block).
constexpr int kRouteRowsPerWave = 1;

// Logits of token t for the rows [r0, r1) of the router, in fp64, by one block: row e < N is
// W_g[e] (z = x . W_g[e] + bias[e] to logits_ws and logits_out), row N is the shared
// block's gate row (sgate[t] = sigmoid(x . w_sg)).  bf16 x bf16 and fp32 x fp32 products
// are exact in fp64, so only the summation rounds.  Wave w owns the rows r0 + w + nw b
// (b < kRouteRowsPerWave); lane l sums the 16-byte chunks l, l + 64, ...; every load of a
// batch of kRounds such chunk rounds is issued before the first is used.
template <int DT>
__device__ void route_logits_rows(const RouteArgs& a, int t, int r0, int r1) {
    using E = RouteElem<DT>;
    constexpr int V = E::V, es = E::es;
    constexpr int kRows = kRouteRowsPerWave;
    constexpr int kRounds = DT == SPICE_BF16 ? 4 : 2;  // 64-chunk rounds per load batch
    const int N = a.N, d = a.d;
    const int lane = threadIdx.x & 63;
    const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int nw = blockDim.x >> 6;
    const int nchunk = d / V;
    const char* xb = static_cast<const char*>(a.x) + (size_t)t * d * es;
    for (int e0 = r0 + w; e0 < r1; e0 += nw * kRows) {
        const char* rb[kRows];
        bool live[kRows];  // uniform per wave
#pragma unroll
        for (int b = 0; b < kRows; ++b) {
            const int e = e0 + nw * b;
            live[b] = e < r1;
            // rows past r1 read router row 0 as zeros (their sums are dropped)
            rb[b] = (e < N) ? static_cast<const char*>(a.wg) + (size_t)e * d * es
                            : (e == N && live[b] ? static_cast<const char*>(a.w_sg) : static_cast<const char*>(a.wg));
        }
        double acc[kRows];
#pragma unroll
        for (int b = 0; b < kRows; ++b) acc[b] = 0.0;
        for (int c0 = 0; c0 < nchunk; c0 += 64 * kRounds) {
            uint4 xq[kRounds], wq[kRows][kRounds];
            // chunks past the row's end load its last chunk as zeros
#pragma unroll
            for (int r = 0; r < kRounds; ++r) {
                const int c = c0 + 64 * r + lane;
                xq[r] = load16_or_zero(xb + (size_t)min(c, nchunk - 1) * 16, c < nchunk);
            }
#pragma unroll
            for (int b = 0; b < kRows; ++b)
#pragma unroll
                for (int r = 0; r < kRounds; ++r) {
                    const int c = c0 + 64 * r + lane;
                    wq[b][r] = load16_or_zero(rb[b] + (size_t)min(c, nchunk - 1) * 16, live[b] && c < nchunk);
                }
            // every load of the batch is in flight before the first is used (left to itself the
            // scheduler interleaves them with the arithmetic: one memory round trip per round)
            __builtin_amdgcn_sched_barrier(0);
#pragma unroll
            for (int r = 0; r < kRounds; ++r) {
                double xd[V];
                E::widen(xq[r], xd);
#pragma unroll
                for (int b = 0; b < kRows; ++b) {
                    double wd[V];
                    E::widen(wq[b][r], wd);
#pragma unroll
                    for (int j = 0; j < V; ++j) acc[b] = fma(xd[j], wd[j], acc[b]);
                }
            }
        }
#pragma unroll
        for (int b = 0; b < kRows; ++b) {
            const int e = e0 + nw * b;
            const double sum = route_wave_sum(acc[b]);
            if (lane == 0 && e < r1) {
                if (e < N) {
                    const double z = sum + (a.bias ? (double)a.bias[e] : 0.0);
                    // written through to the device-coherent level: the token's last routing
                    // block reads it without an L2 write-back or invalidate (route_last_block)
                    __hip_atomic_store(reinterpret_cast<unsigned long long*>(a.logits_ws) + (size_t)t * N + e,
                                       (unsigned long long)__double_as_longlong(z), __ATOMIC_RELAXED,
                                       __HIP_MEMORY_SCOPE_AGENT);
                    if (a.logits_out) a.logits_out[(size_t)t * N + e] = z;
                } else {
                    a.sgate[t] = (float)(1.0 / (1.0 + exp(-sum)));
                }
            }
        }
    }
}

// Routing blocks per token: enough for every wave of an nt-thread block to own
// kRouteRowsPerWave rows (the router rows plus the gate row when there is one).
inline __host__ __device__ int route_blocks_per_token(int n_rows, int nt) {
    const int per = (nt / 64) * kRouteRowsPerWave;
    return (n_rows + per - 1) / per;
}

// Order-preserving map of a logit to an unsigned key: a larger double gives a larger key
// (after -0 is made +0, so equal doubles give equal keys).
__device__ __forceinline__ unsigned long long logit_key(double z) {
    const unsigned long long u = (unsigned long long)__double_as_longlong(z + 0.0);
    return (u >> 63) ? ~u : (u | 0x8000000000000000ull);
}

// LDS of block_topk.
struct TopkLds {
    double z[SPICE_MAX_EXPERTS];
    unsigned long long key[SPICE_MAX_EXPERTS];
    int res[SPICE_MAX_EXPERTS];
    int rank[SPICE_MAX_EXPERTS];
    int pick[64];
};

// The gates, confidence and classes of token t's K picks, by one wave: z = its N logits,
// res = resident_slot, pick = its experts in rank order (all in LDS).  Lane k < K returns
// its slot's bucket key (class * N + expert), the other lanes -1.  kPublish: the outputs
// and the key (control word kWordSlotKeys + slot) are written through to the
// device-coherent level, for a block of the same launch on another XCD.
template <bool kPublish = false>
__device__ int wave_topk_gates(const RouteArgs& a, int t, const double* z, const int* res, const int* pick,
                               int lane, float conf_in) {
    constexpr int kJ = SPICE_MAX_EXPERTS / 64;
    const int N = a.N, K = a.K;
    const double m = z[pick[0]];  // the largest logit
    double part = 0.0;
#pragma unroll
    for (int j = 0; j < kJ; ++j)
        if (lane + 64 * j < N) part += exp(z[lane + 64 * j] - m);
    const int my_e = lane < K ? pick[lane] : 0;
    const double my_ex = lane < K ? exp(z[my_e] - m) : 0.0;
    const double denom = route_wave_sum(part);
    double g = my_ex / denom;
    if (a.norm_topk) g = g / route_wave_sum(lane < K ? g : 0.0);
    const double gsum = (a.conf_mode == SPICE_CONF_GATE_RENORM) ? route_wave_sum(lane < K ? g : 0.0) : 1.0;
    if (lane < K) {
        const size_t s = (size_t)t * K + lane;
        float conf;
        if (a.conf_mode == SPICE_CONF_INPUT) conf = conf_in;
        else if (a.conf_mode == SPICE_CONF_GATE) conf = (float)g;
        else conf = (float)(g / gsum);
        int32_t slot = res[my_e];
        if (slot < -1 || slot >= a.C) {
            atomicOr(&a.ctrl[kWordFlags], (uint32_t)SPICE_FLAG_BAD_SLOT);
            slot = -1;
        }
        uint8_t cls;
        if (slot >= 0) cls = SPICE_CLASS_HIT;
        else if (conf < a.tau) cls = SPICE_CLASS_LORE;
        else cls = SPICE_CLASS_EXACT;
        if (kPublish) {
            __hip_atomic_store(a.topk_idx + s, my_e, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            __hip_atomic_store(a.topk_w + s, (float)g, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            __hip_atomic_store(a.slot_class + s, cls, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            __hip_atomic_store(a.ctrl + kWordSlotKeys + s, (uint32_t)(cls * N + my_e), __ATOMIC_RELAXED,
                               __HIP_MEMORY_SCOPE_AGENT);
        } else {
            a.topk_idx[s] = my_e;
            a.topk_w[s] = (float)g;
            a.slot_class[s] = cls;
        }
        return cls * N + my_e;
    }
    return -1;
}

// Top-K of token t from its N logits zg (fp64, bias included; global memory) by one block
// of NT threads (NT >= 64).  Expert e's rank is the number of experts that come before it
// (a larger logit, or an equal one with a smaller id); each wave counts a share of the
// experts ee against every e, and rank k < K makes e the k-th pick (descending, the lower id
// wins ties).  Then the softmax over all N, the gate of each pick (its probability,
// optionally renormalised over the K), its confidence and its class (kPublish: see
// wave_topk_gates).
template <int NT, bool kCoherent, bool kPublish = false>
__device__ void block_topk(const RouteArgs& a, int t, const double* zg, TopkLds& L) {
    constexpr int NW = NT / 64;
    constexpr int kJ = SPICE_MAX_EXPERTS / 64;
    const int N = a.N, K = a.K;
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    // everything this block reads from memory, in one round trip; kCoherent: the logits
    // were written by this launch's routing blocks and are read from the device-coherent
    // level (route_logits_rows stores them there)
    for (int e = tid; e < N; e += NT) {
        const double z =
            kCoherent ? __longlong_as_double((long long)__hip_atomic_load(
                            reinterpret_cast<const unsigned long long*>(zg) + e, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT))
                      : zg[e];
        L.z[e] = z;
        L.key[e] = logit_key(z);
        L.res[e] = a.resident_slot[e];
        L.rank[e] = 0;
    }
    const float conf_in = (a.conf_mode == SPICE_CONF_INPUT && tid < K) ? a.conf[(size_t)t * K + tid] : 0.f;
    __syncthreads();
    const int e_lo = w * N / NW, e_hi = (w + 1) * N / NW;  // this wave's share of the experts ee
#pragma unroll
    for (int j = 0; j < kJ; ++j) {
        if (64 * j >= N) break;  // uniform
        const int e = lane + 64 * j;
        const unsigned long long k = e < N ? L.key[e] : 0ull;
        int r = 0;
#pragma unroll 8  // several LDS reads in flight
        for (int ee = e_lo; ee < e_hi; ++ee) {
            const unsigned long long ke = L.key[ee];
            const unsigned gt = ke > k, eq = ke == k, lt = ee < e;
            r += (int)(gt | (eq & lt));
        }
        if (e < N && r) atomicAdd(&L.rank[e], r);
    }
    __syncthreads();
    for (int e = tid; e < N; e += NT)
        if (L.rank[e] < K) L.pick[L.rank[e]] = e;
    __syncthreads();
    if (w == 0) wave_topk_gates<kPublish>(a, t, L.z, L.res, L.pick, lane, conf_in);
}

// The last of a token's routing blocks to finish, found with an arrival counter.  A block's
// logits are agent-scope stores (written through to the device-coherent level), so ordering
// them before its increment needs only that every wave's stores have completed (s_waitcnt
// vmcnt(0)), not an L2 write-back; the last block reads them with agent-scope loads, not
// after an L2 invalidate.  Neither disturbs the tiles that stream beside the routing
// blocks.  The last block resets the counter, so it is zero again for the next call.
__device__ __forceinline__ bool route_last_block(uint32_t* counter, uint32_t n_blocks, int* s_flag) {
    __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0): this wave's stores have completed
    __syncthreads();
    if (threadIdx.x == 0) {
        const uint32_t prev = __hip_atomic_fetch_add(counter, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        const bool last = prev == n_blocks - 1;
        if (last) __hip_atomic_store(counter, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        *s_flag = last ? 1 : 0;
    }
    __syncthreads();
    return *s_flag != 0;
}

// Bucket key of slot s (class * N + expert), or -1 (flagged) for a value no gating step
// can produce.
__device__ __forceinline__ int route_slot_key(const RouteArgs& a, int s) {
    const int c = a.slot_class[s], e = a.topk_idx[s];
    if (c > SPICE_CLASS_EXACT || e < 0 || e >= a.N) {
        atomicOr(&a.ctrl[kWordFlags], (uint32_t)SPICE_FLAG_BAD_INDEX);
        return -1;
    }
    return c * a.N + e;
}

// Bucket key of slot s as the bucketing reads it: from the slot's top-K outputs, or, with
// kCoherentKeys, the key its routing block published in this launch (always valid).
template <bool kCoherentKeys>
__device__ __forceinline__ int bucket_key(const RouteArgs& a, int s) {
    if (kCoherentKeys)
        return (int)__hip_atomic_load(a.ctrl + kWordSlotKeys + s, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    return route_slot_key(a, s);
}

// LDS of bucket_slots for NT threads: two [NT/64][3N] int tables, the [3N] key totals, a
// few words and the key cache of `cache` slots (the keys of up to that many slots stay in
// LDS between the two passes; more slots are read twice).
constexpr size_t bucket_lds_bytes(int nt, int n_experts, int cache) {
    return (size_t)(2 * (nt / 64) + 1) * 3 * n_experts * sizeof(int) + 16 * sizeof(int) + (size_t)cache * sizeof(int);
}

// Stable counting sort of the S = T*K slots by key = class * N + expert, by one block of
// NT threads: per-wave histograms over contiguous slot ranges, one block-wide exclusive
// scan over (key, wave), then ranks of equal keys inside each 64-slot chunk by ballot
// matching.  Writes offsets, perm and inv_perm, the work lists (for class c, record j =
// {expert, pool slot (HIT) or -1, bucket start, bucket size} of the j-th non-empty bucket
// of that class in ascending expert order) with their counts, and the class counts to the
// host copy when a.h_counts is set.  kCoherentKeys: the keys come from bucket_key's
// published words (the routing ran in this launch).
template <int NT, int kKeyCache, bool kCoherentKeys = false>
__device__ void bucket_slots(const RouteArgs& a, int* lds) {
    constexpr int kW = NT / 64;
    constexpr int kBatch = 8;  // 64-slot chunks whose keys one round trip reads
    const int N = a.N, S = a.T * a.K, NK = 3 * N;
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    int* s_base = lds;                 // [kW][NK]
    int* s_run = lds + kW * NK;        // [kW][NK]
    int* s_tot = lds + 2 * kW * NK;    // [NK] slots per key
    int* s_misc = s_tot + NK;          // [0..3): class counts, [4..4+kW): wave sums
    int* s_keys = s_misc + 16;         // [S] when S <= kKeyCache
    const bool cached = S <= kKeyCache;
    for (int i = tid; i < kW * NK; i += NT) { s_base[i] = 0; s_run[i] = 0; }
    if (tid < 3) s_misc[tid] = 0;
    __syncthreads();
    const int per = (S + kW - 1) / kW;
    const int lo = min(S, w * per), hi = min(S, lo + per);
    for (int base = lo; base < hi; base += 64 * kBatch) {
        int key[kBatch];
#pragma unroll
        for (int u = 0; u < kBatch; ++u) {
            const int s = base + 64 * u + lane;
            key[u] = s < hi ? bucket_key<kCoherentKeys>(a, s) : -1;
        }
#pragma unroll
        for (int u = 0; u < kBatch; ++u) {
            const int s = base + 64 * u + lane;
            if (key[u] >= 0) atomicAdd(&s_base[w * NK + key[u]], 1);
            if (cached && s < hi) s_keys[s] = key[u];
        }
    }
    __syncthreads();

    // exclusive scan over keys in order; thread tid owns keys [kPer*tid, kPer*tid + kPer)
    constexpr int kPer = (3 * SPICE_MAX_EXPERTS + NT - 1) / NT;
    int tot = 0;
    int cnt[kPer];
#pragma unroll
    for (int q = 0; q < kPer; ++q) {
        const int key = kPer * tid + q;
        int v = 0;
        if (key < NK)
            for (int ww = 0; ww < kW; ++ww) v += s_base[ww * NK + key];
        cnt[q] = v;
        tot += v;
        if (key < NK) s_tot[key] = v;
        if (v) atomicAdd(&s_misc[key / N], v);
    }
    int incl = tot;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
        const int up = __shfl_up(incl, o);
        if (lane >= o) incl += up;
    }
    if (lane == 63) s_misc[4 + w] = incl;
    __syncthreads();
    int run = incl - tot;
    for (int ww = 0; ww < w; ++ww) run += s_misc[4 + ww];
#pragma unroll
    for (int q = 0; q < kPer; ++q) {
        const int key = kPer * tid + q;
        if (key < NK) {
            const int c = key / N, e = key - c * N;
            a.offsets[c * (N + 1) + e] = run;
            int acc = run;
            for (int ww = 0; ww < kW; ++ww) {
                const int h = s_base[ww * NK + key];
                s_base[ww * NK + key] = acc;
                acc += h;
            }
            if (e == N - 1) a.offsets[c * (N + 1) + N] = acc;
            run += cnt[q];
        }
    }
    __syncthreads();
    if (tid < 3 && a.h_counts) a.h_counts[tid] = s_misc[tid];

    // work lists: wave c (< 3) ranks the non-empty buckets of class c by expert id
    if (a.worklist && w < 3) {
        const int c = w;
        int seen = 0;
        const unsigned long long lt = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
        for (int e0 = 0; e0 < N; e0 += 64) {
            const int e = e0 + lane;
            int st = 0, n = 0;
            if (e < N) {
                st = s_base[c * N + e];  // wave 0's base of the key = the bucket start
                n = s_tot[c * N + e];
            }
            const unsigned long long m = __ballot(n > 0);
            if (n > 0) {
                int slot = -1;
                if (c == SPICE_CLASS_HIT) {
                    slot = a.resident_slot[e];
                    if (slot < 0 || slot >= a.C) slot = -1;  // routing flagged it already
                }
                *reinterpret_cast<int4*>(a.worklist + 4 * (c * N + seen + __popcll(m & lt))) = make_int4(e, slot, st, n);
            }
            seen += __popcll(m);
        }
        if (lane == 0) a.wl_count[c] = seen;
    }

    const unsigned long long lt_mask = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
    for (int base0 = lo; base0 < hi; base0 += 64 * kBatch) {
        int keys[kBatch];
#pragma unroll
        for (int u = 0; u < kBatch; ++u) {
            const int s = base0 + 64 * u + lane;
            keys[u] = s < hi ? (cached ? s_keys[s] : bucket_key<kCoherentKeys>(a, s)) : -1;
        }
#pragma unroll
        for (int u = 0; u < kBatch; ++u) {  // chunks in slot order: ranks stay stable
            const int s = base0 + 64 * u + lane;
            const int key = keys[u];
            const bool valid = key >= 0;
            unsigned long long match = __ballot(valid);
#pragma unroll
            for (int b = 0; b < 10; ++b) {
                const bool bit = (key >> b) & 1;
                const unsigned long long bb = __ballot(valid && bit);
                match &= bit ? bb : ~bb;
            }
            if (valid) {
                const int rank = __popcll(match & lt_mask);
                const int pos = s_base[w * NK + key] + s_run[w * NK + key] + rank;
                if (pos >= 0 && pos < S) {
                    a.perm[pos] = s;
                    a.inv_perm[s] = pos;
                } else {
                    atomicOr(&a.ctrl[kWordFlags], (uint32_t)SPICE_FLAG_BAD_INDEX);
                }
                if ((match >> lane) == 1ull) s_run[w * NK + key] += __popcll(match);
            }
        }
    }
}

// The CPU path's host copies (x, top-K, gates, classes; the class counts are written by
// bucket_slots) by one block, then the ready word: every wave waits for its own stores to
// complete (a system-scope fence) before thread 0 stores a.ready_value, so a host that
// sees the value also sees every copy.
template <int NT, bool kCoherent = false>
__device__ void mirror_host(const RouteArgs& a) {
    const int tid = threadIdx.x;
    const int es = a.dtype == SPICE_BF16 ? 2 : 4;
    if (a.hx) {
        const size_t nq = (size_t)a.T * a.d * es / 16;
        const uint4* src = static_cast<const uint4*>(a.x);
        uint4* dst = static_cast<uint4*>(a.hx);
        for (size_t i = tid; i < nq; i += NT) dst[i] = src[i];
    }
    const int S = a.T * a.K;
    for (int s = tid; s < S; s += NT) {
        if (kCoherent) {  // written in this launch by routing blocks on any XCD
            if (a.h_idx) a.h_idx[s] = __hip_atomic_load(a.topk_idx + s, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            if (a.h_w) a.h_w[s] = __hip_atomic_load(a.topk_w + s, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            if (a.h_cls) a.h_cls[s] = __hip_atomic_load(a.slot_class + s, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        } else {
            if (a.h_idx) a.h_idx[s] = a.topk_idx[s];
            if (a.h_w) a.h_w[s] = a.topk_w[s];
            if (a.h_cls) a.h_cls[s] = a.slot_class[s];
        }
    }
    if (a.h_ready) {
        __threadfence_system();
        __syncthreads();
        if (tid == 0) __hip_atomic_store(a.h_ready, a.ready_value, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_SYSTEM);
    }
}

}  // namespace
}  // namespace spice
