// Router logits, softmax top-K gating, per-slot classification and (class, expert)
// bucketing in one launch (Eq. 1; Sec. 2.1, 4.2, 4.3).
//
// Grid: (ceil(N/8) expert groups) x (ceil(T/TT) token tiles), 512 threads (8 waves).
//   1. every block: fp64 logits of TT tokens x 8 experts.  The block stages its
//      TT token rows in LDS; each wave owns one expert row and loads all of its
//      16-byte chunks at once, so the step costs about one memory round trip.
//      bf16 x bf16 and fp32 x fp32 products are exact in fp64, so only the
//      summation rounds;
//   2. the last block of a token tile to finish: softmax and top-K of its tokens
//      (one wave per token, wave-wide argmax with the lower id winning ties),
//      gate scores, confidence and class;
//   3. the last token tile to finish: stable counting sort of all T*K slots by
//      key (class, expert) with per-wave histograms, a block scan, and ballot
//      matching to rank equal keys inside each 64-slot chunk.
// Optional host copies for the CPU path (x, top-K, gates, classes, class counts)
// are stored straight into the caller's pinned host memory along the way.
// "Last block" is decided with an agent-scope atomic counter in the workspace
// control region after a device fence; the last block resets the counter.
#include <float.h>
#include <limits.h>

#include <hip/hip_runtime.h>

#include "spice_internal.h"

namespace spice {
namespace {

constexpr int kThreads = 512;
constexpr int kWaves = kThreads / 64;
constexpr int kMaxKeys = 3 * SPICE_MAX_EXPERTS;
constexpr int kKeysPerThread = (kMaxKeys + kThreads - 1) / kThreads;
constexpr int kMaxRowChunks = 16;  // 16-byte chunks of a router row per lane (d*es <= 16 KiB)
constexpr int kBatch = 8;          // 64-slot chunks whose keys are read per round trip when bucketing
constexpr int kRouteFusedMaxTiles = 16;  // token tiles up to which the three steps share one launch

__device__ __forceinline__ float bf16_bits_to_float(uint32_t bits16) {
    return __uint_as_float(bits16 << 16);
}

// 16-byte chunk of `n` elements widened to double.
template <int DT>
struct Chunk;

template <>
struct Chunk<SPICE_BF16> {
    static constexpr int n = 8;
    __device__ __forceinline__ static void widen(uint4 q, double* v) {
        const uint32_t w[4] = {q.x, q.y, q.z, q.w};
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            v[2 * i] = (double)bf16_bits_to_float(w[i] & 0xFFFFu);
            v[2 * i + 1] = (double)bf16_bits_to_float(w[i] >> 16);
        }
    }
    __device__ __forceinline__ static void load(const void* base, size_t elem, double* v) {
        const uint4 q = *reinterpret_cast<const uint4*>(static_cast<const uint16_t*>(base) + elem);
        const uint32_t w[4] = {q.x, q.y, q.z, q.w};
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            v[2 * i] = (double)bf16_bits_to_float(w[i] & 0xFFFFu);
            v[2 * i + 1] = (double)bf16_bits_to_float(w[i] >> 16);
        }
    }
};

template <>
struct Chunk<SPICE_F32> {
    static constexpr int n = 4;
    __device__ __forceinline__ static void widen(uint4 q, double* v) {
        v[0] = __uint_as_float(q.x); v[1] = __uint_as_float(q.y);
        v[2] = __uint_as_float(q.z); v[3] = __uint_as_float(q.w);
    }
    __device__ __forceinline__ static void load(const void* base, size_t elem, double* v) {
        const float4 q = *reinterpret_cast<const float4*>(static_cast<const float*>(base) + elem);
        v[0] = q.x; v[1] = q.y; v[2] = q.z; v[3] = q.w;
    }
};

__device__ __forceinline__ double wave_sum_lane0(double v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
    return __shfl(v, 0);  // every lane takes lane 0's association order
}

// The block barrier orders every thread's stores before thread 0's device-scope
// release fence (one L2 write-back per block, not per wave); the last block's
// thread 0 takes the acquire fence before the barrier releases the others.
__device__ __forceinline__ bool is_last_arrival(uint32_t* counter, uint32_t n_expected, int* s_flag) {
    __syncthreads();
    if (threadIdx.x == 0) {
        __threadfence();
        uint32_t prev = atomicAdd(counter, 1u);
        const bool last = (prev == n_expected - 1);
        if (last) {
            atomicExch(counter, 0u);
            __threadfence();
        }
        *s_flag = last ? 1 : 0;
    }
    __syncthreads();
    return *s_flag != 0;
}

// Step 2 for one token: wave-wide softmax over N logits, K rounds of argmax.
__device__ void topk_one_token(const RouteArgs& a, int t, int lane) {
    const int N = a.N, K = a.K;
    constexpr int kJ = SPICE_MAX_EXPERTS / 64;
    double z[kJ];
    bool taken[kJ];
    double m = -DBL_MAX;
#pragma unroll
    for (int j = 0; j < kJ; ++j) {
        const int e = lane + 64 * j;
        z[j] = (e < N) ? a.logits_ws[(size_t)t * N + e] : -DBL_MAX;
        taken[j] = (e >= N);
        if (e < N) m = fmax(m, z[j]);
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) m = fmax(m, __shfl_xor(m, o));
    double part = 0.0;
#pragma unroll
    for (int j = 0; j < kJ; ++j)
        if (lane + 64 * j < N) part += exp(z[j] - m);
    const double denom = wave_sum_lane0(part);

    int my_e = -1;
    double my_z = 0.0;
    for (int k = 0; k < K; ++k) {
        double bv = -DBL_MAX;
        int bi = INT_MAX;
#pragma unroll
        for (int j = 0; j < kJ; ++j) {
            const int e = lane + 64 * j;
            if (!taken[j] && (bi == INT_MAX || z[j] > bv)) { bv = z[j]; bi = e; }
        }
#pragma unroll
        for (int o = 32; o > 0; o >>= 1) {
            const double ov = __shfl_xor(bv, o);
            const int oi = __shfl_xor(bi, o);
            if (oi != INT_MAX && (bi == INT_MAX || ov > bv || (ov == bv && oi < bi))) { bv = ov; bi = oi; }
        }
        if (bi != INT_MAX && (bi & 63) == lane) taken[bi >> 6] = true;
        if (lane == k) { my_e = bi; my_z = bv; }
    }

    double g = 0.0;
    if (lane < K) g = exp(my_z - m) / denom;
    if (a.norm_topk) g = g / wave_sum_lane0(lane < K ? g : 0.0);
    const double gsum = (a.conf_mode == SPICE_CONF_GATE_RENORM) ? wave_sum_lane0(lane < K ? g : 0.0) : 1.0;
    if (lane < K) {
        const size_t s = (size_t)t * K + lane;
        float conf;
        if (a.conf_mode == SPICE_CONF_INPUT) conf = a.conf[s];
        else if (a.conf_mode == SPICE_CONF_GATE) conf = (float)g;
        else conf = (float)(g / gsum);
        int32_t slot = -1;
        if (my_e >= 0 && my_e < N) slot = a.resident_slot[my_e];
        if (slot < -1 || slot >= a.C) {
            atomicOr(&a.ctrl[kWordFlags], (uint32_t)SPICE_FLAG_BAD_SLOT);
            slot = -1;
        }
        uint8_t cls;
        if (slot >= 0) cls = SPICE_CLASS_HIT;
        else if (conf < a.tau) cls = SPICE_CLASS_LORE;
        else cls = SPICE_CLASS_EXACT;
        a.topk_idx[s] = my_e;
        a.topk_w[s] = (float)g;
        a.slot_class[s] = cls;
        if (a.h_idx) a.h_idx[s] = my_e;
        if (a.h_w) a.h_w[s] = (float)g;
        if (a.h_cls) a.h_cls[s] = cls;
    }
}

// Bucket key of slot s, or -1 (flagged) for a value no gating step can produce.
__device__ __forceinline__ int slot_key(const RouteArgs& a, int s) {
    const int c = a.slot_class[s], e = a.topk_idx[s];
    if (c > SPICE_CLASS_EXACT || e < 0 || e >= a.N) {
        atomicOr(&a.ctrl[kWordFlags], (uint32_t)SPICE_FLAG_BAD_INDEX);
        return -1;
    }
    return c * a.N + e;
}

// Step 3: stable counting sort of the T*K slots by key = class*N + expert.
__device__ void bucket_all(const RouteArgs& a, int* s_base, int* s_run, int* s_wsum, int* s_ccount) {
    const int N = a.N, S = a.T * a.K, NK = 3 * N;
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    for (int i = tid; i < kWaves * NK; i += kThreads) { s_base[i] = 0; s_run[i] = 0; }
    if (tid < 3) s_ccount[tid] = 0;
    __syncthreads();
    const int per = (S + kWaves - 1) / kWaves;
    const int lo = min(S, w * per), hi = min(S, lo + per);
    // keys are read kBatch chunks of 64 at a time, so that one memory round trip
    // serves kBatch chunks (large batches of tokens have thousands of slots)
    for (int base = lo; base < hi; base += 64 * kBatch) {
        int key[kBatch];
#pragma unroll
        for (int u = 0; u < kBatch; ++u) {
            const int s = base + 64 * u + lane;
            key[u] = s < hi ? slot_key(a, s) : -1;
        }
#pragma unroll
        for (int u = 0; u < kBatch; ++u)
            if (key[u] >= 0) atomicAdd(&s_base[w * NK + key[u]], 1);
    }
    __syncthreads();

    // Block-wide exclusive scan over keys; thread `tid` owns kKeysPerThread consecutive keys.
    int tot = 0;
    int cnt[kKeysPerThread];
#pragma unroll
    for (int q = 0; q < kKeysPerThread; ++q) {
        const int key = kKeysPerThread * tid + q;
        int v = 0;
        if (key < NK)
            for (int ww = 0; ww < kWaves; ++ww) v += s_base[ww * NK + key];
        cnt[q] = v;
        tot += v;
        if (v) atomicAdd(&s_ccount[key / N], v);
    }
    int incl = tot;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
        const int up = __shfl_up(incl, o);
        if (lane >= o) incl += up;
    }
    if (lane == 63) s_wsum[w] = incl;
    __syncthreads();
    int run = incl - tot;
    for (int ww = 0; ww < w; ++ww) run += s_wsum[ww];
#pragma unroll
    for (int q = 0; q < kKeysPerThread; ++q) {
        const int key = kKeysPerThread * tid + q;
        if (key < NK) {
            const int c = key / N, e = key - c * N;
            a.offsets[c * (N + 1) + e] = run;
            int acc = run;
            for (int ww = 0; ww < kWaves; ++ww) {
                const int h = s_base[ww * NK + key];
                s_base[ww * NK + key] = acc;
                acc += h;
            }
            if (e == N - 1) a.offsets[c * (N + 1) + N] = acc;
            run += cnt[q];
        }
    }
    __syncthreads();
    if (a.h_counts && tid < 3) a.h_counts[tid] = s_ccount[tid];

    const unsigned long long lt_mask = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
    for (int base0 = lo; base0 < hi; base0 += 64 * kBatch) {
      int keys[kBatch];
#pragma unroll
      for (int u = 0; u < kBatch; ++u) {
          const int s = base0 + 64 * u + lane;
          keys[u] = s < hi ? slot_key(a, s) : -1;
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

// kFused: one launch, later steps run in the last block to arrive (small T);
// kLogitsOnly: step 1 only (large T: steps 2 and 3 are launches of their own, so no
// block pays a device-scope fence; thousands of such fences cost more than launches).
enum : int { kFused = 0, kLogitsOnly = 1 };

template <int DT, int kMode>
__global__ __launch_bounds__(kThreads) void route_bucket_kernel(RouteArgs a, int tt_tok) {
    extern __shared__ __align__(16) unsigned char s_dyn[];
    __shared__ int s_wsum[kWaves];
    __shared__ int s_ccount[3];
    __shared__ int s_flag;
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const int t0 = blockIdx.y * tt_tok;
    const int nt = min(tt_tok, a.T - t0);
    constexpr int V = Chunk<DT>::n;
    constexpr int es = (DT == SPICE_BF16) ? 2 : 4;
    const int nchunk = a.d / V;  // 16-byte chunks per row

    // 1a. this wave's router row: every chunk it owns, loaded at once
    const int e = blockIdx.x * kRouteExp + w;
    uint4 wrow[kMaxRowChunks];
    if (e < a.N) {
#pragma unroll
        for (int i = 0; i < kMaxRowChunks; ++i) {
            const int c = lane + 64 * i;
            if (c < nchunk)
                wrow[i] = *reinterpret_cast<const uint4*>(static_cast<const char*>(a.wg) +
                                                          ((size_t)e * a.d + (size_t)c * V) * es);
        }
    }
    // 1b. the block's token rows into LDS
    uint4* s_x = reinterpret_cast<uint4*>(s_dyn);
    const bool mirror_x = a.hx != nullptr && blockIdx.x == 0;  // one expert group copies x to the host
    for (int i = threadIdx.x; i < nt * nchunk; i += kThreads) {
        const int tok = i / nchunk, c = i - tok * nchunk;
        const size_t off = ((size_t)(t0 + tok) * a.d + (size_t)c * V) * es;
        const uint4 q = *reinterpret_cast<const uint4*>(static_cast<const char*>(a.x) + off);
        s_x[i] = q;
        if (mirror_x) *reinterpret_cast<uint4*>(static_cast<char*>(a.hx) + off) = q;
    }
    __syncthreads();
    if (e < a.N) {
        double acc[kRouteTok];
#pragma unroll
        for (int i = 0; i < kRouteTok; ++i) acc[i] = 0.0;
#pragma unroll
        for (int i = 0; i < kMaxRowChunks; ++i) {
            const int c = lane + 64 * i;
            if (c < nchunk) {
                double wv[V];
                Chunk<DT>::widen(wrow[i], wv);
#pragma unroll
                for (int tok = 0; tok < kRouteTok; ++tok) {
                    if (tok < nt) {
                        double xv[V];
                        Chunk<DT>::widen(s_x[tok * nchunk + c], xv);
#pragma unroll
                        for (int j = 0; j < V; ++j) acc[tok] += xv[j] * wv[j];
                    }
                }
            }
        }
        const double b = a.bias ? (double)a.bias[e] : 0.0;
#pragma unroll
        for (int tok = 0; tok < kRouteTok; ++tok) {
            if (tok < nt) {
                const double zi = wave_sum_lane0(acc[tok]) + b;
                if (lane == 0) {
                    a.logits_ws[(size_t)(t0 + tok) * a.N + e] = zi;
                    if (a.logits_out) a.logits_out[(size_t)(t0 + tok) * a.N + e] = zi;
                }
            }
        }
    }

    if (kMode == kLogitsOnly) return;
    // 2. the last expert group of this token tile runs the gating (one wave per token)
    if (!is_last_arrival(&a.ctrl[kWordTileCounters + blockIdx.y], gridDim.x, &s_flag)) return;
    for (int i = w; i < nt; i += kWaves) topk_one_token(a, t0 + i, lane);

    // 3. the last token tile buckets every slot
    if (!is_last_arrival(&a.ctrl[kWordRouteDone], gridDim.y, &s_flag)) return;
    int* s_base = reinterpret_cast<int*>(s_dyn);
    bucket_all(a, s_base, s_base + kWaves * kMaxKeys, s_wsum, s_ccount);
}

// Step 2 on its own: one wave per token.
__global__ __launch_bounds__(kThreads) void route_topk_kernel(RouteArgs a) {
    const int t = blockIdx.x * kWaves + (threadIdx.x >> 6);
    if (t < a.T) topk_one_token(a, t, threadIdx.x & 63);
}

// Step 3 on its own: one block.
__global__ __launch_bounds__(kThreads) void route_sort_kernel(RouteArgs a) {
    extern __shared__ __align__(16) unsigned char s_dyn[];
    __shared__ int s_wsum[kWaves];
    __shared__ int s_ccount[3];
    int* s_base = reinterpret_cast<int*>(s_dyn);
    bucket_all(a, s_base, s_base + kWaves * kMaxKeys, s_wsum, s_ccount);
}

}  // namespace

hipError_t launch_route_bucket(const RouteArgs& a, hipStream_t s) {
    const int es = a.dtype == SPICE_BF16 ? 2 : 4;
    const int tt = route_tokens_per_block(a.d, es);
    const size_t x_lds = (size_t)tt * a.d * es;
    const size_t bucket_lds = (size_t)2 * kWaves * kMaxKeys * sizeof(int);
    const size_t lds = x_lds > bucket_lds ? x_lds : bucket_lds;
    dim3 grid((a.N + kRouteExp - 1) / kRouteExp, (a.T + tt - 1) / tt);
    if ((int)grid.y <= kRouteFusedMaxTiles) {
        if (a.dtype == SPICE_BF16)
            hipLaunchKernelGGL((route_bucket_kernel<SPICE_BF16, kFused>), grid, dim3(kThreads), lds, s, a, tt);
        else
            hipLaunchKernelGGL((route_bucket_kernel<SPICE_F32, kFused>), grid, dim3(kThreads), lds, s, a, tt);
        return hipGetLastError();
    }
    if (a.dtype == SPICE_BF16)
        hipLaunchKernelGGL((route_bucket_kernel<SPICE_BF16, kLogitsOnly>), grid, dim3(kThreads), x_lds, s, a, tt);
    else
        hipLaunchKernelGGL((route_bucket_kernel<SPICE_F32, kLogitsOnly>), grid, dim3(kThreads), x_lds, s, a, tt);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(route_topk_kernel, dim3((a.T + kWaves - 1) / kWaves), dim3(kThreads), 0, s, a);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(route_sort_kernel, dim3(1), dim3(kThreads), bucket_lds, s, a);
    return hipGetLastError();
}

}  // namespace spice
