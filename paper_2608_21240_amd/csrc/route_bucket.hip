// Router logits, softmax top-K gating, per-slot classification and (class, expert)
// bucketing (Eq. 1; Sec. 2.1, 4.2, 4.3).  No block waits for another block.
//
// T <= kRouteTokenMaxT (decode), two launches:
//   1. route_logits_kernel: a token's router rows are spread over a few blocks (4 rows per
//      wave), each summing its logits in fp64; the last of the token's blocks to finish (an
//      arrival counter per token) takes the token's top-K, gates, confidence and classes;
//   2. route_bucket_kernel: one block sorts the T*K slots by (class, expert), writes the
//      work lists and, when asked, the CPU path's host copies and their ready word.
// Larger T (prefill): the logits as fp64 MFMA tiles of 16 experts x 16 tokens, a block per
// token for the top-K, then the same bucketing block.
//
// bf16 x bf16 and fp32 x fp32 products are exact in fp64, so on every path only the
// summation order of the logits differs from a plain loop.
#include <hip/hip_runtime.h>

#include "route_device.h"

namespace spice {
namespace {

constexpr int kLogitThreads = 256;   // routing logits: 4 waves, 4 router rows each
constexpr int kBucketThreads = 512;  // bucketing block
constexpr int kMfmaThreads = 256;    // fp64 MFMA logits: 4 waves, one 16-token tile per block
constexpr int kBucketCache = 2048;   // slots whose keys stay in LDS while bucketing (LDS <= 64 KiB at N = 256)

typedef double f64x4_t __attribute__((ext_vector_type(4)));

template <int DT>
__global__ __launch_bounds__(kLogitThreads) void route_logits_kernel(RouteArgs a, int g_per_tok) {
    __shared__ TopkLds lds;
    __shared__ int s_flag;
    const int t = blockIdx.x / g_per_tok, g = blockIdx.x % g_per_tok;
    const int rows = (kLogitThreads / 64) * kRouteRowsPerWave;
    const int n_rows = a.N + (a.w_sg ? 1 : 0);
    route_logits_rows<DT>(a, t, g * rows, min(n_rows, (g + 1) * rows));
    if (!route_last_block(&a.ctrl[kWordTokCount + t], g_per_tok, &s_flag)) return;
    block_topk<kLogitThreads, true>(a, t, a.logits_ws + (size_t)t * a.N, lds);
}

__global__ __launch_bounds__(kBucketThreads) void route_bucket_kernel(RouteArgs a) {
    extern __shared__ __align__(16) int s_lds[];
    bucket_slots<kBucketThreads, kBucketCache>(a, s_lds);
    if (a.hx || a.h_idx || a.h_w || a.h_cls || a.h_ready) mirror_host<kBucketThreads>(a);
}

// Large T: z = x W_g^T (+ bias) with v_mfma_f64_16x16x4f64.  Block = 16 tokens; wave w
// takes the 16-expert tiles w, w + 4, ...  A 16-byte load gives each lane 8 (bf16) or 4
// (fp32) consecutive k of one row: lane (m = lane % 16, q = lane / 16) holds row m's
// elements q*V .. q*V + V-1 of a 4V-wide k chunk, and MFMA step u takes element u of
// every lane, so the 4 k of step u are {u, V + u, 2V + u, 3V + u} for both operands and
// each chunk's products are all summed once.  Rows beyond N and tokens beyond T load
// zero and their outputs are dropped; d is a multiple of V (the ABI's alignment).
template <int DT>
__global__ __launch_bounds__(kMfmaThreads) void route_logits_mfma_kernel(RouteArgs a) {
    using E = RouteElem<DT>;
    constexpr int V = E::V, es = E::es;
    const int lane = threadIdx.x & 63, m = lane & 15, q = lane >> 4;
    const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int t0 = blockIdx.x * 16;
    const int tok = t0 + m;
    const bool tok_ok = tok < a.T;
    const char* xr = static_cast<const char*>(a.x) + (size_t)(tok_ok ? tok : 0) * a.d * es;
    const int ntile = (a.N + 15) / 16;
    for (int tile = w; tile < ntile; tile += kMfmaThreads / 64) {
        const int e = tile * 16 + m;
        const bool e_ok = e < a.N;
        const char* wr = static_cast<const char*>(a.wg) + (size_t)(e_ok ? e : 0) * a.d * es;
        f64x4_t acc0 = {0.0, 0.0, 0.0, 0.0}, acc1 = {0.0, 0.0, 0.0, 0.0};
        for (int k0 = 0; k0 < a.d; k0 += 8 * V) {  // two 4V-wide chunks per pass
            uint4 xq[2], wq[2];
#pragma unroll
            for (int c = 0; c < 2; ++c) {
                const int k = k0 + c * 4 * V + q * V;
                const bool in = k < a.d;
                const size_t kk = (size_t)(in ? k : 0) * es;  // out-of-range chunks load chunk 0 as zeros
                xq[c] = load16_or_zero(xr + kk, in && tok_ok);
                wq[c] = load16_or_zero(wr + kk, in && e_ok);
            }
#pragma unroll
            for (int c = 0; c < 2; ++c) {
                double xd[V], wd[V];
                E::widen(xq[c], xd);
                E::widen(wq[c], wd);
#pragma unroll
                for (int u = 0; u < V; u += 2) {  // two accumulators: no MFMA waits on the one before
                    acc0 = __builtin_amdgcn_mfma_f64_16x16x4f64(wd[u], xd[u], acc0, 0, 0, 0);
                    acc1 = __builtin_amdgcn_mfma_f64_16x16x4f64(wd[u + 1], xd[u + 1], acc1, 0, 0, 0);
                }
            }
        }
        // the f64 16x16x4 result layout: acc[v] = D[row 4v + q][column m], i.e. the logit of
        // expert tile*16 + 4v + q for token t0 + m (a probe of the instruction fixed this)
#pragma unroll
        for (int v = 0; v < 4; ++v) {
            const int ee = tile * 16 + 4 * v + q;
            if (ee < a.N && tok_ok) {
                const double z = (acc0[v] + acc1[v]) + (a.bias ? (double)a.bias[ee] : 0.0);
                a.logits_ws[(size_t)tok * a.N + ee] = z;
                if (a.logits_out) a.logits_out[(size_t)tok * a.N + ee] = z;
            }
        }
    }
}

// Top-K of the logits in the workspace: one block per token.
__global__ __launch_bounds__(kLogitThreads) void route_topk_kernel(RouteArgs a) {
    __shared__ TopkLds lds;
    block_topk<kLogitThreads, false>(a, blockIdx.x, a.logits_ws + (size_t)blockIdx.x * a.N, lds);
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
        const unsigned nb = (unsigned)((a.T + 15) / 16);
        if (a.dtype == SPICE_BF16)
            hipLaunchKernelGGL(route_logits_mfma_kernel<SPICE_BF16>, dim3(nb), dim3(kMfmaThreads), 0, s, a);
        else
            hipLaunchKernelGGL(route_logits_mfma_kernel<SPICE_F32>, dim3(nb), dim3(kMfmaThreads), 0, s, a);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
        hipLaunchKernelGGL(route_topk_kernel, dim3((unsigned)a.T), dim3(kLogitThreads), 0, s, a);
    }
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(route_bucket_kernel, dim3(1), dim3(kBucketThreads),
                       bucket_lds_bytes(kBucketThreads, a.N, kBucketCache), s, a);
    return hipGetLastError();
}

}  // namespace spice
