// One depth of the speculative-prefetch draft rollout (Sec. 4.1, Alg. 1 steps 2-4),
// after the routing and the surrogate FFN of that depth have run:
//   the router's top-K of each running token is its prediction (Eq. 2) and is enqueued;
//   its confidence is the top-K probability mass (Eq. 5);
//   a token at depth >= l_min whose confidence is below tau stops (its prediction stays);
//   the others move their draft state one layer on,
//     h <- Attn(h) + sum_k pi_k (S(h) + B_k A_k h),  Ẽ_k = S + B_k A_k (Eq. 11),
//   with the target layer's attention replaced by the identity.
// S(h) comes from the shared block's FFN (y_shared) and B_k A_k h from the LoRE FFN
// of the slots (y_slots at the slot's bucket position); the routing of the depth put
// every slot in the LoRE class, so every predicted expert has its surrogate row.
//
// One block per token.  Thread 0 reads the K predictions, writes the queue entries and
// takes the halting decision; then every thread updates (or copies) 4 features at a time
// of the token's draft state in fp32 and stores it in the activation dtype (bf16 with
// round-to-nearest-even).
#include <hip/hip_runtime.h>

#include "spice_internal.h"

namespace spice {
namespace {

constexpr int kThreads = 256;
constexpr int kMaxK = 64;

__device__ __forceinline__ uint32_t bf16_rne(float f) {
    const uint32_t u = __float_as_uint(f);
    if ((u & 0x7FFFFFFFu) > 0x7F800000u) return 0x7FC0u;  // NaN stays NaN
    return (u + 0x7FFFu + ((u >> 16) & 1u)) >> 16;
}

template <int DT>
__device__ __forceinline__ float4 load4(const void* p, size_t i) {
    if constexpr (DT == SPICE_BF16) {
        const uint2 v = *reinterpret_cast<const uint2*>(static_cast<const uint16_t*>(p) + i);
        return make_float4(__uint_as_float(v.x << 16), __uint_as_float(v.x & 0xFFFF0000u),
                           __uint_as_float(v.y << 16), __uint_as_float(v.y & 0xFFFF0000u));
    } else {
        return *reinterpret_cast<const float4*>(static_cast<const float*>(p) + i);
    }
}

template <int DT>
__device__ __forceinline__ void store4(void* p, size_t i, float4 v) {
    if constexpr (DT == SPICE_BF16) {
        uint2 o;
        o.x = bf16_rne(v.x) | (bf16_rne(v.y) << 16);
        o.y = bf16_rne(v.z) | (bf16_rne(v.w) << 16);
        *reinterpret_cast<uint2*>(static_cast<uint16_t*>(p) + i) = o;
    } else {
        *reinterpret_cast<float4*>(static_cast<float*>(p) + i) = v;
    }
}

template <int DT>
__global__ __launch_bounds__(kThreads) void spec_update_kernel(SpecArgs a) {
    __shared__ int s_update;
    __shared__ float s_w[kMaxK];
    __shared__ int s_pos[kMaxK];
    const int t = blockIdx.x, K = a.K;
    if (threadIdx.x == 0) {
        int update = 0;
        const size_t r0 = (size_t)t * K;
        if (a.halted[t]) {
            for (int k = 0; k < K; ++k) {
                a.pred_idx[r0 + k] = -1;
                a.pred_prob[r0 + k] = 0.f;
                if (a.h_pred_idx) a.h_pred_idx[r0 + k] = -1;
                if (a.h_pred_prob) a.h_pred_prob[r0 + k] = 0.f;
            }
            a.conf[t] = __builtin_nanf("");
            if (a.h_conf) a.h_conf[t] = __builtin_nanf("");
        } else {
            double c = 0.0;
            bool ok = true;
            for (int k = 0; k < K; ++k) {
                const int e = a.topk_idx[r0 + k];
                const float w = a.topk_w[r0 + k];
                a.pred_idx[r0 + k] = e;
                a.pred_prob[r0 + k] = w;
                if (a.h_pred_idx) a.h_pred_idx[r0 + k] = e;
                if (a.h_pred_prob) a.h_pred_prob[r0 + k] = w;
                c += (double)w;
                const int pos = a.inv_perm[r0 + k];
                if (pos < 0 || pos >= a.T * K) ok = false;
                s_w[k] = w;
                s_pos[k] = pos;
            }
            a.conf[t] = (float)c;
            if (a.h_conf) a.h_conf[t] = (float)c;
            if (!ok) atomicOr(&a.ctrl[kWordFlags], (uint32_t)SPICE_FLAG_BAD_INDEX);
            if (a.delta >= a.l_min && c < (double)a.tau)
                a.halted[t] = 1;  // the prediction stays queued; no deeper speculation
            else if (!a.last && ok)
                update = 1;
        }
        s_update = update;
    }
    __syncthreads();
    const size_t row = (size_t)t * a.d;
    if (s_update) {
        for (int i = threadIdx.x * 4; i < a.d; i += kThreads * 4) {
            const float4 h = load4<DT>(a.h_in, row + i);
            const float4 s = *reinterpret_cast<const float4*>(a.y_shared + row + i);
            float4 acc = h;
            for (int k = 0; k < K; ++k) {
                float4 y = s;
                if (a.lore) {
                    const float4 dl = *reinterpret_cast<const float4*>(a.y_slots + (size_t)s_pos[k] * a.d + i);
                    y.x += dl.x; y.y += dl.y; y.z += dl.z; y.w += dl.w;
                }
                const float w = s_w[k];
                acc.x += w * y.x; acc.y += w * y.y; acc.z += w * y.z; acc.w += w * y.w;
            }
            store4<DT>(a.h_out, row + i, acc);
        }
    } else if (a.h_out != a.h_in) {
        for (int i = threadIdx.x * 4; i < a.d; i += kThreads * 4) store4<DT>(a.h_out, row + i, load4<DT>(a.h_in, row + i));
    }
}

}  // namespace

hipError_t launch_spec_update(const SpecArgs& a, hipStream_t s) {
    if (a.T == 0) return hipSuccess;
    if (a.dtype == SPICE_BF16)
        hipLaunchKernelGGL(spec_update_kernel<SPICE_BF16>, dim3((unsigned)a.T), dim3(kThreads), 0, s, a);
    else
        hipLaunchKernelGGL(spec_update_kernel<SPICE_F32>, dim3((unsigned)a.T), dim3(kThreads), 0, s, a);
    return hipGetLastError();
}

}  // namespace spice
