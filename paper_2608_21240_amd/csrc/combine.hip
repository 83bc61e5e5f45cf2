// Gate-weighted combine (Sec. 2.1) with LoRE substitution (Eq. 11) and the merge
// of the CPU exact residual (Sec. 4.3), plus a small fill kernel.
//
// One thread per 4 consecutive hidden features of one token; grid (d/1024, T).
// out = (1 + sum_{LORE} g) * S(x) + sum_{HIT,LORE,EXACT_GPU} g * y_slots[inv_perm[slot]] + resid,
// summed over the slots in order k = 0..K-1.
#include <hip/hip_runtime.h>

#include "spice_internal.h"

namespace spice {
namespace {

typedef float f32x4_t __attribute__((ext_vector_type(4)));

__device__ __forceinline__ uint32_t f32_to_bf16_rne(float f) {
    const uint32_t u = __float_as_uint(f);
    if ((u & 0x7FFFFFFFu) > 0x7F800000u) return 0x7FC0u;
    return (u + 0x7FFFu + ((u >> 16) & 1u)) >> 16;
}

// The loads are issued in two independent rounds per 8 slots (class, row and gate of each
// slot; then their y rows), so a call costs two memory round trips, not two per slot.
template <int DT>
__global__ __launch_bounds__(256) void combine_kernel(CombineArgs a) {
    constexpr int kB = 8;  // slots per round
    const int t = blockIdx.y;
    const int dim = (blockIdx.x * blockDim.x + threadIdx.x) * 4;
    if (dim >= a.d) return;
    const f32x4_t zero = {0.f, 0.f, 0.f, 0.f};
    const f32x4_t ys = *reinterpret_cast<const f32x4_t*>(a.y_shared + (size_t)t * a.d + dim);
    const f32x4_t rs = a.resid ? *reinterpret_cast<const f32x4_t*>(a.resid + (size_t)t * a.d + dim) : zero;
    f32x4_t acc = zero;
    float coef = 1.0f;
    const int S = a.T * a.K;
    for (int k0 = 0; k0 < a.K; k0 += kB) {
        int pos[kB];
        float g[kB];
        uint8_t c[kB];
#pragma unroll
        for (int u = 0; u < kB; ++u) {
            const int k = k0 + u;
            const int s = t * a.K + (k < a.K ? k : 0);
            c[u] = k < a.K ? a.slot_class[s] : (uint8_t)SPICE_CLASS_EXACT;
            pos[u] = a.inv_perm[s];
            g[u] = a.topk_w[s];
        }
        f32x4_t y[kB];
#pragma unroll
        for (int u = 0; u < kB; ++u) {
            const bool use = (c[u] == SPICE_CLASS_HIT || c[u] == SPICE_CLASS_LORE || c[u] == SPICE_CLASS_EXACT_GPU) &&
                             pos[u] >= 0 && pos[u] < S;
            if (!use) c[u] = (uint8_t)SPICE_CLASS_EXACT;  // not summed
            y[u] = use ? *reinterpret_cast<const f32x4_t*>(a.y_slots + (size_t)pos[u] * a.d + dim) : zero;
        }
#pragma unroll
        for (int u = 0; u < kB; ++u) {  // slots in order, as the sum is defined
            if (c[u] == SPICE_CLASS_EXACT) continue;
            acc += g[u] * y[u];
            if (c[u] == SPICE_CLASS_LORE) coef += g[u];
        }
    }
    f32x4_t o = coef * ys + acc;
    if (a.resid) o += rs;
    if (DT == SPICE_BF16) {
        uint2 p;
        p.x = f32_to_bf16_rne(o.x) | (f32_to_bf16_rne(o.y) << 16);
        p.y = f32_to_bf16_rne(o.z) | (f32_to_bf16_rne(o.w) << 16);
        *reinterpret_cast<uint2*>(static_cast<uint16_t*>(a.out) + (size_t)t * a.d + dim) = p;
    } else {
        *reinterpret_cast<f32x4_t*>(static_cast<float*>(a.out) + (size_t)t * a.d + dim) = o;
    }
}

__global__ void fill_u32_kernel(uint32_t* p, size_t n, uint32_t v) {
    for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x)
        p[i] = v;
}

}  // namespace

hipError_t launch_combine(const CombineArgs& a, hipStream_t s) {
    dim3 grid((a.d / 4 + 255) / 256, a.T);
    if (a.dtype == SPICE_BF16)
        hipLaunchKernelGGL(combine_kernel<SPICE_BF16>, grid, dim3(256), 0, s, a);
    else
        hipLaunchKernelGGL(combine_kernel<SPICE_F32>, grid, dim3(256), 0, s, a);
    return hipGetLastError();
}

hipError_t launch_fill_u32(uint32_t* p, size_t words, uint32_t value, hipStream_t s) {
    if (words == 0) return hipSuccess;
    const size_t blocks = (words + 255) / 256;
    hipLaunchKernelGGL(fill_u32_kernel, dim3((unsigned)(blocks < 1024 ? blocks : 1024)), dim3(256), 0, s, p,
                       words, value);
    return hipGetLastError();
}

}  // namespace spice
