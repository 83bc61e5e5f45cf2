// Output gate of the shared block for a Qwen2-style shared expert: the shared block's
// output S(x) is scaled by sigmoid(w_sg . x) before it enters the combine and every LoRE
// slot's S(x) + B_e A_e x (Eq. 7 / 11, with S the model's native shared expert).
//
// One block of 256 threads per token: products of the stored values are exact in fp64
// and summed in fp64 (strided per thread, then a shuffle and LDS reduction), so only the
// final sigmoid rounds to fp32.
#include <hip/hip_runtime.h>

#include "spice_internal.h"

namespace spice {
namespace {

constexpr int kGateThreads = 256;

template <int DT>
__device__ __forceinline__ double load_elem(const void* p, size_t i) {
    if constexpr (DT == SPICE_BF16)
        return (double)__uint_as_float((uint32_t)static_cast<const uint16_t*>(p)[i] << 16);
    else
        return (double)static_cast<const float*>(p)[i];
}

template <int DT>
__global__ __launch_bounds__(kGateThreads) void shared_gate_kernel(const void* x, const void* w, int d, float* g) {
    __shared__ double part[kGateThreads / 64];
    const int t = blockIdx.x;
    double acc = 0.0;
    for (int i = threadIdx.x; i < d; i += kGateThreads) acc += load_elem<DT>(x, (size_t)t * d + i) * load_elem<DT>(w, i);
    for (int o = 32; o > 0; o >>= 1) acc += __shfl_xor(acc, o);
    if ((threadIdx.x & 63) == 0) part[threadIdx.x >> 6] = acc;
    __syncthreads();
    if (threadIdx.x == 0) {
        double z = 0.0;
        for (int k = 0; k < kGateThreads / 64; ++k) z += part[k];
        g[t] = (float)(1.0 / (1.0 + exp(-z)));
    }
}

}  // namespace

hipError_t launch_shared_gate(const void* x, const void* w_sg, int32_t T, int32_t d, int32_t dtype, float* sgate,
                              hipStream_t s) {
    if (T <= 0) return hipSuccess;
    if (dtype == SPICE_BF16)
        hipLaunchKernelGGL(shared_gate_kernel<SPICE_BF16>, dim3((unsigned)T), dim3(kGateThreads), 0, s, x, w_sg, d, sgate);
    else
        hipLaunchKernelGGL(shared_gate_kernel<SPICE_F32>, dim3((unsigned)T), dim3(kGateThreads), 0, s, x, w_sg, d, sgate);
    return hipGetLastError();
}

}  // namespace spice
