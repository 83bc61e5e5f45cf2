// Device steps of the LoRE calibration fit (Sec. 4.2, Eq. 8-10) for one expert:
//   fit_setup      a one-expert bucket of all n calibration tokens (perm = identity,
//                  HIT class only) for the grouped FFN, which computes E_e(x) and S(x);
//   fit_residual   Y = E_e(x) - S(x), the target of Eq. 8, in place;
//   fit_gram       n x n Gram matrices of the rows of X (dtype) or Y (fp32), accumulated in
//                  fp64 (one 16 x 16 output tile per block, 64-column panels through LDS);
//   fit_project    rows of A = (X^T Z)^T and of B = Y^T V from n x r host coefficients.
// The n x n eigen-decomposition and solve between gram and project run on the host.
#include <hip/hip_runtime.h>

#include "spice_internal.h"

namespace spice {
namespace {

constexpr int kGramTile = 16;
constexpr int kGramThreads = 256;

__global__ void fit_setup_kernel(int32_t n, int32_t* perm, int32_t* offsets, int32_t* resident) {
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n) perm[i] = i;
    if (i == 0) {
        // classes x (N + 1) with N = 1: HIT [0, n), LORE and EXACT empty
        offsets[0] = 0; offsets[1] = n;
        offsets[2] = n; offsets[3] = n;
        offsets[4] = n; offsets[5] = n;
        resident[0] = 0;
    }
}

__global__ void fit_residual_kernel(size_t count, float* y, const float* s) {
    const size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i < count) y[i] -= s[i];
}

__device__ __forceinline__ double elem(const void* p, int dtype, size_t i) {
    if (dtype == SPICE_BF16) return (double)__uint_as_float((uint32_t)static_cast<const uint16_t*>(p)[i] << 16);
    return (double)static_cast<const float*>(p)[i];
}

// G[i][j] = sum_k M[i][k] M[j][k] for the 16 x 16 tile (blockIdx.y, blockIdx.x); only tiles
// on or above the diagonal are computed and mirrored.  The two 16-row panels go through
// LDS 64 columns at a time (coalesced row reads, widened to fp64); each thread owns one
// (i, j) of the tile.
__global__ __launch_bounds__(kGramThreads) void fit_gram_kernel(int32_t n, int32_t d, int dtype, const void* M,
                                                                 double* G) {
    constexpr int kChunk = 64;
    const int ti = blockIdx.y, tj = blockIdx.x;
    if (tj < ti) return;
    __shared__ double pi[kGramTile][kChunk + 1];
    __shared__ double pj[kGramTile][kChunk + 1];
    const int tid = threadIdx.x;
    const int oi = tid / kGramTile, oj = tid % kGramTile;
    double acc = 0.0;
    for (int k0 = 0; k0 < d; k0 += kChunk) {
        for (int e = tid; e < kGramTile * kChunk; e += kGramThreads) {
            const int row = e / kChunk, col = e % kChunk, k = k0 + col;
            const int gi = ti * kGramTile + row, gj = tj * kGramTile + row;
            pi[row][col] = (gi < n && k < d) ? elem(M, dtype, (size_t)gi * d + k) : 0.0;
            pj[row][col] = (gj < n && k < d) ? elem(M, dtype, (size_t)gj * d + k) : 0.0;
        }
        __syncthreads();
        for (int c = 0; c < kChunk; ++c) acc += pi[oi][c] * pj[oj][c];
        __syncthreads();
    }
    const int i = ti * kGramTile + oi, j = tj * kGramTile + oj;
    if (i < n && j < n) {
        G[(size_t)i * n + j] = acc;
        G[(size_t)j * n + i] = acc;
    }
}

// out[k][j] (b_layout) or out[j][k] = sum_i M[i][k] C[i][j]: one thread per (feature k,
// column j); a block takes 256 consecutive features of one column, so the rows of M are
// read coalesced and C[i][j] is the same for the whole block.
__global__ __launch_bounds__(256) void fit_project_kernel(int32_t n, int32_t d, int32_t r, int dtype, const void* M,
                                                          const double* C, float* out, int b_layout) {
    const int k = blockIdx.x * blockDim.x + threadIdx.x, j = blockIdx.y;
    if (k >= d) return;
    double acc = 0.0;
    for (int i = 0; i < n; ++i) acc += elem(M, dtype, (size_t)i * d + k) * C[(size_t)i * r + j];
    if (b_layout) out[(size_t)k * r + j] = (float)acc;
    else out[(size_t)j * d + k] = (float)acc;
}

}  // namespace

hipError_t launch_fit_setup(int32_t n, int32_t* perm, int32_t* offsets, int32_t* resident, hipStream_t s) {
    hipLaunchKernelGGL(fit_setup_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, n, perm, offsets,
                       resident);
    return hipGetLastError();
}

hipError_t launch_fit_residual(size_t count, float* y, const float* shared, hipStream_t s) {
    if (count == 0) return hipSuccess;
    hipLaunchKernelGGL(fit_residual_kernel, dim3((unsigned)((count + 255) / 256)), dim3(256), 0, s, count, y,
                       shared);
    return hipGetLastError();
}

hipError_t launch_fit_gram(int32_t n, int32_t d, int dtype, const void* M, double* G, hipStream_t s) {
    const unsigned t = (unsigned)((n + kGramTile - 1) / kGramTile);
    hipLaunchKernelGGL(fit_gram_kernel, dim3(t, t), dim3(kGramThreads), 0, s, n, d, dtype, M, G);
    return hipGetLastError();
}

hipError_t launch_fit_project(int32_t n, int32_t d, int32_t r, int dtype, const void* M, const double* C, float* out,
                              bool b_layout, hipStream_t s) {
    hipLaunchKernelGGL(fit_project_kernel, dim3((unsigned)((d + 255) / 256), (unsigned)r), dim3(256), 0, s, n, d, r,
                       dtype, M, C, out, b_layout ? 1 : 0);
    return hipGetLastError();
}

}  // namespace spice
