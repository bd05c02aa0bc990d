// Per-expert selection counts (the bincount behind the load-balancing statistic f,
// Appendix "Training"): counts[e] = #{(t, j) : idx[t][j] == e}.
//
// Small expert counts use a per-workgroup LDS histogram flushed with one global atomic per
// non-empty bin; large ones add straight into global memory.  Counts are cleared by a fill
// kernel (not a memset) so the sequence stays valid inside a captured HIP graph.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "lowrank.h"

namespace more {

constexpr int32_t kLdsBins = 16384;

__global__ __launch_bounds__(256) void fill_zero_kernel(int32_t* __restrict__ p, int64_t n) {
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
         i += (int64_t)gridDim.x * blockDim.x)
        p[i] = 0;
}

__global__ __launch_bounds__(256) void histogram_lds_kernel(const int32_t* __restrict__ idx,
                                                            int64_t n, int32_t M,
                                                            int32_t* __restrict__ counts) {
    __shared__ int32_t bins[kLdsBins];
    for (int32_t e = threadIdx.x; e < M; e += blockDim.x) bins[e] = 0;
    __syncthreads();
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
         i += (int64_t)gridDim.x * blockDim.x) {
        const int32_t e = idx[i];
        if (e >= 0 && e < M) atomicAdd(&bins[e], 1);
    }
    __syncthreads();
    for (int32_t e = threadIdx.x; e < M; e += blockDim.x) {
        const int32_t c = bins[e];
        if (c) atomicAdd(&counts[e], c);
    }
}

__global__ __launch_bounds__(256) void histogram_global_kernel(const int32_t* __restrict__ idx,
                                                               int64_t n, int32_t M,
                                                               int32_t* __restrict__ counts) {
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
         i += (int64_t)gridDim.x * blockDim.x) {
        const int32_t e = idx[i];
        if (e >= 0 && e < M) atomicAdd(&counts[e], 1);
    }
}

hipError_t histogram_launch(const int32_t* idx, int64_t n, int32_t M, int32_t* counts,
                            hipStream_t st) {
    {
        int64_t blocks = ((int64_t)M + 255) / 256;
        if (blocks > 1024) blocks = 1024;
        hipLaunchKernelGGL(fill_zero_kernel, dim3((unsigned)blocks), dim3(256), 0, st, counts,
                           (int64_t)M);
    }
    if (n > 0) {
        if (M <= kLdsBins) {
            int64_t blocks = n / 8192;
            blocks = blocks < 1 ? 1 : (blocks > 128 ? 128 : blocks);
            hipLaunchKernelGGL(histogram_lds_kernel, dim3((unsigned)blocks), dim3(256), 0, st, idx,
                               n, M, counts);
        } else {
            int64_t blocks = (n + 255) / 256;
            blocks = blocks > 2048 ? 2048 : blocks;
            hipLaunchKernelGGL(histogram_global_kernel, dim3((unsigned)blocks), dim3(256), 0, st,
                               idx, n, M, counts);
        }
    }
    return hipGetLastError();
}

}  // namespace more
