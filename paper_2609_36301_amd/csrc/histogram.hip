// Per-expert selection counts (the bincount behind the load-balancing statistic f,
// Appendix "Training"): counts[e] = #{(t, j) : idx[t][j] == e}.
//
// Up to 16384 experts, each workgroup counts one slice of the ids in an LDS histogram and
// flushes it with one global atomic per non-empty bin; larger expert sets use an LDS hash table
// per slice instead (one pass over the ids rather than one per range of 16384 bins).  Counts are cleared by a
// fill kernel (not a memset) so the sequence stays valid inside a captured HIP graph; the
// routing call clears them in its threshold kernel instead.
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

// Counts the ids in [b0, b0 + kLdsBins) over one slice of idx in an LDS histogram, then adds
// the non-empty bins to counts with one global atomic each.  blockIdx.y selects the bin range,
// blockIdx.x the slice; the per-workgroup aggregation keeps hot experts from serialising on
// one global address.
__global__ __launch_bounds__(256) void histogram_lds_kernel(const int32_t* __restrict__ idx,
                                                            int64_t n, int32_t M,
                                                            int32_t* __restrict__ counts) {
    __shared__ int32_t bins[kLdsBins];
    const int32_t b0 = (int32_t)blockIdx.y * kLdsBins;
    const int32_t nb = M - b0 < kLdsBins ? M - b0 : kLdsBins;
    for (int32_t e = threadIdx.x; e < nb; e += blockDim.x) bins[e] = 0;
    __syncthreads();
    const int64_t per = (n + gridDim.x - 1) / gridDim.x;
    const int64_t i0 = (int64_t)blockIdx.x * per;
    const int64_t i1 = i0 + per < n ? i0 + per : n;
    for (int64_t i = i0 + threadIdx.x; i < i1; i += blockDim.x) {
        const int32_t e = idx[i] - b0;
        if (e >= 0 && e < nb) atomicAdd(&bins[e], 1);
    }
    __syncthreads();
    for (int32_t e = threadIdx.x; e < nb; e += blockDim.x) {
        const int32_t c = bins[e];
        if (c) atomicAdd(&counts[b0 + e], c);
    }
}

// Larger expert sets (M > kHashMinExperts): each workgroup aggregates one slice of kHashSlice
// ids in an LDS hash table (linear probing, twice as many slots as ids) and adds every distinct
// expert of the slice to counts with one global atomic, so an expert chosen by many tokens gets
// one atomic per slice instead of one per selection.
constexpr int kHashSlice = 1024;
constexpr int kHashSlots = 2 * kHashSlice;  // power of two
constexpr int32_t kHashMinExperts = kLdsBins;  // up to one LDS bin range: dense bins

__global__ __launch_bounds__(256) void histogram_hash_kernel(const int32_t* __restrict__ idx,
                                                             int64_t n, int32_t M,
                                                             int32_t* __restrict__ counts) {
    __shared__ int32_t key[kHashSlots], cnt[kHashSlots];
    for (int i = threadIdx.x; i < kHashSlots; i += blockDim.x) {
        key[i] = -1;
        cnt[i] = 0;
    }
    __syncthreads();
    const int64_t i0 = (int64_t)blockIdx.x * kHashSlice;
    const int64_t i1 = i0 + kHashSlice < n ? i0 + kHashSlice : n;
    for (int64_t i = i0 + threadIdx.x; i < i1; i += blockDim.x) {
        const int32_t e = idx[i];
        if (e < 0 || e >= M) continue;
        uint32_t hh = ((uint32_t)e * 2654435761u) & (kHashSlots - 1);
        // at most kHashSlice distinct keys in kHashSlots slots: a free or matching slot exists
        for (int probe = 0; probe < kHashSlots; ++probe) {
            const int32_t old = atomicCAS(&key[hh], -1, e);
            if (old == -1 || old == e) {
                atomicAdd(&cnt[hh], 1);
                break;
            }
            hh = (hh + 1) & (kHashSlots - 1);
        }
    }
    __syncthreads();
    for (int i = threadIdx.x; i < kHashSlots; i += blockDim.x)
        if (key[i] >= 0) atomicAdd(&counts[key[i]], cnt[i]);
}

hipError_t histogram_launch(const int32_t* idx, int64_t n, int32_t M, int32_t* counts,
                            hipStream_t st, bool counts_zeroed) {
    if (!counts_zeroed) {
        int64_t blocks = ((int64_t)M + 255) / 256;
        if (blocks > 1024) blocks = 1024;
        hipLaunchKernelGGL(fill_zero_kernel, dim3((unsigned)blocks), dim3(256), 0, st, counts,
                           (int64_t)M);
    }
    if (n > 0 && M > kHashMinExperts) {
        hipLaunchKernelGGL(histogram_hash_kernel, dim3((unsigned)((n + kHashSlice - 1) / kHashSlice)),
                           dim3(256), 0, st, idx, n, M, counts);
    } else if (n > 0) {
        const int64_t ranges = ((int64_t)M + kLdsBins - 1) / kLdsBins;
        int64_t slices = n / 4096;
        const int64_t max_slices = 256 / ranges > 1 ? 256 / ranges : 1;
        slices = slices < 1 ? 1 : (slices > max_slices ? max_slices : slices);
        hipLaunchKernelGGL(histogram_lds_kernel, dim3((unsigned)slices, (unsigned)ranges),
                           dim3(256), 0, st, idx, n, M, counts);
    }
    return hipGetLastError();
}

}  // namespace more
