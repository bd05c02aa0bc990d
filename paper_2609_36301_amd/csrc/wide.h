// Wide low-rank route: ranks beyond the register-tiled kernels (r a multiple of 16 up to 256,
// other than 16, 32 and 64) and 17 <= k <= 32.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "lowrank.h"

namespace more {

constexpr int32_t kWideMaxRank = 256;

struct WidePlan {
    int32_t nblocks;      // rank-column blocks of z = x R1, each 64, 32 or 16 columns wide
    int32_t j0[8], w[8];  // first column and width of each block (r <= 256: at most 6 blocks)
    FusedFullrankPlan ff; // the fused sweep over the 3r-wide split of z
    bool stack;           // r not a multiple of 64: R2t rows stacked three times (W3)
    size_t off_z, off_zscratch, off_zs, off_w3, off_ff, workspace_bytes;
};

// The wide route serves (r, k) exactly when the register-tiled routes do not.
bool wide_route_needed(int32_t r, int32_t k);
bool wide_make_plan(int64_t T, int32_t h, int32_t r, int32_t M, int32_t k, WidePlan* plan);

// The fused standard router's sweep (fullrank_fused.hip) over x [T][h] against weight rows
// stored ldw wide (ldw a multiple of 64 dividing h): the contraction's 64-wide chunk c reads
// stored chunk c mod (ldw / 64), so the h / ldw chunk groups of x all meet the same row.
hipError_t fullrank_fused_launch_periodic(const FusedFullrankPlan& plan, const uint16_t* x,
                                          const uint16_t* Wt, int32_t ldw, int64_t T, int32_t h,
                                          int32_t M, int32_t k, int32_t* idx, float* gate,
                                          float* topval, void* workspace, hipStream_t stream);
hipError_t wide_launch(const WidePlan& plan, const uint16_t* x, const uint16_t* R1t,
                       const uint16_t* R2t, int64_t T, int32_t h, int32_t r, int32_t M, int32_t k,
                       int32_t* idx, float* gate, float* topval, void* workspace,
                       hipStream_t stream);

}  // namespace more
