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
    size_t off_z, off_zscratch, off_zs, off_w3, off_ff, workspace_bytes;
};

// The wide route serves (r, k) exactly when the register-tiled routes do not.
bool wide_route_needed(int32_t r, int32_t k);
bool wide_make_plan(int64_t T, int32_t h, int32_t r, int32_t M, int32_t k, WidePlan* plan);
hipError_t wide_launch(const WidePlan& plan, const uint16_t* x, const uint16_t* R1t,
                       const uint16_t* R2t, int64_t T, int32_t h, int32_t r, int32_t M, int32_t k,
                       int32_t* idx, float* gate, float* topval, void* workspace,
                       hipStream_t stream);

}  // namespace more
