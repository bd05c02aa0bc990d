// Internal interface of the training backward pass (backward.hip).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "lowrank.h"

namespace more {

// Training backward pass (backward.hip).
struct TokGrid {         // grid of a token-major sweep
    int32_t WT;          // token slots per workgroup
    int64_t ntb;         // token blocks
    int32_t splits;      // expert splits
    int32_t parts;       // partials per token: splits x (8 / WT)
};

struct BackwardPlan {
    int32_t RC;
    int32_t balance;     // 1: pbar given (the softmax terms and their sweeps)
    TokGrid gsweep;      // sweep 1 (g)
    TokGrid dzsweep;     // sweep 2, token-major (dz)
    int32_t eblocks;     // expert-major sweep: expert blocks
    int32_t esplits;     //   x token splits
    int64_t Tp;          // T rounded up to 64
    int32_t r1splits;    // token splits of dR1
    int64_t nchunks;     // chunks of the sorted selections in the segmented dtop sum of dR2
    size_t off_z, off_zscratch, off_zhl, off_zb, off_bias, off_g, off_gpart, off_dzpart,
        off_dzsum, off_dzhl, off_dzT, off_r1, off_r2part, off_r1part, off_offsets, off_sorted,
        off_dispatch, off_bpart;
    size_t workspace_bytes;
};

struct BackwardArgs {
    const uint16_t *x, *R1t, *R2t;
    int32_t T, h, r, M, k;
    const int32_t* idx;
    const float *dtop, *pbar, *m, *Z;
    float *dx, *dR1t, *dR2t;
};

bool backward_make_plan(int64_t T, int32_t h, int32_t r, int32_t M, int32_t k, bool balance,
                        BackwardPlan* plan);
hipError_t backward_launch(const BackwardPlan& plan, const BackwardArgs& a, void* workspace,
                           hipStream_t stream);

}  // namespace more
