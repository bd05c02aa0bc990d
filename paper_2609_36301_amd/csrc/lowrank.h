// Internal interface between the C ABI layer and the low-rank router kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace more {

// How one low-rank routing call is split into launches and where its scratch lives.
struct LowrankPlan {
    int32_t RC;               // rank chunks of 16 (r = 16 RC)
    int32_t RT;               // 32-row tiles of the rank axis in the z pass
    int32_t K;                // top-K list length (power of two >= k)
    int32_t fused;            // 1: one fused route kernel per 64 tokens (small expert sets)
    int32_t local;            // 1: the fused kernel also computes z (one launch in all)
    int32_t ntb;              // token blocks of the route kernels
    int32_t chunks;           // expert-axis chunks, each resident in one workgroup's LDS
                              // (1 for the fused route)
    int32_t splits;           // token-block ranges per chunk (route grid = chunks * splits)
    int32_t cap;              // candidate slots per token
    int32_t theta_group;      // threads per token in the threshold kernel
    int32_t hsplit;           // workgroups sharing the h axis of one token group in the z pass
    int32_t steps_per_split;  // 64-wide h chunks per z-pass workgroup
    size_t off_zparts, off_z, off_zhi, off_cz, off_top, off_gnorm, off_tau, off_count, off_cand;
    // single-pass route (zscreen, collect and finalize kernels of resident.hip)
    int32_t single_pass;      // 1: this route
    int32_t sub_tiles;        // expert tiles of the prescreen
    int32_t slots;            // entry slots per lane and token group in the collect kernel
    size_t off_theta0, off_rec, off_scratch;
    size_t workspace_bytes;
};

// Arguments of the single-pass route (pointers into the caller's buffers and workspace).
struct SinglePassArgs {
    const uint16_t *x, *R1t, *R2t;
    int32_t T, h, r, M, k;
    float* z;
    uint16_t* zhi;
    float *cz, *theta0;
    int32_t* count;
    int2* rec;
    void* scratch;
    int32_t* hist;
    int32_t* idx;
    float *gate, *topval;
};

hipError_t single_pass_launch(const LowrankPlan& plan, const SinglePassArgs& a, hipStream_t stream);

// Bytes of the collect kernel's entry scratch for `grid` workgroups.
size_t collect_scratch_bytes(int64_t grid, int32_t slots);

// Returns false when m_chunks is not 0, 1 or a multiple of 8 up to 1024.
bool lowrank_make_plan(int64_t T, int32_t h, int32_t r, int32_t M, int32_t k, int32_t m_chunks,
                       LowrankPlan* plan);

// counts (nullable) is cleared by the launch, ready for histogram_launch(..., true).
hipError_t lowrank_launch(const LowrankPlan& plan, const uint16_t* x, const uint16_t* R1t,
                          const uint16_t* R2t, int64_t T, int32_t h, int32_t r, int32_t M,
                          int32_t k, int32_t* idx, float* gate, float* topval,
                          int32_t* counts, void* workspace, hipStream_t stream);

// counts_zeroed: the caller has already cleared counts on this stream.
hipError_t histogram_launch(const int32_t* idx, int64_t n, int32_t M, int32_t* counts,
                            hipStream_t stream, bool counts_zeroed = false);

struct FullrankPlan {
    int32_t K;
    int32_t logit_bits;
    size_t off_logits, off_gemm_ws, gemm_ws_bytes;
    size_t workspace_bytes;
};

bool fullrank_make_plan(int64_t T, int32_t h, int32_t M, int32_t k, int32_t logit_bits,
                        FullrankPlan* plan);

hipError_t fullrank_launch(const FullrankPlan& plan, const uint16_t* x, const uint16_t* Wt,
                           int64_t T, int32_t h, int32_t M, int32_t k, int32_t* idx, float* gate,
                           float* topval, void* workspace, hipStream_t stream, int* blas_status);

// z = x R1 alone, fp32 [T][r] at z, for callers other than the routes (the h-split partials
// and the z_hi / error-scale byproducts of the z pass go to scratch).
size_t zonly_workspace_bytes(int64_t T, int32_t h, int32_t r);
hipError_t zonly_launch(const uint16_t* x, const uint16_t* R1t, int64_t T, int32_t h, int32_t r,
                        float* z, void* scratch, hipStream_t stream);

// Softmax statistics of the training forward pass (stats.hip).
struct StatsPlan {
    int32_t RC;
    int32_t chunks, splits;     // Z sweep: expert chunks x token splits
    int32_t eblocks, psplits;   // psum sweep: expert blocks x token splits
    int32_t gz, gp;             // threads per output summing the Z and psum partials
    int32_t own_z;              // 1: z is computed here (the routing call keeps none)
    size_t off_tv, off_z, off_zscratch, off_zhl, off_mb, off_Zp, off_bias, off_part;
    size_t workspace_bytes;
};

struct StatsArgs {
    const uint16_t *x, *R1t, *R2t;
    const float* z;      // z = x R1 [T][r] (unused with own_z)
    const float* mtop;   // top-1 logit of token t at mtop[t ks]
    int32_t ks;
    int32_t T, h, r, M;
    float *m, *Z, *psum;
};

bool stats_make_plan(int64_t T, int32_t h, int32_t r, int32_t M, int32_t k, bool own_z,
                     StatsPlan* plan);
hipError_t stats_launch(const StatsPlan& plan, const StatsArgs& a, void* workspace,
                        hipStream_t stream);
hipError_t stats_zero_psum(float* psum, int32_t M, hipStream_t stream);

// Fused standard router (fullrank_fused.hip): x rows of a token block resident in LDS, the
// logits of each expert tile folded into register top-K lists.
struct FusedFullrankPlan {
    int32_t NT;        // 32-token tiles per workgroup
    int32_t K;         // list length (power of two >= k)
    int32_t esplits;   // workgroups sharing the expert axis of one token block
    size_t workspace_bytes;  // the splits' lists (none with one split)
};

// false when the x rows of one 32-token tile do not fit the workgroup's LDS (h > 2112) or k > 32
bool fullrank_fused_make_plan(int64_t T, int32_t h, int32_t M, int32_t k, FusedFullrankPlan* plan);
hipError_t fullrank_fused_launch(const FusedFullrankPlan& plan, const uint16_t* x,
                                 const uint16_t* Wt, int64_t T, int32_t h, int32_t M, int32_t k,
                                 int32_t* idx, float* gate, float* topval, void* workspace,
                                 hipStream_t stream);

// Dispatch bookkeeping (dispatch.hip): N = T k entries, keys 0 .. M.
int dispatch_passes(int32_t M);
size_t dispatch_workspace_bytes(int64_t N);
hipError_t dispatch_launch(const int32_t* idx, int64_t N, int32_t M, int32_t* offsets,
                           int32_t* sorted, void* workspace, hipStream_t stream);

}  // namespace more
