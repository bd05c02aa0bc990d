// Full-rank (standard) router baseline: softmax(TopK(x W)) with the logits materialised.
// ("Preliminaries", standard router; the paper's unfused router is a GEMM followed by
// top-k and softmax as separate kernels.)
//
//   1. hipBLASLt GEMM  L[T][M] = x[T][h] * Wt[M][h]^T, fp32 accumulate, fp32 or bf16 output,
//      into the caller's workspace;
//   2. rows_topk: one wave per token row; each lane scans its strided share of the row in
//      16-byte pieces keeping a sorted register list, then a butterfly of list merges across
//      the wave; lane 0 applies the softmax and stores the row.
#include <hip/hip_runtime.h>
#include <hipblaslt/hipblaslt.h>
#include <stdint.h>

#include <map>
#include <mutex>
#include <tuple>

#include "device_common.h"
#include "lowrank.h"

namespace more {

// One wave per token row.  When a row starts on a 16-byte boundary (M a multiple of 8 for bf16
// logits, of 4 for fp32), lane l reads 16-byte pieces l, l + 64, ..., four pieces in flight,
// and tests a piece's largest value against the lane's K-th before looking at its elements
// (after the first few hundred logits almost no piece has a candidate), so the loop runs at
// the rate the logits stream in.  Other rows take one logit per lane and step.  Each lane
// visits its ids in increasing order, so a strict > keeps the smaller id on equal logits.
//
// Short rows (at most NPL pieces per lane: 16, or 8 at K = 32; M <= 8192 bf16 or 4096 fp32
// logits) are held in registers by rows_topk_short_kernel and take a threshold path instead: theta = the k-th largest of the 64 lanes'
// maxima (a bitonic sort across the wave) is reached by k distinct logits, so the top k are
// among the logits >= theta, usually a few more than k; those go to LDS and each one's rank is
// counted against the others.  Rows with more than 128 such logits (ties) use the list path.
constexpr int kRowsCap = 128;  // candidates per row on the threshold path

// The wave's LDS writes complete before any of its lanes reads them back (s_waitcnt
// lgkmcnt(0); the other counters keep their maximum).  Waves of a workgroup exit at different
// times here, so there is no workgroup barrier.
__device__ __forceinline__ void wave_lds_sync() {
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_waitcnt((15) | (3 << 14) | (7 << 4));
    __builtin_amdgcn_wave_barrier();
    asm volatile("" ::: "memory");
}

// x sorted descending across the 64 lanes of the wave (lane 0 the largest): bitonic network
// of 21 compare-exchange stages, partners by lane_xor.
__device__ __forceinline__ float wave_sort_desc(float x, int lane) {
#pragma unroll
    for (int size = 2; size <= 64; size <<= 1) {
#pragma unroll
        for (int d = size >> 1; d >= 1; d >>= 1) {
            float y;
            switch (d) {
                case 1: y = lane_xor<1>(x); break;
                case 2: y = lane_xor<2>(x); break;
                case 4: y = lane_xor<4>(x); break;
                case 8: y = lane_xor<8>(x); break;
                case 16: y = lane_xor<16>(x); break;
                default: y = lane_xor<32>(x); break;
            }
            // within blocks of `size`, descending where (lane & size) == 0 (the last stage
            // has size 64: all descending); the lower lane of a pair keeps the larger value
            const bool desc = (lane & size) == 0 || size == 64;
            const bool lower = (lane & d) == 0;
            x = (lower == desc) ? fmaxf(x, y) : fminf(x, y);
        }
    }
    return x;
}

template <int K, bool BF16, int NPL>
__global__ __launch_bounds__(256) void rows_topk_short_kernel(const void* __restrict__ logits,
                                                              int32_t T, int32_t M, int32_t k,
                                                              int32_t* __restrict__ idx,
                                                              float* __restrict__ gate,
                                                              float* __restrict__ topval) {
    constexpr int PER = BF16 ? 8 : 4;  // logits per 16-byte piece
    __shared__ float cv[4][kRowsCap];
    __shared__ int32_t ci[4][kRowsCap];
    __shared__ float tv[4][K];
    const int lane = threadIdx.x & 63;
    const int wv = threadIdx.x >> 6;
    const int64_t row = (int64_t)blockIdx.x * 4 + wv;
    if (row >= T) return;  // wave-uniform
    float v[K];
    int32_t ix[K];
    list_init<K>(v, ix);
    auto piece = [&](const u32x4& q, int t) __attribute__((always_inline)) {
        const uint32_t w = q[BF16 ? t / 2 : t];
        return BF16 ? __builtin_bit_cast(float, (t & 1) ? (w & 0xFFFF0000u) : (w << 16))
                    : __builtin_bit_cast(float, w);
    };
    {  // the caller launches this kernel for M % PER == 0 and M / PER <= 64 NPL
        const u32x4* P = reinterpret_cast<const u32x4*>(
            static_cast<const char*>(logits) + row * (int64_t)M * (BF16 ? 2 : 4));
        const int32_t np = M / PER;
        u32x4 q[NPL];
#pragma unroll
        for (int j = 0; j < NPL; ++j) {
            const int32_t c = lane + 64 * j;
            q[j] = P[c < np ? c : np - 1];  // past the end: a reload, excluded below
        }
        float mx = -__builtin_huge_valf();
#pragma unroll
        for (int j = 0; j < NPL; ++j)
            if (lane + 64 * j < np)
#pragma unroll
                for (int t = 0; t < PER; ++t) mx = fmaxf(mx, piece(q[j], t));
        // k distinct logits (the maxima of k lanes) reach theta
        const float sorted = wave_sort_desc(mx, lane);
        const float theta = __builtin_bit_cast(
            float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, sorted), k - 1));
        int cnt = 0;
#pragma unroll
        for (int j = 0; j < NPL; ++j)
            if (lane + 64 * j < np)
#pragma unroll
                for (int t = 0; t < PER; ++t) cnt += piece(q[j], t) >= theta ? 1 : 0;
        // exclusive prefix of the lanes' counts
        int incl = cnt;
#pragma unroll
        for (int d = 1; d < 64; d <<= 1) {
            const int y = __shfl_up(incl, d, 64);
            incl += lane >= d ? y : 0;
        }
        const int total = __shfl(incl, 63, 64);
        if (total <= kRowsCap) {  // wave-uniform
            int o = incl - cnt;
#pragma unroll
            for (int j = 0; j < NPL; ++j)
                if (lane + 64 * j < np)
#pragma unroll
                    for (int t = 0; t < PER; ++t) {
                        const float x = piece(q[j], t);
                        if (x >= theta) {
                            cv[wv][o] = x;
                            ci[wv][o] = (lane + 64 * j) * PER + t;
                            ++o;
                        }
                    }
            wave_lds_sync();
            // rank of candidates lane and lane + 64 under (larger logit, then smaller id)
            int rk[2] = {0, 0};
            float cx[2];
            int32_t cie[2];
#pragma unroll
            for (int h2 = 0; h2 < 2; ++h2) {
                const int j = lane + 64 * h2;
                cx[h2] = j < total ? cv[wv][j] : -__builtin_huge_valf();
                cie[h2] = j < total ? ci[wv][j] : kNoExpert;
            }
            for (int j = 0; j < total; ++j) {
                const float y = cv[wv][j];
                const int32_t yi = ci[wv][j];
#pragma unroll
                for (int h2 = 0; h2 < 2; ++h2) rk[h2] += better(y, yi, cx[h2], cie[h2]) ? 1 : 0;
            }
#pragma unroll
            for (int h2 = 0; h2 < 2; ++h2)
                if (lane + 64 * h2 < total && rk[h2] < k) tv[wv][rk[h2]] = cx[h2];
            wave_lds_sync();
            // softmax over the k selected logits, summed in rank order as store_selection does
            const float top = tv[wv][0];
            float sum = 0.0f;
            for (int j = 0; j < k; ++j) sum += expf(tv[wv][j] - top);
#pragma unroll
            for (int h2 = 0; h2 < 2; ++h2) {
                if (lane + 64 * h2 < total && rk[h2] < k) {
                    const int64_t o2 = row * k + rk[h2];
                    idx[o2] = cie[h2];
                    gate[o2] = expf(cx[h2] - top) / sum;
                    if (topval) topval[o2] = cx[h2];
                }
            }
            return;
        }
        // many logits reach theta (ties): sorted lists over the held pieces
#pragma unroll
        for (int j = 0; j < NPL; ++j) {
            const int32_t c = lane + 64 * j;
            if (c < np) {
#pragma unroll
                for (int t = 0; t < PER; ++t) {
                    const float x = piece(q[j], t);
                    if (x > v[K - 1]) list_insert_newer<K>(v, ix, x, c * PER + t);
                }
            }
        }
    }
    list_merge_xor<1, K>(v, ix);
    list_merge_xor<2, K>(v, ix);
    list_merge_xor<4, K>(v, ix);
    list_merge_xor<8, K>(v, ix);
    list_merge_xor<16, K>(v, ix);
    list_merge_xor<32, K>(v, ix);
    if (lane == 0) store_selection<K>(v, ix, k, row, idx, gate, topval);
}

template <int K, bool BF16>
__global__ __launch_bounds__(256) void rows_topk_kernel(const void* __restrict__ logits, int32_t T,
                                                        int32_t M, int32_t k,
                                                        int32_t* __restrict__ idx,
                                                        float* __restrict__ gate,
                                                        float* __restrict__ topval) {
    constexpr int PER = BF16 ? 8 : 4;  // logits per 16-byte piece
    constexpr int U = 4;               // pieces in flight per lane
    const int lane = threadIdx.x & 63;
    const int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    if (row >= T) return;  // wave-uniform
    float v[K];
    int32_t ix[K];
    list_init<K>(v, ix);
    if (M % PER == 0) {
        const u32x4* P = reinterpret_cast<const u32x4*>(
            static_cast<const char*>(logits) + row * (int64_t)M * (BF16 ? 2 : 4));
        const int32_t np = M / PER;
        for (int32_t c0 = lane; c0 < np; c0 += 64 * U) {
            u32x4 q[U];
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int32_t c = c0 + 64 * u;
                q[u] = P[c < np ? c : np - 1];  // past the end: a reload, masked below
            }
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int32_t c = c0 + 64 * u;
                float x[PER];
#pragma unroll
                for (int t = 0; t < PER; ++t) {
                    const uint32_t w = q[u][BF16 ? t / 2 : t];
                    x[t] = BF16 ? __builtin_bit_cast(float, (t & 1) ? (w & 0xFFFF0000u) : (w << 16))
                                : __builtin_bit_cast(float, w);
                    if (c >= np) x[t] = -__builtin_huge_valf();
                }
                float mx = x[0];
#pragma unroll
                for (int t = 1; t < PER; ++t) mx = fmaxf(mx, x[t]);
                if (mx > v[K - 1]) {
#pragma unroll
                    for (int t = 0; t < PER; ++t)
                        if (x[t] > v[K - 1]) list_insert_newer<K>(v, ix, x[t], c * PER + t);
                }
            }
        }
    } else if (BF16) {
        const uint16_t* L = static_cast<const uint16_t*>(logits) + row * M;
#pragma unroll 4
        for (int32_t e = lane; e < M; e += 64) {
            const float x = bf16_bits_to_f32(L[e]);
            if (x > v[K - 1]) list_insert_newer<K>(v, ix, x, e);
        }
    } else {
        const float* L = static_cast<const float*>(logits) + row * M;
#pragma unroll 4
        for (int32_t e = lane; e < M; e += 64) {
            const float x = L[e];
            if (x > v[K - 1]) list_insert_newer<K>(v, ix, x, e);
        }
    }
    list_merge_xor<1, K>(v, ix);
    list_merge_xor<2, K>(v, ix);
    list_merge_xor<4, K>(v, ix);
    list_merge_xor<8, K>(v, ix);
    list_merge_xor<16, K>(v, ix);
    list_merge_xor<32, K>(v, ix);
    if (lane == 0) store_selection<K>(v, ix, k, row, idx, gate, topval);
}

// ---------------------------------------------------------------- hipBLASLt state
namespace {

struct GemmKey {
    int device;
    int64_t T;
    int32_t h, M, bits;
    bool operator<(const GemmKey& o) const {
        return std::tie(device, T, h, M, bits) < std::tie(o.device, o.T, o.h, o.M, o.bits);
    }
};

struct GemmEntry {
    hipblasLtMatmulDesc_t desc = nullptr;
    hipblasLtMatrixLayout_t la = nullptr, lb = nullptr, lc = nullptr;
    hipblasLtMatmulHeuristicResult_t heur{};
    bool ok = false;
};

std::mutex g_mu;
std::map<int, hipblasLtHandle_t> g_handles;
std::map<GemmKey, GemmEntry> g_gemms;

constexpr size_t kGemmWorkspace = (size_t)64 << 20;

// Returns nullptr and sets *status on failure.  Caller holds g_mu.
GemmEntry* gemm_entry(int device, int64_t T, int32_t h, int32_t M, int32_t bits, int* status) {
    GemmKey key{device, T, h, M, bits};
    auto it = g_gemms.find(key);
    if (it != g_gemms.end()) return it->second.ok ? &it->second : nullptr;
    hipblasLtHandle_t handle;
    auto hit = g_handles.find(device);
    if (hit == g_handles.end()) {
        hipblasStatus_t s = hipblasLtCreate(&handle);
        if (s != HIPBLAS_STATUS_SUCCESS) {
            *status = (int)s;
            return nullptr;
        }
        g_handles[device] = handle;
    } else {
        handle = hit->second;
    }
    GemmEntry e;
    hipblasStatus_t s = hipblasLtMatmulDescCreate(&e.desc, HIPBLAS_COMPUTE_32F, HIP_R_32F);
    hipblasOperation_t opA = HIPBLAS_OP_T, opB = HIPBLAS_OP_N;
    if (s == HIPBLAS_STATUS_SUCCESS)
        s = hipblasLtMatmulDescSetAttribute(e.desc, HIPBLASLT_MATMUL_DESC_TRANSA, &opA, sizeof(opA));
    if (s == HIPBLAS_STATUS_SUCCESS)
        s = hipblasLtMatmulDescSetAttribute(e.desc, HIPBLASLT_MATMUL_DESC_TRANSB, &opB, sizeof(opB));
    // Column-major view: A = Wt as (h x M), B = x as (h x T), D = L as (M x T).
    if (s == HIPBLAS_STATUS_SUCCESS) s = hipblasLtMatrixLayoutCreate(&e.la, HIP_R_16BF, h, M, h);
    if (s == HIPBLAS_STATUS_SUCCESS) s = hipblasLtMatrixLayoutCreate(&e.lb, HIP_R_16BF, h, T, h);
    if (s == HIPBLAS_STATUS_SUCCESS)
        s = hipblasLtMatrixLayoutCreate(&e.lc, bits == 16 ? HIP_R_16BF : HIP_R_32F, M, T, M);
    hipblasLtMatmulPreference_t pref = nullptr;
    if (s == HIPBLAS_STATUS_SUCCESS) s = hipblasLtMatmulPreferenceCreate(&pref);
    uint64_t wsb = kGemmWorkspace;
    if (s == HIPBLAS_STATUS_SUCCESS)
        s = hipblasLtMatmulPreferenceSetAttribute(pref, HIPBLASLT_MATMUL_PREF_MAX_WORKSPACE_BYTES,
                                                  &wsb, sizeof(wsb));
    int returned = 0;
    if (s == HIPBLAS_STATUS_SUCCESS)
        s = hipblasLtMatmulAlgoGetHeuristic(handle, e.desc, e.la, e.lb, e.lc, e.lc, pref, 1,
                                            &e.heur, &returned);
    if (pref) hipblasLtMatmulPreferenceDestroy(pref);
    e.ok = (s == HIPBLAS_STATUS_SUCCESS && returned > 0);
    if (!e.ok) *status = (s == HIPBLAS_STATUS_SUCCESS) ? (int)HIPBLAS_STATUS_NOT_SUPPORTED : (int)s;
    auto ins = g_gemms.emplace(key, e).first;
    return e.ok ? &ins->second : nullptr;
}

}  // namespace

static int pow2_at_least_fr(int k) {
    int K = 1;
    while (K < k) K <<= 1;
    return K;
}

bool fullrank_make_plan(int64_t T, int32_t h, int32_t M, int32_t k, int32_t logit_bits,
                        FullrankPlan* p) {
    (void)h;
    FullrankPlan q{};
    q.K = pow2_at_least_fr(k);
    q.logit_bits = logit_bits;
    const size_t lbytes = (size_t)T * (size_t)M * (logit_bits == 16 ? 2 : 4);
    q.off_logits = 0;
    q.off_gemm_ws = (lbytes + 255) & ~(size_t)255;
    q.gemm_ws_bytes = kGemmWorkspace;
    q.workspace_bytes = q.off_gemm_ws + q.gemm_ws_bytes;
    *p = q;
    return true;
}

template <int K>
static void launch_rows(const FullrankPlan& p, const void* L, int64_t T, int32_t M, int32_t k,
                        int32_t* idx, float* gate, float* topval, hipStream_t st) {
    dim3 grid((unsigned)((T + 3) / 4));
    constexpr int NPL = K == 32 ? 8 : 16;
    const int per = p.logit_bits == 16 ? 8 : 4;
    if (M % per == 0 && M / per <= 64 * NPL) {
        if (p.logit_bits == 16)
            hipLaunchKernelGGL((rows_topk_short_kernel<K, true, NPL>), grid, dim3(256), 0, st, L,
                               (int32_t)T, M, k, idx, gate, topval);
        else
            hipLaunchKernelGGL((rows_topk_short_kernel<K, false, NPL>), grid, dim3(256), 0, st, L,
                               (int32_t)T, M, k, idx, gate, topval);
        return;
    }
    if (p.logit_bits == 16)
        hipLaunchKernelGGL((rows_topk_kernel<K, true>), grid, dim3(256), 0, st, L, (int32_t)T, M, k,
                           idx, gate, topval);
    else
        hipLaunchKernelGGL((rows_topk_kernel<K, false>), grid, dim3(256), 0, st, L, (int32_t)T, M,
                           k, idx, gate, topval);
}

hipError_t fullrank_launch(const FullrankPlan& p, const uint16_t* x, const uint16_t* Wt, int64_t T,
                           int32_t h, int32_t M, int32_t k, int32_t* idx, float* gate,
                           float* topval, void* workspace, hipStream_t st, int* blas_status) {
    *blas_status = 0;
    int device = 0;
    hipError_t he = hipGetDevice(&device);
    if (he != hipSuccess) return he;
    char* ws = static_cast<char*>(workspace);
    void* L = ws + p.off_logits;
    {
        std::lock_guard<std::mutex> lock(g_mu);
        GemmEntry* e = gemm_entry(device, T, h, M, p.logit_bits, blas_status);
        if (!e) return hipErrorUnknown;
        const float alpha = 1.0f, beta = 0.0f;
        hipblasStatus_t s = hipblasLtMatmul(g_handles[device], e->desc, &alpha, Wt, e->la, x, e->lb,
                                            &beta, L, e->lc, L, e->lc, &e->heur.algo,
                                            ws + p.off_gemm_ws, p.gemm_ws_bytes, st);
        if (s != HIPBLAS_STATUS_SUCCESS) {
            *blas_status = (int)s;
            return hipErrorUnknown;
        }
    }
    switch (p.K) {
        case 1: launch_rows<1>(p, L, T, M, k, idx, gate, topval, st); break;
        case 2: launch_rows<2>(p, L, T, M, k, idx, gate, topval, st); break;
        case 4: launch_rows<4>(p, L, T, M, k, idx, gate, topval, st); break;
        case 8: launch_rows<8>(p, L, T, M, k, idx, gate, topval, st); break;
        case 16: launch_rows<16>(p, L, T, M, k, idx, gate, topval, st); break;
        case 32: launch_rows<32>(p, L, T, M, k, idx, gate, topval, st); break;
        default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

}  // namespace more
