// Low-rank router kernels for gfx950: softmax(TopK(x R1 R2)) without materialising the
// T x M logits (Appendix "Pseudocode", inference algorithm; MoRE layer in "Preliminaries").
//
// Pipeline of one call:
//   zpass    z = x R1 (fp32 accumulate) for 32-token groups; the h axis may be split over
//            several workgroups (hsplit > 1), each writing a partial z;
//   zreduce  sums the partials in a fixed order (only when hsplit > 1);
//   route    for a block of 32*TPW tokens and a chunk of the expert axis: logits
//            z R2 tile by tile on the matrix cores, each lane keeping a running top-K
//            list of its token in registers; lists are merged across lane halves and
//            across the waves of the workgroup; the block either writes the final
//            (idx, gate, topval) or, when the expert axis is split into chunks, a
//            partial top-K list per token;
//   merge    (chunks > 1) merges the chunk lists of each token and writes the result.
//
// MFMA layout.  Every contraction uses v_mfma_f32_32x32x16_bf16 with experts (or rank
// rows) on the 32 A rows and tokens on the 32 B columns.  A lane therefore owns one token
// and 16 logits of it per tile, so the per-token threshold test is lane local.
//
// Phase-1 row permutation.  In zpass, MFMA row m' of tile pt loads rank row
// 32 pt + pi(m') with pi(8j + 4q + i) = 16(j >> 1) + 8q + 4(j & 1) + i.  Lane (n, half)
// then ends up holding, in accumulator elements 8c'..8c'+7, exactly z[n][16 c + 8 half + 0..7]
// for chunk c = 2 pt + c' -- the B-operand layout the expert contraction needs -- so z can
// be written and re-read as plain row-major [T][r] fp32 with 32-byte lane accesses.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "device_common.h"
#include "lowrank.h"

namespace more {

// ------------------------------------------------------------------------------ zpass
template <int RT>
__global__ __launch_bounds__(256) void zpass_kernel(const uint16_t* __restrict__ x,
                                                    const uint16_t* __restrict__ R1t,
                                                    float* __restrict__ zout, int32_t T, int32_t h,
                                                    int32_t r, int32_t steps_per_split) {
    const int lane = threadIdx.x & 63;
    const int w = threadIdx.x >> 6;
    const int n = lane & 31;
    const int half = lane >> 5;
    const int64_t tok = (int64_t)blockIdx.x * 32 + n;
    const bool tok_ok = tok < T;
    const int S = h >> 4;
    const int s0 = blockIdx.y * steps_per_split;
    const int s1 = min(S, s0 + steps_per_split);
    const int len = max(0, s1 - s0);
    const int ws0 = s0 + (len * w) / 4;
    const int ws1 = s0 + (len * (w + 1)) / 4;

    const int jm = n >> 3, qm = (n >> 2) & 1, im = n & 3;
    const int prow = 16 * (jm >> 1) + 8 * qm + 4 * (jm & 1) + im;

    f32x16 acc[RT];
#pragma unroll
    for (int pt = 0; pt < RT; ++pt) acc[pt] = zero_f32x16();

    const uint16_t* xrow = x + (tok_ok ? tok : 0) * (int64_t)h + 8 * half;
    // Operands of 8 consecutive h steps are loaded before their MFMAs so that each wave keeps
    // 8 x 16 bytes of x per lane in flight; steps past the wave's range contribute zeros.
    for (int s = ws0; s < ws1; s += 8) {
        bf16x8 b[8], a[8][RT];
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            const bool ok = s + u < ws1;
            b[u] = (ok && tok_ok) ? load_bf16x8(xrow + 16 * (s + u)) : zero_bf16x8();
#pragma unroll
            for (int pt = 0; pt < RT; ++pt) {
                const int row = 32 * pt + prow;
                a[u][pt] = (ok && row < r)
                               ? load_bf16x8(R1t + (int64_t)row * h + 16 * (s + u) + 8 * half)
                               : zero_bf16x8();
            }
        }
#pragma unroll
        for (int u = 0; u < 8; ++u)
#pragma unroll
            for (int pt = 0; pt < RT; ++pt) acc[pt] = mfma_32x32x16(a[u][pt], b[u], acc[pt]);
    }

    __shared__ f32x16 red[3][RT][64];
    if (w > 0) {
#pragma unroll
        for (int pt = 0; pt < RT; ++pt) red[w - 1][pt][lane] = acc[pt];
    }
    __syncthreads();
    if (w == 0) {
#pragma unroll
        for (int pt = 0; pt < RT; ++pt) {
#pragma unroll
            for (int q = 0; q < 3; ++q) acc[pt] += red[q][pt][lane];
        }
        if (tok_ok) {
            float* zrow = zout + ((int64_t)blockIdx.y * T + tok) * r + 8 * half;
#pragma unroll
            for (int pt = 0; pt < RT; ++pt) {
#pragma unroll
                for (int c2 = 0; c2 < 2; ++c2) {
                    const int c = 2 * pt + c2;
                    if (16 * c < r) {
                        f32x4 lo4, hi4;
#pragma unroll
                        for (int p = 0; p < 4; ++p) {
                            lo4[p] = acc[pt][8 * c2 + p];
                            hi4[p] = acc[pt][8 * c2 + 4 + p];
                        }
                        *reinterpret_cast<f32x4*>(zrow + 16 * c) = lo4;
                        *reinterpret_cast<f32x4*>(zrow + 16 * c + 4) = hi4;
                    }
                }
            }
        }
    }
}

// z[i] = sum over splits s of zparts[s][i], in split order.
__global__ __launch_bounds__(256) void zreduce_kernel(const float* __restrict__ zparts,
                                                      float* __restrict__ z, int64_t n,
                                                      int32_t splits) {
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
         i += (int64_t)gridDim.x * blockDim.x) {
        float s = 0.0f;
        for (int p = 0; p < splits; ++p) s += zparts[(int64_t)p * n + i];
        z[i] = s;
    }
}

// ------------------------------------------------------------------------------ route
constexpr int kRouteWaves = 8;

// Shared-memory layout of one route workgroup (NT tokens, lists of K).
template <int K, int TPW>
struct RouteSmem {
    static constexpr int NT = 32 * TPW;                // tokens of the workgroup
    static constexpr int LPT = 2 * kRouteWaves;        // lanes that see a token's experts
    static constexpr int BL = (2 * K + LPT - 1) / LPT; // screening buckets per lane
    static constexpr int NB = LPT * BL;                // screening buckets per token (>= 2K)
    static constexpr int S = K <= 8 ? 4 : 8;           // private candidate slots per lane
    static constexpr int OCAP = 2 * K + 16;            // shared overflow slots per token
    // Per-token rows have an odd length in 32-bit words so that the 32-64 tokens handled
    // side by side in a wave fall on different LDS banks.
    static constexpr int NBP = NB + 1;
    static constexpr int SLP = LPT * S + 1;
    static constexpr int OCP = OCAP + 1;
    struct Fast {
        float bucket[NT][NBP];
        float theta[NT];
        int32_t lane_count[NT][LPT + 1];
        int32_t ovf_count[NT];
        int32_t fallback;
        float slot_v[NT][SLP];
        int32_t slot_i[NT][SLP];
        float ovf_v[NT][OCP];
        int32_t ovf_i[NT][OCP];
    };
    struct Exact {
        float sv[kRouteWaves / 2][TPW][32][K];
        int32_t si[kRouteWaves / 2][TPW][32][K];
    };
    static constexpr size_t bytes = sizeof(Fast) > sizeof(Exact) ? sizeof(Fast) : sizeof(Exact);
};

template <int RC, int K, int TPW>
struct RouteLane {
    bf16x8 zhi[TPW][RC], zlo[TPW][RC];
};

// z for the lane's token(s) (rows tb*TPW*32 + g*32 + n of the z workspace), split into
// hi/lo bf16 B operands; tokens past T get zeros.
template <int RC, int K, int TPW>
__device__ __forceinline__ void load_z_operands(const float* __restrict__ z, int32_t T, int tb,
                                                int n, int half, RouteLane<RC, K, TPW>& zl) {
    constexpr int R = 16 * RC;
#pragma unroll
    for (int g = 0; g < TPW; ++g) {
        const int64_t tok = ((int64_t)tb * TPW + g) * 32 + n;
#pragma unroll
        for (int c = 0; c < RC; ++c) {
            float v[8];
            if (tok < T) {
                const f32x4* p = reinterpret_cast<const f32x4*>(z + tok * R + 16 * c + 8 * half);
                const f32x4 a0 = p[0], a1 = p[1];
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    v[q] = a0[q];
                    v[4 + q] = a1[q];
                }
            } else {
#pragma unroll
                for (int q = 0; q < 8; ++q) v[q] = 0.0f;
            }
            split_hi_lo(v, zl.zhi[g][c], zl.zlo[g][c]);
        }
    }
}

// A operand of expert tile t: expert row t*32 + n, K half `half` of each 16-wide rank chunk.
template <int RC>
__device__ __forceinline__ void load_expert_rows(const uint16_t* __restrict__ R2t, int32_t M,
                                                 int64_t t, int n, int half, bf16x8 (&a)[RC]) {
    constexpr int R = 16 * RC;
    const int64_t e = t * 32 + n;
    if (e < M) {
        const uint16_t* p = R2t + e * R + 8 * half;
#pragma unroll
        for (int c = 0; c < RC; ++c) a[c] = load_bf16x8(p + 16 * c);
    } else {
#pragma unroll
        for (int c = 0; c < RC; ++c) a[c] = zero_bf16x8();
    }
}

__device__ __forceinline__ void mask_past_end(f32x16& acc, int32_t e0, int32_t M, int half) {
    if (e0 + 32 > M) {
#pragma unroll
        for (int j = 0; j < 16; ++j)
            if (e0 + acc_row(j, half) >= M) acc[j] = -__builtin_huge_valf();
    }
}

__device__ __forceinline__ float max16(const f32x16& a) {
    float m = fmaxf(fmaxf(a[0], a[1]), a[2]);
    m = fmaxf(fmaxf(m, a[3]), a[4]);
    m = fmaxf(fmaxf(m, a[5]), a[6]);
    m = fmaxf(fmaxf(m, a[7]), a[8]);
    m = fmaxf(fmaxf(m, a[9]), a[10]);
    m = fmaxf(fmaxf(m, a[11]), a[12]);
    m = fmaxf(fmaxf(m, a[13]), a[14]);
    return fmaxf(m, a[15]);
}

// Tile loop helper: calls body(a, e0, partial) for the wave's tiles [wb, we); only the
// tile that crosses M (at most one, the last) is visited with partial = true, so full tiles
// carry no bounds checks.  The A operands of the next D tiles are kept in flight in a
// register ring while the current tile is processed.
template <int RC>
struct TileDepth {
    static constexpr int D = RC <= 2 ? 4 : 2;
};

template <int RC, typename Body>
__device__ __forceinline__ void for_each_tile(const uint16_t* __restrict__ R2t, int32_t M,
                                              int64_t wb, int64_t we, int n, int half,
                                              Body&& body) {
    constexpr int D = TileDepth<RC>::D;
    const int64_t full_end = we < (int64_t)(M / 32) ? we : (int64_t)(M / 32);
    if (wb < full_end) {
        bf16x8 ring[D][RC];
#pragma unroll
        for (int d = 0; d < D; ++d)
            if (wb + d < full_end) load_expert_rows<RC>(R2t, M, wb + d, n, half, ring[d]);
        for (int64_t t = wb; t < full_end; t += D) {
#pragma unroll
            for (int d = 0; d < D; ++d) {
                if (t + d < full_end) {
                    body(ring[d], (int32_t)((t + d) * 32), false);
                    if (t + d + D < full_end)
                        load_expert_rows<RC>(R2t, M, t + d + D, n, half, ring[d]);
                }
            }
        }
    }
    if (full_end < we && full_end >= wb) {  // the partial last tile
        bf16x8 a[RC];
        load_expert_rows<RC>(R2t, M, full_end, n, half, a);
        body(a, (int32_t)(full_end * 32), true);
    }
}

// Exact path: every lane keeps a sorted register list of its token over its own experts,
// inserting every logit that beats the list's last entry; lists are then merged across the
// two K halves and across the waves.  Used when the screened path cannot certify a token.
template <int RC, int K, int TPW, bool FINAL>
__device__ __noinline__ void route_exact(const float* __restrict__ z,
                            const uint16_t* __restrict__ R2t,
                            int32_t T, int32_t M, int32_t k, int tb, int chunk, int64_t wb,
                            int64_t we, int w, char* smem, int32_t* __restrict__ idx,
                            float* __restrict__ gate, float* __restrict__ topval,
                            float* __restrict__ part_v, int32_t* __restrict__ part_i) {
    using S = RouteSmem<K, TPW>;
    auto& sm = *reinterpret_cast<typename S::Exact*>(smem);
    const int lane = threadIdx.x & 63;
    const int n = lane & 31;
    const int half = lane >> 5;
    RouteLane<RC, K, TPW> zl;
    load_z_operands<RC, K, TPW>(z, T, tb, n, half, zl);
    float lv[TPW][K];
    int32_t li[TPW][K];
#pragma unroll
    for (int g = 0; g < TPW; ++g) list_init<K>(lv[g], li[g]);
    for_each_tile<RC>(R2t, M, wb, we, n, half, [&](const bf16x8 (&a)[RC], int32_t e0, bool partial) {
#pragma unroll
        for (int g = 0; g < TPW; ++g) {
            f32x16 acc = zero_f32x16();
#pragma unroll
            for (int c = 0; c < RC; ++c) {
                acc = mfma_32x32x16(a[c], zl.zhi[g][c], acc);
                acc = mfma_32x32x16(a[c], zl.zlo[g][c], acc);
            }
            if (partial) mask_past_end(acc, e0, M, half);
            if (max16(acc) > lv[g][K - 1]) {
#pragma unroll
                for (int j = 0; j < 16; ++j) {
                    if (acc[j] > lv[g][K - 1])
                        list_insert_newer<K>(lv[g], li[g], acc[j], e0 + acc_row(j, half));
                }
            }
        }
    });
#pragma unroll
    for (int g = 0; g < TPW; ++g) list_merge_xor<K>(lv[g], li[g], 32);
#pragma unroll
    for (int s = kRouteWaves / 2; s >= 1; s >>= 1) {
        if (w >= s && w < 2 * s && half == 0) {
#pragma unroll
            for (int g = 0; g < TPW; ++g) {
#pragma unroll
                for (int j = 0; j < K; ++j) {
                    sm.sv[w - s][g][n][j] = lv[g][j];
                    sm.si[w - s][g][n][j] = li[g][j];
                }
            }
        }
        __syncthreads();
        if (w < s) {
#pragma unroll
            for (int g = 0; g < TPW; ++g) {
                float pv[K];
                int32_t pi[K];
#pragma unroll
                for (int j = 0; j < K; ++j) {
                    pv[j] = sm.sv[w][g][n][j];
                    pi[j] = sm.si[w][g][n][j];
                }
                list_merge<K>(lv[g], li[g], pv, pi);
            }
        }
        __syncthreads();
    }
    if (w == 0 && half == 0) {
#pragma unroll
        for (int g = 0; g < TPW; ++g) {
            const int64_t tok = ((int64_t)tb * TPW + g) * 32 + n;
            if (tok >= T) continue;
            if (FINAL) {
                store_selection<K>(lv[g], li[g], k, tok, idx, gate, topval);
            } else {
                const int64_t base = ((int64_t)chunk * T + tok) * K;
#pragma unroll
                for (int j = 0; j < K; ++j) {
                    part_v[base + j] = lv[g][j];
                    part_i[base + j] = li[g][j];
                }
            }
        }
    }
}

// Route one block of 32*TPW tokens over one chunk of the expert axis.
//
// Screened path, in three steps:
//  1. screening sweep with z_hi only (one MFMA per rank chunk): each lane keeps the maximum
//     of its experts' screened logits in BL buckets (tiles assigned round robin).  The K-th
//     largest of a token's NB >= 2K bucket maxima comes from K distinct experts, so it is a
//     lower bound on the token's K-th largest screened logit; lowered by a 2^-6 relative
//     margin it becomes the candidate threshold theta;
//  2. exact sweep with z_hi + z_lo: every logit above theta is appended to the lane's
//     private candidate slots in LDS (a shared per-token overflow area takes the rest);
//  3. each token's candidates are ranked under the selection order; ranks < K are the
//     result.
// Certificate: if a token has at least k candidates, every logit >= its k-th largest is above
// theta and therefore a candidate, so the result is exact.  Otherwise (or if the overflow
// area fills) the whole workgroup recomputes its tokens on the exact path.
template <int RC, int K, int TPW, bool FINAL>
__global__ __launch_bounds__(kRouteWaves * 64) void route_kernel(
    const float* __restrict__ z, const uint16_t* __restrict__ R2t, int32_t T, int32_t M,
    int32_t k, int32_t chunks, int32_t ntb, int32_t* __restrict__ idx, float* __restrict__ gate,
    float* __restrict__ topval, float* __restrict__ part_v, int32_t* __restrict__ part_i) {
    using S = RouteSmem<K, TPW>;
    constexpr int R = 16 * RC;
    constexpr int NT = S::NT, NB = S::NB, BL = S::BL, SL = S::S, OCAP = S::OCAP, LPT = S::LPT;
    constexpr int NTHREADS = kRouteWaves * 64;
    constexpr int TPT = NTHREADS / NT;  // threads per token when ranking bucket maxima
    __shared__ __attribute__((aligned(16))) char smem[S::bytes];
    auto& sm = *reinterpret_cast<typename S::Fast*>(smem);

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int n = lane & 31;
    const int half = lane >> 5;
    const int ls = w * 2 + half;  // this lane's index among the lanes of its token

    // Workgroup -> (token block, expert chunk).  With chunks a multiple of 8, the chunk's
    // low three bits equal the XCD the workgroup is dispatched to (workgroups are dealt to
    // the eight XCDs round robin), so each XCD's L2 only ever holds its own R2 slices, and
    // the token blocks of one chunk run back to back on the same XCD.
    int tb, chunk;
    if (chunks == 1) {
        tb = blockIdx.x;
        chunk = 0;
    } else {
        const int local = blockIdx.x >> 3;
        tb = local % ntb;
        chunk = (blockIdx.x & 7) + 8 * (local / ntb);
    }
    if (tid < NT) sm.ovf_count[tid] = 0;
    if (tid == 0) sm.fallback = 0;

    // z for the lane's token(s), split into hi/lo bf16 B operands.
    RouteLane<RC, K, TPW> zl;
    load_z_operands<RC, K, TPW>(z, T, tb, n, half, zl);

    // This wave's range of 32-expert tiles inside the chunk (wave-uniform).
    const int64_t Mt = (M + 31) / 32;
    const int64_t cb = Mt * chunk / chunks;
    const int64_t ce = Mt * (chunk + 1) / chunks;
    const int64_t wb = cb + (ce - cb) * w / kRouteWaves;
    const int64_t we = cb + (ce - cb) * (w + 1) / kRouteWaves;

    // ---- step 1: screening maxima
    float bm[TPW][BL];
#pragma unroll
    for (int g = 0; g < TPW; ++g)
#pragma unroll
        for (int b = 0; b < BL; ++b) bm[g][b] = -__builtin_huge_valf();
    for_each_tile<RC>(R2t, M, wb, we, n, half, [&](const bf16x8 (&a)[RC], int32_t e0, bool partial) {
        const int bsel = BL == 1 ? 0 : (int)(((e0 >> 5) - wb) % BL);
        f32x16 acc[TPW];
#pragma unroll
        for (int g = 0; g < TPW; ++g) {
            acc[g] = zero_f32x16();
#pragma unroll
            for (int c = 0; c < RC; ++c) acc[g] = mfma_32x32x16(a[c], zl.zhi[g][c], acc[g]);
        }
#pragma unroll
        for (int g = 0; g < TPW; ++g) {
            if (partial) mask_past_end(acc[g], e0, M, half);
            const float mx = max16(acc[g]);
#pragma unroll
            for (int b = 0; b < BL; ++b)
                if (b == bsel) bm[g][b] = fmaxf(bm[g][b], mx);
        }
    });
#pragma unroll
    for (int g = 0; g < TPW; ++g)
#pragma unroll
        for (int b = 0; b < BL; ++b) sm.bucket[g * 32 + n][ls * BL + b] = bm[g][b];
    __syncthreads();

    // theta per token: the bucket maximum of rank K-1 (ties ranked by position), lowered.
    {
        const int tt = tid / TPT, sub = tid % TPT;
        for (int q = sub; q < NB; q += TPT) {
            const float v = sm.bucket[tt][q];
            int rank = 0;
            for (int i = 0; i < NB; ++i) {
                const float u = sm.bucket[tt][i];
                rank += (u > v || (u == v && i < q)) ? 1 : 0;
            }
            if (rank == K - 1) sm.theta[tt] = v - fabsf(v) * 0x1p-6f;
        }
    }
    __syncthreads();

    // ---- step 2: exact sweep, candidates above theta into the lane's slots
    float th[TPW];
    int32_t cnt[TPW];
#pragma unroll
    for (int g = 0; g < TPW; ++g) {
        th[g] = sm.theta[g * 32 + n];
        cnt[g] = 0;
    }
    for_each_tile<RC>(R2t, M, wb, we, n, half, [&](const bf16x8 (&a)[RC], int32_t e0, bool partial) {
        f32x16 acc[TPW];
#pragma unroll
        for (int g = 0; g < TPW; ++g) {
            acc[g] = zero_f32x16();
#pragma unroll
            for (int c = 0; c < RC; ++c) {
                acc[g] = mfma_32x32x16(a[c], zl.zhi[g][c], acc[g]);
                acc[g] = mfma_32x32x16(a[c], zl.zlo[g][c], acc[g]);
            }
        }
#pragma unroll
        for (int g = 0; g < TPW; ++g) {
            if (partial) mask_past_end(acc[g], e0, M, half);
            if (max16(acc[g]) > th[g]) {
                const int tl = g * 32 + n;
#pragma unroll
                for (int j = 0; j < 16; ++j) {
                    if (acc[g][j] > th[g]) {
                        const int32_t e = e0 + acc_row(j, half);
                        if (cnt[g] < SL) {
                            sm.slot_v[tl][ls * SL + cnt[g]] = acc[g][j];
                            sm.slot_i[tl][ls * SL + cnt[g]] = e;
                        } else {
                            const int o = atomicAdd(&sm.ovf_count[tl], 1);
                            if (o < OCAP) {
                                sm.ovf_v[tl][o] = acc[g][j];
                                sm.ovf_i[tl][o] = e;
                            }
                        }
                        ++cnt[g];
                    }
                }
            }
        }
    });
#pragma unroll
    for (int g = 0; g < TPW; ++g) sm.lane_count[g * 32 + n][ls] = cnt[g] < SL ? cnt[g] : SL;
    __syncthreads();

    // ---- step 3: one thread per token keeps the best K of its candidates; certificate
    float lv[K];
    int32_t li[K];
    if (tid < NT) {
        list_init<K>(lv, li);
        int P = 0;
        for (int l = 0; l < LPT; ++l) {
            const int c = sm.lane_count[tid][l];
            P += c;
            for (int q = 0; q < c; ++q) {
                const float v = sm.slot_v[tid][l * SL + q];
                const int32_t e = sm.slot_i[tid][l * SL + q];
                if (better(v, e, lv[K - 1], li[K - 1])) list_insert<K>(lv, li, v, e);
            }
        }
        const int ovf = sm.ovf_count[tid];
        const int no = ovf < OCAP ? ovf : OCAP;
        P += no;
        for (int q = 0; q < no; ++q) {
            const float v = sm.ovf_v[tid][q];
            const int32_t e = sm.ovf_i[tid][q];
            if (better(v, e, lv[K - 1], li[K - 1])) list_insert<K>(lv, li, v, e);
        }
        const bool all_in = sm.theta[tid] == -__builtin_huge_valf();  // nothing screened out
        const bool tok_ok = (int64_t)tb * NT + tid < T;
        if (tok_ok && (ovf > OCAP || (P < k && !all_in))) atomicOr(&sm.fallback, 1);
    }
    __syncthreads();

    if (sm.fallback) {  // workgroup-uniform
        __syncthreads();
        route_exact<RC, K, TPW, FINAL>(z, R2t, T, M, k, tb, chunk, wb, we, w, smem, idx, gate,
                                       topval, part_v, part_i);
        return;
    }
    if (tid < NT) {
        const int64_t tok = (int64_t)tb * NT + tid;
        if (tok < T) {
            if (FINAL) {
                store_selection<K>(lv, li, k, tok, idx, gate, topval);
            } else {
                const int64_t base = ((int64_t)chunk * T + tok) * K;
#pragma unroll
                for (int j = 0; j < K; ++j) {
                    part_v[base + j] = lv[j];
                    part_i[base + j] = li[j];
                }
            }
        }
    }
}

// ------------------------------------------------------------------------------ merge
// One wave per token: lane l merges chunk lists l, l+64, ...; then a butterfly over lanes.
template <int K>
__global__ __launch_bounds__(256) void merge_kernel(const float* __restrict__ part_v,
                                                    const int32_t* __restrict__ part_i, int32_t T,
                                                    int32_t chunks, int32_t k,
                                                    int32_t* __restrict__ idx,
                                                    float* __restrict__ gate,
                                                    float* __restrict__ topval) {
    const int lane = threadIdx.x & 63;
    const int64_t tok = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    if (tok >= T) return;  // wave-uniform
    float v[K];
    int32_t ix[K];
    list_init<K>(v, ix);
    for (int c = lane; c < chunks; c += 64) {
        const int64_t base = ((int64_t)c * T + tok) * K;
        float pv[K];
        int32_t pi[K];
#pragma unroll
        for (int j = 0; j < K; ++j) {
            pv[j] = part_v[base + j];
            pi[j] = part_i[base + j];
        }
        list_merge<K>(v, ix, pv, pi);
    }
    for (int s = 1; s < 64 && s < chunks; s <<= 1) list_merge_xor<K>(v, ix, s);
    if (lane == 0) store_selection<K>(v, ix, k, tok, idx, gate, topval);
}

// ------------------------------------------------------------------------------ planning
static int pow2_at_least(int k) {
    int K = 1;
    while (K < k) K <<= 1;
    return K;
}

static size_t align256(size_t b) { return (b + 255) & ~(size_t)255; }

bool lowrank_make_plan(int64_t T, int32_t h, int32_t r, int32_t M, int32_t k, int32_t m_chunks,
                       LowrankPlan* p) {
    LowrankPlan q{};
    q.RC = r / 16;
    q.RT = (q.RC + 1) / 2;
    q.K = pow2_at_least(k);
    q.TPW = (q.RC <= 4 && q.K <= 8) ? 2 : 1;
    q.ntb = (int32_t)((T + 32 * q.TPW - 1) / (32 * q.TPW));
    const int64_t Mt = ((int64_t)M + 31) / 32;
    if (m_chunks > 0) {
        q.chunks = m_chunks;
    } else {
        const int64_t r2_bytes = (int64_t)M * r * 2;
        int64_t C = 1;
        if (r2_bytes > (int64_t)3 << 20) C = 8 * ((r2_bytes + ((int64_t)8 << 20) - 1) >> 23);
        while ((int64_t)q.ntb * C < 256) {
            const int64_t nextC = (C == 1) ? 8 : 2 * C;
            if (nextC > 1024 || Mt < nextC * kRouteWaves) break;
            C = nextC;
        }
        q.chunks = (int32_t)C;
    }
    if (q.chunks != 1 && (q.chunks % 8 != 0 || q.chunks > 1024)) return false;
    const int32_t S = h / 16;
    const int64_t TG = (T + 31) / 32;
    int64_t hs = (256 + TG - 1) / TG;
    hs = hs < 1 ? 1 : hs;
    const int64_t max_hs = S / 4 > 0 ? S / 4 : 1;
    if (hs > max_hs) hs = max_hs;
    q.hsplit = (int32_t)hs;
    q.steps_per_split = (S + q.hsplit - 1) / q.hsplit;
    const size_t zbytes = (size_t)T * r * sizeof(float);
    size_t off = 0;
    q.off_zparts = off;
    off += align256(zbytes * q.hsplit);
    if (q.hsplit > 1) {
        q.off_z = off;
        off += align256(zbytes);
    } else {
        q.off_z = q.off_zparts;
    }
    if (q.chunks > 1) {
        const size_t pbytes = (size_t)q.chunks * T * q.K;
        q.off_part_v = off;
        off += align256(pbytes * sizeof(float));
        q.off_part_i = off;
        off += align256(pbytes * sizeof(int32_t));
    }
    q.workspace_bytes = off;
    *p = q;
    return true;
}

// ------------------------------------------------------------------------------ launch
template <int RT>
static void launch_zpass(const LowrankPlan& p, const uint16_t* x, const uint16_t* R1t, float* zparts,
                         int64_t T, int32_t h, int32_t r, hipStream_t st) {
    dim3 grid((unsigned)((T + 31) / 32), (unsigned)p.hsplit);
    hipLaunchKernelGGL(zpass_kernel<RT>, grid, dim3(256), 0, st, x, R1t, zparts, (int32_t)T, h, r,
                       p.steps_per_split);
}

template <int RC, int K>
static void launch_route(const LowrankPlan& p, const float* z, const uint16_t* R2t, int64_t T,
                         int32_t M, int32_t k, int32_t* idx, float* gate, float* topval,
                         float* pv, int32_t* pi, hipStream_t st) {
    constexpr int TPW = (RC <= 4 && K <= 8) ? 2 : 1;
    dim3 grid((unsigned)((int64_t)p.ntb * p.chunks)), block(kRouteWaves * 64);
    if (p.chunks == 1)
        hipLaunchKernelGGL((route_kernel<RC, K, TPW, true>), grid, block, 0, st, z, R2t,
                           (int32_t)T, M, k, p.chunks, p.ntb, idx, gate, topval, pv, pi);
    else
        hipLaunchKernelGGL((route_kernel<RC, K, TPW, false>), grid, block, 0, st, z, R2t,
                           (int32_t)T, M, k, p.chunks, p.ntb, idx, gate, topval, pv, pi);
}

template <int RC>
static bool dispatch_route_k(const LowrankPlan& p, const float* z, const uint16_t* R2t, int64_t T,
                             int32_t M, int32_t k, int32_t* idx, float* gate, float* topval,
                             float* pv, int32_t* pi, hipStream_t st) {
    switch (p.K) {
        case 1: launch_route<RC, 1>(p, z, R2t, T, M, k, idx, gate, topval, pv, pi, st); return true;
        case 2: launch_route<RC, 2>(p, z, R2t, T, M, k, idx, gate, topval, pv, pi, st); return true;
        case 4: launch_route<RC, 4>(p, z, R2t, T, M, k, idx, gate, topval, pv, pi, st); return true;
        case 8: launch_route<RC, 8>(p, z, R2t, T, M, k, idx, gate, topval, pv, pi, st); return true;
        case 16: launch_route<RC, 16>(p, z, R2t, T, M, k, idx, gate, topval, pv, pi, st); return true;
        case 32: launch_route<RC, 32>(p, z, R2t, T, M, k, idx, gate, topval, pv, pi, st); return true;
    }
    return false;
}

template <int K>
static void launch_merge(const LowrankPlan& p, const float* pv, const int32_t* pi, int64_t T,
                         int32_t k, int32_t* idx, float* gate, float* topval, hipStream_t st) {
    dim3 grid((unsigned)((T + 3) / 4));
    hipLaunchKernelGGL(merge_kernel<K>, grid, dim3(256), 0, st, pv, pi, (int32_t)T, p.chunks, k,
                       idx, gate, topval);
}

hipError_t lowrank_launch(const LowrankPlan& p, const uint16_t* x, const uint16_t* R1t,
                          const uint16_t* R2t, int64_t T, int32_t h, int32_t r, int32_t M,
                          int32_t k, int32_t* idx, float* gate, float* topval, void* workspace,
                          hipStream_t st) {
    char* ws = static_cast<char*>(workspace);
    float* zparts = reinterpret_cast<float*>(ws + p.off_zparts);
    float* z = reinterpret_cast<float*>(ws + p.off_z);
    float* pv = p.chunks > 1 ? reinterpret_cast<float*>(ws + p.off_part_v) : nullptr;
    int32_t* pi = p.chunks > 1 ? reinterpret_cast<int32_t*>(ws + p.off_part_i) : nullptr;

    switch (p.RT) {
        case 1: launch_zpass<1>(p, x, R1t, zparts, T, h, r, st); break;
        case 2: launch_zpass<2>(p, x, R1t, zparts, T, h, r, st); break;
        case 4: launch_zpass<4>(p, x, R1t, zparts, T, h, r, st); break;
        default: return hipErrorInvalidValue;
    }
    if (p.hsplit > 1) {
        const int64_t n = T * r;
        const unsigned blocks = (unsigned)((n + 255) / 256 < 4096 ? (n + 255) / 256 : 4096);
        hipLaunchKernelGGL(zreduce_kernel, dim3(blocks), dim3(256), 0, st, zparts, z, n,
                           p.hsplit);
    }
    bool ok = false;
    switch (p.RC) {
        case 1: ok = dispatch_route_k<1>(p, z, R2t, T, M, k, idx, gate, topval, pv, pi, st); break;
        case 2: ok = dispatch_route_k<2>(p, z, R2t, T, M, k, idx, gate, topval, pv, pi, st); break;
        case 4: ok = dispatch_route_k<4>(p, z, R2t, T, M, k, idx, gate, topval, pv, pi, st); break;
        case 8: ok = dispatch_route_k<8>(p, z, R2t, T, M, k, idx, gate, topval, pv, pi, st); break;
    }
    if (!ok) return hipErrorInvalidValue;
    if (p.chunks > 1) {
        switch (p.K) {
            case 1: launch_merge<1>(p, pv, pi, T, k, idx, gate, topval, st); break;
            case 2: launch_merge<2>(p, pv, pi, T, k, idx, gate, topval, st); break;
            case 4: launch_merge<4>(p, pv, pi, T, k, idx, gate, topval, st); break;
            case 8: launch_merge<8>(p, pv, pi, T, k, idx, gate, topval, st); break;
            case 16: launch_merge<16>(p, pv, pi, T, k, idx, gate, topval, st); break;
            case 32: launch_merge<32>(p, pv, pi, T, k, idx, gate, topval, st); break;
            default: return hipErrorInvalidValue;
        }
    }
    return hipGetLastError();
}

}  // namespace more
