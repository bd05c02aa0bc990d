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
#pragma unroll 4
    for (int s = ws0; s < ws1; ++s) {
        bf16x8 b = tok_ok ? load_bf16x8(xrow + 16 * s) : zero_bf16x8();
#pragma unroll
        for (int pt = 0; pt < RT; ++pt) {
            const int row = 32 * pt + prow;
            bf16x8 a = row < r ? load_bf16x8(R1t + (int64_t)row * h + 16 * s + 8 * half)
                               : zero_bf16x8();
            acc[pt] = mfma_32x32x16(a, b, acc[pt]);
        }
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

template <int RC, int K, int TPW, bool FINAL>
__global__ __launch_bounds__(kRouteWaves * 64) void route_kernel(
    const float* __restrict__ z, const uint16_t* __restrict__ R2t, int32_t T, int32_t M,
    int32_t k, int32_t chunks, int32_t ntb, int32_t* __restrict__ idx, float* __restrict__ gate,
    float* __restrict__ topval, float* __restrict__ part_v, int32_t* __restrict__ part_i) {
    constexpr int R = 16 * RC;
    const int lane = threadIdx.x & 63;
    const int w = threadIdx.x >> 6;
    const int n = lane & 31;
    const int half = lane >> 5;

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

    // z for the lane's token(s), split into hi/lo bf16 B operands.
    bf16x8 zhi[TPW][RC], zlo[TPW][RC];
#pragma unroll
    for (int g = 0; g < TPW; ++g) {
        const int64_t tok = ((int64_t)tb * TPW + g) * 32 + n;
#pragma unroll
        for (int c = 0; c < RC; ++c) {
            float v[8];
            if (tok < T) {
                const f32x4* p = reinterpret_cast<const f32x4*>(z + tok * R + 16 * c + 8 * half);
                f32x4 a0 = p[0], a1 = p[1];
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    v[q] = a0[q];
                    v[4 + q] = a1[q];
                }
            } else {
#pragma unroll
                for (int q = 0; q < 8; ++q) v[q] = 0.0f;
            }
            split_hi_lo(v, zhi[g][c], zlo[g][c]);
        }
    }

    // This wave's range of 32-expert tiles.
    const int64_t Mt = (M + 31) / 32;
    const int64_t cb = Mt * chunk / chunks;
    const int64_t ce = Mt * (chunk + 1) / chunks;
    const int64_t wb = cb + (ce - cb) * w / kRouteWaves;
    const int64_t we = cb + (ce - cb) * (w + 1) / kRouteWaves;

    float lv[TPW][K];
    int32_t li[TPW][K];
#pragma unroll
    for (int g = 0; g < TPW; ++g) list_init<K>(lv[g], li[g]);

    // A operand of tile t: expert row t*32 + n, K half `half` of each 16-wide rank chunk.
    auto load_a = [&](int64_t t, bf16x8 (&a)[RC]) {
        const int64_t e = t * 32 + n;
        if (e < M) {
            const uint16_t* p = R2t + e * R + 8 * half;
#pragma unroll
            for (int c = 0; c < RC; ++c) a[c] = load_bf16x8(p + 16 * c);
        } else {
#pragma unroll
            for (int c = 0; c < RC; ++c) a[c] = zero_bf16x8();
        }
    };

    bf16x8 a_cur[RC], a_nxt[RC];
    if (wb < we) load_a(wb, a_cur);
    for (int64_t t = wb; t < we; ++t) {
        if (t + 1 < we) load_a(t + 1, a_nxt);
        const int32_t e0 = (int32_t)(t * 32);
#pragma unroll
        for (int g = 0; g < TPW; ++g) {
            f32x16 acc = zero_f32x16();
#pragma unroll
            for (int c = 0; c < RC; ++c) {
                acc = mfma_32x32x16(a_cur[c], zhi[g][c], acc);
                acc = mfma_32x32x16(a_cur[c], zlo[g][c], acc);
            }
            if (e0 + 32 > M) {  // last tile: experts past M do not exist
#pragma unroll
                for (int j = 0; j < 16; ++j)
                    if (e0 + acc_row(j, half) >= M) acc[j] = -__builtin_huge_valf();
            }
            float mx = acc[0];
#pragma unroll
            for (int j = 1; j < 16; ++j) mx = fmaxf(mx, acc[j]);
            if (mx > lv[g][K - 1]) {
#pragma unroll
                for (int j = 0; j < 16; ++j) {
                    if (acc[j] > lv[g][K - 1])
                        list_insert_newer<K>(lv[g], li[g], acc[j], e0 + acc_row(j, half));
                }
            }
        }
#pragma unroll
        for (int c = 0; c < RC; ++c) a_cur[c] = a_nxt[c];
    }

    // The two K halves of a lane pair saw disjoint expert rows of the same token.
#pragma unroll
    for (int g = 0; g < TPW; ++g) list_merge_xor<K>(lv[g], li[g], 32);

    // Tree merge across the waves of the workgroup through LDS.
    __shared__ float sv[kRouteWaves / 2][TPW][32][K];
    __shared__ int32_t si[kRouteWaves / 2][TPW][32][K];
#pragma unroll
    for (int s = kRouteWaves / 2; s >= 1; s >>= 1) {
        if (w >= s && w < 2 * s && half == 0) {
#pragma unroll
            for (int g = 0; g < TPW; ++g) {
#pragma unroll
                for (int j = 0; j < K; ++j) {
                    sv[w - s][g][n][j] = lv[g][j];
                    si[w - s][g][n][j] = li[g][j];
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
                    pv[j] = sv[w][g][n][j];
                    pi[j] = si[w][g][n][j];
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
    q.TPW = (q.RC <= 4 && q.K <= 16) ? 2 : 1;
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
    constexpr int TPW = (RC <= 4 && K <= 16) ? 2 : 1;
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
