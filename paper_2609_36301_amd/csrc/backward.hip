// Training backward pass of the low-rank router for gfx950 (Appendix "Pseudocode", backward
// pass: eqs. app_chain, app_jac, app_kernelgrad and the backward algorithm with recompute).
// With l = z R2, z = x R1, P_te = exp(l_te - m_t) / Z_t from the saved statistics, the gradient
// dtop of the loss with respect to the selected logits and pbar with respect to psum:
//   g_t     = sum_e pbar_e P_te                       (one scalar per token)
//   ybar_te = P_te (pbar_e - g_t) + dtop at the selected experts
//   dz      = ybar R2^T,  dR2 = z^T ybar,  dx = dz R1^T,  dR1 = x^T dz
// and no T x M matrix is written: the logits are recomputed tile by tile on the matrix cores.
//
// Kernels of one call (the balancing kernels run only when pbar is given):
//   zonly            z = x R1 (fp32, the z pass of the routing call)
//   bwd_prep         z' = z log2(e) as bf16 hi/lo rows, bf16(z) rows and the token bias
//                    -(m log2(e) + log2 Z); bwd_r1_transpose: R1 as [h][r]
//   bwd_tok<false>   sweep 1, token-major: per (expert split, token) sum_e pbar_e P_te
//   bwd_colsum       g = the split sums in split order
//   bwd_tok<true>    sweep 2, token-major: ybar tile by tile, dz partials per expert split,
//                    summed by bwd_colsum
//   bwd_exp          sweep 2 again, expert-major: ybar tile by tile, dR2 partials per token split
//   dispatch         the selections sorted by expert (Sort + Count kernels)
//   bwd_sparse       the dtop z terms of dR2, a segmented sum over chunks of the sorted selections
//   bwd_dr2          dR2 = partials in order + the dtop terms
//   bwd_dz           dz = the dense sum + the selected experts' dtop R2 rows; dz as bf16 hi/lo rows
//                    [T][2r] and as transposed hi/lo rows [2][r][T]
//   bwd_dx           dx = dz R1^T (dz as hi + lo)
//   bwd_dr1          dR1 = x^T dz over token splits, summed by bwd_colsum in split order
// The paper's algorithm computes dz and dR2 in one sweep per token block and lets token blocks
// add into dR2; here two sweeps (one token-major, one expert-major) each own their output, so
// nothing is added atomically and every sum runs in a fixed order: a shape gives the same bits
// on every run.
//
// Numerics.  The logits are recomputed as in the training forward pass (z' as bf16 hi + lo on
// the matrix cores, the bias entering through the accumulator input, 2^x by v_exp_f32).  The
// dense logit gradient P (pbar - g) is rounded to bf16 for the two contractions, which also
// read bf16(z) (dR2) and the bf16 rows of R2 (dz), with fp32 accumulation; the sparse dtop
// terms use fp32 z and fp32 dtop; dx and dR1 read dz as bf16 hi + lo (about 16 significant
// bits) and the exact bf16 x and R1.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "device_common.h"
#include "lowrank.h"
#include "backward.h"

namespace more {

namespace {

constexpr float kBwLog2e = 1.44269504088896340736f;
constexpr float kBwNoToken = -0x1p100f;  // bias of rows past T: 2^(finite + this) = 0

constexpr int kBwWaves = 8;
constexpr int kBwThreads = 64 * kBwWaves;
// Waves per workgroup and 32-token groups per wave in the token-major sweeps.  The r = 64 dz
// sweep holds one token group per wave: two would not fit two waves per SIMD, and one wave per
// SIMD with two groups (four waves per workgroup, up to 512 registers each) measured 45% slower.
template <int RC, bool DZ>
constexpr int bw_waves() { return 8; }
template <int RC, bool DZ>
constexpr int bw_tpw() { return (RC == 4 && DZ) ? 1 : 2; }
constexpr int kBwStageE = 128;   // experts per LDS stage of the token-major sweeps
constexpr int kBwNE = 2;         // 32-expert tiles per wave in the expert-major sweep
constexpr int kBwStageT = 128;   // tokens per LDS stage of the expert-major sweep
constexpr int kBwFoldParts = 16; // at most this many partials: summed by their consumers

__device__ __forceinline__ float bw_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// eight fp32 -> bf16x8 (round to nearest even)
__device__ __forceinline__ bf16x8 pack_bf16x8(const float* v) {
    bf16x8 o;
#pragma unroll
    for (int i = 0; i < 8; ++i) o[i] = (__bf16)v[i];
    return o;
}

// Two 8-byte LDS pieces (four bf16 each) as one operand.
__device__ __forceinline__ bf16x8 lds_two_quads(const uint16_t* p0, const uint16_t* p1) {
    const uint2 a = *reinterpret_cast<const uint2*>(p0);
    const uint2 b = *reinterpret_cast<const uint2*>(p1);
    return __builtin_bit_cast(bf16x8, u32x4{a.x, a.y, b.x, b.y});
}

}  // namespace

// ------------------------------------------------------------------------------ prep
// One thread per element of z [T][r]: zhl [T][2r] = bf16(z'), bf16(z' - bf16(z')) with
// z' = z log2(e); zb [T][r] = bf16(z); bias[t] = -(m log2(e) + log2 Z) (when m is given).
__global__ __launch_bounds__(256) void bwd_prep_kernel(const float* __restrict__ z,
                                                       const float* __restrict__ m,
                                                       const float* __restrict__ Z, int32_t T,
                                                       int32_t r, uint16_t* __restrict__ zhl,
                                                       uint16_t* __restrict__ zb,
                                                       float* __restrict__ bias) {
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i >= (int64_t)T * r) return;
    const int64_t t = i / r;
    const int32_t j = (int32_t)(i - t * r);
    const float zv = z[i];
    const float v = zv * kBwLog2e;
    const __bf16 hb = (__bf16)v;
    const __bf16 lb = (__bf16)(v - (float)hb);
    zhl[t * 2 * r + j] = __builtin_bit_cast(uint16_t, hb);
    zhl[t * 2 * r + r + j] = __builtin_bit_cast(uint16_t, lb);
    zb[i] = __builtin_bit_cast(uint16_t, (__bf16)zv);
    if (m && j == 0) bias[t] = -(m[t] * kBwLog2e + log2f(Z[t]));
}

// R1 [h][r] from R1t [r][h].
__global__ __launch_bounds__(256) void bwd_r1_transpose_kernel(const uint16_t* __restrict__ R1t,
                                                               int32_t h, int32_t r,
                                                               uint16_t* __restrict__ R1) {
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;  // index into R1
    if (i >= (int64_t)h * r) return;
    const int64_t c = i / r;
    const int32_t j = (int32_t)(i - c * r);
    R1[i] = R1t[(int64_t)j * h + c];
}

// ------------------------------------------------------------------------------ token-major
// Workgroup (token block, expert split); the block's tokens are WT slots of TPW x 32 tokens, and
// the waves of a slot (WE = 8 / WT of them) take the expert tiles of each stage in turn.  A
// wave holds z'_hi and z'_lo of its tokens as B operands (token columns) and reads the expert
// rows of R2t from LDS as A operands, so a lane owns one token column and sixteen expert rows
// of each 32 x 32 logit tile; the token's bias enters through the accumulator input.
//   DZ = false: per lane sum_e pbar_e 2^(l' + bias) -> gpart[(split WE + we)][t]
//   DZ = true : ybar = P (pbar_e - g_t) as bf16 A operands (token rows, expert K order as the
//               accumulator holds them) against R2^T pieces read from a transposed LDS copy
//               with the same K order -> dz partials dzpart[(split WE + we)][t][r]
template <int RC, int NW>
struct TokCfg {
    static constexpr int THREADS = 64 * NW;
    static constexpr int R = 16 * RC;
    static constexpr int RB = (R + 31) / 32;       // 32-row blocks of the rank axis
    static constexpr int RP = R + 8;               // LDS pitch of an expert row (bf16)
    static constexpr int CP = kBwStageE + 8;       // LDS pitch of a transposed row (bf16)
    static constexpr int PIECES = kBwStageE * R / 8;  // 16-byte pieces of R2t per stage
    static constexpr int PPT = (PIECES + THREADS - 1) / THREADS;
};

template <int RC, bool DZ>
__global__ __launch_bounds__((64 * bw_waves<RC, DZ>()), 1) void bwd_tok_kernel(
    const uint16_t* __restrict__ zhl, const float* __restrict__ bias,
    const float* __restrict__ gtok, const float* __restrict__ gpart, int32_t gparts,
    float* gsummed, const float* __restrict__ pbar,
    const uint16_t* __restrict__ R2t, int32_t T, int32_t M, int32_t WT, int32_t splits,
    float* __restrict__ out) {
    constexpr int NW = bw_waves<RC, DZ>();
    using C = TokCfg<RC, NW>;
    constexpr int R = C::R, RB = C::RB, RP = C::RP, CP = C::CP, TPW = bw_tpw<RC, DZ>();
    constexpr int NT = C::THREADS;
    constexpr int TILES = kBwStageE / 32;
    __shared__ __attribute__((aligned(16))) uint16_t rows[2][kBwStageE * RP];
    __shared__ __attribute__((aligned(16))) uint16_t rowsT[DZ ? 2 : 1][DZ ? R * CP : 8];
    __shared__ __attribute__((aligned(16))) float pbs[2][kBwStageE];
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int n = lane & 31, half = lane >> 5;
    const int WE = NW / WT;
    const int wt = w % WT, we = w / WT;
    const int32_t split = (int32_t)(blockIdx.x % (unsigned)splits);
    const int64_t tb = blockIdx.x / (unsigned)splits;
    const int32_t Mt = (M + 31) / 32;
    const int32_t tile0 = (int32_t)((int64_t)Mt * split / splits);
    const int32_t tile1 = (int32_t)((int64_t)Mt * (split + 1) / splits);
    const int nstages = (tile1 - tile0 + TILES - 1) / TILES;
    const int64_t first = (tb * WT + wt) * (32 * TPW);  // first token of this wave

    // the wave's tokens as B operands, its bias and g
    bf16x8 zh[TPW][RC], zl[TPW][RC];
    float bt[TPW], gt[TPW];
#pragma unroll
    for (int g = 0; g < TPW; ++g) {
        const int64_t t = first + 32 * g + n;
        const bool ok = t < T;
        const uint16_t* zr = zhl + (ok ? t : 0) * (2 * R) + 8 * half;
#pragma unroll
        for (int c = 0; c < RC; ++c) {
            const bf16x8 hv = load_bf16x8(zr + 16 * c);
            const bf16x8 lv = load_bf16x8(zr + R + 16 * c);
            zh[g][c] = ok ? hv : zero_bf16x8();
            zl[g][c] = ok ? lv : zero_bf16x8();
        }
        bt[g] = ok ? bias[t] : kBwNoToken;
        // g: the summed array, or (few partials) their sum in order, which the first expert
        // split's first wave column stores for the expert-major sweep
        float gsum = 0.0f;
        if (DZ && ok) {
            if (gparts > 0) {
                for (int32_t p = 0; p < gparts; ++p) gsum += gpart[(int64_t)p * T + t];
                if (split == 0 && we == 0 && half == 0) gsummed[t] = gsum;
            } else {
                gsum = gtok[t];
            }
        }
        gt[g] = gsum;
    }

    // stage loads: piece p = expert p / (R / 8) of the stage, rank piece p % (R / 8)
    u32x4 rg[C::PPT];
    float rp = 0.0f;
    auto gload = [&](int st) __attribute__((always_inline)) {
        const int64_t e0 = (int64_t)(tile0 + st * TILES) * 32;
#pragma unroll
        for (int i = 0; i < C::PPT; ++i) {
            const int p = tid + i * NT;
            int64_t e = e0 + p / (R / 8);
            e = e < M ? e : M - 1;  // rows past M: masked out of the sums below
            if (p < C::PIECES)
                rg[i] = *reinterpret_cast<const u32x4*>(R2t + e * R + 8 * (p % (R / 8)));
        }
        if (tid < kBwStageE) {
            const int64_t e = e0 + tid;
            rp = e < M ? pbar[e] : 0.0f;
        }
    };
    auto stash = [&](int buf) __attribute__((always_inline)) {
#pragma unroll
        for (int i = 0; i < C::PPT; ++i) {
            const int p = tid + i * NT;
            if (p < C::PIECES) {
                const int el = p / (R / 8), q = p % (R / 8);
                *reinterpret_cast<u32x4*>(&rows[buf][el * RP + 8 * q]) = rg[i];
                if constexpr (DZ) {
                    const uint16_t* v = reinterpret_cast<const uint16_t*>(&rg[i]);
#pragma unroll
                    for (int u = 0; u < 8; ++u) rowsT[buf][(8 * q + u) * CP + el] = v[u];
                }
            }
        }
        if (tid < kBwStageE) pbs[buf][tid] = rp;
    };

    float gs[TPW];
    f32x16 dz[TPW][RB];
#pragma unroll
    for (int g = 0; g < TPW; ++g) {
        gs[g] = 0.0f;
#pragma unroll
        for (int b = 0; b < RB; ++b) dz[g][b] = zero_f32x16();
    }
    const bool active = first < T;  // wave-uniform; idle waves still stage experts
    if (nstages > 0) {              // workgroup-uniform
        gload(0);
        stash(0);
        if (nstages > 1) gload(1);
        __syncthreads();
        for (int st = 0; st < nstages; ++st) {
            const int buf = st & 1;
            if (active) {
                for (int tl = we; tl < TILES; tl += WE) {
                    const int32_t tile = tile0 + st * TILES + tl;
                    if (tile >= tile1) break;
                    bf16x8 a[RC];
                    const uint16_t* ar = &rows[buf][(tl * 32 + n) * RP + 8 * half];
#pragma unroll
                    for (int c = 0; c < RC; ++c) a[c] = load_bf16x8(ar + 16 * c);
                    // rows past M in the last tile: no probability
                    const bool ragged = (tile + 1) * 32 > M;
                    bf16x8 rt[2][RB];
                    if constexpr (DZ) {
#pragma unroll
                        for (int q2 = 0; q2 < 2; ++q2)
#pragma unroll
                            for (int b = 0; b < RB; ++b) {
                                int j = 32 * b + n;
                                j = j < R ? j : R - 1;  // columns past r: never stored
                                const uint16_t* pr = &rowsT[buf][j * CP + tl * 32 + 16 * q2 + 4 * half];
                                rt[q2][b] = lds_two_quads(pr, pr + 8);
                            }
                    }
#pragma unroll
                    for (int g = 0; g < TPW; ++g) {
                        // two independent chains (z'_hi with the bias, z'_lo), added at the end
                        f32x16 acc, acl = zero_f32x16();
#pragma unroll
                        for (int i = 0; i < 16; ++i) acc[i] = bt[g];
#pragma unroll
                        for (int c = 0; c < RC; ++c) {
                            acc = mfma_32x32x16(a[c], zh[g][c], acc);
                            acl = mfma_32x32x16(a[c], zl[g][c], acl);
                        }
                        acc += acl;
                        // pbar of this lane's expert rows (re-read per group: fewer live registers)
                        float pb[16];
#pragma unroll
                        for (int q = 0; q < 4; ++q) {
                            const f32x4 v = *reinterpret_cast<const f32x4*>(
                                &pbs[buf][tl * 32 + 8 * q + 4 * half]);
#pragma unroll
                            for (int u = 0; u < 4; ++u) pb[4 * q + u] = v[u];
                        }
                        float p[16];
#pragma unroll
                        for (int i = 0; i < 16; ++i) p[i] = bw_exp2(acc[i]);
                        if (ragged) {
#pragma unroll
                            for (int i = 0; i < 16; ++i)
                                p[i] = tile * 32 + acc_row(i, half) < M ? p[i] : 0.0f;
                        }
                        if constexpr (!DZ) {
                            float s = 0.0f;
#pragma unroll
                            for (int i = 0; i < 16; ++i) s += pb[i] * p[i];
                            gs[g] += s;
                        } else {
                            float y[16];
#pragma unroll
                            for (int i = 0; i < 16; ++i) y[i] = p[i] * (pb[i] - gt[g]);
                            const bf16x8 y0 = pack_bf16x8(y), y1 = pack_bf16x8(y + 8);
#pragma unroll
                            for (int b = 0; b < RB; ++b) {
                                dz[g][b] = mfma_32x32x16(y0, rt[0][b], dz[g][b]);
                                dz[g][b] = mfma_32x32x16(y1, rt[1][b], dz[g][b]);
                            }
                        }
                    }
                }
            }
            if (st + 1 < nstages) stash(buf ^ 1);
            if (st + 2 < nstages) gload(st + 2);
            __syncthreads();
        }
    }
    const int64_t slot = (int64_t)split * WE + we;
    if constexpr (!DZ) {
#pragma unroll
        for (int g = 0; g < TPW; ++g) {
            const float tot = sum_pair32(gs[g]);  // the two lane halves hold disjoint rows
            const int64_t t = first + 32 * g + n;
            if (half == 0 && t < T) out[slot * T + t] = tot;
        }
    } else {
        // lane: rank column 32 b + n, token rows acc_row(i, half) of group g
#pragma unroll
        for (int g = 0; g < TPW; ++g)
#pragma unroll
            for (int b = 0; b < RB; ++b) {
                const int j = 32 * b + n;
                if (j < R) {
#pragma unroll
                    for (int i = 0; i < 16; ++i) {
                        const int64_t t = first + 32 * g + acc_row(i, half);
                        if (t < T) out[(slot * T + t) * R + j] = dz[g][b][i];
                    }
                }
            }
    }
}

// out[j] = sum over p < P of in[p N + j] in a fixed order (0 when P == 0): G threads per output
// (blocks of 256 / G consecutive outputs, so that loads coalesce); thread q sums p = q, q + G, ...
// in increasing order with eight loads in flight, and the G partials are added in order of q.
__global__ __launch_bounds__(256) void bwd_colsum_kernel(const float* __restrict__ in, int32_t P,
                                                         int64_t N, int32_t G,
                                                         float* __restrict__ out) {
    __shared__ float red[256];
    const int per = 256 / G;
    const int q = threadIdx.x / per, jj = threadIdx.x % per;
    const int64_t j = (int64_t)blockIdx.x * per + jj;
    float s = 0.0f;
    if (j < N) {
        int32_t p = q;
        for (; p + 7 * G < P; p += 8 * G) {
            float v[8];
#pragma unroll
            for (int u = 0; u < 8; ++u) v[u] = in[(int64_t)(p + u * G) * N + j];
#pragma unroll
            for (int u = 0; u < 8; ++u) s += v[u];
        }
        for (; p < P; p += G) s += in[(int64_t)p * N + j];
    }
    red[threadIdx.x] = s;
    __syncthreads();
    if (q == 0 && j < N) {
        float t = red[jj];
        for (int qq = 1; qq < G; ++qq) t += red[qq * per + jj];
        out[j] = t;
    }
}

// ------------------------------------------------------------------------------ dz
// One workgroup per 32 tokens, eight threads per token, each owning VPT = r / 8 consecutive rank
// columns: dz[t][j] = the dense part (dzsum, or the dz sweep's partials summed here in order when
// there are few), then dtop[t][q] R2t[e][j] for the
// token's selections q = 0 .. k-1 with e = idx[t][q] in [0, M) (one VPT-wide gather each).
// Writes dz as bf16 hi/lo rows dzhl [T][2r] and, through LDS, as transposed rows dzT [2][r][Tp]
// (Tp = T rounded up to 64; the columns past T are zero).
template <int RC>
__global__ __launch_bounds__(256) void bwd_dz_kernel(const float* __restrict__ dzsum,
                                                     const float* __restrict__ dzpart,
                                                     int32_t dzparts,
                                                     const int32_t* __restrict__ idx,
                                                     const float* __restrict__ dtop, int32_t k,
                                                     const uint16_t* __restrict__ R2t, int32_t T,
                                                     int32_t M, int64_t Tp,
                                                     uint16_t* __restrict__ dzhl,
                                                     uint16_t* __restrict__ dzT) {
    constexpr int R = 16 * RC, VPT = R / 8;
    __shared__ uint16_t sh[2][R * 33];  // [hi/lo][j][token] with 33 columns per row
    const int tl = threadIdx.x >> 3, jg = threadIdx.x & 7;
    const int64_t t0 = (int64_t)blockIdx.x * 32;
    const int64_t t = t0 + tl;
    const int j0 = jg * VPT;
    float s[VPT];
#pragma unroll
    for (int v = 0; v < VPT; ++v) s[v] = 0.0f;
    if (t < T) {
        if (dzparts > 0) {  // the dz sweep's partials in order (few), else their sum
            for (int32_t p = 0; p < dzparts; ++p) {
#pragma unroll
                for (int v = 0; v < VPT; ++v) s[v] += dzpart[((int64_t)p * T + t) * R + j0 + v];
            }
        } else if (dzsum) {
#pragma unroll
            for (int v = 0; v < VPT; ++v) s[v] = dzsum[t * R + j0 + v];
        }
        for (int32_t u0 = 0; u0 < k; u0 += 8) {  // eight selections' rows in flight, added in order
            int32_t ee[8];
            float dd[8];
            uint16_t w[8][VPT];
#pragma unroll
            for (int q = 0; q < 8; ++q) {
                const int32_t u = u0 + q;
                const int32_t e = u < k ? idx[t * k + u] : -1;
                const bool ok = e >= 0 && e < M;
                ee[q] = ok ? e : -1;
                dd[q] = ok ? dtop[t * k + u] : 0.0f;
                const uint16_t* row = R2t + (int64_t)(ok ? e : 0) * R + j0;
                if constexpr (VPT == 8) {
                    const u32x4 v = *reinterpret_cast<const u32x4*>(row);
                    __builtin_memcpy(w[q], &v, sizeof w[q]);
                } else if constexpr (VPT == 4) {
                    const uint2 v = *reinterpret_cast<const uint2*>(row);
                    __builtin_memcpy(w[q], &v, sizeof w[q]);
                } else {
                    const uint32_t v = *reinterpret_cast<const uint32_t*>(row);
                    __builtin_memcpy(w[q], &v, sizeof w[q]);
                }
            }
#pragma unroll
            for (int q = 0; q < 8; ++q) {
                if (ee[q] >= 0) {
#pragma unroll
                    for (int v = 0; v < VPT; ++v) s[v] += dd[q] * bf16_bits_to_f32(w[q][v]);
                }
            }
        }
    }
#pragma unroll
    for (int v = 0; v < VPT; ++v) {
        const __bf16 hb = (__bf16)s[v];
        const __bf16 lb = (__bf16)(s[v] - (float)hb);
        const uint16_t hv = __builtin_bit_cast(uint16_t, hb), lv = __builtin_bit_cast(uint16_t, lb);
        if (t < T) {
            dzhl[t * 2 * R + j0 + v] = hv;
            dzhl[t * 2 * R + R + j0 + v] = lv;
        }
        sh[0][(j0 + v) * 33 + tl] = hv;
        sh[1][(j0 + v) * 33 + tl] = lv;
    }
    __syncthreads();
    for (int q = threadIdx.x; q < 32 * R; q += 256) {
        const int j = q / 32, c = q % 32;
        dzT[(int64_t)j * Tp + t0 + c] = sh[0][j * 33 + c];
        dzT[((int64_t)R + j) * Tp + t0 + c] = sh[1][j * 33 + c];
    }
}

// ------------------------------------------------------------------------------ expert-major
// Workgroup (expert block, token split): wave w owns NE expert tiles of the block, held as B
// operands (expert columns) in registers, and the workgroup streams the 32-token tiles of its
// split through LDS (z'_hi/z'_lo rows, bias and g of each token, and bf16(z) transposed), stages
// of 128 tokens, double buffered.  A lane owns one expert column and sixteen token rows of each
// logit tile; ybar = P (pbar_e - g_t) is then an A operand (expert rows, token K order as the
// accumulator holds them) against bf16(z) pieces read from the transposed copy in the same K
// order, accumulating dR2^T rows: part[split][e][r].  Rows past M are computed and not stored;
// rows past T have bias kBwNoToken (P = 0) and zero z.
template <int RC>
struct ExpCfg {
    static constexpr int R = 16 * RC;
    static constexpr int RB = (R + 31) / 32;
    static constexpr int ROW = 2 * R + 8;                  // LDS pitch of a z'_hi|z'_lo row
    static constexpr int ZP = kBwStageT + 8;               // LDS pitch of a transposed z row
    static constexpr int ZH_PIECES = kBwStageT * 2 * R / 8;
    static constexpr int ZB_PIECES = kBwStageT * R / 8;
    static constexpr int ZH_PPT = ZH_PIECES / kBwThreads;
    static constexpr int ZB_PPT = (ZB_PIECES + kBwThreads - 1) / kBwThreads;
    static constexpr int EXPERTS = 32 * kBwNE * kBwWaves;  // experts per workgroup
    static_assert(ZH_PIECES % kBwThreads == 0, "whole pieces per thread");
};

template <int RC>
__global__ __launch_bounds__(kBwThreads, 1) void bwd_exp_kernel(
    const uint16_t* __restrict__ zhl, const uint16_t* __restrict__ zb,
    const float* __restrict__ bias, const float* __restrict__ gtok,
    const float* __restrict__ pbar, const uint16_t* __restrict__ R2t, int32_t T, int32_t M,
    int32_t eblocks, int32_t splits, float* __restrict__ part) {
    using C = ExpCfg<RC>;
    constexpr int R = C::R, RB = C::RB, ROW = C::ROW, ZP = C::ZP, NE = kBwNE;
    constexpr int TILES = kBwStageT / 32;
    __shared__ __attribute__((aligned(16))) uint16_t zs[2][kBwStageT * ROW];
    __shared__ __attribute__((aligned(16))) uint16_t zt[2][R * ZP];
    __shared__ __attribute__((aligned(16))) float bs[2][kBwStageT];
    __shared__ __attribute__((aligned(16))) float gss[2][kBwStageT];
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int n = lane & 31, half = lane >> 5;
    const int32_t eb = (int32_t)(blockIdx.x % (unsigned)eblocks);
    const int32_t split = (int32_t)(blockIdx.x / (unsigned)eblocks);
    const int64_t Tt = ((int64_t)T + 31) / 32;
    const int64_t tt0 = Tt * split / splits, tt1 = Tt * (split + 1) / splits;
    const int ntiles = (int)(tt1 - tt0);
    const int nstages = (ntiles + TILES - 1) / TILES;
    const int32_t Mt = (M + 31) / 32;
    const int32_t etile0 = (eb * kBwWaves + w) * NE;
    const bool active = etile0 < Mt;  // wave-uniform; idle waves still stage tokens
    bf16x8 b[NE][RC];
    float pb[NE];
#pragma unroll
    for (int j = 0; j < NE; ++j) {
        int64_t e = (int64_t)32 * (etile0 + j) + n;
        const bool ok = e < M;
        e = ok ? e : M - 1;  // columns past M: never stored
#pragma unroll
        for (int c = 0; c < RC; ++c) b[j][c] = load_bf16x8(R2t + e * R + 16 * c + 8 * half);
        pb[j] = ok ? pbar[e] : 0.0f;
    }
    u32x4 rh[C::ZH_PPT], rz[C::ZB_PPT];
    float rb = 0.0f, rgv = 0.0f;
    auto gload = [&](int st) __attribute__((always_inline)) {
        const int64_t tok0 = (tt0 + (int64_t)st * TILES) * 32;
#pragma unroll
        for (int i = 0; i < C::ZH_PPT; ++i) {
            const int p = tid + i * kBwThreads;
            int64_t t = tok0 + p / (2 * R / 8);
            t = t < T ? t : T - 1;  // rows past T: bias kBwNoToken below
            rh[i] = *reinterpret_cast<const u32x4*>(zhl + t * (2 * R) + 8 * (p % (2 * R / 8)));
        }
#pragma unroll
        for (int i = 0; i < C::ZB_PPT; ++i) {
            const int p = tid + i * kBwThreads;
            const int64_t t = tok0 + p / (R / 8);
            const int64_t tc = t < T ? t : T - 1;
            u32x4 v = u32x4{0u, 0u, 0u, 0u};
            if (p < C::ZB_PIECES) v = *reinterpret_cast<const u32x4*>(zb + tc * R + 8 * (p % (R / 8)));
            rz[i] = t < T ? v : u32x4{0u, 0u, 0u, 0u};
        }
        if (tid < kBwStageT) {
            const int64_t t = tok0 + tid;
            const int64_t tc = t < T ? t : T - 1;
            const float bv = bias[tc], gv = gtok[tc];
            rb = t < T ? bv : kBwNoToken;
            rgv = t < T ? gv : 0.0f;
        }
    };
    auto stash = [&](int buf) __attribute__((always_inline)) {
#pragma unroll
        for (int i = 0; i < C::ZH_PPT; ++i) {
            const int p = tid + i * kBwThreads;
            *reinterpret_cast<u32x4*>(&zs[buf][(p / (2 * R / 8)) * ROW + 8 * (p % (2 * R / 8))]) =
                rh[i];
        }
#pragma unroll
        for (int i = 0; i < C::ZB_PPT; ++i) {
            const int p = tid + i * kBwThreads;
            if (p < C::ZB_PIECES) {
                const int tl = p / (R / 8), q = p % (R / 8);
                const uint16_t* v = reinterpret_cast<const uint16_t*>(&rz[i]);
#pragma unroll
                for (int u = 0; u < 8; ++u) zt[buf][(8 * q + u) * ZP + tl] = v[u];
            }
        }
        if (tid < kBwStageT) {
            bs[buf][tid] = rb;
            gss[buf][tid] = rgv;
        }
    };
    f32x16 dr[NE][RB];
#pragma unroll
    for (int j = 0; j < NE; ++j)
#pragma unroll
        for (int q = 0; q < RB; ++q) dr[j][q] = zero_f32x16();
    if (nstages > 0) {  // workgroup-uniform
        gload(0);
        stash(0);
        if (nstages > 1) gload(1);
        __syncthreads();
        for (int st = 0; st < nstages; ++st) {
            const int buf = st & 1;
            const int cnt = min(TILES, ntiles - st * TILES);
            if (active) {
                for (int tl = 0; tl < cnt; ++tl) {
                    const uint16_t* zr = &zs[buf][(tl * 32 + n) * ROW + 8 * half];
                    bf16x8 a[2 * RC];
#pragma unroll
                    for (int c = 0; c < 2 * RC; ++c) a[c] = load_bf16x8(zr + 16 * c);
                    f32x16 cin;
                    float gv[16];
#pragma unroll
                    for (int q = 0; q < 4; ++q) {
                        const f32x4 v =
                            *reinterpret_cast<const f32x4*>(&bs[buf][tl * 32 + 8 * q + 4 * half]);
                        const f32x4 u =
                            *reinterpret_cast<const f32x4*>(&gss[buf][tl * 32 + 8 * q + 4 * half]);
#pragma unroll
                        for (int p = 0; p < 4; ++p) {
                            cin[4 * q + p] = v[p];
                            gv[4 * q + p] = u[p];
                        }
                    }
                    bf16x8 zf[2][RB];
#pragma unroll
                    for (int q2 = 0; q2 < 2; ++q2)
#pragma unroll
                        for (int q = 0; q < RB; ++q) {
                            int jr = 32 * q + n;
                            jr = jr < R ? jr : R - 1;  // columns past r: never stored
                            const uint16_t* pr = &zt[buf][jr * ZP + tl * 32 + 16 * q2 + 4 * half];
                            zf[q2][q] = lds_two_quads(pr, pr + 8);
                        }
#pragma unroll
                    for (int j = 0; j < NE; ++j) {
                        f32x16 acc = cin;
                        if constexpr (RC < 4) {
                            // two independent chains (z'_hi with the bias, z'_lo), added at the
                            // end (at r = 64 the NE tiles' chains suffice and registers are short)
                            f32x16 acl = zero_f32x16();
#pragma unroll
                            for (int c = 0; c < RC; ++c) {
                                acc = mfma_32x32x16(a[c], b[j][c], acc);
                                acl = mfma_32x32x16(a[RC + c], b[j][c], acl);
                            }
                            acc += acl;
                        } else {
#pragma unroll
                            for (int c = 0; c < 2 * RC; ++c) acc = mfma_32x32x16(a[c], b[j][c % RC], acc);
                        }
                        float y[16];
#pragma unroll
                        for (int i = 0; i < 16; ++i) y[i] = bw_exp2(acc[i]) * (pb[j] - gv[i]);
                        const bf16x8 y0 = pack_bf16x8(y), y1 = pack_bf16x8(y + 8);
#pragma unroll
                        for (int q = 0; q < RB; ++q) {
                            dr[j][q] = mfma_32x32x16(y0, zf[0][q], dr[j][q]);
                            dr[j][q] = mfma_32x32x16(y1, zf[1][q], dr[j][q]);
                        }
                    }
                }
            }
            if (st + 1 < nstages) stash(buf ^ 1);
            if (st + 2 < nstages) gload(st + 2);
            __syncthreads();
        }
    }
    // lane: rank column 32 q + n, expert rows acc_row(i, half) of tile j
#pragma unroll
    for (int j = 0; j < NE; ++j) {
        if (etile0 + j >= Mt) break;
#pragma unroll
        for (int q = 0; q < RB; ++q) {
            const int jr = 32 * q + n;
            if (jr < R) {
#pragma unroll
                for (int i = 0; i < 16; ++i) {
                    const int64_t e = (int64_t)32 * (etile0 + j) + acc_row(i, half);
                    if (e < M) part[((int64_t)split * M + e) * R + jr] = dr[j][q][i];
                }
            }
        }
    }
}

// The dtop terms of dR2, sum over the selections p of expert e of dtop[p] z[p / k][:], as a
// segmented sum over the sorted selections: one wave per chunk of kBwChunk consecutive sorted
// entries (lane j < r holds rank column j) walks its entries in order and sums each run of one
// expert.  An expert whose entries lie in one chunk gets its sum written to dR2t[e][:] (read
// back, after the dense part, by bwd_dr2); for an expert spanning chunks c0 < c1 each chunk
// stores its run in bpart[c][s][:], with s = 1 in c0 (the chunk's last run) and s = 0 in the
// others (the chunk's first run), and bwd_dr2 adds them in chunk order.
constexpr int kBwChunk = 64;

__global__ __launch_bounds__(256) void bwd_sparse_kernel(const int32_t* __restrict__ sorted,
                                                         const int32_t* __restrict__ offsets,
                                                         const int32_t* __restrict__ idx,
                                                         const float* __restrict__ dtop,
                                                         const float* __restrict__ z, int32_t k,
                                                         int32_t r, int32_t M, int64_t nchunks,
                                                         int32_t accumulate,
                                                         float* __restrict__ dR2t,
                                                         float* __restrict__ bpart) {
    const int lane = threadIdx.x & 63;
    const int64_t c = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    if (c >= nchunks) return;  // wave-uniform
    const int64_t nv = offsets[M];  // entries with a valid id
    const int64_t q0 = c * kBwChunk;
    const int cnt = (int)min((int64_t)kBwChunk, nv - q0);
    if (cnt <= 0) return;  // wave-uniform
    int32_t pl = 0, el = 0, o0l = 0, o1l = 1;
    float vl = 0.0f;
    if (lane < cnt) {
        pl = sorted[q0 + lane];
        el = idx[pl];
        vl = dtop[pl];
        o0l = offsets[el];  // the entry's expert range, loaded for all entries at once
        o1l = offsets[el + 1];
    }
    // run ending at entry u (its expert's range read from lane u; dense: its dR2 row's value when
    // accumulating)
    auto flush = [&](int32_t e, int u, float acc, float dense) __attribute__((always_inline)) {
        const int64_t o0 = __builtin_amdgcn_readlane(o0l, u);
        const int64_t o1 = __builtin_amdgcn_readlane(o1l, u);
        const int64_t c0 = o0 / kBwChunk, c1 = (o1 - 1) / kBwChunk;
        if (lane < r) {
            if (c0 == c1)
                dR2t[(int64_t)e * r + lane] = accumulate ? dense + acc : acc;
            else
                bpart[(c * 2 + (c == c0 ? 1 : 0)) * r + lane] = acc;
        }
    };
    int32_t cur = __builtin_amdgcn_readfirstlane(el);
    float acc = 0.0f;
    const int32_t vbits = __builtin_bit_cast(int32_t, vl);
    // the z rows of all the chunk's entries in flight at once (lane j < r: column j), then the
    // entries in order
    float zv[kBwChunk];
#pragma unroll
    for (int u = 0; u < kBwChunk; ++u) {
        const int32_t p = __builtin_amdgcn_readlane(pl, u);  // 0 past cnt: a valid row
        zv[u] = lane < r ? z[(int64_t)(p / k) * r + lane] : 0.0f;
    }
    // accumulating: the dense dR2 rows of the entries' experts, also all in flight at once
    float dv[kBwChunk];
#pragma unroll
    for (int u = 0; u < kBwChunk; ++u) {
        const int32_t e = __builtin_amdgcn_readlane(el, u);  // 0 past cnt: a valid row
        dv[u] = (accumulate && lane < r) ? dR2t[(int64_t)e * r + lane] : 0.0f;
    }
#pragma unroll
    for (int u = 0; u < kBwChunk; ++u) {
        if (u < cnt) {
            const int32_t e = __builtin_amdgcn_readlane(el, u);
            const float v = __builtin_bit_cast(float, __builtin_amdgcn_readlane(vbits, u));
            if (e != cur) {
                flush(cur, u - 1, acc, dv[u > 0 ? u - 1 : 0]);
                cur = e;
                acc = 0.0f;
            }
            acc += v * zv[u];
            if (u == cnt - 1) flush(cur, u, acc, dv[u]);
        }
    }
}

// dR2t[e][j] = the P partials in order, then the dtop terms of bwd_sparse (in chunk order for an
// expert spanning chunks).  One thread per element.  With one token split the expert-major sweep
// writes dR2t itself and bwd_sparse adds the sums of the experts inside one chunk to it
// (accumulate = 1); bwd_dr2_fix then adds the chunk sums of the experts spanning chunks, in the
// same order of operations.
__global__ __launch_bounds__(256) void bwd_dr2_kernel(const float* __restrict__ part, int32_t P,
                                                      const int32_t* __restrict__ offsets,
                                                      const float* __restrict__ bpart, int32_t M,
                                                      int32_t r, float* __restrict__ dR2t) {
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i >= (int64_t)M * r) return;
    const int64_t e = i / r;
    const int32_t j = (int32_t)(i - e * r);
    const int64_t N = (int64_t)M * r;
    float s = 0.0f;
    int32_t p = 0;
    for (; p + 8 <= P; p += 8) {
        float v[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) v[u] = part[(int64_t)(p + u) * N + i];
#pragma unroll
        for (int u = 0; u < 8; ++u) s += v[u];
    }
    for (; p < P; ++p) s += part[(int64_t)p * N + i];
    const int64_t o0 = offsets[e], o1 = offsets[e + 1];
    if (o1 > o0) {
        const int64_t c0 = o0 / kBwChunk, c1 = (o1 - 1) / kBwChunk;
        if (c0 == c1) {
            s += dR2t[i];
        } else {
            s += bpart[(c0 * 2 + 1) * r + j];
            for (int64_t c = c0 + 1; c <= c1; ++c) s += bpart[(c * 2) * r + j];
        }
    }
    dR2t[i] = s;
}

__global__ __launch_bounds__(256) void bwd_dr2_fix_kernel(const int32_t* __restrict__ offsets,
                                                          const float* __restrict__ bpart,
                                                          int32_t M, int32_t r,
                                                          float* __restrict__ dR2t) {
    // lane l of a wave checks expert 64 w + l; the wave then fixes each spanning one, lane = column
    const int lane = threadIdx.x & 63;
    const int64_t e0 = ((int64_t)blockIdx.x * 4 + (threadIdx.x >> 6)) * 64;
    const int64_t e = e0 + lane;
    int64_t o0 = 0, o1 = 0;
    if (e < M) {
        o0 = offsets[e];
        o1 = offsets[e + 1];
    }
    const bool span = o1 > o0 && o0 / kBwChunk != (o1 - 1) / kBwChunk;
    uint64_t m = __ballot(span);
    while (m) {  // wave-uniform
        const int src = __builtin_ctzll(m);
        m &= m - 1;
        const int64_t ee = e0 + src;
        const int64_t c0 = (int64_t)__builtin_amdgcn_readlane((int32_t)o0, src) / kBwChunk;
        const int64_t c1 = ((int64_t)__builtin_amdgcn_readlane((int32_t)o1, src) - 1) / kBwChunk;
        if (lane < r) {
            float s = dR2t[ee * r + lane];
            s += bpart[(c0 * 2 + 1) * r + lane];
            for (int64_t c = c0 + 1; c <= c1; ++c) s += bpart[(c * 2) * r + lane];
            dR2t[ee * r + lane] = s;
        }
    }
}

// ------------------------------------------------------------------------------ dx
// dx [T][h] = dz R1^T with dz = hi + lo: a wave takes 32 tokens (A operands: dz rows) and
// kBwDxTiles 32-column tiles (B operands: rows of R1 [h][r]); a lane stores one column.
constexpr int kBwDxTiles = 4;

template <int RC>
__global__ __launch_bounds__(256) void bwd_dx_kernel(const uint16_t* __restrict__ dzhl,
                                                     const uint16_t* __restrict__ R1, int32_t T,
                                                     int32_t h, int32_t ctiles_per_wg,
                                                     float* __restrict__ dx) {
    constexpr int R = 16 * RC;
    const int lane = threadIdx.x & 63;
    const int w = threadIdx.x >> 6;
    const int n = lane & 31, half = lane >> 5;
    const int32_t Ct = (h + 31) / 32;
    const int32_t cgroups = (Ct + ctiles_per_wg - 1) / ctiles_per_wg;
    const int64_t tt = blockIdx.x / (unsigned)cgroups;
    const int32_t cg = (int32_t)(blockIdx.x % (unsigned)cgroups);
    const int64_t t = tt * 32 + n;
    const bool tok_ok = t < T;
    bf16x8 ah[RC], al[RC];
    const uint16_t* dr = dzhl + (tok_ok ? t : 0) * (2 * R) + 8 * half;
#pragma unroll
    for (int c = 0; c < RC; ++c) {
        const bf16x8 hv = load_bf16x8(dr + 16 * c), lv = load_bf16x8(dr + R + 16 * c);
        ah[c] = tok_ok ? hv : zero_bf16x8();
        al[c] = tok_ok ? lv : zero_bf16x8();
    }
    const int32_t ct_end = min(Ct, (cg + 1) * ctiles_per_wg);
    for (int32_t ct = cg * ctiles_per_wg + w; ct < ct_end; ct += 4) {
        int64_t col = (int64_t)ct * 32 + n;
        const bool col_ok = col < h;
        const uint16_t* br = R1 + (col_ok ? col : h - 1) * R + 8 * half;
        f32x16 acc = zero_f32x16();
#pragma unroll
        for (int c = 0; c < RC; ++c) {
            const bf16x8 bv = load_bf16x8(br + 16 * c);
            acc = mfma_32x32x16(ah[c], bv, acc);
            acc = mfma_32x32x16(al[c], bv, acc);
        }
        if (col_ok) {
#pragma unroll
            for (int i = 0; i < 16; ++i) {
                const int64_t tr = tt * 32 + acc_row(i, half);
                if (tr < T) dx[tr * h + col] = acc[i];
            }
        }
    }
}

// ------------------------------------------------------------------------------ dR1
// part[s][j][c] = sum over the tokens of split s of dz[t][j] x[t][c]: a workgroup of 4 waves
// takes 128 columns (wave w: columns 32 w ..) and stages 64-token slices of x and of dzT's rows
// (hi and lo) through LDS, one slice ahead in registers; the A operands are dz^T rows read from
// the staged slice, the B operands eight x values of one column read down the LDS slice.
constexpr int kBwR1Tok = 64;
constexpr int kBwR1Cols = 128;
constexpr int kBwR1Pitch = kBwR1Cols + 8;

template <int RC>
__global__ __launch_bounds__(256) void bwd_dr1_kernel(const uint16_t* __restrict__ x,
                                                      const uint16_t* __restrict__ dzT,
                                                      int64_t Tp, int32_t T, int32_t h,
                                                      int32_t splits, float* __restrict__ part) {
    constexpr int R = 16 * RC, RB = (R + 31) / 32;
    constexpr int PIECES = kBwR1Tok * kBwR1Cols / 8;  // 1024
    constexpr int PPT = PIECES / 256;
    // the stage's dz columns: rows 0 .. 2R - 1 of dzT (hi, then lo), kBwR1Tok tokens each,
    // staged beside x so that the A operands come from LDS
    constexpr int DZP = kBwR1Tok + 8;
    constexpr int DPT = 2 * R * (kBwR1Tok / 8) / 256;  // 16-byte pieces per thread (= RC)
    __shared__ __attribute__((aligned(16))) uint16_t xs[2][kBwR1Tok * kBwR1Pitch];
    __shared__ __attribute__((aligned(16))) uint16_t dzs[2][2 * R * DZP];
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int w = tid >> 6;
    const int n = lane & 31, half = lane >> 5;
    const int32_t cblocks = (h + kBwR1Cols - 1) / kBwR1Cols;
    const int32_t cb = (int32_t)(blockIdx.x % (unsigned)cblocks);
    const int32_t split = (int32_t)(blockIdx.x / (unsigned)cblocks);
    const int64_t Ts = Tp / kBwR1Tok;  // 64-token slices
    const int64_t s0 = Ts * split / splits, s1 = Ts * (split + 1) / splits;
    const int nst = (int)(s1 - s0);
    const int64_t c0 = (int64_t)cb * kBwR1Cols;
    u32x4 rg[PPT], dg[DPT];
    auto gload = [&](int st) __attribute__((always_inline)) {
        const int64_t tok0 = (s0 + st) * kBwR1Tok;
#pragma unroll
        for (int i = 0; i < DPT; ++i) {  // piece p: dzT row p / 8, tokens tok0 + 8 (p % 8) + 0..7
            const int p = tid + i * 256;
            dg[i] = *reinterpret_cast<const u32x4*>(dzT + (int64_t)(p >> 3) * Tp + tok0 +
                                                    8 * (p & 7));
        }
#pragma unroll
        for (int i = 0; i < PPT; ++i) {
            const int p = tid + i * 256;
            const int64_t t = tok0 + p / (kBwR1Cols / 8);
            const int64_t c = c0 + 8 * (p % (kBwR1Cols / 8));
            const bool ok = t < T && c < h;
            const u32x4 v = *reinterpret_cast<const u32x4*>(x + (ok ? t * h + c : 0));
            rg[i] = ok ? v : u32x4{0u, 0u, 0u, 0u};
        }
    };
    auto stash = [&](int buf) __attribute__((always_inline)) {
#pragma unroll
        for (int i = 0; i < DPT; ++i) {
            const int p = tid + i * 256;
            *reinterpret_cast<u32x4*>(&dzs[buf][(p >> 3) * DZP + 8 * (p & 7)]) = dg[i];
        }
#pragma unroll
        for (int i = 0; i < PPT; ++i) {
            const int p = tid + i * 256;
            *reinterpret_cast<u32x4*>(
                &xs[buf][(p / (kBwR1Cols / 8)) * kBwR1Pitch + 8 * (p % (kBwR1Cols / 8))]) = rg[i];
        }
    };
    f32x16 acc[RB];
#pragma unroll
    for (int q = 0; q < RB; ++q) acc[q] = zero_f32x16();
    if (nst > 0) {
        gload(0);
        stash(0);
        if (nst > 1) gload(1);
        __syncthreads();
        for (int st = 0; st < nst; ++st) {
            const int buf = st & 1;
#pragma unroll
            for (int ks = 0; ks < kBwR1Tok / 16; ++ks) {
                bf16x8 bx;
                const uint16_t* xp = &xs[buf][(16 * ks + 8 * half) * kBwR1Pitch + 32 * w + n];
#pragma unroll
                for (int u = 0; u < 8; ++u)
                    bx[u] = __builtin_bit_cast(__bf16, xp[u * kBwR1Pitch]);
#pragma unroll
                for (int q = 0; q < RB; ++q) {
                    int jr = 32 * q + n;
                    jr = jr < R ? jr : R - 1;  // rows past r: never stored
                    const int off = 16 * ks + 8 * half;
                    const bf16x8 ahv =
                        *reinterpret_cast<const bf16x8*>(&dzs[buf][jr * DZP + off]);
                    const bf16x8 alv =
                        *reinterpret_cast<const bf16x8*>(&dzs[buf][(R + jr) * DZP + off]);
                    acc[q] = mfma_32x32x16(ahv, bx, acc[q]);
                    acc[q] = mfma_32x32x16(alv, bx, acc[q]);
                }
            }
            if (st + 1 < nst) stash(buf ^ 1);
            if (st + 2 < nst) gload(st + 2);
            __syncthreads();
        }
    }
    const int64_t c = c0 + 32 * w + n;
    if (c < h) {
#pragma unroll
        for (int q = 0; q < RB; ++q)
#pragma unroll
            for (int i = 0; i < 16; ++i) {
                const int jr = 32 * q + acc_row(i, half);
                if (jr < R) part[((int64_t)split * R + jr) * h + c] = acc[q][i];
            }
    }
}

// ------------------------------------------------------------------------------ host side
namespace {

size_t al256(size_t b) { return (b + 255) & ~(size_t)255; }

// Threads per output of bwd_colsum for P partials: about eight partials per thread, at most 16.
int32_t colsum_group(int64_t P) {
    int32_t G = 1;
    while (G < 16 && (int64_t)G * 8 < P) G *= 2;
    return G;
}

void launch_colsum(const float* in, int32_t P, int64_t N, float* out, hipStream_t st) {
    const int32_t G = colsum_group(P);
    const int64_t per = 256 / G;
    hipLaunchKernelGGL(bwd_colsum_kernel, dim3((unsigned)((N + per - 1) / per)), dim3(256), 0, st,
                       in, P, N, G, out);
}

}  // namespace

bool backward_make_plan(int64_t T, int32_t h, int32_t r, int32_t M, int32_t k, bool balance,
                        BackwardPlan* out) {
    if (T < 0 || M <= 0 || k < 1 || (r != 16 && r != 32 && r != 64) || h <= 0 || h % 16 != 0)
        return false;
    BackwardPlan q{};
    q.RC = r / 16;
    q.balance = balance ? 1 : 0;
    const int64_t Mt = ((int64_t)M + 31) / 32;
    const int64_t Tt = (T + 31) / 32;
    // token-major sweeps: WT token slots per workgroup, about 256 workgroups
    auto tok_grid = [&](int nw, int tpw, TokGrid* g) {
        const int64_t slot = 32 * tpw;
        const int64_t slots_needed = (T + slot - 1) / slot;
        int32_t WT = nw;  // token slots per workgroup; the WE = nw / WT waves of a slot (<= 4)
        while (WT > nw / 4 && (int64_t)WT / 2 >= slots_needed) WT /= 2;
        g->WT = WT;
        g->ntb = (T + WT * slot - 1) / (WT * slot);
        int64_t S = (256 + g->ntb - 1) / (g->ntb > 0 ? g->ntb : 1);
        const int64_t stages = (Mt + kBwStageE / 32 - 1) / (kBwStageE / 32);
        if (S > stages) S = stages;
        if (S < 1) S = 1;
        g->splits = (int32_t)S;
        g->parts = (int32_t)(S * (nw / WT));
    };
    switch (q.RC) {
        case 1:
            tok_grid(bw_waves<1, false>(), bw_tpw<1, false>(), &q.gsweep);
            tok_grid(bw_waves<1, true>(), bw_tpw<1, true>(), &q.dzsweep);
            break;
        case 2:
            tok_grid(bw_waves<2, false>(), bw_tpw<2, false>(), &q.gsweep);
            tok_grid(bw_waves<2, true>(), bw_tpw<2, true>(), &q.dzsweep);
            break;
        default:
            tok_grid(bw_waves<4, false>(), bw_tpw<4, false>(), &q.gsweep);
            tok_grid(bw_waves<4, true>(), bw_tpw<4, true>(), &q.dzsweep);
            break;
    }
    // expert-major sweep: expert blocks of 32 NE waves tiles, about 512 workgroups
    const int64_t per_block = 32 * kBwNE * kBwWaves;
    q.eblocks = (int32_t)((M + per_block - 1) / per_block);
    int64_t P = (512 + q.eblocks - 1) / q.eblocks;
    if (P > Tt) P = Tt;
    if (P < 1) P = 1;
    q.esplits = (int32_t)P;
    // dR1: 128-column blocks x token splits, about 512 workgroups
    q.Tp = ((T + 63) / 64) * 64;
    const int64_t cblocks = (h + kBwR1Cols - 1) / kBwR1Cols;
    int64_t S3 = (512 + cblocks - 1) / cblocks;
    if (S3 > q.Tp / 64) S3 = q.Tp / 64;
    if (S3 < 1) S3 = 1;
    q.r1splits = (int32_t)S3;
    size_t o = 0;
    auto take = [&](size_t bytes) {
        const size_t at = o;
        o += al256(bytes);
        return at;
    };
    q.off_z = take((size_t)T * r * 4);
    q.off_zscratch = take(zonly_workspace_bytes(T > 0 ? T : 1, h, r));
    q.off_zhl = take((size_t)T * 2 * r * 2);
    q.off_zb = take((size_t)T * r * 2);
    q.off_bias = take((size_t)T * 4);
    q.off_g = take((size_t)T * 4);
    q.off_gpart = balance ? take((size_t)q.gsweep.parts * T * 4) : take(0);
    q.off_dzpart = balance ? take((size_t)q.dzsweep.parts * T * r * 4) : take(0);
    q.off_dzsum = balance ? take((size_t)T * r * 4) : take(0);
    q.off_dzhl = take((size_t)T * 2 * r * 2);
    q.off_dzT = take((size_t)2 * r * q.Tp * 2);
    q.off_r1 = take((size_t)h * r * 2);
    q.off_r2part = (balance && q.esplits > 1) ? take((size_t)q.esplits * M * r * 4) : take(0);
    q.off_r1part = take((size_t)q.r1splits * r * h * 4);
    q.off_offsets = take(((size_t)M + 1) * 4);
    q.off_sorted = take((size_t)T * k * 4);
    q.off_dispatch = take(dispatch_workspace_bytes(T * k));
    q.nchunks = (T * k + kBwChunk - 1) / kBwChunk;
    q.off_bpart = take((size_t)q.nchunks * 2 * r * 4);
    q.workspace_bytes = o;
    *out = q;
    return true;
}

template <int RC>
static void launch_balance(const BackwardPlan& p, const BackwardArgs& a, char* ws,
                           hipStream_t st) {
    const uint16_t* zhl = reinterpret_cast<const uint16_t*>(ws + p.off_zhl);
    const uint16_t* zb = reinterpret_cast<const uint16_t*>(ws + p.off_zb);
    const float* bias = reinterpret_cast<const float*>(ws + p.off_bias);
    float* g = reinterpret_cast<float*>(ws + p.off_g);
    float* gpart = reinterpret_cast<float*>(ws + p.off_gpart);
    float* dzpart = reinterpret_cast<float*>(ws + p.off_dzpart);
    float* r2part = reinterpret_cast<float*>(ws + p.off_r2part);
    float* dzsum = reinterpret_cast<float*>(ws + p.off_dzsum);
    const TokGrid& G = p.gsweep;
    const TokGrid& D = p.dzsweep;
    hipLaunchKernelGGL((bwd_tok_kernel<RC, false>), dim3((unsigned)(G.ntb * G.splits)),
                       dim3(64 * bw_waves<RC, false>()), 0, st, zhl, bias, nullptr, nullptr, 0,
                       nullptr, a.pbar, a.R2t, a.T, a.M, G.WT, G.splits, gpart);
    // few partials: the dz sweep sums them (and stores g); many: one summing launch
    const int32_t gp = G.parts <= kBwFoldParts ? G.parts : 0;
    if (gp == 0) launch_colsum(gpart, G.parts, a.T, g, st);
    hipLaunchKernelGGL((bwd_tok_kernel<RC, true>), dim3((unsigned)(D.ntb * D.splits)),
                       dim3(64 * bw_waves<RC, true>()), 0, st, zhl, bias, gp ? nullptr : g, gpart, gp,
                       gp ? g : nullptr, a.pbar, a.R2t, a.T, a.M, D.WT, D.splits, dzpart);
    if (D.parts > kBwFoldParts) launch_colsum(dzpart, D.parts, (int64_t)a.T * a.r, dzsum, st);
    // one token split: the sweep's partials are dR2's dense part, written in place
    hipLaunchKernelGGL((bwd_exp_kernel<RC>), dim3((unsigned)((int64_t)p.eblocks * p.esplits)),
                       dim3(kBwThreads), 0, st, zhl, zb, bias, g, a.pbar, a.R2t, a.T, a.M,
                       p.eblocks, p.esplits, p.esplits == 1 ? a.dR2t : r2part);
}

template <int RC>
static void launch_phase3(const BackwardPlan& p, const BackwardArgs& a, char* ws,
                          hipStream_t st) {
    const uint16_t* dzhl = reinterpret_cast<const uint16_t*>(ws + p.off_dzhl);
    const uint16_t* dzT = reinterpret_cast<const uint16_t*>(ws + p.off_dzT);
    const uint16_t* R1 = reinterpret_cast<const uint16_t*>(ws + p.off_r1);
    float* r1part = reinterpret_cast<float*>(ws + p.off_r1part);
    // dz = the dense sum (when pbar is given) plus the dtop rows of R2, as hi/lo rows and transposed
    const bool fold = p.balance && p.dzsweep.parts <= kBwFoldParts;
    hipLaunchKernelGGL((bwd_dz_kernel<RC>), dim3((unsigned)(p.Tp / 32)), dim3(256), 0, st,
                       (p.balance && !fold) ? reinterpret_cast<const float*>(ws + p.off_dzsum)
                                            : nullptr,
                       fold ? reinterpret_cast<const float*>(ws + p.off_dzpart) : nullptr,
                       fold ? p.dzsweep.parts : 0, a.idx, a.dtop, a.k, a.R2t, a.T, a.M, p.Tp,
                       reinterpret_cast<uint16_t*>(ws + p.off_dzhl),
                       reinterpret_cast<uint16_t*>(ws + p.off_dzT));
    const int32_t Ct = (a.h + 31) / 32;
    const int32_t per_wg = 4 * kBwDxTiles;
    const int64_t cgroups = (Ct + per_wg - 1) / per_wg;
    const int64_t Tt = ((int64_t)a.T + 31) / 32;
    if (Tt > 0)
        hipLaunchKernelGGL((bwd_dx_kernel<RC>), dim3((unsigned)(Tt * cgroups)), dim3(256), 0, st,
                           dzhl, R1, a.T, a.h, per_wg, a.dx);
    const int64_t cblocks = (a.h + kBwR1Cols - 1) / kBwR1Cols;
    hipLaunchKernelGGL((bwd_dr1_kernel<RC>), dim3((unsigned)(cblocks * p.r1splits)), dim3(256), 0,
                       st, a.x, dzT, p.Tp, a.T, a.h, p.r1splits, r1part);
    launch_colsum(r1part, p.r1splits, (int64_t)a.r * a.h, a.dR1t, st);
}

hipError_t backward_launch(const BackwardPlan& p, const BackwardArgs& a, void* workspace,
                           hipStream_t st) {
    char* ws = static_cast<char*>(workspace);
    const int32_t r = a.r;
    if (a.T == 0) {  // no tokens: zero weight gradients
        launch_colsum(nullptr, 0, (int64_t)r * a.h, a.dR1t, st);
        launch_colsum(nullptr, 0, (int64_t)a.M * r, a.dR2t, st);
        return hipGetLastError();
    }
    float* z = reinterpret_cast<float*>(ws + p.off_z);
    hipError_t e = zonly_launch(a.x, a.R1t, a.T, a.h, r, z, ws + p.off_zscratch, st);
    if (e != hipSuccess) return e;
    const int64_t nz = (int64_t)a.T * r;
    hipLaunchKernelGGL(bwd_prep_kernel, dim3((unsigned)((nz + 255) / 256)), dim3(256), 0, st, z,
                       p.balance ? a.m : nullptr, a.Z, a.T, r,
                       reinterpret_cast<uint16_t*>(ws + p.off_zhl),
                       reinterpret_cast<uint16_t*>(ws + p.off_zb),
                       reinterpret_cast<float*>(ws + p.off_bias));
    const int64_t nr1 = (int64_t)a.h * r;
    hipLaunchKernelGGL(bwd_r1_transpose_kernel, dim3((unsigned)((nr1 + 255) / 256)), dim3(256), 0,
                       st, a.R1t, a.h, r, reinterpret_cast<uint16_t*>(ws + p.off_r1));
    if (p.balance) {
        switch (p.RC) {
            case 1: launch_balance<1>(p, a, ws, st); break;
            case 2: launch_balance<2>(p, a, ws, st); break;
            case 4: launch_balance<4>(p, a, ws, st); break;
            default: return hipErrorInvalidValue;
        }
    }
    int32_t* offsets = reinterpret_cast<int32_t*>(ws + p.off_offsets);
    int32_t* sorted = reinterpret_cast<int32_t*>(ws + p.off_sorted);
    e = dispatch_launch(a.idx, (int64_t)a.T * a.k, a.M, offsets, sorted, ws + p.off_dispatch, st);
    if (e != hipSuccess) return e;
    float* bpart = reinterpret_cast<float*>(ws + p.off_bpart);
    const bool direct = p.balance && p.esplits == 1;  // dR2t holds the dense part already
    hipLaunchKernelGGL(bwd_sparse_kernel, dim3((unsigned)((p.nchunks + 3) / 4)), dim3(256), 0, st,
                       sorted, offsets, a.idx, a.dtop, z, a.k, r, a.M, p.nchunks,
                       direct ? 1 : 0, a.dR2t, bpart);
    const int64_t nr2 = (int64_t)a.M * r;
    if (direct)
        hipLaunchKernelGGL(bwd_dr2_fix_kernel, dim3((unsigned)(((int64_t)a.M + 255) / 256)),
                           dim3(256), 0, st, offsets, bpart, a.M, r, a.dR2t);  // 64 experts a wave
    else
        hipLaunchKernelGGL(bwd_dr2_kernel, dim3((unsigned)((nr2 + 255) / 256)), dim3(256), 0, st,
                           reinterpret_cast<const float*>(ws + p.off_r2part),
                           p.balance ? p.esplits : 0, offsets, bpart, a.M, r, a.dR2t);
    switch (p.RC) {
        case 1: launch_phase3<1>(p, a, ws, st); break;
        case 2: launch_phase3<2>(p, a, ws, st); break;
        case 4: launch_phase3<4>(p, a, ws, st); break;
        default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

}  // namespace more
