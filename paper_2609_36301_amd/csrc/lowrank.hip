// Low-rank router kernels for gfx950: softmax(TopK(x R1 R2)) without materialising the
// T x M logits (Appendix "Pseudocode", inference algorithm; MoRE layer in "Preliminaries").
//
// Routes of one call (chosen per shape by lowrank_make_plan):
//   expert-resident  zpass (z = x R1, fp32, and the group norms of R2t's rows unless the screen
//                    kernel takes them) [+ zreduce when the h axis is split over workgroups],
//                    then screen, threshold, collect and finalize kernels; screen and collect
//                    workgroups hold one chunk of the expert axis in LDS;
//   fused            zpass, then one fused_route_kernel: a workgroup of 64 tokens sweeps the
//                    whole expert axis (operands streamed from L2) through the same four steps;
//   local            one fused_local_kernel: the fused workgroup also computes z and one norm
//                    bound per wave, and keeps its expert rows in registers.
// The steps: screening bounds on z_hi = bf16(z) give a per-token threshold that k experts
// provably reach, the candidates above it are collected, and their logits are evaluated exactly
// in fp32 for the final top k (see the route section).
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

#include <utility>

#include "device_common.h"
#include "lowrank.h"
#include "route_device.h"

namespace more {

// ------------------------------------------------------------------------------ zpass
// One workgroup = 4 waves = 128 tokens, wave w owning tokens 32w..32w+31 of the block.  The h
// axis is walked in chunks of 64 (4 MFMA k-steps); the chunk of R1 (all rank rows) is staged
// in LDS and shared by the four waves; x and R1 are prefetched D chunks ahead in registers.  With
// hsplit > 1 the chunks are split over hsplit workgroups and each split writes a partial z.
constexpr int kZWaves = 4;
constexpr int kZTokens = 32 * kZWaves;
constexpr int kZChunk = 64;
constexpr int kGroupNormBlocks = 4;  // 256-segment blocks per group-norm workgroup

// Group norms: the largest Euclidean norm among expert rows 4g..4g+3 of R2t, rounded up, for
// every group of the rows < `rows` (all tiles).  A group holding a row past M gets the norm bound
// 2^100 instead: its screening bounds s -+ c 2^100 then never raise a threshold and always pass
// the collect test, so the sweeps need no masking of the rows past M (they re-read row M - 1)
// and the candidate expansion drops the ids >= M.  Within each tile of
// 32 rows the 8 groups are stored in the order [half][q] (group 2q + half at 4 half + q), so
// that MFMA lane half `half` reads the norms of its four accumulator groups q with one 16-byte
// load.  Lane (row, 16-byte segment) layout: the
// r/8 segments of a row sit in consecutive lanes and the 4 rows of a group next to each other.
template <int SPR>
__device__ __forceinline__ void group_norms(const uint16_t* __restrict__ R2t, int32_t M,
                                            int64_t rows, int64_t gid0, float* __restrict__ gnorm) {
    constexpr int R = 8 * SPR;
    constexpr int NB = kGroupNormBlocks;  // segments gid0 + 256 b, all loaded before any is used
    bf16x8 v[NB];
#pragma unroll
    for (int b = 0; b < NB; ++b) {
        const int64_t gid = gid0 + 256 * b;
        const int64_t row = gid / SPR;
        v[b] = row < M ? load_bf16x8(R2t + row * R + (gid % SPR) * 8) : zero_bf16x8();
    }
#pragma unroll
    for (int b = 0; b < NB; ++b) {
        const int64_t gid = gid0 + 256 * b;
        const int64_t row = gid / SPR;
        const int col = (int)(gid % SPR);
        float ss = 0.0f;
#pragma unroll
        for (int q = 0; q < 8; ++q) ss = fmaf((float)v[b][q], (float)v[b][q], ss);
#pragma unroll
        for (int m = 1; m < SPR; m <<= 1) ss += __shfl_xor(ss, m, kWave);
        ss = fmaxf(ss, __shfl_xor(ss, SPR, kWave));
        ss = fmaxf(ss, __shfl_xor(ss, 2 * SPR, kWave));
        if (col == 0 && (row & 3) == 0 && row < rows) {
            // slot of group g4 = (row mod 32) / 4 = 2q + half of tile row / 32: [tile][half][q]
            const int g4 = (int)(row & 31) >> 2;
            gnorm[(row >> 5) * 8 + (g4 & 1) * 4 + (g4 >> 1)] =
                row + 3 < M ? sqrtf(ss) * (1.0f + 0x1p-20f) : kPhantomNorm;
        }
    }
}

template <int RT, int D>
__global__ __launch_bounds__(256) void zpass_kernel(const uint16_t* __restrict__ x,
                                                    const uint16_t* __restrict__ R1t,
                                                    float* __restrict__ zout, int32_t T, int32_t h,
                                                    int32_t r, int32_t chunks_per_split,
                                                    const uint16_t* __restrict__ R2t, int32_t M,
                                                    int32_t zblocks, int32_t hsplit,
                                                    float* __restrict__ gnorm,
                                                    uint16_t* __restrict__ zhi_out,
                                                    float* __restrict__ c_out) {
    // Workgroups [0, zblocks * hsplit) compute z (token block bx % zblocks, h split
    // bx / zblocks); the rest compute group norms.
    if ((int)blockIdx.x >= zblocks * hsplit) {  // workgroup-uniform: a group-norm workgroup
        const int64_t gid = ((int64_t)blockIdx.x - (int64_t)zblocks * hsplit) * 256 *
                                kGroupNormBlocks + threadIdx.x;
        const int64_t rows = ((int64_t)M + 31) / 32 * 32;
        switch (r) {
            case 16: group_norms<2>(R2t, M, rows, gid, gnorm); break;
            case 32: group_norms<4>(R2t, M, rows, gid, gnorm); break;
            case 64: group_norms<8>(R2t, M, rows, gid, gnorm); break;
        }
        return;
    }
    constexpr int RR = 32 * RT;         // rank rows held by the MFMA tiles (r rounded up)
    constexpr int LROW = kZChunk + 8;   // padded LDS row of R1, bf16 elements
    constexpr int RLOADS = RR * (kZChunk / 8) / 256;  // 16-byte R1 segments per thread
    __shared__ __attribute__((aligned(16))) uint16_t r1s[2][RR * LROW];
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int w = tid >> 6;
    const int n = lane & 31;
    const int half = lane >> 5;
    const int zb = (int)(blockIdx.x % (unsigned)zblocks);
    const int split = (int)(blockIdx.x / (unsigned)zblocks);
    const int64_t tok = ((int64_t)zb * kZWaves + w) * 32 + n;
    const bool tok_ok = tok < T;
    const int S = h >> 4;               // 16-wide k-steps
    const int NC = (S + 3) / 4;         // 64-wide chunks
    const int cbeg = split * chunks_per_split;
    const int nc = max(0, min(NC, cbeg + chunks_per_split) - cbeg);

    const int jm = n >> 3, qm = (n >> 2) & 1, im = n & 3;
    const int prow = 16 * (jm >> 1) + 8 * qm + 4 * (jm & 1) + im;

    // All loads are issued unconditionally with clamped addresses (chunks past the range
    // re-read the last step, rows past r re-read row r - 1), so that every lane issues the
    // same loads and the compiler can keep D chunks in flight.  Clamped values never reach a
    // stored result: their MFMAs are skipped, or they land in rank rows that are not stored.
    const uint16_t* xrow = x + (tok_ok ? tok : 0) * (int64_t)h + 8 * half;
    u32x4 xb[D][4];
    auto xload = [&](auto slot, int c) __attribute__((always_inline)) {
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            int step = 4 * (cbeg + c) + j;
            step = step < S ? step : S - 1;
            xb[decltype(slot)::value][j] = *reinterpret_cast<const u32x4*>(xrow + 16 * step);
        }
    };
    // R1 chunks use the same D-deep register ring as x: chunk c sits in ring slot c mod D,
    // is stored to LDS buffer c mod 2 one chunk ahead of its use, and its slot is then
    // refilled with chunk c + D.
    u32x4 rb[D][RLOADS];
    auto rload = [&](auto slot, int c) __attribute__((always_inline)) {
#pragma unroll
        for (int i = 0; i < RLOADS; ++i) {
            const int seg = tid + 256 * i;
            const int row = seg >> 3, col = seg & 7;
            const int rr = row < r ? row : r - 1;
            int hc = (cbeg + c) * kZChunk + col * 8;
            hc = hc < h ? hc : h - 8;
            rb[decltype(slot)::value][i] = *reinterpret_cast<const u32x4*>(R1t + (int64_t)rr * h + hc);
        }
    };
    auto rstash = [&](auto slot, int buf) __attribute__((always_inline)) {
#pragma unroll
        for (int i = 0; i < RLOADS; ++i) {
            const int seg = tid + 256 * i;
            const int row = seg >> 3, col = seg & 7;
            *reinterpret_cast<u32x4*>(&r1s[buf][row * LROW + col * 8]) = rb[decltype(slot)::value][i];
        }
    };

    f32x16 acc[RT];
#pragma unroll
    for (int pt = 0; pt < RT; ++pt) acc[pt] = zero_f32x16();
    if (nc > 0) {
        unroll<D>([&](auto s) __attribute__((always_inline)) {
            xload(s, decltype(s)::value);
            rload(s, decltype(s)::value);
        });
        rstash(std::integral_constant<int, 0>{}, 0);
        rload(std::integral_constant<int, 0>{}, D);
        __syncthreads();
        for (int cb = 0; cb < nc; cb += D) {
            unroll<D>([&](auto p) __attribute__((always_inline)) {
                constexpr int P = decltype(p)::value;
                const int c = cb + P;
                if (c < nc) {
                    const int buf = c & 1;
#pragma unroll
                    for (int j = 0; j < 4; ++j) {
                        if (4 * (cbeg + c) + j < S) {
                            const bf16x8 b = __builtin_bit_cast(bf16x8, xb[P][j]);
#pragma unroll
                            for (int pt = 0; pt < RT; ++pt) {
                                const bf16x8 a = load_bf16x8(
                                    &r1s[buf][(32 * pt + prow) * LROW + 16 * j + 8 * half]);
                                acc[pt] = mfma_32x32x16(a, b, acc[pt]);
                            }
                        }
                    }
                    xload(p, c + D);
                    rstash(std::integral_constant<int, (P + 1) % D>{}, buf ^ 1);
                    rload(std::integral_constant<int, (P + 1) % D>{}, c + 1 + D);
                    __syncthreads();
                }
            });
        }
    }

    // Lane (n, half) holds z[n][16 c + 8 half + 0..7] in accumulator elements 8 c2 .. 8 c2 + 7
    // of tile pt (c = 2 pt + c2).  Without an h split the z pass also writes the screening
    // operands: z_hi = bf16(z) in the same layout and the error scale c of the token.
    float lo2 = 0.0f, hi2 = 0.0f;
    float* zrow = zout + ((int64_t)split * T + (tok_ok ? tok : 0)) * r + 8 * half;
    uint16_t* hrow = zhi_out + (tok_ok ? tok : 0) * (int64_t)r + 8 * half;
#pragma unroll
    for (int pt = 0; pt < RT; ++pt) {
#pragma unroll
        for (int c2 = 0; c2 < 2; ++c2) {
            const int c = 2 * pt + c2;
            if (16 * c < r) {
                f32x4 lo4, hi4;
                bf16x8 hb;
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    lo4[q] = acc[pt][8 * c2 + q];
                    hi4[q] = acc[pt][8 * c2 + 4 + q];
                }
#pragma unroll
                for (int q = 0; q < 8; ++q) {
                    const float v = acc[pt][8 * c2 + q];
                    hb[q] = (__bf16)v;
                    const float hf = (float)hb[q];
                    const float lf = v - hf;
                    hi2 = fmaf(hf, hf, hi2);
                    lo2 = fmaf(lf, lf, lo2);
                }
                if (tok_ok) {
                    *reinterpret_cast<f32x4*>(zrow + 16 * c) = lo4;
                    *reinterpret_cast<f32x4*>(zrow + 16 * c + 4) = hi4;
                    if (hsplit == 1)
                        *reinterpret_cast<u32x4*>(hrow + 16 * c) = __builtin_bit_cast(u32x4, hb);
                }
            }
        }
    }
    if (hsplit == 1) {
        hi2 += __shfl_xor(hi2, 32, kWave);
        lo2 += __shfl_xor(lo2, 32, kWave);
        if (tok_ok && half == 0) c_out[tok] = screen_scale(lo2, hi2, r);
    }
}

// Sums the h-split partials of z (per element, splits in increasing order), then writes z,
// z_hi = bf16(z) and the token's error scale c.  256 threads = 256 / r tokens, one thread per
// element; the r threads of a token are consecutive lanes of one wave.
__global__ __launch_bounds__(256) void zreduce_kernel(const float* __restrict__ zparts,
                                                      float* __restrict__ z,
                                                      uint16_t* __restrict__ zhi,
                                                      float* __restrict__ cz, int32_t T,
                                                      int32_t r, int32_t splits) {
    const int64_t n = (int64_t)T * r;
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    const bool ok = i < n;
    float s = 0.0f;
    if (ok) {
        // 16 partials are loaded before they are added (still in split order).
        int p = 0;
        for (; p + 16 <= splits; p += 16) {
            float v[16];
#pragma unroll
            for (int j = 0; j < 16; ++j) v[j] = zparts[(int64_t)(p + j) * n + i];
#pragma unroll
            for (int j = 0; j < 16; ++j) s += v[j];
        }
        for (; p < splits; ++p) s += zparts[(int64_t)p * n + i];
    }
    const __bf16 hb = (__bf16)s;
    const float hf = (float)hb;
    const float lf = s - hf;
    float hi2 = hf * hf, lo2 = lf * lf;
    for (int m = 1; m < r; m <<= 1) {
        hi2 += __shfl_xor(hi2, m, kWave);
        lo2 += __shfl_xor(lo2, m, kWave);
    }
    if (ok) {
        z[i] = s;
        zhi[i] = __builtin_bit_cast(uint16_t, hb);
        if (i % r == 0) cz[i / r] = screen_scale(lo2, hi2, r);
    }
}

// Screening sweep.  For each accumulator group q of a tile the lane forms the lower bound
// max_{e in group} s_e - c N_g (attained by one expert of the group) and keeps the maxima of
// these bounds in L = 4U buckets (group q of tile t goes to bucket 4 (t mod U) + q).  The
// buckets of a token's two lanes partition the chunk's experts into 2L >= 2K groups, so the
// K largest bucket maxima belong to K distinct experts, each with logit >= its value.
// Output per token and chunk: those K values, descending, in top[chunk][token][0..K-1].
template <int RC, int K>
__global__ __launch_bounds__(kRouteThreads, 2) void screen_kernel(
    const uint16_t* __restrict__ zh, const float* __restrict__ cz,
    const uint16_t* __restrict__ R2t, int32_t T, int32_t M, int32_t chunks, int32_t splits,
    float* __restrict__ gnorm, float* __restrict__ top) {
    using C = RouteCfg<RC, K>;
    constexpr int L = C::L, TPW = C::TPW;
    __shared__ __attribute__((aligned(16))) uint16_t rows[C::EMAX * C::R];
    __shared__ __attribute__((aligned(16))) float gn[C::EMAX / 4];
    const RouteSplit sp = route_split(T, M, chunks, splits, C::TOK);
    // With one token split (small T) the group norms of the chunk are computed here from LDS
    // and published for the collect kernel; otherwise the z pass has written them.
    load_chunk<RC, K>(R2t, gnorm, M, sp.t0, sp.t1, rows, gn, splits > 1);
    if (splits == 1) chunk_group_norms<RC, K>(rows, M, sp.t0, sp.t1, gn, gnorm);
    const int lane = threadIdx.x & 63;
    const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int n = lane & 31, half = lane >> 5;
    const LdsRows<RC, K> src(rows, gn, n, half);

    TokenGroups<RC, TPW> tg, nx;
    const int64_t wofs = (int64_t)w * 32 * TPW;
    if constexpr (C::PREFETCH) {
        if (sp.blk0 < sp.blk1 && sp.blk0 * C::TOK + wofs < T)
            tg.load(zh, cz, T, sp.blk0 * C::TOK + wofs, n, half);
    }
    for (int64_t blk = sp.blk0; blk < sp.blk1; ++blk) {
        const int64_t first = blk * C::TOK + wofs;
        if (first >= T) break;  // wave-uniform
        const bool has_next = blk + 1 < sp.blk1 && first + C::TOK < T;
        if constexpr (C::PREFETCH) {
            // the next block's operands are loaded while the current block is swept
            if (has_next) nx.load(zh, cz, T, first + C::TOK, n, half);
        } else {
            tg.load(zh, cz, T, first, n, half);
        }
        float bm[TPW][L];
#pragma unroll
        for (int g = 0; g < TPW; ++g)
#pragma unroll
            for (int b = 0; b < L; ++b) bm[g][b] = -__builtin_huge_valf();
        sweep<RC, K, TPW, 1>(
            src, (int)(sp.t1 - sp.t0), (int32_t)(sp.t0 * 32), M, half, tg.zhi,
            [&](auto gg, f32x16& acc, int32_t e0, auto u, const f32x4& nq)
                __attribute__((always_inline)) {
                constexpr int g = decltype(gg)::value;
                constexpr int UB = 4 * decltype(u)::value;
                (void)e0;
#pragma unroll
                for (int q = 0; q < 4; ++q)
                    bm[g][UB + q] = fmaxf(bm[g][UB + q], max4(acc, q) - tg.c[g] * nq[q]);
            });
        // K largest of each token's 2L bucket maxima.
#pragma unroll
        for (int g = 0; g < TPW; ++g) {
            sort_desc<L>(bm[g]);
            float pb[L];  // the two lanes' lists (merging is symmetric)
#pragma unroll
            for (int b = 0; b < L; ++b) lane_pair32(bm[g][b], bm[g][b], pb[b]);
            vlist_merge<L>(bm[g], pb);
            if (half == 0 && tg.tok_ok(g, n)) {
                float* o = top + ((int64_t)sp.chunk * T + tg.tok(g, n)) * K;
#pragma unroll
                for (int j = 0; j < K; ++j) o[j] = bm[g][j];
            }
        }
        if constexpr (C::PREFETCH) {
            if (has_next) tg = nx;
        }
    }
}

// Threshold per token: theta = the k-th largest of the union of all chunks' lists, lowered by
// a rounding guard.  k distinct experts have logit >= theta, so the k-th largest logit is >=
// theta and every expert of the top k has s_e + c N_g >= theta.  G threads per token (a power
// of two <= 64) share the chunk lists.  Also clears the token's candidate count and, when
// hist is set, the per-expert histogram.
template <int K>
__global__ __launch_bounds__(256) void theta_kernel(const float* __restrict__ top, int32_t T,
                                                    int32_t chunks, int32_t k, int32_t G,
                                                    float* __restrict__ theta,
                                                    int32_t* __restrict__ count,
                                                    int32_t* __restrict__ hist, int32_t M) {
    const int64_t gid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (hist) {  // clear the per-expert histogram for this call
        for (int64_t e = gid; e < M; e += (int64_t)gridDim.x * blockDim.x) hist[e] = 0;
    }
    const int64_t tok = gid / G;
    const int g = (int)(gid % G);
    const bool ok = tok < T;
    const int64_t t = ok ? tok : 0;
    float v[K];
#pragma unroll
    for (int j = 0; j < K; ++j) v[j] = -__builtin_huge_valf();
    // Lists are loaded B at a time before they are merged, so that their loads overlap.
    constexpr int B = K <= 8 ? 4 : (K <= 16 ? 2 : 1);
    for (int c0 = g; c0 < chunks; c0 += B * G) {
        float b[B][K];
#pragma unroll
        for (int u = 0; u < B; ++u) {
            const int c = c0 + u * G;
            const bool in = c < chunks;
            const f32x4* p = reinterpret_cast<const f32x4*>(top + ((int64_t)(in ? c : 0) * T + t) * K);
#pragma unroll
            for (int j = 0; j < K; j += 4) {
                if (K >= 4) {
                    const f32x4 q = p[j / 4];
#pragma unroll
                    for (int i = 0; i < 4; ++i) b[u][j + i] = in ? q[i] : -__builtin_huge_valf();
                } else {
#pragma unroll
                    for (int i = 0; i < K; ++i)
                        b[u][i] = in ? top[((int64_t)c * T + t) * K + i] : -__builtin_huge_valf();
                }
            }
        }
#pragma unroll
        for (int u = 0; u < B; ++u) vlist_merge<K>(v, b[u]);
    }
    for (int s = 1; s < G; s <<= 1) {
        float b[K];
#pragma unroll
        for (int j = 0; j < K; ++j) b[j] = __shfl_xor(v[j], s, kWave);
        vlist_merge<K>(v, b);
    }
    if (!ok || g != 0) return;
    float th = v[0];
#pragma unroll
    for (int j = 1; j < K; ++j)
        if (j == k - 1) th = v[j];
    // Clamped to -2^100: logits are finite and far smaller in magnitude, and masked (-inf)
    // entries stay below every threshold derived from it.
    theta[tok] = fmaxf(th - fabsf(th) * 0x1p-20f, -0x1p100f);
    count[tok] = 0;
}

// Collect sweep: recomputes s for the chunk and appends every expert with s_e + c N_g >=
// theta[token] to the token's candidate list cand[token][0..cap-1] (order of arrival,
// count[token] entries).  A lane buffers its hits in SLOTS LDS slots per token group (16-bit
// offsets in the chunk); the token's two lanes reserve their list space with one atomic add
// at the end of the token block.  A lane with more hits marks the token as overflowed (count
// > cap), which sends it to the exact sweep of the finalize kernel.
template <int RC, int K>
__global__ __launch_bounds__(kRouteThreads, 2) void collect_kernel(
    const uint16_t* __restrict__ zh, const float* __restrict__ cz,
    const uint16_t* __restrict__ R2t, int32_t T, int32_t M, int32_t chunks, int32_t splits,
    const float* __restrict__ theta, const float* __restrict__ gnorm,
    int32_t* __restrict__ count, int32_t* __restrict__ cand, int32_t cap) {
    using C = RouteCfg<RC, K>;
    constexpr int TPW = C::TPW, S = C::SLOTS;
    __shared__ __attribute__((aligned(16))) uint16_t rows[C::EMAX * C::R];
    __shared__ __attribute__((aligned(16))) float gn[C::EMAX / 4];
    __shared__ uint16_t slots[S][TPW][kRouteThreads];
    const RouteSplit sp = route_split(T, M, chunks, splits, C::TOK);
    load_chunk<RC, K>(R2t, gnorm, M, sp.t0, sp.t1, rows, gn);
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int n = lane & 31, half = lane >> 5;
    const int32_t ebase = (int32_t)(sp.t0 * 32);
    const LdsRows<RC, K> src(rows, gn, n, half);

    TokenGroups<RC, TPW> tg, nx;
    float th[TPW], nth[TPW];
    auto load_theta = [&](const TokenGroups<RC, TPW>& q, float (&o)[TPW])
                          __attribute__((always_inline)) {
#pragma unroll
        for (int g = 0; g < TPW; ++g)  // lanes past T never qualify (+inf threshold)
            o[g] = q.tok_ok(g, n) ? theta[q.tok(g, n)] : __builtin_huge_valf();
    };
    const int64_t wofs = (int64_t)w * 32 * TPW;
    if constexpr (C::PREFETCH) {
        if (sp.blk0 < sp.blk1 && sp.blk0 * C::TOK + wofs < T) {
            tg.load(zh, cz, T, sp.blk0 * C::TOK + wofs, n, half);
            load_theta(tg, th);
        }
    }
    for (int64_t blk = sp.blk0; blk < sp.blk1; ++blk) {
        const int64_t first = blk * C::TOK + wofs;
        if (first >= T) break;  // wave-uniform
        const bool has_next = blk + 1 < sp.blk1 && first + C::TOK < T;
        if constexpr (C::PREFETCH) {
            // the next block's operands and thresholds are loaded while this block is swept
            if (has_next) {
                nx.load(zh, cz, T, first + C::TOK, n, half);
                load_theta(nx, nth);
            }
        } else {
            tg.load(zh, cz, T, first, n, half);
            load_theta(tg, th);
        }
        int cnt[TPW];
#pragma unroll
        for (int g = 0; g < TPW; ++g) cnt[g] = 0;
        sweep<RC, K, TPW, 1>(
            src, (int)(sp.t1 - sp.t0), (int32_t)(sp.t0 * 32), M, half, tg.zhi,
            [&](auto gg, f32x16& acc, int32_t e0, auto u, const f32x4& nq)
                __attribute__((always_inline)) {
                constexpr int g = decltype(gg)::value;
                (void)u;
                cnt[g] = collect_tile<S>(acc, th[g], tg.c[g], nq, (e0 - ebase) / 4 + half, cnt[g],
                                         [&](int i) { return &slots[i][g][tid]; });
            });
#pragma unroll
        for (int g = 0; g < TPW; ++g) {
            auto slot = [&](int i) { return &slots[i][g][tid]; };
            const int ne = slot_experts<S>(cnt[g], slot, ebase, M);
            const int pe = __shfl_xor(ne, 32, kWave);
            const int pc = __shfl_xor(cnt[g], 32, kWave);
            const bool over = cnt[g] > S || pc > S;
            const int total = ne + pe;
            int base = 0;
            const int64_t tk = tg.tok(g, n);
            if (half == 0 && tk < T && total > 0)
                base = atomicAdd(&count[tk], over ? cap + 1 : total);
            base = __shfl(base, n, kWave);  // lane half 1 reads its partner's reservation
            if (tk < T && !over) {
                const int off = base + (half ? pe : 0);
                if (off < cap)
                    slot_expand(cnt[g], slot, ebase, M, cand + tk * cap + off, cap - off);
            }
        }
        if constexpr (C::PREFETCH) {
            if (has_next) {
                tg = nx;
#pragma unroll
                for (int g = 0; g < TPW; ++g) th[g] = nth[g];
            }
        }
    }
}

// Final selection over the global candidate lists of the collect kernel, 32 tokens per
// workgroup.  With RCAP > 0 tokens with up to RCAP candidates take the rank-counting path:
// shorter latency, chosen when there are few workgroups (small T); with many workgroups the
// list path's fewer barriers and LDS round trips win.
template <int RC, int K, int RCAP>
__global__ __launch_bounds__(256) void finalize_kernel(
    const float* __restrict__ z, const uint16_t* __restrict__ R2t, int32_t T, int32_t M,
    int32_t k, const int32_t* __restrict__ count, const int32_t* __restrict__ cand, int32_t cap,
    int32_t* __restrict__ idx, float* __restrict__ gate, float* __restrict__ topval) {
    __shared__ __attribute__((aligned(16))) float lv[32 * (RCAP > 0 ? RCAP : 1)];
    __shared__ __attribute__((aligned(16))) int32_t le[32 * (RCAP > 0 ? RCAP : 1)];
    const int64_t tok0 = (int64_t)blockIdx.x * 32;
    finalize_tokens<RC, K, 256, RCAP>(
        [&](int j) __attribute__((always_inline)) {
            return z + (tok0 + j < T ? tok0 + j : 0) * (16 * RC);
        },
        R2t, T, M, k, tok0, cap,
        [&](int j) __attribute__((always_inline)) { return count[tok0 + j]; },
        [&](int j, int i) __attribute__((always_inline)) { return cand[(tok0 + j) * cap + i]; },
        lv, le, idx, gate, topval);
}

// ------------------------------------------------------------------------------ fused route
// One workgroup routes 64 tokens against the whole expert axis, for expert sets small enough
// that every workgroup can hold or re-read all of R2t: wave w sweeps tiles [Mt w / 8,
// Mt (w + 1) / 8) for the workgroup's two token groups.  The screening pass, the threshold, the
// collect pass and the final selection run in the workgroup with LDS for the exchanges, so one
// launch replaces the screen, threshold, collect and finalize kernels (same screening bounds,
// same candidate guarantee, same exact evaluation).
//   fused_route_kernel  reads z, z_hi and the group norms written by the z pass and streams the
//                       A operands from L2, D tiles ahead (r M <= 2^18);
//   fused_local_kernel  also computes z for its tokens and a norm bound for its tiles, and
//                       keeps the A operands in registers for both passes (r M <= 2^17, K <= 8):
//                       the whole routing call is one launch.  Its z sums the h axis in four
//                       quarters (one per wave pair) added in order, so its logits may differ
//                       from the z pass's in the last bits.
constexpr int kFusedTokens = 64;
constexpr int kFusedCap = 128;   // candidates per token
constexpr int kFusedSlots = 8;   // slot entries per lane and token group in the collect pass
constexpr int kFusedRankCap = 32;  // candidates per token selected by rank counting
// A-operand ring depth (tiles loaded ahead), bounded by the registers at r = 64
__host__ __device__ constexpr int fused_ring(int RC) { return RC == 2 ? 8 : (RC == 1 ? 4 : 2); }
constexpr int kFusedMaxTiles = 512;  // expert tiles whose norms fit the LDS copy (M <= 16384)
// h values per LDS-staged chunk of the local kernel's z pass: (64 + r) rows of this many bf16
// stay within 96 KiB.
__host__ __device__ constexpr int local_zchunk(int RC) { return RC <= 2 ? 512 : 256; }
// (r M <= 2^17), 64 at r = 64 (M <= 1024), next to the z pass operands).
__host__ __device__ constexpr int fused_reg_tiles(int RC) { return RC == 4 ? 4 : 32 / RC; }

// LDS of the fused phases.
template <int K>
struct FusedLds {
    // per token and wave: K best bucket maxima (the token's row padded by 16 bytes, so that
    // the 32 tokens a wave writes at once spread over the banks)
    float tops[kFusedTokens][kRouteWaves * K + 4];
    int32_t cand[kFusedTokens * kFusedCap];    // candidate lists
    union {
        uint32_t slots[kFusedSlots + 1][2][kRouteThreads];  // collect pass (+ overflow slot)
        struct {                                        // final selection (rank path)
            float lv[kFusedTokens][kFusedRankCap];
            int32_t le[kFusedTokens][kFusedRankCap];
        } fin;
    };
    float theta[kFusedTokens];
    int32_t count[kFusedTokens];
};

// Screening pass, threshold, collect pass and final selection of a fused workgroup;
// run_sweep(cin, body) sweeps the wave's tiles for its two token groups (operands tg, initial
// accumulators cin), zrow_of(j) is the fp32 z row of local token j.  Reached by every thread of
// the workgroup.
//
// Norm bounds.  With WN the wave uses one bound nw >= every row norm of its tiles instead of
// the per-group norms (looser by c (nw - N_g), a few 1e-3 of a logit at unit-variance rows):
//  - screen keeps bucket maxima of s itself (two v_max3 per 4-expert group) and subtracts c nw
//    once at the end; rows past M (copies of row M - 1) are set to -inf first, in the one tile
//    that has them, so that no bucket maximum is attained by a phantom row;
//  - collect starts each accumulator at b = c nw - theta + guard, so the test s_e + c nw >=
//    theta becomes the sign of the MFMA result (collect_tile_sign).  The guard (r + 2) 2^-23
//    (|theta| + c nw) covers the rounding of b and the accumulation error that |b| adds to the
//    MFMA sum (r + 1 terms, at most r 2^-24 relative each); the products' own accumulation
//    error is inside c.  So every expert with l_e >= theta gets s_e + b >= +0.
template <int RC, int K, bool WN, typename Sweep, typename WaveNorm, typename ZRowOf>
__device__ __forceinline__ void fused_phases(Sweep&& run_sweep, const TokenGroups<RC, 2>& tg,
                                             WaveNorm&& wave_norm, FusedLds<K>& sh,
                                             ZRowOf&& zrow_of,
                                             const uint16_t* __restrict__ R2t, int32_t T,
                                             int32_t M, int32_t k, int64_t tok0,
                                             int32_t* __restrict__ idx, float* __restrict__ gate,
                                             float* __restrict__ topval) {
    using C = RouteCfg<RC, K>;
    constexpr int L = C::L, TPW = 2, S = kFusedSlots, R = 16 * RC;
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int n = lane & 31, half = lane >> 5;
    float nw = 0.0f;  // the wave's norm bound (WN), taken after the screening sweep
    // Screening pass (as in screen_kernel): the wave's bucket maxima per token.
    {
        float bm[TPW][L];
        f32x16 cz[TPW];
#pragma unroll
        for (int g = 0; g < TPW; ++g) {
            cz[g] = zero_f32x16();
#pragma unroll
            for (int b = 0; b < L; ++b) bm[g][b] = -__builtin_huge_valf();
        }
        run_sweep(cz, [&](auto gg, f32x16& acc, int32_t e0, auto u, const f32x4& nq)
                          __attribute__((always_inline)) {
                              constexpr int g = decltype(gg)::value;
                              constexpr int UB = 4 * decltype(u)::value;
                              if constexpr (WN) {
                                  if (e0 + 32 > M) {  // wave-uniform: the tile reaching past M
#pragma unroll
                                      for (int i = 0; i < 16; ++i)
                                          if (e0 + acc_row(i, half) >= M)
                                              acc[i] = -__builtin_huge_valf();
                                  }
#pragma unroll
                                  for (int q = 0; q < 4; ++q) {  // two v_max3
                                      const float t = fmaxf(fmaxf(bm[g][UB + q], acc[4 * q]),
                                                            acc[4 * q + 1]);
                                      bm[g][UB + q] =
                                          fmaxf(fmaxf(t, acc[4 * q + 2]), acc[4 * q + 3]);
                                  }
                              } else {
#pragma unroll
                                  for (int q = 0; q < 4; ++q)
                                      bm[g][UB + q] =
                                          fmaxf(bm[g][UB + q], max4(acc, q) - tg.c[g] * nq[q]);
                              }
                          });
        if constexpr (WN) nw = wave_norm();
#pragma unroll
        for (int g = 0; g < TPW; ++g) {
            if constexpr (WN) {
#pragma unroll
                for (int b = 0; b < L; ++b) bm[g][b] = fmaf(-tg.c[g], nw, bm[g][b]);
            }
            sort_desc<L>(bm[g]);
            float pb[L];  // the two lanes' lists (merging is symmetric)
#pragma unroll
            for (int b = 0; b < L; ++b) lane_pair32(bm[g][b], bm[g][b], pb[b]);
            vlist_merge<L>(bm[g], pb);
            if (half == 0) {
#pragma unroll
                for (int j = 0; j < K; ++j) sh.tops[32 * g + n][w * K + j] = bm[g][j];
            }
        }
    }
    __syncthreads();
    // Threshold per token (as in theta_kernel): 8 threads per token merge the waves' lists.
    {
        const int jt = tid >> 3, sub = tid & 7;
        float v[K];
#pragma unroll
        for (int j = 0; j < K; ++j) v[j] = sh.tops[jt][sub * K + j];
        unroll<3>([&](auto ss) __attribute__((always_inline)) {
            float b[K];
#pragma unroll
            for (int j = 0; j < K; ++j) b[j] = lane_xor<(1 << decltype(ss)::value)>(v[j]);
            vlist_merge<K>(v, b);
        });
        if (sub == 0) {
            float th = v[0];
#pragma unroll
            for (int j = 1; j < K; ++j)
                if (j == k - 1) th = v[j];
            sh.theta[jt] = fmaxf(th - fabsf(th) * 0x1p-20f, -0x1p100f);
            sh.count[jt] = 0;
        }
    }
    __syncthreads();
    // Collect pass (as in collect_kernel): entries go to lane-private slots first, then their
    // experts into the token's LDS list with one reservation per lane (a lane with more than S
    // entries overflows the token, which is then swept exactly).
    {
        int cnt[TPW];
        float th[TPW];
        f32x16 cb[TPW];
#pragma unroll
        for (int g = 0; g < TPW; ++g) {
            cnt[g] = 0;  // tokens past T never qualify (+inf threshold, -inf start)
            const bool ok = tg.tok_ok(g, n);
            th[g] = ok ? sh.theta[32 * g + n] : __builtin_huge_valf();
            float b = 0.0f;
            if constexpr (WN) {
                const float cn = tg.c[g] * nw;
                b = fmaf(tg.c[g], nw, -th[g]) +
                    (float)(R + 2) * 0x1p-23f * (fabsf(th[g]) + cn);
                b = ok ? b : -__builtin_huge_valf();
            }
#pragma unroll
            for (int i = 0; i < 16; ++i) cb[g][i] = b;
        }
        run_sweep(cb, [&](auto gg, f32x16& acc, int32_t e0, auto u, const f32x4& nq)
                          __attribute__((always_inline)) {
                              constexpr int g = decltype(gg)::value;
                              (void)u;
                              auto slot = [&](int i) { return &sh.slots[i][g][tid]; };
                              if constexpr (WN)
                                  cnt[g] = collect_tile_sign<S>(acc, e0 / 16 + half, cnt[g], slot);
                              else
                                  cnt[g] = collect_tile16<S>(acc, th[g], tg.c[g], nq,
                                                             e0 / 16 + half, cnt[g], slot);
                          });
        // Expansion.  The lane's entries of both token groups are read at once (independent LDS
        // reads), counted, reserved with one LDS atomic per group, then expanded.
        const LastTileMask ltm(M);
        uint32_t ent[TPW][S];
#pragma unroll
        for (int g = 0; g < TPW; ++g)
#pragma unroll
            for (int i = 0; i < S; ++i) ent[g][i] = i < cnt[g] ? sh.slots[i][g][tid] : 0u;
        int base[TPW];
#pragma unroll
        for (int g = 0; g < TPW; ++g) {
            int ne = 0;
#pragma unroll
            for (int i = 0; i < S; ++i) ne += __builtin_popcount(ltm.bits(ent[g][i]));
            base[g] = 0;
            if (cnt[g] > 0)
                base[g] = atomicAdd(&sh.count[32 * g + n], cnt[g] > S ? kFusedCap + 1 : ne);
        }
#pragma unroll
        for (int g = 0; g < TPW; ++g) {
            if (cnt[g] > 0 && cnt[g] <= S) {
                const int tl = 32 * g + n;
                int o = base[g];
#pragma unroll
                for (int i = 0; i < S; ++i) {
                    const uint32_t v = ent[g][i];
                    uint32_t m = ltm.bits(v);  // 0 for i >= cnt
                    const int32_t e = (int32_t)(v >> 17) * 32 + 4 * (int32_t)((v >> 16) & 1);
                    while (m) {
                        const int bt = __builtin_ctz(m);
                        m &= m - 1;
                        if (o < kFusedCap) sh.cand[tl * kFusedCap + o] = e + 8 * (bt >> 2) + (bt & 3);
                        ++o;
                    }
                }
            }
        }
    }
    __syncthreads();
    finalize_tokens<RC, K, kRouteThreads, kFusedRankCap>(
        zrow_of, R2t, T, M, k, tok0, kFusedCap,
        [&](int j) __attribute__((always_inline)) { return sh.count[j]; },
        [&](int j, int i) __attribute__((always_inline)) { return sh.cand[j * kFusedCap + i]; },
        &sh.fin.lv[0][0], &sh.fin.le[0][0], idx, gate, topval);
}

template <int RC, int K>
__global__ __launch_bounds__(kRouteThreads, 2) void fused_route_kernel(
    const float* __restrict__ z, const uint16_t* __restrict__ zh, const float* __restrict__ cz,
    const uint16_t* __restrict__ R2t, const float* __restrict__ gnorm, int32_t T, int32_t M,
    int32_t k, int32_t* __restrict__ hist, int32_t* __restrict__ idx, float* __restrict__ gate,
    float* __restrict__ topval) {
    constexpr int TPW = 2;
    __shared__ FusedLds<K> sh;
    __shared__ __attribute__((aligned(16))) float gn[kFusedMaxTiles * 8];
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int n = lane & 31, half = lane >> 5;
    const int64_t tok0 = (int64_t)blockIdx.x * kFusedTokens;
    if (hist) {  // clear the per-expert histogram for this call
        for (int64_t e = (int64_t)blockIdx.x * kRouteThreads + tid; e < M;
             e += (int64_t)gridDim.x * kRouteThreads)
            hist[e] = 0;
    }
    const int64_t Mt = ((int64_t)M + 31) / 32;
    for (int i = tid; i < (int)Mt * 8; i += kRouteThreads) gn[i] = gnorm[i];
    __syncthreads();

    TokenGroups<RC, TPW> tg;
    tg.load(zh, cz, T, tok0, n, half);
    const int64_t t0 = Mt * w / kRouteWaves, t1 = Mt * (w + 1) / kRouteWaves;
    const GlobalRows<RC> src(R2t, gn, M, t0, n, half);
    const int nt = (int)(t1 - t0);
    const int32_t e00 = (int32_t)(t0 * 32);
    fused_phases<RC, K, false>(
        [&](const f32x16(&)[TPW], auto&& body) __attribute__((always_inline)) {
            sweep<RC, K, TPW, fused_ring(RC)>(src, nt, e00, M, half, tg.zhi, body);
        },
        tg, [] { return 0.0f; }, sh,
        [&](int j) __attribute__((always_inline)) {
            return z + (tok0 + j < T ? tok0 + j : 0) * (16 * RC);
        },
        R2t, T, M, k, tok0, idx, gate, topval);
}

template <int RC, int K>
__global__ __launch_bounds__(kRouteThreads, 2) void fused_local_kernel(
    const uint16_t* __restrict__ x, const uint16_t* __restrict__ R1t,
    const uint16_t* __restrict__ R2t, int32_t T, int32_t h, int32_t r, int32_t M, int32_t k,
    int32_t* __restrict__ hist, int32_t* __restrict__ idx, float* __restrict__ gate,
    float* __restrict__ topval) {
    constexpr int R = 16 * RC, RT = (RC + 1) / 2, TPW = 2, NTW = fused_reg_tiles(RC);
    constexpr int ZRED = 4 * 2 * RT * 64 * 16;  // floats: [h quarter][group][tile][quad][lane][4]
    constexpr int ZSP = R + 4;  // z row stride in floats: an odd count of 16-byte segments
    constexpr int ZHC = local_zchunk(RC);       // h per staged chunk
    constexpr int STAGE = (kFusedTokens + R) * ZHC * 2;  // bytes: x rows, then R1t rows
    constexpr int POOL0 = (int)sizeof(FusedLds<K>) > 4 * ZRED ? (int)sizeof(FusedLds<K>) : 4 * ZRED;
    constexpr int POOL = POOL0 > STAGE ? POOL0 : STAGE;
    // The partial sums of z share their LDS with the later phases.
    __shared__ __attribute__((aligned(16))) unsigned char pool[POOL];
    FusedLds<K>& sh = *reinterpret_cast<FusedLds<K>*>(pool);
    float* zred = reinterpret_cast<float*>(pool);
    __shared__ __attribute__((aligned(16))) float zs[kFusedTokens * ZSP];  // z rows, fp32
    __shared__ float csp[4][2][kFusedTokens];  // shares of the squared norms of z_lo, z_hi
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int n = lane & 31, half = lane >> 5;
    const int64_t tok0 = (int64_t)blockIdx.x * kFusedTokens;
    if (hist) {  // clear the per-expert histogram for this call
        for (int64_t e = (int64_t)blockIdx.x * kRouteThreads + tid; e < M;
             e += (int64_t)gridDim.x * kRouteThreads)
            hist[e] = 0;
    }
    // The wave's expert tiles (they stay in registers for both passes).  Register slot J < nt
    // holds tile (J + rot) mod nt of the wave's slice: the rotation by workgroup spreads the
    // 32 CUs of an XCD that read the same R2t rows at once over the L2 channels.
    const int64_t Mt = ((int64_t)M + 31) / 32;
    const int64_t t0 = Mt * w / kRouteWaves, t1 = Mt * (w + 1) / kRouteWaves;
    const int nt = (int)(t1 - t0);
    const int rot = nt > 0 ? (int)(blockIdx.x % (unsigned)nt) : 0;
    const int32_t e00 = (int32_t)(t0 * 32);
    const GlobalRows<RC> src(R2t, nullptr, M, t0, n, half);  // A operands only
    bf16x8 areg[NTW][RC];
    // Slot J < nt loads tile (J + rot) mod nt, slots past nt copies of tile nt - 1.  The first
    // half of the slots is loaded during the z pass, the second half right before the screening
    // sweep, whose first tiles then run while those loads complete.
    auto load_tiles = [&](auto part) __attribute__((always_inline)) {
        unroll<NTW / 2>([&](auto jj) __attribute__((always_inline)) {
            constexpr int J = decltype(jj)::value + decltype(part)::value * (NTW / 2);
            int tj = J < nt ? J + rot : nt - 1;
            tj = tj < nt ? tj : tj - nt;
            src.load_a(tj > 0 ? tj : 0, areg[J]);
        });
    };

    // z = x R1 for the 64 tokens: wave w takes token group w & 1 and the h quarter w >> 1 of each
    // staged chunk, in the MFMA layout of the z pass (rank rows permuted so that z lands in the
    // B-operand layout).  The x rows and R1t rows of a chunk of ZHC h values are staged in LDS
    // by direct-to-LDS loads, each instruction a contiguous 1 KiB of LDS filled from whole
    // 128-byte lines (a B-operand load straight from memory touches 32 rows for 32 bytes each).
    // In LDS, 16-byte segment s of row t sits at position s ^ (t & swm), so that the 32 rows of
    // an operand read hit distinct banks.  The expert tiles are issued after the first chunk's
    // loads; the chunk barrier then waits for the staged loads only (loads complete in order).
    {
        const int zg = w & 1, hq = w >> 1;
        const int jm = n >> 3, qm = (n >> 2) & 1, im = n & 3;
        const int prow = 16 * (jm >> 1) + 8 * qm + 4 * (jm & 1) + im;
        f32x16 za[RT];
#pragma unroll
        for (int pt = 0; pt < RT; ++pt) za[pt] = zero_f32x16();
        for (int h0 = 0; h0 < h; h0 += ZHC) {
            const int hc = h - h0 < ZHC ? h - h0 : ZHC;  // multiple of 16
            const int segs = hc >> 3;                     // 16-byte segments per row
            const int swm = ((segs & -segs) < 32 ? (segs & -segs) : 32) - 1;
            const int ns = (kFusedTokens + r) * segs;
            // staging: LDS slot q = 512 i + 64 w + lane = row * segs + p; rows [0, 64) are x rows
            // tok0 + row (clamped to T - 1), rows [64, 64 + r) R1t rows.  Row offsets times h fit
            // a 24-bit multiply (h < 2^24, checked by the plan).
            int row = tid / segs, p = tid - row * segs;
            const int drow = kRouteThreads / segs, dp = kRouteThreads - drow * segs;
            const int xlast = (int)(T - 1 - tok0 < kFusedTokens ? T - 1 - tok0 : kFusedTokens - 1);
            const uint16_t* xb = x + tok0 * h + h0;
            const uint16_t* rb = R1t + h0;
            for (int q0 = 0; q0 < ns; q0 += kRouteThreads) {
                if (q0 + tid < ns) {
                    const int sg = p ^ (row & swm);
                    const bool isx = row < kFusedTokens;
                    const int roff = isx ? (row < xlast ? row : xlast) : row - kFusedTokens;
                    const uint16_t* gp =
                        (isx ? xb : rb) + __umul24((unsigned)roff, (unsigned)h) + 8 * sg;
                    lds_dma16(gp, pool + 16 * (q0 + 64 * w));
                }
                row += drow;
                p += dp;
                if (p >= segs) {
                    p -= segs;
                    ++row;
                }
            }
            if (h0 == 0) {
                __builtin_amdgcn_sched_barrier(0);
                load_tiles(std::integral_constant<int, 0>{});
                __builtin_amdgcn_sched_barrier(0);
                lds_barrier<NTW / 2 * RC>();
            } else {
                lds_barrier<0>();
            }
            const int S = hc >> 4;
            const int s0 = S * hq / 4, s1 = S * (hq + 1) / 4;
            const unsigned char* xr = pool + (32 * zg + n) * segs * 16;
            const int xsw = (32 * zg + n) & swm;
            const unsigned char* ar[RT];
            int asw[RT];
#pragma unroll
            for (int pt = 0; pt < RT; ++pt) {
                const int rr = 32 * pt + prow < r ? 32 * pt + prow : r - 1;
                ar[pt] = pool + (kFusedTokens + rr) * segs * 16;
                asw[pt] = (kFusedTokens + rr) & swm;
            }
            constexpr int ZD = 4;  // k-steps whose operands are read before they are used
            for (int sb = s0; sb < s1; sb += ZD) {
                bf16x8 xb[ZD], ab[ZD][RT];
#pragma unroll
                for (int i = 0; i < ZD; ++i) {
                    const int sg = 2 * (sb + i < s1 ? sb + i : s1 - 1) + half;
                    xb[i] = *reinterpret_cast<const bf16x8*>(xr + 16 * (sg ^ xsw));
#pragma unroll
                    for (int pt = 0; pt < RT; ++pt)
                        ab[i][pt] = *reinterpret_cast<const bf16x8*>(ar[pt] + 16 * (sg ^ asw[pt]));
                }
#pragma unroll
                for (int i = 0; i < ZD; ++i)
                    if (sb + i < s1)
#pragma unroll
                        for (int pt = 0; pt < RT; ++pt) za[pt] = mfma_32x32x16(ab[i][pt], xb[i], za[pt]);
            }
            lds_barrier();  // the chunk is consumed (the next one, or zred, reuses the LDS)
        }
#pragma unroll
        for (int pt = 0; pt < RT; ++pt) {
            f32x4* dst = reinterpret_cast<f32x4*>(zred + (((hq * 2 + zg) * RT + pt) * 256 + lane) * 4);
#pragma unroll
            for (int q = 0; q < 4; ++q)
                dst[64 * q] = f32x4{za[pt][4 * q], za[pt][4 * q + 1], za[pt][4 * q + 2], za[pt][4 * q + 3]};
        }
    }
    lds_barrier();  // (the expert tiles may still be in flight)
    {
        // The four h quarters of token group w & 1 added in order, by all 8 waves: wave w takes
        // accumulator elements 4 (w >> 1) .. 4 (w >> 1) + 3 of each tile.  z rows go to LDS, and
        // each wave's share of the token's squared norms of z_hi = bf16(z) and z_lo = z - z_hi
        // (as in the z pass) to csp; the screening scale adds the four shares in order.
        const int zg = w & 1, part = w >> 1;
        const int jt = 32 * zg + n;
        const int c2 = part >> 1, q0 = 4 * (part & 1);
        float hi2 = 0.0f, lo2 = 0.0f;
#pragma unroll
        for (int pt = 0; pt < RT; ++pt) {
            const int c = 2 * pt + c2;
            f32x4 zsum;
#pragma unroll
            for (int hq = 0; hq < 4; ++hq) {
                const f32x4 v = *reinterpret_cast<const f32x4*>(
                    zred + ((((hq * 2 + zg) * RT + pt) * 4 + part) * 64 + lane) * 4);
#pragma unroll
                for (int i = 0; i < 4; ++i) zsum[i] = hq == 0 ? v[i] : zsum[i] + v[i];
            }
            if (16 * c < r) {  // wave-uniform
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const float hf = (float)(__bf16)zsum[i];
                    const float lf = zsum[i] - hf;
                    hi2 = fmaf(hf, hf, hi2);
                    lo2 = fmaf(lf, lf, lo2);
                }
                *reinterpret_cast<f32x4*>(&zs[jt * ZSP + 16 * c + 8 * half + q0]) = zsum;
            }
        }
        hi2 = sum_pair32(hi2);
        lo2 = sum_pair32(lo2);
        if (half == 0) {
            csp[part][0][jt] = lo2;
            csp[part][1][jt] = hi2;
        }
    }
    // The wave's norm bound nw >= the norm of every row of its tiles, from the registers: a lane
    // holds half of row n of each tile, the other half sits in lane n + 32.  The squared sums use
    // bf16 dot products; their rounding (a relative 2^-18 at most) is covered by the 2^-20 and
    // 2^-10 slacks.  Slots past nt hold copies of tile nt - 1, and rows past M copies of row
    // M - 1, so they do not raise the bound.  It is evaluated after the screening sweep, whose
    // first tiles then need not wait for the last tiles' loads.
    auto wave_norm = [&]() __attribute__((always_inline)) {
        float ssn[NTW];
        unroll<NTW>([&](auto jj) __attribute__((always_inline)) {
            constexpr int J = decltype(jj)::value;
            float ss = 0.0f;
#pragma unroll
            for (int c = 0; c < RC; ++c)
#pragma unroll
                for (int q = 0; q < 8; q += 2) {
                    const bf16x2 p = {areg[J][c][q], areg[J][c][q + 1]};
                    ss = __builtin_amdgcn_fdot2_f32_bf16(p, p, ss, false);
                }
            ssn[J] = ss;
        });
        // Row n of tile J has squared norm a_J + b_J (this lane's half and lane n + 32's), at most
        // max_J a_J + max_J b_J: one pair sum after the per-lane maximum.
        float mx = 0.0f;
        unroll<NTW>([&](auto jj) __attribute__((always_inline)) {
            mx = fmaxf(mx, ssn[decltype(jj)::value]);
        });
        mx = sum_pair32(mx);
        mx = fmaxf(mx, lane_xor<1>(mx));
        mx = fmaxf(mx, lane_xor<2>(mx));
        mx = fmaxf(mx, lane_xor<4>(mx));
        mx = fmaxf(mx, lane_xor<8>(mx));
        mx = fmaxf(mx, lane_xor<16>(mx));
        return __builtin_bit_cast(float, __builtin_amdgcn_readfirstlane(
                                             __builtin_bit_cast(int, sqrtf(mx) * (1.0f + 0x1p-20f))));
    };
    lds_barrier();
    load_tiles(std::integral_constant<int, 1>{});
    __builtin_amdgcn_s_waitcnt(vmcnt_imm(NTW / 2 * RC));  // the first half is in registers
    TokenGroups<RC, TPW> tg;
    tg.first = tok0;
    tg.T = T;
#pragma unroll
    for (int g = 0; g < TPW; ++g) {
        const int jt = 32 * g + n;
        const bool ok = tg.tok_ok(g, n);
#pragma unroll
        for (int c = 0; c < RC; ++c) {
            bf16x8 v;
#pragma unroll
            for (int q = 0; q < 8; ++q) v[q] = (__bf16)zs[jt * ZSP + 16 * c + 8 * half + q];
            tg.zhi[g][c] = ok ? v : zero_bf16x8();
        }
        const float lo2 = ((csp[0][0][jt] + csp[1][0][jt]) + csp[2][0][jt]) + csp[3][0][jt];
        const float hi2 = ((csp[0][1][jt] + csp[1][1][jt]) + csp[2][1][jt]) + csp[3][1][jt];
        tg.c[g] = ok ? screen_scale(lo2, hi2, r) : 0.0f;
    }
    fused_phases<RC, K, true>(
        [&](const f32x16(&cin)[TPW], auto&& body) __attribute__((always_inline)) {
            sweep_regs<RC, K, TPW, NTW, false>(areg, nullptr, nt, rot, e00, M, half, tg.zhi, cin,
                                               body);
        },
        tg, wave_norm, sh, [&](int j) __attribute__((always_inline)) { return zs + j * ZSP; }, R2t, T,
        M, k, tok0, idx, gate, topval);
}

// ------------------------------------------------------------------------------ planning
static int pow2_at_least(int k) {
    int K = 1;
    while (K < k) K <<= 1;
    return K;
}

static size_t align256(size_t b) { return (b + 255) & ~(size_t)255; }

// Split of the z pass's h axis: 64-wide chunks per split and the number of splits.
static void zpass_split(int64_t T, int32_t h, int32_t* steps_per_split, int32_t* hsplit) {
    const int32_t NC = (h / 16 + 3) / 4;
    const int64_t ntbz = (T + kZTokens - 1) / kZTokens;
    int64_t hs = ntbz >= 256 ? 1 : (256 + ntbz - 1) / ntbz;
    if (hs > NC) hs = NC;
    *steps_per_split = (int32_t)((NC + hs - 1) / hs);
    *hsplit = (NC + *steps_per_split - 1) / *steps_per_split;
}

bool lowrank_make_plan(int64_t T, int32_t h, int32_t r, int32_t M, int32_t k, int32_t m_chunks,
                       LowrankPlan* p) {
    LowrankPlan q{};
    q.RC = r / 16;
    q.RT = (q.RC + 1) / 2;
    q.K = pow2_at_least(k);
    const int64_t Mt = ((int64_t)M + 31) / 32;
    // Library's choice on a small expert set (r M <= 2^18, i.e. R2t <= 512 KiB, read from L2 by
    // every workgroup twice): the fused route kernel.
    q.fused = m_chunks == 0 && (int64_t)r * M <= (1 << 18) && Mt <= kFusedMaxTiles;
    // ... and when the wave's tiles fit in registers (r M <= 2^17) and K <= 8, the local kernel,
    // which needs no z pass and no workspace.
    q.local = q.fused && q.K <= 8 && (Mt + kRouteWaves - 1) / kRouteWaves <= fused_reg_tiles(q.RC) &&
              h < (1 << 24);
    const int tokens_per_block = q.fused ? kFusedTokens : 32 * kRouteTPW * kRouteWaves;
    q.ntb = (int32_t)((T + tokens_per_block - 1) / tokens_per_block);
    const int64_t emax_tiles = (int64_t)kChunkBytes / (2 * r) / 32;
    if (q.fused) {
        q.chunks = 1;
    } else if (m_chunks > 0) {
        q.chunks = m_chunks;
    } else {
        // Chunks that fit the resident LDS rows, and at least 256 workgroups when there are
        // enough token blocks and tiles.
        int64_t C = (Mt + emax_tiles - 1) / emax_tiles;
        const int64_t want = (256 + q.ntb - 1) / q.ntb;
        if (C < want) C = want < Mt ? want : Mt;
        q.chunks = (int32_t)(C < 1024 ? C : 1024);
    }
    if (q.chunks < 1 || q.chunks > 1024) return false;
    // Resident rows must fit in LDS (m_chunks is a request: the result does not depend on
    // the chunking).
    while (!q.fused && (Mt + q.chunks - 1) / q.chunks > emax_tiles) {
        if (q.chunks >= (1 << 20)) return false;
        q.chunks *= 2;
    }
    // Token splits: about 256 workgroups in all, each split holding whole token blocks.
    int64_t S = q.fused ? q.ntb : 256 / q.chunks;
    if (S < 1) S = 1;
    if (S > q.ntb) S = q.ntb;
    q.splits = (int32_t)S;
    q.theta_group = 1;
    // threads per token in the threshold kernel: one per 4 chunk lists, at most 64
    while (q.theta_group < 64 && q.theta_group * 4 < q.chunks) q.theta_group *= 2;
    // z pass: 128-token blocks; the h chunks are split over workgroups when there are fewer
    // token blocks than CUs (one workgroup of 4 waves per CU streams x too slowly to leave
    // CUs idle: at T = 16384, h = 4096 two splits and the partial-sum reduction take 46 us
    // against 59 us unsplit).
    zpass_split(T, h, &q.steps_per_split, &q.hsplit);
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
    q.off_zhi = off;
    off += align256((size_t)T * r * sizeof(uint16_t));
    q.off_cz = off;
    off += align256((size_t)T * sizeof(float));
    // (the fused route keeps its lists, thresholds and candidates in LDS)
    const size_t route_ws = q.fused ? 0 : 1;
    q.off_top = off;
    off += route_ws * align256((size_t)q.chunks * T * q.K * sizeof(float));
    q.off_gnorm = off;
    off += align256((size_t)Mt * 8 * sizeof(float));
    q.off_tau = off;
    off += route_ws * align256((size_t)T * sizeof(float));
    q.cap = q.fused ? kFusedCap : 512;
    q.off_count = off;
    off += route_ws * align256((size_t)T * sizeof(int32_t));
    q.off_cand = off;
    off += route_ws * align256((size_t)T * q.cap * sizeof(int32_t));
    q.workspace_bytes = q.local ? 0 : off;
    // Single-pass route: the library's choice for expert sets of at least 32768 (below that the
    // resident route's two sweeps cost less than the single pass's records) and enough tokens to
    // fill the chip with 64-token workgroups of the z pass.  Its prescreen assumes that its tiles
    // lie below M (32 sub_tiles <= M, true at these sizes).
    q.single_pass = m_chunks == 0 && !q.fused && T >= 4096 && M >= 32768 && M <= (1 << 24) &&
                    q.K <= 16 && h < (1 << 24) &&
                    32 * ((Mt + 3) / 4 > 8 ? (Mt + 3) / 4 : 8) <= M;
    if (q.single_pass) {
        q.ntb = (int32_t)((T + 511) / 512);  // collect blocks of 512 tokens
        int64_t C = (Mt + emax_tiles - 1) / emax_tiles;
        const int64_t want = (256 + q.ntb - 1) / q.ntb;
        if (C < want) C = want < Mt ? want : Mt;
        q.chunks = (int32_t)(C < 1024 ? C : 1024);
        while ((Mt + q.chunks - 1) / q.chunks > emax_tiles) q.chunks *= 2;
        int64_t Sp = 256 / q.chunks;
        if (Sp < 1) Sp = 1;
        if (Sp > q.ntb) Sp = q.ntb;
        q.splits = (int32_t)Sp;
        // prescreen: a quarter of the expert tiles, at least 8 (one per wave); an eighth leaves
        // a looser threshold and more records for collect and finalize (2% slower on fine_grained)
        int64_t st = (Mt + 3) / 4;
        if (st < 8) st = 8;
        if (st > Mt) st = Mt;
        q.sub_tiles = (int32_t)st;
        q.cap = M > 16384 ? 1024 : 512;  // records per token (more on large expert sets)
        q.slots = 16;
        size_t o = 0;
        q.off_z = o;
        o += align256((size_t)T * r * sizeof(float));
        q.off_zhi = o;
        o += align256((size_t)T * r * sizeof(uint16_t));
        q.off_cz = o;
        o += align256((size_t)T * sizeof(float));
        q.off_theta0 = o;
        o += align256((size_t)T * sizeof(float));
        q.off_count = o;
        o += align256((size_t)T * sizeof(int32_t));
        q.off_rec = o;
        o += align256((size_t)T * q.cap * 2 * sizeof(int32_t));
        q.off_scratch = o;
        o += align256(collect_scratch_bytes((int64_t)q.chunks * q.splits, q.slots));
        q.workspace_bytes = o;
    }
    *p = q;
    return true;
}

// ------------------------------------------------------------------------------ launch
template <int RT>
static void launch_zpass(const LowrankPlan& p, const uint16_t* x, const uint16_t* R1t, float* zparts,
                         int64_t T, int32_t h, int32_t r, const uint16_t* R2t, int32_t M,
                         float* gnorm, uint16_t* zhi, float* cz, hipStream_t st) {
    const int64_t zblocks = (T + kZTokens - 1) / kZTokens;
    // group-norm workgroups, unless the expert-resident route runs one token split: then its
    // screen kernel computes the norms from its LDS chunk (each chunk is loaded once)
    const int64_t nblocks =
        p.fused || p.splits > 1
            ? (((int64_t)M + 31) / 32 * 32 * (r / 8) + 256 * kGroupNormBlocks - 1) /
                  (256 * kGroupNormBlocks)
            : 0;
    dim3 grid((unsigned)(zblocks * p.hsplit + nblocks));
    constexpr int D = 2;
    hipLaunchKernelGGL((zpass_kernel<RT, D>), grid, dim3(256), 0, st, x, R1t, zparts, (int32_t)T,
                       h, r, p.steps_per_split, R2t, M, (int32_t)zblocks, p.hsplit, gnorm, zhi,
                       cz);
}

struct RouteArgs {
    const float* z;
    uint16_t* zhi;
    float* cz;
    const uint16_t* R2t;
    int32_t T, M, k;
    float *top, *gnorm, *theta;
    int32_t *count, *cand, *hist;
    int32_t* idx;
    float *gate, *topval;
};

template <int RC, int K>
static void launch_route(const LowrankPlan& p, const RouteArgs& a, hipStream_t st) {
    if (p.fused) {
        hipLaunchKernelGGL((fused_route_kernel<RC, K>), dim3((unsigned)p.ntb),
                           dim3(kRouteThreads), 0, st, a.z, a.zhi, a.cz, a.R2t, a.gnorm, a.T,
                           a.M, a.k, a.hist, a.idx, a.gate, a.topval);
        return;
    }
    const dim3 grid((unsigned)((int64_t)p.splits * p.chunks));
    hipLaunchKernelGGL((screen_kernel<RC, K>), grid, dim3(kRouteThreads), 0, st, a.zhi, a.cz,
                       a.R2t, a.T, a.M, p.chunks, p.splits, a.gnorm, a.top);
    const int64_t nth = (int64_t)a.T * p.theta_group;
    hipLaunchKernelGGL((theta_kernel<K>), dim3((unsigned)((nth + 255) / 256)), dim3(256), 0, st,
                       a.top, a.T, p.chunks, a.k, p.theta_group, a.theta, a.count, a.hist, a.M);
    hipLaunchKernelGGL((collect_kernel<RC, K>), grid, dim3(kRouteThreads), 0, st, a.zhi, a.cz,
                       a.R2t, a.T, a.M, p.chunks, p.splits, a.theta, a.gnorm, a.count, a.cand,
                       p.cap);
    const dim3 fgrid((unsigned)((a.T + 31) / 32));
    if (a.T <= 32 * 256)  // at most one workgroup per CU
        hipLaunchKernelGGL((finalize_kernel<RC, K, 32>), fgrid, dim3(256), 0, st, a.z, a.R2t, a.T,
                           a.M, a.k, a.count, a.cand, p.cap, a.idx, a.gate, a.topval);
    else
        hipLaunchKernelGGL((finalize_kernel<RC, K, 0>), fgrid, dim3(256), 0, st, a.z, a.R2t, a.T,
                           a.M, a.k, a.count, a.cand, p.cap, a.idx, a.gate, a.topval);
}

template <int RC>
static bool dispatch_route_k(const LowrankPlan& p, const RouteArgs& a, hipStream_t st) {
    switch (p.K) {
        case 1: launch_route<RC, 1>(p, a, st); return true;
        case 2: launch_route<RC, 2>(p, a, st); return true;
        case 4: launch_route<RC, 4>(p, a, st); return true;
        case 8: launch_route<RC, 8>(p, a, st); return true;
        case 16: launch_route<RC, 16>(p, a, st); return true;
    }
    return false;
}

template <int RC, int K>
static void launch_local(const LowrankPlan& p, const uint16_t* x, const uint16_t* R1t,
                         const uint16_t* R2t, int64_t T, int32_t h, int32_t r, int32_t M,
                         int32_t k, int32_t* hist, int32_t* idx, float* gate, float* topval,
                         hipStream_t st) {
    hipLaunchKernelGGL((fused_local_kernel<RC, K>), dim3((unsigned)p.ntb), dim3(kRouteThreads), 0,
                       st, x, R1t, R2t, (int32_t)T, h, r, M, k, hist, idx, gate, topval);
}

template <int RC>
static bool dispatch_local_k(const LowrankPlan& p, const uint16_t* x, const uint16_t* R1t,
                             const uint16_t* R2t, int64_t T, int32_t h, int32_t r, int32_t M,
                             int32_t k, int32_t* hist, int32_t* idx, float* gate, float* topval,
                             hipStream_t st) {
    switch (p.K) {
        case 1: launch_local<RC, 1>(p, x, R1t, R2t, T, h, r, M, k, hist, idx, gate, topval, st);
            return true;
        case 2: launch_local<RC, 2>(p, x, R1t, R2t, T, h, r, M, k, hist, idx, gate, topval, st);
            return true;
        case 4: launch_local<RC, 4>(p, x, R1t, R2t, T, h, r, M, k, hist, idx, gate, topval, st);
            return true;
        case 8: launch_local<RC, 8>(p, x, R1t, R2t, T, h, r, M, k, hist, idx, gate, topval, st);
            return true;
    }
    return false;
}

size_t zonly_workspace_bytes(int64_t T, int32_t h, int32_t r) {
    int32_t sps, hs;
    zpass_split(T, h, &sps, &hs);
    return (hs > 1 ? align256((size_t)hs * T * r * sizeof(float)) : 0) +
           align256((size_t)T * r * sizeof(uint16_t)) + align256((size_t)T * sizeof(float));
}

hipError_t zonly_launch(const uint16_t* x, const uint16_t* R1t, int64_t T, int32_t h, int32_t r,
                        float* z, void* scratch, hipStream_t st) {
    int32_t sps, hs;
    zpass_split(T, h, &sps, &hs);
    char* s = static_cast<char*>(scratch);
    float* zparts = hs > 1 ? reinterpret_cast<float*>(s) : z;
    const size_t o1 = hs > 1 ? align256((size_t)hs * T * r * sizeof(float)) : 0;
    uint16_t* zhi = reinterpret_cast<uint16_t*>(s + o1);
    float* cz = reinterpret_cast<float*>(s + o1 + align256((size_t)T * r * sizeof(uint16_t)));
    const int64_t zblocks = (T + kZTokens - 1) / kZTokens;
    const dim3 grid((unsigned)(zblocks * hs));  // no group-norm workgroups
    constexpr int D = 2;
    switch ((r / 16 + 1) / 2) {
        case 1:
            hipLaunchKernelGGL((zpass_kernel<1, D>), grid, dim3(256), 0, st, x, R1t, zparts,
                               (int32_t)T, h, r, sps, nullptr, 0, (int32_t)zblocks, hs, nullptr,
                               zhi, cz);
            break;
        case 2:
            hipLaunchKernelGGL((zpass_kernel<2, D>), grid, dim3(256), 0, st, x, R1t, zparts,
                               (int32_t)T, h, r, sps, nullptr, 0, (int32_t)zblocks, hs, nullptr,
                               zhi, cz);
            break;
        default: return hipErrorInvalidValue;
    }
    if (hs > 1) {
        const int64_t n = T * r;
        hipLaunchKernelGGL(zreduce_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, st,
                           zparts, z, zhi, cz, (int32_t)T, r, hs);
    }
    return hipGetLastError();
}

hipError_t lowrank_launch(const LowrankPlan& p, const uint16_t* x, const uint16_t* R1t,
                          const uint16_t* R2t, int64_t T, int32_t h, int32_t r, int32_t M,
                          int32_t k, int32_t* idx, float* gate, float* topval, int32_t* counts,
                          void* workspace, hipStream_t st) {
    if (p.local) {  // one launch, no workspace
        bool ok = false;
        switch (p.RC) {
            case 1: ok = dispatch_local_k<1>(p, x, R1t, R2t, T, h, r, M, k, counts, idx, gate, topval, st); break;
            case 2: ok = dispatch_local_k<2>(p, x, R1t, R2t, T, h, r, M, k, counts, idx, gate, topval, st); break;
            case 4: ok = dispatch_local_k<4>(p, x, R1t, R2t, T, h, r, M, k, counts, idx, gate, topval, st); break;
        }
        if (!ok) return hipErrorInvalidValue;
        return hipGetLastError();
    }
    char* ws = static_cast<char*>(workspace);
    if (p.single_pass) {
        SinglePassArgs s;
        s.x = x;
        s.R1t = R1t;
        s.R2t = R2t;
        s.T = (int32_t)T;
        s.h = h;
        s.r = r;
        s.M = M;
        s.k = k;
        s.z = reinterpret_cast<float*>(ws + p.off_z);
        s.zhi = reinterpret_cast<uint16_t*>(ws + p.off_zhi);
        s.cz = reinterpret_cast<float*>(ws + p.off_cz);
        s.theta0 = reinterpret_cast<float*>(ws + p.off_theta0);
        s.count = reinterpret_cast<int32_t*>(ws + p.off_count);
        s.rec = reinterpret_cast<int2*>(ws + p.off_rec);
        s.scratch = ws + p.off_scratch;
        s.hist = counts;
        s.idx = idx;
        s.gate = gate;
        s.topval = topval;
        return single_pass_launch(p, s, st);
    }
    float* zparts = reinterpret_cast<float*>(ws + p.off_zparts);
    RouteArgs a;
    a.z = reinterpret_cast<float*>(ws + p.off_z);
    a.zhi = reinterpret_cast<uint16_t*>(ws + p.off_zhi);
    a.cz = reinterpret_cast<float*>(ws + p.off_cz);
    a.R2t = R2t;
    a.T = (int32_t)T;
    a.M = M;
    a.k = k;
    a.top = reinterpret_cast<float*>(ws + p.off_top);
    a.gnorm = reinterpret_cast<float*>(ws + p.off_gnorm);
    a.theta = reinterpret_cast<float*>(ws + p.off_tau);
    a.count = reinterpret_cast<int32_t*>(ws + p.off_count);
    a.cand = reinterpret_cast<int32_t*>(ws + p.off_cand);
    a.hist = counts;
    a.idx = idx;
    a.gate = gate;
    a.topval = topval;

    switch (p.RT) {
        case 1: launch_zpass<1>(p, x, R1t, zparts, T, h, r, R2t, M, a.gnorm, a.zhi, a.cz, st);
            break;
        case 2: launch_zpass<2>(p, x, R1t, zparts, T, h, r, R2t, M, a.gnorm, a.zhi, a.cz, st);
            break;
        default: return hipErrorInvalidValue;
    }
    if (p.hsplit > 1) {
        const int64_t n = T * r;
        hipLaunchKernelGGL(zreduce_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, st,
                           zparts, const_cast<float*>(a.z), a.zhi, a.cz, (int32_t)T, r,
                           p.hsplit);
    }
    bool ok = false;
    switch (p.RC) {
        case 1: ok = dispatch_route_k<1>(p, a, st); break;
        case 2: ok = dispatch_route_k<2>(p, a, st); break;
        case 4: ok = dispatch_route_k<4>(p, a, st); break;
    }
    if (!ok) return hipErrorInvalidValue;
    return hipGetLastError();
}

}  // namespace more
