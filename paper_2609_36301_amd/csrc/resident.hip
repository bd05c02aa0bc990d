// Single-pass expert-resident route of the low-rank router (gfx950), for many tokens and large
// expert sets: softmax(TopK(x R1 R2)) in three launches (plus the histogram kernel), without the
// T x M logits in memory (Appendix "Pseudocode", inference algorithm; MoRE layer in
// "Preliminaries").
//
//   zscreen_kernel   z = x R1 for 64 tokens per workgroup (x read once, straight into the MFMA
//                    B operands), z_hi = bf16(z) and the screening scale c; then a prescreen of
//                    the first `sub_tiles` expert tiles (staged per wave through LDS) gives each
//                    token a threshold theta0 that k distinct experts provably reach;
//   collect_kernel1  one MFMA pass over the whole expert axis, each workgroup holding one chunk
//                    of expert rows in LDS: every expert whose screened upper bound reaches the
//                    token's theta0 is recorded as (expert, upper bound);
//   finalize_kernel2 per token: the records with the largest upper bounds are evaluated exactly
//                    in fp32, the k-th of those logits, theta1, is a tighter lower bound of the
//                    k-th logit, and the records whose upper bound reaches theta1 are evaluated
//                    as well; the top k of the exact logits and their softmax.
//
// The paper's kernel keeps a running top-k buffer per token block over all expert tiles; here
// the expert axis is split over workgroups, so a token's threshold must exist before the expert
// pass: the prescreen provides it, from a fraction of the experts, and the exact evaluation of
// the few records above it replaces the running buffer.  Every step is exact: the result is
// the top k under the total order (larger logit first, then smaller expert id) of the fp32
// logits z . u_e, with z in fp32 and the expert rows in bf16.
//
// Screening bounds.  s_e = z_hi . u_e is computed on the matrix cores; with the token's scale
// c (route_device.h) and N >= ||u_e||, s_e - c N <= l_e <= s_e + c N.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "device_common.h"
#include "lowrank.h"
#include "route_device.h"

namespace more {

constexpr int kZsTokens = 64;          // tokens per zscreen workgroup (two groups of 32)
constexpr int kCollectTPW = 2;         // token groups of 32 per collect wave
constexpr int kCollectTokens = 32 * kCollectTPW * kRouteWaves;  // tokens per collect block

// ------------------------------------------------------------------------------ zscreen
// LDS of a zscreen workgroup.  The staged x chunks, then the k-split partial sums of z, then
// the waves' top-K lists of the prescreen share one buffer.
constexpr int kZsChunk = 256;          // h values per staged chunk (32 segments of 16 bytes)
constexpr int kZsStages = 4;           // staged chunks in the ring (three in flight)
template <int RC, int K>
struct ZsLds {
    static constexpr int R = 16 * RC;
    static constexpr int RT = (RC + 1) / 2;
    static constexpr int ZSP = R + 4;  // z row stride in floats (odd count of 16 B)
    static constexpr int LPC = kZsTokens * (kZsChunk / 8) / kRouteThreads;  // loads per thread
    static constexpr int STAGE = kZsTokens * kZsChunk;                         // bf16 per stage
    union {
        uint16_t stage[kZsStages][STAGE];
        float zred[16 * 4 * 64 * 4];  // [(k-split * 2 + group) * RT + tile][quad][lane][4]
        float tops[kZsTokens][kRouteWaves * K + 4];
    };
    float zs[kZsTokens * ZSP];  // z rows, fp32
    float csp[4][2][kZsTokens];  // shares of the squared norms of z_lo and z_hi
};

// Grid: ceil(T / 64) workgroups of 8 waves.  The h axis is walked in chunks of 256: the 64 x
// rows of a chunk are staged in LDS by direct-to-LDS loads (each instruction fills a contiguous
// 1 KiB of LDS from whole 128-byte lines), four chunks in a ring with three in flight; in LDS,
// 16-byte segment p of row t sits at position p ^ (t & 31), so that the 32 rows of an operand
// read hit distinct banks.  Wave w takes rank tile w % RT and k-split w / RT (8 / RT k-splits,
// each a contiguous run of the chunk's 16 k-steps) for both token groups: its R1t operands (rank
// rows, permuted) come from L2 into a register ring one chunk ahead, its x operands from LDS, so
// each workgroup reads R1t once.  Rank row m' of tile pt is R1t row 32 pt + pi(m') with
// pi(8j + 4q + i) = 16 (j >> 1) + 8 q + 4 (j & 1) + i, so that lane (n, half) ends up holding
// z[n][16 c + 8 half + 0..7] in accumulator elements 8 c' .. 8 c' + 7 of tile pt (c = 2 pt +
// c'), the B-operand layout of the expert contraction.  The k-split partials are added in order
// in LDS.
//
// Prescreen: wave w sweeps tiles [St w / 8, St (w + 1) / 8) of the first St = sub_tiles expert
// tiles for both token groups, keeping per lane L = 4 max(1, K / 4) bucket maxima of s (group q
// of the j-th tile of the wave in bucket 4 (j mod U) + q) and the largest half-row squared norm
// it loads.  With N_w >= every row norm of the wave's tiles, bucket maximum - c N_w is a lower
// bound of the logit of the expert attaining it, and the buckets of a token's two lanes
// partition the wave's experts, so the K largest of the 2 L values belong to K distinct
// experts.  theta0 = the k-th largest of the 8 waves' K-lists, lowered by a 2^-20 relative
// guard (clamped to -2^100): k distinct experts have logits >= theta0.
//
// Also clears the record counts of its tokens and, with hist != nullptr, the histogram.
template <int RC, int K>
__global__ __launch_bounds__(kRouteThreads, 1) void zscreen_kernel(
    const uint16_t* __restrict__ x, const uint16_t* __restrict__ R1t,
    const uint16_t* __restrict__ R2t, int32_t T, int32_t h, int32_t r, int32_t M, int32_t k,
    int32_t sub_tiles, float* __restrict__ zout, uint16_t* __restrict__ zhi_out,
    float* __restrict__ cz, float* __restrict__ theta0, int32_t* __restrict__ count,
    int32_t* __restrict__ hist) {
    using Z = ZsLds<RC, K>;
    constexpr int R = 16 * RC, RT = Z::RT, ZSP = Z::ZSP;
    constexpr int U = K / 4 > 1 ? K / 4 : 1, L = 4 * U;
    __shared__ Z sh;
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int n = lane & 31, half = lane >> 5;
    const int64_t tok0 = (int64_t)blockIdx.x * kZsTokens;

    // ---- z = x R1
    {
        constexpr int LPC = Z::LPC, NS = kZsStages, KS = 8 / RT, SPW = 16 / KS;
        const int pt = w % RT, ks = w / RT;
        const int NC = (h + kZsChunk - 1) / kZsChunk;
        const int xlast = (int)(T - 1 - tok0 < kZsTokens ? T - 1 - tok0 : kZsTokens - 1);
        // staging: thread tid, load j fills LDS slot q = 512 j + tid of the stage (row q / 32,
        // position q % 32), from global segment (q % 32) ^ (row & 31) of that row
        const uint16_t* gsrc[LPC];  // x row of each of the thread's staging loads
#pragma unroll
        for (int jj = 0; jj < LPC; ++jj) {
            const int row = (kRouteThreads * jj + tid) >> 5;
            gsrc[jj] = x + (tok0 + (row < xlast ? row : xlast)) * (int64_t)h;
        }
        auto issue = [&](int c) __attribute__((always_inline)) {
            uint16_t* dst = sh.stage[c % NS];  // free: chunk c - NS is consumed
            const int h0 = (c < NC ? c : NC - 1) * kZsChunk;  // past the end: a harmless reload
#pragma unroll
            for (int jj = 0; jj < LPC; ++jj) {
                // segments past h (last chunk) re-read the row's last 16 bytes
                const int q = kRouteThreads * jj + tid;
                const int col = h0 + 8 * ((q & 31) ^ ((q >> 5) & 31));
                lds_dma16(gsrc[jj] + (col < h ? col : h - 8), dst + 8 * (kRouteThreads * jj + 64 * w));
            }
        };
        const int jm = n >> 3, qm = (n >> 2) & 1, im = n & 3;
        const int prow = 16 * (jm >> 1) + 8 * qm + 4 * (jm & 1) + im;
        const int rr = 32 * pt + prow < r ? 32 * pt + prow : r - 1;
        const uint16_t* ap = R1t + (int64_t)rr * h + 8 * half;
        // R1t operands of chunk c (the wave's SPW k-steps), in a ring of NS chunks issued right
        // before the chunk's x stage, so that one vmcnt wait covers both; k-steps past h re-read
        // the row's last 16 values (their MFMAs are skipped)
        bf16x8 ab[NS][SPW];
        auto fetch_a = [&](auto buf, int c) __attribute__((always_inline)) {
#pragma unroll
            for (int i = 0; i < SPW; ++i) {
                int col = c * kZsChunk + 16 * (ks * SPW + i);
                col = col < h ? col : h - 16;
                ab[decltype(buf)::value][i] = load_bf16x8(ap + col);
            }
        };
        f32x16 za[2] = {zero_f32x16(), zero_f32x16()};
        // One chunk; FULL: all 16 k-steps exist (no guard, so that the compiler's wait counts stay
        // exact and the staged chunks remain in flight).
        auto chunk = [&](auto buf, auto full, int c) __attribute__((always_inline)) {
            constexpr int B = decltype(buf)::value;
            // chunk c (x stage and R1t operands) has arrived and every wave is done with c - 1
            lds_barrier<(NS - 2) * (LPC + SPW)>();
            fetch_a(std::integral_constant<int, (B + NS - 1) % NS>{}, c + NS - 1);
            issue(c + NS - 1);
            const uint16_t* st = sh.stage[B];
            const int steps = (h - c * kZsChunk) >> 4;  // 16-wide k-steps in this chunk
#pragma unroll
            for (int i = 0; i < SPW; ++i) {
                const int s = ks * SPW + i;
                if (decltype(full)::value || s < steps) {
                    const int seg = 2 * s + half;
#pragma unroll
                    for (int g = 0; g < 2; ++g) {
                        const int brow = 32 * g + n;
                        const bf16x8 b = *reinterpret_cast<const bf16x8*>(
                            st + brow * kZsChunk + 8 * (seg ^ (brow & 31)));
                        za[g] = mfma_32x32x16(ab[B][i], b, za[g]);
                    }
                }
            }
        };
        unroll<NS - 1>([&](auto c) __attribute__((always_inline)) {
            fetch_a(c, decltype(c)::value);
            issue(decltype(c)::value);
        });
        const int NCF = h / kZsChunk;  // full chunks
        int c0 = 0;
        for (; c0 + NS <= NCF; c0 += NS)
            unroll<NS>([&](auto jj) __attribute__((always_inline)) {
                chunk(jj, std::true_type{}, c0 + decltype(jj)::value);
            });
        unroll<NS>([&](auto jj) __attribute__((always_inline)) {
            if (c0 + decltype(jj)::value < NC) chunk(jj, std::false_type{}, c0 + decltype(jj)::value);
        });
        lds_barrier<0>();  // the ring is dead: zred reuses it
#pragma unroll
        for (int g = 0; g < 2; ++g) {
            f32x4* dst = reinterpret_cast<f32x4*>(sh.zred + (((ks * 2 + g) * RT + pt) * 256 + lane) * 4);
#pragma unroll
            for (int q = 0; q < 4; ++q)
                dst[64 * q] = f32x4{za[g][4 * q], za[g][4 * q + 1], za[g][4 * q + 2], za[g][4 * q + 3]};
        }
    }
    __syncthreads();
    {
        // The k-split partials of token group w & 1 added in order, by all 8 waves: wave w takes
        // accumulator elements 4 (w >> 1) .. 4 (w >> 1) + 3 of each tile; each wave's share of
        // the squared norms of z_hi and z_lo goes to csp.
        constexpr int KS = 8 / RT;
        const int zg = w & 1, part = w >> 1;
        const int jt = 32 * zg + n;
        const int c2 = part >> 1, q0 = 4 * (part & 1);
        float hi2 = 0.0f, lo2 = 0.0f;
#pragma unroll
        for (int pt = 0; pt < RT; ++pt) {
            const int c = 2 * pt + c2;
            f32x4 zsum;
#pragma unroll
            for (int ks = 0; ks < KS; ++ks) {
                const f32x4 v = *reinterpret_cast<const f32x4*>(
                    sh.zred + ((((ks * 2 + zg) * RT + pt) * 4 + part) * 64 + lane) * 4);
#pragma unroll
                for (int i = 0; i < 4; ++i) zsum[i] = ks == 0 ? v[i] : zsum[i] + v[i];
            }
            if (16 * c < R) {
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const float hf = (float)(__bf16)zsum[i];
                    const float lf = zsum[i] - hf;
                    hi2 = fmaf(hf, hf, hi2);
                    lo2 = fmaf(lf, lf, lo2);
                }
                *reinterpret_cast<f32x4*>(&sh.zs[jt * ZSP + 16 * c + 8 * half + q0]) = zsum;
            }
        }
        hi2 = sum_pair32(hi2);
        lo2 = sum_pair32(lo2);
        if (half == 0) {
            sh.csp[part][0][jt] = lo2;
            sh.csp[part][1][jt] = hi2;
        }
    }
    __syncthreads();
    // z, z_hi and c to memory (tokens < T): 16 bytes of z per thread and step
    for (int i = tid; i < kZsTokens * (R / 4); i += kRouteThreads) {
        const int jt = i / (R / 4), q = i % (R / 4);
        const int64_t t = tok0 + jt;
        if (t < T) {
            const f32x4 v = *reinterpret_cast<const f32x4*>(&sh.zs[jt * ZSP + 4 * q]);
            *reinterpret_cast<f32x4*>(zout + t * R + 4 * q) = v;
            uint32_t b01 = f32_to_bf16_bits(v[0]) | (f32_to_bf16_bits(v[1]) << 16);
            uint32_t b23 = f32_to_bf16_bits(v[2]) | (f32_to_bf16_bits(v[3]) << 16);
            *reinterpret_cast<uint2*>(zhi_out + t * R + 4 * q) = uint2{b01, b23};
        }
    }

    // ---- prescreen
    TokenGroups<RC, 2> tg;
    tg.first = tok0;
    tg.T = T;
#pragma unroll
    for (int g = 0; g < 2; ++g) {
        const int jt = 32 * g + n;
        const bool ok = tg.tok_ok(g, n);
#pragma unroll
        for (int c = 0; c < RC; ++c) {
            bf16x8 v;
#pragma unroll
            for (int q = 0; q < 8; ++q) v[q] = (__bf16)sh.zs[jt * ZSP + 16 * c + 8 * half + q];
            tg.zhi[g][c] = ok ? v : zero_bf16x8();
        }
        const float lo2 = ((sh.csp[0][0][jt] + sh.csp[1][0][jt]) + sh.csp[2][0][jt]) + sh.csp[3][0][jt];
        const float hi2 = ((sh.csp[0][1][jt] + sh.csp[1][1][jt]) + sh.csp[2][1][jt]) + sh.csp[3][1][jt];
        tg.c[g] = ok ? screen_scale(lo2, hi2, r) : 0.0f;
        if (ok && half == 0 && w == 0) cz[tok0 + jt] = tg.c[g];
    }
    const int tb = sub_tiles * w / kRouteWaves, nt = sub_tiles * (w + 1) / kRouteWaves - tb;
    float bm[2][L];
#pragma unroll
    for (int g = 0; g < 2; ++g)
#pragma unroll
        for (int b = 0; b < L; ++b) bm[g][b] = -__builtin_huge_valf();
    float ssmax = 0.0f;  // largest squared norm of the lane's half rows
    // The wave's tiles pass through a private ring of DA tiles in the (now free) staging area,
    // filled by direct-to-LDS loads (whole 128-byte lines) DA - 1 tiles ahead; rows are stored
    // with the swizzle of LdsRows, so the A-operand reads hit distinct banks.
    using RCfg = RouteCfg<RC, K>;
    constexpr int DA = 4;
    constexpr int TILE = 32 * R;            // bf16 per tile
    constexpr int TLOADS = TILE / 8 / 64;   // 16-byte direct-to-LDS loads per lane and tile
    static_assert(kRouteWaves * DA * TILE * 2 <= (int)sizeof(sh.stage), "prescreen ring");
    uint16_t* ring = sh.stage[0] + w * DA * TILE;
    auto stage_tile = [&](int slot, int j) __attribute__((always_inline)) {
        const int jt = j < nt ? j : (nt > 0 ? nt - 1 : 0);  // past the end: a harmless reload
        const uint16_t* g0 = R2t + (int64_t)(tb + jt) * TILE;
#pragma unroll
        for (int i = 0; i < TLOADS; ++i) {
            const int q = 64 * i + lane;  // slot in the tile: row q / SPR, position q % SPR
            const int row = q / RCfg::SPR, pos = q % RCfg::SPR;
            lds_dma16(g0 + row * R + 8 * (pos ^ RCfg::swz(row)), ring + slot * TILE + 512 * i);
        }
    };
    const LdsRows<RC, K> lsrc(ring, nullptr, n, half);
    constexpr int V = U > DA ? U : DA;
    bf16x8 a[RC];
    // [tile parity][group]; the set of the "previous" tile before the first one holds -inf
    f32x16 acc[2][2];
#pragma unroll
    for (int g = 0; g < 2; ++g)
#pragma unroll
        for (int i = 0; i < 16; ++i) acc[1][g][i] = -__builtin_huge_valf();
    // epilogue of the tile in accumulator set P (bucket UB / 4 = its index in the wave mod U);
    // the subset lies below M (the plan keeps 32 sub_tiles <= M), so no row is masked
    auto finish = [&](auto pp, auto uu) __attribute__((always_inline)) {
        constexpr int P = decltype(pp)::value, UB = 4 * decltype(uu)::value;
#pragma unroll
        for (int g = 0; g < 2; ++g)
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const float t = fmaxf(fmaxf(bm[g][UB + q], acc[P][g][4 * q]), acc[P][g][4 * q + 1]);
                bm[g][UB + q] = fmaxf(fmaxf(t, acc[P][g][4 * q + 2]), acc[P][g][4 * q + 3]);
            }
    };
    // tile j of the wave (ring slot J mod DA, parity J & 1): wait for its staged rows, read the
    // A operands, refill the slot with tile j + DA, MFMAs, norm of the rows, then the epilogue
    // of tile j - 1
    auto step = [&](auto jj, int j) __attribute__((always_inline)) {
        constexpr int J = decltype(jj)::value;
        constexpr int SA = J % DA, P = J & 1;
        __builtin_amdgcn_s_waitcnt(vmcnt_imm((DA - 1) * TLOADS));  // tile j has arrived
        lsrc.load_a(SA, a);
        __builtin_amdgcn_s_waitcnt(vmcnt_imm(63) & ~(15 << 8));   // lgkmcnt(0): slot read
        stage_tile(SA, j + DA);
#pragma unroll
        for (int g = 0; g < 2; ++g) {
            acc[P][g] = mfma_32x32x16(a[0], tg.zhi[g][0], zero_f32x16());
#pragma unroll
            for (int c = 1; c < RC; ++c) acc[P][g] = mfma_32x32x16(a[c], tg.zhi[g][c], acc[P][g]);
        }
        float ss = 0.0f;
#pragma unroll
        for (int c = 0; c < RC; ++c)
#pragma unroll
            for (int q = 0; q < 8; q += 2) {
                const bf16x2 pq = {a[c][q], a[c][q + 1]};
                ss = __builtin_amdgcn_fdot2_f32_bf16(pq, pq, ss, false);
            }
        ssmax = fmaxf(ssmax, ss);
        finish(std::integral_constant<int, P ^ 1>{}, std::integral_constant<int, (J + V - 1) % U>{});
    };
#pragma unroll
    for (int d = 0; d < DA; ++d) stage_tile(d, d);
    int j0 = 0;
    for (; j0 + V <= nt; j0 += V)  // unguarded steady state
        unroll<V>([&](auto jj) __attribute__((always_inline)) { step(jj, j0 + decltype(jj)::value); });
    unroll<V>([&](auto jj) __attribute__((always_inline)) {
        if (j0 + decltype(jj)::value < nt) step(jj, j0 + decltype(jj)::value);
    });
    // the last tile's epilogue (its parity and bucket dispatched to compile-time values)
    unroll<V>([&](auto jj) __attribute__((always_inline)) {
        constexpr int J = decltype(jj)::value;
        if (nt > 0 && (nt - 1) % V == J)
            finish(std::integral_constant<int, J & 1>{}, std::integral_constant<int, J % U>{});
    });
    __builtin_amdgcn_s_waitcnt(vmcnt_imm(0));  // the ring's last (unused) loads
    // wave norm bound: row n of the wave's tiles has squared norm a + b (this lane's half and
    // lane n + 32's), at most max a + max b over the tiles
    float mx = sum_pair32(ssmax);
    mx = fmaxf(mx, lane_xor<1>(mx));
    mx = fmaxf(mx, lane_xor<2>(mx));
    mx = fmaxf(mx, lane_xor<4>(mx));
    mx = fmaxf(mx, lane_xor<8>(mx));
    mx = fmaxf(mx, lane_xor<16>(mx));
    const float nw = __builtin_bit_cast(
        float, __builtin_amdgcn_readfirstlane(__builtin_bit_cast(int, sqrtf(mx) * (1.0f + 0x1p-20f))));
    __syncthreads();  // every wave's ring is dead: tops reuses the staging area
#pragma unroll
    for (int g = 0; g < 2; ++g) {
#pragma unroll
        for (int b = 0; b < L; ++b) bm[g][b] = fmaf(-tg.c[g], nw, bm[g][b]);
        sort_desc<L>(bm[g]);
        float pb[L];
#pragma unroll
        for (int b = 0; b < L; ++b) lane_pair32(bm[g][b], bm[g][b], pb[b]);
        vlist_merge<L>(bm[g], pb);
        if (half == 0) {
#pragma unroll
            for (int j = 0; j < K; ++j) sh.tops[32 * g + n][w * K + j] = bm[g][j];
        }
    }
    __syncthreads();
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
        const int64_t t = tok0 + jt;
        if (sub == 0 && t < T) {
            float th = v[0];
#pragma unroll
            for (int j = 1; j < K; ++j)
                if (j == k - 1) th = v[j];
            theta0[t] = fmaxf(th - fabsf(th) * 0x1p-20f, -0x1p100f);
            count[t] = 0;
        }
    }
    if (hist) {  // cleared for the finalize kernel's counts (no memset: graph-safe)
        for (int64_t e = (int64_t)blockIdx.x * kRouteThreads + tid; e < M;
             e += (int64_t)gridDim.x * kRouteThreads)
            hist[e] = 0;
    }
}

// ------------------------------------------------------------------------------ collect
// Grid: chunks x splits workgroups (route_split).  A workgroup loads its chunk of expert rows
// (<= 128 KiB) into LDS with the chunk norm N_c (the largest row norm, rounded up), then sweeps
// it for blocks of 512 tokens (wave w: token groups of 32 at 64 w and 64 w + 32).
//
// Test.  Every accumulator starts at b = c N_c - theta0 + delta (the MFMA's C operand), with
// delta = (r + 2) 2^-23 (|theta0| + c N_c) covering the rounding of b and the accumulation
// error |b| adds; the MFMA returns acc_e = s_e + b, and l_e <= acc_e + theta0 holds exactly
// (real arithmetic on the fp32 values).  An expert with l_e >= theta0 therefore has acc_e >= +0,
// and acc_e + theta0 is an upper bound of its logit.  The sixteen sign bits of a lane's
// accumulator become a mask; a lane with a hit stores one entry (tile, lane half, mask) with the
// largest acc of its sixteen, in its private slots of the workgroup's scratch.
//
// Records.  After a block, a lane reserves room for its hits in the token's record list with
// one atomic add (issued before the next block's sweep, consumed after it) and then writes one
// record (expert, upper bound) per hit: ub = (max acc + theta0) rounded up by 2^-22 relative.
// A lane with more than S entries in a block marks its token overflowed (count > cap), and so
// does a list that would exceed cap: finalize then sweeps all experts exactly for that token.
struct CollectEntry {
    uint32_t code;  // tile in chunk << 17 | lane half << 16 | 16-bit element mask
    float amax;     // the largest acc of the lane's sixteen
};

template <int RC, int K>
__global__ __launch_bounds__(kRouteThreads, 1) void collect_kernel1(
    const uint16_t* __restrict__ zh, const float* __restrict__ cz,
    const float* __restrict__ theta0, const uint16_t* __restrict__ R2t, int32_t T, int32_t M,
    int32_t chunks, int32_t splits, int32_t* __restrict__ count, int2* __restrict__ rec,
    int32_t cap, CollectEntry* __restrict__ scratch, int32_t S) {
    using C = RouteCfg<RC, K>;
    constexpr int TPW = kCollectTPW, R = C::R;
    __shared__ __attribute__((aligned(16))) uint16_t rows[C::EMAX * C::R];
    __shared__ float nred[kRouteWaves];
    const RouteSplit sp = route_split(T, M, chunks, splits, kCollectTokens);
    load_chunk<RC, K>(R2t, nullptr, M, sp.t0, sp.t1, rows, nullptr, false);
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int n = lane & 31, half = lane >> 5;
    const int nt = (int)(sp.t1 - sp.t0);
    const int32_t ebase = (int32_t)(sp.t0 * 32);
    // chunk norm bound from the resident rows (rows past M are copies of row M - 1)
    float nc;
    {
        float mx = 0.0f;
        for (int e = tid; e < nt * 32; e += kRouteThreads) {
            const int sw = C::swz(e);
            float ss = 0.0f;
#pragma unroll
            for (int sg = 0; sg < C::SPR; ++sg) {
                const bf16x8 v = load_bf16x8(rows + e * R + ((sg ^ sw) * 8));
#pragma unroll
                for (int q = 0; q < 8; q += 2) {
                    const bf16x2 pq = {v[q], v[q + 1]};
                    ss = __builtin_amdgcn_fdot2_f32_bf16(pq, pq, ss, false);
                }
            }
            mx = fmaxf(mx, ss);
        }
        mx = fmaxf(mx, lane_xor<1>(mx));
        mx = fmaxf(mx, lane_xor<2>(mx));
        mx = fmaxf(mx, lane_xor<4>(mx));
        mx = fmaxf(mx, lane_xor<8>(mx));
        mx = fmaxf(mx, lane_xor<16>(mx));
        mx = fmaxf(mx, __shfl_xor(mx, 32, kWave));
        if (lane == 0) nred[w] = mx;
        __syncthreads();
        mx = nred[0];
#pragma unroll
        for (int i = 1; i < kRouteWaves; ++i) mx = fmaxf(mx, nred[i]);
        // the squared sums use bf16 dot products, whose rounding (2^-18 relative at most) the
        // 2^-20 here and the 2^-10 of the screening scale cover
        nc = sqrtf(mx) * (1.0f + 0x1p-20f);
    }
    const LdsRows<RC, K> src(rows, nullptr, n, half);
    const LastTileMask ltm(M);
    const uint32_t lmask = half ? ltm.m[1] : ltm.m[0];  // experts < M of the last tile
    const uint32_t hcode = (uint32_t)half << 16;
    const int32_t tile0 = (int32_t)sp.t0;
    // the lane's private entry slots: [buffer][group][slot][lane] of this workgroup
    CollectEntry* my = scratch + (int64_t)blockIdx.x * 2 * TPW * (S + 1) * kRouteThreads + tid;
    auto slot = [&](int buf, int g, int i) __attribute__((always_inline)) {
        return my + ((buf * TPW + g) * (S + 1) + i) * kRouteThreads;
    };
    // block state kept for the deferred record writes
    int pcnt[TPW], pbase[TPW];
    int64_t ptok[TPW];
    float pth[TPW];
    bool pending = false;
    // The lane's entries of one group are loaded together (one memory latency), then expanded.
    constexpr int SB = 16;  // entries loaded per batch
    auto write_records = [&](int buf) __attribute__((always_inline)) {
#pragma unroll
        for (int g = 0; g < TPW; ++g) {
            const int cnt = pcnt[g];
            if (cnt <= 0 || cnt > S || ptok[g] >= T) continue;
            int o = pbase[g];
            int2* out = rec + ptok[g] * cap;
            for (int i0 = 0; i0 < cnt; i0 += SB) {
                CollectEntry ent[SB];
#pragma unroll
                for (int i = 0; i < SB; ++i)
                    ent[i] = i0 + i < cnt ? *slot(buf, g, i0 + i) : CollectEntry{0u, 0.0f};
#pragma unroll
                for (int i = 0; i < SB; ++i) {
                    uint32_t m = ent[i].code & 0xFFFFu;  // 0 past cnt
                    const int32_t tl = (int32_t)(ent[i].code >> 17);
                    const int hf = (int)((ent[i].code >> 16) & 1u);
                    if (tile0 + tl == ltm.last) m &= ltm.m[hf];
                    float ub = ent[i].amax + pth[g];
                    ub = fmaf(fabsf(ub), 0x1p-22f, ub);
                    const int32_t e = ebase + 32 * tl + 4 * hf;
                    while (m) {
                        const int bt = __builtin_ctz(m);
                        m &= m - 1;
                        if (o < cap) out[o] = int2{e + 8 * (bt >> 2) + (bt & 3), __builtin_bit_cast(int, ub)};
                        ++o;
                    }
                }
            }
        }
    };

    int buf = 0;
    TokenGroups<RC, TPW> tg;
    const int64_t wofs = (int64_t)w * 32 * TPW;
    for (int64_t blk = sp.blk0; blk < sp.blk1; ++blk) {
        const int64_t first = blk * kCollectTokens + wofs;
        if (first >= T) break;  // wave-uniform
        tg.load(zh, cz, T, first, n, half);
        f32x16 cb[TPW];
        float th[TPW];
#pragma unroll
        for (int g = 0; g < TPW; ++g) {
            const bool ok = tg.tok_ok(g, n);
            th[g] = ok ? theta0[tg.tok(g, n)] : 0.0f;
            const float cn = tg.c[g] * nc;
            float b = fmaf(tg.c[g], nc, -th[g]) + (float)(R + 2) * 0x1p-23f * (fabsf(th[g]) + cn);
            b = ok ? b : -__builtin_huge_valf();  // tokens past T never pass
#pragma unroll
            for (int i = 0; i < 16; ++i) cb[g][i] = b;
        }
        int cnt[TPW], nh[TPW];
        CollectEntry* sbase[TPW];  // the lane's slot 0 of each group in this block's buffer
#pragma unroll
        for (int g = 0; g < TPW; ++g) {
            cnt[g] = nh[g] = 0;
            sbase[g] = slot(buf, g, 0);
        }
        sweep_cin<RC, K, TPW, 1>(
            src, nt, half, tg.zhi, cb,
            [&](auto gg, const f32x16& acc, int tl) __attribute__((always_inline)) {
                constexpr int g = decltype(gg)::value;
                const float a15 = acc[15];
                uint32_t m = __builtin_bit_cast(uint32_t, a15) >> 31;
#pragma unroll
                for (int i = 14; i >= 0; --i) {
                    const float ai = acc[i];
                    m = __builtin_amdgcn_alignbit(m, __builtin_bit_cast(uint32_t, ai), 31);
                }
                if (m != 0xFFFFu) {  // some element has acc >= +0 (its sign bit clear)
                    m ^= 0xFFFFu;
                    float amax = acc[0];
#pragma unroll
                    for (int i = 1; i < 16; ++i) amax = fmaxf(amax, acc[i]);
                    const bool last = tile0 + tl == ltm.last;  // wave-uniform
                    sbase[g][(cnt[g] < S ? cnt[g] : S) * kRouteThreads] =
                        CollectEntry{((uint32_t)tl << 17) | hcode | m, amax};
                    ++cnt[g];
                    nh[g] += __builtin_popcount(last ? (m & lmask) : m);
                }
            });
        // reserve this block's records (the return values are consumed after the next sweep)
        int base[TPW];
#pragma unroll
        for (int g = 0; g < TPW; ++g) {
            base[g] = 0;
            const int64_t t = tg.tok(g, n);
            if (t < T && (nh[g] > 0 || cnt[g] > S))
                base[g] = atomicAdd(&count[t], cnt[g] > S ? cap + 1 : nh[g]);
        }
        if (pending) write_records(buf ^ 1);
#pragma unroll
        for (int g = 0; g < TPW; ++g) {
            pcnt[g] = cnt[g];
            pbase[g] = base[g];
            ptok[g] = tg.tok(g, n);
            pth[g] = th[g];
        }
        pending = true;
        buf ^= 1;
    }
    if (pending) write_records(buf ^ 1);
}

// ------------------------------------------------------------------------------ finalize
// Sixteen lanes per token and sixteen tokens per workgroup of 256 threads (eight lanes and
// twice the records per lane measured slower, despite twice the tokens in flight per CU).  Lane
// sub of token j keeps records sub, sub + 16, ... of the token's list in registers (one round
// of 256; longer lists are walked in rounds, reloaded for each pass).  Per token:
//  1. kub: each lane offers the two largest upper bounds of its records; kub = the
//     min(2k, n)-th largest of those (at most 32) values, so at least that many (>= k) records
//     reach it;
//  2. pass 0: the records with ub >= kub are evaluated exactly (z from LDS, the rows of two
//     candidates per lane loaded together) into the token's candidate table in LDS; each
//     candidate's rank under the selection order is counted against the others, and theta1 = the
//     logit of rank k - 1: k distinct experts reach it, so the k-th logit does too;
//  3. pass 1: the records with theta1 <= ub < kub, the only others that can still reach the top k
//     (l <= ub), are evaluated and appended the same way;
//  4. ranks over the whole table give the top k: idx, topval, and gate (softmax in rank order).
// A token whose record list overflowed (count > cap) or whose candidates overflow the table is
// swept over all M experts by the whole workgroup.
constexpr int kFinLanes = 16;                        // lanes per token
constexpr int kFinThreads = 256;
constexpr int kFinTokens = kFinThreads / kFinLanes;  // tokens per workgroup
constexpr int kFinRegs = 16;                         // records per lane and round
constexpr int kFinRound = kFinLanes * kFinRegs;      // records per round
constexpr int kFinCand = 256;                        // candidate table entries per token

template <int RC, int K>
__global__ __launch_bounds__(kFinThreads) void finalize_kernel2(
    const float* __restrict__ z, const uint16_t* __restrict__ R2t, int32_t T, int32_t M,
    int32_t k, const int32_t* __restrict__ count, const int2* __restrict__ rec, int32_t cap,
    int32_t* __restrict__ idx, float* __restrict__ gate, float* __restrict__ topval) {
    constexpr int R = 16 * RC, NW = kFinThreads / 64;
    __shared__ __attribute__((aligned(16))) float zs[kFinTokens * R];
    __shared__ __attribute__((aligned(16))) float cv[kFinTokens * kFinCand];    // candidate logits
    __shared__ __attribute__((aligned(16))) int32_t ce[kFinTokens * kFinCand];  // candidate experts
    __shared__ float u2[kFinTokens * 2 * kFinLanes];
    __shared__ float thr[kFinTokens];
    __shared__ float ex[kFinTokens][K];
    __shared__ int32_t over_tok[kFinTokens];
    __shared__ float wv[NW][K];
    __shared__ int32_t wi[NW][K];
    const int tid = threadIdx.x;
    const int sub = tid & (kFinLanes - 1), j = tid / kFinLanes;
    const int64_t tok0 = (int64_t)blockIdx.x * kFinTokens;
    const int64_t tok = tok0 + j;
    const bool ok = tok < T;
    const int32_t n = ok ? count[tok] : 0;
    bool live = ok && n <= cap && n >= k;
    for (int i = 4 * sub; i < R; i += 4 * kFinLanes)
        *reinterpret_cast<f32x4*>(zs + j * R + i) =
            live ? *reinterpret_cast<const f32x4*>(z + tok * R + i) : f32x4{0.0f, 0.0f, 0.0f, 0.0f};
    const float* zj = zs + j * R;
    float* cvj = cv + j * kFinCand;
    int32_t* cej = ce + j * kFinCand;
    const int2* rj = rec + (ok ? tok : 0) * (int64_t)cap;
    const int nrounds = live ? (n + kFinRound - 1) / kFinRound : 0;
    int2 q[kFinRegs];
    auto load_round = [&](int rd) __attribute__((always_inline)) {
#pragma unroll
        for (int b = 0; b < kFinRegs; ++b) {
            const int i = rd * kFinRound + sub + kFinLanes * b;
            q[b] = i < n ? rj[i] : int2{kNoExpert, __builtin_bit_cast(int, -__builtin_huge_valf())};
        }
    };
    if (nrounds == 1) load_round(0);
    // f(expert, ub) for every record of the lane
    auto scan = [&](auto&& f) __attribute__((always_inline)) {
        for (int rd = 0; rd < nrounds; ++rd) {
            if (nrounds > 1) load_round(rd);
#pragma unroll
            for (int b = 0; b < kFinRegs; ++b)
                if (rd * kFinRound + sub + kFinLanes * b < n) f(q[b].x, __builtin_bit_cast(float, q[b].y));
        }
    };
    // 1. kub = the nk-th largest of the lanes' two largest bounds (x is it when fewer than nk
    //    offered values exceed x and at least nk reach it)
    {
        float m1 = -__builtin_huge_valf(), m2 = -__builtin_huge_valf();
        scan([&](int32_t, float u) __attribute__((always_inline)) {
            m2 = fmaxf(m2, fminf(m1, u));
            m1 = fmaxf(m1, u);
        });
        u2[j * 2 * kFinLanes + sub] = m1;
        u2[j * 2 * kFinLanes + kFinLanes + sub] = m2;
    }
    __syncthreads();
    int nk = 2 * k < n ? 2 * k : n;
    nk = nk < 2 * kFinLanes ? nk : 2 * kFinLanes;  // >= k: k <= 16 <= 2 kFinLanes
    if (live) {
        const float a = u2[j * 2 * kFinLanes + sub], b = u2[j * 2 * kFinLanes + kFinLanes + sub];
        int ga = 0, gb = 0, ea = 0, eb = 0;
        for (int i = 0; i < 2 * kFinLanes; ++i) {
            const float o = u2[j * 2 * kFinLanes + i];
            ga += o > a;
            ea += o >= a;
            gb += o > b;
            eb += o >= b;
        }
        if (ga < nk && ea >= nk) thr[j] = a;  // equal values from several lanes: same value
        if (gb < nk && eb >= nk) thr[j] = b;
    }
    __syncthreads();
    const float kub = thr[j];
    // exact logits of candidates cl = experts e0, e1 into table slots i0, i1 (i1 < 0: none)
    auto eval2 = [&](int32_t e0, int i0, int32_t e1, int i1) __attribute__((always_inline)) {
        // table entries are written before they are read; the clamp keeps any row address in
        // bounds regardless
        e0 = (uint32_t)e0 < (uint32_t)M ? e0 : 0;
        e1 = (uint32_t)e1 < (uint32_t)M ? e1 : 0;
        bf16x8 w0[2 * RC], w1[2 * RC];
#pragma unroll
        for (int c = 0; c < 2 * RC; ++c) {
            w0[c] = load_bf16x8(R2t + (int64_t)e0 * R + 8 * c);
            w1[c] = load_bf16x8(R2t + (int64_t)(i1 >= 0 ? e1 : e0) * R + 8 * c);
        }
        float l0 = 0.0f, l1 = 0.0f;  // rank entries in increasing order
#pragma unroll
        for (int c = 0; c < 2 * RC; ++c) {
            // z is read from LDS one segment at a time (the empty asm keeps the compiler from
            // hoisting all of it into registers next to the two rows)
            asm volatile("" ::: "memory");
            const f32x4 za = *reinterpret_cast<const f32x4*>(zj + 8 * c);
            const f32x4 zb = *reinterpret_cast<const f32x4*>(zj + 8 * c + 4);
#pragma unroll
            for (int t = 0; t < 4; ++t) {
                l0 = fmaf(za[t], (float)w0[c][t], l0);
                l1 = fmaf(za[t], (float)w1[c][t], l1);
            }
#pragma unroll
            for (int t = 0; t < 4; ++t) {
                l0 = fmaf(zb[t], (float)w0[c][4 + t], l0);
                l1 = fmaf(zb[t], (float)w1[c][4 + t], l1);
            }
        }
        // both chains are computed unconditionally, so that the second row's loads are issued
        // with the first (not sunk into the store's branch)
        asm volatile("" ::"v"(l0), "v"(l1));
        cvj[i0] = l0;
        if (i1 >= 0) cvj[i1] = l1;
    };
    // ranks of table entries ia and ib (ib < 0: none) among entries [0, cnt) under the selection
    // order; the table is read four entries at a time (entries cnt .. cnt4 - 1 are sentinels)
    auto rank2 = [&](int ia, int ib, int cnt4, int& ra, int& rb) __attribute__((always_inline)) {
        const float la = cvj[ia], lb = cvj[ib >= 0 ? ib : ia];
        const int32_t ea = cej[ia], eb = cej[ib >= 0 ? ib : ia];
        ra = 0;
        rb = 0;
#pragma nounroll
        for (int t = 0; t < cnt4; t += 4) {
            const f32x4 tv = *reinterpret_cast<const f32x4*>(cvj + t);
            const i32x4 te = *reinterpret_cast<const i32x4*>(cej + t);
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                ra += better(tv[u], te[u], la, ea) ? 1 : 0;
                rb += better(tv[u], te[u], lb, eb) ? 1 : 0;
            }
        }
    };
    // 2. pass 0 (lo = kub, hi = inf) and 3. pass 1 (lo = theta1, hi = kub): the selected records
    //    are appended to the table (positions from a prefix sum over the token's lanes, within
    //    one 16-lane DPP row), evaluated, and ranked
    float lo = kub, hi = __builtin_huge_valf();
    int cnt = 0;
#pragma nounroll
    for (int pass = 0; pass < 2; ++pass) {
        int base = cnt;
        for (int rd = 0; rd < nrounds; ++rd) {
            if (nrounds > 1) load_round(rd);
            uint32_t m = 0;
#pragma unroll
            for (int b = 0; b < kFinRegs; ++b) {
                const float u = __builtin_bit_cast(float, q[b].y);
                if (rd * kFinRound + sub + kFinLanes * b < n && u >= lo && u < hi) m |= 1u << b;
            }
            const int c = __builtin_popcount(m);
            int incl = c;  // inclusive prefix over the row
            // row_shr:d reads lane - d of the 16-lane DPP row.  Each move runs with all of the
            // token's lanes active (a lane whose source lane is inactive would read 0), and its
            // value is then dropped where the source lies in another token or outside the row.
            const int s1 = __builtin_amdgcn_update_dpp(0, incl, 0x111, 0xF, 0xF, false);
            incl += sub >= 1 ? s1 : 0;
            const int s2 = __builtin_amdgcn_update_dpp(0, incl, 0x112, 0xF, 0xF, false);
            incl += sub >= 2 ? s2 : 0;
            const int s4 = __builtin_amdgcn_update_dpp(0, incl, 0x114, 0xF, 0xF, false);
            incl += sub >= 4 ? s4 : 0;
            if constexpr (kFinLanes > 8) {
                const int s8 = __builtin_amdgcn_update_dpp(0, incl, 0x118, 0xF, 0xF, false);
                incl += sub >= 8 ? s8 : 0;
            }
            int o = base + incl - c;
#pragma unroll
            for (int b = 0; b < kFinRegs; ++b) {
                if (m & (1u << b)) {
                    if (o < kFinCand) cej[o] = q[b].x;
                    ++o;
                }
            }
            base += __shfl(incl, (threadIdx.x & ~(kFinLanes - 1)) + kFinLanes - 1, kWave);
        }
        if (base > kFinCand) live = false;  // token-uniform: swept exactly below
        const int hiend = live ? base : cnt;
        __syncthreads();
#pragma nounroll
        for (int i = cnt + sub; i < hiend; i += 2 * kFinLanes) {
            const int i1 = i + kFinLanes < hiend ? i + kFinLanes : -1;
            eval2(cej[i], i, i1 >= 0 ? cej[i1] : 0, i1);
        }
        cnt = hiend;
        const int cnt4 = (cnt + 3) & ~3;
        if (cnt + sub < cnt4) {
            cvj[cnt + sub] = -__builtin_huge_valf();
            cej[cnt + sub] = kNoExpert;
        }
        __syncthreads();
        if (pass == 0) {
            // theta1: the logit of rank k - 1 (exactly one entry has it: the order is total)
            for (int i = sub; i < cnt; i += 2 * kFinLanes) {
                const int ib = i + kFinLanes < cnt ? i + kFinLanes : -1;
                int ra, rb;
                rank2(i, ib, cnt4, ra, rb);
                if (ra == k - 1) thr[j] = cvj[i];
                if (ib >= 0 && rb == k - 1) thr[j] = cvj[ib];
            }
            __syncthreads();
            hi = lo;
            lo = thr[j];
        }
    }
    // 4. the top k by rank (only entries reaching theta1 can have rank < k); gate = softmax in
    //    rank order
    {
        const int cnt4 = (cnt + 3) & ~3;
        for (int i = sub; live && i < cnt; i += 2 * kFinLanes) {
            const int ib = i + kFinLanes < cnt ? i + kFinLanes : -1;
            const bool ua = cvj[i] >= lo, ub = ib >= 0 && cvj[ib] >= lo;
            if (!ua && !ub) continue;
            int ra, rb;
            rank2(i, ib, cnt4, ra, rb);
            if (ua && ra < k) {
                idx[tok * k + ra] = cej[i];
                if (topval) topval[tok * k + ra] = cvj[i];
                ex[j][ra] = cvj[i];
            }
            if (ub && rb < k) {
                idx[tok * k + rb] = cej[ib];
                if (topval) topval[tok * k + rb] = cvj[ib];
                ex[j][rb] = cvj[ib];
            }
        }
    }
    __syncthreads();
    if (live) {
        const float lmax = ex[j][0];
        float e[K];
        float sum = 0.0f;
#pragma unroll
        for (int i = 0; i < K; ++i) {
            e[i] = i < k ? expf(ex[j][i] - lmax) : 0.0f;
            sum += e[i];
        }
#pragma unroll
        for (int i = 0; i < K; ++i)
            if (i < k && i % kFinLanes == sub) gate[tok * k + i] = e[i] / sum;
    }
    // Tokens left over (an overflowed record list or candidate table; rare): the whole workgroup
    // sweeps all experts, thread tid taking experts tid, tid + kFinThreads, ...
    const bool over = ok && !live;
    if (sub == 0) over_tok[j] = over;
    if (!__syncthreads_or(over)) return;  // workgroup-uniform
    for (int jt = 0; jt < kFinTokens; ++jt) {
        if (!over_tok[jt]) continue;  // workgroup-uniform
        const int64_t t = tok0 + jt;
        const float* zp = z + t * R;
        float v[K];
        int32_t ix[K];
        list_init<K>(v, ix);
        for (int32_t e = tid; e < M; e += kFinThreads) {
            const float l = exact_logit<RC>([&](int i) { return zp[i]; }, R2t + (int64_t)e * R);
            if (better(l, e, v[K - 1], ix[K - 1])) list_insert<K>(v, ix, l, e);
        }
        list_merge_xor<1, K>(v, ix);
        list_merge_xor<2, K>(v, ix);
        list_merge_xor<4, K>(v, ix);
        list_merge_xor<8, K>(v, ix);
        list_merge_xor<16, K>(v, ix);
        list_merge_xor<32, K>(v, ix);
        if ((tid & 63) == 0) {
#pragma unroll
            for (int i = 0; i < K; ++i) {
                wv[tid >> 6][i] = v[i];
                wi[tid >> 6][i] = ix[i];
            }
        }
        __syncthreads();
        if (tid == 0) {
            for (int w = 1; w < NW; ++w) {
                float bv[K];
                int32_t bi[K];
#pragma unroll
                for (int i = 0; i < K; ++i) {
                    bv[i] = wv[w][i];
                    bi[i] = wi[w][i];
                }
                list_merge<K>(v, ix, bv, bi);
            }
            store_selection<K>(v, ix, k, t, idx, gate, topval);
        }
        __syncthreads();
    }
}

// ------------------------------------------------------------------------------ launch
template <int RC, int K>
static void launch_single_pass_k(const LowrankPlan& p, const SinglePassArgs& a, hipStream_t st) {
    const int64_t T = a.T;
    hipLaunchKernelGGL((zscreen_kernel<RC, K>), dim3((unsigned)((T + kZsTokens - 1) / kZsTokens)),
                       dim3(kRouteThreads), 0, st, a.x, a.R1t, a.R2t, (int32_t)T, a.h, a.r, a.M,
                       a.k, p.sub_tiles, a.z, a.zhi, a.cz, a.theta0, a.count, a.hist);
    hipLaunchKernelGGL((collect_kernel1<RC, K>), dim3((unsigned)((int64_t)p.splits * p.chunks)),
                       dim3(kRouteThreads), 0, st, a.zhi, a.cz, a.theta0, a.R2t, (int32_t)T, a.M,
                       p.chunks, p.splits, a.count, a.rec, p.cap,
                       reinterpret_cast<CollectEntry*>(a.scratch), p.slots);
    hipLaunchKernelGGL((finalize_kernel2<RC, K>),
                       dim3((unsigned)((T + kFinTokens - 1) / kFinTokens)), dim3(kFinThreads), 0, st, a.z, a.R2t, (int32_t)T, a.M, a.k, a.count,
                       a.rec, p.cap, a.idx, a.gate, a.topval);
}

template <int RC>
static bool launch_single_pass_rc(const LowrankPlan& p, const SinglePassArgs& a, hipStream_t st) {
    switch (p.K) {
        case 1: launch_single_pass_k<RC, 1>(p, a, st); return true;
        case 2: launch_single_pass_k<RC, 2>(p, a, st); return true;
        case 4: launch_single_pass_k<RC, 4>(p, a, st); return true;
        case 8: launch_single_pass_k<RC, 8>(p, a, st); return true;
        case 16: launch_single_pass_k<RC, 16>(p, a, st); return true;
    }
    return false;
}

hipError_t single_pass_launch(const LowrankPlan& p, const SinglePassArgs& a, hipStream_t st) {
    bool ok = false;
    switch (p.RC) {
        case 1: ok = launch_single_pass_rc<1>(p, a, st); break;
        case 2: ok = launch_single_pass_rc<2>(p, a, st); break;
        case 4: ok = launch_single_pass_rc<4>(p, a, st); break;
    }
    return ok ? hipGetLastError() : hipErrorInvalidValue;
}

size_t collect_scratch_bytes(int64_t grid, int32_t slots) {
    return (size_t)grid * 2 * kCollectTPW * (slots + 1) * kRouteThreads * sizeof(CollectEntry);
}

}  // namespace more
