// Device helpers of the low-rank router kernels (gfx950): compile-time unrolling, the
// screening error scale, expert-chunk staging in LDS, token-group operands, the MFMA sweeps over
// expert tiles (operands from LDS, L2 or registers), the collect tests, the exact logit of a
// candidate and the final selection of a workgroup's tokens, and LDS barrier helpers.
//
// MFMA layout.  Every contraction uses v_mfma_f32_32x32x16_bf16 with experts (or rank
// rows) on the 32 A rows and tokens on the 32 B columns.  A lane therefore owns one token
// and 16 logits of it per tile, so the per-token threshold test is lane local.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <utility>

#include "device_common.h"

namespace more {
// Calls f(std::integral_constant<int, i>) for i = 0 .. N-1 (compile-time positions).
template <typename F, int... I>
__device__ __forceinline__ void unroll_impl(F&& f, std::integer_sequence<int, I...>) {
    (f(std::integral_constant<int, I>{}), ...);
}
template <int N, typename F>
__device__ __forceinline__ void unroll(F&& f) {
    unroll_impl(f, std::make_integer_sequence<int, N>{});
}

// Error scale of the screened logits of one token (see the route section):
// c = (||z_lo|| + r 2^-23 ||z_hi||) (1 + 2^-10), from the squared norms.
// It is kept >= 2^-126 (a looser bound), so that c 2^100 always dominates a logit.
__device__ __forceinline__ float screen_scale(float lo2, float hi2, int r) {
    return fmaxf((sqrtf(lo2) + (float)r * 0x1p-23f * sqrtf(hi2)) * (1.0f + 0x1p-10f), 0x1p-126f);
}


constexpr float kPhantomNorm = 0x1p100f;  // norm bound of a 4-expert group reaching past M

// ------------------------------------------------------------------------------ route
// Screen and collect workgroups are expert-resident: a workgroup loads one chunk of the
// expert axis (up to 128 KiB of R2t rows, with their group norms) into LDS once, then its 8
// waves sweep that chunk for token blocks of 8 * 32 * TPW tokens (wave w takes the TPW groups
// of 32 tokens starting at 32 TPW w), with no barrier inside the token loop.  Each A operand
// read from LDS feeds TPW MFMAs, so a larger TPW means less LDS traffic per MFMA.
//
// Screening precision.  The sweeps compute s_e = z_hi . u_e on the matrix cores, with z_hi =
// bf16(z) and fp32 accumulation, instead of the logit l_e = z . u_e.  With z_lo = z - z_hi,
//   |l_e - s_e| <= ||z_lo|| ||u_e|| + r 2^-24 sum_i |z_hi,i u_e,i| <= c ||u_e||,
//   c = ||z_lo|| + r 2^-23 ||z_hi||  (Cauchy-Schwarz; accumulation bound taken twice over),
// and ||u_e|| <= N_g, the largest row norm of the 4-expert group g holding e.  So s_e - c N_g
// is a lower and s_e + c N_g an upper bound of l_e.
constexpr int kRouteWaves = 8;
constexpr int kRouteThreads = 64 * kRouteWaves;
constexpr int kChunkBytes = 128 * 1024;       // LDS for the resident expert rows

// Token groups of 32 per wave: 2.  (Four at r = 64 and K <= 8 halve the LDS reads per MFMA but
// need more than 256 registers: the screen and collect kernels spilled 32-100 bytes per lane, and
// the two-group version, spill-free, runs the mid workload in the same time.)
constexpr int kRouteTPW = 2;

template <int RC, int K>
struct RouteCfg {
    static constexpr int R = 16 * RC;
    static constexpr int SPR = R / 8;                     // 16-byte segments per expert row
    static constexpr int U = K / 4 > 1 ? K / 4 : 1;       // bucket period, in tiles
    static constexpr int L = 4 * U;                       // bucket maxima per lane (>= K)
    static constexpr int EMAX = kChunkBytes / (2 * R);    // experts per chunk (multiple of 32)
    static constexpr int TPW = kRouteTPW;                 // token groups per wave
    static constexpr int TOK = 32 * TPW * kRouteWaves;    // tokens per block
    // candidate slots per lane and token group (the collect kernel's LDS must stay <= 160 KiB)
    static constexpr int SLOTS = TPW == 4 ? 7 : 8;
    // The next token block's operands are prefetched into registers only at TPW = 2.
    static constexpr bool PREFETCH = TPW == 2;
    // Rows are stored unpadded; segment s of row e sits at position s ^ swz(e), which spreads
    // the 16-byte reads of 16 consecutive rows over all 64 banks.
    static constexpr int RPL = 16 / SPR;                  // rows per 256-byte bank line
    __device__ static constexpr int swz(int e) { return (e / RPL) % SPR; }
};

template <int N>
__device__ __forceinline__ void sort_desc(float (&v)[N]) {
#pragma unroll
    for (int size = 2; size <= N; size <<= 1) {
#pragma unroll
        for (int stride = size / 2; stride > 0; stride >>= 1) {
#pragma unroll
            for (int i = 0; i < N; ++i) {
                const int j = i ^ stride;
                if (j > i) {
                    const bool desc = (i & size) == 0;
                    const float a = v[i], b = v[j];
                    v[i] = desc ? fmaxf(a, b) : fminf(a, b);
                    v[j] = desc ? fminf(a, b) : fmaxf(a, b);
                }
            }
        }
    }
}

// a <- the K largest of a and b (both sorted descending); result sorted descending.
template <int K>
__device__ __forceinline__ void vlist_merge(float (&a)[K], const float (&b)[K]) {
#pragma unroll
    for (int j = 0; j < K; ++j) a[j] = fmaxf(a[j], b[K - 1 - j]);
#pragma unroll
    for (int s = K / 2; s >= 1; s >>= 1) {
#pragma unroll
        for (int j = 0; j < K; ++j) {
            if ((j & s) == 0) {
                const float x = a[j], y = a[j + s];
                a[j] = fmaxf(x, y);
                a[j + s] = fminf(x, y);
            }
        }
    }
}

__device__ __forceinline__ float max4(const f32x16& a, int q) {
    return fmaxf(fmaxf(a[4 * q], a[4 * q + 1]), fmaxf(a[4 * q + 2], a[4 * q + 3]));
}

// Work split of a route launch: workgroup -> (expert chunk, range of token blocks).
struct RouteSplit {
    int32_t chunk;
    int64_t t0, t1;        // tiles of the chunk
    int64_t blk0, blk1;    // token blocks
};

__device__ __forceinline__ RouteSplit route_split(int32_t T, int32_t M, int32_t chunks,
                                                  int32_t splits, int tokens_per_block) {
    RouteSplit q;
    q.chunk = (int32_t)(blockIdx.x % (unsigned)chunks);
    const int32_t split = (int32_t)(blockIdx.x / (unsigned)chunks);
    const int64_t Mt = ((int64_t)M + 31) / 32;
    q.t0 = Mt * q.chunk / chunks;
    q.t1 = Mt * (q.chunk + 1) / chunks;
    const int64_t ntb = ((int64_t)T + tokens_per_block - 1) / tokens_per_block;
    q.blk0 = ntb * split / splits;
    q.blk1 = ntb * (split + 1) / splits;
    return q;
}

// Loads the rows of tiles [t0, t1) (rows past M re-read row M - 1; see group_norms) and
// their group norms into LDS; every thread of the workgroup takes part.
template <int RC, int K>
__device__ __forceinline__ void load_chunk(const uint16_t* __restrict__ R2t,
                                           const float* __restrict__ gnorm, int32_t M,
                                           int64_t t0, int64_t t1, uint16_t* rows, float* gn,
                                           bool copy_gn = true) {
    using C = RouteCfg<RC, K>;
    const int tid = threadIdx.x;
    const int nseg = (int)(t1 - t0) * 32 * C::SPR;
    const int64_t e0 = t0 * 32;
    constexpr int UNR = 8;  // loads in flight per thread
    for (int base = 0; base < nseg; base += UNR * kRouteThreads) {
        u32x4 v[UNR];
#pragma unroll
        for (int i = 0; i < UNR; ++i) {
            int seg = base + i * kRouteThreads + tid;
            seg = seg < nseg ? seg : nseg - 1;
            const int e = seg / C::SPR, s = seg % C::SPR;
            int64_t ge = e0 + e;
            ge = ge < M ? ge : M - 1;
            v[i] = *reinterpret_cast<const u32x4*>(R2t + ge * C::R + s * 8);
        }
#pragma unroll
        for (int i = 0; i < UNR; ++i) {
            const int seg = base + i * kRouteThreads + tid;
            if (seg < nseg) {
                const int e = seg / C::SPR, s = seg % C::SPR;
                *reinterpret_cast<u32x4*>(rows + e * C::R + ((s ^ C::swz(e)) * 8)) = v[i];
            }
        }
    }
    if (copy_gn) {
        const int ngr = (int)(t1 - t0) * 8;
        for (int g = tid; g < ngr; g += kRouteThreads) gn[g] = gnorm[t0 * 8 + g];
    }
    __syncthreads();
}

// Group norms of a chunk resident in LDS (as group_norms computes them from memory), written to
// the LDS copy gn and, with out != nullptr, to the chunk's part of the global array for the
// collect kernel.  Every thread of the workgroup takes part; rows past M hold copies of row
// M - 1 and their groups get the bound 2^100.
template <int RC, int K>
__device__ __forceinline__ void chunk_group_norms(const uint16_t* rows, int32_t M, int64_t t0,
                                                  int64_t t1, float* gn,
                                                  float* __restrict__ out) {
    using C = RouteCfg<RC, K>;
    const int tid = threadIdx.x;
    const int nrows = (int)(t1 - t0) * 32;
    for (int rb = 0; rb < nrows; rb += kRouteThreads) {  // workgroup-uniform trip count
        const int rr = rb + tid < nrows ? rb + tid : nrows - 1;
        const int sw = C::swz(rr);
        float ss = 0.0f;
#pragma unroll
        for (int sg = 0; sg < C::SPR; ++sg) {
            const bf16x8 v = load_bf16x8(rows + rr * C::R + ((sg ^ sw) * 8));
#pragma unroll
            for (int q = 0; q < 8; q += 2) {
                const bf16x2 pq = {v[q], v[q + 1]};
                ss = __builtin_amdgcn_fdot2_f32_bf16(pq, pq, ss, false);
            }
        }
        ss = fmaxf(ss, lane_xor<1>(ss));  // the 4 rows of the group sit in 4 consecutive lanes
        ss = fmaxf(ss, lane_xor<2>(ss));
        const int64_t row = t0 * 32 + rr;
        if (rb + tid < nrows && (rr & 3) == 0) {
            const int g4 = (rr & 31) >> 2;
            const int slot = (rr >> 5) * 8 + (g4 & 1) * 4 + (g4 >> 1);
            const float nb = row + 3 < M ? sqrtf(ss) * (1.0f + 0x1p-20f) : kPhantomNorm;
            gn[slot] = nb;
            if (out) out[t0 * 8 + slot] = nb;
        }
    }
    __syncthreads();
}

// Token ids, z_hi operands and error scales of one lane, for each of the wave's TPW groups of
// 32 tokens starting at `first` (written by the z pass; zeros past T).
template <int RC, int TPW>
struct TokenGroups {
    int64_t first;  // wave-uniform
    int32_t T;
    bf16x8 zhi[TPW][RC];
    float c[TPW];

    __device__ __forceinline__ int64_t tok(int g, int n) const { return first + 32 * g + n; }
    __device__ __forceinline__ bool tok_ok(int g, int n) const { return tok(g, n) < T; }

    __device__ __forceinline__ void load(const uint16_t* __restrict__ zh,
                                         const float* __restrict__ cz, int32_t T_, int64_t first_,
                                         int n, int half) {
        constexpr int R = 16 * RC;
        first = first_;
        T = T_;
#pragma unroll
        for (int g = 0; g < TPW; ++g) {
            const bool ok = tok_ok(g, n);
            const int64_t t = ok ? tok(g, n) : 0;
#pragma unroll
            for (int cc = 0; cc < RC; ++cc) {
                const bf16x8 v = load_bf16x8(zh + t * R + 16 * cc + 8 * half);
                zhi[g][cc] = ok ? v : zero_bf16x8();
            }
            c[g] = ok ? cz[t] : 0.0f;
        }
    }
};

// Operand sources of a sweep: the A operands (expert rows 32 t + n, rank entries 16 c + 8 half
// + 0..7 for c < RC) and the norm bounds of lane half `half` for tile t of the sweep.
//
// LdsRows: a chunk resident in LDS (rows stored with the XOR swizzle of RouteCfg).
template <int RC, int K>
struct LdsRows {
    const uint16_t* rows;
    const float* gn;
    int off[RC];
    int half;
    __device__ __forceinline__ LdsRows(const uint16_t* rows_, const float* gn_, int n, int half_)
        : rows(rows_), gn(gn_), half(half_) {
        using C = RouteCfg<RC, K>;
        const int sw = C::swz(n);
#pragma unroll
        for (int c = 0; c < RC; ++c) off[c] = n * C::R + (((2 * c + half) ^ sw) * 8);
    }
    __device__ __forceinline__ void load_a(int tile, bf16x8 (&a)[RC]) const {
        const uint16_t* base = rows + tile * 32 * RouteCfg<RC, K>::R;
#pragma unroll
        for (int c = 0; c < RC; ++c) a[c] = load_bf16x8(base + off[c]);
    }
    __device__ __forceinline__ f32x4 load_nq(int tile) const {
        return *reinterpret_cast<const f32x4*>(gn + tile * 8 + 4 * half);
    }
};

// GlobalRows: rows read straight from R2t (L2-resident when the expert set is small), norms
// from a copy of the group norms in LDS; tiles are counted from global tile tile0, rows past M
// re-read row M - 1 (see group_norms).
template <int RC>
struct GlobalRows {
    const uint16_t* row;   // R2t + (32 tile0 + n) * R + 8 half
    const float* gn;       // LDS group norms + 8 tile0 + 4 half
    int32_t rmax;          // rows past this one (M - 1 - 32 tile0 - n) are clamped
    __device__ __forceinline__ GlobalRows(const uint16_t* R2t, const float* gn_lds, int32_t M,
                                          int64_t tile0, int n, int half)
        : row(R2t + (tile0 * 32 + n) * (16 * RC) + 8 * half),
          gn(gn_lds + tile0 * 8 + 4 * half),
          rmax((int32_t)(M - 1 - tile0 * 32 - n)) {}
    __device__ __forceinline__ void load_a(int tile, bf16x8 (&a)[RC]) const {
        int rr = tile * 32;
        rr = rr < rmax ? rr : rmax;
        const uint16_t* p = row + (int64_t)rr * (16 * RC);
#pragma unroll
        for (int c = 0; c < RC; ++c) a[c] = load_bf16x8(p + 16 * c);
    }
    __device__ __forceinline__ f32x4 load_nq(int tile) const {
        return *reinterpret_cast<const f32x4*>(gn + tile * 8);
    }
};

// Sweeps nt tiles (experts e00 .. e00 + 32 nt - 1) for one lane's token groups and calls
// body(g, acc, e0, u, nq) once per token group g and tile: acc holds s for the group's
// 32 tokens and the tile's 32 experts starting at e0, nq[q] is the norm bound of accumulator
// group q, u = tile mod U the bucket index (g and u are std::integral_constant).
//
// Schedule.  The token groups form two halves H0 = [0, TPW/2) and H1 = [TPW/2, TPW), with one
// accumulator per group.  Per tile t the wave issues the MFMAs of H0(t), finishes H1(t - 1),
// issues the MFMAs of H1(t) and finishes H0(t): every epilogue runs while the other half's
// MFMAs execute.  The A operands and norms of the next D tiles are held in a register ring (the
// refill of a slot is issued once its last reader has been issued).  The steady-state loop runs
// groups of V = max(U, D, 2) tiles, so that ring slots and bucket indices are compile-time
// constants there and each tile is one basic block.
template <int RC, int K, int TPW, int D, typename Src, typename Body>
__device__ __forceinline__ void sweep(const Src& src, int nt, int32_t e00, int32_t M, int half,
                                      const bf16x8 (&zhi)[TPW][RC], Body&& body) {
    using C = RouteCfg<RC, K>;
    constexpr int H = TPW / 2;
    constexpr int U = C::U;
    constexpr int ND = 2;  // norm slots (norms come from LDS; a slot lives for two steps)
    constexpr int V = U > D ? (U > ND ? U : ND) : (D > ND ? D : ND);
    if (nt <= 0) return;
    f32x16 acc[TPW];
    f32x4 nq[ND];
    bf16x8 a[D][RC];
    auto fetch = [&](auto slot, int tile) __attribute__((always_inline)) {
        src.load_a(tile < nt ? tile : nt - 1, a[decltype(slot)::value]);  // past the end: unused
    };
    auto fetch_nq = [&](auto slot, int tile) __attribute__((always_inline)) {
        nq[decltype(slot)::value] = src.load_nq(tile < nt ? tile : nt - 1);
    };
    auto mfmas = [&](auto slot, auto hh) __attribute__((always_inline)) {
        constexpr int A = decltype(slot)::value;
        constexpr int G0 = decltype(hh)::value * H;
#pragma unroll
        for (int g = G0; g < G0 + H; ++g) acc[g] = zero_f32x16();
#pragma unroll
        for (int c = 0; c < RC; ++c)
#pragma unroll
            for (int g = G0; g < G0 + H; ++g) acc[g] = mfma_32x32x16(a[A][c], zhi[g][c], acc[g]);
    };
    auto finish = [&](auto nslot, auto hh, int tile, auto u) __attribute__((always_inline)) {
        constexpr int NS = decltype(nslot)::value;
        constexpr int G0 = decltype(hh)::value * H;
        const int32_t e0 = e00 + tile * 32;
        unroll<H>([&](auto gg) __attribute__((always_inline)) {
            constexpr int G = G0 + decltype(gg)::value;
            body(std::integral_constant<int, G>{}, acc[G], e0, u, nq[NS]);
        });
    };
    using I0 = std::integral_constant<int, 0>;
    using I1 = std::integral_constant<int, 1>;
    // Tile `tile` = j (mod V) with j = J: A slot j mod D, norm slot j mod ND, bucket j mod U.
    auto step = [&](auto jj, auto has_prev, int tile) __attribute__((always_inline)) {
        constexpr int J = decltype(jj)::value;
        using SA = std::integral_constant<int, J % D>;
        using SN = std::integral_constant<int, J % ND>;
        using SP = std::integral_constant<int, (J + ND - 1) % ND>;
        mfmas(SA{}, I0{});
        if constexpr (decltype(has_prev)::value) {
            finish(SP{}, I1{}, tile - 1, std::integral_constant<int, (J + V - 1) % U>{});
            fetch_nq(SP{}, tile - 1 + ND);
        }
        mfmas(SA{}, I1{});
        fetch(SA{}, tile + D);
        finish(SN{}, I0{}, tile, std::integral_constant<int, J % U>{});
    };
    unroll<D>([&](auto s) __attribute__((always_inline)) { fetch(s, decltype(s)::value); });
    unroll<ND>([&](auto s) __attribute__((always_inline)) { fetch_nq(s, decltype(s)::value); });
    step(I0{}, std::false_type{}, 0);
    // Tiles 1 .. nt - 2 (t = 1 mod V in the loop, so tile t + VV has residue 1 + VV).
    int t = 1;
    for (; t + V <= nt - 1; t += V)
        unroll<V>([&](auto vv) __attribute__((always_inline)) {
            step(std::integral_constant<int, (1 + decltype(vv)::value) % V>{}, std::true_type{},
                 t + decltype(vv)::value);
        });
    unroll<V>([&](auto vv) __attribute__((always_inline)) {
        if (t + decltype(vv)::value < nt - 1)
            step(std::integral_constant<int, (1 + decltype(vv)::value) % V>{}, std::true_type{},
                 t + decltype(vv)::value);
    });
    // Last tile (when nt > 1), then the second half of the last tile; residues dispatched to
    // compile-time values.
    unroll<V>([&](auto vv) __attribute__((always_inline)) {
        constexpr int J = decltype(vv)::value;
        if ((nt - 1) % V == J) {
            if (nt > 1) step(vv, std::true_type{}, nt - 1);
            finish(std::integral_constant<int, J % ND>{}, I1{}, nt - 1,
                   std::integral_constant<int, J % U>{});
        }
    });
}

// Sweeps tiles 0 .. nt - 1 of src for a lane's TPW token groups with every accumulator chain
// starting from cin[g] (the MFMA adds it for free) and calls body(g, acc, tile) once per token
// group and tile (g a std::integral_constant).  Same schedule as sweep: the token groups form two
// halves, and per tile the wave issues the MFMAs of the first half, finishes the second half of
// the previous tile, issues the MFMAs of the second half, refills the A-operand ring slot and
// finishes the first half; a D-deep ring of A operands, slots fixed at compile time.
template <int RC, int K, int TPW, int D, typename Src, typename Body>
__device__ __forceinline__ void sweep_cin(const Src& src, int nt, int half,
                                          const bf16x8 (&zhi)[TPW][RC],
                                          const f32x16 (&cin)[TPW], Body&& body) {
    static_assert(TPW % 2 == 0, "two halves of token groups");
    constexpr int H = TPW / 2;
    if (nt <= 0) return;
    f32x16 acc[TPW];
    bf16x8 a[D][RC];
    auto fetch = [&](auto slot, int tile) __attribute__((always_inline)) {
        src.load_a(tile < nt ? tile : nt - 1, a[decltype(slot)::value]);
    };
    auto mfmas = [&](auto slot, auto hh) __attribute__((always_inline)) {
        constexpr int A = decltype(slot)::value, G0 = decltype(hh)::value * H;
#pragma unroll
        for (int g = G0; g < G0 + H; ++g) acc[g] = mfma_32x32x16(a[A][0], zhi[g][0], cin[g]);
#pragma unroll
        for (int c = 1; c < RC; ++c)
#pragma unroll
            for (int g = G0; g < G0 + H; ++g) acc[g] = mfma_32x32x16(a[A][c], zhi[g][c], acc[g]);
    };
    auto finish = [&](auto hh, int tile) __attribute__((always_inline)) {
        constexpr int G0 = decltype(hh)::value * H;
        unroll<H>([&](auto gg) __attribute__((always_inline)) {
            constexpr int G = G0 + decltype(gg)::value;
            body(std::integral_constant<int, G>{}, acc[G], tile);
        });
    };
    using I0 = std::integral_constant<int, 0>;
    using I1 = std::integral_constant<int, 1>;
    // the first tile is peeled (no previous tile to finish), so that the steady-state loop has
    // no branch and the compiler's wait counts stay exact
    auto step = [&](auto slot, int tile) __attribute__((always_inline)) {
        mfmas(slot, I0{});
        finish(I1{}, tile - 1);
        mfmas(slot, I1{});
        fetch(slot, tile + D);
        finish(I0{}, tile);
    };
    unroll<D>([&](auto s) __attribute__((always_inline)) { fetch(s, decltype(s)::value); });
    using S0 = std::integral_constant<int, 0>;
    mfmas(S0{}, I0{});
    mfmas(S0{}, I1{});
    fetch(S0{}, D);
    finish(I0{}, 0);
    // tiles 1 .. nt - 1: slot of tile t is t mod D
    int t = 1;
    if constexpr (D == 1) {
        for (; t < nt; ++t) step(S0{}, t);
    } else {
        for (; t < nt && t % D != 0; ++t)  // up to the next multiple of D (runtime slot)
            unroll<D>([&](auto s) __attribute__((always_inline)) {
                if (t % D == decltype(s)::value) step(s, t);
            });
        for (; t + D <= nt; t += D)
            unroll<D>([&](auto s) __attribute__((always_inline)) { step(s, t + decltype(s)::value); });
        unroll<D>([&](auto s) __attribute__((always_inline)) {
            if (t + decltype(s)::value < nt) step(s, t + decltype(s)::value);
        });
    }
    finish(I1{}, nt - 1);
}

// The same sweep over tiles whose A operands are held in registers (slot J < nt <= NTW holds
// tile (J + rot) mod nt, loaded by the caller).  The accumulator of token group g starts from
// cin[g] (the MFMA adds it for free); with NQ the norms come from LDS (gn + 8 t + 4 half),
// otherwise nq is zero.  Slots are fully unrolled, so register indices are compile-time
// constants; the bucket of slot J is J mod U.
template <int RC, int K, int TPW, int NTW, bool NQ, typename Body>
__device__ __forceinline__ void sweep_regs(const bf16x8 (&a)[NTW][RC], const float* gn, int nt,
                                           int rot, int32_t e00, int32_t M, int half,
                                           const bf16x8 (&zhi)[TPW][RC],
                                           const f32x16 (&cin)[TPW], Body&& body) {
    using C = RouteCfg<RC, K>;
    constexpr int H = TPW / 2;
    constexpr int U = C::U;
    f32x16 acc[TPW];
    f32x4 nq[2] = {f32x4{0.0f, 0.0f, 0.0f, 0.0f}, f32x4{0.0f, 0.0f, 0.0f, 0.0f}};
    auto mfmas = [&](auto jj, auto hh) __attribute__((always_inline)) {
        constexpr int J = decltype(jj)::value;
        constexpr int G0 = decltype(hh)::value * H;
#pragma unroll
        for (int g = G0; g < G0 + H; ++g) acc[g] = mfma_32x32x16(a[J][0], zhi[g][0], cin[g]);
#pragma unroll
        for (int c = 1; c < RC; ++c)
#pragma unroll
            for (int g = G0; g < G0 + H; ++g) acc[g] = mfma_32x32x16(a[J][c], zhi[g][c], acc[g]);
    };
    auto finish = [&](auto jj, auto hh) __attribute__((always_inline)) {
        constexpr int J = decltype(jj)::value;
        constexpr int G0 = decltype(hh)::value * H;
        unroll<H>([&](auto gg) __attribute__((always_inline)) {
            constexpr int G = G0 + decltype(gg)::value;
            const int tj = J + rot < nt ? J + rot : J + rot - nt;  // the slot's tile
            body(std::integral_constant<int, G>{}, acc[G], e00 + tj * 32,
                 std::integral_constant<int, J % U>{}, nq[J & 1]);
        });
    };
    using I0 = std::integral_constant<int, 0>;
    using I1 = std::integral_constant<int, 1>;
    unroll<NTW>([&](auto jj) __attribute__((always_inline)) {
        constexpr int J = decltype(jj)::value;
        if (J < nt) {  // wave-uniform
            if constexpr (NQ) {
                const int tj = J + rot < nt ? J + rot : J + rot - nt;
                nq[J & 1] = *reinterpret_cast<const f32x4*>(gn + tj * 8 + 4 * half);
            }
            mfmas(jj, I0{});
            if constexpr (J > 0) finish(std::integral_constant<int, J - 1>{}, I1{});
            mfmas(jj, I1{});
            finish(jj, I0{});
        }
    });
    unroll<NTW>([&](auto jj) __attribute__((always_inline)) {
        if (decltype(jj)::value == nt - 1) finish(jj, I1{});
    });
}

// Collect test of one token group and tile.  For every accumulator group q of the lane (rows
// 8q + 4 half + 0..3 of the tile, i.e. 4-expert group 2q + half) holding an expert with
// s_e + c N_g >= theta, appends one entry (group index gbase + 2q << 4 | bit mask of those
// experts) to the lane's slots (slot(i) = address of entry i, the last slot takes every
// entry past it) and returns the new entry count.  A first test with the lane's largest group
// norm (one compare) skips most tiles.
template <int S, typename Slot>
__device__ __forceinline__ int collect_tile(const f32x16& acc, float th, float c, const f32x4& nq,
                                            int32_t gbase, int cnt, Slot&& slot) {
    const float nmax = fmaxf(fmaxf(nq[0], nq[1]), fmaxf(nq[2], nq[3]));
    const float m16 = fmaxf(fmaxf(fmaxf(max4(acc, 0), max4(acc, 1)), max4(acc, 2)), max4(acc, 3));
    if (m16 >= th - c * nmax) {
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const float tq = th - c * nq[q];
            if (max4(acc, q) >= tq) {
                const uint32_t m = (acc[4 * q] >= tq ? 1u : 0u) | (acc[4 * q + 1] >= tq ? 2u : 0u) |
                                   (acc[4 * q + 2] >= tq ? 4u : 0u) | (acc[4 * q + 3] >= tq ? 8u : 0u);
                *slot(cnt < S ? cnt : S - 1) = (uint16_t)(((uint32_t)(gbase + 2 * q) << 4) | m);
                ++cnt;
            }
        }
    }
    return cnt;
}

// Bit mask of the experts of slot entry v that exist (ebase + 4 group + bit < M).
__device__ __forceinline__ uint32_t slot_bits(uint32_t v, int32_t ebase, int32_t M) {
    const int32_t left = M - ebase - 4 * (int32_t)(v >> 4);  // experts of the group below M
    return v & (left >= 4 ? 15u : (left > 0 ? (1u << left) - 1u : 0u));
}

// Collect test of the fused kernels (LDS for 32-bit entries): one entry per lane and tile with a
// hit, (2 tile + half) << 16 | the 16-bit mask of accumulator elements with s_e + c N_g >= theta
// (element 4q + i is expert 32 tile + 8q + 4 half + i), built without branches.
template <int S, typename Slot>
__device__ __forceinline__ int collect_tile16(const f32x16& acc, float th, float c, const f32x4& nq,
                                              int32_t code, int cnt, Slot&& slot) {
    uint32_t m = 0;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        const float tq = th - c * nq[q];
#pragma unroll
        for (int i = 0; i < 4; ++i) m |= acc[4 * q + i] >= tq ? (1u << (4 * q + i)) : 0u;
    }
    if (m) {
        *slot(cnt < S ? cnt : S - 1) = ((uint32_t)code << 16) | m;
        ++cnt;
    }
    return cnt;
}

// The same entry from an accumulator that already holds s_e + b, where b = c N_w - theta plus a
// rounding guard was fed to the MFMA as its initial value (N_w bounds every row norm of the
// wave): an element passes iff its sign bit is clear, and v_alignbit shifts the 16 sign bits
// into a mask, one instruction per element.
template <int S, typename Slot>
__device__ __forceinline__ int collect_tile_sign(const f32x16& acc, int32_t code, int cnt,
                                                 Slot&& slot) {
    // (Each element is copied to a scalar first: a bit cast applied directly to a vector element
    // reads element 0 with this compiler.)
    const float a15 = acc[15];
    uint32_t m = __builtin_bit_cast(uint32_t, a15) >> 31;
#pragma unroll
    for (int i = 14; i >= 0; --i) {
        const float ai = acc[i];
        m = __builtin_amdgcn_alignbit(m, __builtin_bit_cast(uint32_t, ai), 31);
    }
    m ^= 0xFFFFu;  // element i (bit i) passes iff acc[i] >= +0
    // Stored without a branch: an entry with no hit sits in the next free slot until a hit
    // overwrites it; slot S takes every entry past the first S (the token then overflows).
    *slot(cnt < S ? cnt : S) = ((uint32_t)code << 16) | m;
    return cnt + (m != 0u ? 1 : 0);
}

// Masks of the accumulator elements of lane half 0 and 1 that hold experts < M in the last
// tile (all ones when M is a multiple of 32): element b is row 8 (b >> 2) + 4 half + (b & 3).
struct LastTileMask {
    int32_t last;     // index of the last tile
    uint32_t m[2];
    __device__ __forceinline__ explicit LastTileMask(int32_t M) : last((M - 1) >> 5) {
        const int32_t rows = M - 32 * last;  // 1 .. 32
#pragma unroll
        for (int hf = 0; hf < 2; ++hf) {
            uint32_t mm = 0;
#pragma unroll
            for (int b = 0; b < 16; ++b)
                mm |= (8 * (b >> 2) + 4 * hf + (b & 3) < rows ? 1u : 0u) << b;
            m[hf] = mm;
        }
    }
    // Experts of a 32-bit entry that exist (< M), as a 16-bit mask.
    __device__ __forceinline__ uint32_t bits(uint32_t v) const {
        const int32_t tile = (int32_t)(v >> 17);
        const uint32_t hm = (v >> 16) & 1u ? m[1] : m[0];
        return v & (tile == last ? hm : 0xFFFFu);
    }
};

// Number of experts in the first min(cnt, S) slot entries of a lane.
template <int S, typename Slot>
__device__ __forceinline__ int slot_experts(int cnt, Slot&& slot, int32_t ebase, int32_t M) {
    int ne = 0;
    for (int i = 0; i < cnt && i < S; ++i) ne += __builtin_popcount(slot_bits(*slot(i), ebase, M));
    return ne;
}

// Writes the experts of a lane's slot entries (ebase + 4 group + bit, ids < M only) to
// out[0..), at most `room` of them.
template <typename Slot>
__device__ __forceinline__ void slot_expand(int cnt, Slot&& slot, int32_t ebase, int32_t M,
                                            int32_t* out, int room) {
    int o = 0;
    for (int i = 0; i < cnt; ++i) {
        const uint32_t v = *slot(i);
        const uint32_t m = slot_bits(v, ebase, M);
        const int32_t e = ebase + 4 * (int32_t)(v >> 4);
#pragma unroll
        for (int b = 0; b < 4; ++b) {
            if ((m >> b) & 1u) {
                if (o < room) out[o] = e + b;
                ++o;
            }
        }
    }
}

// z . u_e in fp32, rank entries in increasing order (z from registers or memory).
template <int RC, typename ZRow>
__device__ __forceinline__ float exact_logit(const ZRow& zr, const uint16_t* __restrict__ ur) {
    float acc = 0.0f;
#pragma unroll
    for (int c = 0; c < RC; ++c) {
        const bf16x8 u0 = load_bf16x8(ur + 16 * c), u1 = load_bf16x8(ur + 16 * c + 8);
#pragma unroll
        for (int i = 0; i < 8; ++i) acc = fmaf(zr(16 * c + i), (float)u0[i], acc);
#pragma unroll
        for (int i = 0; i < 8; ++i) acc = fmaf(zr(16 * c + 8 + i), (float)u1[i], acc);
    }
    return acc;
}

// Final selection for the NTOK = NTHREADS / 8 tokens tok0 .. tok0 + NTOK - 1 of a workgroup.  8
// lanes per token evaluate the token's candidates exactly (fp32 z times the bf16 expert rows, rank
// entries in increasing order).  zrow_of(j) is the fp32 z row of local token j (any address for
// tokens past T), count_of(j) the number of its candidates and cand_of(j, i) the i-th.
//  - up to RCAP candidates (the common case; RCAP = 0 turns this path off): the logits and
//    experts go to the LDS arrays lv and le ([NTOK][RCAP], given by the caller), each candidate's
//    rank under the selection order is counted against the others, ranks below k write their
//    output slot;
//  - up to cap: each lane keeps a top-K list, the 8 lists are merged, lane 0 writes;
//  - more (an overflowed list): the whole workgroup sweeps all M experts for the token.
// Either way the softmax adds exp(l - l_max) in rank order, so every path gives the same bits.
// Must be reached by every thread of the workgroup.
// on_select(e) is called once for every selected expert (for a histogram), by some thread.
struct NoSelectHook {
    __device__ __forceinline__ void operator()(int32_t) const {}
};

template <int RC, int K, int NTHREADS, int RCAP, typename ZRowOf, typename CountOf,
          typename CandOf, typename OnSelect = NoSelectHook>
__device__ __forceinline__ void finalize_tokens(ZRowOf&& zrow_of,
                                                const uint16_t* __restrict__ R2t, int32_t T,
                                                int32_t M, int32_t k, int64_t tok0, int32_t cap,
                                                CountOf&& count_of, CandOf&& cand_of,
                                                float* lv, int32_t* le,
                                                int32_t* __restrict__ idx,
                                                float* __restrict__ gate,
                                                float* __restrict__ topval,
                                                OnSelect&& on_select = OnSelect{}) {
    constexpr int R = 16 * RC;
    constexpr int NTOK = NTHREADS / 8, NW = NTHREADS / 64;
    __shared__ int32_t over_flag[NTOK];
    __shared__ float wv[NW][K];
    __shared__ int32_t wi[NW][K];
    __shared__ float ex[NTOK][K];       // exp(l - l_max) by rank
    const int tid = threadIdx.x;
    const int sub = tid & 7;
    const int j = tid >> 3;
    const int64_t tok = tok0 + j;
    const bool ok = tok < T;
    const int32_t n = ok ? count_of(j) : 0;
    // n >= k always holds (k experts reach theta); the test is a guard, not a path.
    const bool exact_sweep = ok && (n > cap || n < k);
    const bool by_rank = RCAP > 0 && ok && !exact_sweep && n <= RCAP;  // same for the token's lanes
    if (sub == 0) over_flag[j] = exact_sweep;
    float v[K];
    int32_t ix[K];
    list_init<K>(v, ix);
    if (!exact_sweep && n > sub) {
        const float* zp = zrow_of(j);
        float zreg[R];
#pragma unroll
        for (int i = 0; i < R; i += 4) {
            const f32x4 q = *reinterpret_cast<const f32x4*>(zp + i);
#pragma unroll
            for (int jj = 0; jj < 4; ++jj) zreg[i + jj] = q[jj];
        }
        // Candidates sub, sub + 8, ...: FB per round, all their rows loaded before any is used.
        constexpr int FB = 2;
        for (int i0 = sub; i0 < n; i0 += 8 * FB) {
            int32_t e[FB];
            bf16x8 u[FB][2 * RC];
#pragma unroll
            for (int b = 0; b < FB; ++b) {
                const int i = i0 + 8 * b;
                e[b] = cand_of(j, i < n ? i : i0);
            }
#pragma unroll
            for (int b = 0; b < FB; ++b)
#pragma unroll
                for (int c = 0; c < 2 * RC; ++c) u[b][c] = load_bf16x8(R2t + (int64_t)e[b] * R + 8 * c);
#pragma unroll
            for (int b = 0; b < FB; ++b) {
                float l = 0.0f;
#pragma unroll
                for (int c = 0; c < 2 * RC; ++c)
#pragma unroll
                    for (int q = 0; q < 8; ++q) l = fmaf(zreg[8 * c + q], (float)u[b][c][q], l);
                const int i = i0 + 8 * b;
                if (i < n) {
                    if (RCAP > 0 && by_rank) {
                        lv[j * RCAP + i] = l;
                        le[j * RCAP + i] = e[b];
                    } else if (better(l, e[b], v[K - 1], ix[K - 1])) {
                        list_insert<K>(v, ix, l, e[b]);
                    }
                }
            }
        }
    }
    if (!by_rank) {  // list path
        list_merge_xor<1, K>(v, ix);
        list_merge_xor<2, K>(v, ix);
        list_merge_xor<4, K>(v, ix);
        if (ok && sub == 0 && !exact_sweep) store_selection<K>(v, ix, k, tok, idx, gate, topval);
        if (ok && !exact_sweep) {
#pragma unroll
            for (int q = 0; q < K; ++q)
                if (q < k && (q & 7) == sub) on_select(ix[q]);
        }
    }
    if constexpr (RCAP > 0) {
    static_assert(RCAP % 8 == 0, "rank path: chunks of 8 entries");
    __syncthreads();
    // The token's entries are read in chunks of 8 (two 16-byte LDS reads per array); chunks
    // at or past the wave's largest candidate count are skipped (wave-uniform), entries past
    // the token's own count are masked to -inf, which no candidate ranks below.
    int nmx = by_rank ? n : 0;  // the 8 lanes of a token share n
    nmx = max(nmx, lane_xor<8>(nmx));
    nmx = max(nmx, lane_xor<16>(nmx));
    nmx = max(nmx, lane_xor<32>(nmx));
    const int nch = __builtin_amdgcn_readfirstlane((nmx + 7) >> 3);
    float L[RCAP];
    int32_t E[RCAP];
    float lmax = -__builtin_huge_valf();  // the rank-0 logit
    const float* lvj = lv + j * RCAP;
    const int32_t* lej = le + j * RCAP;
#pragma unroll
    for (int c = 0; c < RCAP / 8; ++c) {
        if (c < nch) {
#pragma unroll
            for (int h4 = 0; h4 < 2; ++h4) {
                const f32x4 a = *reinterpret_cast<const f32x4*>(lvj + 8 * c + 4 * h4);
                const i32x4 b = *reinterpret_cast<const i32x4*>(lej + 8 * c + 4 * h4);
#pragma unroll
                for (int t = 0; t < 4; ++t) {
                    const int i = 8 * c + 4 * h4 + t;
                    L[i] = i < n ? a[t] : -__builtin_huge_valf();
                    E[i] = b[t];
                    lmax = fmaxf(lmax, L[i]);
                }
            }
        }
    }
    if (by_rank) {
#pragma unroll
        for (int m = 0; m < RCAP / 8; ++m) {
            const int i = sub + 8 * m;
            if (m < nch && i < n) {
                const float l = lvj[i];
                const int32_t e = lej[i];
                int rank = 0;
#pragma unroll
                for (int c = 0; c < RCAP / 8; ++c) {
                    if (c < nch) {
#pragma unroll
                        for (int t = 0; t < 8; ++t)
                            rank += better(L[8 * c + t], E[8 * c + t], l, e) ? 1 : 0;
                    }
                }
                if (rank < k) {
                    idx[tok * k + rank] = e;
                    if (topval) topval[tok * k + rank] = l;
                    ex[j][rank] = expf(l - lmax);
                    on_select(e);
                }
            }
        }
    }
    __syncthreads();
    if (by_rank) {
        float sum = 0.0f;  // in rank order, as store_selection
#pragma unroll
        for (int i = 0; i < K; ++i)
            if (i < k) sum += ex[j][i];
#pragma unroll
        for (int i = sub; i < K; i += 8)
            if (i < k) gate[tok * k + i] = ex[j][i] / sum;
    }
    }
    // Overflowed tokens (rare): the whole workgroup sweeps all experts, thread tid taking
    // experts tid, tid + NTHREADS, ...
    if (!__syncthreads_or(exact_sweep)) return;  // workgroup-uniform
    for (int jt = 0; jt < NTOK; ++jt) {
        if (!over_flag[jt]) continue;  // workgroup-uniform
        const int64_t t = tok0 + jt;
        const float* zp = zrow_of(jt);
        list_init<K>(v, ix);
        for (int32_t e = tid; e < M; e += NTHREADS) {
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
            for (int q = 0; q < K; ++q) {
                wv[tid >> 6][q] = v[q];
                wi[tid >> 6][q] = ix[q];
            }
        }
        __syncthreads();
        if (tid == 0) {
            for (int q = 1; q < NW; ++q) {
                float bv[K];
                int32_t bi[K];
#pragma unroll
                for (int e = 0; e < K; ++e) {
                    bv[e] = wv[q][e];
                    bi[e] = wi[q][e];
                }
                list_merge<K>(v, ix, bv, bi);
            }
            store_selection<K>(v, ix, k, t, idx, gate, topval);
            for (int q = 0; q < k; ++q) on_select(ix[q]);
        }
        __syncthreads();
    }
}


// s_waitcnt immediate that waits until at most n vector memory operations are outstanding
// (n < 64; expcnt and lgkmcnt not waited for).
__host__ __device__ constexpr int vmcnt_imm(int n) {
    return (n & 15) | ((n >> 4) << 14) | (7 << 4) | (15 << 8);
}
// Direct-to-LDS load of 16 bytes per lane: lane l of the wave writes lds + 16 l (lds must be
// wave-uniform).  Completion is counted by vmcnt.
__device__ __forceinline__ void lds_dma16(const void* g, void* lds) {
    __builtin_amdgcn_global_load_lds(g, lds, 16, 0, 0);
}
// Workgroup barrier for LDS data: waits for the wave's own LDS operations and, with vmcnt_left
// < 64, until at most that many vector memory operations are outstanding (direct-to-LDS loads
// complete in order with the others).  Unlike __syncthreads it does not drain the remaining
// global loads.  The empty asm statements keep the compiler from moving memory accesses across.
template <int VM = 63>
__device__ __forceinline__ void lds_barrier() {
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_waitcnt(vmcnt_imm(VM) & ~(15 << 8));  // lgkmcnt(0)
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
}
// Tiles per wave whose A operands stay in registers in the local kernel (128 registers at r <= 32

}  // namespace more
