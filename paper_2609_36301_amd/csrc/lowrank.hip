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

// ------------------------------------------------------------------------------ zpass
// One workgroup = 4 waves = 128 tokens, wave w owning tokens 32w..32w+31 of the block.  The h
// axis is walked in chunks of 64 (4 MFMA k-steps); the chunk of R1 (all rank rows) is staged
// in LDS and shared by the four waves; x and R1 are prefetched D chunks ahead in registers.  With
// hsplit > 1 the chunks are split over hsplit workgroups and each split writes a partial z.
constexpr int kZWaves = 4;
constexpr float kPhantomNorm = 0x1p100f;  // norm bound of a 4-expert group reaching past M
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

// Token groups of 32 per wave: 4 at r = 64 and K <= 8 (the A-operand reads from LDS, which do not
// overlap the MFMAs, then cost half as much per MFMA), else 2.
__host__ __device__ constexpr int route_tpw(int RC, int K) { return RC == 4 && K <= 8 ? 4 : 2; }

template <int RC, int K>
struct RouteCfg {
    static constexpr int R = 16 * RC;
    static constexpr int SPR = R / 8;                     // 16-byte segments per expert row
    static constexpr int U = K / 4 > 1 ? K / 4 : 1;       // bucket period, in tiles
    static constexpr int L = 4 * U;                       // bucket maxima per lane (>= K)
    static constexpr int EMAX = kChunkBytes / (2 * R);    // experts per chunk (multiple of 32)
    static constexpr int TPW = route_tpw(RC, K);          // token groups per wave
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
template <int RC, int K, int NTHREADS, int RCAP, typename ZRowOf, typename CountOf,
          typename CandOf>
__device__ __forceinline__ void finalize_tokens(ZRowOf&& zrow_of,
                                                const uint16_t* __restrict__ R2t, int32_t T,
                                                int32_t M, int32_t k, int64_t tok0, int32_t cap,
                                                CountOf&& count_of, CandOf&& cand_of,
                                                float* lv, int32_t* le,
                                                int32_t* __restrict__ idx,
                                                float* __restrict__ gate,
                                                float* __restrict__ topval) {
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
        }
        __syncthreads();
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
    const int tokens_per_block = q.fused ? kFusedTokens : 32 * route_tpw(q.RC, q.K) * kRouteWaves;
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
    const int32_t NC = (h / 16 + 3) / 4;
    const int64_t ntbz = (T + kZTokens - 1) / kZTokens;
    int64_t hs = ntbz >= 256 ? 1 : (256 + ntbz - 1) / ntbz;
    if (hs > NC) hs = NC;
    q.steps_per_split = (int32_t)((NC + hs - 1) / hs);  // chunks per split
    q.hsplit = (NC + q.steps_per_split - 1) / q.steps_per_split;
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
