// Low-rank router kernels for gfx950: softmax(TopK(x R1 R2)) without materialising the
// T x M logits (Appendix "Pseudocode", inference algorithm; MoRE layer in "Preliminaries").
//
// Pipeline of one call:
//   zpass    z = x R1 (fp32 accumulate) for 32-token groups; the h axis may be split over
//            several workgroups (hsplit > 1), each writing a partial z;
//   zreduce  sums the partials in a fixed order (only when hsplit > 1);
//   route    for a block of 32*NW tokens and a chunk of the expert axis: logits
//            z R2 tile by tile on the matrix cores (expert rows streamed through LDS),
//            a screening sweep that fixes a per-token candidate threshold, an exact sweep
//            that collects the candidates, and a per-token top-K of them; the block
//            either writes the final (idx, gate, topval) or, when the expert axis is
//            split into chunks, a partial top-K list per token;
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

#include <utility>

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

    // Partial sums of waves 1..3, element-major so that a wave's 64 lanes touch 64 consecutive
    // words for each accumulator element.
    __shared__ float red[3][RT][16][64];
    if (w > 0) {
#pragma unroll
        for (int pt = 0; pt < RT; ++pt)
#pragma unroll
            for (int j = 0; j < 16; ++j) red[w - 1][pt][j][lane] = acc[pt][j];
    }
    __syncthreads();
    if (w == 0) {
#pragma unroll
        for (int pt = 0; pt < RT; ++pt) {
#pragma unroll
            for (int q = 0; q < 3; ++q)
#pragma unroll
                for (int j = 0; j < 16; ++j) acc[pt][j] += red[q][pt][j][lane];
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
// Route workgroups: 8 waves, wave w owning the 32 tokens tb*256 + 32w + (0..31), sweeping the
// expert tiles of one chunk.  The chunk's expert rows stream through LDS in blocks of BT tiles
// shared by all eight waves, so each R2 byte leaves L2 once per 256 tokens.
//
// Screening precision.  The sweeps compute s_e = z_hi . u_e on the matrix cores, with z_hi =
// bf16(z) and fp32 accumulation, instead of the logit l_e = z . u_e.  With z_lo = z - z_hi,
//   |l_e - s_e| <= ||z_lo|| ||u_e|| + r 2^-24 sum_i |z_hi,i u_e,i| <= c ||u_e||,
//   c = ||z_lo|| + r 2^-23 ||z_hi||  (Cauchy-Schwarz; accumulation bound taken twice over),
// and ||u_e|| <= N_g, the largest row norm of the 4-expert group g holding e.  So s_e - c N_g
// is a lower and s_e + c N_g an upper bound of l_e.
constexpr int kRouteWaves = 8;
constexpr int kRouteThreads = 64 * kRouteWaves;
constexpr int kRouteTokens = 32 * kRouteWaves;
constexpr int kLaneSlots = 16;         // candidate slots per lane in the collect kernel
constexpr int kMaxChunkExperts = 65536;  // slots hold 16-bit offsets inside the chunk

template <int RC, int K>
struct RouteCfg {
    static constexpr int R = 16 * RC;
    static constexpr int U = K / 4 > 1 ? K / 4 : 1;  // bucket period, in tiles
    static constexpr int L = 4 * U;                  // bucket maxima per lane (>= K)
    static constexpr int BT0 = RC <= 2 ? 8 : 4;
    static constexpr int BT = U > BT0 ? U : BT0;     // tiles per LDS block (a multiple of U)
    static constexpr int ROW = R + 8;                // padded LDS row, bf16 elements
    static constexpr int BLOCK = BT * 32 * ROW;      // bf16 elements per block buffer
    static constexpr int SPR = R / 8;                // 16-byte segments per expert row
    static constexpr int SEGS = BT * 32 * SPR;
    static constexpr int LOADS = (SEGS + kRouteThreads - 1) / kRouteThreads;
    static constexpr int GROUPS = BT * 8;            // 4-expert groups per block
    // Blocks in flight: a block is fetched DEPTH blocks ahead of its use into registers and
    // stored to one of DEPTH + 1 LDS buffers one block ahead.
    static constexpr int DEPTH = 3 * BLOCK * 2 <= 120 * 1024 ? 2 : 1;
    static constexpr int NBUF = DEPTH + 1;
    static_assert(GROUPS <= kRouteThreads, "one group norm per thread");
};

template <typename F, int... I>
__device__ __forceinline__ void unroll_impl(F&& f, std::integer_sequence<int, I...>) {
    (f(std::integral_constant<int, I>{}), ...);
}
template <int N, typename F>
__device__ __forceinline__ void unroll(F&& f) {
    unroll_impl(f, std::make_integer_sequence<int, N>{});
}

__device__ __forceinline__ float max4(const f32x16& a, int q) {
    return fmaxf(fmaxf(a[4 * q], a[4 * q + 1]), fmaxf(a[4 * q + 2], a[4 * q + 3]));
}

__device__ __forceinline__ void mask_past_end(f32x16& acc, int32_t e0, int32_t M, int half) {
#pragma unroll
    for (int j = 0; j < 16; ++j)
        if (e0 + acc_row(j, half) >= M) acc[j] = -__builtin_huge_valf();
}

// Sort N = 2^m values in descending order (bitonic network).
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

// LDS position of group g4 = (row mod 32) / 4 = 2q + half of a tile: [tile][half][q], so that a
// lane reads the norms of its four accumulator groups with one 16-byte load.
__device__ __forceinline__ int gnorm_slot(int tile, int g4) {
    return tile * 8 + (g4 & 1) * 4 + (g4 >> 1);
}

// The tiles [t0, t1) of one expert chunk, streamed through NBUF LDS block buffers, with the
// group norms N_g of each block.  OWN_NORMS: the norms are computed from the rows (and, when
// gnorm_out is set, written to gnorm_out[group]); otherwise they are read from gnorm_in.
template <int RC, int K, bool OWN_NORMS>
struct ChunkStream {
    using C = RouteCfg<RC, K>;
    const uint16_t* __restrict__ R2t;
    int32_t M;
    int64_t t0, t1;
    uint16_t* lds;   // NBUF * C::BLOCK elements
    float* lds_gn;   // NBUF * C::GROUPS
    const float* __restrict__ gnorm_in;
    float* __restrict__ gnorm_out;
    u32x4 g[C::DEPTH][C::LOADS];
    float gn[C::DEPTH];

    // Loads block b of the chunk into register set S.  Every lane always issues the same
    // loads (so that the compiler can count them and wait for one set while the next is in
    // flight): blocks past the end re-read the last block, tiles past the chunk re-read its
    // last tile and rows past M re-read row M - 1.  None of those values reaches a result:
    // such tiles are skipped and such rows are masked.
    template <int S>
    __device__ __forceinline__ void fetch(int64_t b, int64_t nblk, int tid) {
        const int64_t bb = b < nblk ? b : nblk - 1;
#pragma unroll
        for (int i = 0; i < C::LOADS; ++i) {
            const int seg = (tid + i * kRouteThreads) % C::SEGS;
            const int row = seg / C::SPR, col = seg % C::SPR;
            int64_t t = t0 + bb * C::BT + row / 32;
            t = t < t1 ? t : t1 - 1;
            int64_t e = t * 32 + (row % 32);
            e = e < M ? e : M - 1;
            g[S][i] = *reinterpret_cast<const u32x4*>(R2t + e * C::R + col * 8);
        }
        if (!OWN_NORMS) {
            int64_t t = t0 + bb * C::BT + (tid % C::GROUPS) / 8;
            t = t < t1 ? t : t1 - 1;
            gn[S] = gnorm_in[t * 8 + tid % 8];
        }
    }
    template <int S>
    __device__ __forceinline__ void stash(int64_t b, int buf, int tid, bool write_out) {
#pragma unroll
        for (int i = 0; i < C::LOADS; ++i) {
            const int seg = tid + i * kRouteThreads;
            if (seg < C::SEGS) {
                const int row = seg / C::SPR, col = seg % C::SPR;
                *reinterpret_cast<u32x4*>(lds + buf * C::BLOCK + row * C::ROW + col * 8) = g[S][i];
            }
        }
        if (OWN_NORMS) {
#pragma unroll
            for (int i = 0; i < C::LOADS; ++i) {
                const int seg = tid + i * kRouteThreads;
                const int row = seg / C::SPR, col = seg % C::SPR;
                const bf16x8 v = __builtin_bit_cast(bf16x8, g[S][i]);
                float ss = 0.0f;
#pragma unroll
                for (int q = 0; q < 8; ++q) ss = fmaf((float)v[q], (float)v[q], ss);
                // row norm^2 over the SPR lanes of the row, then the max over 4 rows
#pragma unroll
                for (int m = 1; m < C::SPR; m <<= 1) ss += __shfl_xor(ss, m, kWave);
                ss = fmaxf(ss, __shfl_xor(ss, C::SPR, kWave));
                ss = fmaxf(ss, __shfl_xor(ss, 2 * C::SPR, kWave));
                if (seg < C::SEGS && col == 0 && (row & 3) == 0) {
                    const float nrm = sqrtf(ss) * (1.0f + 0x1p-20f);
                    const int tile = row / 32;
                    lds_gn[buf * C::GROUPS + gnorm_slot(tile, (row % 32) / 4)] = nrm;
                    const int64_t t = t0 + b * C::BT + tile;
                    if (write_out && t < t1) gnorm_out[t * 8 + (row % 32) / 4] = nrm;
                }
            }
        } else if (tid < C::GROUPS) {
            lds_gn[buf * C::GROUPS + gnorm_slot(tid / 8, tid % 8)] = gn[S];
        }
    }

    // Calls body(a, e0, partial, tt, nq) for every tile of the chunk in increasing order,
    // where a[c] is this lane's A operand (expert row e0 + n, K half `half`, rank chunk c), tt
    // the tile's compile-time position in its block and nq[q] the norm bound of the lane's
    // accumulator group q.  Every thread of the workgroup must call this together.
    template <typename Body>
    __device__ __forceinline__ void sweep(int tid, int n, int half, bool write_out, Body&& body) {
        constexpr int D = C::DEPTH;
        const int64_t nblk = (t1 - t0 + C::BT - 1) / C::BT;
        if (nblk <= 0) return;
        unroll<D>([&](auto s) __attribute__((always_inline)) {
            fetch<decltype(s)::value>(decltype(s)::value, nblk, tid);
        });
        stash<0>(0, 0, tid, write_out);
        __syncthreads();
        for (int64_t b0 = 0; b0 < nblk; b0 += D) {
            unroll<D>([&](auto p) __attribute__((always_inline)) {
                constexpr int P = decltype(p)::value;  // b mod D
                const int64_t b = b0 + P;
                if (b < nblk) {
                    // register set P (block b, already in LDS) is free: fetch block b + D
                    fetch<P>(b + D, nblk, tid);
                    const int buf = (int)(b % C::NBUF);
                    const uint16_t* base = lds + buf * C::BLOCK + n * C::ROW + 8 * half;
                    unroll<C::BT>([&](auto tt) __attribute__((always_inline)) {
                        constexpr int TT = decltype(tt)::value;
                        const int64_t t = t0 + b * C::BT + TT;
                        if (t < t1) {
                            bf16x8 a[RC];
#pragma unroll
                            for (int c = 0; c < RC; ++c)
                                a[c] = load_bf16x8(base + TT * 32 * C::ROW + 16 * c);
                            const f32x4 nq = *reinterpret_cast<const f32x4*>(
                                lds_gn + buf * C::GROUPS + TT * 8 + 4 * half);
                            body(a, (int32_t)(t * 32), t * 32 + 32 > M, tt, nq);
                        }
                    });
                    if (b + 1 < nblk) stash<(P + 1) % D>(b + 1, (int)((b + 1) % C::NBUF), tid, write_out);
                    __syncthreads();
                }
            });
        }
    }
};

// Token ids, z operands and the error scale c of one lane of a route workgroup.
template <int RC>
struct RouteLane {
    int tid, lane, w, n, half, chunk, tb;
    int64_t tok;
    bool tok_ok;
    bf16x8 zhi[RC];
    float c;

    __device__ __forceinline__ RouteLane(const float* __restrict__ z, int32_t T, int32_t chunks) {
        tid = threadIdx.x;
        lane = tid & 63;
        w = __builtin_amdgcn_readfirstlane(tid >> 6);
        n = lane & 31;
        half = lane >> 5;
        // Consecutive workgroups take consecutive chunks: with chunks a multiple or a divisor
        // of 8, a chunk always lands on the same XCD(s) (workgroups are dealt to the eight XCDs
        // round robin) and its expert rows stay in that XCD's L2.
        chunk = (int)(blockIdx.x % (unsigned)chunks);
        tb = (int)(blockIdx.x / (unsigned)chunks);
        tok = ((int64_t)tb * kRouteWaves + w) * 32 + n;
        tok_ok = tok < T;
        constexpr int R = 16 * RC;
        float lo2 = 0.0f, hi2 = 0.0f;
#pragma unroll
        for (int cc = 0; cc < RC; ++cc) {
            float v[8];
            if (tok_ok) {
                const f32x4* p = reinterpret_cast<const f32x4*>(z + tok * R + 16 * cc + 8 * half);
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
#pragma unroll
            for (int q = 0; q < 8; ++q) {
                const __bf16 h = (__bf16)v[q];
                const float hf = (float)h;
                const float lf = v[q] - hf;
                zhi[cc][q] = h;
                hi2 = fmaf(hf, hf, hi2);
                lo2 = fmaf(lf, lf, lo2);
            }
        }
        hi2 += __shfl_xor(hi2, 32, kWave);
        lo2 += __shfl_xor(lo2, 32, kWave);
        c = (sqrtf(lo2) + (float)R * 0x1p-23f * sqrtf(hi2)) * (1.0f + 0x1p-10f);
    }
};

template <int RC>
__device__ __forceinline__ f32x16 screened_tile(const bf16x8 (&a)[RC], const bf16x8 (&zhi)[RC]) {
    f32x16 acc = zero_f32x16();
#pragma unroll
    for (int c = 0; c < RC; ++c) acc = mfma_32x32x16(a[c], zhi[c], acc);
    return acc;
}

// Screening sweep.  For each accumulator group q of a tile the lane forms the lower bound
// max_{e in group} s_e - c N_g (attained by one expert of the group) and keeps the maxima of
// these bounds in L = 4U buckets (group q of tile t goes to bucket 4 (t mod U) + q).  The
// buckets of a token's two lanes partition the chunk's experts into 2L >= 2K groups, so the
// K largest bucket maxima belong to K distinct experts, each with logit >= its value.
// Output per token and chunk: those K values, descending, in top[chunk][token][0..K-1].
// Workgroups of token block 0 also write the group norms of their chunk to gnorm[].
template <int RC, int K>
__global__ __launch_bounds__(kRouteThreads, 4) void screen_kernel(
    const float* __restrict__ z, const uint16_t* __restrict__ R2t, int32_t T, int32_t M,
    int32_t chunks, float* __restrict__ top, float* __restrict__ gnorm) {
    using C = RouteCfg<RC, K>;
    constexpr int U = C::U, L = C::L;
    __shared__ __attribute__((aligned(16))) uint16_t a_lds[C::NBUF * C::BLOCK];
    __shared__ __attribute__((aligned(16))) float gn_lds[C::NBUF * C::GROUPS];
    const RouteLane<RC> ln(z, T, chunks);
    const bool wave_active = ((int64_t)ln.tb * kRouteWaves + ln.w) * 32 < T;  // wave-uniform
    const int64_t Mt = ((int64_t)M + 31) / 32;
    ChunkStream<RC, K, true> st{R2t, M, Mt * ln.chunk / chunks, Mt * (ln.chunk + 1) / chunks,
                                a_lds, gn_lds, nullptr, gnorm};

    float bm[L];
#pragma unroll
    for (int b = 0; b < L; ++b) bm[b] = -__builtin_huge_valf();
    st.sweep(ln.tid, ln.n, ln.half, ln.tb == 0,
             [&](const bf16x8 (&a)[RC], int32_t e0, bool partial, auto tt, const f32x4& nq)
                 __attribute__((always_inline)) {
                 if (!wave_active) return;
                 f32x16 acc = screened_tile<RC>(a, ln.zhi);
                 if (partial) mask_past_end(acc, e0, M, ln.half);
                 constexpr int u = decltype(tt)::value % U;
#pragma unroll
                 for (int q = 0; q < 4; ++q)
                     bm[4 * u + q] = fmaxf(bm[4 * u + q], max4(acc, q) - ln.c * nq[q]);
             });

    // K largest of the token's 2L bucket maxima.
    sort_desc<L>(bm);
    float pb[L];
#pragma unroll
    for (int b = 0; b < L; ++b) pb[b] = __shfl_xor(bm[b], 32, kWave);
    vlist_merge<L>(bm, pb);
    if (ln.half == 0 && ln.tok_ok) {
        float* o = top + ((int64_t)ln.chunk * T + ln.tok) * K;
#pragma unroll
        for (int j = 0; j < K; ++j) o[j] = bm[j];
    }
}

// Threshold per token: theta = the k-th largest of the union of all chunks' lists, lowered by
// a rounding guard.  k distinct experts have logit >= theta, so the k-th largest logit is >=
// theta and every expert of the top k has s_e + c N_g >= theta.  G threads per token (a power
// of two <= 64) share the chunk lists.  Also clears the token's candidate count.
template <int K>
__global__ __launch_bounds__(256) void theta_kernel(const float* __restrict__ top, int32_t T,
                                                    int32_t chunks, int32_t k, int32_t G,
                                                    float* __restrict__ theta,
                                                    int32_t* __restrict__ count) {
    const int64_t gid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
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
    theta[tok] = th - fabsf(th) * 0x1p-20f;
    count[tok] = 0;
}

// Collect sweep: recomputes s for the chunk and appends every expert with s_e + c N_g >=
// theta[token] to the token's candidate list cand[token][0..cap-1] (order of arrival,
// count[token] entries).  A lane buffers its hits in kLaneSlots LDS slots (16-bit offsets in
// the chunk); the token's two lanes reserve their list space with one atomic add at the end.
// A lane with more hits marks the token as overflowed (count > cap), which sends it to the
// exact sweep of the finalize kernel.
template <int RC, int K>
__global__ __launch_bounds__(kRouteThreads, 4) void collect_kernel(
    const float* __restrict__ z, const uint16_t* __restrict__ R2t, int32_t T, int32_t M,
    int32_t chunks, const float* __restrict__ theta, const float* __restrict__ gnorm,
    int32_t* __restrict__ count, int32_t* __restrict__ cand, int32_t cap) {
    using C = RouteCfg<RC, K>;
    __shared__ __attribute__((aligned(16))) uint16_t a_lds[C::NBUF * C::BLOCK];
    __shared__ __attribute__((aligned(16))) float gn_lds[C::NBUF * C::GROUPS];
    __shared__ uint16_t slots[kLaneSlots][kRouteThreads];
    const RouteLane<RC> ln(z, T, chunks);
    const bool wave_active = ((int64_t)ln.tb * kRouteWaves + ln.w) * 32 < T;
    const int64_t Mt = ((int64_t)M + 31) / 32;
    ChunkStream<RC, K, false> st{R2t, M, Mt * ln.chunk / chunks, Mt * (ln.chunk + 1) / chunks,
                                 a_lds, gn_lds, gnorm, nullptr};
    const int32_t ebase = (int32_t)(st.t0 * 32);
    // Lanes past T never qualify (+inf threshold).
    const float th = ln.tok_ok ? theta[ln.tok] : __builtin_huge_valf();

    int cnt = 0;
    st.sweep(ln.tid, ln.n, ln.half, false,
             [&](const bf16x8 (&a)[RC], int32_t e0, bool partial, auto tt, const f32x4& nq)
                 __attribute__((always_inline)) {
                 (void)tt;
                 if (!wave_active) return;
                 f32x16 acc = screened_tile<RC>(a, ln.zhi);
                 if (partial) mask_past_end(acc, e0, M, ln.half);
                 float tq[4];
#pragma unroll
                 for (int q = 0; q < 4; ++q) tq[q] = fmaxf(th - ln.c * nq[q], -__FLT_MAX__);
                 const float m = fmaxf(fmaxf(max4(acc, 0) - tq[0], max4(acc, 1) - tq[1]),
                                       fmaxf(max4(acc, 2) - tq[2], max4(acc, 3) - tq[3]));
                 if (m >= 0.0f) {
#pragma unroll
                     for (int j = 0; j < 16; ++j) {
                         if (acc[j] >= tq[j >> 2]) {
                             if (cnt < kLaneSlots)
                                 slots[cnt][ln.tid] = (uint16_t)(e0 - ebase + acc_row(j, ln.half));
                             ++cnt;
                         }
                     }
                 }
             });

    const int pc = __shfl_xor(cnt, 32, kWave);
    const bool over = cnt > kLaneSlots || pc > kLaneSlots;
    const int total = cnt + pc;
    int base = 0;
    if (ln.half == 0 && ln.tok_ok && total > 0)
        base = atomicAdd(&count[ln.tok], over ? cap + 1 : total);
    base = __shfl(base, ln.n, kWave);  // lane half 1 reads its partner's reservation
    if (ln.tok_ok && !over) {
        const int off = base + (ln.half ? pc : 0);
        for (int i = 0; i < cnt; ++i)
            if (off + i < cap) cand[ln.tok * cap + off + i] = ebase + (int32_t)slots[i][ln.tid];
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

// Final selection: 8 lanes per token evaluate the token's candidates exactly, keep a top-K
// list each and merge; lane 0 of the group writes the softmax over the best k.  Tokens whose
// candidate list overflowed are recomputed by the whole workgroup with an exact sweep over
// all M experts.
template <int RC, int K>
__global__ __launch_bounds__(256) void finalize_kernel(
    const float* __restrict__ z, const uint16_t* __restrict__ R2t, int32_t T, int32_t M,
    int32_t k, const int32_t* __restrict__ count, const int32_t* __restrict__ cand, int32_t cap,
    int32_t* __restrict__ idx, float* __restrict__ gate, float* __restrict__ topval) {
    constexpr int R = 16 * RC;
    __shared__ int32_t over_flag[32];
    __shared__ float wv[4][K];
    __shared__ int32_t wi[4][K];
    const int tid = threadIdx.x;
    const int sub = tid & 7;
    const int64_t tok = (int64_t)blockIdx.x * 32 + (tid >> 3);
    const bool ok = tok < T;
    const int32_t n = ok ? count[tok] : 0;
    // n >= k always holds (k experts reach theta); the test is a guard, not a path.
    const bool exact_sweep = ok && (n > cap || n < k);
    if (sub == 0) over_flag[tid >> 3] = exact_sweep;
    float v[K];
    int32_t ix[K];
    list_init<K>(v, ix);
    if (!exact_sweep && n > sub) {
        const float* zp = z + (ok ? tok : 0) * R;
        auto eval = [&](auto zr) __attribute__((always_inline)) {
            // candidates sub, sub + 8, ...: two per round so that their loads overlap
            for (int i = sub; i < n; i += 16) {
                const bool two = i + 8 < n;
                const int32_t e0 = cand[tok * cap + i];
                const int32_t e1 = two ? cand[tok * cap + i + 8] : e0;
                const float l0 = exact_logit<RC>(zr, R2t + (int64_t)e0 * R);
                const float l1 = exact_logit<RC>(zr, R2t + (int64_t)e1 * R);
                if (better(l0, e0, v[K - 1], ix[K - 1])) list_insert<K>(v, ix, l0, e0);
                if (two && better(l1, e1, v[K - 1], ix[K - 1])) list_insert<K>(v, ix, l1, e1);
            }
        };
        if constexpr (RC <= 4) {
            float zreg[R];
#pragma unroll
            for (int i = 0; i < R; i += 4) {
                const f32x4 q = *reinterpret_cast<const f32x4*>(zp + i);
#pragma unroll
                for (int j = 0; j < 4; ++j) zreg[i + j] = q[j];
            }
            eval([&](int i) __attribute__((always_inline)) { return zreg[i]; });
        } else {
            eval([&](int i) __attribute__((always_inline)) { return zp[i]; });
        }
    }
#pragma unroll
    for (int s = 1; s < 8; s <<= 1) list_merge_xor<K>(v, ix, s);
    if (ok && sub == 0 && !exact_sweep) store_selection<K>(v, ix, k, tok, idx, gate, topval);
    __syncthreads();
    // Overflowed tokens (rare): the whole workgroup sweeps all experts, thread tid taking
    // experts tid, tid + 256, ...
    for (int j = 0; j < 32; ++j) {
        if (!over_flag[j]) continue;  // workgroup-uniform
        const int64_t t = (int64_t)blockIdx.x * 32 + j;
        const float* zp = z + t * R;
        list_init<K>(v, ix);
        for (int32_t e = tid; e < M; e += 256) {
            const float l = exact_logit<RC>([&](int i) { return zp[i]; }, R2t + (int64_t)e * R);
            if (better(l, e, v[K - 1], ix[K - 1])) list_insert<K>(v, ix, l, e);
        }
#pragma unroll
        for (int s = 1; s < 64; s <<= 1) list_merge_xor<K>(v, ix, s);
        if ((tid & 63) == 0) {
#pragma unroll
            for (int q = 0; q < K; ++q) {
                wv[tid >> 6][q] = v[q];
                wi[tid >> 6][q] = ix[q];
            }
        }
        __syncthreads();
        if (tid == 0) {
            for (int q = 1; q < 4; ++q) {
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
    q.ntb = (int32_t)((T + kRouteTokens - 1) / kRouteTokens);
    const int64_t Mt = ((int64_t)M + 31) / 32;
    const int U = q.K / 4 > 1 ? q.K / 4 : 1;
    const int BT0 = q.RC <= 2 ? 8 : 4;
    const int BT = U > BT0 ? U : BT0;
    if (m_chunks > 0) {
        q.chunks = m_chunks;
    } else {
        // Two route workgroups per CU (512 in all), expert slices of at most 2 MiB (an XCD's
        // L2 keeps the slice while the token blocks pass over it), at least one full LDS
        // block per chunk.
        const int64_t r2_bytes = (int64_t)M * r * 2;
        int64_t C = 1;
        while (C < 1024 && ((int64_t)q.ntb * C < 512 || r2_bytes / C > ((int64_t)2 << 20)) &&
               Mt / (2 * C) >= BT)
            C *= 2;
        q.chunks = (int32_t)C;
    }
    if (q.chunks < 1 || q.chunks > 1024) return false;
    // Candidate slots hold 16-bit offsets inside a chunk.
    while (Mt * 32 / q.chunks + 32 > kMaxChunkExperts) q.chunks *= 2;
    q.theta_group = 1;
    while (q.theta_group < 64 && q.theta_group * 16 < q.chunks) q.theta_group *= 2;
    q.cap = 512;
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
    q.off_top = off;
    off += align256((size_t)q.chunks * T * q.K * sizeof(float));
    q.off_gnorm = off;
    off += align256((size_t)Mt * 8 * sizeof(float));
    q.off_tau = off;
    off += align256((size_t)T * sizeof(float));
    q.off_count = off;
    off += align256((size_t)T * sizeof(int32_t));
    q.off_cand = off;
    off += align256((size_t)T * q.cap * sizeof(int32_t));
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

struct RouteArgs {
    const float* z;
    const uint16_t* R2t;
    int32_t T, M, k;
    float *top, *gnorm, *theta;
    int32_t *count, *cand;
    int32_t* idx;
    float *gate, *topval;
};

template <int RC, int K>
static void launch_route(const LowrankPlan& p, const RouteArgs& a, hipStream_t st) {
    const dim3 grid((unsigned)((int64_t)p.ntb * p.chunks));
    hipLaunchKernelGGL((screen_kernel<RC, K>), grid, dim3(kRouteThreads), 0, st, a.z, a.R2t, a.T,
                       a.M, p.chunks, a.top, a.gnorm);
    const int64_t nth = (int64_t)a.T * p.theta_group;
    hipLaunchKernelGGL((theta_kernel<K>), dim3((unsigned)((nth + 255) / 256)), dim3(256), 0, st,
                       a.top, a.T, p.chunks, a.k, p.theta_group, a.theta, a.count);
    hipLaunchKernelGGL((collect_kernel<RC, K>), grid, dim3(kRouteThreads), 0, st, a.z, a.R2t, a.T,
                       a.M, p.chunks, a.theta, a.gnorm, a.count, a.cand, p.cap);
    hipLaunchKernelGGL((finalize_kernel<RC, K>), dim3((unsigned)((a.T + 31) / 32)), dim3(256), 0,
                       st, a.z, a.R2t, a.T, a.M, a.k, a.count, a.cand, p.cap, a.idx, a.gate,
                       a.topval);
}

template <int RC>
static bool dispatch_route_k(const LowrankPlan& p, const RouteArgs& a, hipStream_t st) {
    switch (p.K) {
        case 1: launch_route<RC, 1>(p, a, st); return true;
        case 2: launch_route<RC, 2>(p, a, st); return true;
        case 4: launch_route<RC, 4>(p, a, st); return true;
        case 8: launch_route<RC, 8>(p, a, st); return true;
        case 16: launch_route<RC, 16>(p, a, st); return true;
        case 32: launch_route<RC, 32>(p, a, st); return true;
    }
    return false;
}

hipError_t lowrank_launch(const LowrankPlan& p, const uint16_t* x, const uint16_t* R1t,
                          const uint16_t* R2t, int64_t T, int32_t h, int32_t r, int32_t M,
                          int32_t k, int32_t* idx, float* gate, float* topval, void* workspace,
                          hipStream_t st) {
    char* ws = static_cast<char*>(workspace);
    float* zparts = reinterpret_cast<float*>(ws + p.off_zparts);
    RouteArgs a;
    a.z = reinterpret_cast<float*>(ws + p.off_z);
    a.R2t = R2t;
    a.T = (int32_t)T;
    a.M = M;
    a.k = k;
    a.top = reinterpret_cast<float*>(ws + p.off_top);
    a.gnorm = reinterpret_cast<float*>(ws + p.off_gnorm);
    a.theta = reinterpret_cast<float*>(ws + p.off_tau);
    a.count = reinterpret_cast<int32_t*>(ws + p.off_count);
    a.cand = reinterpret_cast<int32_t*>(ws + p.off_cand);
    a.idx = idx;
    a.gate = gate;
    a.topval = topval;

    switch (p.RT) {
        case 1: launch_zpass<1>(p, x, R1t, zparts, T, h, r, st); break;
        case 2: launch_zpass<2>(p, x, R1t, zparts, T, h, r, st); break;
        case 4: launch_zpass<4>(p, x, R1t, zparts, T, h, r, st); break;
        default: return hipErrorInvalidValue;
    }
    if (p.hsplit > 1) {
        const int64_t n = T * r;
        const unsigned blocks = (unsigned)((n + 255) / 256 < 4096 ? (n + 255) / 256 : 4096);
        hipLaunchKernelGGL(zreduce_kernel, dim3(blocks), dim3(256), 0, st, zparts,
                           const_cast<float*>(a.z), n, p.hsplit);
    }
    bool ok = false;
    switch (p.RC) {
        case 1: ok = dispatch_route_k<1>(p, a, st); break;
        case 2: ok = dispatch_route_k<2>(p, a, st); break;
        case 4: ok = dispatch_route_k<4>(p, a, st); break;
        case 8: ok = dispatch_route_k<8>(p, a, st); break;
    }
    if (!ok) return hipErrorInvalidValue;
    return hipGetLastError();
}

}  // namespace more
