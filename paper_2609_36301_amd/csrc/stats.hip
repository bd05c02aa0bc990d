// Softmax statistics of the training forward pass for gfx950 (Appendix "Pseudocode", training
// forward algorithm; eqs. app_softmax, app_psum and app_online):
//   m[t]    = max_e l_te                         (the top-1 logit of the routing call)
//   Z[t]    = sum_e exp(l_te - m[t])             (the softmax normaliser over all M experts)
//   psum[e] = sum_t exp(l_te - m[t]) / Z[t]      (column sums of the row softmax)
// with l = z R2 and z = x R1, never written out as a T x M matrix.  Z needs every logit of a
// token and psum needs Z, so the experts are swept twice, as in the paper's algorithm: once
// for Z (tokens held in registers, expert rows resident in LDS) and once for psum (expert rows
// held in registers, tokens streamed).
//
// Kernels of one call, after the routing call has produced z and the top-1 logits:
//   stats_prep     z' = z log2(e) as bf16 hi/lo rows (about 16 significant bits) and
//                  -m' = -m log2(e) per token;
//   stats_z        per (expert chunk, token): sum over the chunk of 2^(z' u_e - m'), the MFMA
//                  adding -m' through its accumulator input (C operand);
//   stats_combine  Z = the chunk sums in chunk order; m; the token's bias -(m' + log2 Z);
//   stats_psum     per (token split, expert): sum over the split of 2^(z' u_e - m' - log2 Z);
//   stats_reduce   psum = the split sums in split order.
// Every sum runs in a fixed order, so results are reproducible bit for bit on a given shape.
//
// Numerics.  The expert contraction reads z' as hi + lo, whose rounding (2^-18 relative) and the
// fp32 accumulation put every exponent within about 2^-18 sum_i |z'_i u_ei| + 2r 2^-24
// (|m'| + sum_i |z'_i u_ei|) of its exact value; 2^x is v_exp_f32 (1 ulp).
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "device_common.h"
#include "lowrank.h"
#include "route_device.h"

namespace more {

constexpr float kLog2e = 1.44269504088896340736f;
constexpr float kNoToken = -0x1p100f;   // bias of columns past T: 2^(finite + kNoToken) = 0

__device__ __forceinline__ float exp2_fast(float x) { return __builtin_amdgcn_exp2f(x); }

// ------------------------------------------------------------------------------ prep
// One thread per element of z [T][r]: zhl [T][2][r] holds bf16(z') then bf16(z' - bf16(z')).
__global__ __launch_bounds__(256) void stats_prep_kernel(const float* __restrict__ z,
                                                         const float* __restrict__ mtop,
                                                         int32_t ks, int32_t T, int32_t r,
                                                         uint16_t* __restrict__ zhl,
                                                         float* __restrict__ mb) {
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i >= (int64_t)T * r) return;
    const int64_t t = i / r;
    const int32_t j = (int32_t)(i - t * r);
    const float v = z[i] * kLog2e;
    const __bf16 hb = (__bf16)v;
    const __bf16 lb = (__bf16)(v - (float)hb);
    zhl[t * 2 * r + j] = __builtin_bit_cast(uint16_t, hb);
    zhl[t * 2 * r + r + j] = __builtin_bit_cast(uint16_t, lb);
    if (j == 0) mb[t] = -(mtop[t * ks] * kLog2e);
}

// ------------------------------------------------------------------------------ Z sweep
// Expert-resident like the routing sweeps: a workgroup of 8 waves loads one chunk of R2t rows
// into LDS and sweeps it for blocks of 512 tokens, wave w taking tokens 64 w .. 64 w + 63 of a
// block (two groups of 32, one per MFMA column tile).  Each A operand (32 expert rows) read
// from LDS feeds four MFMA chains steps: hi and lo of both token groups.
constexpr int kStatsTPW = 2;
constexpr int kStatsTokens = 32 * kStatsTPW * kRouteWaves;

// A-operand source that returns each LDS row fragment twice: chunks 0 .. RC-1 pair with z'_hi,
// chunks RC .. 2RC-1 (the same registers) with z'_lo.
template <int RC>
struct HiLoRows {
    LdsRows<RC, 1> rows;
    __device__ __forceinline__ void load_a(int tile, bf16x8 (&a)[2 * RC]) const {
        bf16x8 t[RC];
        rows.load_a(tile, t);
#pragma unroll
        for (int c = 0; c < RC; ++c) {
            a[c] = t[c];
            a[RC + c] = t[c];
        }
    }
};

template <int RC>
__global__ __launch_bounds__(kRouteThreads, 1) void stats_z_kernel(
    const uint16_t* __restrict__ zhl, const float* __restrict__ mb,
    const uint16_t* __restrict__ R2t, int32_t T, int32_t M, int32_t chunks, int32_t splits,
    float* __restrict__ Zp) {
    using C = RouteCfg<RC, 1>;
    constexpr int TPW = kStatsTPW, R = C::R;
    __shared__ __attribute__((aligned(16))) uint16_t rows[C::EMAX * C::R];
    const RouteSplit sp = route_split(T, M, chunks, splits, kStatsTokens);
    load_chunk<RC, 1>(R2t, nullptr, M, sp.t0, sp.t1, rows, nullptr, false);
    const int lane = threadIdx.x & 63;
    const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int n = lane & 31, half = lane >> 5;
    const int nt = (int)(sp.t1 - sp.t0);
    const HiLoRows<RC> src{LdsRows<RC, 1>(rows, nullptr, n, half)};
    // rows past M in the last tile re-read row M - 1 (load_chunk) and are left out of the sums
    const LastTileMask ltm(M);
    const uint32_t lmask = half ? ltm.m[1] : ltm.m[0];
    const int tlast = (int)(ltm.last - sp.t0);  // chunk-local index of the last tile (or outside)
    for (int64_t blk = sp.blk0; blk < sp.blk1; ++blk) {
        const int64_t first = blk * kStatsTokens + (int64_t)w * 32 * TPW;
        if (first >= T) break;  // wave-uniform
        bf16x8 zz[TPW][2 * RC];
        f32x16 cin[TPW];
        float zs[TPW];
#pragma unroll
        for (int g = 0; g < TPW; ++g) {
            const int64_t t = first + 32 * g + n;
            const bool ok = t < T;
            const uint16_t* zr = zhl + (ok ? t : 0) * (2 * R) + 8 * half;
#pragma unroll
            for (int c = 0; c < RC; ++c) {
                const bf16x8 hv = load_bf16x8(zr + 16 * c);
                const bf16x8 lv = load_bf16x8(zr + R + 16 * c);
                zz[g][c] = ok ? hv : zero_bf16x8();
                zz[g][RC + c] = ok ? lv : zero_bf16x8();
            }
            const float b = ok ? mb[t] : 0.0f;
#pragma unroll
            for (int i = 0; i < 16; ++i) cin[g][i] = b;
            zs[g] = 0.0f;
        }
        sweep_cin<2 * RC, 1, TPW, 1>(
            src, nt, half, zz, cin,
            [&](auto gg, const f32x16& acc, int tl) __attribute__((always_inline)) {
                constexpr int g = decltype(gg)::value;
                float s = 0.0f;
                if (tl != tlast) {
#pragma unroll
                    for (int i = 0; i < 16; ++i) s += exp2_fast(acc[i]);
                } else {
#pragma unroll
                    for (int i = 0; i < 16; ++i) s += (lmask >> i) & 1u ? exp2_fast(acc[i]) : 0.0f;
                }
                zs[g] += s;
            });
#pragma unroll
        for (int g = 0; g < TPW; ++g) {
            const float tot = sum_pair32(zs[g]);  // the two lane halves hold disjoint rows
            const int64_t t = first + 32 * g + n;
            if (half == 0 && t < T) Zp[(int64_t)sp.chunk * T + t] = tot;
        }
    }
}

// ------------------------------------------------------------------------------ partial sums
// out[j] = sum over p < P of in[p N + j] in a fixed order: G threads per output (consecutive
// blocks of 256 / G outputs per workgroup, the outputs fastest so that loads coalesce); thread q
// sums p = q, q + G, ... in increasing order, then the G partials are added in order of q.
template <typename Epilogue>
__device__ __forceinline__ void column_sums(const float* __restrict__ in, int32_t P, int64_t N,
                                            int G, float* red, Epilogue&& epi) {
    const int per = 256 / G;
    const int q = threadIdx.x / per, jj = threadIdx.x % per;
    const int64_t j = (int64_t)blockIdx.x * per + jj;
    float s = 0.0f;
    if (j < N) {
        int32_t p = q;
        for (; p + 7 * G < P; p += 8 * G) {  // eight loads in flight, added in order
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
        epi(j, t);
    }
}

// Z[t] = the chunk partials in order; m[t]; bias[t] = -(m' + log2 Z) for the psum sweep.
__global__ __launch_bounds__(256) void stats_combine_kernel(const float* __restrict__ Zp,
                                                            int32_t chunks, int32_t G,
                                                            const float* __restrict__ mtop,
                                                            int32_t ks,
                                                            const float* __restrict__ mb,
                                                            int32_t T, float* __restrict__ m_out,
                                                            float* __restrict__ Z_out,
                                                            float* __restrict__ bias) {
    __shared__ float red[256];
    column_sums(Zp, chunks, T, G, red, [&](int64_t t, float z) {
        m_out[t] = mtop[t * ks];
        Z_out[t] = z;
        bias[t] = mb[t] - log2f(z);
    });
}

// ------------------------------------------------------------------------------ psum sweep
// A workgroup of 8 waves owns 8 NE expert tiles (wave w tiles NE w .. NE w + NE - 1 of its
// block), held as B operands (expert columns) in registers, and streams the 32-token tiles of
// its token split through LDS: stages of SB tiles (z'_hi, z'_lo and the bias of each token),
// double buffered, loaded by the whole workgroup one stage ahead.  Tokens are the MFMA rows, so
// a lane holds one expert column and sixteen token rows of each tile, adds the sixteen
// probabilities, and keeps one running sum per expert tile; the two lane halves (disjoint token
// rows) are added at the end.  The bias -(m' + log2 Z) of a row enters through the MFMA's C
// operand, read from LDS as four 16-byte pieces per tile.
constexpr int kPsumWaves = 8;
constexpr int kPsumThreads = 64 * kPsumWaves;
constexpr int kPsumSB = 4;  // token tiles per stage

template <int RC>
struct PsumCfg {
    static constexpr int R = 16 * RC;
    static constexpr int NE = 4;                                  // expert tiles per wave
    static constexpr int EXPERTS = 32 * NE * kPsumWaves;          // experts per workgroup
    static constexpr int ROW = 2 * R + 8;                         // bf16 per token row in LDS
    static constexpr int SEGS = kPsumSB * 32 * (2 * R / 8);       // 16-byte pieces per stage
    static constexpr int SEG_PER_THREAD = SEGS / kPsumThreads;
    static_assert(SEGS % kPsumThreads == 0, "whole pieces per thread");
};

template <int RC>
__global__ __launch_bounds__(kPsumThreads, 1) void stats_psum_kernel(
    const uint16_t* __restrict__ zhl, const float* __restrict__ bias,
    const uint16_t* __restrict__ R2t, int32_t T, int32_t M, int32_t eblocks, int32_t splits,
    float* __restrict__ part) {
    using C = PsumCfg<RC>;
    constexpr int R = C::R, NE = C::NE, ROW = C::ROW, SB = kPsumSB, SPT = C::SEG_PER_THREAD;
    constexpr int RSEG = 2 * R / 8;  // 16-byte pieces per token (hi then lo)
    __shared__ __attribute__((aligned(16))) uint16_t zs[2][SB * 32 * ROW];
    __shared__ __attribute__((aligned(16))) float bs[2][SB * 32];
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int n = lane & 31, half = lane >> 5;
    const int32_t eb = (int32_t)(blockIdx.x % (unsigned)eblocks);
    const int32_t split = (int32_t)(blockIdx.x / (unsigned)eblocks);
    const int64_t Tt = ((int64_t)T + 31) / 32;
    const int64_t tt0 = Tt * split / splits, tt1 = Tt * (split + 1) / splits;
    const int ntiles = (int)(tt1 - tt0);
    const int nstages = (ntiles + SB - 1) / SB;
    const int32_t Mt = (M + 31) / 32;
    const int32_t tile0 = (eb * kPsumWaves + w) * NE;
    const bool active = tile0 < Mt;  // wave-uniform; idle waves still stage tokens
    bf16x8 b[NE][RC];
#pragma unroll
    for (int j = 0; j < NE; ++j) {
        int64_t e = (int64_t)32 * (tile0 + j) + n;
        e = e < M ? e : M - 1;  // columns past M: copies of expert M - 1, never stored
#pragma unroll
        for (int c = 0; c < RC; ++c) b[j][c] = load_bf16x8(R2t + e * R + 16 * c + 8 * half);
    }
    // Stage loads: piece g of a stage is token g / RSEG of the stage, piece g % RSEG of its row.
    u32x4 rg[SPT];
    float rb = 0.0f;
    auto gload = [&](int st) __attribute__((always_inline)) {
        const int64_t tok0 = (tt0 + (int64_t)st * SB) * 32;
#pragma unroll
        for (int i = 0; i < SPT; ++i) {
            const int g = tid + i * kPsumThreads;
            int64_t t = tok0 + g / RSEG;
            t = t < T ? t : T - 1;  // rows past T: bias kNoToken below
            rg[i] = *reinterpret_cast<const u32x4*>(zhl + t * (2 * R) + 8 * (g % RSEG));
        }
        if (tid < SB * 32) {
            const int64_t t = tok0 + tid;
            const float v = bias[t < T ? t : T - 1];
            rb = t < T ? v : kNoToken;
        }
    };
    auto stash = [&](int buf) __attribute__((always_inline)) {
#pragma unroll
        for (int i = 0; i < SPT; ++i) {
            const int g = tid + i * kPsumThreads;
            *reinterpret_cast<u32x4*>(&zs[buf][(g / RSEG) * ROW + 8 * (g % RSEG)]) = rg[i];
        }
        if (tid < SB * 32) bs[buf][tid] = rb;
    };
    float pacc[NE];
#pragma unroll
    for (int j = 0; j < NE; ++j) pacc[j] = 0.0f;
    if (nstages > 0) {  // workgroup-uniform
        gload(0);
        stash(0);
        if (nstages > 1) gload(1);
        __syncthreads();
        for (int st = 0; st < nstages; ++st) {
            const int buf = st & 1;
            const int cnt = min(SB, ntiles - st * SB);
            if (active) {
#pragma unroll
                for (int tl = 0; tl < SB; ++tl) {
                    if (tl < cnt) {
                        const uint16_t* zr = &zs[buf][(tl * 32 + n) * ROW + 8 * half];
                        bf16x8 a[2 * RC];
#pragma unroll
                        for (int c = 0; c < 2 * RC; ++c) a[c] = load_bf16x8(zr + 16 * c);
                        f32x16 cin;
#pragma unroll
                        for (int q = 0; q < 4; ++q) {
                            const f32x4 v = *reinterpret_cast<const f32x4*>(
                                &bs[buf][tl * 32 + 8 * q + 4 * half]);
#pragma unroll
                            for (int p = 0; p < 4; ++p) cin[4 * q + p] = v[p];
                        }
                        f32x16 acc[NE];
#pragma unroll
                        for (int j = 0; j < NE; ++j) acc[j] = mfma_32x32x16(a[0], b[j][0], cin);
#pragma unroll
                        for (int c = 1; c < 2 * RC; ++c)
#pragma unroll
                            for (int j = 0; j < NE; ++j)
                                acc[j] = mfma_32x32x16(a[c], b[j][c % RC], acc[j]);
#pragma unroll
                        for (int j = 0; j < NE; ++j) {
                            float s = 0.0f;
#pragma unroll
                            for (int i = 0; i < 16; ++i) s += exp2_fast(acc[j][i]);
                            pacc[j] += s;
                        }
                    }
                }
            }
            if (st + 1 < nstages) stash(buf ^ 1);
            if (st + 2 < nstages) gload(st + 2);
            __syncthreads();
        }
    }
    // the two lane halves hold disjoint token rows of the same expert column
#pragma unroll
    for (int j = 0; j < NE; ++j) {
        const float tot = sum_pair32(pacc[j]);
        const int32_t e = 32 * (tile0 + j) + n;
        if (half == 0 && tile0 + j < Mt && e < M) part[(int64_t)split * M + e] = tot;
    }
}

// psum[e] = the split partials in order (0 when there are none).
__global__ __launch_bounds__(256) void stats_reduce_kernel(const float* __restrict__ part,
                                                           int32_t splits, int32_t G, int32_t M,
                                                           float* __restrict__ psum) {
    __shared__ float red[256];
    column_sums(part, splits, M, G, red, [&](int64_t e, float v) { psum[e] = v; });
}

// ------------------------------------------------------------------------------ host side
static size_t align256s(size_t b) { return (b + 255) & ~(size_t)255; }

// Threads per output of column_sums for P partials: about eight partials per thread, at most 16.
static int32_t sum_group(int64_t P) {
    int32_t G = 1;
    while (G < 16 && (int64_t)G * 8 < P) G *= 2;
    return G;
}

bool stats_make_plan(int64_t T, int32_t h, int32_t r, int32_t M, int32_t k, bool own_z,
                     StatsPlan* out) {
    if (T <= 0 || M <= 0 || (r != 16 && r != 32 && r != 64)) return false;
    StatsPlan q{};
    q.RC = r / 16;
    const int64_t Mt = ((int64_t)M + 31) / 32;
    // Z sweep: chunks that fit the LDS rows, about 256 workgroups in all
    const int64_t emax_tiles = (int64_t)kChunkBytes / (2 * r) / 32;
    const int64_t ntb = (T + kStatsTokens - 1) / kStatsTokens;
    int64_t C = (Mt + emax_tiles - 1) / emax_tiles;
    const int64_t want = (256 + ntb - 1) / ntb;
    if (C < want) C = want < Mt ? want : Mt;
    while ((Mt + C - 1) / C > emax_tiles) ++C;
    if (C > (1 << 20)) return false;
    q.chunks = (int32_t)C;
    int64_t S = 256 / C;
    if (S < 1) S = 1;
    if (S > ntb) S = ntb;
    q.splits = (int32_t)S;
    // psum sweep: expert blocks of 32 NE waves tiles, about 512 workgroups in all
    const int64_t Tt = (T + 31) / 32;
    const int64_t per_block = PsumCfg<1>::EXPERTS;  // the same for every rank
    const int64_t eb = (M + per_block - 1) / per_block;
    int64_t P = (512 + eb - 1) / eb;
    if (P > Tt) P = Tt;
    if (P < 1) P = 1;
    q.eblocks = (int32_t)eb;
    q.psplits = (int32_t)P;
    q.gz = sum_group(C);
    q.gp = sum_group(P);
    q.own_z = own_z ? 1 : 0;
    size_t o = 0;
    q.off_tv = o;
    o += align256s((size_t)T * k * sizeof(float));
    q.off_z = o;
    o += own_z ? align256s((size_t)T * r * sizeof(float)) : 0;
    q.off_zscratch = o;
    o += own_z ? align256s(zonly_workspace_bytes(T, h, r)) : 0;
    q.off_zhl = o;
    o += align256s((size_t)T * 2 * r * sizeof(uint16_t));
    q.off_mb = o;
    o += align256s((size_t)T * sizeof(float));
    q.off_Zp = o;
    o += align256s((size_t)C * T * sizeof(float));
    q.off_bias = o;
    o += align256s((size_t)T * sizeof(float));
    q.off_part = o;
    o += align256s((size_t)P * M * sizeof(float));
    q.workspace_bytes = o;
    *out = q;
    return true;
}

template <int RC>
static void launch_stats_sweeps(const StatsPlan& p, const StatsArgs& a, const uint16_t* zhl,
                                const float* mb, float* Zp, float* bias, float* part,
                                hipStream_t st) {
    hipLaunchKernelGGL((stats_z_kernel<RC>), dim3((unsigned)((int64_t)p.chunks * p.splits)),
                       dim3(kRouteThreads), 0, st, zhl, mb, a.R2t, a.T, a.M, p.chunks, p.splits,
                       Zp);
    const int64_t zper = 256 / p.gz;
    hipLaunchKernelGGL(stats_combine_kernel, dim3((unsigned)((a.T + zper - 1) / zper)), dim3(256),
                       0, st, Zp, p.chunks, p.gz, a.mtop, a.ks, mb, a.T, a.m, a.Z, bias);
    hipLaunchKernelGGL((stats_psum_kernel<RC>), dim3((unsigned)((int64_t)p.eblocks * p.psplits)),
                       dim3(kPsumThreads), 0, st, zhl, bias, a.R2t, a.T, a.M, p.eblocks,
                       p.psplits, part);
}

hipError_t stats_launch(const StatsPlan& p, const StatsArgs& a, void* workspace, hipStream_t st) {
    char* ws = static_cast<char*>(workspace);
    const float* z = a.z;
    if (p.own_z) {
        float* zown = reinterpret_cast<float*>(ws + p.off_z);
        const hipError_t e = zonly_launch(a.x, a.R1t, a.T, a.h, a.r, zown, ws + p.off_zscratch, st);
        if (e != hipSuccess) return e;
        z = zown;
    }
    uint16_t* zhl = reinterpret_cast<uint16_t*>(ws + p.off_zhl);
    float* mb = reinterpret_cast<float*>(ws + p.off_mb);
    float* Zp = reinterpret_cast<float*>(ws + p.off_Zp);
    float* bias = reinterpret_cast<float*>(ws + p.off_bias);
    float* part = reinterpret_cast<float*>(ws + p.off_part);
    const int64_t nz = (int64_t)a.T * a.r;
    hipLaunchKernelGGL(stats_prep_kernel, dim3((unsigned)((nz + 255) / 256)), dim3(256), 0, st, z,
                       a.mtop, a.ks, a.T, a.r, zhl, mb);
    switch (p.RC) {
        case 1: launch_stats_sweeps<1>(p, a, zhl, mb, Zp, bias, part, st); break;
        case 2: launch_stats_sweeps<2>(p, a, zhl, mb, Zp, bias, part, st); break;
        case 4: launch_stats_sweeps<4>(p, a, zhl, mb, Zp, bias, part, st); break;
        default: return hipErrorInvalidValue;
    }
    const int64_t pper = 256 / p.gp;
    hipLaunchKernelGGL(stats_reduce_kernel, dim3((unsigned)((a.M + pper - 1) / pper)), dim3(256), 0,
                       st, part, p.psplits, p.gp, a.M, a.psum);
    return hipGetLastError();
}

hipError_t stats_zero_psum(float* psum, int32_t M, hipStream_t st) {
    hipLaunchKernelGGL(stats_reduce_kernel, dim3((unsigned)((M + 255) / 256)), dim3(256), 0, st,
                       nullptr, 0, 1, M, psum);
    return hipGetLastError();
}

}  // namespace more
