// Fused standard router: softmax(TopK(x W)) without writing the T x M logits (the fused standard
// MoE router of the efficiency appendix, "Fusing a standard MoE layer": the low-rank router's
// fusion with the rank replaced by the hidden size h).  The stronger full-rank baseline on
// small hidden sizes; the paper finds the benefit of the fusion vanishing as h grows, since the
// weight tile is re-read for every token block.
//
// One workgroup of 8 waves owns 32 NT tokens, whose rows of x stay in LDS for the whole call,
// and a range of expert tiles (the expert axis split over esplits workgroups per token block);
// wave w takes a contiguous share of the range.  Per expert tile of 32 rows of Wt the wave runs
// the h contraction on the matrix cores (v_mfma_f32_32x32x16_bf16, experts on the A rows, tokens
// on the B columns; products of bf16 values are exact and the sum is fp32), so the accumulators
// hold the final fp32 logits, and each lane folds its sixteen logits of a token into a sorted
// register list of K (largest first; a strict > keeps the smaller id on equal logits, since a
// lane visits its experts in increasing order).  At the end the two lane halves, then the eight
// waves (through LDS) merge their lists; with one split the workgroup applies the softmax and
// stores, otherwise the lists of the splits are merged by fullrank_merge_kernel.
//
// h order within a 64-wide chunk.  MFMA step s of chunk c takes h values c 64 + 8 s + 0..7 from
// lane half 0 and c 64 + 32 + 8 s + 0..7 from lane half 1 (the same order for both operands), so
// a lane reads its 32 h values of a row of Wt as one contiguous 64-byte piece per chunk.  The x
// rows in LDS are zero from h up to the next multiple of 64, so a partial last chunk needs no
// special path.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "device_common.h"
#include "lowrank.h"
#include "route_device.h"
#include "wide.h"

namespace more {

constexpr int kFfWaves = 8;
constexpr int kFfThreads = 64 * kFfWaves;
constexpr int kFfLdsBytes = 136 * 1024;  // the x rows of a token block (row stride h + 8)
constexpr int kFfRing = 3;               // chunks of Wt rows in flight per wave

template <int NT, int K>
__global__ __launch_bounds__(kFfThreads, 1) void fullrank_fused_kernel(
    const uint16_t* __restrict__ x, const uint16_t* __restrict__ Wt, int32_t ldw, int32_t wmod,
    int32_t T, int32_t h, int32_t M, int32_t k, int32_t esplits, float* __restrict__ pv,
    int32_t* __restrict__ pi, int32_t* __restrict__ idx, float* __restrict__ gate,
    float* __restrict__ topval) {
    // Row e of the weights starts at Wt + e ldw and chunk c of the contraction reads its chunk
    // c mod wmod: ldw = h and wmod = the chunk count for a plain [M][h] matrix; with ldw = h / p
    // (a multiple of 64) and wmod = ldw / 64 the p chunk groups of x meet the same stored row
    // (the wide route's three pieces of z against one copy of R2).
    constexpr int BT = 32 * NT;
    static_assert(kFfWaves * BT * K * 8 <= kFfLdsBytes, "merge lists fit the LDS block");
    __shared__ __attribute__((aligned(16))) uint16_t xs[kFfLdsBytes / 2];
    const int HP = (h + 63) & ~63;  // h rounded up to whole 64-wide chunks (zero-padded in LDS)
    const int XS = HP + 8;          // bf16 per LDS row: 16-byte pad spreads 16 rows over the banks
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int n = lane & 31, half = lane >> 5;
    const int64_t tb = blockIdx.x / (unsigned)esplits;
    const int es = (int)(blockIdx.x % (unsigned)esplits);
    const int64_t tok0 = tb * BT;
    // x rows tok0 .. tok0 + BT - 1 into LDS (rows past T re-read row T - 1; never stored), zeros
    // from h up to HP
    {
        const int spr = HP >> 3;  // 16-byte pieces per padded row
        const int nseg = BT * spr;
        for (int base = 0; base < nseg; base += 8 * kFfThreads) {
            u32x4 v[8];
#pragma unroll
            for (int u = 0; u < 8; ++u) {
                int seg = base + u * kFfThreads + tid;
                seg = seg < nseg ? seg : nseg - 1;
                const int row = seg / spr, col = seg - (seg / spr) * spr;
                int64_t t = tok0 + row;
                t = t < T ? t : T - 1;
                const int cc = 8 * col < h ? col : 0;
                const u32x4 ld = *reinterpret_cast<const u32x4*>(x + t * h + 8 * cc);
                v[u] = 8 * col < h ? ld : u32x4{0u, 0u, 0u, 0u};
            }
#pragma unroll
            for (int u = 0; u < 8; ++u) {
                const int seg = base + u * kFfThreads + tid;
                if (seg < nseg) {
                    const int row = seg / spr, col = seg - (seg / spr) * spr;
                    *reinterpret_cast<u32x4*>(&xs[row * XS + 8 * col]) = v[u];
                }
            }
        }
    }
    __syncthreads();

    const int32_t Mt = (M + 31) / 32;
    const int32_t et0 = (int32_t)((int64_t)Mt * es / esplits);
    const int32_t et1 = (int32_t)((int64_t)Mt * (es + 1) / esplits);
    const int32_t wt0 = et0 + (int32_t)((int64_t)(et1 - et0) * w / kFfWaves);
    const int32_t wt1 = et0 + (int32_t)((int64_t)(et1 - et0) * (w + 1) / kFfWaves);
    const int nch = HP >> 6;  // 64-wide chunks; pieces at or past h read x as zero
    float lv[NT][K];
    int32_t li[NT][K];
#pragma unroll
    for (int g = 0; g < NT; ++g) list_init<K>(lv[g], li[g]);
    const uint16_t* xb = &xs[n * XS + 32 * half];  // token n of tile 0, the lane's h half
    // The wave's 64-wide chunks, numbered q = (tile - wt0) nch + c, stream through a ring of
    // kFfRing register slots: slot q mod kFfRing is refilled with chunk q + kFfRing as soon as chunk
    // q's MFMAs are issued, so each load has kFfRing - 1 chunks of MFMAs to arrive.  Every load is
    // unconditional (loads past the wave's last chunk re-read it; pieces at or past h re-read the
    // row's first piece, which meets zeros of x), and the steady-state loop has no load on a
    // conditional path, so the compiler's wait counts stay exact across the loop.
    const int Q = (wt1 - wt0) * nch;
    auto loadq = [&](int q, u32x4 (&a)[4]) __attribute__((always_inline)) {
        q = q < Q ? q : Q - 1;
        const int32_t tile = wt0 + q / nch;
        const int c = q - (q / nch) * nch;
        const int cw = c - (c / wmod) * wmod;  // the stored chunk
        int32_t e = tile * 32 + n;
        e = e < M ? e : M - 1;  // rows past M: copies of row M - 1, masked in the epilogue
        const uint16_t* rowp = Wt + (int64_t)e * ldw;
#pragma unroll
        for (int s = 0; s < 4; ++s) {
            int off = 64 * cw + 32 * half + 8 * s;
            off = off < ldw ? off : 0;
            a[s] = *reinterpret_cast<const u32x4*>(rowp + off);
        }
    };
    f32x16 acc[NT];
#pragma unroll
    for (int g = 0; g < NT; ++g) acc[g] = zero_f32x16();
    // the list update of a finished tile; acc is cleared for the next one
    auto finish_tile = [&](int32_t tile) __attribute__((always_inline)) {
        if (tile == Mt - 1) {  // rows past M out
#pragma unroll
            for (int g = 0; g < NT; ++g)
#pragma unroll
                for (int i = 0; i < 16; ++i)
                    if (tile * 32 + acc_row(i, half) >= M) acc[g][i] = -__builtin_huge_valf();
        }
        if (tile == wt0) {  // empty lists: every logit goes in (no lane idles)
#pragma unroll
            for (int g = 0; g < NT; ++g)
#pragma unroll
                for (int i = 0; i < 16; ++i)
                    if (acc[g][i] > lv[g][K - 1])
                        list_insert_newer<K>(lv[g], li[g], acc[g][i], tile * 32 + acc_row(i, half));
        } else {
            // Later tiles: a lane's logits above its K-th form a 16-bit mask, inserted one per
            // round in increasing id order, so the wave runs as many rounds as its busiest lane
            // has hits (a few per tile once the lists hold the larger logits) instead of a
            // masked insertion per element.
#pragma unroll
            for (int g = 0; g < NT; ++g) {
                const float th = lv[g][K - 1];
                uint32_t m = 0;
#pragma unroll
                for (int i = 0; i < 16; ++i) m |= (acc[g][i] > th ? 1u : 0u) << i;
                while (m) {
                    const int i = __builtin_ctz(m);
                    m &= m - 1;
                    float v = acc[g][0];
#pragma unroll
                    for (int j = 1; j < 16; ++j) v = i == j ? acc[g][j] : v;
                    if (v > lv[g][K - 1])
                        list_insert_newer<K>(lv[g], li[g], v,
                                             tile * 32 + 8 * (i >> 2) + 4 * half + (i & 3));
                }
            }
        }
#pragma unroll
        for (int g = 0; g < NT; ++g) acc[g] = zero_f32x16();
    };
    auto chunk = [&](auto slot, int q, u32x4 (&a)[4]) __attribute__((always_inline)) {
        (void)slot;
        const int c = q - (q / nch) * nch;
#pragma unroll
        for (int s = 0; s < 4; ++s) {
            const bf16x8 av = __builtin_bit_cast(bf16x8, a[s]);
#pragma unroll
            for (int g = 0; g < NT; ++g)
                acc[g] = mfma_32x32x16(av, load_bf16x8(xb + g * 32 * XS + 64 * c + 8 * s), acc[g]);
        }
        loadq(q + kFfRing, a);
        if (c == nch - 1) finish_tile(wt0 + q / nch);
    };
    if (Q > 0) {  // wave-uniform
        u32x4 ring[kFfRing][4];
        unroll<kFfRing>([&](auto ss) __attribute__((always_inline)) {
            loadq(decltype(ss)::value, ring[decltype(ss)::value]);
        });
        int q0 = 0;
        for (; q0 + kFfRing <= Q; q0 += kFfRing)
            unroll<kFfRing>([&](auto ss) __attribute__((always_inline)) {
                chunk(ss, q0 + decltype(ss)::value, ring[decltype(ss)::value]);
            });
        unroll<kFfRing>([&](auto ss) __attribute__((always_inline)) {
            if (q0 + decltype(ss)::value < Q)
                chunk(ss, q0 + decltype(ss)::value, ring[decltype(ss)::value]);
        });
    }
    // lanes n and n + 32 hold disjoint expert rows of the same tokens
#pragma unroll
    for (int g = 0; g < NT; ++g) list_merge_xor<32, K>(lv[g], li[g]);
    __syncthreads();  // the x rows are no longer read: the LDS block takes the waves' lists
    float* sv = reinterpret_cast<float*>(xs);
    int32_t* si = reinterpret_cast<int32_t*>(xs) + kFfWaves * BT * K;
    if (half == 0) {
#pragma unroll
        for (int g = 0; g < NT; ++g)
#pragma unroll
            for (int j = 0; j < K; ++j) {
                sv[(w * BT + 32 * g + n) * K + j] = lv[g][j];
                si[(w * BT + 32 * g + n) * K + j] = li[g][j];
            }
    }
    __syncthreads();
    if (tid < BT) {
        float v[K], bv[K];
        int32_t vi[K], bi[K];
#pragma unroll
        for (int j = 0; j < K; ++j) {
            v[j] = sv[tid * K + j];
            vi[j] = si[tid * K + j];
        }
        for (int ww = 1; ww < kFfWaves; ++ww) {
#pragma unroll
            for (int j = 0; j < K; ++j) {
                bv[j] = sv[(ww * BT + tid) * K + j];
                bi[j] = si[(ww * BT + tid) * K + j];
            }
            list_merge<K>(v, vi, bv, bi);
        }
        const int64_t t = tok0 + tid;
        if (t < T) {
            if (esplits == 1) {
                store_selection<K>(v, vi, k, t, idx, gate, topval);
            } else {
                float* ov = pv + ((int64_t)es * T + t) * K;
                int32_t* oi = pi + ((int64_t)es * T + t) * K;
#pragma unroll
                for (int j = 0; j < K; ++j) {
                    ov[j] = v[j];
                    oi[j] = vi[j];
                }
            }
        }
    }
}

// The lists of the expert splits of each token merged in split order, then softmax and store.
template <int K>
__global__ __launch_bounds__(256) void fullrank_merge_kernel(const float* __restrict__ pv,
                                                             const int32_t* __restrict__ pi,
                                                             int32_t T, int32_t k, int32_t esplits,
                                                             int32_t* __restrict__ idx,
                                                             float* __restrict__ gate,
                                                             float* __restrict__ topval) {
    const int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (t >= T) return;
    float v[K], bv[K];
    int32_t vi[K], bi[K];
#pragma unroll
    for (int j = 0; j < K; ++j) {
        v[j] = pv[t * K + j];
        vi[j] = pi[t * K + j];
    }
    for (int s = 1; s < esplits; ++s) {
#pragma unroll
        for (int j = 0; j < K; ++j) {
            bv[j] = pv[((int64_t)s * T + t) * K + j];
            bi[j] = pi[((int64_t)s * T + t) * K + j];
        }
        list_merge<K>(v, vi, bv, bi);
    }
    store_selection<K>(v, vi, k, t, idx, gate, topval);
}

// ------------------------------------------------------------------------------ host side
static int ff_pow2(int k) {
    int K = 1;
    while (K < k) K <<= 1;
    return K;
}

bool fullrank_fused_make_plan(int64_t T, int32_t h, int32_t M, int32_t k, FusedFullrankPlan* p) {
    FusedFullrankPlan q{};
    q.K = ff_pow2(k);
    // token tiles per workgroup: the x rows fit the LDS block and the lists (NT K pairs per lane)
    // stay at most 16, or 32 with one tile (more spilled registers: 76 bytes per lane at
    // NT = 4, K = 8, for no gain in speed)
    const int64_t xs_row = (((int64_t)h + 63) & ~(int64_t)63) + 8;  // bf16 per LDS row
    int NT = 4;
    while (NT > 1 && (32 * NT * xs_row * 2 > kFfLdsBytes || NT * q.K > 16)) NT >>= 1;
    if (32 * NT * xs_row * 2 > kFfLdsBytes || NT * q.K > 32) return false;
    // Expert splits give each wave at least 16 tiles (fewer leave the register lists filling up
    // for most of the sweep, where almost every logit is inserted); narrower token blocks then
    // bring the grid to 256 workgroups (one per CU) where the tokens allow.
    const int64_t Mt = ((int64_t)M + 31) / 32;
    const int64_t es_max = Mt / (kFfWaves * 16) > 1 ? Mt / (kFfWaves * 16) : 1;
    int64_t es = 1;
    for (;; NT >>= 1) {
        const int64_t nb = (T + 32 * NT - 1) / (32 * NT);
        es = (256 + nb - 1) / nb;
        if (es > es_max) es = es_max;
        if (es > 1024) es = 1024;
        if (nb * es >= 256 || NT == 1) break;
    }
    q.NT = NT;
    q.esplits = (int32_t)es;
    q.workspace_bytes = es > 1 ? (size_t)es * T * q.K * 8 : 0;
    *p = q;
    return true;
}

template <int NT, int K>
static void launch_ff(const FusedFullrankPlan& p, const uint16_t* x, const uint16_t* Wt,
                      int32_t ldw, int32_t wmod, int64_t T, int32_t h, int32_t M, int32_t k,
                      int32_t* idx, float* gate, float* topval, void* ws, hipStream_t st) {
    const int64_t nb = (T + 32 * NT - 1) / (32 * NT);
    float* pv = static_cast<float*>(ws);
    int32_t* pi = p.esplits > 1 ? reinterpret_cast<int32_t*>(pv + (int64_t)p.esplits * T * K)
                                : nullptr;
    hipLaunchKernelGGL((fullrank_fused_kernel<NT, K>), dim3((unsigned)(nb * p.esplits)),
                       dim3(kFfThreads), 0, st, x, Wt, ldw, wmod, (int32_t)T, h, M, k,
                       p.esplits, pv, pi, idx, gate, topval);
    if (p.esplits > 1)
        hipLaunchKernelGGL((fullrank_merge_kernel<K>), dim3((unsigned)((T + 255) / 256)),
                           dim3(256), 0, st, pv, pi, (int32_t)T, k, p.esplits, idx, gate, topval);
}

static hipError_t launch_ff_any(const FusedFullrankPlan& p, const uint16_t* x,
                                const uint16_t* Wt, int32_t ldw, int32_t wmod, int64_t T,
                                int32_t h, int32_t M, int32_t k, int32_t* idx, float* gate,
                                float* topval, void* workspace, hipStream_t st) {
#define MORE_FF(NT_, K_)                                                                   \
    if (p.NT == NT_ && p.K == K_) {                                                        \
        launch_ff<NT_, K_>(p, x, Wt, ldw, wmod, T, h, M, k, idx, gate, topval, workspace, st); \
        return hipGetLastError();                                                          \
    }
    MORE_FF(4, 1) MORE_FF(4, 2) MORE_FF(4, 4)
    MORE_FF(2, 1) MORE_FF(2, 2) MORE_FF(2, 4) MORE_FF(2, 8)
    MORE_FF(1, 1) MORE_FF(1, 2) MORE_FF(1, 4) MORE_FF(1, 8) MORE_FF(1, 16) MORE_FF(1, 32)
#undef MORE_FF
    return hipErrorInvalidValue;
}

hipError_t fullrank_fused_launch(const FusedFullrankPlan& p, const uint16_t* x, const uint16_t* Wt,
                                 int64_t T, int32_t h, int32_t M, int32_t k, int32_t* idx,
                                 float* gate, float* topval, void* workspace, hipStream_t st) {
    return launch_ff_any(p, x, Wt, h, (h + 63) / 64, T, h, M, k, idx, gate, topval, workspace,
                         st);
}

hipError_t fullrank_fused_launch_periodic(const FusedFullrankPlan& p, const uint16_t* x,
                                          const uint16_t* Wt, int32_t ldw, int64_t T, int32_t h,
                                          int32_t M, int32_t k, int32_t* idx, float* gate,
                                          float* topval, void* workspace, hipStream_t st) {
    if (ldw < 64 || ldw % 64 != 0 || h % ldw != 0) return hipErrorInvalidValue;
    return launch_ff_any(p, x, Wt, ldw, ldw / 64, T, h, M, k, idx, gate, topval, workspace, st);
}

}  // namespace more
