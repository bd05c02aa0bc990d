// Wide low-rank route: softmax(TopK(x R1 R2)) (Section "Preliminaries") for the ranks of the
// paper's rank sweeps that the register-tiled routes do not hold (r a multiple of 16 up to 256,
// Section "Routing expressivity") and for 17 <= k <= 32.
//
// Three launches in sequence on the caller's stream:
//   1. z = x R1 in fp32, by the z pass of the other routes, run once per block of 64, 32 or 16
//      rank columns (a block's columns are independent rows of the contraction, so z is the
//      same as from one pass over all r columns);
//   2. z is split into three bfloat16 pieces per element whose sum is z exactly, stored as the
//      rows [z_hi | z_mid | z_lo] of a 3r-wide operand; when r is not a multiple of 64 the rows
//      of R2t are stacked three times into a matching [M][3r] operand, otherwise the sweep
//      reads each 64-wide chunk of R2t for all three pieces;
//   3. the fused standard router sweeps that pair: its fp32 logits are sums of exact bf16
//      products, i.e. the fp32 dot products of the fp32 z with the bfloat16 expert rows up to
//      the summation order, and it returns their exact top k (ties to the smaller id), the
//      softmax over the k and, optionally, the selected logits.
// The executed matrix work is three times the algorithmic z R2; the route trades that for
// kernels that keep every rank width and list length in registers without new tilings.
//
// Exactness of the split: z = m u with |m| < 2^24 (u the fp32 unit of z's binade).  z_hi =
// bf16(z) leaves z - z_hi = m1 u with |m1| <= 2^16, exact in fp32; z_mid = bf16(z - z_hi) leaves
// m2 u with |m2| <= 2^8, which one bfloat16 holds exactly.  (Magnitudes near the bottom of the
// fp32 range, below about 2^-110, could lose low bits to subnormal flushing; no logit of a
// bf16 router comes near it.)
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "wide.h"

namespace more {

namespace {

typedef uint32_t wide_u32x4 __attribute__((ext_vector_type(4)));

constexpr int kWideThreads = 256;
constexpr int64_t kWideMaxGrid = 1 << 20;

__device__ __forceinline__ uint16_t wide_bits(__bf16 v) { return __builtin_bit_cast(uint16_t, v); }

// z as written by the block passes: block b holds z[t][j0 + c] at zb[T j0 + t w + c].  Columns
// below n64 sit in 64-wide blocks, then one 32-wide block (when r mod 64 >= 32), then one
// 16-wide block (when r mod 32 == 16).
__global__ __launch_bounds__(kWideThreads) void wide_split_kernel(const float* __restrict__ zb,
                                                                  int64_t T, int32_t r,
                                                                  uint16_t* __restrict__ zs) {
    const int64_t n = T * r;
    const int32_t n64 = r / 64 * 64;
    const int32_t n32 = n64 + (r % 64 >= 32 ? 32 : 0);
    for (int64_t i = (int64_t)blockIdx.x * kWideThreads + threadIdx.x; i < n;
         i += (int64_t)gridDim.x * kWideThreads) {
        const int64_t t = i / r;
        const int32_t j = (int32_t)(i - t * r);
        const int32_t j0 = j < n64 ? (j & ~63) : (j < n32 ? n64 : n32);
        const int32_t w = j < n64 ? 64 : (j < n32 ? 32 : 16);
        const float v = zb[T * j0 + t * w + (j - j0)];
        const __bf16 a = (__bf16)v;
        const float r1 = v - (float)a;
        const __bf16 b = (__bf16)r1;
        const float r2 = r1 - (float)b;
        const __bf16 c = (__bf16)r2;
        uint16_t* row = zs + t * 3 * r;
        row[j] = wide_bits(a);
        row[r + j] = wide_bits(b);
        row[2 * r + j] = wide_bits(c);
    }
}

// W3[e] = [R2t[e] | R2t[e] | R2t[e]], copied in 16-byte pieces (r / 8 per row of R2t).
__global__ __launch_bounds__(kWideThreads) void wide_stack_kernel(const uint16_t* __restrict__ R2t,
                                                                  int32_t M, int32_t r,
                                                                  uint16_t* __restrict__ W3) {
    const int32_t pr = r / 8;
    const int64_t n = (int64_t)M * 3 * pr;
    for (int64_t i = (int64_t)blockIdx.x * kWideThreads + threadIdx.x; i < n;
         i += (int64_t)gridDim.x * kWideThreads) {
        const int64_t e = i / (3 * pr);
        const int32_t q = (int32_t)(i - e * 3 * pr);
        const wide_u32x4 v =
            *reinterpret_cast<const wide_u32x4*>(R2t + e * r + 8 * (q % pr));
        *reinterpret_cast<wide_u32x4*>(W3 + e * 3 * r + 8 * q) = v;
    }
}

size_t wide_align(size_t b) { return (b + 255) & ~(size_t)255; }

unsigned wide_grid(int64_t n) {
    const int64_t g = (n + kWideThreads - 1) / kWideThreads;
    return (unsigned)(g < 1 ? 1 : (g > kWideMaxGrid ? kWideMaxGrid : g));
}

}  // namespace

bool wide_route_needed(int32_t r, int32_t k) {
    return !(r == 16 || r == 32 || r == 64) || k > 16;
}

bool wide_make_plan(int64_t T, int32_t h, int32_t r, int32_t M, int32_t k, WidePlan* out) {
    if (T < 1 || h < 16 || h % 16 != 0 || r < 16 || r % 16 != 0 || r > kWideMaxRank || M < 1 ||
        k < 1 || k > M)
        return false;
    WidePlan q{};
    int32_t j = 0;
    size_t zscr = 0;
    while (j < r) {
        const int32_t left = r - j;
        const int32_t w = left >= 64 ? 64 : (left >= 32 ? 32 : 16);
        q.j0[q.nblocks] = j;
        q.w[q.nblocks] = w;
        ++q.nblocks;
        const size_t s = zonly_workspace_bytes(T, h, w);
        zscr = s > zscr ? s : zscr;
        j += w;
    }
    if (!fullrank_fused_make_plan(T, 3 * r, M, k, &q.ff)) return false;
    size_t o = 0;
    q.off_z = o;
    o += wide_align((size_t)T * r * sizeof(float));
    q.off_zscratch = o;
    o += wide_align(zscr);
    q.off_zs = o;
    o += wide_align((size_t)T * 3 * r * sizeof(uint16_t));
    q.stack = r % 64 != 0;
    q.off_w3 = o;
    if (q.stack) o += wide_align((size_t)M * 3 * r * sizeof(uint16_t));
    q.off_ff = o;
    o += wide_align(q.ff.workspace_bytes);
    q.workspace_bytes = o;
    *out = q;
    return true;
}

hipError_t wide_launch(const WidePlan& p, const uint16_t* x, const uint16_t* R1t,
                       const uint16_t* R2t, int64_t T, int32_t h, int32_t r, int32_t M, int32_t k,
                       int32_t* idx, float* gate, float* topval, void* workspace,
                       hipStream_t st) {
    char* ws = static_cast<char*>(workspace);
    float* z = reinterpret_cast<float*>(ws + p.off_z);
    for (int32_t b = 0; b < p.nblocks; ++b) {
        const hipError_t e = zonly_launch(x, R1t + (int64_t)p.j0[b] * h, T, h, p.w[b],
                                          z + T * p.j0[b], ws + p.off_zscratch, st);
        if (e != hipSuccess) return e;
    }
    uint16_t* zs = reinterpret_cast<uint16_t*>(ws + p.off_zs);
    uint16_t* w3 = reinterpret_cast<uint16_t*>(ws + p.off_w3);
    hipLaunchKernelGGL(wide_split_kernel, dim3(wide_grid(T * r)), dim3(kWideThreads), 0, st, z,
                       T, r, zs);
    void* ffws = p.ff.workspace_bytes > 0 ? ws + p.off_ff : nullptr;
    if (!p.stack)  // r a multiple of 64: the three pieces read the one copy of R2t
        return fullrank_fused_launch_periodic(p.ff, zs, R2t, r, T, 3 * r, M, k, idx, gate,
                                              topval, ffws, st);
    hipLaunchKernelGGL(wide_stack_kernel, dim3(wide_grid((int64_t)M * 3 * (r / 8))),
                       dim3(kWideThreads), 0, st, R2t, M, r, w3);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    return fullrank_fused_launch(p.ff, zs, w3, T, 3 * r, M, k, idx, gate, topval, ffws, st);
}

}  // namespace more
