// Device helpers shared by the router kernels (gfx950 only).
//
// Contents: operand vector types and 16-byte loads, the 32x32x16 bf16 MFMA, the fp32 ->
// bf16 hi/lo split used to carry z into the expert contraction, and the per-lane
// register top-K list with its total order (larger logit first, then smaller expert id).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace more {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef int32_t i32x4 __attribute__((ext_vector_type(4)));

constexpr int kWave = 64;

__device__ __forceinline__ bf16x8 load_bf16x8(const uint16_t* p) {
    return __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>(p));
}

__device__ __forceinline__ bf16x8 zero_bf16x8() {
    return __builtin_bit_cast(bf16x8, u32x4{0u, 0u, 0u, 0u});
}

__device__ __forceinline__ f32x16 zero_f32x16() {
    f32x16 z;
#pragma unroll
    for (int i = 0; i < 16; ++i) z[i] = 0.0f;
    return z;
}

// D = A (32 x 16) * B (16 x 32) + C, fp32 accumulate.  Lane l supplies A row (l % 32) and B
// column (l % 32), eight consecutive K values each, K half (l / 32); lane l receives
// C[8j + 4(l/32) + i][l % 32] in element 4j + i (j, i = 0..3).
__device__ __forceinline__ f32x16 mfma_32x32x16(bf16x8 a, bf16x8 b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

// Row of the 32x32 accumulator tile held in element `e` by a lane in K half `half`.
__device__ __forceinline__ constexpr int acc_row(int e, int half) {
    return 8 * (e >> 2) + 4 * half + (e & 3);
}

// fp32 -> bfloat16 bits, round to nearest even (finite inputs).
__device__ __forceinline__ uint32_t f32_to_bf16_bits(float f) {
    uint32_t u = __builtin_bit_cast(uint32_t, f);
    return (u + 0x7FFFu + ((u >> 16) & 1u)) >> 16;
}

__device__ __forceinline__ float bf16_bits_to_f32(uint32_t b) {
    return __builtin_bit_cast(float, b << 16);
}

// Split eight fp32 values into bf16 hi = bf16(z) and lo = bf16(z - hi), both rounded to
// nearest even (v_cvt_pk_bf16_f32).  z - hi is exact in fp32, so hi + lo carries about 16
// significant bits of z.
__device__ __forceinline__ void split_hi_lo(const float (&z)[8], bf16x8& hi, bf16x8& lo) {
#pragma unroll
    for (int q = 0; q < 8; ++q) {
        const __bf16 h = (__bf16)z[q];
        hi[q] = h;
        lo[q] = (__bf16)(z[q] - (float)h);
    }
}

// ---------------------------------------------------------------- top-K lists
// A list holds K (value, expert) pairs sorted by the selection order.  Empty slots hold
// (-inf, INT32_MAX), which every real candidate beats.
constexpr int32_t kNoExpert = 0x7FFFFFFF;

__device__ __forceinline__ bool better(float av, int32_t ai, float bv, int32_t bi) {
    return av > bv || (av == bv && ai < bi);
}

template <int K>
__device__ __forceinline__ void list_init(float (&v)[K], int32_t (&ix)[K]) {
#pragma unroll
    for (int j = 0; j < K; ++j) {
        v[j] = -__builtin_huge_valf();
        ix[j] = kNoExpert;
    }
}

// Insert a candidate whose expert id is larger than every id already in the list (a lane
// visits its experts in increasing order): it goes after every entry with a value at least its
// own (a strict value compare), and the entries after it shift down by one in their order (an
// entry carried down is never compared again: with equal values it must stay ahead of the
// entries it was ahead of).  The last pair falls off the end.
template <int K>
__device__ __forceinline__ void list_insert_newer(float (&v)[K], int32_t (&ix)[K], float nv,
                                                  int32_t ni) {
    bool placed = false;
#pragma unroll
    for (int j = 0; j < K; ++j) {
        const bool b = placed || nv > v[j];
        float tv = v[j];
        int32_t ti = ix[j];
        v[j] = b ? nv : tv;
        ix[j] = b ? ni : ti;
        nv = b ? tv : nv;
        ni = b ? ti : ni;
        placed = b;
    }
}

// Insert any candidate (general position in the selection order); the last pair falls off.
template <int K>
__device__ __forceinline__ void list_insert(float (&v)[K], int32_t (&ix)[K], float nv, int32_t ni) {
#pragma unroll
    for (int j = 0; j < K; ++j) {
        bool b = better(nv, ni, v[j], ix[j]);
        float tv = v[j];
        int32_t ti = ix[j];
        v[j] = b ? nv : tv;
        ix[j] = b ? ni : ti;
        nv = b ? tv : nv;
        ni = b ? ti : ni;
    }
}

// (av, ai) <- the best K of (av, ai) and (bv, bi), both sorted; result sorted.
// First half-cleaner against the reversed partner, then a bitonic merge network.
template <int K>
__device__ __forceinline__ void list_merge(float (&av)[K], int32_t (&ai)[K], const float (&bv)[K],
                                           const int32_t (&bi)[K]) {
#pragma unroll
    for (int j = 0; j < K; ++j) {
        float ov = bv[K - 1 - j];
        int32_t oi = bi[K - 1 - j];
        bool b = better(ov, oi, av[j], ai[j]);
        av[j] = b ? ov : av[j];
        ai[j] = b ? oi : ai[j];
    }
#pragma unroll
    for (int s = K / 2; s >= 1; s >>= 1) {
#pragma unroll
        for (int j = 0; j < K; ++j) {
            if ((j & s) == 0) {
                bool b = better(av[j + s], ai[j + s], av[j], ai[j]);
                float tv = av[j];
                int32_t ti = ai[j];
                av[j] = b ? av[j + s] : tv;
                ai[j] = b ? ai[j + s] : ti;
                av[j + s] = b ? tv : av[j + s];
                ai[j + s] = b ? ti : ai[j + s];
            }
        }
    }
}

// ---------------------------------------------------------------- cross-lane moves
// The value of x held by lane (lane ^ M).  M = 1 and 2 are DPP quad permutations, M = 4 a
// half-row mirror followed by a quad reversal (lane i of an 8-lane group reads 7 - (i ^ 3) =
// i ^ 4); these stay in the VALU instead of going through the LDS crossbar of a general
// shuffle.  Other M use __shfl_xor.
template <int M, typename T>
__device__ __forceinline__ T lane_xor(T x) {
    static_assert(sizeof(T) == 4, "32-bit values only");
    const int v = __builtin_bit_cast(int, x);
    int r;
    if constexpr (M == 1) {
        r = __builtin_amdgcn_mov_dpp(v, 0xB1, 0xF, 0xF, false);  // quad_perm [1,0,3,2]
    } else if constexpr (M == 2) {
        r = __builtin_amdgcn_mov_dpp(v, 0x4E, 0xF, 0xF, false);  // quad_perm [2,3,0,1]
    } else if constexpr (M == 4) {
        const int h = __builtin_amdgcn_mov_dpp(v, 0x141, 0xF, 0xF, false);  // row_half_mirror
        r = __builtin_amdgcn_mov_dpp(h, 0x1B, 0xF, 0xF, false);             // quad_perm [3,2,1,0]
    } else {
        r = __shfl_xor(v, M, kWave);
    }
    return __builtin_bit_cast(T, r);
}

// The values of x in lane l and in lane l ^ 32, in some order (both lanes of a pair get the
// same two values): one gfx950 permlane32 swap, for symmetric combinations (sums, merges).
__device__ __forceinline__ void lane_pair32(float x, float& a, float& b) {
    const unsigned v = __builtin_bit_cast(unsigned, x);
    const auto r = __builtin_amdgcn_permlane32_swap(v, v, false, false);
    a = __builtin_bit_cast(float, (unsigned)r[0]);
    b = __builtin_bit_cast(float, (unsigned)r[1]);
}

// x plus its value in lane l ^ 32.
__device__ __forceinline__ float sum_pair32(float x) {
    float a, b;
    lane_pair32(x, a, b);
    return a + b;
}

// Merge with the list held by lane (lane ^ M) of the same wave.
template <int M, int K>
__device__ __forceinline__ void list_merge_xor(float (&v)[K], int32_t (&ix)[K]) {
    float pv[K];
    int32_t pi[K];
#pragma unroll
    for (int j = 0; j < K; ++j) {
        pv[j] = lane_xor<M>(v[j]);
        pi[j] = lane_xor<M>(ix[j]);
    }
    list_merge<K>(v, ix, pv, pi);
}

// softmax over the first k entries of a sorted list, then store idx / gate / topval row.
template <int K>
__device__ __forceinline__ void store_selection(const float (&v)[K], const int32_t (&ix)[K], int k,
                                                int64_t token, int32_t* __restrict__ idx,
                                                float* __restrict__ gate,
                                                float* __restrict__ topval) {
    float e[K];
    float sum = 0.0f;
#pragma unroll
    for (int j = 0; j < K; ++j) {
        e[j] = (j < k) ? expf(v[j] - v[0]) : 0.0f;
        sum += e[j];
    }
    const int64_t base = token * k;
#pragma unroll
    for (int j = 0; j < K; ++j) {
        if (j < k) {
            idx[base + j] = ix[j];
            gate[base + j] = e[j] / sum;
            if (topval) topval[base + j] = v[j];
        }
    }
}

}  // namespace more
