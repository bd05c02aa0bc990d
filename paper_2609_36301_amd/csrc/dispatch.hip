// Dispatch bookkeeping of an MoE layer ("Sort + Count" in the layer's forward-pass figure of the
// efficiency appendix): the N = T k expert ids of a routing result become the positions
// p = t k + j grouped by expert (ascending p within an expert, ids outside [0, M) last) and the
// per-expert offsets.
//
// A least-significant-digit radix sort on the key (expert id, or M for an id outside [0, M)),
// 8 bits per pass, each pass stable, so that equal keys keep their position order:
//   dsort_hist_kernel     per block of 1024 entries, the count of each digit value;
//   dsort_scan_kernel     one workgroup per digit value: the exclusive scan of that digit's
//                         block counts, and the digit's total;
//   dsort_scatter_kernel  each entry's rank among the block's earlier entries with its digit
//                         (wave ballots within a wave, then counts of the earlier waves and
//                         rounds), added to its (digit, block) start: the totals of the smaller
//                         digits (a 256-wide scan in LDS) plus the digit's block prefix.
// dsort_offsets_kernel derives offsets from the sorted keys: offsets[e] = the first slot whose
// key is at least e.  Up to 4096 entries (decode-sized batches) one workgroup runs all passes in
// LDS instead (dsort_small_kernel); with at most 8191 experts one counting pass replaces the
// radix passes (dsort_whist, dsort_wscan, dsort_wscatter).
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "lowrank.h"

namespace more {

constexpr int kDsThreads = 256;
constexpr int kDsRounds = 4;                          // entries per thread and block
constexpr int kDsBlock = kDsThreads * kDsRounds;      // 1024 entries per block
constexpr int kDsDigits = 256;                        // 8-bit digits
constexpr int kDsGroups = kDsRounds * (kDsThreads / 64);  // (round, wave) groups in entry order

__device__ __forceinline__ int32_t ds_key(int32_t e, int32_t M) {
    return (e >= 0 && e < M) ? e : M;
}

// Digit counts of block b: hist[d * nblocks + b].  Pass 0 reads the keys from idx.
__global__ __launch_bounds__(kDsThreads) void dsort_hist_kernel(const int32_t* __restrict__ idx,
                                                                const int32_t* __restrict__ keys,
                                                                int64_t N, int32_t M, int shift,
                                                                int32_t* __restrict__ hist) {
    __shared__ int32_t cnt[kDsDigits];
    const int tid = threadIdx.x;
    cnt[tid] = 0;
    __syncthreads();
    const int64_t b0 = (int64_t)blockIdx.x * kDsBlock;
    for (int r = 0; r < kDsRounds; ++r) {
        const int64_t g = b0 + r * kDsThreads + tid;
        if (g < N) {
            const int32_t key = idx ? ds_key(idx[g], M) : keys[g];
            atomicAdd(&cnt[(key >> shift) & (kDsDigits - 1)], 1);
        }
    }
    __syncthreads();
    hist[(int64_t)tid * gridDim.x + blockIdx.x] = cnt[tid];
}

// Workgroup d: in-place exclusive scan of hist[d][0 .. nb) (the digit's block counts, in
// tiles of 1024, four consecutive counts per thread) and total[d], the digit's entry count.
__global__ __launch_bounds__(kDsThreads) void dsort_scan_kernel(int32_t* __restrict__ hist,
                                                                int64_t nb,
                                                                int32_t* __restrict__ total) {
    __shared__ int32_t part[kDsThreads];
    const int tid = threadIdx.x;
    int32_t* a = hist + (int64_t)blockIdx.x * nb;
    int32_t carry = 0;
    for (int64_t t0 = 0; t0 < nb; t0 += 4 * kDsThreads) {
        int32_t v[4];
        int32_t sum = 0;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int64_t j = t0 + 4 * tid + i;
            v[i] = j < nb ? a[j] : 0;
            sum += v[i];
        }
        part[tid] = sum;
        __syncthreads();
        for (int d = 1; d < kDsThreads; d <<= 1) {  // inclusive scan of the threads' sums
            const int32_t u = tid >= d ? part[tid - d] : 0;
            __syncthreads();
            part[tid] += u;
            __syncthreads();
        }
        int32_t run = carry + part[tid] - sum;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int64_t j = t0 + 4 * tid + i;
            if (j < nb) a[j] = run;
            run += v[i];
        }
        carry += part[kDsThreads - 1];
        __syncthreads();  // part is rewritten by the next tile
    }
    if (tid == 0) total[blockIdx.x] = carry;
}

// Stable scatter of one pass.  Entry g = b0 + r 256 + tid of block b belongs to group
// (r, wave); groups are in entry order, lanes within a group too.  keys_out may be null (not
// needed after the last pass); pass 0 reads keys from idx and takes the position as value.
__global__ __launch_bounds__(kDsThreads) void dsort_scatter_kernel(
    const int32_t* __restrict__ idx, const int32_t* __restrict__ keys_in,
    const int32_t* __restrict__ vals_in, int64_t N, int32_t M, int shift,
    const int32_t* __restrict__ start, const int32_t* __restrict__ total,
    int32_t* __restrict__ keys_out, int32_t* __restrict__ vals_out) {
    __shared__ int32_t cnt[kDsGroups][kDsDigits];  // count per group, then the group's offset
    __shared__ int32_t base[kDsDigits];            // entries of the smaller digits
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    for (int i = tid; i < kDsGroups * kDsDigits; i += kDsThreads) (&cnt[0][0])[i] = 0;
    base[tid] = total[tid];
    __syncthreads();
    for (int d = 1; d < kDsDigits; d <<= 1) {  // inclusive scan of the digit totals
        const int32_t u = tid >= d ? base[tid - d] : 0;
        __syncthreads();
        base[tid] += u;
        __syncthreads();
    }
    const int32_t mybase = base[tid] - total[tid];  // exclusive, digit tid
    __syncthreads();
    base[tid] = mybase;
    __syncthreads();
    const int64_t b0 = (int64_t)blockIdx.x * kDsBlock;
    const uint64_t below = (1ull << lane) - 1ull;
    int32_t key[kDsRounds], val[kDsRounds], rank[kDsRounds];
    for (int r = 0; r < kDsRounds; ++r) {
        const int64_t g = b0 + r * kDsThreads + tid;
        const bool ok = g < N;
        key[r] = ok ? (idx ? ds_key(idx[g], M) : keys_in[g]) : 0;
        val[r] = ok ? (idx ? (int32_t)g : vals_in[g]) : 0;
        const int d = (key[r] >> shift) & (kDsDigits - 1);
        // lanes of this wave holding the same digit (all 64 lanes take part in every ballot)
        uint64_t peers = __ballot(ok);
#pragma unroll
        for (int bit = 0; bit < 8; ++bit) {
            const uint64_t m = __ballot((d >> bit) & 1);
            peers &= ((d >> bit) & 1) ? m : ~m;
        }
        rank[r] = __popcll(peers & below);
        if (ok && (peers & below) == 0) cnt[r * 4 + w][d] = __popcll(peers);
    }
    __syncthreads();
    {  // thread tid = digit: exclusive offsets of the groups, in entry order
        int32_t run = 0;
        for (int gi = 0; gi < kDsGroups; ++gi) {
            const int32_t c = cnt[gi][tid];
            cnt[gi][tid] = run;
            run += c;
        }
    }
    __syncthreads();
    for (int r = 0; r < kDsRounds; ++r) {
        const int64_t g = b0 + r * kDsThreads + tid;
        if (g >= N) continue;
        const int d = (key[r] >> shift) & (kDsDigits - 1);
        const int64_t dest = (int64_t)base[d] + start[(int64_t)d * gridDim.x + blockIdx.x] +
                             cnt[r * 4 + w][d] + rank[r];
        if (dest < N) {  // always true; keeps every write in bounds regardless
            if (keys_out) keys_out[dest] = key[r];
            vals_out[dest] = val[r];
        }
    }
}

// ------------------------------------------------------------------------------ one pass
// Keys 0 .. M with M + 1 <= kDsWideBins (up to 8191 experts) need one counting pass instead of two
// radix passes: per-block key counts, the scan of each key's block counts (dsort_wscan_kernel),
// and a scatter that also writes the offsets.  The counts are stored block-major,
// hist[b * (M + 1) + key], so that every kernel reads and writes whole rows of keys.
constexpr int kDsWideBins = 8192;
constexpr int kDsWideBits = 13;

// Key counts of block b: hist[b * (M + 1) + key].
__global__ __launch_bounds__(kDsThreads) void dsort_whist_kernel(const int32_t* __restrict__ idx,
                                                                 int64_t N, int32_t M,
                                                                 int32_t* __restrict__ hist) {
    __shared__ int32_t cnt[kDsWideBins];
    const int tid = threadIdx.x;
    const int D = M + 1;
    for (int i = tid; i < D; i += kDsThreads) cnt[i] = 0;
    __syncthreads();
    const int64_t b0 = (int64_t)blockIdx.x * kDsBlock;
    for (int r = 0; r < kDsRounds; ++r) {
        const int64_t g = b0 + r * kDsThreads + tid;
        if (g < N) atomicAdd(&cnt[ds_key(idx[g], M)], 1);
    }
    __syncthreads();
    for (int i = tid; i < D; i += kDsThreads) hist[(int64_t)blockIdx.x * D + i] = cnt[i];
}

// Keys 64 q .. 64 q + 63 for workgroup q, one per lane; wave w takes the w-th quarter of the
// nb blocks.  Each thread sums its key's counts over its blocks, the four sums give each wave's
// start, and a second pass over the same counts replaces them with the exclusive prefix in
// block order (start of the key's entries of block b among the key's entries); total[key]
// = the key's entry count.
__global__ __launch_bounds__(kDsThreads) void dsort_wscan_kernel(int32_t* __restrict__ hist,
                                                                 int64_t nb, int32_t D,
                                                                 int32_t* __restrict__ total) {
    constexpr int NW = kDsThreads / 64;
    __shared__ int32_t part[NW][64];
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const int32_t key = 64 * (int32_t)blockIdx.x + lane;
    const bool ok = key < D;
    const int64_t b0 = nb * w / NW, b1 = nb * (w + 1) / NW;
    int32_t sum = 0;
    if (ok) {
        int64_t b = b0;
        for (; b + 8 <= b1; b += 8) {
            int32_t v[8];
#pragma unroll
            for (int j = 0; j < 8; ++j) v[j] = hist[(b + j) * D + key];
#pragma unroll
            for (int j = 0; j < 8; ++j) sum += v[j];
        }
        for (; b < b1; ++b) sum += hist[b * D + key];
    }
    part[w][lane] = sum;
    __syncthreads();
    int32_t run = 0;
    for (int ww = 0; ww < w; ++ww) run += part[ww][lane];
    if (ok && w == NW - 1) total[key] = run + sum;
    if (ok) {
        int64_t b = b0;
        for (; b + 8 <= b1; b += 8) {
            int32_t v[8];
#pragma unroll
            for (int j = 0; j < 8; ++j) v[j] = hist[(b + j) * D + key];
#pragma unroll
            for (int j = 0; j < 8; ++j) {
                hist[(b + j) * D + key] = run;
                run += v[j];
            }
        }
        for (; b < b1; ++b) {
            const int32_t v = hist[b * D + key];
            hist[b * D + key] = run;
            run += v;
        }
    }
}

// Block b: base[key] = entries with a smaller key (the exclusive scan of the key totals, in LDS;
// block 0 writes it as the offsets) plus the block's prefix of the key (start, scanned per key).
// Wave w then places entries 256 w .. 256 w + 255 of the block in entry order.  The waves' counts
// of each key, 16-bit fields packed two to a word (waves 0 and 1 in wc[0], 2 and 3 in wc[1]), are
// turned into each wave's exclusive prefix over the earlier waves; in each group of 64 a lane's
// slot is base[key] + its wave's field + its rank among the group's lanes with that key (13
// ballots), and the group's first lane of each key advances the wave's field by the group's count
// of that key (an atomic add on the word, so the other half is never overwritten).
__global__ __launch_bounds__(kDsThreads) void dsort_wscatter_kernel(
    const int32_t* __restrict__ idx, int64_t N, int32_t M, const int32_t* __restrict__ start,
    const int32_t* __restrict__ total, int32_t* __restrict__ sorted,
    int32_t* __restrict__ offsets) {
    constexpr int PER = kDsWideBins / kDsThreads;  // keys per thread in the scan
    constexpr int WG = kDsRounds;                  // groups of 64 per wave (256 entries)
    __shared__ int32_t base[kDsWideBins];
    __shared__ uint32_t wc[2][kDsWideBins];
    __shared__ int32_t part[kDsThreads];
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const int D = M + 1;
    for (int i = tid; i < D; i += kDsThreads) {
        wc[0][i] = 0u;
        wc[1][i] = 0u;
    }
    int32_t v[PER];
    int32_t sum = 0;
#pragma unroll
    for (int i = 0; i < PER; ++i) {
        const int key = PER * tid + i;
        v[i] = key < D ? total[key] : 0;
        sum += v[i];
    }
    part[tid] = sum;
    __syncthreads();
    for (int d = 1; d < kDsThreads; d <<= 1) {  // inclusive scan of the threads' sums
        const int32_t u = tid >= d ? part[tid - d] : 0;
        __syncthreads();
        part[tid] += u;
        __syncthreads();
    }
    int32_t run = part[tid] - sum;
#pragma unroll
    for (int i = 0; i < PER; ++i) {
        base[PER * tid + i] = run;
        run += v[i];
    }
    __syncthreads();
    if (blockIdx.x == 0)
        for (int e = tid; e <= M; e += kDsThreads) offsets[e] = base[e];
    for (int key = tid; key < D; key += kDsThreads)
        base[key] += start[(int64_t)blockIdx.x * D + key];
    // the wave's keys, and its count of each key
    const int64_t b0 = (int64_t)blockIdx.x * kDsBlock + (int64_t)w * 64 * WG;
    const uint32_t one = 1u << (16 * (w & 1));
    int32_t keys[WG];
#pragma unroll
    for (int gi = 0; gi < WG; ++gi) {
        const int64_t g = b0 + gi * 64 + lane;
        keys[gi] = g < N ? ds_key(idx[g], M) : 0;
        if (g < N) atomicAdd(&wc[w >> 1][keys[gi]], one);
    }
    __syncthreads();
    for (int key = tid; key < D; key += kDsThreads) {  // per wave: the counts of earlier waves
        const uint32_t a = wc[0][key], c = wc[1][key];
        const uint32_t c0 = a & 0xFFFFu, c1 = a >> 16, c2 = c & 0xFFFFu;
        wc[0][key] = (c0 << 16);
        wc[1][key] = (c0 + c1) | ((c0 + c1 + c2) << 16);
    }
    __syncthreads();
    const uint64_t below = (1ull << lane) - 1ull;
    const int sh = 16 * (w & 1);
#pragma unroll
    for (int gi = 0; gi < WG; ++gi) {
        const int64_t g = b0 + gi * 64 + lane;
        const bool ok = g < N;
        const int d = keys[gi];
        uint64_t peers = __ballot(ok);
#pragma unroll
        for (int bit = 0; bit < kDsWideBits; ++bit) {
            const uint64_t m = __ballot((d >> bit) & 1);
            peers &= ((d >> bit) & 1) ? m : ~m;
        }
        const uint64_t before = peers & below;
        // every lane reads its wave's field before the group's first lane of each key advances
        // it (one wave: its LDS operations complete in order; the other wave of the word only
        // adds to its own field)
        const int32_t slot =
            base[d] + (int32_t)((wc[w >> 1][d] >> sh) & 0xFFFFu) + __popcll(before);
        if (ok && before == 0) atomicAdd(&wc[w >> 1][d], (uint32_t)__popcll(peers) << sh);
        if (ok && slot < N) sorted[slot] = (int32_t)g;
    }
}

// offsets[e] = the first slot i whose key is at least e (N if none), for e = 0 .. M.  With at
// least as many entries as experts, slot i writes the e in (key[i - 1], key[i]] (the last slot
// also those above its key): a few writes per slot.  With fewer entries, one thread per expert
// searches the sorted keys (coalesced writes; the first levels of neighbouring threads' searches
// read the same slots), since the gaps between keys would make the per-slot writes long.
__global__ __launch_bounds__(256) void dsort_offsets_gap_kernel(const int32_t* __restrict__ keys,
                                                                int64_t N, int32_t M,
                                                                int32_t* __restrict__ offsets) {
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i <= N;
         i += (int64_t)gridDim.x * blockDim.x) {
        const int32_t lo = i == 0 ? -1 : keys[i - 1];
        const int32_t hi = i == N ? M : keys[i];
        for (int32_t e = lo + 1; e <= hi && e <= M; ++e) offsets[e] = (int32_t)i;
    }
}

__global__ __launch_bounds__(256) void dsort_offsets_kernel(const int32_t* __restrict__ keys,
                                                            int64_t N, int32_t M,
                                                            int32_t* __restrict__ offsets) {
    const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (e > M) return;
    int64_t lo = 0, hi = N;  // keys[lo - 1] < e <= keys[hi] (virtual ends)
    while (lo < hi) {
        const int64_t mid = (lo + hi) >> 1;
        if (keys[mid] < e)
            lo = mid + 1;
        else
            hi = mid;
    }
    offsets[e] = (int32_t)lo;
}

// All passes of the sort in one workgroup, for at most kDsSmallN entries: keys and positions
// ping-pong between two LDS buffers; per pass a digit histogram, its exclusive scan, then the
// entries in rounds of 1024 (entry order): ranks within a wave from ballots, counts of the
// earlier waves of the round per digit, and each digit's running base across rounds.  The
// sorted keys go to keys_out (for the offsets) and the positions to sorted.
constexpr int kDsSmallThreads = 1024;
constexpr int kDsSmallN = 4096;
constexpr int kDsSmallWaves = kDsSmallThreads / 64;

__global__ __launch_bounds__(kDsSmallThreads) void dsort_small_kernel(
    const int32_t* __restrict__ idx, int32_t N, int32_t M, int passes,
    int32_t* __restrict__ keys_out, int32_t* __restrict__ sorted) {
    __shared__ int32_t kbuf[2][kDsSmallN];
    __shared__ int32_t vbuf[2][kDsSmallN];
    __shared__ int32_t cnt[kDsSmallWaves][kDsDigits];
    __shared__ int32_t base[kDsDigits];
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const uint64_t below = (1ull << lane) - 1ull;
    for (int i = tid; i < N; i += kDsSmallThreads) {
        kbuf[0][i] = ds_key(idx[i], M);
        vbuf[0][i] = i;
    }
    int cur = 0;
    for (int p = 0; p < passes; ++p) {
        const int shift = 8 * p;
        if (tid < kDsDigits) base[tid] = 0;
        __syncthreads();
        for (int i = tid; i < N; i += kDsSmallThreads)
            atomicAdd(&base[(kbuf[cur][i] >> shift) & (kDsDigits - 1)], 1);
        __syncthreads();
        if (tid < 64) {  // exclusive scan of the 256 digit counts by one wave, four per lane
            int32_t v[4], sum = 0;
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                v[i] = base[4 * tid + i];
                sum += v[i];
            }
            int32_t incl = sum;
            for (int d = 1; d < 64; d <<= 1) {
                const int32_t u = __shfl_up(incl, d, 64);
                incl += tid >= d ? u : 0;
            }
            int32_t run = incl - sum;
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                base[4 * tid + i] = run;
                run += v[i];
            }
        }
        __syncthreads();
        for (int r0 = 0; r0 < N; r0 += kDsSmallThreads) {
            for (int i = tid; i < kDsSmallWaves * kDsDigits; i += kDsSmallThreads)
                (&cnt[0][0])[i] = 0;
            __syncthreads();
            const int g = r0 + tid;
            const bool ok = g < N;
            const int32_t key = ok ? kbuf[cur][g] : 0;
            const int32_t val = ok ? vbuf[cur][g] : 0;
            const int d = (key >> shift) & (kDsDigits - 1);
            uint64_t peers = __ballot(ok);  // lanes of this wave with the same digit
#pragma unroll
            for (int bit = 0; bit < 8; ++bit) {
                const uint64_t m = __ballot((d >> bit) & 1);
                peers &= ((d >> bit) & 1) ? m : ~m;
            }
            const int rank = __popcll(peers & below);
            if (ok && (peers & below) == 0) cnt[w][d] = __popcll(peers);
            __syncthreads();
            if (tid < kDsDigits) {  // digit tid: exclusive offsets of the waves, then the base
                int32_t run = base[tid];
                for (int ww = 0; ww < kDsSmallWaves; ++ww) {
                    const int32_t c = cnt[ww][tid];
                    cnt[ww][tid] = run;
                    run += c;
                }
                base[tid] = run;  // the next round's entries of this digit follow
            }
            __syncthreads();
            if (ok) {
                const int dest = cnt[w][d] + rank;
                if (dest < N) {  // always true; keeps every write in bounds regardless
                    kbuf[cur ^ 1][dest] = key;
                    vbuf[cur ^ 1][dest] = val;
                }
            }
            __syncthreads();
        }
        cur ^= 1;
    }
    for (int i = tid; i < N; i += kDsSmallThreads) {
        keys_out[i] = kbuf[cur][i];
        sorted[i] = vbuf[cur][i];
    }
}

__global__ __launch_bounds__(256) void dsort_fill_kernel(int32_t* __restrict__ p, int64_t n,
                                                         int32_t v) {
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
         i += (int64_t)gridDim.x * blockDim.x)
        p[i] = v;
}

int dispatch_passes(int32_t M) {
    int bits = 1;
    while (bits < 31 && ((int64_t)1 << bits) <= (int64_t)M) ++bits;  // keys 0 .. M
    return (bits + 7) / 8;
}

size_t dispatch_workspace_bytes(int64_t N) {
    if (N == 0) return 0;
    const int64_t nblocks = (N + kDsBlock - 1) / kDsBlock;
    auto al = [](size_t b) { return (b + 255) & ~(size_t)255; };
    // room for the key counts of the one-pass sort (kDsWideBins >= kDsDigits)
    return 4 * al((size_t)N * 4) + al((size_t)nblocks * kDsWideBins * 4) + al(kDsWideBins * 4);
}

hipError_t dispatch_launch(const int32_t* idx, int64_t N, int32_t M, int32_t* offsets,
                           int32_t* sorted, void* workspace, hipStream_t st) {
    if (N == 0) {
        const int64_t n = (int64_t)M + 1;
        const unsigned blocks = (unsigned)((n + 255) / 256 < 1024 ? (n + 255) / 256 : 1024);
        hipLaunchKernelGGL(dsort_fill_kernel, dim3(blocks), dim3(256), 0, st, offsets, n, 0);
        return hipGetLastError();
    }
    const int64_t nblocks = (N + kDsBlock - 1) / kDsBlock;
    auto al = [](size_t b) { return (b + 255) & ~(size_t)255; };
    char* ws = static_cast<char*>(workspace);
    const unsigned oblocks = (unsigned)(((int64_t)M + 1 + 255) / 256);
    if (N <= kDsSmallN) {  // one workgroup sorts, a second launch derives the offsets
        int32_t* keys = reinterpret_cast<int32_t*>(ws);
        hipLaunchKernelGGL(dsort_small_kernel, dim3(1), dim3(kDsSmallThreads), 0, st, idx,
                           (int32_t)N, M, dispatch_passes(M), keys, sorted);
        hipLaunchKernelGGL(dsort_offsets_kernel, dim3(oblocks), dim3(256), 0, st, keys, N, M,
                           offsets);
        return hipGetLastError();
    }
    if ((int64_t)M + 1 <= kDsWideBins) {  // one counting pass: three launches
        int32_t* hist = reinterpret_cast<int32_t*>(ws + 4 * al((size_t)N * 4));
        int32_t* total = reinterpret_cast<int32_t*>(ws + 4 * al((size_t)N * 4) +
                                                    al((size_t)nblocks * kDsWideBins * 4));
        hipLaunchKernelGGL(dsort_whist_kernel, dim3((unsigned)nblocks), dim3(kDsThreads), 0, st,
                           idx, N, M, hist);
        hipLaunchKernelGGL(dsort_wscan_kernel, dim3((unsigned)((M + 1 + 63) / 64)),
                           dim3(kDsThreads), 0, st, hist, nblocks, (int32_t)(M + 1), total);
        hipLaunchKernelGGL(dsort_wscatter_kernel, dim3((unsigned)nblocks), dim3(kDsThreads), 0, st,
                           idx, N, M, hist, total, sorted, offsets);
        return hipGetLastError();
    }
    int32_t* keys[2] = {reinterpret_cast<int32_t*>(ws), reinterpret_cast<int32_t*>(ws + al((size_t)N * 4))};
    int32_t* vals[2] = {reinterpret_cast<int32_t*>(ws + 2 * al((size_t)N * 4)),
                        reinterpret_cast<int32_t*>(ws + 3 * al((size_t)N * 4))};
    int32_t* hist = reinterpret_cast<int32_t*>(ws + 4 * al((size_t)N * 4));
    int32_t* total = reinterpret_cast<int32_t*>(ws + 4 * al((size_t)N * 4) +
                                                al((size_t)nblocks * kDsDigits * 4));
    const int passes = dispatch_passes(M);
    for (int p = 0; p < passes; ++p) {
        const int shift = 8 * p;
        const int32_t* kin = p == 0 ? nullptr : keys[(p - 1) & 1];
        const int32_t* vin = p == 0 ? nullptr : vals[(p - 1) & 1];
        const int32_t* src_idx = p == 0 ? idx : nullptr;
        int32_t* kout = keys[p & 1];
        int32_t* vout = p == passes - 1 ? sorted : vals[p & 1];
        hipLaunchKernelGGL(dsort_hist_kernel, dim3((unsigned)nblocks), dim3(kDsThreads), 0, st,
                           src_idx, kin, N, M, shift, hist);
        hipLaunchKernelGGL(dsort_scan_kernel, dim3(kDsDigits), dim3(kDsThreads), 0, st, hist,
                           nblocks, total);
        hipLaunchKernelGGL(dsort_scatter_kernel, dim3((unsigned)nblocks), dim3(kDsThreads), 0, st,
                           src_idx, kin, vin, N, M, shift, hist, total, kout, vout);
    }
    if (N >= M) {
        const int64_t nth = N + 1;
        const unsigned blocks = (unsigned)((nth + 255) / 256 < 4096 ? (nth + 255) / 256 : 4096);
        hipLaunchKernelGGL(dsort_offsets_gap_kernel, dim3(blocks), dim3(256), 0, st,
                           keys[(passes - 1) & 1], N, M, offsets);
    } else {
        hipLaunchKernelGGL(dsort_offsets_kernel, dim3(oblocks), dim3(256), 0, st,
                           keys[(passes - 1) & 1], N, M, offsets);
    }
    return hipGetLastError();
}

}  // namespace more
