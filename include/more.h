/*
 * more.h -- C ABI of the MoRE low-rank router library for AMD Instinct MI355X (gfx950).
 *
 * The library computes the MoRE router output (Section "Preliminaries", MoRE layer):
 *
 *     g(x; R1, R2) = softmax(TopK(x R1 R2))
 *
 * for T tokens at once, x [T x h], R1 [h x r], R2 [r x M].  In the paper's own notation the
 * same logits are x R2_paper^T R1_paper^T with the down-projection R2_paper (r x h) and the
 * expert matrix R1_paper (M x r, row e = expert vector u_e); so R1 = R2_paper^T and
 * R2 = R1_paper^T (Appendix "Pseudocode", logits equation).  TopK keeps the k largest logits
 * of the M experts; the softmax runs over those k logits only.  The T x M logit matrix is
 * never written to memory (Appendix "Pseudocode", inference algorithm).
 *
 * Calls: the routing (more_route_lowrank and its variants), the training forward pass with the
 * softmax statistics (more_route_lowrank_train), the training backward pass
 * (more_route_lowrank_backward), the full-rank baselines (more_route_fullrank,
 * more_route_fullrank_fused), the per-expert histogram and the dispatch bookkeeping
 * (more_dispatch_sort).
 *
 * Conventions shared by every call
 * --------------------------------
 *  - Element types: bfloat16 inputs are passed as uint16_t bit patterns.  Accumulation is
 *    fp32.  Outputs: int32 expert ids, fp32 gates and logits.
 *  - Storage: x is row-major [T][h] (token rows).  Both router factors are passed
 *    TRANSPOSED, i.e. in the paper's row-major orientation:
 *        R1t = R1^T stored row-major [r][h]   (= R2_paper, one row per rank direction)
 *        R2t = R2^T stored row-major [M][r]   (= R1_paper, one row per expert vector)
 *    so every contraction reads contiguous rows along its reduction axis.
 *  - Pointers are device pointers on the current HIP device unless marked "host".  Every
 *    device pointer must be 16-byte aligned.  Inputs are read only; outputs must not alias
 *    inputs or one another.  The caller owns and allocates every buffer, including the
 *    workspace; the router calls never allocate, free or synchronise.
 *  - `stream` is a hipStream_t (NULL = the default stream).  Work is enqueued on it and the
 *    call returns after launching.  Launch failures return MORE_ERR_HIP; faults during
 *    execution surface at the caller's next synchronisation.
 *  - Arguments are validated on the host before anything is launched; an error status means
 *    nothing was enqueued.  T == 0 returns MORE_OK without launching (apart from clearing
 *    the per-expert outputs counts and psum, and the weight gradients dR1t and dR2t of the
 *    backward pass); the token-sized pointers (x, idx, gate, topval, m, Z, dtop, dx) may then
 *    be NULL.
 *  - Selection order: experts are ranked by logit, larger first; equal logits are ranked by
 *    expert id, smaller first.  idx[t][0..k-1] lists the selected experts in that order.
 *    (The paper's buffer leaves both the slot order and tie handling open; this total
 *    order makes every plan and every run bitwise reproducible.)
 *  - Limits: 1 <= k <= min(M, MORE_K_MAX) for the full-rank router and
 *    1 <= k <= min(M, MORE_LOWRANK_K_MAX) for the low-rank router, with r a multiple of 16 up
 *    to 256 (the paper's rank sweeps, Section "Routing expressivity"); the training forward
 *    and backward passes take r in {16, 32, 64}, and the training forward k <=
 *    MORE_LOWRANK_TRAIN_K_MAX; h a positive multiple of 16; M >= 1 (any value; the last expert tile is masked to -inf, as
 *    the paper's inference algorithm does for out-of-range experts); T <= 2^31 - 1.
 *  - Numerics: z = x R1 is accumulated in fp32.  The expert sweeps run on the matrix cores
 *    with z rounded to bfloat16 and a rigorous bound on the resulting logit error, which
 *    selects a small candidate set that provably holds the top k; the candidates' logits
 *    are then evaluated exactly in fp32 (fp32 z times the bfloat16 expert rows).  The paper's
 *    kernel instead narrows z to one bfloat16 for the whole contraction.  Shapes outside the
 *    register-tiled routes (r not in {16, 32, 64}, or k > 16) take the wide route
 *    (MORE_ROUTE_WIDE): fp32 z split exactly into three bfloat16 pieces and one fused sweep of
 *    the matrix cores over the 3r-wide pair, i.e. the same fp32 logits up to summation order.
 */
#ifndef MORE_H
#define MORE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum more_status {
    MORE_OK = 0,
    MORE_ERR_INVALID_ARG = 1, /* NULL/misaligned pointer, negative or zero size, k out of range */
    MORE_ERR_UNSUPPORTED = 2, /* valid arguments outside the limits listed above               */
    MORE_ERR_WORKSPACE = 3,   /* workspace NULL or smaller than the matching size query        */
    MORE_ERR_HIP = 4          /* the HIP runtime or hipBLASLt reported an error                */
} more_status;

#define MORE_K_MAX 32
#define MORE_LOWRANK_K_MAX 32
#define MORE_LOWRANK_TRAIN_K_MAX 16

/*
 * Low-rank router (Section "Preliminaries", MoRE layer; Appendix "Pseudocode", inference
 * algorithm).
 *   x       bf16 [T][h]            tokens
 *   R1t     bf16 [r][h]            R1 transposed (the paper's down-projection R2_paper)
 *   R2t     bf16 [M][r]            R2 transposed (the paper's expert matrix R1_paper)
 *   idx     int32 [T][k]  out      selected experts, in selection order
 *   gate    fp32  [T][k]  out      softmax over the k selected logits, same order
 *   topval  fp32  [T][k]  out      the selected logits, or NULL
 *   counts  int32 [M]     out      per-expert number of selections over all T tokens
 *                                  (overwritten), or NULL to skip
 *   workspace / workspace_bytes    scratch of at least more_route_lowrank_workspace_size()
 *                                  bytes (NULL/0 allowed when that size is 0)
 */
more_status more_route_lowrank(const uint16_t* x, const uint16_t* R1t, const uint16_t* R2t,
                               int64_t T, int32_t h, int32_t r, int32_t M, int32_t k,
                               int32_t* idx, float* gate, float* topval, int32_t* counts,
                               void* workspace, size_t workspace_bytes, void* stream);

/* Workspace bytes more_route_lowrank needs for this shape (written to *bytes, host). */
more_status more_route_lowrank_workspace_size(int64_t T, int32_t h, int32_t r, int32_t M,
                                              int32_t k, size_t* bytes);

/*
 * Same as more_route_lowrank with the expert axis split into (at least) `m_chunks` slices
 * processed by separate workgroups and merged afterwards (0 = the library's choice, which may be
 * a fused route on small expert sets; 1 = no split, else a multiple of 8 up to 1024; the library
 * raises it when a slice would not fit in one workgroup's LDS).  Every m_chunks >= 1 returns
 * bitwise identical results, and so does the fused route that reads the z pass (r M <= 2^18).
 * The one-launch fused route (r M <= 2^17 with K <= 8, and M <= 1024 at r = 64) computes z
 * inside the routing workgroup, summing the h axis in another order: its logits can differ from
 * the others' in the last bits (selections only where logits tie to rounding); so can those of
 * the single-pass route, which m_chunks = 0 picks for T >= 4096 and M >= 32768.  This entry
 * point exists for tuning and for tests of these properties.  The wide route ignores m_chunks
 * (any valid value gives the same result).  Its workspace size comes from
 * more_route_lowrank_workspace_size_ex with the same m_chunks (0 bytes for the one-launch
 * route).
 */
more_status more_route_lowrank_ex(const uint16_t* x, const uint16_t* R1t, const uint16_t* R2t,
                                  int64_t T, int32_t h, int32_t r, int32_t M, int32_t k,
                                  int32_t m_chunks, int32_t* idx, float* gate, float* topval,
                                  int32_t* counts, void* workspace, size_t workspace_bytes,
                                  void* stream);
more_status more_route_lowrank_workspace_size_ex(int64_t T, int32_t h, int32_t r, int32_t M,
                                                 int32_t k, int32_t m_chunks, size_t* bytes);

/* The m_chunks value the library picks for this shape (written to *m_chunks, host): the
 * number of expert-axis slices of the expert-resident route, or 0 when the library routes this
 * shape with a route that no m_chunks >= 1 selects: a fused route (expert sets with
 * r * M <= 2^18 and M <= 16384: one workgroup per 64 tokens sweeps all experts) or the
 * single-pass route (T >= 4096 and M >= 32768: one screening sweep over all experts after a
 * prescreen of a quarter of them; see more_route_lowrank_ex) or the wide route. */
more_status more_route_lowrank_plan(int64_t T, int32_t h, int32_t r, int32_t M, int32_t k,
                                    int32_t* m_chunks);

/* The route more_route_lowrank takes for this shape (written to *route, host): one of the
 * MORE_ROUTE_* codes below.  Routes differ in speed and in the summation order of z = x R1 (see
 * more_route_lowrank_ex); every route returns the exact top k of its own fp32 logits. */
#define MORE_ROUTE_RESIDENT 0    /* z pass; screen, threshold, collect and finalize per chunk  */
#define MORE_ROUTE_FUSED 1       /* z pass; one fused kernel per 64 tokens over all experts     */
#define MORE_ROUTE_FUSED_LOCAL 2 /* one launch: the fused kernel also computes z                */
#define MORE_ROUTE_SINGLE_PASS 3 /* z + prescreen, one collect sweep, finalize (+ histogram)    */
#define MORE_ROUTE_WIDE 4        /* z per rank block; exact 3-piece split; fused 3r-wide sweep */
more_status more_route_lowrank_route(int64_t T, int32_t h, int32_t r, int32_t M, int32_t k,
                                     int32_t* route);

/*
 * Training forward pass of the low-rank router (Appendix "Pseudocode", training forward
 * algorithm; eqs. app_softmax, app_psum and app_online): the routing of more_route_lowrank plus
 * the statistics of the full row softmax over all M experts that the switch load-balancing
 * loss L_bal = (M / T) sum_e f_e psum[e] needs (f_e = counts[e] / (T k); the loss itself is
 * left to the caller):
 *   m[t]    = max_e l_te                       (the token's top-1 logit)
 *   Z[t]    = sum_e exp(l_te - m[t])           (the normaliser of the online softmax)
 *   psum[e] = sum_t exp(l_te - m[t]) / Z[t]    (column sums of the softmax probabilities)
 * with l = x R1 R2; no T x M matrix is written.
 *   x, R1t, R2t, T, h, r, M, k, idx, gate, topval, counts   as in more_route_lowrank
 *   m       fp32 [T]  out
 *   Z       fp32 [T]  out
 *   psum    fp32 [M]  out     (all zero when T == 0)
 *   workspace / workspace_bytes   at least more_route_lowrank_train_workspace_size() bytes,
 *                                 256-byte aligned
 * Numerics: m is the top-1 logit of the routing (topval[t][0]).  Z and psum take the logits
 * from the matrix cores with z carried as a bfloat16 hi/lo pair (about 16 significant bits):
 * each exponent is within 2^-18 sum_i |z_i u_ei| + 2^-24 (2r + 1)(|m| + sum_i |z_i u_ei|)
 * (times log2 e) of exact, and the sums run in fp32 in a fixed order, so a shape gives the same
 * bits on every run.  Limits: r in {16, 32, 64} and k <= MORE_LOWRANK_TRAIN_K_MAX (the
 * register-tiled routes; other shapes return MORE_ERR_UNSUPPORTED), otherwise as for
 * more_route_lowrank.
 */
more_status more_route_lowrank_train(const uint16_t* x, const uint16_t* R1t, const uint16_t* R2t,
                                     int64_t T, int32_t h, int32_t r, int32_t M, int32_t k,
                                     int32_t* idx, float* gate, float* topval, int32_t* counts,
                                     float* m, float* Z, float* psum, void* workspace,
                                     size_t workspace_bytes, void* stream);
more_status more_route_lowrank_train_workspace_size(int64_t T, int32_t h, int32_t r, int32_t M,
                                                    int32_t k, size_t* bytes);

/*
 * Training backward pass of the low-rank router with recompute (Appendix "Pseudocode",
 * backward pass: eqs. app_chain, app_jac, app_kernelgrad and the backward algorithm).  Given
 * the selection of the forward pass, the gradient of the loss with respect to the selected
 * logits and (optionally) with respect to psum, it returns the gradients with respect to x,
 * R1 and R2.  With l = x R1 R2 recomputed tile by tile (never written) and
 * P_te = exp(l_te - m[t]) / Z[t]:
 *   g_t      = sum_e pbar[e] P_te
 *   ybar_te  = P_te (pbar[e] - g_t) + sum_{j : idx[t][j] == e} dtop[t][j]
 *   dx       = ybar R2^T R1^T     dR1t = (x^T ybar R2^T)^T     dR2t = (R1^T x^T ybar)^T
 * i.e. dz = ybar R2^T [T][r], dx = dz R1^T, dR1t[i][c] = sum_t dz[t][i] x[t][c],
 * dR2t[e][i] = sum_t ybar_te z[t][i].
 *   x, R1t, R2t, T, h, r, M   as in more_route_lowrank (device, bf16)
 *   k         selections per token, 1 <= k <= min(M, MORE_K_MAX)
 *   idx       int32 [T][k]  the selection (device); entries outside [0, M) add nothing
 *   dtop      fp32 [T][k]   gradient with respect to the selected logits l_t[idx[t][j]] (device)
 *   pbar      fp32 [M]      gradient with respect to psum (device), or NULL: no balancing term
 *                           (then m and Z are not read and may be NULL)
 *   m, Z      fp32 [T]      the statistics saved by more_route_lowrank_train (device)
 *   dx        fp32 [T][h]   out (device), overwritten
 *   dR1t      fp32 [r][h]   out (device), overwritten; zero when T == 0
 *   dR2t      fp32 [M][r]   out (device), overwritten; zero when T == 0
 *   workspace / workspace_bytes   at least more_route_lowrank_backward_workspace_size() bytes
 *             with balance = (pbar != NULL), 256-byte aligned (device; NULL allowed when T == 0)
 * Numerics: the recomputed logits are those of the training forward pass's statistics (z as a
 * bf16 hi/lo pair); P (pbar - g) is rounded to bf16 for the two contractions over experts and
 * tokens, which read bf16(z) and R2 with fp32 accumulation; the dtop terms use fp32 z; dx and
 * dR1t read dz as a bf16 hi/lo pair.  Every sum runs in a fixed order, so a shape gives the
 * same bits on every run.  Errors: MORE_ERR_INVALID_ARG (NULL or misaligned pointers, negative
 * sizes), MORE_ERR_UNSUPPORTED (r outside {16, 32, 64}, h not a multiple of 16, k > MORE_K_MAX),
 * MORE_ERR_WORKSPACE; nothing is enqueued on an error.
 */
more_status more_route_lowrank_backward(const uint16_t* x, const uint16_t* R1t,
                                        const uint16_t* R2t, int64_t T, int32_t h, int32_t r,
                                        int32_t M, int32_t k, const int32_t* idx,
                                        const float* dtop, const float* pbar, const float* m,
                                        const float* Z, float* dx, float* dR1t, float* dR2t,
                                        void* workspace, size_t workspace_bytes, void* stream);
more_status more_route_lowrank_backward_workspace_size(int64_t T, int32_t h, int32_t r,
                                                       int32_t M, int32_t k, int32_t balance,
                                                       size_t* bytes);

/*
 * Full-rank (standard) router, the baseline (Section "Preliminaries": softmax(TopK(R x)) with
 * R in R^{M x h}).  The logits x W^T are formed with a hipBLASLt GEMM into the workspace
 * (fp32 when logit_bits == 32, bf16 when logit_bits == 16) and a row top-k kernel then
 * selects and normalises, as the paper's unfused standard router does.
 *   Wt      bf16 [M][h]            the router matrix, one row per expert (the paper's R)
 *   other arguments as in more_route_lowrank (no histogram).
 * The library keeps one hipBLASLt handle per device, created on first use and never freed;
 * calls may run concurrently from several threads.
 */
more_status more_route_fullrank(const uint16_t* x, const uint16_t* Wt, int64_t T, int32_t h,
                                int32_t M, int32_t k, int32_t logit_bits, int32_t* idx,
                                float* gate, float* topval, void* workspace,
                                size_t workspace_bytes, void* stream);
more_status more_route_fullrank_workspace_size(int64_t T, int32_t h, int32_t M, int32_t k,
                                               int32_t logit_bits, size_t* bytes);

/*
 * Fused full-rank (standard) router, the stronger baseline (efficiency appendix, "Fusing a
 * standard MoE layer": the low-rank router's fusion with the rank replaced by h).  Same result
 * definition and arguments as more_route_fullrank with fp32 logits, but the T x M logits are
 * never written: a workgroup keeps the x rows of 32-128 tokens in LDS, streams the rows of Wt
 * through the matrix cores (fp32 accumulation of exact bf16 products) and folds each logit
 * into register top-k lists.  The rows of Wt are re-read for every token block, so this suits
 * small h and M (the paper finds the fusion's benefit vanishing at large h).
 *   workspace   at least more_route_fullrank_fused_workspace_size() bytes (the lists of the
 *               expert splits; 0 bytes when one workgroup sweeps all experts of a token block)
 * Limits: h <= 2112 (the x rows of 32 tokens fit one workgroup's LDS), k <= 32; larger h returns
 * MORE_ERR_UNSUPPORTED.  Logits can differ from more_route_fullrank's in the last bits (another
 * fp32 summation order).
 */
more_status more_route_fullrank_fused(const uint16_t* x, const uint16_t* Wt, int64_t T, int32_t h,
                                      int32_t M, int32_t k, int32_t* idx, float* gate,
                                      float* topval, void* workspace, size_t workspace_bytes,
                                      void* stream);
more_status more_route_fullrank_fused_workspace_size(int64_t T, int32_t h, int32_t M, int32_t k,
                                                     size_t* bytes);

/*
 * Per-expert histogram of a selection (the bincount behind the load-balancing statistic,
 * Appendix "Training"): counts[e] = #{(t, j) : idx[t][j] == e}.
 *   idx     int32 [T][k]   selections; every entry must lie in [0, M)
 *   counts  int32 [M] out  overwritten
 * Entries outside [0, M) are not counted (no error is raised for them).
 */
more_status more_expert_histogram(const int32_t* idx, int64_t T, int32_t k, int32_t M,
                                  int32_t* counts, void* stream);

/*
 * Dispatch bookkeeping that consumes a selection ("Sort + Count" of the MoE layer's forward
 * pass in the efficiency appendix: the (N, k) expert ids become N k sorted positions plus
 * per-expert offsets).  The T k entries of idx are numbered p = t k + j (row-major); an entry's
 * key is its expert id, or M when the id lies outside [0, M).
 *   idx      int32 [T][k]           expert ids (e.g. the idx output of a routing call)
 *   offsets  int32 [M + 1]  out     offsets[e] = number of entries whose key is below e;
 *                                   offsets[M] = number of entries with a valid id
 *   sorted   int32 [T k]    out     the positions p ordered by key, increasing p within a key
 *                                   (expert e's entries are sorted[offsets[e] .. offsets[e+1]);
 *                                   entries with invalid ids follow all experts)
 *   workspace / workspace_bytes     at least more_dispatch_sort_workspace_size() bytes,
 *                                   256-byte aligned (0 bytes when T = 0)
 * Limits: T k <= 2^31 - 1, M < 2^30.  T == 0 writes offsets (all zero).  A stable radix sort
 * on the key: the result is unique, so every run gives the same bits.
 */
more_status more_dispatch_sort(const int32_t* idx, int64_t T, int32_t k, int32_t M,
                               int32_t* offsets, int32_t* sorted, void* workspace,
                               size_t workspace_bytes, void* stream);
more_status more_dispatch_sort_workspace_size(int64_t T, int32_t k, int32_t M, size_t* bytes);

/*
 * For callers that cannot allocate (code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc): more_route_lowrank without a workspace argument.  The
 * scratch is a static device array of MORE_NOALLOC_SCRATCH_BYTES bytes per device, placed on
 * a device by the first call there and held until the process ends; this call allocates and
 * frees nothing.  Arguments, outputs and results are those of more_route_lowrank (bitwise
 * identical).  A shape whose more_route_lowrank_workspace_size exceeds the array returns
 * MORE_ERR_WORKSPACE before anything is launched.  Every call on a device shares its array:
 * calls ordered on one stream are safe, calls that overlap in time on one device (other
 * streams, other threads) race and give undefined results.  MORE_ERR_HIP when the array's
 * device address cannot be obtained.
 */
#define MORE_NOALLOC_SCRATCH_BYTES ((size_t)256 << 20)
more_status more_route_lowrank_noalloc(const uint16_t* x, const uint16_t* R1t, const uint16_t* R2t,
                                       int64_t T, int32_t h, int32_t r, int32_t M, int32_t k,
                                       int32_t* idx, float* gate, float* topval, int32_t* counts,
                                       void* stream);

/* Static, never NULL. */
const char* more_status_string(more_status s);

/* Library version string, e.g. "0.1.0 gfx950". Static, never NULL. */
const char* more_version(void);

#ifdef __cplusplus
}
#endif

#endif /* MORE_H */
