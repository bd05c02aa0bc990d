/*
 * Router oracle: a plain, slow, fp64 evaluation of the MoRE router output.
 *
 * TEST INFRASTRUCTURE ONLY.  This file is the checker the HIP library is compared
 * against.  Only the test suite, the smoke check and the benchmark's CPU-baseline
 * leg may load it.  It shares no code, header, table or helper with the library.
 *
 * What it computes is the definition itself (Section "Preliminaries", MoRE layer):
 *     g(x; R1, R2) = softmax(TopK(x R1 R2))
 * written here in the library's orientation, x [T][h], R1 [h][r], R2 [r][M]
 * (the paper writes the same product as R1_paper R2_paper x, with
 * R1_paper = R2^T and R2_paper = R1^T; Appendix "Pseudocode", eq. for the logits).
 * Steps, per token t:
 *   1. decode the bfloat16 inputs exactly to double;
 *   2. z_t = sum_j x[t][j] * R1[j][:]                        (fp64)
 *   3. l_t[e] = sum_i z_t[i] * R2[i][e] for every expert e     (fp64; z is never narrowed)
 *   4. S_t = the first k experts in the total order "logit descending, then expert
 *      index ascending" (a full sort of all M candidates with qsort);
 *   5. gate_t[j] = exp(l_(j) - l_(1)) / sum_{i<k} exp(l_(i) - l_(1))   (softmax over the k
 *      selected logits, standard router definition in "Preliminaries");
 *   6. also report the selected logits and l_(k+1), the best unselected logit, so the
 *      caller can tell near-ties at the selection boundary.
 * The full-rank entry points run steps 4-6 on logits x W with a given W [h][M]
 * (standard router, "Preliminaries").  The histogram is the per-expert count of
 * selections (bincount of the chosen indices, Appendix "Training", load-balancing
 * statistic f).
 *
 * oracle_route_stats gives the softmax statistics of the training forward pass: the row maximum
 * m, the normaliser Z and the column sums psum of the full softmax over all experts.
 *
 * oracle_route_backward is the training backward pass: the gradients of a loss with respect to
 * x, R1 and R2, given its gradients with respect to the selected logits and to psum.
 *
 * oracle_dispatch_sort is the dispatch bookkeeping that consumes a selection: the selected
 * (token, slot) positions grouped by expert, with per-expert offsets.
 *
 * oracle_logits_at evaluates steps 2-3 at given (token, expert) pairs only, so that a
 * selection made by another implementation can be checked expert by expert;
 * oracle_fullrank_logits_at does the same for the full-rank logits x W.
 *
 * Non-finite inputs are rejected (return value ORACLE_ERR_NONFINITE).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#ifdef _OPENMP
#include <omp.h>
#endif

#define ORACLE_OK 0
#define ORACLE_ERR_ARG 1
#define ORACLE_ERR_NONFINITE 2
#define ORACLE_ERR_NOMEM 3

static double bf16_bits_to_double(uint16_t b) {
    uint32_t u = ((uint32_t)b) << 16;
    float f;
    memcpy(&f, &u, sizeof f);
    return (double)f;
}

/* Decode n bf16 values; returns 0 if any is NaN or infinite. */
static int decode_all(const uint16_t* src, int64_t n, double* dst) {
    int finite = 1;
    for (int64_t i = 0; i < n; ++i) {
        dst[i] = bf16_bits_to_double(src[i]);
        if (!isfinite(dst[i])) finite = 0;
    }
    return finite;
}

typedef struct {
    double value;
    int32_t expert;
} candidate;

/* Total order used for selection: larger logit first; equal logits -> smaller index first. */
static int candidate_order(const void* pa, const void* pb) {
    const candidate* a = (const candidate*)pa;
    const candidate* b = (const candidate*)pb;
    if (a->value > b->value) return -1;
    if (a->value < b->value) return 1;
    if (a->expert < b->expert) return -1;
    if (a->expert > b->expert) return 1;
    return 0;
}

/* Steps 4-6 for one token, given all M logits. */
static void select_and_gate(const double* logit, int32_t M, int32_t k, candidate* work,
                            int32_t* idx, double* gate, double* topval, double* next) {
    for (int32_t e = 0; e < M; ++e) {
        work[e].value = logit[e];
        work[e].expert = e;
    }
    qsort(work, (size_t)M, sizeof(candidate), candidate_order);
    double top = work[0].value;
    double denom = 0.0;
    for (int32_t j = 0; j < k; ++j) {
        idx[j] = work[j].expert;
        topval[j] = work[j].value;
        gate[j] = exp(work[j].value - top);
        denom += gate[j];
    }
    for (int32_t j = 0; j < k; ++j) gate[j] /= denom;
    *next = (k < M) ? work[k].value : -INFINITY;
}

static int check_shape(int64_t T, int32_t h, int32_t r, int32_t M, int32_t k,
                       const int64_t* rows, int64_t nrows) {
    if (T < 0 || h <= 0 || r <= 0 || M <= 0 || k < 1 || k > M) return 0;
    if (rows) {
        if (nrows < 0) return 0;
        for (int64_t i = 0; i < nrows; ++i)
            if (rows[i] < 0 || rows[i] >= T) return 0;
    }
    return 1;
}

/*
 * Low-rank router.  x: bf16 [T][h]; R1: bf16 [h][r]; R2: bf16 [r][M]  (all row-major).
 * rows: the tokens to evaluate (nrows of them), or NULL for all T tokens in order.
 * Outputs, one row per evaluated token: idx int32 [n][k], gate/topval double [n][k],
 * next double [n] (the (k+1)-th logit, -inf when k == M).
 */
int oracle_route_lowrank(const uint16_t* x, const uint16_t* R1, const uint16_t* R2,
                         int64_t T, int32_t h, int32_t r, int32_t M, int32_t k,
                         const int64_t* rows, int64_t nrows,
                         int32_t* idx, double* gate, double* topval, double* next,
                         int32_t nthreads) {
    if (!x || !R1 || !R2 || !idx || !gate || !topval || !next) return ORACLE_ERR_ARG;
    if (!check_shape(T, h, r, M, k, rows, nrows)) return ORACLE_ERR_ARG;
    int64_t n = rows ? nrows : T;
    double* r1 = (double*)malloc(sizeof(double) * (size_t)h * (size_t)r);
    double* r2 = (double*)malloc(sizeof(double) * (size_t)r * (size_t)M);
    if (!r1 || !r2) {
        free(r1);
        free(r2);
        return ORACLE_ERR_NOMEM;
    }
    int ok = decode_all(R1, (int64_t)h * r, r1) & decode_all(R2, (int64_t)r * M, r2);
    int status = ok ? ORACLE_OK : ORACLE_ERR_NONFINITE;
    if (status == ORACLE_OK) {
#ifdef _OPENMP
        if (nthreads > 0) omp_set_num_threads(nthreads);
#endif
#pragma omp parallel
        {
            double* xrow = (double*)malloc(sizeof(double) * (size_t)h);
            double* z = (double*)malloc(sizeof(double) * (size_t)r);
            double* logit = (double*)malloc(sizeof(double) * (size_t)M);
            candidate* work = (candidate*)malloc(sizeof(candidate) * (size_t)M);
            int local_ok = xrow && z && logit && work;
#pragma omp for schedule(dynamic, 4)
            for (int64_t t = 0; t < n; ++t) {
                if (!local_ok) continue;
                int64_t tok = rows ? rows[t] : t;
                if (!decode_all(x + tok * (int64_t)h, h, xrow)) {
#pragma omp atomic write
                    status = ORACLE_ERR_NONFINITE;
                    continue;
                }
                /* step 2: z = x R1 */
                for (int32_t i = 0; i < r; ++i) z[i] = 0.0;
                for (int32_t j = 0; j < h; ++j) {
                    const double* r1row = r1 + (int64_t)j * r;
                    for (int32_t i = 0; i < r; ++i) z[i] += xrow[j] * r1row[i];
                }
                /* step 3: logits = z R2 */
                for (int32_t e = 0; e < M; ++e) logit[e] = 0.0;
                for (int32_t i = 0; i < r; ++i) {
                    const double* r2row = r2 + (int64_t)i * M;
                    for (int32_t e = 0; e < M; ++e) logit[e] += z[i] * r2row[e];
                }
                /* steps 4-6 */
                select_and_gate(logit, M, k, work, idx + t * k, gate + t * k, topval + t * k,
                                next + t);
            }
            if (!local_ok) {
#pragma omp atomic write
                status = ORACLE_ERR_NOMEM;
            }
            free(xrow);
            free(z);
            free(logit);
            free(work);
        }
    }
    free(r1);
    free(r2);
    return status;
}

/*
 * Logits at chosen (token, expert) pairs, for checking a selection made elsewhere against the
 * definition: out[i][j] = l_{rows[i], experts[i][j]} with z and the logit summed exactly as in
 * steps 2 and 3 above (z over h in increasing order, the logit over r in increasing order), so
 * every value equals the corresponding logit of oracle_route_lowrank bit for bit.
 * x, R1, R2 as in oracle_route_lowrank; rows [nrows] token ids; experts [nrows][m] ids in
 * [0, M); out double [nrows][m].
 */
int oracle_logits_at(const uint16_t* x, const uint16_t* R1, const uint16_t* R2, int64_t T,
                     int32_t h, int32_t r, int32_t M, const int64_t* rows, int64_t nrows,
                     const int32_t* experts, int32_t m, double* out, int32_t nthreads) {
    if (!x || !R1 || !R2 || !rows || !experts || !out || m < 0) return ORACLE_ERR_ARG;
    if (!check_shape(T, h, r, M, 1, rows, nrows)) return ORACLE_ERR_ARG;
    for (int64_t i = 0; i < nrows * (int64_t)m; ++i)
        if (experts[i] < 0 || experts[i] >= M) return ORACLE_ERR_ARG;
    double* r1 = (double*)malloc(sizeof(double) * (size_t)h * (size_t)r);
    double* r2 = (double*)malloc(sizeof(double) * (size_t)r * (size_t)M);
    if (!r1 || !r2) {
        free(r1);
        free(r2);
        return ORACLE_ERR_NOMEM;
    }
    int ok = decode_all(R1, (int64_t)h * r, r1) & decode_all(R2, (int64_t)r * M, r2);
    int status = ok ? ORACLE_OK : ORACLE_ERR_NONFINITE;
    if (status == ORACLE_OK) {
#ifdef _OPENMP
        if (nthreads > 0) omp_set_num_threads(nthreads);
#endif
#pragma omp parallel
        {
            double* xrow = (double*)malloc(sizeof(double) * (size_t)h);
            double* z = (double*)malloc(sizeof(double) * (size_t)r);
            int local_ok = xrow && z;
#pragma omp for schedule(dynamic, 16)
            for (int64_t t = 0; t < nrows; ++t) {
                if (!local_ok) continue;
                if (!decode_all(x + rows[t] * (int64_t)h, h, xrow)) {
#pragma omp atomic write
                    status = ORACLE_ERR_NONFINITE;
                    continue;
                }
                for (int32_t i = 0; i < r; ++i) z[i] = 0.0;
                for (int32_t j = 0; j < h; ++j) {
                    const double* w1 = r1 + (int64_t)j * r; /* row j of R1 */
                    for (int32_t i = 0; i < r; ++i) z[i] += xrow[j] * w1[i];
                }
                for (int32_t j = 0; j < m; ++j) {
                    const int64_t e = experts[t * m + j];
                    double l = 0.0;
                    for (int32_t i = 0; i < r; ++i) l += z[i] * r2[(int64_t)i * M + e];
                    out[t * m + j] = l;
                }
            }
            if (!local_ok) {
#pragma omp atomic write
                status = ORACLE_ERR_NOMEM;
            }
            free(xrow);
            free(z);
        }
    }
    free(r1);
    free(r2);
    return status;
}

/* Shared body of the two full-rank entry points; W is already decoded to double [h][M]. */
static int fullrank_body(const uint16_t* x, const double* W, int64_t T, int32_t h, int32_t M,
                         int32_t k, const int64_t* rows, int64_t nrows, int32_t* idx,
                         double* gate, double* topval, double* next, int32_t nthreads) {
    int64_t n = rows ? nrows : T;
    int status = ORACLE_OK;
#ifdef _OPENMP
    if (nthreads > 0) omp_set_num_threads(nthreads);
#endif
#pragma omp parallel
    {
        double* xrow = (double*)malloc(sizeof(double) * (size_t)h);
        double* logit = (double*)malloc(sizeof(double) * (size_t)M);
        candidate* work = (candidate*)malloc(sizeof(candidate) * (size_t)M);
        int local_ok = xrow && logit && work;
#pragma omp for schedule(dynamic, 4)
        for (int64_t t = 0; t < n; ++t) {
            if (!local_ok) continue;
            int64_t tok = rows ? rows[t] : t;
            if (!decode_all(x + tok * (int64_t)h, h, xrow)) {
#pragma omp atomic write
                status = ORACLE_ERR_NONFINITE;
                continue;
            }
            for (int32_t e = 0; e < M; ++e) logit[e] = 0.0;
            for (int32_t j = 0; j < h; ++j) {
                const double* wrow = W + (int64_t)j * M;
                for (int32_t e = 0; e < M; ++e) logit[e] += xrow[j] * wrow[e];
            }
            select_and_gate(logit, M, k, work, idx + t * k, gate + t * k, topval + t * k, next + t);
        }
        if (!local_ok) {
#pragma omp atomic write
            status = ORACLE_ERR_NOMEM;
        }
        free(xrow);
        free(logit);
        free(work);
    }
    return status;
}

/* Full-rank router with W given in double, [h][M] row-major. */
int oracle_route_fullrank_f64(const uint16_t* x, const double* W, int64_t T, int32_t h,
                              int32_t M, int32_t k, const int64_t* rows, int64_t nrows,
                              int32_t* idx, double* gate, double* topval, double* next,
                              int32_t nthreads) {
    if (!x || !W || !idx || !gate || !topval || !next) return ORACLE_ERR_ARG;
    if (!check_shape(T, h, 1, M, k, rows, nrows)) return ORACLE_ERR_ARG;
    for (int64_t i = 0; i < (int64_t)h * M; ++i)
        if (!isfinite(W[i])) return ORACLE_ERR_NONFINITE;
    return fullrank_body(x, W, T, h, M, k, rows, nrows, idx, gate, topval, next, nthreads);
}

/* Full-rank router with W given as bf16 bit patterns, [h][M] row-major. */
int oracle_route_fullrank_bf16(const uint16_t* x, const uint16_t* W, int64_t T, int32_t h,
                               int32_t M, int32_t k, const int64_t* rows, int64_t nrows,
                               int32_t* idx, double* gate, double* topval, double* next,
                               int32_t nthreads) {
    if (!x || !W || !idx || !gate || !topval || !next) return ORACLE_ERR_ARG;
    if (!check_shape(T, h, 1, M, k, rows, nrows)) return ORACLE_ERR_ARG;
    double* w = (double*)malloc(sizeof(double) * (size_t)h * (size_t)M);
    if (!w) return ORACLE_ERR_NOMEM;
    int status = decode_all(W, (int64_t)h * M, w)
                     ? fullrank_body(x, w, T, h, M, k, rows, nrows, idx, gate, topval, next,
                                     nthreads)
                     : ORACLE_ERR_NONFINITE;
    free(w);
    return status;
}

/*
 * Full-rank logits at chosen (token, expert) pairs: out[i][j] = sum_h x[rows[i]][h] W[h][e]
 * with e = experts[i][j], W given as bf16 bits [h][M], summed over h in increasing order as
 * the full-rank router above does, so the values equal its logits bit for bit.
 */
int oracle_fullrank_logits_at(const uint16_t* x, const uint16_t* W, int64_t T, int32_t h,
                              int32_t M, const int64_t* rows, int64_t nrows,
                              const int32_t* experts, int32_t m, double* out) {
    if (!x || !W || !rows || !experts || !out || m < 0) return ORACLE_ERR_ARG;
    if (!check_shape(T, h, 1, M, 1, rows, nrows)) return ORACLE_ERR_ARG;
    for (int64_t i = 0; i < nrows * (int64_t)m; ++i)
        if (experts[i] < 0 || experts[i] >= M) return ORACLE_ERR_ARG;
    for (int64_t t = 0; t < nrows; ++t) {
        const uint16_t* xr = x + rows[t] * (int64_t)h;
        for (int32_t j = 0; j < m; ++j) {
            const int64_t e = experts[t * m + j];
            double l = 0.0;
            for (int32_t q = 0; q < h; ++q) {
                const double xv = bf16_bits_to_double(xr[q]);
                const double wv = bf16_bits_to_double(W[(int64_t)q * M + e]);
                if (!isfinite(xv) || !isfinite(wv)) return ORACLE_ERR_NONFINITE;
                l += xv * wv;
            }
            out[t * m + j] = l;
        }
    }
    return ORACLE_OK;
}

/* counts[e] = number of (token, slot) pairs with idx == e.  Out-of-range ids -> error. */
/*
 * Dispatch bookkeeping of the MoE layer ("Sort + Count" of the layer's forward-pass figure in the
 * efficiency appendix: the (N, k) expert ids become N k sorted positions plus per-expert
 * offsets).  The N k entries of idx are numbered p = t k + j in row-major order.  Each entry's
 * key is its expert id, or M for an id outside [0, M) (such entries go after every expert).
 *   offsets[e] = number of entries whose key is below e, for e = 0 .. M (offsets[M] is the
 *                number of valid entries);
 *   sorted[i]  = the positions ordered by key, positions in increasing order within a key
 *                (a stable counting sort: each key's entries are placed in position order,
 *                starting at its offset).
 * offsets int64 [M + 1]; sorted int64 [N k].
 */
/*
 * Softmax statistics of the training forward pass (Appendix "Pseudocode", training forward:
 * the row softmax P of the logits, eq. app_softmax; its column sums psum, eq. app_psum; the row
 * maximum m and the normaliser Z that the online softmax keeps, eq. app_online):
 *   m[t]    = max_e l_t[e]
 *   Z[t]    = sum_e exp(l_t[e] - m[t])
 *   psum[e] = sum_t exp(l_t[e] - m[t]) / Z[t]
 * with the logits l = x R1 R2 of steps 2-3 above, in fp64 over all M experts.  x, R1, R2 as
 * in oracle_route_lowrank; m, Z double [T]; psum double [M].  Tokens are summed into psum in
 * increasing order within fixed blocks of 64 tokens, then block by block, so the result does
 * not depend on the thread count.
 */
int oracle_route_stats(const uint16_t* x, const uint16_t* R1, const uint16_t* R2, int64_t T,
                       int32_t h, int32_t r, int32_t M, double* m, double* Z, double* psum,
                       int32_t nthreads) {
    if (!x || !R1 || !R2 || !m || !Z || !psum) return ORACLE_ERR_ARG;
    if (T < 0 || h <= 0 || r <= 0 || M <= 0) return ORACLE_ERR_ARG;
    const int64_t nb = (T + 63) / 64;
    double* f1 = (double*)malloc(sizeof(double) * (size_t)h * (size_t)r);
    double* f2 = (double*)malloc(sizeof(double) * (size_t)r * (size_t)M);
    double* part = (double*)calloc((size_t)(nb > 0 ? nb : 1) * (size_t)M, sizeof(double));
    if (!f1 || !f2 || !part) {
        free(f1);
        free(f2);
        free(part);
        return ORACLE_ERR_NOMEM;
    }
    int ok = decode_all(R1, (int64_t)h * r, f1) & decode_all(R2, (int64_t)r * M, f2);
    int status = ok ? ORACLE_OK : ORACLE_ERR_NONFINITE;
    if (status == ORACLE_OK) {
#ifdef _OPENMP
        if (nthreads > 0) omp_set_num_threads(nthreads);
#endif
#pragma omp parallel
        {
            double* xs = (double*)malloc(sizeof(double) * (size_t)h);
            double* zz = (double*)malloc(sizeof(double) * (size_t)r);
            double* lg = (double*)malloc(sizeof(double) * (size_t)M);
            int local_ok = xs && zz && lg;
#pragma omp for schedule(dynamic, 1)
            for (int64_t b = 0; b < nb; ++b) {
                if (!local_ok) continue;
                double* pb = part + b * (int64_t)M;
                for (int64_t t = 64 * b; t < T && t < 64 * b + 64; ++t) {
                    if (!decode_all(x + t * (int64_t)h, h, xs)) {
#pragma omp atomic write
                        status = ORACLE_ERR_NONFINITE;
                        continue;
                    }
                    for (int32_t i = 0; i < r; ++i) zz[i] = 0.0;
                    for (int32_t j = 0; j < h; ++j)
                        for (int32_t i = 0; i < r; ++i) zz[i] += xs[j] * f1[(int64_t)j * r + i];
                    for (int32_t e = 0; e < M; ++e) lg[e] = 0.0;
                    for (int32_t i = 0; i < r; ++i)
                        for (int32_t e = 0; e < M; ++e) lg[e] += zz[i] * f2[(int64_t)i * M + e];
                    double mx = lg[0];
                    for (int32_t e = 1; e < M; ++e) mx = lg[e] > mx ? lg[e] : mx;
                    double zs = 0.0;
                    for (int32_t e = 0; e < M; ++e) zs += exp(lg[e] - mx);
                    m[t] = mx;
                    Z[t] = zs;
                    for (int32_t e = 0; e < M; ++e) pb[e] += exp(lg[e] - mx) / zs;
                }
            }
            if (!local_ok) {
#pragma omp atomic write
                status = ORACLE_ERR_NOMEM;
            }
            free(xs);
            free(zz);
            free(lg);
        }
        for (int32_t e = 0; e < M; ++e) psum[e] = 0.0;
        for (int64_t b = 0; b < nb; ++b)
            for (int32_t e = 0; e < M; ++e) psum[e] += part[b * (int64_t)M + e];
    }
    free(f1);
    free(f2);
    free(part);
    return status;
}

/* Key of an entry: its expert id, or M when the id lies outside [0, M). */
static int32_t dispatch_key(int32_t e, int32_t M) { return (e >= 0 && e < M) ? e : M; }

int oracle_dispatch_sort(const int32_t* idx, int64_t n, int32_t k, int32_t M, int64_t* offsets,
                         int64_t* sorted) {
    if (!idx || !offsets || !sorted || n < 0 || k < 1 || M < 1) return ORACLE_ERR_ARG;
    const int64_t N = n * (int64_t)k;
    int64_t* start = (int64_t*)calloc((size_t)M + 2, sizeof(int64_t));
    if (!start) return ORACLE_ERR_NOMEM;
    /* count the entries of each key */
    for (int64_t p = 0; p < N; ++p) start[dispatch_key(idx[p], M) + 1] += 1;
    /* first slot of each key: the number of entries with a smaller key */
    for (int32_t e = 0; e <= M; ++e) start[e + 1] += start[e];
    for (int32_t e = 0; e <= M; ++e) offsets[e] = start[e];
    /* place the positions in increasing order */
    for (int64_t p = 0; p < N; ++p) {
        const int32_t key = dispatch_key(idx[p], M);
        sorted[start[key]] = p;
        start[key] += 1;
    }
    free(start);
    return ORACLE_OK;
}

int oracle_histogram(const int32_t* idx, int64_t n, int32_t k, int32_t M, int64_t* counts) {
    if (!idx || !counts || n < 0 || k < 1 || M < 1) return ORACLE_ERR_ARG;
    for (int32_t e = 0; e < M; ++e) counts[e] = 0;
    for (int64_t i = 0; i < n * (int64_t)k; ++i) {
        if (idx[i] < 0 || idx[i] >= M) return ORACLE_ERR_ARG;
        counts[idx[i]] += 1;
    }
    return ORACLE_OK;
}

/*
 * Training backward pass of the low-rank router (Appendix "Pseudocode", backward pass: eqs.
 * app_chain, app_jac and app_kernelgrad and the backward algorithm with recompute), in this
 * file's orientation x [T][h], R1 [h][r], R2 [r][M] (the paper's appendix names the expert
 * factor R1 [M][r], which is R2^T here, and the hidden factor R2 [r][h], which is R1^T here).
 * Inputs: the selection idx [T][k]; dtop [T][k], the gradient of the loss with respect to the
 * selected logits l_t[idx[t][j]]; pbar [M], the gradient with respect to psum (NULL: no
 * balancing term); m [T] and Z [T], the saved softmax statistics (read only when pbar is given).
 * Per token t:
 *   z_t      = x_t R1
 *   l_t[e]   = z_t R2[:, e]
 *   P_te     = exp(l_t[e] - m_t) / Z_t
 *   g_t      = sum_e pbar_e P_te                                  (eq. app_kernelgrad)
 *   ybar_te  = P_te (pbar_e - g_t), then dtop[t][j] added at e = idx[t][j] for j = 0 .. k-1
 *   dz_t[i]  = sum_e ybar_te R2[i][e]
 *   dx_t[c]  = sum_i dz_t[i] R1[c][i]
 * and over all tokens
 *   dR1[c][i] = sum_t x[t][c] dz_t[i]
 *   dR2[i][e] = sum_t z_t[i] ybar_te
 * Entries of idx outside [0, M) add nothing.  Every sum runs in increasing order of its index
 * (t, e, i or j), so the result does not depend on the thread count.  g [T] and dz [T][r] are
 * outputs too (g is 0 without pbar).
 */
int oracle_route_backward(const uint16_t* x, const uint16_t* R1, const uint16_t* R2, int64_t T,
                          int32_t h, int32_t r, int32_t M, int32_t k, const int32_t* idx,
                          const double* dtop, const double* pbar, const double* m,
                          const double* Z, double* dx, double* dR1, double* dR2, double* g,
                          double* dz, int32_t nthreads) {
    if (!x || !R1 || !R2 || !dR1 || !dR2) return ORACLE_ERR_ARG;
    if (T < 0 || h <= 0 || r <= 0 || M <= 0 || k < 1) return ORACLE_ERR_ARG;
    if (T > 0 && (!idx || !dtop || !dx || !g || !dz || (pbar && (!m || !Z)))) return ORACLE_ERR_ARG;
    for (int64_t i = 0; i < T * (int64_t)k; ++i)
        if (!isfinite(dtop[i])) return ORACLE_ERR_NONFINITE;
    if (pbar) {
        for (int32_t e = 0; e < M; ++e)
            if (!isfinite(pbar[e])) return ORACLE_ERR_NONFINITE;
        for (int64_t t = 0; t < T; ++t) {
            if (!isfinite(m[t]) || !isfinite(Z[t])) return ORACLE_ERR_NONFINITE;
            if (!(Z[t] > 0.0)) return ORACLE_ERR_ARG;
        }
    }
    double* f1 = (double*)malloc(sizeof(double) * (size_t)h * (size_t)r);
    double* f2 = (double*)malloc(sizeof(double) * (size_t)r * (size_t)M);
    double* zall = (double*)malloc(sizeof(double) * (size_t)(T > 0 ? T : 1) * (size_t)r);
    if (!f1 || !f2 || !zall) {
        free(f1);
        free(f2);
        free(zall);
        return ORACLE_ERR_NOMEM;
    }
    int status = (decode_all(R1, (int64_t)h * r, f1) & decode_all(R2, (int64_t)r * M, f2))
                     ? ORACLE_OK
                     : ORACLE_ERR_NONFINITE;
#ifdef _OPENMP
    if (nthreads > 0) omp_set_num_threads(nthreads);
#endif
    /* Per token: z, the logits, P, g, ybar, dz and dx. */
    if (status == ORACLE_OK) {
#pragma omp parallel
        {
            double* xs = (double*)malloc(sizeof(double) * (size_t)h);
            double* lg = (double*)malloc(sizeof(double) * (size_t)M);
            double* yb = (double*)malloc(sizeof(double) * (size_t)M);
            int local_ok = xs && lg && yb;
#pragma omp for schedule(dynamic, 4)
            for (int64_t t = 0; t < T; ++t) {
                if (!local_ok) continue;
                if (!decode_all(x + t * (int64_t)h, h, xs)) {
#pragma omp atomic write
                    status = ORACLE_ERR_NONFINITE;
                    continue;
                }
                double* zt = zall + t * (int64_t)r;
                for (int32_t i = 0; i < r; ++i) zt[i] = 0.0;
                for (int32_t c = 0; c < h; ++c)
                    for (int32_t i = 0; i < r; ++i) zt[i] += xs[c] * f1[(int64_t)c * r + i];
                double gt = 0.0;
                if (pbar) {
                    for (int32_t e = 0; e < M; ++e) lg[e] = 0.0;
                    for (int32_t i = 0; i < r; ++i)
                        for (int32_t e = 0; e < M; ++e) lg[e] += zt[i] * f2[(int64_t)i * M + e];
                    for (int32_t e = 0; e < M; ++e) lg[e] = exp(lg[e] - m[t]) / Z[t];  /* P */
                    for (int32_t e = 0; e < M; ++e) gt += pbar[e] * lg[e];
                    for (int32_t e = 0; e < M; ++e) yb[e] = lg[e] * (pbar[e] - gt);
                } else {
                    for (int32_t e = 0; e < M; ++e) yb[e] = 0.0;
                }
                for (int32_t j = 0; j < k; ++j) {
                    const int32_t e = idx[t * k + j];
                    if (e >= 0 && e < M) yb[e] += dtop[t * k + j];
                }
                g[t] = gt;
                double* dzt = dz + t * (int64_t)r;
                for (int32_t i = 0; i < r; ++i) {
                    double s = 0.0;
                    for (int32_t e = 0; e < M; ++e) s += yb[e] * f2[(int64_t)i * M + e];
                    dzt[i] = s;
                }
                double* dxt = dx + t * (int64_t)h;
                for (int32_t c = 0; c < h; ++c) {
                    double s = 0.0;
                    for (int32_t i = 0; i < r; ++i) s += dzt[i] * f1[(int64_t)c * r + i];
                    dxt[c] = s;
                }
            }
            if (!local_ok) {
#pragma omp atomic write
                status = ORACLE_ERR_NOMEM;
            }
            free(xs);
            free(lg);
            free(yb);
        }
    }
    /* dR2 = z^T ybar: blocks of 64 experts, every token in order, ybar recomputed as above. */
    const int32_t EB = 64;
    if (status == ORACLE_OK) {
        const int32_t nblk = (M + EB - 1) / EB;
#pragma omp parallel
        {
            double* acc = (double*)malloc(sizeof(double) * (size_t)EB * (size_t)r);
            double* yb = (double*)malloc(sizeof(double) * (size_t)EB);
            int local_ok = acc && yb;
#pragma omp for schedule(dynamic, 1)
            for (int32_t b = 0; b < nblk; ++b) {
                if (!local_ok) continue;
                const int32_t e0 = b * EB, e1 = (e0 + EB < M) ? e0 + EB : M;
                for (int64_t q = 0; q < (int64_t)EB * r; ++q) acc[q] = 0.0;
                for (int64_t t = 0; t < T; ++t) {
                    const double* zt = zall + t * (int64_t)r;
                    for (int32_t e = e0; e < e1; ++e) {
                        double y = 0.0;
                        if (pbar) {
                            double l = 0.0;
                            for (int32_t i = 0; i < r; ++i) l += zt[i] * f2[(int64_t)i * M + e];
                            const double p = exp(l - m[t]) / Z[t];
                            y = p * (pbar[e] - g[t]);
                        }
                        yb[e - e0] = y;
                    }
                    for (int32_t j = 0; j < k; ++j) {
                        const int32_t e = idx[t * k + j];
                        if (e >= e0 && e < e1) yb[e - e0] += dtop[t * k + j];
                    }
                    for (int32_t e = e0; e < e1; ++e)
                        for (int32_t i = 0; i < r; ++i)
                            acc[(int64_t)(e - e0) * r + i] += zt[i] * yb[e - e0];
                }
                for (int32_t e = e0; e < e1; ++e)
                    for (int32_t i = 0; i < r; ++i)
                        dR2[(int64_t)i * M + e] = acc[(int64_t)(e - e0) * r + i];
            }
            if (!local_ok) {
#pragma omp atomic write
                status = ORACLE_ERR_NOMEM;
            }
            free(acc);
            free(yb);
        }
    }
    /* dR1 = x^T dz: blocks of 64 hidden columns, every token in order. */
    const int32_t CB = 64;
    if (status == ORACLE_OK) {
        const int32_t nblk = (h + CB - 1) / CB;
#pragma omp parallel
        {
            double* acc = (double*)malloc(sizeof(double) * (size_t)CB * (size_t)r);
            double* xs = (double*)malloc(sizeof(double) * (size_t)CB);
            int local_ok = acc && xs;
#pragma omp for schedule(dynamic, 1)
            for (int32_t b = 0; b < nblk; ++b) {
                if (!local_ok) continue;
                const int32_t c0 = b * CB, c1 = (c0 + CB < h) ? c0 + CB : h;
                for (int64_t q = 0; q < (int64_t)CB * r; ++q) acc[q] = 0.0;
                for (int64_t t = 0; t < T; ++t) {
                    decode_all(x + t * (int64_t)h + c0, c1 - c0, xs);
                    const double* dzt = dz + t * (int64_t)r;
                    for (int32_t c = c0; c < c1; ++c)
                        for (int32_t i = 0; i < r; ++i)
                            acc[(int64_t)(c - c0) * r + i] += xs[c - c0] * dzt[i];
                }
                for (int32_t c = c0; c < c1; ++c)
                    for (int32_t i = 0; i < r; ++i)
                        dR1[(int64_t)c * r + i] = acc[(int64_t)(c - c0) * r + i];
            }
            if (!local_ok) {
#pragma omp atomic write
                status = ORACLE_ERR_NOMEM;
            }
            free(acc);
            free(xs);
        }
    }
    free(f1);
    free(f2);
    free(zall);
    return status;
}
