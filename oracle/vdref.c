/*
 * vdref.c -- reference oracle for the ValueDiff eviction pass.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product path may link, load or
 * call this file; only the test suite, the smoke check and the CPU-baseline
 * leg of the benchmark do.  It shares no source, header, table or helper with
 * the HIP library.
 *
 * Everything is computed in double precision with plain loops, one unit
 * (sequence, layer, KV head) at a time, in the order the paper states:
 *
 *   1. mean of the n cached value vectors, v_bar = (1/n) sum_i v_i
 *      (Sec. 3.2, Eq. vd; the n cached tokens include the block just
 *      appended, Sec. 2.2, Eq. block_processing);
 *   2. a score per token (Sec. 3.2):
 *        L2   s_j = ||v_j - v_bar||                       (Eq. vd)
 *        Dir  s_j = 1 - cos(v_j, v_bar)                   (variant after Eq. decomp)
 *        Norm s_j = ||v_j||                               (variant after Eq. decomp)
 *   3. keep the N highest scores whenever n exceeds the budget N
 *      (Sec. 2.1, Eq. eviction), ties going to the lower slot index;
 *   4. gather K and V onto the kept set with the slot-reuse layout: the
 *      evicted slots below N, ascending, receive the kept slots at or above N,
 *      ascending (the layout reading of "gather" used by this project).
 *
 * Key-side scores (Sec. 4, Baselines, key geometry): the same three scores
 * taken on the key rows instead of the value rows -- L2 on K (ManifoldKV),
 * Dir on K (KeyDiff) and Norm on K (KeyNorm), the last keeping the SMALLEST
 * norms (the opposite radial preference to the value-side Norm).
 *
 * Decode attention of one query row (Sec. 2.1, Eq. attention; grouped-query
 * heads share a KV head): softmax of the scaled dot products with every cached
 * key, applied to the values, in fp64.
 *
 * FastCAOTE scores of one decode step (App. A, Eq. app_fastcaote; Sec. 4,
 * Baselines): s_j = a_j / (1 - a_j) * ||v_j - v_bar||, where a_j is the
 * observed attention weight of row j, taken as the mean over the G query
 * heads of the KV head of their softmax weights (a reading: the paper does
 * not say how grouped heads combine), and +infinity when a_j = 1.
 *
 * Geometry diagnostics of one unit (Sec. 3.1 and the bos-cosim equation of
 * Sec. 4), from their definitions: sigma_X = std_i ||x_i - x_bar|| for X = K
 * and V (the population standard deviation over the n tokens), the mean of
 * those distances, and bos-cosim = cos(k_0, (1/(n-1)) sum_{i>0} k_i).
 *
 * Readings of points the paper leaves open:
 *   - Dir when ||v_j|| * ||v_bar|| == 0: cos is taken as 0, so s_j = 1.
 *   - Norm keeps the largest norms.
 *   - n <= N is a no-op (eviction happens only when the cache exceeds N).
 *   - std is the population one (divide by n); bos-cosim is 0 when either
 *     vector is zero or n < 2.
 *
 * Pins: every function here is checked by the CPU tests against identities
 * and brute force that do not reuse this code (minimal-disturbance identity
 * of Sec. 3.3 Eq. recon_error, law of cosines Eq. decomp, the Dirichlet
 * closed form of App. A Eq. app_claim, invariances, brute-force subset
 * search, hand-worked examples).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

#define VDREF_BF16 0
#define VDREF_F32 1

#define VDREF_L2 0
#define VDREF_DIR 1
#define VDREF_NORM 2
#define VDREF_KEY_L2 3
#define VDREF_KEY_DIR 4
#define VDREF_KEY_NORM 5

#define VDREF_OK 0
#define VDREF_BAD_ARG 1

/* ---- element access ---------------------------------------------------- */

/* A bfloat16 number is the upper half of an IEEE binary32 number. */
static double bf16_bits_to_double(uint16_t bits)
{
    uint32_t w = ((uint32_t)bits) << 16;
    float f;
    memcpy(&f, &w, sizeof f);
    return (double)f;
}

static double get_elem(const void *rows, int dtype, int64_t idx)
{
    if (dtype == VDREF_BF16)
        return bf16_bits_to_double(((const uint16_t *)rows)[idx]);
    return (double)((const float *)rows)[idx];
}

static size_t elem_size(int dtype) { return dtype == VDREF_BF16 ? 2 : 4; }

/* Exposed for the decoding pin. */
double vdref_decode_elem(const void *rows, int dtype, int64_t idx)
{
    return get_elem(rows, dtype, idx);
}

/* ---- step 1: mean (Sec. 3.2, Eq. vd) ----------------------------------- */

/* v: n rows of d elements, row r starting at element r*row_stride. */
int vdref_mean(const void *v, int dtype, int64_t n, int d, int64_t row_stride,
               double *mean)
{
    if (n <= 0 || d <= 0 || !v || !mean)
        return VDREF_BAD_ARG;
    for (int c = 0; c < d; ++c) {
        double sum = 0.0;
        for (int64_t i = 0; i < n; ++i)
            sum += get_elem(v, dtype, i * row_stride + c);
        mean[c] = sum / (double)n;
    }
    return VDREF_OK;
}

/* ---- step 2: scores (Sec. 3.2) ----------------------------------------- */

/* The rows `v` are the scored rows: value rows for the value-side scores,
 * key rows for the key-side ones (which take the same three forms). */
int vdref_score(const void *v, int dtype, int64_t n, int d, int64_t row_stride,
                int variant, double *scores, double *mean_out)
{
    if (n <= 0 || d <= 0 || !v || !scores)
        return VDREF_BAD_ARG;
    if (variant < VDREF_L2 || variant > VDREF_KEY_NORM)
        return VDREF_BAD_ARG;
    if (variant >= VDREF_KEY_L2)
        variant -= VDREF_KEY_L2;

    double *mean = (double *)malloc(sizeof(double) * (size_t)d);
    if (!mean)
        return VDREF_BAD_ARG;
    vdref_mean(v, dtype, n, d, row_stride, mean);

    double mean_norm2 = 0.0;
    for (int c = 0; c < d; ++c)
        mean_norm2 += mean[c] * mean[c];
    double mean_norm = sqrt(mean_norm2);

    for (int64_t j = 0; j < n; ++j) {
        if (variant == VDREF_L2) {
            /* s_j = || v_j - v_bar || */
            double acc = 0.0;
            for (int c = 0; c < d; ++c) {
                double diff = get_elem(v, dtype, j * row_stride + c) - mean[c];
                acc += diff * diff;
            }
            scores[j] = sqrt(acc);
        } else if (variant == VDREF_NORM) {
            /* s_j = || v_j || */
            double acc = 0.0;
            for (int c = 0; c < d; ++c) {
                double x = get_elem(v, dtype, j * row_stride + c);
                acc += x * x;
            }
            scores[j] = sqrt(acc);
        } else {
            /* s_j = 1 - cos(v_j, v_bar), cos := 0 when either norm is zero */
            double dot = 0.0, vn2 = 0.0;
            for (int c = 0; c < d; ++c) {
                double x = get_elem(v, dtype, j * row_stride + c);
                dot += x * mean[c];
                vn2 += x * x;
            }
            double denom = sqrt(vn2) * mean_norm;
            double cosv = denom > 0.0 ? dot / denom : 0.0;
            scores[j] = 1.0 - cosv;
        }
    }
    if (mean_out)
        memcpy(mean_out, mean, sizeof(double) * (size_t)d);
    free(mean);
    return VDREF_OK;
}

/* ---- step 3: top-N (Sec. 2.1, Eq. eviction) ---------------------------- */

typedef struct {
    double s;
    int64_t j;
} scored_index;

/* Higher score first; equal scores: lower index first. */
static int by_score_desc_index_asc(const void *pa, const void *pb)
{
    const scored_index *a = (const scored_index *)pa;
    const scored_index *b = (const scored_index *)pb;
    if (a->s > b->s)
        return -1;
    if (a->s < b->s)
        return 1;
    if (a->j < b->j)
        return -1;
    if (a->j > b->j)
        return 1;
    return 0;
}

/* keep[j] = 1 for the N kept slots, 0 otherwise, for j < n. */
int vdref_select_topn(const double *scores, int64_t n, int64_t N, uint8_t *keep)
{
    if (n < 0 || N < 1 || !keep || (n > 0 && !scores))
        return VDREF_BAD_ARG;
    if (n <= N) {
        for (int64_t j = 0; j < n; ++j)
            keep[j] = 1;
        return VDREF_OK;
    }
    scored_index *order = (scored_index *)malloc(sizeof(scored_index) * (size_t)n);
    if (!order)
        return VDREF_BAD_ARG;
    for (int64_t j = 0; j < n; ++j) {
        order[j].s = scores[j];
        order[j].j = j;
    }
    qsort(order, (size_t)n, sizeof(scored_index), by_score_desc_index_asc);
    for (int64_t j = 0; j < n; ++j)
        keep[j] = 0;
    for (int64_t r = 0; r < N; ++r)
        keep[order[r].j] = 1;
    free(order);
    return VDREF_OK;
}

/* Lower score first; equal scores: lower index first. */
static int by_score_asc_index_asc(const void *pa, const void *pb)
{
    const scored_index *a = (const scored_index *)pa;
    const scored_index *b = (const scored_index *)pb;
    if (a->s < b->s)
        return -1;
    if (a->s > b->s)
        return 1;
    if (a->j < b->j)
        return -1;
    if (a->j > b->j)
        return 1;
    return 0;
}

/* keep[j] = 1 for the N slots of smallest score (KeyNorm), ties to the lower index. */
int vdref_select_smallest(const double *scores, int64_t n, int64_t N, uint8_t *keep)
{
    if (n < 0 || N < 1 || !keep || (n > 0 && !scores))
        return VDREF_BAD_ARG;
    if (n <= N) {
        for (int64_t j = 0; j < n; ++j)
            keep[j] = 1;
        return VDREF_OK;
    }
    scored_index *order = (scored_index *)malloc(sizeof(scored_index) * (size_t)n);
    if (!order)
        return VDREF_BAD_ARG;
    for (int64_t j = 0; j < n; ++j) {
        order[j].s = scores[j];
        order[j].j = j;
    }
    qsort(order, (size_t)n, sizeof(scored_index), by_score_asc_index_asc);
    for (int64_t j = 0; j < n; ++j)
        keep[j] = 0;
    for (int64_t r = 0; r < N; ++r)
        keep[order[r].j] = 1;
    free(order);
    return VDREF_OK;
}

/* ---- step 4: gather with slot reuse ------------------------------------ */

static void copy_row(void *base, int dtype, int64_t row_stride, int d,
                     int64_t dst, int64_t src)
{
    size_t es = elem_size(dtype);
    char *b = (char *)base;
    memmove(b + (size_t)(dst * row_stride) * es, b + (size_t)(src * row_stride) * es,
            (size_t)d * es);
}

/*
 * holes  = evicted slots in [0, N), ascending
 * movers = kept slots in [N, n), ascending
 * the k-th mover's K row, V row and pos entry are copied onto the k-th hole.
 * Afterwards the kept tokens occupy slots [0, N).
 */
int vdref_compact(void *k, void *v, int dtype, int64_t n, int64_t N, int d,
                  int64_t row_stride, const uint8_t *keep, int32_t *pos)
{
    if (n < 0 || N < 1 || d <= 0 || !keep)
        return VDREF_BAD_ARG;
    if (n <= N)
        return VDREF_OK;
    int64_t next_mover = N;
    for (int64_t hole = 0; hole < N; ++hole) {
        if (keep[hole])
            continue;
        while (next_mover < n && !keep[next_mover])
            ++next_mover;
        if (next_mover >= n)
            break;
        if (k)
            copy_row(k, dtype, row_stride, d, hole, next_mover);
        if (v)
            copy_row(v, dtype, row_stride, d, hole, next_mover);
        if (pos)
            pos[hole] = pos[next_mover];
        ++next_mover;
    }
    return VDREF_OK;
}

/* ---- the whole pass over a batch of units ------------------------------ */

/*
 * k, v       : [U][cap][d] contiguous, in place (either may be NULL)
 * n_unit[u]  : cached tokens of unit u before eviction (0 <= n <= cap)
 * N_unit[u]  : budget of unit u (>= 1)
 * scores     : optional [U][cap] output (first n of each unit written)
 * keep       : optional [U][cap] output (first n of each unit written)
 * mean_out   : optional [U][d] output (units with n > 0)
 * pos        : optional [U][cap] payload moved with the rows
 * nthreads   : OpenMP threads over units (<= 0: library default)
 */
int vdref_evict_step(void *k, void *v, int dtype, int64_t U, int64_t cap, int d,
                     const int32_t *n_unit, const int32_t *N_unit, int variant,
                     double *scores, uint8_t *keep, double *mean_out,
                     int32_t *pos, int nthreads)
{
    if (U < 0 || cap < 0 || d <= 0 || !v || !n_unit || !N_unit)
        return VDREF_BAD_ARG;
    if (dtype != VDREF_BF16 && dtype != VDREF_F32)
        return VDREF_BAD_ARG;
    if (variant < VDREF_L2 || variant > VDREF_KEY_NORM)
        return VDREF_BAD_ARG;
    int key_side = variant >= VDREF_KEY_L2;
    if (key_side && !k)
        return VDREF_BAD_ARG;
    for (int64_t u = 0; u < U; ++u)
        if (n_unit[u] < 0 || n_unit[u] > cap || N_unit[u] < 1)
            return VDREF_BAD_ARG;

    size_t es = elem_size(dtype);
    int status = VDREF_OK;
#ifdef _OPENMP
    if (nthreads <= 0)
        nthreads = omp_get_max_threads();
#pragma omp parallel for schedule(dynamic, 1) num_threads(nthreads)
#endif
    for (int64_t u = 0; u < U; ++u) {
        int64_t n = n_unit[u], N = N_unit[u];
        if (n == 0)
            continue;
        char *vu = (char *)v + (size_t)(u * cap * d) * es;
        char *ku = k ? (char *)k + (size_t)(u * cap * d) * es : NULL;
        int32_t *pu = pos ? pos + u * cap : NULL;
        double *su = (double *)malloc(sizeof(double) * (size_t)n);
        uint8_t *keepu = (uint8_t *)malloc((size_t)n);
        if (!su || !keepu) {
            free(su);
            free(keepu);
            status = VDREF_BAD_ARG;
            continue;
        }
        /* the scored rows: V, or K for a key-side score */
        vdref_score(key_side ? ku : vu, dtype, n, d, d, variant, su,
                    mean_out ? mean_out + u * d : NULL);
        if (variant == VDREF_KEY_NORM)
            vdref_select_smallest(su, n, N, keepu);
        else
            vdref_select_topn(su, n, N, keepu);
        vdref_compact(ku, vu, dtype, n, N, d, d, keepu, pu);
        if (scores)
            memcpy(scores + u * cap, su, sizeof(double) * (size_t)n);
        if (keep)
            memcpy(keep + u * cap, keepu, (size_t)n);
        free(su);
        free(keepu);
    }
    return status;
}

/* ---- geometry diagnostics (Sec. 3.1, Sec. 4 bos-cosim) ----------------- */

/* Mean and population standard deviation over i of ||x_i - x_bar||. */
static void dispersion(const void *x, int dtype, int64_t n, int d, int64_t row_stride,
                       double *mean_dist, double *sigma)
{
    double *xbar = (double *)malloc(sizeof(double) * (size_t)d);
    double *dist = (double *)malloc(sizeof(double) * (size_t)n);
    if (!xbar || !dist) {
        free(xbar);
        free(dist);
        *mean_dist = *sigma = 0.0;
        return;
    }
    vdref_mean(x, dtype, n, d, row_stride, xbar);
    double sum = 0.0;
    for (int64_t i = 0; i < n; ++i) {
        double acc = 0.0;
        for (int c = 0; c < d; ++c) {
            double diff = get_elem(x, dtype, i * row_stride + c) - xbar[c];
            acc += diff * diff;
        }
        dist[i] = sqrt(acc);
        sum += dist[i];
    }
    double mu = sum / (double)n;
    double var = 0.0;
    for (int64_t i = 0; i < n; ++i)
        var += (dist[i] - mu) * (dist[i] - mu);
    *mean_dist = mu;
    *sigma = sqrt(var / (double)n);
    free(xbar);
    free(dist);
}

/*
 * out[0] = sigma_K, out[1] = sigma_V, out[2] = mean ||k_i - k_bar||,
 * out[3] = mean ||v_i - v_bar||, out[4] = bos-cosim; all zero when n == 0.
 */
int vdref_geometry(const void *k, const void *v, int dtype, int64_t n, int d,
                   int64_t row_stride, double *out)
{
    if (n < 0 || d <= 0 || !k || !v || !out)
        return VDREF_BAD_ARG;
    for (int i = 0; i < 5; ++i)
        out[i] = 0.0;
    if (n == 0)
        return VDREF_OK;
    dispersion(k, dtype, n, d, row_stride, &out[2], &out[0]);
    dispersion(v, dtype, n, d, row_stride, &out[3], &out[1]);
    if (n >= 2) {
        /* cos(k_0, (1/(n-1)) sum_{i>0} k_i) */
        double dot = 0.0, n0 = 0.0, nm = 0.0;
        for (int c = 0; c < d; ++c) {
            double m = 0.0;
            for (int64_t i = 1; i < n; ++i)
                m += get_elem(k, dtype, i * row_stride + c);
            m /= (double)(n - 1);
            double k0 = get_elem(k, dtype, c);
            dot += k0 * m;
            n0 += k0 * k0;
            nm += m * m;
        }
        double denom = sqrt(n0) * sqrt(nm);
        out[4] = denom > 0.0 ? dot / denom : 0.0;
    }
    return VDREF_OK;
}

/* ---- decode attention (Sec. 2.1, Eq. attention) ------------------------ */

/*
 * One query row of one head against rows 0 .. n-1 of its KV head:
 * out = sum_j softmax_j(scale * q . k_j) v_j.  For the newest token the causal
 * mask keeps every cached row, so it does not appear.  The largest logit is
 * subtracted before exponentiation (softmax does not change under a common
 * shift of its arguments).
 */
int vdref_attention(const double *q, const void *k, const void *v, int dtype, int64_t n,
                    int d, int64_t row_stride, double scale, double *out)
{
    if (n <= 0 || d <= 0 || !q || !k || !v || !out)
        return VDREF_BAD_ARG;
    double *w = (double *)malloc(sizeof(double) * (size_t)n);
    if (!w)
        return VDREF_BAD_ARG;
    double top = -INFINITY;
    for (int64_t j = 0; j < n; ++j) {
        double dot = 0.0;
        for (int c = 0; c < d; ++c)
            dot += q[c] * get_elem(k, dtype, j * row_stride + c);
        w[j] = scale * dot;
        if (w[j] > top)
            top = w[j];
    }
    double den = 0.0;
    for (int64_t j = 0; j < n; ++j) {
        w[j] = exp(w[j] - top);
        den += w[j];
    }
    for (int c = 0; c < d; ++c) {
        double acc = 0.0;
        for (int64_t j = 0; j < n; ++j)
            acc += w[j] * get_elem(v, dtype, j * row_stride + c);
        out[c] = acc / den;
    }
    free(w);
    return VDREF_OK;
}

/* ---- FastCAOTE scores of one decode step (App. A, Eq. app_fastcaote) -- */

/*
 * q: the G query rows of the KV head, [G][d] doubles; k, v: rows 0 .. n-1.
 * a_j = (1/G) sum_g softmax_j(scale * q_g . k_j), the observed attention of
 * row j averaged over the heads; scores[j] = a_j / (1 - a_j) * ||v_j - v_bar||
 * with v_bar the mean of the n value rows; +infinity where a_j = 1.
 */
int vdref_fastcaote_scores(const double *q, int G, const void *k, const void *v, int dtype,
                           int64_t n, int d, int64_t row_stride, double scale, double *scores)
{
    if (n <= 0 || d <= 0 || G < 1 || !q || !k || !v || !scores)
        return VDREF_BAD_ARG;
    double *a = (double *)calloc((size_t)n, sizeof(double));
    double *w = (double *)malloc(sizeof(double) * (size_t)n);
    double *dist = (double *)malloc(sizeof(double) * (size_t)n);
    if (!a || !w || !dist) {
        free(a);
        free(w);
        free(dist);
        return VDREF_BAD_ARG;
    }
    for (int g = 0; g < G; ++g) {
        /* softmax of head g over the n rows, the largest logit subtracted first */
        double top = -INFINITY;
        for (int64_t j = 0; j < n; ++j) {
            double dot = 0.0;
            for (int c = 0; c < d; ++c)
                dot += q[g * d + c] * get_elem(k, dtype, j * row_stride + c);
            w[j] = scale * dot;
            if (w[j] > top)
                top = w[j];
        }
        double den = 0.0;
        for (int64_t j = 0; j < n; ++j) {
            w[j] = exp(w[j] - top);
            den += w[j];
        }
        for (int64_t j = 0; j < n; ++j)
            a[j] += w[j] / den / (double)G;
    }
    /* the distances of the value rows to their mean (the L2 scores) */
    vdref_score(v, dtype, n, d, row_stride, VDREF_L2, dist, NULL);
    for (int64_t j = 0; j < n; ++j)
        scores[j] = a[j] < 1.0 ? a[j] / (1.0 - a[j]) * dist[j] : INFINITY;
    free(a);
    free(w);
    free(dist);
    return VDREF_OK;
}
