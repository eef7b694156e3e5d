/* Runs every function of the C oracle on small inputs (edge cases included)
 * so that the sanitizer build catches out-of-bounds accesses, leaks and
 * undefined behaviour.  Built and run by tests/test_sanitizers.py. */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

int vdref_mean(const void *v, int dtype, int64_t n, int d, int64_t row_stride, double *mean);
int vdref_score(const void *v, int dtype, int64_t n, int d, int64_t row_stride, int variant,
                double *scores, double *mean_out);
int vdref_select_topn(const double *scores, int64_t n, int64_t N, uint8_t *keep);
int vdref_select_smallest(const double *scores, int64_t n, int64_t N, uint8_t *keep);
int vdref_compact(void *k, void *v, int dtype, int64_t n, int64_t N, int d, int64_t row_stride,
                  const uint8_t *keep, int32_t *pos);
int vdref_evict_step(void *k, void *v, int dtype, int64_t U, int64_t cap, int d,
                     const int32_t *n_unit, const int32_t *N_unit, int variant, double *scores,
                     uint8_t *keep, double *mean_out, int32_t *pos, int nthreads);
int vdref_geometry(const void *k, const void *v, int dtype, int64_t n, int d, int64_t row_stride,
                   double *out);
int vdref_attention(const double *q, const void *k, const void *v, int dtype, int64_t n, int d,
                    int64_t row_stride, double scale, double *out);
int vdref_fastcaote_scores(const double *q, int G, const void *k, const void *v, int dtype,
                           int64_t n, int d, int64_t row_stride, double scale, double *scores);

static unsigned long long rng = 88172645463325252ull;
static double unif(void)
{
    rng ^= rng << 13;
    rng ^= rng >> 7;
    rng ^= rng << 17;
    return (double)(rng >> 11) / 9007199254740992.0 - 0.5;
}

#define CHECK(x)                                                          \
    do {                                                                  \
        if (!(x)) {                                                       \
            fprintf(stderr, "check failed at line %d: %s\n", __LINE__, #x); \
            return 1;                                                     \
        }                                                                 \
    } while (0)

int main(void)
{
    const int ds[] = {1, 3, 8};
    for (int di = 0; di < 3; ++di) {
        int d = ds[di];
        for (int n = 1; n <= 9; ++n) {
            /* exactly-sized buffers, so that any overrun is caught */
            float *vf = malloc(sizeof(float) * n * d);
            float *kf = malloc(sizeof(float) * n * d);
            uint16_t *vb = malloc(sizeof(uint16_t) * n * d);
            uint16_t *kb = malloc(sizeof(uint16_t) * n * d);
            double *s = malloc(sizeof(double) * n);
            double *m = malloc(sizeof(double) * d);
            double *q = malloc(sizeof(double) * 4 * d);
            uint8_t *keep = malloc(n);
            int32_t *pos = malloc(sizeof(int32_t) * n);
            double out5[5], *att = malloc(sizeof(double) * d);
            for (int i = 0; i < n * d; ++i) {
                vf[i] = (float)unif();
                kf[i] = (float)unif();
                uint32_t w;
                memcpy(&w, &vf[i], 4);
                vb[i] = (uint16_t)(w >> 16);
                memcpy(&w, &kf[i], 4);
                kb[i] = (uint16_t)(w >> 16);
            }
            for (int i = 0; i < 4 * d; ++i)
                q[i] = unif();
            for (int dt = 0; dt < 2; ++dt) {
                void *vv = dt ? (void *)vf : (void *)vb;
                void *kk = dt ? (void *)kf : (void *)kb;
                CHECK(vdref_mean(vv, dt, n, d, d, m) == 0);
                for (int var = 0; var < 6; ++var) {
                    CHECK(vdref_score(vv, dt, n, d, d, var, s, m) == 0);
                    for (int j = 0; j < n; ++j)
                        CHECK(isfinite(s[j]) && s[j] >= -1e-12);   /* 1 - cos rounds below 0 */
                }
                for (int N = 1; N <= n + 1; ++N) {
                    CHECK(vdref_select_topn(s, n, N, keep) == 0);
                    CHECK(vdref_select_smallest(s, n, N, keep) == 0);
                    for (int j = 0; j < n; ++j)
                        pos[j] = j;
                    CHECK(vdref_compact(kk, vv, dt, n, N, d, d, keep, pos) == 0);
                }
                CHECK(vdref_geometry(kk, vv, dt, n, d, d, out5) == 0);
                CHECK(vdref_attention(q, kk, vv, dt, n, d, d, 0.5, att) == 0);
                for (int G = 1; G <= 4; G *= 2)
                    CHECK(vdref_fastcaote_scores(q, G, kk, vv, dt, n, d, d, 0.5, s) == 0);
            }
            free(vf); free(kf); free(vb); free(kb); free(s); free(m); free(q);
            free(keep); free(pos); free(att);
        }
    }
    /* the batched pass with ragged units, n = 0 included, every variant */
    {
        const int U = 5, cap = 7, d = 4;
        int32_t n_unit[5] = {0, 1, 7, 5, 6}, N_unit[5] = {1, 1, 3, 5, 2};
        for (int var = 0; var < 6; ++var) {
            float *k = malloc(sizeof(float) * U * cap * d), *v = malloc(sizeof(float) * U * cap * d);
            double *sc = malloc(sizeof(double) * U * cap), *mo = malloc(sizeof(double) * U * d);
            uint8_t *kp = malloc(U * cap);
            int32_t *pos = malloc(sizeof(int32_t) * U * cap);
            for (int i = 0; i < U * cap * d; ++i) {
                k[i] = (float)unif();
                v[i] = (float)unif();
            }
            for (int i = 0; i < U * cap; ++i)
                pos[i] = i;
            CHECK(vdref_evict_step(k, v, 1, U, cap, d, n_unit, N_unit, var, sc, kp, mo, pos, 1) == 0);
            free(k); free(v); free(sc); free(mo); free(kp); free(pos);
        }
    }
    /* rejections */
    double s1[1];
    uint8_t k1[1];
    CHECK(vdref_select_topn(s1, 1, 0, k1) != 0);
    CHECK(vdref_score(NULL, 1, 1, 1, 1, 0, s1, NULL) != 0);
    CHECK(vdref_fastcaote_scores(NULL, 1, NULL, NULL, 1, 1, 1, 1, 1.0, s1) != 0);
    puts("oracle sanitizer run ok");
    return 0;
}
