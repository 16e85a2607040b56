/* Drives every function of the C oracle (oracle/precog_oracle.c) on small
 * problems whose buffers are allocated at their exact sizes, for a build with
 * AddressSanitizer and UndefinedBehaviorSanitizer: any read or write past a
 * buffer, use after free, leak or undefined arithmetic in the oracle is
 * reported by the sanitizers (and makes the process exit nonzero).  It also
 * checks the results it can check without a second implementation: return
 * codes, finite outputs, indices in range, the Theorem 1 split (the state
 * after a prefix, injected as h0, continues the scan bit for bit), the
 * trajectory's last slot equal to the final state, thread-count invariance.
 * Test infrastructure only. */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

int oracle_scan_f64(int64_t B, int64_t L, int64_t D, int64_t N, const double *x,
                    const double *dt, const double *A, const double *Bm, const double *Cm,
                    const double *z, const double *Dskip, const double *h0, double *y,
                    double *hT, int nthreads);
int oracle_scan_complex_f64(int64_t B, int64_t L, int64_t D, int64_t N, const double *x,
                            const double *dt, const double *Are, const double *Aim,
                            const double *Bm, const double *Cm, const double *z,
                            const double *Dskip, const double *h0, double *y, double *hT);
int oracle_trajectory_f64(int64_t B, int64_t L, int64_t D, int64_t N, int64_t k,
                          const double *x, const double *dt, const double *A, const double *Bm,
                          const double *h0, double *traj);
int oracle_top1_f64(int64_t Q, int64_t M, int64_t E, const float *q, const float *K,
                    int32_t *idx, double *best, int nthreads);

static int failures = 0;
#define CHECK(c)                                                          \
    do {                                                                  \
        if (!(c)) {                                                       \
            fprintf(stderr, "check failed at line %d: %s\n", __LINE__, #c); \
            ++failures;                                                   \
        }                                                                 \
    } while (0)

static uint64_t rng = 0x9e3779b97f4a7c15ull;
static double urand(void) /* uniform in [0, 1), xorshift64* */
{
    rng ^= rng >> 12;
    rng ^= rng << 25;
    rng ^= rng >> 27;
    return (double)((rng * 2685821657736338717ull) >> 11) / 9007199254740992.0;
}

/* exact-size buffers (one element when empty: the oracle requires its
 * input pointers whenever L > 0, even with no rows) */
static double *dbuf(int64_t n, double lo, double hi)
{
    double *p = (double *)malloc((size_t)(n > 0 ? n : 1) * sizeof(double));
    for (int64_t i = 0; i < n; ++i)
        p[i] = lo + (hi - lo) * urand();
    return p;
}
static int all_finite(const double *p, int64_t n)
{
    for (int64_t i = 0; i < n; ++i)
        if (!isfinite(p[i]))
            return 0;
    return 1;
}

static void scan_case(int64_t B, int64_t L, int64_t D, int64_t N, int with_opts, int nthr)
{
    double *x = dbuf(B * L * D, -1, 1), *dt = dbuf(B * L * D, 0.01, 0.9);
    double *A = dbuf(D * N, 1, 16), *Bm = dbuf(B * L * N, -0.5, 0.5);
    double *Cm = dbuf(B * L * N, -0.5, 0.5);
    double *z = with_opts ? dbuf(B * L * D, -2, 2) : NULL;
    double *Ds = with_opts ? dbuf(D, -1, 1) : NULL;
    double *h0 = with_opts ? dbuf(B * D * N, -1, 1) : NULL;
    double *y = B * L * D > 0 ? (double *)malloc((size_t)(B * L * D) * sizeof(double)) : NULL;
    double *hT = B * D * N > 0 ? (double *)malloc((size_t)(B * D * N) * sizeof(double)) : NULL;
    double *y1 = B * L * D > 0 ? (double *)malloc((size_t)(B * L * D) * sizeof(double)) : NULL;
    double *hT1 = B * D * N > 0 ? (double *)malloc((size_t)(B * D * N) * sizeof(double)) : NULL;
    CHECK(oracle_scan_f64(B, L, D, N, x, dt, A, Bm, Cm, z, Ds, h0, y, hT, nthr) == 0);
    CHECK(all_finite(y, B * L * D) && all_finite(hT, B * D * N));
    /* one thread gives the same bits */
    CHECK(oracle_scan_f64(B, L, D, N, x, dt, A, Bm, Cm, z, Ds, h0, y1, hT1, 1) == 0);
    if (B * L * D > 0)
        CHECK(memcmp(y, y1, (size_t)(B * L * D) * sizeof(double)) == 0);
    if (B * D * N > 0)
        CHECK(memcmp(hT, hT1, (size_t)(B * D * N) * sizeof(double)) == 0);
    /* state only, no readout inputs */
    CHECK(oracle_scan_f64(B, L, D, N, x, dt, A, Bm, NULL, NULL, NULL, h0, NULL, hT1, nthr) == 0);
    if (B * D * N > 0)
        CHECK(memcmp(hT, hT1, (size_t)(B * D * N) * sizeof(double)) == 0);
    /* Theorem 1 split at s for B = 1: prefix, then the rest from its state */
    if (B == 1 && L >= 2) {
        const int64_t s = L / 2;
        double *hs = (double *)malloc((size_t)(D * N) * sizeof(double));
        double *ys = (double *)malloc((size_t)(L * D) * sizeof(double));
        double *hE = (double *)malloc((size_t)(D * N) * sizeof(double));
        CHECK(oracle_scan_f64(1, s, D, N, x, dt, A, Bm, Cm, z, Ds, h0, ys, hs, 1) == 0);
        CHECK(oracle_scan_f64(1, L - s, D, N, x + s * D, dt + s * D, A, Bm + s * N, Cm + s * N,
                              z ? z + s * D : NULL, Ds, hs, ys + s * D, hE, 1) == 0);
        CHECK(memcmp(ys, y, (size_t)(L * D) * sizeof(double)) == 0);
        CHECK(memcmp(hE, hT, (size_t)(D * N) * sizeof(double)) == 0);
        free(hs);
        free(ys);
        free(hE);
    }
    free(x); free(dt); free(A); free(Bm); free(Cm); free(z); free(Ds); free(h0);
    free(y); free(hT); free(y1); free(hT1);
}

static void complex_case(int64_t B, int64_t L, int64_t D, int64_t N, int with_opts)
{
    double *x = dbuf(B * L * D, -1, 1), *dt = dbuf(B * L * D, 0.01, 0.9);
    double *Ar = dbuf(D * N, 1, 16), *Ai = dbuf(D * N, 0, 40);
    double *Bm = dbuf(B * L * N, -0.5, 0.5), *Cm = dbuf(B * L * N, -0.5, 0.5);
    double *z = with_opts ? dbuf(B * L * D, -2, 2) : NULL;
    double *Ds = with_opts ? dbuf(D, -1, 1) : NULL;
    double *h0 = with_opts ? dbuf(2 * B * D * N, -1, 1) : NULL;
    double *y = B * L * D > 0 ? (double *)malloc((size_t)(B * L * D) * sizeof(double)) : NULL;
    double *hT = B * D * N > 0 ? (double *)malloc((size_t)(2 * B * D * N) * sizeof(double)) : NULL;
    CHECK(oracle_scan_complex_f64(B, L, D, N, x, dt, Ar, Ai, Bm, Cm, z, Ds, h0, y, hT) == 0);
    CHECK(all_finite(y, B * L * D) && all_finite(hT, 2 * B * D * N));
    CHECK(oracle_scan_complex_f64(B, L, D, N, x, dt, Ar, Ai, Bm, NULL, NULL, NULL, h0, NULL,
                                  hT) == 0);
    free(x); free(dt); free(Ar); free(Ai); free(Bm); free(Cm); free(z); free(Ds); free(h0);
    free(y); free(hT);
}

static void trajectory_case(int64_t B, int64_t L, int64_t D, int64_t N, int64_t k)
{
    double *x = dbuf(B * L * D, -1, 1), *dt = dbuf(B * L * D, 0.01, 0.9);
    double *A = dbuf(D * N, 1, 16), *Bm = dbuf(B * L * N, -0.5, 0.5);
    double *h0 = dbuf(B * D * N, -1, 1);
    const int64_t K = L / k;
    double *tr = B * K * D * N > 0 ? (double *)malloc((size_t)(B * K * D * N) * sizeof(double)) : NULL;
    double *hT = B * D * N > 0 ? (double *)malloc((size_t)(B * D * N) * sizeof(double)) : NULL;
    CHECK(oracle_trajectory_f64(B, L, D, N, k, x, dt, A, Bm, h0, tr) == 0);
    CHECK(all_finite(tr, B * K * D * N));
    CHECK(oracle_scan_f64(B, L, D, N, x, dt, A, Bm, NULL, NULL, NULL, h0, NULL, hT, 1) == 0);
    if (K > 0 && K * k == L) /* the last kept state is the final state */
        for (int64_t b = 0; b < B; ++b)
            CHECK(memcmp(tr + ((b * K + K - 1) * D) * N, hT + b * D * N,
                         (size_t)(D * N) * sizeof(double)) == 0);
    free(x); free(dt); free(A); free(Bm); free(h0); free(tr); free(hT);
}

static void top1_case(int64_t Q, int64_t M, int64_t E, int nthr)
{
    float *q = Q * E > 0 ? (float *)malloc((size_t)(Q * E) * sizeof(float)) : NULL;
    float *K = M * E > 0 ? (float *)malloc((size_t)(M * E) * sizeof(float)) : NULL;
    for (int64_t i = 0; i < Q * E; ++i)
        q[i] = (float)(urand() - 0.5);
    for (int64_t i = 0; i < M * E; ++i)
        K[i] = (float)(urand() - 0.5);
    if (M > 1 && E > 0) /* a duplicated row: ties go to the lower index */
        memcpy(K + (M - 1) * E, K, (size_t)E * sizeof(float));
    int32_t *idx = Q > 0 ? (int32_t *)malloc((size_t)Q * sizeof(int32_t)) : NULL;
    double *best = Q > 0 ? (double *)malloc((size_t)Q * sizeof(double)) : NULL;
    CHECK(oracle_top1_f64(Q, M, E, q, K, idx, best, nthr) == 0);
    for (int64_t i = 0; i < Q; ++i) {
        CHECK(M == 0 ? idx[i] == -1 : (idx[i] >= 0 && idx[i] < M - (M > 1 ? 1 : 0)));
    }
    CHECK(oracle_top1_f64(Q, M, E, q, K, idx, NULL, nthr) == 0); /* best is optional */
    free(q); free(K); free(idx); free(best);
}

int main(void)
{
    const int64_t shapes[][4] = {{1, 1, 1, 1}, {2, 17, 3, 4}, {1, 40, 8, 16}, {3, 33, 5, 2},
                                 {2, 0, 5, 2}, {0, 5, 3, 2}, {1, 64, 2, 64}};
    for (size_t i = 0; i < sizeof(shapes) / sizeof(shapes[0]); ++i) {
        const int64_t *s = shapes[i];
        for (int opts = 0; opts < 2; ++opts) {
            scan_case(s[0], s[1], s[2], s[3], opts, 3);
            scan_case(s[0], s[1], s[2], s[3], opts, 64);
            if (s[3] <= 16)
                complex_case(s[0], s[1], s[2], s[3], opts);
        }
        trajectory_case(s[0], s[1], s[2], s[3], 1);
        trajectory_case(s[0], s[1], s[2], s[3], 3);
        if (s[1] > 0) {
            trajectory_case(s[0], s[1], s[2], s[3], s[1]);
            trajectory_case(s[0], s[1], s[2], s[3], s[1] + 1);
        }
    }
    const int64_t rs[][3] = {{0, 5, 4}, {3, 0, 4}, {5, 7, 3}, {9, 100, 16}, {1, 1, 1}};
    for (size_t i = 0; i < sizeof(rs) / sizeof(rs[0]); ++i) {
        top1_case(rs[i][0], rs[i][1], rs[i][2], 1);
        top1_case(rs[i][0], rs[i][1], rs[i][2], 4);
    }
    /* malformed arguments are refused */
    CHECK(oracle_scan_f64(-1, 1, 1, 1, NULL, NULL, NULL, NULL, NULL, NULL, NULL, NULL, NULL, NULL,
                          1) != 0);
    CHECK(oracle_scan_f64(1, 1, 1, 0, NULL, NULL, NULL, NULL, NULL, NULL, NULL, NULL, NULL, NULL,
                          1) != 0);
    CHECK(oracle_trajectory_f64(1, 4, 1, 1, 0, NULL, NULL, NULL, NULL, NULL, NULL) != 0);
    CHECK(oracle_top1_f64(-1, 1, 1, NULL, NULL, NULL, NULL, 1) != 0);
    if (failures) {
        fprintf(stderr, "%d checks failed\n", failures);
        return 1;
    }
    printf("oracle driver: all checks passed\n");
    return 0;
}
