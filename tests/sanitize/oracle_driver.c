/*
 * Drives every function of the oracle (oracle/mpm_oracle.c) on random inputs whose
 * buffers are allocated at their exact sizes, for a build with AddressSanitizer and
 * UndefinedBehaviorSanitizer (or ThreadSanitizer, for the threaded nearest-neighbour
 * search). Exits 0 when every call returned what its contract states; the
 * sanitizers abort the run on an out-of-bounds access, a use after free, undefined
 * behaviour or a data race.
 */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>

int mpm_oracle_nearest(const double* x, int n, int D, int threads, int32_t* nb, double* top1, double* top2);
int mpm_oracle_nearest_from_affinity(const double* S, int n, int32_t* nb);
int mpm_oracle_pairs(const int32_t* nb, int n, int32_t* map, int32_t* src_a, int32_t* src_b);
void mpm_oracle_average(const double* x, int D, const int32_t* src_a, const int32_t* src_b, int m, int dtype,
                        double* y);
void mpm_oracle_compose(const int32_t* r1, int n, const int32_t* r2, int32_t* out);
void mpm_oracle_unmerge(const double* z, int D, const int32_t* rstar, int n, double* out);
double mpm_oracle_cosine(const double* x, int n, int D, int i, int j);
void mpm_oracle_round(const double* v, int64_t count, int dtype, double* out);

static uint64_t state = 0x9E3779B97F4A7C15ull;
static uint64_t next(void)
{
    state ^= state << 13;
    state ^= state >> 7;
    state ^= state << 17;
    return state;
}
static double uniform(void) { return (double)(next() >> 11) / 9007199254740992.0 * 2.0 - 1.0; }

#define CHECK(c)                                                     \
    do {                                                             \
        if (!(c)) {                                                  \
            fprintf(stderr, "check failed at line %d: %s\n", __LINE__, #c); \
            return 1;                                                \
        }                                                            \
    } while (0)

static int one_case(int n, int D, int threads, int dtype, int zero_row)
{
    double* x = malloc(sizeof(double) * (size_t)n * D);
    int32_t* nb = malloc(sizeof(int32_t) * n);
    double* t1 = malloc(sizeof(double) * n);
    double* t2 = malloc(sizeof(double) * n);
    int32_t* map = malloc(sizeof(int32_t) * n);
    int32_t* sa = malloc(sizeof(int32_t) * n);
    int32_t* sb = malloc(sizeof(int32_t) * n);
    for (int k = 0; k < n * D; ++k) x[k] = uniform() * ((next() & 7) == 0 ? 1e-3 : 10.0);
    if (zero_row) for (int c = 0; c < D; ++c) x[c] = 0.0;
    mpm_oracle_round(x, (int64_t)n * D, dtype, x);
    CHECK(mpm_oracle_nearest(x, n, D, threads, nb, t1, t2) == 0);
    for (int i = 0; i < n; ++i) {
        CHECK(n == 1 ? nb[i] == -1 : (nb[i] >= 0 && nb[i] < n && nb[i] != i));
        CHECK(n == 1 || t1[i] >= t2[i]);
        if (n > 1) CHECK(fabs(mpm_oracle_cosine(x, n, D, i, nb[i]) - t1[i]) < 1e-12);
    }
    const int m = mpm_oracle_pairs(nb, n, map, sa, sb);
    CHECK(m >= (n + 1) / 2 && m <= (n > 1 ? n - 1 : 1));
    double* y = malloc(sizeof(double) * (size_t)m * D);
    mpm_oracle_average(x, D, sa, sb, m, dtype, y);
    int32_t* r2 = malloc(sizeof(int32_t) * m);
    for (int k = 0; k < m; ++k) r2[k] = (int32_t)(next() % (uint64_t)m);
    int32_t* rs = malloc(sizeof(int32_t) * n);
    mpm_oracle_compose(map, n, r2, rs);
    double* up = malloc(sizeof(double) * (size_t)n * D);
    mpm_oracle_unmerge(y, D, rs, n, up);
    /* A given affinity: the same argmax rule on a random symmetric matrix. */
    double* S = malloc(sizeof(double) * (size_t)n * n);
    for (int i = 0; i < n; ++i)
        for (int j = 0; j <= i; ++j) S[(size_t)i * n + j] = S[(size_t)j * n + i] = (double)(next() % 3);
    CHECK(mpm_oracle_nearest_from_affinity(S, n, nb) == 0);
    free(S); free(up); free(rs); free(r2); free(y);
    free(sb); free(sa); free(map); free(t2); free(t1); free(nb); free(x);
    return 0;
}

int main(void)
{
    int cases = 0;
    for (int n = 1; n <= 40; n += (n < 8 ? 1 : 7))
        for (int D = 1; D <= 20; D += 6)
            for (int threads = 1; threads <= 5; threads += 2)
                for (int dtype = 0; dtype <= 1; ++dtype) {
                    if (one_case(n, D, threads, dtype, (n + D) % 3 == 0)) {
                        fprintf(stderr, "case n=%d D=%d threads=%d dtype=%d failed\n", n, D, threads, dtype);
                        return 1;
                    }
                    ++cases;
                }
    /* Bad arguments are refused, not dereferenced. */
    int32_t nb1[1];
    if (mpm_oracle_nearest(NULL, 1, 1, 1, nb1, NULL, NULL) != -1 || mpm_oracle_pairs(NULL, 1, nb1, NULL, NULL) != -1 ||
        mpm_oracle_nearest_from_affinity(NULL, 1, nb1) != -1 || !isnan(mpm_oracle_cosine(NULL, 2, 1, 0, 0))) {
        fprintf(stderr, "bad arguments accepted\n");
        return 1;
    }
    printf("oracle driver: %d cases ok\n", cases);
    return 0;
}
