/*
 * Mutual Pair Merging -- CPU reference oracle (plain C, float64).
 *
 * TEST INFRASTRUCTURE. Only the test suite, the smoke check and the
 * benchmark's CPU-baseline leg load this library. The product path (the HIP
 * library) never calls it and shares no code with it.
 *
 * It computes, per image, exactly what the paper defines, written out as
 * brute force:
 *   Eq. 1      : row L2 normalisation and the dense cosine affinity S, with the
 *                diagonal excluded;
 *   Sec. 3.2   : nearest neighbour b(i) = argmax_{j != i} S_ij and the set of
 *                mutual pairs (b(b(i)) = i), lower index as representative;
 *   Alg. 1     : RepMask and compact ids by a left-to-right scan (partners
 *                inherit their representative's id);
 *   Eq. 2      : each cluster (one token or a mutual pair) is replaced by the
 *                mean of its members;
 *   Eq. 3      : composition of two merge maps, r*(i) = r2(r1(i));
 *   Eq. 4      : gather reconstruction, Z_up[i] = Z[r*(i)];
 *   Sec. 5     : the locality constraint the paper proposes against the quadratic
 *                affinity (also Sec. 4.3): candidates restricted to a spatial window
 *                around each token (reading: Chebyshev radius on the token grid; a
 *                merged token sits at its representative's position).
 *
 * Readings where the paper is silent:
 *   - ties in the argmax go to the lowest index j;
 *   - a row's norm is clamped below at 1e-12 before dividing;
 *   - ids are 0-based;
 *   - the mean is taken in float64 and rounded once (nearest even) to the
 *     storage type (float32 or bfloat16).
 *
 * S is made bitwise symmetric: the cosine of an unordered pair {i, j} is always
 * evaluated as dot(xt[min], xt[max]) over k = 0..D-1 in order.
 */
#include <math.h>
#include <pthread.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define ORACLE_DTYPE_F32 0
#define ORACLE_DTYPE_BF16 1

/* ------------------------------------------------------------------ */
/* Storage rounding                                                    */
/* ------------------------------------------------------------------ */

/* Round a float64 value to the nearest bfloat16 (8 significant bits, exponent
 * range of float32), ties to even; returned as the float64 value it equals. */
static double round_to_bf16(double v)
{
    if (isnan(v)) return v;
    if (v == 0.0 || isinf(v)) return v;
    double a = fabs(v);
    int e;
    frexp(a, &e);                 /* a = m * 2^e with m in [0.5, 1) */
    int lsb = (e - 1) - 7;        /* weight of the last of 8 significant bits */
    if (lsb < -133) lsb = -133;   /* spacing of the smallest (subnormal) bfloat16 */
    double q = ldexp(a, -lsb);    /* exact scaling by a power of two */
    double fl = floor(q);
    double frac = q - fl;
    double r = fl;
    if (frac > 0.5) r = fl + 1.0;
    else if (frac == 0.5 && fmod(fl, 2.0) != 0.0) r = fl + 1.0;
    double y = ldexp(r, lsb);
    if (y >= 0x1p128) y = INFINITY;  /* beyond the largest finite bfloat16 */
    return v < 0 ? -y : y;
}

static double round_to_storage(double v, int dtype)
{
    if (dtype == ORACLE_DTYPE_F32) return (double)(float)v;  /* C conversion rounds to nearest even */
    return round_to_bf16(v);
}

void mpm_oracle_round(const double* v, int64_t count, int dtype, double* out)
{
    for (int64_t i = 0; i < count; ++i) out[i] = round_to_storage(v[i], dtype);
}

/* ------------------------------------------------------------------ */
/* Eq. 1: normalisation and cosine affinity                            */
/* ------------------------------------------------------------------ */

/* xt[i] = x[i] / max(||x[i]||_2, 1e-12) */
static void normalise_rows(const double* x, int n, int D, double* xt)
{
    for (int i = 0; i < n; ++i) {
        double ss = 0.0;
        for (int k = 0; k < D; ++k) ss += x[(int64_t)i * D + k] * x[(int64_t)i * D + k];
        double nu = sqrt(ss);
        if (nu < 1e-12) nu = 1e-12;
        for (int k = 0; k < D; ++k) xt[(int64_t)i * D + k] = x[(int64_t)i * D + k] / nu;
    }
}

/* S_ij for i != j, symmetric by construction. */
static double cosine_of(const double* xt, int D, int i, int j)
{
    int lo = i < j ? i : j, hi = i < j ? j : i;
    const double* a = xt + (int64_t)lo * D;
    const double* b = xt + (int64_t)hi * D;
    double s = 0.0;
    for (int k = 0; k < D; ++k) s += a[k] * b[k];
    return s;
}

double mpm_oracle_cosine(const double* x, int n, int D, int i, int j)
{
    if (i < 0 || j < 0 || i >= n || j >= n || i == j) return NAN;
    double* xt = (double*)malloc(sizeof(double) * 2 * (size_t)D);
    if (!xt) return NAN;
    int lo = i < j ? i : j, hi = i < j ? j : i;
    normalise_rows(x + (int64_t)lo * D, 1, D, xt);
    normalise_rows(x + (int64_t)hi * D, 1, D, xt + D);
    double s = cosine_of(xt, D, 0, 1);
    free(xt);
    return s;
}

/* ------------------------------------------------------------------ */
/* Sec. 3.2: nearest neighbour with the diagonal masked                */
/* ------------------------------------------------------------------ */

typedef struct {
    const double* xt;
    int n, D;
    int row_begin, row_end;
    int32_t* nb;
    double* top1;
    double* top2;
    const int32_t* pos;  /* NULL: every j != i is a candidate */
    int grid_w, window;
} nn_job;

/* Whether token j is a candidate of token i under the locality constraint: both grid
 * positions (raster indices on a grid of grid_w columns) within `window` rows and
 * `window` columns of each other. */
static int in_window(const nn_job* job, int i, int j)
{
    if (!job->pos) return 1;
    const int ri = job->pos[i] / job->grid_w, ci = job->pos[i] % job->grid_w;
    const int rj = job->pos[j] / job->grid_w, cj = job->pos[j] % job->grid_w;
    return abs(ri - rj) <= job->window && abs(ci - cj) <= job->window;
}

/* For each row i: b(i) = argmax_{j != i} S_ij, lowest j among equal maxima;
 * top1 = the maximum, top2 = the second largest value over j != i (equal to
 * top1 when the maximum is attained twice). */
static void* nearest_rows(void* p)
{
    nn_job* job = (nn_job*)p;
    for (int i = job->row_begin; i < job->row_end; ++i) {
        int best = -1;
        double v1 = -INFINITY, v2 = -INFINITY;
        for (int j = 0; j < job->n; ++j) {
            if (j == i) continue;  /* S_ii is -inf */
            if (!in_window(job, i, j)) continue;  /* outside the locality window: not a candidate */
            double s = cosine_of(job->xt, job->D, i, j);
            if (best < 0 || s > v1) {
                v2 = v1;
                v1 = s;
                best = j;
            } else if (s > v2) {
                v2 = s;
            }
        }
        job->nb[i] = best;  /* -1 when the image has a single token (or the window no other one) */
        if (job->top1) job->top1[i] = v1;
        if (job->top2) job->top2[i] = v2;
    }
    return NULL;
}

/* x: n x D float64 (the storage values, converted exactly). Writes nb[n] and,
 * when non-NULL, top1[n] / top2[n]. Rows are split over `threads` threads.
 * Returns 0, or -1 on bad arguments / allocation failure. */
static int nearest_impl(const double* x, int n, int D, int threads, int32_t* nb, double* top1, double* top2,
                        const int32_t* pos, int grid_w, int window)
{
    if (!x || !nb || n < 1 || D < 1) return -1;
    double* xt = (double*)malloc(sizeof(double) * (size_t)n * (size_t)D);
    if (!xt) return -1;
    normalise_rows(x, n, D, xt);
    if (threads < 1) threads = 1;
    if (threads > n) threads = n;
    nn_job* jobs = (nn_job*)calloc((size_t)threads, sizeof(nn_job));
    pthread_t* tids = (pthread_t*)calloc((size_t)threads, sizeof(pthread_t));
    if (!jobs || !tids) {
        free(xt); free(jobs); free(tids);
        return -1;
    }
    for (int t = 0; t < threads; ++t) {
        jobs[t].xt = xt; jobs[t].n = n; jobs[t].D = D;
        jobs[t].row_begin = (int)((int64_t)n * t / threads);
        jobs[t].row_end = (int)((int64_t)n * (t + 1) / threads);
        jobs[t].nb = nb; jobs[t].top1 = top1; jobs[t].top2 = top2;
        jobs[t].pos = pos; jobs[t].grid_w = grid_w; jobs[t].window = window;
    }
    int spawned = 0;
    for (int t = 1; t < threads; ++t) {
        if (pthread_create(&tids[t], NULL, nearest_rows, &jobs[t]) != 0) break;
        spawned = t;
    }
    nearest_rows(&jobs[0]);
    for (int t = 1; t <= spawned; ++t) pthread_join(tids[t], NULL);
    for (int t = spawned + 1; t < threads; ++t) nearest_rows(&jobs[t]);  /* threads that failed to start */
    free(jobs); free(tids); free(xt);
    return 0;
}

int mpm_oracle_nearest(const double* x, int n, int D, int threads,
                       int32_t* nb, double* top1, double* top2)
{
    return nearest_impl(x, n, D, threads, nb, top1, top2, NULL, 1, 0);
}

/* mpm_oracle_nearest under the locality constraint: pos[i] = grid position of token i
 * (row * grid_w + col), window >= 0. Returns -1 on bad arguments. */
int mpm_oracle_nearest_window(const double* x, int n, int D, const int32_t* pos, int grid_w, int window,
                              int threads, int32_t* nb, double* top1, double* top2)
{
    if (!pos || grid_w < 1 || window < 0) return -1;
    for (int i = 0; i < n; ++i)
        if (pos[i] < 0) return -1;
    return nearest_impl(x, n, D, threads, nb, top1, top2, pos, grid_w, window);
}

/* Same argmax rule applied to a given n x n matrix S (row-major); the diagonal
 * is ignored. Used to check the pairing steps on hand-made affinities. */
int mpm_oracle_nearest_from_affinity(const double* S, int n, int32_t* nb)
{
    if (!S || !nb || n < 1) return -1;
    for (int i = 0; i < n; ++i) {
        int best = -1;
        double v1 = -INFINITY;
        for (int j = 0; j < n; ++j) {
            if (j == i) continue;
            double s = S[(int64_t)i * n + j];
            if (best < 0 || s > v1) { v1 = s; best = j; }
        }
        nb[i] = best;
    }
    return 0;
}

/* ------------------------------------------------------------------ */
/* Sec. 3.2 + Alg. 1: mutual pairs, RepMask, compact ids               */
/* ------------------------------------------------------------------ */

/* From nb[n] compute:
 *   map[i]   : compact cluster id r(i) in [0, n');
 *   src_a[k] : representative (lowest index) of cluster k;
 *   src_b[k] : its partner, or src_a[k] for a singleton.
 * Returns n' (>= 1 for n >= 1), or -1 on bad arguments. */
int mpm_oracle_pairs(const int32_t* nb, int n, int32_t* map, int32_t* src_a, int32_t* src_b)
{
    if (!nb || !map || n < 1) return -1;
    /* A token is in a mutual pair with j = b(i) iff b(j) = i. */
    unsigned char* mutual = (unsigned char*)calloc((size_t)n, 1);
    if (!mutual) return -1;
    for (int i = 0; i < n; ++i) {
        int j = nb[i];
        mutual[i] = (j >= 0 && j < n && j != i && nb[j] == i);
    }
    /* RepMask: the lower index of a pair, or a singleton. Ids by left-to-right scan. */
    int next_id = 0;
    for (int i = 0; i < n; ++i) {
        int is_rep = !mutual[i] || i < nb[i];
        if (is_rep) {
            map[i] = next_id;
            if (src_a) src_a[next_id] = i;
            if (src_b) src_b[next_id] = mutual[i] ? nb[i] : i;
            ++next_id;
        }
    }
    /* Partners inherit their representative's id (the representative has a lower index). */
    for (int i = 0; i < n; ++i)
        if (mutual[i] && i > nb[i]) map[i] = map[nb[i]];
    free(mutual);
    return next_id;
}

/* ------------------------------------------------------------------ */
/* Eq. 2: cluster means                                                */
/* ------------------------------------------------------------------ */

/* y[k] = mean of the members of cluster k, rounded to the storage dtype. */
void mpm_oracle_average(const double* x, int D, const int32_t* src_a, const int32_t* src_b,
                        int m, int dtype, double* y)
{
    for (int k = 0; k < m; ++k) {
        const double* xa = x + (int64_t)src_a[k] * D;
        const double* xb = x + (int64_t)src_b[k] * D;
        double* yk = y + (int64_t)k * D;
        if (src_a[k] == src_b[k]) {
            for (int c = 0; c < D; ++c) yk[c] = xa[c];  /* |C_k| = 1 */
        } else {
            for (int c = 0; c < D; ++c) yk[c] = round_to_storage((xa[c] + xb[c]) / 2.0, dtype);
        }
    }
}

/* ------------------------------------------------------------------ */
/* Eq. 3 and Eq. 4                                                     */
/* ------------------------------------------------------------------ */

/* out[i] = r2[r1[i]] (or -1 where r1[i] < 0). */
void mpm_oracle_compose(const int32_t* r1, int n, const int32_t* r2, int32_t* out)
{
    for (int i = 0; i < n; ++i) out[i] = r1[i] < 0 ? -1 : r2[r1[i]];
}

/* out[i] = z[rstar[i]] row by row (a plain copy). */
void mpm_oracle_unmerge(const double* z, int D, const int32_t* rstar, int n, double* out)
{
    for (int i = 0; i < n; ++i)
        memcpy(out + (int64_t)i * D, z + (int64_t)rstar[i] * D, sizeof(double) * (size_t)D);
}
