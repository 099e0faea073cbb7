/*
 * CPU oracle for the k-means hot path -- TEST INFRASTRUCTURE ONLY.
 *
 * Only the test suite, the package smoke check and the benchmark's CPU
 * baseline leg may load this code.  The GPU library never links it and shares
 * no code with it.
 *
 * What it computes: plain Lloyd's k-means in float64 with no pruning.
 * MTI pruning (paper section III-C) is an exact acceleration -- every distance
 * it skips is provably not smaller than the incumbent's -- and the merged
 * MM step of ||Lloyd's (section III-B) reorders the work without changing the
 * result, so the path's assignments and centroids are exactly those of this
 * definition.
 *
 *   distance   : Euclidean d of Table I, written out over the d coordinates;
 *                compared in squared form (argmin of d == argmin of d^2).
 *   assignment : a_i = argmin_j ||x_i - c_j||^2 (section IV-A).  Ties: the
 *                previous assignment wins an exact tie, otherwise the lowest
 *                index wins (the paper is silent; this rule makes "<=" pruning
 *                result-preserving).
 *   update     : c_j = mean of the points assigned to j (section IV-A); an
 *                empty cluster keeps its previous centroid (paper silent).
 *   objective  : inertia J = sum_i ||x_i - c_{a_i}||^2, the squared form of
 *                the objective of section IV-A, which Lloyd's never increases.
 *   stopping   : after the update of iteration t, stop if the number of
 *                points whose assignment changed is < tol * n (strict), or
 *                after max_iters assignment steps (paper silent for k-means).
 *
 * Inputs are float32 (exactly representable in float64); all arithmetic is
 * float64.  The assignment loop is parallel over points (OpenMP, static
 * schedule); each point's decision does not depend on the thread count.  The
 * update sums points sequentially in index order.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

void oracle_set_threads(int32_t t) {
#ifdef _OPENMP
    if (t > 0) omp_set_num_threads(t);
#else
    (void)t;
#endif
}

int32_t oracle_get_threads(void) {
#ifdef _OPENMP
    return (int32_t)omp_get_max_threads();
#else
    return 1;
#endif
}

/* ||x - c||^2 summed over the d coordinates in order (Table I). */
static double sq_euclid(const float* x, const double* c, int32_t d) {
    double s = 0.0;
    for (int32_t m = 0; m < d; ++m) {
        double t = (double)x[m] - c[m];
        s += t * t;
    }
    return s;
}

/*
 * One assignment step.  prev (nullable) is the previous assignment, -1 for
 * "none".  out[i] receives the new assignment.  best[i] / second[i]
 * (nullable) receive the smallest squared distance and the smallest squared
 * distance over the other centroids (+inf when k == 1).  Returns the number
 * of points whose assignment differs from prev (n when prev is NULL).
 */
int64_t oracle_assign(const float* X, int64_t n, int32_t d, const double* C, int32_t k,
                      const int32_t* prev, int32_t* out, double* best, double* second) {
    int64_t changed = 0;
#pragma omp parallel for schedule(static) reduction(+ : changed)
    for (int64_t i = 0; i < n; ++i) {
        const float* x = X + i * (int64_t)d;
        double b = INFINITY, s2 = INFINITY;
        int32_t arg = -1;
        double dprev = INFINITY;
        int32_t p = prev ? prev[i] : -1;
        for (int32_t j = 0; j < k; ++j) {
            double D = sq_euclid(x, C + (int64_t)j * d, d);
            if (j == p) dprev = D;
            if (D < b) {
                s2 = b;
                b = D;
                arg = j;
            } else if (D < s2) {
                s2 = D;
            }
        }
        if (p >= 0 && p != arg && dprev == b) arg = p;   /* incumbent wins an exact tie */
        out[i] = arg;
        if (best) best[i] = b;
        if (second) second[i] = s2;
        if (arg != p) changed += 1;
    }
    return changed;
}

/*
 * One update step: C_new[j] = mean of rows with assign == j, or C_old[j]
 * when no row is assigned to j.  counts (nullable) receives the cluster
 * sizes.  Rows are summed in index order.
 */
int32_t oracle_update(const float* X, int64_t n, int32_t d, const int32_t* assign, int32_t k,
                      const double* C_old, double* C_new, int64_t* counts) {
    double* S = (double*)calloc((size_t)k * (size_t)d, sizeof(double));
    int64_t* N = (int64_t*)calloc((size_t)k, sizeof(int64_t));
    if (!S || !N) {
        free(S);
        free(N);
        return -1;
    }
    for (int64_t i = 0; i < n; ++i) {
        int32_t j = assign[i];
        const float* x = X + i * (int64_t)d;
        double* s = S + (int64_t)j * d;
        for (int32_t m = 0; m < d; ++m) s[m] += (double)x[m];
        N[j] += 1;
    }
    for (int32_t j = 0; j < k; ++j) {
        for (int32_t m = 0; m < d; ++m) {
            int64_t o = (int64_t)j * d + m;
            C_new[o] = N[j] > 0 ? S[o] / (double)N[j] : C_old[o];
        }
        if (counts) counts[j] = N[j];
    }
    free(S);
    free(N);
    return 0;
}

/*
 * Whole run of Lloyd's k-means from C0.
 *
 * Outputs: assign_out[n] (last assignment step), C_out[k*d] (centroids after
 * the last update), *iters_out (assignment steps executed).  Per-iteration
 * arrays of length max_iters (nullable): inertia[t] = J_t measured against
 * the centroids used in step t, changed[t].  best/second (nullable, length n)
 * hold the last step's smallest and second-smallest squared distances.
 * assign_hist (nullable, max_iters*n) keeps every step's assignment and
 * C_hist (nullable, (max_iters+1)*k*d) the centroids before step 0 and after
 * every update.  Returns 0, or -1 on bad arguments / allocation failure.
 */
int32_t oracle_lloyd(const float* X, int64_t n, int32_t d, int32_t k, const double* C0,
                     int32_t max_iters, double tol, int32_t* assign_out, double* C_out,
                     int32_t* iters_out, double* inertia, int64_t* changed, double* best,
                     double* second, int32_t* assign_hist, double* C_hist) {
    if (!X || !C0 || !assign_out || !C_out || !iters_out || n < 1 || d < 1 || k < 1 || k > n ||
        max_iters < 1 || !(tol >= 0.0))
        return -1;
    const size_t kd = (size_t)k * (size_t)d;
    double* C = (double*)malloc(kd * sizeof(double));
    double* Cn = (double*)malloc(kd * sizeof(double));
    int32_t* a = (int32_t*)malloc((size_t)n * sizeof(int32_t));
    int32_t* an = (int32_t*)malloc((size_t)n * sizeof(int32_t));
    double* b = (double*)malloc((size_t)n * sizeof(double));
    double* s2 = second ? second : (double*)malloc((size_t)n * sizeof(double));
    if (!C || !Cn || !a || !an || !b || !s2) {
        free(C); free(Cn); free(a); free(an); free(b);
        if (!second) free(s2);
        return -1;
    }
    memcpy(C, C0, kd * sizeof(double));
    if (C_hist) memcpy(C_hist, C, kd * sizeof(double));
    int32_t t = 0;
    for (; t < max_iters; ++t) {
        int64_t ch = oracle_assign(X, n, d, C, k, t == 0 ? NULL : a, an, b, s2);
        double J = 0.0;
        for (int64_t i = 0; i < n; ++i) J += b[i];
        if (inertia) inertia[t] = J;
        if (changed) changed[t] = ch;
        if (assign_hist) memcpy(assign_hist + (int64_t)t * n, an, (size_t)n * sizeof(int32_t));
        if (oracle_update(X, n, d, an, k, C, Cn, NULL) != 0) {
            t = -1;
            break;
        }
        { int32_t* tmp = a; a = an; an = tmp; }
        { double* tmp = C; C = Cn; Cn = tmp; }
        if (C_hist) memcpy(C_hist + (size_t)(t + 1) * kd, C, kd * sizeof(double));
        if ((double)ch < tol * (double)n) {
            t += 1;
            break;
        }
    }
    int32_t rc = 0;
    if (t < 0) {
        rc = -1;
    } else {
        *iters_out = t;
        memcpy(assign_out, a, (size_t)n * sizeof(int32_t));
        memcpy(C_out, C, kd * sizeof(double));
        if (best) memcpy(best, b, (size_t)n * sizeof(double));
    }
    free(C); free(Cn); free(a); free(an); free(b);
    if (!second) free(s2);
    return rc;
}
