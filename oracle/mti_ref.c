/*
 * CPU reference of MTI-pruned Lloyd's k-means -- TEST INFRASTRUCTURE ONLY.
 *
 * Only the test suite and the benchmark's CPU leg may load this code; the GPU
 * library shares nothing with it.  It exists to pin a property, not a value:
 * MTI pruning (paper section III-C) never changes an assignment relative to
 * unpruned Lloyd's, so at every iteration its assignments must equal those of
 * the plain oracle in lloyd.c (written separately, on purpose).
 *
 * State (section III-C, Table I): an upper bound u_i >= d(x_i, c_{a_i}) per
 * point (O(n) memory), the centroid drift f(c) = d(c^t, c^{t-1}) and the
 * centroid-to-centroid distances (O(k^2)).  Readings of the paper taken here:
 *   - the clause thresholds are half the centroid-to-centroid distance,
 *     h(a, c) = d(c_a, c) / 2 (Elkan's lemma; without the factor 1/2 a point
 *     can be kept away from a closer centroid -- the "halve = 0" switch below
 *     plants exactly that mistake for the negative-control test);
 *   - Clause 1 takes the minimum over the other centroids, s(a) = min_{c != a} h(a, c);
 *   - the bound is maintained as u <- u + f(c_a) after every update and
 *     reset to the exact distance whenever that distance is computed;
 *   - the scan keeps a running best b (Elkan's order): the incumbent is
 *     tightened first, then the other centroids in ascending index, and a
 *     centroid c is skipped when the current bound is <= h(b, c);
 *   - iteration 0 has no bounds: it scans all centroids with the running-best
 *     skip only.
 * Ties follow the oracle's rule (incumbent wins, else the lowest index); with
 * the scan order above a strict "<" implements it.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

static double mti_sqdist(const float* x, const double* c, int32_t d) {
    double acc = 0.0;
    for (int32_t m = 0; m < d; ++m) {
        double diff = (double)x[m] - c[m];
        acc += diff * diff;
    }
    return acc;
}

static double mti_cdist(const double* p, const double* q, int32_t d) {
    double acc = 0.0;
    for (int32_t m = 0; m < d; ++m) {
        double diff = p[m] - q[m];
        acc += diff * diff;
    }
    return sqrt(acc);
}

/* h[i*k+j] = scale * d(c_i, c_j); s[i] = min over j != i (+inf when k == 1). */
static void mti_centroid_table(const double* C, int32_t k, int32_t d, double scale, double* h,
                               double* s) {
    for (int32_t i = 0; i < k; ++i) {
        s[i] = INFINITY;
        for (int32_t j = 0; j < k; ++j) {
            double v = i == j ? 0.0 : scale * mti_cdist(C + (int64_t)i * d, C + (int64_t)j * d, d);
            h[(int64_t)i * k + j] = v;
            if (j != i && v < s[i]) s[i] = v;
        }
    }
}

/*
 * Whole MTI run.  halve = 1 is the method; halve = 0 drops the factor 1/2
 * (negative control).  Outputs as in oracle_lloyd, plus per-iteration
 * counters (nullable, length max_iters): computed[t] = point-centroid
 * distances evaluated (tightenings included), clause1[t] = points skipped by
 * Clause 1.  bound_violations (nullable): if non-null, after every
 * assignment step the exact distance to the assigned centroid is recomputed
 * and the number of points with u_i < that distance is accumulated here.
 */
int32_t mti_lloyd(const float* X, int64_t n, int32_t d, int32_t k, const double* C0,
                  int32_t max_iters, double tol, int32_t halve, int32_t* assign_out,
                  double* C_out, int32_t* iters_out, int64_t* changed, int64_t* computed,
                  int64_t* clause1, int32_t* assign_hist, int64_t* bound_violations) {
    if (!X || !C0 || !assign_out || !C_out || !iters_out || n < 1 || d < 1 || k < 1 || k > n ||
        max_iters < 1 || !(tol >= 0.0))
        return -1;
    const double scale = halve ? 0.5 : 1.0;
    const size_t kd = (size_t)k * (size_t)d;
    double* C = (double*)malloc(kd * sizeof(double));
    double* Cold = (double*)malloc(kd * sizeof(double));
    double* S = (double*)malloc(kd * sizeof(double));
    int64_t* N = (int64_t*)malloc((size_t)k * sizeof(int64_t));
    double* h = (double*)malloc((size_t)k * (size_t)k * sizeof(double));
    double* s = (double*)malloc((size_t)k * sizeof(double));
    double* f = (double*)malloc((size_t)k * sizeof(double));
    int32_t* a = (int32_t*)malloc((size_t)n * sizeof(int32_t));
    double* u = (double*)malloc((size_t)n * sizeof(double));
    if (!C || !Cold || !S || !N || !h || !s || !f || !a || !u) {
        free(C); free(Cold); free(S); free(N); free(h); free(s); free(f); free(a); free(u);
        return -1;
    }
    memcpy(C, C0, kd * sizeof(double));
    if (bound_violations) *bound_violations = 0;
    int32_t t = 0;
    for (; t < max_iters; ++t) {
        mti_centroid_table(C, k, d, scale, h, s);
        int64_t n_changed = 0, n_computed = 0, n_clause1 = 0;
        /* Points are independent within a step (each reads the shared tables
           and writes only its own a[i], u[i]), so they run in parallel; the
           counts are integer sums, the same for any thread count. */
#pragma omp parallel for schedule(static) reduction(+ : n_changed, n_computed, n_clause1)
        for (int64_t i = 0; i < n; ++i) {
            const float* x = X + i * (int64_t)d;
            if (t == 0) {
                /* No bounds yet: running-best scan over all centroids. */
                int32_t b = 0;
                double Db = mti_sqdist(x, C, d);
                double ub = sqrt(Db);
                n_computed += 1;
                for (int32_t j = 1; j < k; ++j) {
                    if (ub <= h[(int64_t)b * k + j]) continue;
                    double Dj = mti_sqdist(x, C + (int64_t)j * d, d);
                    n_computed += 1;
                    if (Dj < Db) {
                        Db = Dj;
                        b = j;
                        ub = sqrt(Db);
                    }
                }
                a[i] = b;
                u[i] = ub;
                n_changed += 1;
                continue;
            }
            const int32_t inc = a[i];
            u[i] += f[inc];                               /* bound update */
            if (u[i] <= s[inc]) {                         /* Clause 1 */
                n_clause1 += 1;
                continue;
            }
            int32_t b = inc;
            double ub = u[i];
            double Db = 0.0;
            int tight = 0;
            for (int32_t j = 0; j < k; ++j) {
                if (j == inc) continue;
                if (ub <= h[(int64_t)b * k + j]) continue;          /* Clause 2 (loose) / 3 (tight) */
                if (!tight) {                                      /* U(u): tighten once */
                    Db = mti_sqdist(x, C + (int64_t)inc * d, d);
                    ub = sqrt(Db);
                    tight = 1;
                    n_computed += 1;
                    if (ub <= h[(int64_t)b * k + j]) continue;      /* Clause 3 */
                }
                double Dj = mti_sqdist(x, C + (int64_t)j * d, d);
                n_computed += 1;
                if (Dj < Db) {
                    Db = Dj;
                    b = j;
                    ub = sqrt(Db);
                }
            }
            u[i] = ub;
            if (b != inc) {
                a[i] = b;
                n_changed += 1;
            }
        }
        if (changed) changed[t] = n_changed;
        if (computed) computed[t] = n_computed;
        if (clause1) clause1[t] = n_clause1;
        if (assign_hist) memcpy(assign_hist + (int64_t)t * n, a, (size_t)n * sizeof(int32_t));
        if (bound_violations) {
            for (int64_t i = 0; i < n; ++i) {
                double e = sqrt(mti_sqdist(X + i * (int64_t)d, C + (int64_t)a[i] * d, d));
                if (u[i] < e * (1.0 - 1e-12)) *bound_violations += 1;   /* fp64 rounding slack */
            }
        }
        /* Update: member means, empty clusters keep their centroid; drift f. */
        memset(S, 0, kd * sizeof(double));
        memset(N, 0, (size_t)k * sizeof(int64_t));
        for (int64_t i = 0; i < n; ++i) {
            const float* x = X + i * (int64_t)d;
            double* row = S + (int64_t)a[i] * d;
            for (int32_t m = 0; m < d; ++m) row[m] += (double)x[m];
            N[a[i]] += 1;
        }
        memcpy(Cold, C, kd * sizeof(double));
        for (int32_t j = 0; j < k; ++j) {
            if (N[j] > 0)
                for (int32_t m = 0; m < d; ++m)
                    C[(int64_t)j * d + m] = S[(int64_t)j * d + m] / (double)N[j];
            f[j] = mti_cdist(C + (int64_t)j * d, Cold + (int64_t)j * d, d);
        }
        if ((double)n_changed < tol * (double)n) {
            t += 1;
            break;
        }
    }
    *iters_out = t;
    memcpy(assign_out, a, (size_t)n * sizeof(int32_t));
    memcpy(C_out, C, kd * sizeof(double));
    free(C); free(Cold); free(S); free(N); free(h); free(s); free(f); free(a); free(u);
    return 0;
}
