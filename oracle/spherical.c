/*
 * CPU oracle for spherical k-means -- TEST INFRASTRUCTURE ONLY.
 *
 * Only the test suite, the package smoke check and the benchmark's CPU
 * baseline leg may load this code.  The GPU library never links it and shares
 * no code with it.
 *
 * What it computes (paper, section on spherical k-means among the
 * applications): every data point is projected to the unit sphere before
 * k-means runs, and point-to-centroid proximity is the cosine
 * cos(v, c) = v.c / (|v| |c|).  Written out here in float64, no pruning:
 *
 *   assignment : a_i = argmax_j cos(x_i, c_j), computed from the raw row and
 *                the centroid.  Ties: the previous assignment wins an exact
 *                tie, otherwise the lowest index (as for k-means).  A zero
 *                row has cosine 0 with every centroid (all tie).
 *   update     : the paper does not give the update; the reading taken is the
 *                mean of the members' unit vectors projected to the sphere,
 *                c_j = S_j / |S_j| with S_j the sum of the members' unit
 *                vectors; a cluster with no member or S_j = 0 keeps its
 *                centroid.  The cosine ignores |c_j|, so the assignments are
 *                those of any positive multiple of the mean.
 *   objective  : J = sum_i (2 - 2 cos(x_i, c_{a_i})), the squared chord
 *                distance between the unit vectors (what the Euclidean form
 *                on the sphere minimises).
 *   stopping   : as for k-means: stop after the update of step t when fewer
 *                than tol * n points changed, or after max_iters steps.
 *
 * C0 rows must be nonzero; they are projected to the sphere first.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

/* Unit vector of a float32 row in float64 (zero stays zero). */
static void unit_row(const float* x, int32_t d, double* out) {
    double s = 0.0;
    for (int32_t m = 0; m < d; ++m) s += (double)x[m] * (double)x[m];
    const double r = sqrt(s);
    for (int32_t m = 0; m < d; ++m) out[m] = r > 0.0 ? (double)x[m] / r : 0.0;
}

/* cos(x, c) from the raw float32 row x and a float64 centroid c. */
static double cosine(const float* x, const double* c, int32_t d) {
    double xc = 0.0, xx = 0.0, cc = 0.0;
    for (int32_t m = 0; m < d; ++m) {
        xc += (double)x[m] * c[m];
        xx += (double)x[m] * (double)x[m];
        cc += c[m] * c[m];
    }
    if (xx == 0.0 || cc == 0.0) return 0.0;
    return xc / (sqrt(xx) * sqrt(cc));
}

/*
 * Whole spherical run from C0 (k x d, any nonzero rows).  Outputs as for
 * oracle_lloyd: assign_out[n], C_out[k*d] (unit centroids after the last
 * update), *iters_out, and per step (nullable, length max_iters) the
 * objective and the changed count; best/second (nullable, length n) receive
 * the last step's smallest and second-smallest squared chord distances
 * 2 - 2 cos.  Returns 0, or -1 on bad arguments (including a zero C0 row) or
 * allocation failure.
 */
int32_t oracle_spherical(const float* X, int64_t n, int32_t d, int32_t k, const double* C0,
                         int32_t max_iters, double tol, int32_t* assign_out, double* C_out,
                         int32_t* iters_out, double* objective, int64_t* changed, double* best,
                         double* second) {
    if (!X || !C0 || !assign_out || !C_out || !iters_out || n < 1 || d < 1 || k < 1 || k > n ||
        max_iters < 1 || !(tol >= 0.0))
        return -1;
    const size_t kd = (size_t)k * (size_t)d;
    double* C = (double*)malloc(kd * sizeof(double));
    double* S = (double*)malloc(kd * sizeof(double));
    double* u = (double*)malloc((size_t)d * sizeof(double));
    int64_t* N = (int64_t*)malloc((size_t)k * sizeof(int64_t));
    int32_t* a = (int32_t*)malloc((size_t)n * sizeof(int32_t));
    double* b = (double*)malloc((size_t)n * sizeof(double));
    double* s2 = (double*)malloc((size_t)n * sizeof(double));
    int32_t rc = 0;
    if (!C || !S || !u || !N || !a || !b || !s2) {
        rc = -1;
        goto done;
    }
    for (int32_t j = 0; j < k; ++j) {   /* C0 projected to the sphere */
        double s = 0.0;
        for (int32_t m = 0; m < d; ++m) s += C0[(size_t)j * d + m] * C0[(size_t)j * d + m];
        if (!(s > 0.0)) {
            rc = -1;
            goto done;
        }
        const double r = sqrt(s);
        for (int32_t m = 0; m < d; ++m) C[(size_t)j * d + m] = C0[(size_t)j * d + m] / r;
    }
    int32_t t = 0;
    for (; t < max_iters; ++t) {
        int64_t ch = 0;
        double J = 0.0;
        for (int64_t i = 0; i < n; ++i) {
            const float* x = X + i * (int64_t)d;
            double cb = -INFINITY, c2 = -INFINITY, cprev = -INFINITY;
            int32_t arg = -1;
            const int32_t p = t == 0 ? -1 : a[i];
            for (int32_t j = 0; j < k; ++j) {
                const double cj = cosine(x, C + (size_t)j * d, d);
                if (j == p) cprev = cj;
                if (cj > cb) {
                    c2 = cb;
                    cb = cj;
                    arg = j;
                } else if (cj > c2) {
                    c2 = cj;
                }
            }
            if (p >= 0 && p != arg && cprev == cb) arg = p;   /* incumbent wins an exact tie */
            if (arg != p) ch += 1;
            a[i] = arg;
            b[i] = 2.0 - 2.0 * cb;
            s2[i] = c2 == -INFINITY ? INFINITY : 2.0 - 2.0 * c2;
            J += b[i];
        }
        if (objective) objective[t] = J;
        if (changed) changed[t] = ch;
        memset(S, 0, kd * sizeof(double));
        memset(N, 0, (size_t)k * sizeof(int64_t));
        for (int64_t i = 0; i < n; ++i) {   /* members' unit vectors, in index order */
            unit_row(X + i * (int64_t)d, d, u);
            double* sj = S + (size_t)a[i] * d;
            for (int32_t m = 0; m < d; ++m) sj[m] += u[m];
            N[a[i]] += 1;
        }
        for (int32_t j = 0; j < k; ++j) {
            double s = 0.0;
            for (int32_t m = 0; m < d; ++m) s += S[(size_t)j * d + m] * S[(size_t)j * d + m];
            if (N[j] > 0 && s > 0.0) {
                const double r = sqrt(s);
                for (int32_t m = 0; m < d; ++m) C[(size_t)j * d + m] = S[(size_t)j * d + m] / r;
            }
        }
        if ((double)ch < tol * (double)n) {
            t += 1;
            break;
        }
    }
    *iters_out = t;
    memcpy(assign_out, a, (size_t)n * sizeof(int32_t));
    memcpy(C_out, C, kd * sizeof(double));
    if (best) memcpy(best, b, (size_t)n * sizeof(double));
    if (second) memcpy(second, s2, (size_t)n * sizeof(double));
done:
    free(C); free(S); free(u); free(N); free(a); free(b); free(s2);
    return rc;
}
