/*
 * CPU oracle for k-means++ seeding -- TEST INFRASTRUCTURE ONLY.
 *
 * Only the test suite, the package smoke check and the benchmark's CPU
 * baseline leg may load this code.  The GPU library never links it and shares
 * no code with it.
 *
 * What it computes (paper section IV-C, equation of the D^2 weighting): the
 * first seed is a uniformly drawn data point; every further seed is a data
 * point drawn with probability D(v)^2 / sum_v D(v)^2, where D(v) is the
 * distance from v to the nearest seed chosen so far.  The uniform numbers
 * are inputs (u[0..k-1], each in [0, 1)), so a run is a pure function of
 * (X, k, u).  Written out plainly:
 *
 *   D^2      : squared Euclidean distance of a float32 row to a seed row,
 *              in float64, coordinate differences summed in index order with
 *              a fused multiply-add (acc = fma(x_m - c_m, x_m - c_m, acc)), so
 *              that any implementation following the same order reaches the
 *              same value bit for bit.  D2[i] = min over the seeds so far.
 *   first    : i_0 = min(floor(u_0 * n), n - 1).
 *   weights  : the draw of seed t+1 (after D2 holds the distances to seeds
 *              0..t) uses integer weights w_i = floor(D2[i] * 2^S_t) whose sum
 *              is exact in any order, so the draw is D2 / sum D2 up to the
 *              rounding of each weight.  S_t = 62 - e - L, where L is the
 *              smallest integer with n <= 2^L and e the smallest integer with
 *              M < 2^e for M = max_i D2[i], the current maximum; then every
 *              w_i < 2^(62 - L) and the sum is <= 2^62.  M = 0 gives all-zero
 *              weights.  The largest weight keeps at least 61 - L
 *              significant bits, and each weight is D2[i] * 2^S_t less a
 *              fraction below one unit.
 *   draw     : W = sum_i w_i, T = min(floor(u_{t+1} * W), W - 1) (the
 *              product in float64), and seed t+1 is the smallest i whose
 *              inclusive prefix sum of w exceeds T.  If W = 0 (every point
 *              coincides with a seed) the draw is uniform as for i_0.
 *
 * Outputs: idx_out[k] (the seed indices in draw order) and, nullable,
 * D2_out[n] (the distances to the nearest of all k seeds).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

/* Squared distance of row x to row c, float64, index order, fused. */
static double dist2_rows(const float* x, const float* c, int32_t d) {
    double acc = 0.0;
    for (int32_t m = 0; m < d; ++m) {
        const double df = (double)x[m] - (double)c[m];
        acc = fma(df, df, acc);
    }
    return acc;
}

static int64_t uniform_index(double u, int64_t n) {
    int64_t i = (int64_t)(u * (double)n);
    return i < n - 1 ? i : n - 1;
}

/* The scale exponent S for the bound M (see the header). */
static int32_t weight_scale(double M, int64_t n) {
    if (!(M > 0.0)) return 0;
    int e = 0;
    (void)frexp(M, &e);   /* M = f * 2^e, 0.5 <= f < 1, so M < 2^e */
    int32_t L = 0;
    while (((int64_t)1 << L) < n) ++L;
    return 62 - e - L;
}

static uint64_t weight_of(double d2, int32_t S) {
    return (uint64_t)floor(ldexp(d2, S));
}

/* One update of D2 with seed row c (first: D2 starts empty); returns the max. */
static double update_d2(const float* X, int64_t n, int32_t d, const float* c, int first, double* D2) {
    double M = 0.0;
#pragma omp parallel for schedule(static) reduction(max : M)
    for (int64_t i = 0; i < n; ++i) {
        const double v = dist2_rows(X + i * (int64_t)d, c, d);
        const double nv = first ? v : (v < D2[i] ? v : D2[i]);
        D2[i] = nv;
        if (nv > M) M = nv;
    }
    return M;
}

/*
 * Seeds k rows of X (n x d).  Returns 0, or -1 on bad arguments (k outside
 * 1..n, a u outside [0, 1)) or allocation failure.
 */
int32_t oracle_kmeanspp(const float* X, int64_t n, int32_t d, int32_t k, const double* u, int64_t* idx_out,
                        double* D2_out) {
    if (!X || !u || !idx_out || n < 1 || d < 1 || k < 1 || k > n) return -1;
    for (int32_t t = 0; t < k; ++t)
        if (!(u[t] >= 0.0 && u[t] < 1.0)) return -1;
    double* D2 = (double*)malloc((size_t)n * sizeof(double));
    if (!D2) return -1;

    idx_out[0] = uniform_index(u[0], n);
    for (int32_t t = 0; t < k; ++t) {
        const double M = update_d2(X, n, d, X + idx_out[t] * (int64_t)d, t == 0, D2);
        if (t == k - 1) break;   /* the last update only completes D2_out */
        const int32_t S = weight_scale(M, n);
        uint64_t W = 0;
        for (int64_t i = 0; i < n; ++i) W += weight_of(D2[i], S);
        int64_t pick;
        if (W == 0) {
            pick = uniform_index(u[t + 1], n);
        } else {
            uint64_t T = (uint64_t)(u[t + 1] * (double)W);
            if (T >= W) T = W - 1;
            uint64_t P = 0;
            pick = n - 1;
            for (int64_t i = 0; i < n; ++i) {
                P += weight_of(D2[i], S);
                if (P > T) {
                    pick = i;
                    break;
                }
            }
        }
        idx_out[t + 1] = pick;
    }
    if (D2_out) memcpy(D2_out, D2, (size_t)n * sizeof(double));
    free(D2);
    return 0;
}
