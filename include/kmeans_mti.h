/*
 * kmeans_mti.h -- C ABI of the MI355X (gfx950) k-means hot path:
 * Lloyd's k-means with Minimal Triangle Inequality (MTI) pruning.
 *
 * Method (Mhembere et al., "clusterNOR: A NUMA-Optimized Clustering
 * Framework", arXiv 1902.09527):
 *   - one iteration is the merged assignment + update step of ||Lloyd's
 *     (section III-B): every point is assigned to its nearest centroid under
 *     the Euclidean distance of Table I, then each centroid becomes the mean
 *     of its members (section IV-A);
 *   - MTI pruning (section III-C) keeps one upper bound u per point and the
 *     centroid-to-centroid distances; a point whose bound is within half the
 *     distance from its centroid to the nearest other centroid keeps its
 *     assignment with no distance work (Clause 1), and single point-centroid
 *     distances are skipped by the same test per centroid before and after
 *     the bound is tightened (Clauses 2 and 3); after each update the bound
 *     grows by the drift f(c) = d(c^t, c^{t-1}) of its centroid (Table I).
 * MTI is exact: the results are those of unpruned Lloyd's.
 *
 * Results.  Assignment ties: the previous assignment wins an exact tie,
 * otherwise the lowest centroid index.  A cluster with no member keeps its
 * centroid.  Per-cluster sums are exact integer sums of the inputs in a fixed
 * binary point (scale 2^S with S chosen at init so that no sum can
 * overflow), so results do not depend on thread scheduling: two runs on the
 * same inputs are bitwise identical.  Distances run in float32; a point
 * whose best and second-best float32 distances are within the float32 error
 * bound is decided again in float64 against float64 master centroids.
 *
 * Memory.  X, C0, assign_out and C_out are DEVICE pointers (HIP device
 * memory of the current device).  X is n rows of d contiguous float32
 * (row-major, row stride d); C0 / C_out are k rows of d float32; assign_out
 * is n int32.  The library borrows X for the lifetime of a context (it is
 * read every iteration and must not change) and never frees caller memory.
 * A context owns all its scratch (bounds, assignments, float64 centroids,
 * per-block partial sums, counters).
 *
 * Streams.  All device work is ordered on the hip_stream given at init
 * (NULL = the null stream).  Calls marked "synchronizes" wait for that
 * stream.  A context is not thread-safe: use one context per host thread.
 *
 * Errors.  Every int-returning entry point returns KM_OK or a negative
 * KM_ERR_* code and never throws.  On KM_ERR_HIP the HIP runtime's message
 * is available from kmeans_mti_last_hip_error() (per host thread).  After a
 * failed init *out is NULL.  A context whose device work failed returns
 * KM_ERR_STATE from later calls except kmeans_mti_destroy.
 */
#ifndef KMEANS_MTI_H
#define KMEANS_MTI_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct km_ctx km_ctx;

enum {
    KM_OK = 0,
    KM_ERR_INVALID_ARG = -1,   /* null pointer, bad size, k > n, tol < 0 or NaN, n*d overflow */
    KM_ERR_OOM = -2,           /* a device or host allocation failed */
    KM_ERR_HIP = -3,           /* a HIP runtime call failed; see kmeans_mti_last_hip_error() */
    KM_ERR_UNSUPPORTED = -4,   /* no kernel path handles this shape */
    KM_ERR_STATE = -5,         /* context is unusable (earlier device failure) */
    KM_ERR_NONFINITE = -6      /* KM_FLAG_VALIDATE: X or C0 holds a NaN or an infinity */
};

enum {
    KM_FLAG_NO_PRUNE = 1u,     /* compute all k distances every iteration (plain Lloyd's) */
    KM_FLAG_STATS = 2u,        /* also accumulate the inertia sum_i ||x_i - c_{a_i}||^2 */
    KM_FLAG_VALIDATE = 4u,     /* reject non-finite X or C0 at init with KM_ERR_NONFINITE */
    KM_FLAG_TIMING = 8u,       /* record HIP events around every kernel (kmeans_mti_get_timing) */
    KM_FLAG_VECTOR_ONLY = 16u, /* use the per-point vector distance loop even where the
                                  matrix-core (MFMA) survivor path applies; same results */
    KM_FLAG_LARGE_PATH = 32u,  /* use the global-memory path (dense MFMA survivors, sums by
                                  counting sort) even where the LDS path fits; same results */
    KM_FLAG_GENERIC = 64u,     /* use the general assignment kernel and separate reduction,
                                  update and table launches even where the streaming step
                                  (d = 16, k <= 16) applies; same results */
    KM_FLAG_FULL_SUMS = 128u,  /* recompute the per-cluster sums from every point (one full
                                  read of X) in every step instead of moving the sums of the
                                  points whose assignment changed, where only the Clause-1
                                  survivors' rows are read after the first step (the
                                  streaming path, d = 16 and k <= 16, and the incremental
                                  matrix-core path, d = 16 or 32 and k <= 128); same results.
                                  Implied by KM_FLAG_STATS. */
    KM_FLAG_SPHERICAL = 256u,  /* spherical k-means (the paper's sk-means application): the
                                  rows of X are projected to the unit sphere (into a copy the
                                  context owns; a zero row stays zero) and C0 likewise, the
                                  assignment maximises the cosine (the nearest unit centroid),
                                  and each update projects the members' mean to the sphere (a
                                  cluster with no member or a zero mean keeps its centroid).
                                  C0 rows must be nonzero (else KM_ERR_INVALID_ARG).  Centroid
                                  outputs are unit vectors; the inertia is the sum of squared
                                  chord distances 2 - 2 cos. */
    KM_FLAG_ELKAN = 512u       /* comparator: Elkan's triangle-inequality pruning (the TI that
                                  MTI relaxes, section III-C) instead of MTI: one lower bound per
                                  point and centroid (4 n k bytes of device memory), a centroid
                                  is skipped when the point's bound is within its lower bound or
                                  within half the centroid distance, and the incumbent's
                                  distance is computed only when some centroid passes both
                                  tests.  Centroids and sums must fit in LDS (else
                                  KM_ERR_UNSUPPORTED); not with KM_FLAG_LARGE_PATH.  Same
                                  results as MTI; path "lds-elkan". */
};

/* Totals over the iterations run so far (kmeans_mti_get_stats, kmeans_mti_run). */
typedef struct {
    int32_t iterations;        /* assignment steps executed */
    int32_t converged;         /* run only: 1 if it stopped on the tol test before max_iters */
    int64_t changed_last;      /* points whose assignment changed in the last step */
    int64_t dist_computed;     /* float32 point-centroid distances evaluated, tightenings included */
    int64_t dist_lloyd;        /* n * k * iterations: what unpruned Lloyd's evaluates */
    int64_t clause1_skips;     /* point-iterations skipped whole by Clause 1 */
    int64_t rechecks;          /* points decided again in float64 (near ties) */
    double inertia_last;       /* last step's inertia (float32 distances summed exactly); NaN without KM_FLAG_STATS */
    double device_ms;          /* run only: device time of the iteration loop (HIP events); else 0 */
} km_stats;

/*
 * Create a context for one k-means problem and compute the centroid table of
 * C0.  X: device, n x d float32, borrowed until kmeans_mti_destroy.  C0:
 * device, k x d float32, copied (may be freed after the call).  Requires
 * n >= 1, 1 <= d, 1 <= k <= n.  hip_stream: a hipStream_t or NULL.  flags:
 * KM_FLAG_*.  Synchronizes.  On success *out owns the context.
 */
int kmeans_mti_init(km_ctx** out, const float* X, int64_t n, int32_t d, int32_t k,
                    const float* C0, void* hip_stream, uint32_t flags);

/*
 * Enqueue one iteration: the assignment step with MTI pruning, then the
 * update of the centroids, their drift and their distance table (one
 * ||Lloyd's iteration, section III-B).  Asynchronous unless changed_out is
 * non-NULL, in which case it synchronizes and stores the number of points
 * whose assignment changed in this step (n in the first step).
 */
int kmeans_mti_iterate(km_ctx* ctx, int64_t* changed_out);

/*
 * Copy the current state into caller device buffers (either may be NULL):
 * assign_out (n int32) = assignment of the last step, C_out (k x d float32)
 * = centroids after the last update (C0 before the first iteration).
 * Stream-ordered, asynchronous.  KM_ERR_STATE before the first iteration
 * when assign_out is non-NULL.
 */
int kmeans_mti_get(km_ctx* ctx, int32_t* assign_out, float* C_out);

/* Copy the float64 master centroids (k x d) into a HOST buffer.  Synchronizes. */
int kmeans_mti_get_centroids64(km_ctx* ctx, double* C_out);

/* Totals over the iterations run so far.  Synchronizes. */
int kmeans_mti_get_stats(km_ctx* ctx, km_stats* stats);

/*
 * Per-iteration history into HOST arrays of length cap (any may be NULL):
 * changed, distances computed, Clause-1 skips, float64 rechecks, inertia
 * (NaN without KM_FLAG_STATS).  Returns the number of iterations written
 * (min(iterations, cap, 4096): the context keeps the last 4096), or a
 * negative KM_ERR_*.  Synchronizes.
 */
int kmeans_mti_get_history(km_ctx* ctx, int64_t* changed, int64_t* computed, int64_t* clause1,
                           int64_t* rechecks, double* inertia, int32_t cap);

/*
 * Device time per kernel over the iterations enqueued so far, measured with
 * HIP events recorded on the context's stream around every launch (needs
 * KM_FLAG_TIMING at init).  ms (HOST, 4 doubles) receives the total
 * milliseconds of the assignment, reduction, update and centroid-table
 * kernels (on the global-memory path the assignment slot holds the Clause-1
 * pass and the matrix-core distances, and the refinement of their
 * candidates is timed with the reduction); *iters (nullable) the number of
 * iterations timed.  Synchronizes.
 * KM_ERR_STATE without KM_FLAG_TIMING.
 */
int kmeans_mti_get_timing(km_ctx* ctx, double* ms, int64_t* iters);

/*
 * Whole run (the paper's base::run): iterate from C0 until fewer than
 * tol * n points change assignment in a step (checked after that step's
 * update; tol = 0 runs all steps) or max_iters steps ran.  Outputs as in
 * kmeans_mti_get.  All iterations are enqueued without host round trips;
 * steps after convergence return at once.  Synchronizes once at the end.
 * stats: HOST pointer, may be NULL.
 */
int kmeans_mti_run(const float* X, int64_t n, int32_t d, int32_t k, const float* C0,
                   int32_t max_iters, double tol, int32_t* assign_out, float* C_out,
                   void* hip_stream, uint32_t flags, km_stats* stats);

/*
 * Name of the kernel path the context uses, a static string: "stream-d16"
 * (d = 16, k <= 16: the streaming kernel k_small in the first step, then
 * the incremental kernel k_inc, each launch of which also ends the step
 * before it; the one-block update k_small_finish runs after k_small and
 * before results are read), "stream-d16-full" (k_small every step, each
 * followed by k_small_finish, with KM_FLAG_FULL_SUMS or KM_FLAG_STATS),
 * "lds-vector" /
 * "lds-mfma" (centroids and sums in LDS: k_assign with vector or matrix-core
 * survivors, then k_reduce, k_update, k_centroid_table), "lds-inc" (d = 16
 * or 32, k <= 128, where the streaming path does not apply: k_inc_mm reads
 * the point states and only the Clause-1 survivors' rows, settles the
 * survivors on the matrix cores and sums the moves of the points whose
 * cluster changed; then k_reduce, k_update, k_centroid_table), "lds-elkan" (the
 * same with KM_FLAG_ELKAN's lower-bound scan), "global-mfma"
 * (centroids or sums too large for LDS: dense MFMA survivors, sums by
 * counting sort).  "" for a NULL context.
 */
const char* kmeans_mti_path(const km_ctx* ctx);

/*
 * k-means++ seeding (section IV-C, the equation of the D^2 weighting): seed 0
 * is row min(floor(u[0] * n), n - 1); seed t+1 is row i drawn with probability
 * D2_i / sum D2, D2_i the squared distance from row i to its nearest seed so
 * far.  The caller draws the uniforms, so the result is a deterministic
 * function of (X, k, u):
 *   - D2 is float64 with the coordinate differences summed in index order by
 *     fused multiply-add;
 *   - the draw of seed t+1 uses integer weights w_i = floor(D2_i * 2^S),
 *     S = 62 - e - ceil(log2 n) with M < 2^e for M = max D2 after the pass
 *     with seed t (the current maximum); W = sum w_i,
 *     T = min(floor(u[t+1] * W), W - 1)
 *     (float64 product), and the seed is the smallest i whose inclusive
 *     prefix sum of w exceeds T; W = 0 (every row lies on a seed) draws
 *     min(floor(u[t+1] * n), n - 1).
 * A pass skips row i when its nearest seed a satisfies
 * ||c_a - c_new||^2 >= 4 D2_i (with rounding margins): exact, since such a
 * seed cannot be nearer (KM_PP_NO_PRUNE computes every distance; same
 * results).
 *
 * X: device, n x d float32 rows (finite; non-finite rows give unspecified
 * seeds).  u: HOST, k doubles in [0, 1), read before the call returns.
 * C_out: device, k x d float32, receives the seed rows in draw order.
 * idx_out: device int64[k] (nullable), the seed row indices.  d2_out: device
 * float64[n] (nullable), each row's squared distance to its nearest seed.
 * workspace: device, at least kmeans_pp_workspace_bytes(n, d, k) bytes,
 * 256-byte aligned, owned by the caller; its contents on entry do not matter
 * and it must not be used by another call until this one's work completes.
 * Requires 1 <= k <= n, d >= 1.  Work is ordered on hip_stream (NULL = null
 * stream) with at most 4k kernel launches and no allocation; asynchronous unless
 * stats (HOST, nullable) is given, in which case it synchronizes and fills
 * it.  Errors: KM_ERR_INVALID_ARG for bad sizes or pointers, a u outside
 * [0, 1), unknown flags or a short or misaligned workspace; KM_ERR_HIP on a
 * launch failure.
 */
enum {
    KM_PP_NO_PRUNE = 1u,   /* compute every point-seed distance (same results) */
    KM_PP_TIMING = 2u      /* with stats: HIP events around every launch */
};

typedef struct {
    int64_t computed;      /* point-seed distances evaluated over all passes */
    int64_t improved;      /* rows whose D2 decreased, summed over the passes after the first */
    int32_t passes;        /* passes over the points (k) */
    int32_t pad_;
    double pass_ms;        /* KM_PP_TIMING: device time of the k passes (k_pp_step), else 0 */
    double later_pass_ms;  /* KM_PP_TIMING: of passes 2..k only */
    double draw_ms;        /* KM_PP_TIMING: set-up, first weights, the k - 1 draws and seed tables */
} km_pp_stats;

size_t kmeans_pp_workspace_bytes(int64_t n, int32_t d, int32_t k);   /* 0 for bad sizes */
int kmeans_pp_seed(const float* X, int64_t n, int32_t d, int32_t k, const double* u, float* C_out,
                   int64_t* idx_out, double* d2_out, void* workspace, size_t workspace_bytes,
                   uint32_t flags, void* hip_stream, km_pp_stats* stats);

/*
 * kmeans_pp_seed for callers that cannot allocate (code under HIP stream
 * capture, tight serving loops, harnesses that forbid hipMalloc): the
 * workspace is a fixed device array of KMEANS_PP_STATIC_WORKSPACE_BYTES
 * (64 MiB) that the library holds on every device it runs on until the
 * process ends, instead of a caller's buffer.  The call makes no hipMalloc,
 * hipFree, event or host allocation.
 *
 * Arguments, results and errors as kmeans_pp_seed (without workspace and
 * stats), except: KM_ERR_INVALID_ARG when kmeans_pp_workspace_bytes(n, d, k)
 * exceeds KMEANS_PP_STATIC_WORKSPACE_BYTES (about 12 bytes per row: n up to
 * about 5.5 million for small k), and when flags hold anything but
 * KM_PP_NO_PRUNE.  The first call on a device looks up the array's device
 * address there (hipGetSymbolAddress, with that device current).
 *
 * All calls on one device share its array and leave their contents in it
 * (each call overwrites what it reads).  Calls that overlap on one device --
 * on different streams, or from host threads without ordering between them --
 * race and give unspecified seeds; calls ordered on one stream are safe.
 */
#define KMEANS_PP_STATIC_WORKSPACE_BYTES ((size_t)64 << 20)
int kmeans_pp_seed_noalloc(const float* X, int64_t n, int32_t d, int32_t k, const double* u, float* C_out,
                           int64_t* idx_out, double* d2_out, uint32_t flags, void* hip_stream);

/*
 * k-means++ with restarts (section IV-C: the best of several seeded runs).
 * For each run q = 0..r-1: seed k rows with kmeans_pp_seed from the uniforms
 * U[q*k .. q*k + k - 1], run k-means from those seeds as kmeans_mti_run does
 * (max_iters, tol, flags with KM_FLAG_STATS added), and keep the run with the
 * least final inertia (float32 distances summed exactly); an exact tie keeps
 * the earlier run.
 *
 * X: device, n x d float32.  U: HOST, r * k doubles in [0, 1).  assign_out
 * (n int32) and C_out (k x d float32): device, receive the kept run's
 * assignment and centroids.  best_out (HOST, nullable): the kept run's index.
 * inertia_out (HOST, nullable, r doubles): every run's final inertia.  stats
 * (HOST, nullable): the kept run's totals.  Requires r >= 1 and the sizes of
 * kmeans_mti_run; flags as for kmeans_mti_run (KM_FLAG_NO_PRUNE also
 * computes every seeding distance).  Allocates its device workspace (the
 * seeding workspace, the seeds and one spare run's outputs) and frees it
 * before returning.  Synchronizes.  Errors as kmeans_mti_run and
 * kmeans_pp_seed.
 */
int kmeans_pp_run_best(const float* X, int64_t n, int32_t d, int32_t k, const double* U, int32_t r,
                       int32_t max_iters, double tol, int32_t* assign_out, float* C_out,
                       void* hip_stream, uint32_t flags, int32_t* best_out, double* inertia_out,
                       km_stats* stats);

/*
 * Release a context.  NULL-safe.  Synchronizes.  Its device buffers are kept
 * by the library (per device and size, at most 8 GiB in all) for the next
 * context that needs the same sizes, so that repeated runs of a problem make
 * no hipMalloc / hipFree calls; kmeans_mti_release_cache frees them.
 */
void kmeans_mti_destroy(km_ctx* ctx);

/* Free the device buffers kept from released contexts (all devices).  Call
 * it with no context in use on another host thread. */
void kmeans_mti_release_cache(void);

/* Static text for a KM_* status code. */
const char* kmeans_mti_strerror(int status);

/* Text of the last HIP error seen on this host thread ("" if none). */
const char* kmeans_mti_last_hip_error(void);

#ifdef __cplusplus
}
#endif

#endif /* KMEANS_MTI_H */
