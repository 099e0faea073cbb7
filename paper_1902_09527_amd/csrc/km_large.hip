// Global-memory path of the MTI k-means hot path for gfx950 (MI355X), used
// when the centroids or the per-cluster sums do not fit in LDS (large k*d,
// e.g. k = 1000, d = 256).  One iteration (one ||Lloyd's MM step, paper
// section III-B) is:
//   k_bound_large       drift-updated bound and Clause 1 (section III-C) for
//                       every point; survivors compacted into a global list;
//   k_mfma_large        float32 MFMA distances of the survivors to all
//                       centroids (dense 64-survivor x 128-centroid tiles,
//                       expanded form), a top-4 candidate list per survivor,
//                       direct-form refinement of the candidates within the
//                       expanded form's error bound, float64 near-tie rule;
//   k_hist_large        per-block cluster counts of the new assignment;
//   k_scan_large_cols,
//   k_scan_large_clusters  cluster starts and per-block write offsets;
//   k_scatter_large     point indices grouped by cluster (counting sort);
//   k_segsum_large      exact fixed-point sums over chunks of each cluster;
//   k_chunk_reduce_large  per-cluster sums, counts and the inertia into the
//                       reduced row read by k_update;
//   k_centroid_table_tiled  half centroid distances for the next step.
// The order of points inside a cluster segment is not fixed, but every sum
// is an exact integer sum, so results are bitwise reproducible.
#include <limits.h>
#include <math.h>

#include "kmeans_mti.h"
#include "km_device.h"
#include "km_internal.h"

namespace km {

namespace {

constexpr int kTiTile = 16;   // centroid rows per block of the tiled centroid table

// Insert (v, j) into an ascending 4-list ordered by value, then index.
__device__ inline void top4_insert(float (&L)[4], int (&J)[4], float v, int j) {
    if (!(v < L[3] || (v == L[3] && j < J[3]))) return;
    L[3] = v;
    J[3] = j;
#pragma unroll
    for (int q = 3; q > 0; --q) {
        const bool sw = L[q] < L[q - 1] || (L[q] == L[q - 1] && J[q] < J[q - 1]);
        if (sw) {
            const float tv = L[q];
            L[q] = L[q - 1];
            L[q - 1] = tv;
            const int tj = J[q];
            J[q] = J[q - 1];
            J[q - 1] = tj;
        }
    }
}

__device__ inline float quad_sum(float v) {
    v += __shfl_xor(v, 1);
    v += __shfl_xor(v, 2);
    return v;
}
__device__ inline double quad_sum(double v) {
    v += __shfl_xor(v, 1);
    v += __shfl_xor(v, 2);
    return v;
}

}  // namespace

// ---------------------------------------------------------------------------
// Bound update and Clause 1 for every point; survivors to the global list.

__global__ __launch_bounds__(256) void k_bound_large(Dev P, Large Lg) {
    IterState* st = P.st;
    if (st->done) {
        if (blockIdx.x == 0 && threadIdx.x == 0) st->active = 0;
        return;
    }
    if (blockIdx.x == 0 && threadIdx.x == 0) st->active = 1;
    const bool first = st->t == 0;
    const bool prune = !(P.flags & KM_FLAG_NO_PRUNE);
    const int lane = threadIdx.x & 63;
    uint64_t c1 = 0;
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t i0 = (int64_t)blockIdx.x * blockDim.x; i0 < P.n; i0 += stride) {
        const int64_t i = i0 + threadIdx.x;
        bool surv = false;
        if (i < P.n) {
            if (first) {
                surv = true;
            } else {
                const int a = P.a[i];
                const float u = (P.u[i] + P.f[a]) * kUp;
                if (!prune || u > P.s[a]) {
                    surv = true;
                } else {
                    c1 += 1;
                    P.u[i] = u;
                }
            }
        }
        const uint64_t m = __ballot(surv);
        if (m) {
            uint32_t b = 0;
            if (lane == 0) b = atomicAdd(Lg.nsurv, (uint32_t)__popcll(m));
            b = __shfl(b, 0);
            if (surv) Lg.surv[b + __popcll(m & ((1ull << lane) - 1ull))] = (int32_t)i;
        }
    }
    c1 = wave_sum_u64(c1);
    if (lane == 0 && c1)
        atomicAdd(reinterpret_cast<unsigned long long*>(&P.total[(int64_t)P.k * P.d + P.k + kStClause1]),
                  (unsigned long long)c1);
}

// ---------------------------------------------------------------------------
// Dense survivor distances on the matrix cores.  Workgroup tile: 64
// survivors (two 32-column MFMA blocks) x 128 centroids (32 per wave); the
// survivor tile stays in LDS dimension-major for all centroid tiles, the
// centroid tile streams through LDS in 32-dimension chunks (double
// buffered).  MFMA k-step s pairs chunk dimensions s and 16 + s.

__global__ __launch_bounds__(256) void k_mfma_large(Dev P, Large Lg) {
    IterState* st = P.st;
    if (!st->active) return;
    const int k = P.k, d = P.d, dp = Lg.dp;
    const bool first = st->t == 0;
    const uint32_t ns = *Lg.nsurv;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, col = lane & 31, half = lane >> 5;
    constexpr int XW = kLgSurvTile + 1;   // padded survivor-tile row (per dimension)
    constexpr int CW = kLgCentTile + 1;   // padded centroid-chunk row (per dimension)
    extern __shared__ __align__(16) unsigned char smem[];
    float* XT = reinterpret_cast<float*>(smem);             // [dp][XW]
    float* CT = XT + dp * XW;                                // [2][32][CW]
    float* candD = CT + 2 * 32 * CW;                         // [64][32]
    int* candJ = reinterpret_cast<int*>(candD + kLgSurvTile * 32);
    float* x2s = reinterpret_cast<float*>(candJ + kLgSurvTile * 32);   // [64]
    float* red = x2s + kLgSurvTile;                          // [16]

    const float ecm = st->ec_max;
    const float gamma = P.gamma;
    const float gexp = (float)(d + 8) * 0x1p-24f;
    // Largest centroid norm (for the expanded-form error bound).
    float m2 = 0.f;
    for (int j = tid; j < k; j += blockDim.x) m2 = fmaxf(m2, P.cn2[j]);
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) m2 = fmaxf(m2, __shfl_xor(m2, off));
    if (lane == 0) red[wave] = m2;
    __syncthreads();
    const float cnmax = sqrtf(fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]))) * kUp;

    uint64_t my_changed = 0, my_comp = 0, my_rc = 0;
    const int ntiles = (int)((ns + kLgSurvTile - 1) / kLgSurvTile);
    const int nct = (k + kLgCentTile - 1) / kLgCentTile;
    const int nch = dp / 32;

    for (int tile = blockIdx.x; tile < ntiles; tile += gridDim.x) {
        const int s0 = tile * kLgSurvTile;
        const int rows = min(kLgSurvTile, (int)ns - s0);
        __syncthreads();   // the previous tile's LDS data is consumed
        // Survivor tile, dimension-major, zero padded.
        for (int e = tid; e < kLgSurvTile * dp; e += blockDim.x) {
            const int c = e / dp, m = e - c * dp;
            float v = 0.f;
            if (c < rows && m < d) v = P.X[(int64_t)Lg.surv[s0 + c] * d + m];
            XT[m * XW + c] = v;
        }
        __syncthreads();
        if (tid < kLgSurvTile) {
            float acc = 0.f;
            for (int m = 0; m < d; ++m) acc = fmaf(XT[m * XW + tid], XT[m * XW + tid], acc);
            x2s[tid] = acc;
        }
        float L0[4], L1[4];
        int J0[4], J1[4];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            L0[q] = L1[q] = INFINITY;
            J0[q] = J1[q] = INT_MAX;
        }
        int g = 0;   // running chunk count: buffer parity alternates across centroid tiles too
        for (int ct = 0; ct < nct; ++ct) {
            f32x16 acc0, acc1;
#pragma unroll
            for (int e = 0; e < 16; ++e) acc0[e] = acc1[e] = 0.f;
            for (int c = 0; c < nch; ++c, ++g) {
                float* cb = CT + (g & 1) * 32 * CW;
                for (int e = tid; e < kLgCentTile * 32; e += blockDim.x) {
                    const int cj = e >> 5, m = e & 31;
                    const int j = ct * kLgCentTile + cj, dim = c * 32 + m;
                    cb[m * CW + cj] = (j < k && dim < d) ? P.C32[(int64_t)j * d + dim] : 0.f;
                }
                __syncthreads();
                const float* xb = XT + (c * 32) * XW;
#pragma unroll
                for (int s = 0; s < 16; ++s) {
                    const int dm = s + 16 * half;
                    const float a = cb[dm * CW + wave * 32 + col];
                    const float b0 = xb[dm * XW + col];
                    const float b1 = xb[dm * XW + 32 + col];
                    acc0 = __builtin_amdgcn_mfma_f32_32x32x2f32(a, b0, acc0, 0, 0, 0);
                    acc1 = __builtin_amdgcn_mfma_f32_32x32x2f32(a, b1, acc1, 0, 0, 0);
                }
            }
            // Register e holds centroid ct*128 + wave*32 + 8*(e/4) + 4*half + e%4.
            const float xa = x2s[col], xb2 = x2s[32 + col];
#pragma unroll
            for (int e = 0; e < 16; ++e) {
                const int j = ct * kLgCentTile + wave * 32 + 8 * (e >> 2) + 4 * half + (e & 3);
                const float cn = j < k ? P.cn2[j] : INFINITY;
                top4_insert(L0, J0, xa + cn - 2.f * acc0[e], j);
                top4_insert(L1, J1, xb2 + cn - 2.f * acc1[e], j);
            }
        }
        // Merge the 8 partial lists of each survivor (4 waves x 2 halves).
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int slot = (wave * 2 + half) * 4 + q;
            candD[col * 32 + slot] = L0[q];
            candJ[col * 32 + slot] = J0[q];
            candD[(32 + col) * 32 + slot] = L1[q];
            candJ[(32 + col) * 32 + slot] = J1[q];
        }
        __syncthreads();

        // Refinement: 4 threads per survivor, each a quarter of the dimensions.
        const int c = tid >> 2, part = tid & 3;
        if (c < rows) {
            float T[4];
            int TJ[4];
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                T[q] = INFINITY;
                TJ[q] = INT_MAX;
            }
            for (int q = 0; q < 32; ++q) top4_insert(T, TJ, candD[c * 32 + q], candJ[c * 32 + q]);
            const int64_t i = Lg.surv[s0 + c];
            const int inc = first ? -1 : P.a[i];
            const int qd = (d + 3) / 4, m0 = part * qd, m1 = min(d, m0 + qd);
            const float R = sqrtf(fmaxf(x2s[c], 0.f)) * kUp + cnmax;
            const float thr = T[0] + 2.f * (gexp * R * R + 4.f * R * ecm + 2.f * ecm * ecm);
            // A fourth candidate inside the bound means more may lie outside
            // the list: decide in float64 then.
            bool re = T[3] <= thr;
            float d1 = INFINITY, d2 = INFINITY;
            int rk1 = INT_MAX, j1 = 0;
            if (!re) {
                for (int q = 0; q < 3; ++q) {
                    if (!(T[q] <= thr) || TJ[q] >= k) continue;   // uniform in the quad
                    const int j = TJ[q];
                    const float* cr = P.C32 + (int64_t)j * d;
                    float acc = 0.f;
                    for (int m = m0; m < m1; ++m) {
                        const float t = XT[m * XW + c] - cr[m];
                        acc = fmaf(t, t, acc);
                    }
                    const float Dd = quad_sum(acc);
                    const int rk = j == inc ? -1 : j;
                    if (Dd < d1 || (Dd == d1 && rk < rk1)) {
                        d2 = d1;
                        d1 = Dd;
                        rk1 = rk;
                        j1 = j;
                    } else if (Dd < d2) {
                        d2 = Dd;
                    }
                }
                if (d2 != INFINITY) {
                    const float band =
                        2.f * gamma * (d1 + d2) + 4.f * (sqrtf(d1) + sqrtf(d2)) * ecm + 8.f * ecm * ecm;
                    if (d2 - d1 <= band) re = true;
                }
            }
            int b = j1;
            float ub = upper_bound(d1, P.ec[j1], gamma);
            if (re) {
                // float64 decision against the master centroids, oracle's tie rule.
                double Dbb = INFINITY;
                int bb = -1;
                auto d64 = [&](int j) {
                    const double* cr = P.C64 + (int64_t)j * d;
                    double acc = 0.0;
                    for (int m = m0; m < m1; ++m) {
                        const double t = (double)XT[m * XW + c] - cr[m];
                        acc = fma(t, t, acc);
                    }
                    return quad_sum(acc);
                };
                if (inc >= 0) {
                    Dbb = d64(inc);
                    bb = inc;
                }
                for (int j = 0; j < k; ++j) {
                    if (j == inc) continue;
                    const double Dj = d64(j);
                    if (Dj < Dbb) {
                        Dbb = Dj;
                        bb = j;
                    }
                }
                b = bb < 0 ? 0 : bb;
                ub = f32_up(sqrt(Dbb) * (1.0 + 0x1p-40));
            }
            if (part == 0) {
                if (b != inc) {
                    P.a[i] = b;
                    my_changed += 1;
                }
                P.u[i] = ub;
                my_comp += (uint64_t)k;
                my_rc += re ? 1 : 0;
            }
        }
    }
    my_changed = wave_sum_u64(my_changed);
    my_comp = wave_sum_u64(my_comp);
    my_rc = wave_sum_u64(my_rc);
    if (lane == 0) {
        unsigned long long* sc =
            reinterpret_cast<unsigned long long*>(P.total + (int64_t)k * d + k);
        if (my_changed) atomicAdd(&sc[kStChanged], (unsigned long long)my_changed);
        if (my_comp) atomicAdd(&sc[kStComputed], (unsigned long long)my_comp);
        if (my_rc) atomicAdd(&sc[kStRecheck], (unsigned long long)my_rc);
    }
}

// ---------------------------------------------------------------------------
// Counting sort of the points by their new cluster.

__global__ __launch_bounds__(256) void k_hist_large(Dev P, Large Lg) {
    if (!P.st->active) return;
    extern __shared__ __align__(16) unsigned char smem[];
    uint32_t* h = reinterpret_cast<uint32_t*>(smem);
    const int k = P.k;
    if (blockIdx.x == 0 && threadIdx.x == 0) *Lg.nsurv = 0;   // for the next step
    for (int j = threadIdx.x; j < k; j += blockDim.x) h[j] = 0;
    __syncthreads();
    const int64_t lo = (int64_t)blockIdx.x * Lg.span;
    const int64_t hi = min(P.n, lo + Lg.span);
    for (int64_t i = lo + threadIdx.x; i < hi; i += blockDim.x) atomicAdd(&h[P.a[i]], 1u);
    __syncthreads();
    for (int j = threadIdx.x; j < k; j += blockDim.x) Lg.cnt[(int64_t)blockIdx.x * k + j] = h[j];
}

// Per cluster j: exclusive prefix of the block counts (write offsets
// relative to the cluster start) and the cluster size into base[j].
__global__ __launch_bounds__(256) void k_scan_large_cols(Dev P, Large Lg) {
    if (!P.st->active) return;
    const int j = blockIdx.x * blockDim.x + threadIdx.x;
    if (j >= P.k) return;
    uint32_t run = 0;
    for (int g = 0; g < Lg.Gs; ++g) {
        const int64_t o = (int64_t)g * P.k + j;
        const uint32_t c = Lg.cnt[o];
        Lg.off[o] = run;
        run += c;
    }
    Lg.base[j] = run;
}

// One block: cluster starts (exclusive scan of the sizes) and the first
// segment chunk of every cluster.  base[k] = n, cbase[k] = chunk count.
__global__ __launch_bounds__(1024) void k_scan_large_clusters(Dev P, Large Lg) {
    if (!P.st->active) return;
    const int k = P.k, t = threadIdx.x, T = blockDim.x;
    __shared__ uint32_t ps[1024], pc[1024];
    const int per = (k + T - 1) / T, j0 = t * per, j1 = min(k, j0 + per);
    uint32_t s = 0, sc = 0;
    for (int j = j0; j < j1; ++j) {
        const uint32_t sz = Lg.base[j];
        s += sz;
        sc += (sz + kLgChunkRows - 1) / kLgChunkRows;
    }
    ps[t] = s;
    pc[t] = sc;
    __syncthreads();
    for (int w = 1; w < T; w <<= 1) {   // inclusive Hillis-Steele scan
        const uint32_t a = t >= w ? ps[t - w] : 0, b = t >= w ? pc[t - w] : 0;
        __syncthreads();
        ps[t] += a;
        pc[t] += b;
        __syncthreads();
    }
    uint32_t run = ps[t] - s, crun = pc[t] - sc;
    for (int j = j0; j < j1; ++j) {
        const uint32_t sz = Lg.base[j];
        Lg.base[j] = run;
        Lg.cbase[j] = crun;
        run += sz;
        crun += (sz + kLgChunkRows - 1) / kLgChunkRows;
    }
    if (t == T - 1) {
        Lg.base[k] = ps[T - 1];
        Lg.cbase[k] = pc[T - 1];
    }
}

__global__ __launch_bounds__(256) void k_scatter_large(Dev P, Large Lg) {
    if (!P.st->active) return;
    extern __shared__ __align__(16) unsigned char smem[];
    uint32_t* pos = reinterpret_cast<uint32_t*>(smem);
    const int k = P.k;
    for (int j = threadIdx.x; j < k; j += blockDim.x)
        pos[j] = Lg.base[j] + Lg.off[(int64_t)blockIdx.x * k + j];
    __syncthreads();
    const int64_t lo = (int64_t)blockIdx.x * Lg.span;
    const int64_t hi = min(P.n, lo + Lg.span);
    for (int64_t i = lo + threadIdx.x; i < hi; i += blockDim.x)
        Lg.perm[atomicAdd(&pos[P.a[i]], 1u)] = (int32_t)i;
}

// One block per chunk of <= kLgChunkRows points of one cluster: exact
// fixed-point coordinate sums (and, with KM_FLAG_STATS, the squared
// distances to the cluster's current centroid, element by element).
__global__ __launch_bounds__(256) void k_segsum_large(Dev P, Large Lg) {
    if (!P.st->active) return;
    const int c = blockIdx.x;
    const int k = P.k, d = P.d;
    if (c >= (int)Lg.cbase[k]) return;
    int lo = 0, hi = k;   // cluster j with cbase[j] <= c < cbase[j + 1]
    while (hi - lo > 1) {
        const int mid = (lo + hi) >> 1;
        if ((int)Lg.cbase[mid] <= c) lo = mid;
        else hi = mid;
    }
    const int j = lo;
    const uint32_t r0 = Lg.base[j] + (uint32_t)(c - (int)Lg.cbase[j]) * kLgChunkRows;
    const uint32_t r1 = min(Lg.base[j + 1], r0 + kLgChunkRows);
    const bool want_inertia = (P.flags & KM_FLAG_STATS) != 0;
    uint64_t iq = 0;
    for (int m = threadIdx.x; m < d; m += blockDim.x) {
        const float cj = P.C32[(int64_t)j * d + m];
        uint64_t acc = 0;
        for (uint32_t r = r0; r < r1; ++r) {
            const float x = P.X[(int64_t)Lg.perm[r] * d + m];
            acc += fixed_bits((double)x, P.qscale);
            if (want_inertia) {
                const float t = x - cj;
                iq += fixed_bits((double)(t * t), P.iscale) - kMagicBits;
            }
        }
        Lg.cpart[(int64_t)c * d + m] = acc;
    }
    if (want_inertia) {
        __shared__ uint64_t rs[4];
        iq = wave_sum_u64(iq);
        if ((threadIdx.x & 63) == 0) rs[threadIdx.x >> 6] = iq;
        __syncthreads();
        if (threadIdx.x == 0) Lg.ciq[c] = rs[0] + rs[1] + rs[2] + rs[3];
    }
}

// Per-cluster sums (over the cluster's chunks) and counts into the reduced
// row; block 0 also adds the inertia partials.
__global__ __launch_bounds__(256) void k_chunk_reduce_large(Dev P, Large Lg) {
    if (!P.st->active) return;
    const int k = P.k, d = P.d;
    const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (e < (int64_t)k * d) {
        const int j = (int)(e / d), m = (int)(e - (int64_t)j * d);
        uint64_t acc = 0;
        for (uint32_t cc = Lg.cbase[j]; cc < Lg.cbase[j + 1]; ++cc) acc += Lg.cpart[(int64_t)cc * d + m];
        P.total[e] = acc;
        if (m == 0) P.total[(int64_t)k * d + j] = Lg.base[j + 1] - Lg.base[j];
    }
    if (blockIdx.x == 0 && (P.flags & KM_FLAG_STATS)) {
        __shared__ uint64_t rs[4];
        uint64_t s = 0;
        const uint32_t nc = Lg.cbase[k];
        for (uint32_t cc = threadIdx.x; cc < nc; cc += blockDim.x) s += Lg.ciq[cc];
        s = wave_sum_u64(s);
        if ((threadIdx.x & 63) == 0) rs[threadIdx.x >> 6] = s;
        __syncthreads();
        if (threadIdx.x == 0) P.total[(int64_t)k * d + k + kStInertia] = rs[0] + rs[1] + rs[2] + rs[3];
    }
}

// ---------------------------------------------------------------------------
// Centroid table for large k*d: a block stages kTiTile float64 rows in LDS
// and streams every centroid once against them.

__global__ __launch_bounds__(256) void k_centroid_table_tiled(Dev P, int force) {
    if (!force && !P.st->active) return;
    const int k = P.k, d = P.d;
    const int i0 = blockIdx.x * kTiTile, ni = min(kTiTile, k - i0);
    extern __shared__ __align__(16) unsigned char smem[];
    double* ci = reinterpret_cast<double*>(smem);                  // [kTiTile][d]
    float* mins = reinterpret_cast<float*>(ci + kTiTile * d);      // [kTiTile][256]
    for (int e = threadIdx.x; e < kTiTile * d; e += blockDim.x) {
        const int r = e / d;
        ci[e] = r < ni ? P.C64[(int64_t)(i0 + r) * d + (e - r * d)] : 0.0;
    }
    __syncthreads();
    float mn[kTiTile];
#pragma unroll
    for (int r = 0; r < kTiTile; ++r) mn[r] = INFINITY;
    for (int j = threadIdx.x; j < k; j += blockDim.x) {
        const double* cj = P.C64 + (int64_t)j * d;
        double acc[kTiTile];
#pragma unroll
        for (int r = 0; r < kTiTile; ++r) acc[r] = 0.0;
        for (int m = 0; m < d; ++m) {
            const double v = cj[m];
#pragma unroll
            for (int r = 0; r < kTiTile; ++r) {
                const double t = ci[r * d + m] - v;
                acc[r] = fma(t, t, acc[r]);
            }
        }
#pragma unroll
        for (int r = 0; r < kTiTile; ++r) {
            if (r >= ni) continue;
            const int i = i0 + r;
            float hv = 0.f;
            if (j != i) {
                hv = f32_down(0.5 * sqrt(acc[r]) * (1.0 - 0x1p-40));
                mn[r] = fminf(mn[r], hv);
            }
            P.h[(int64_t)i * k + j] = hv;
        }
    }
#pragma unroll
    for (int r = 0; r < kTiTile; ++r) mins[r * 256 + threadIdx.x] = mn[r];
    __syncthreads();
    if (threadIdx.x < ni) {
        const int r = threadIdx.x, i = i0 + r;
        float m = INFINITY;
        for (int q = 0; q < (int)blockDim.x; ++q) m = fminf(m, mins[r * 256 + q]);
        P.s[i] = m;
        const float* c32 = P.C32 + (int64_t)i * d;
        double n2 = 0.0;
        for (int q = 0; q < d; ++q) n2 = fma((double)c32[q], (double)c32[q], n2);
        P.cn2[i] = (float)n2;
    }
    if (blockIdx.x == 0) {
        float em = 0.f;
        for (int j = threadIdx.x; j < k; j += blockDim.x) em = fmaxf(em, P.ec[j]);
#pragma unroll
        for (int off = 32; off > 0; off >>= 1) em = fmaxf(em, __shfl_xor(em, off));
        __syncthreads();
        if ((threadIdx.x & 63) == 0) mins[threadIdx.x >> 6] = em;
        __syncthreads();
        if (threadIdx.x == 0)
            P.st->ec_max = fmaxf(fmaxf(mins[0], mins[1]), fmaxf(mins[2], mins[3]));
    }
}

// ---------------------------------------------------------------------------
// Launchers

const void* large_mfma_symbol() { return reinterpret_cast<const void*>(&k_mfma_large); }

hipError_t launch_large_assign(const Dev& dv, const Large& lg, int gb, hipStream_t s) {
    hipLaunchKernelGGL(k_bound_large, dim3(gb), dim3(256), 0, s, dv, lg);
    hipLaunchKernelGGL(k_mfma_large, dim3(lg.Gm), dim3(256), large_mfma_lds(lg.dp), s, dv, lg);
    return hipGetLastError();
}

hipError_t launch_large_reduce(const Dev& dv, const Large& lg, hipStream_t s) {
    const int hl = 4 * dv.k;
    hipLaunchKernelGGL(k_hist_large, dim3(lg.Gs), dim3(256), hl, s, dv, lg);
    hipLaunchKernelGGL(k_scan_large_cols, dim3((dv.k + 255) / 256), dim3(256), 0, s, dv, lg);
    hipLaunchKernelGGL(k_scan_large_clusters, dim3(1), dim3(1024), 0, s, dv, lg);
    hipLaunchKernelGGL(k_scatter_large, dim3(lg.Gs), dim3(256), hl, s, dv, lg);
    hipLaunchKernelGGL(k_segsum_large, dim3(lg.NCmax), dim3(256), 0, s, dv, lg);
    const int64_t kd = (int64_t)dv.k * dv.d;
    hipLaunchKernelGGL(k_chunk_reduce_large, dim3((unsigned)((kd + 255) / 256)), dim3(256), 0, s, dv, lg);
    return hipGetLastError();
}

int large_table_lds(int d) { return 8 * kTiTile * d + 4 * kTiTile * 256; }

hipError_t large_set_attributes(int k, int d, int dp) {
    hipError_t e;
    const auto attr = hipFuncAttributeMaxDynamicSharedMemorySize;
    if ((e = hipFuncSetAttribute(reinterpret_cast<const void*>(&k_mfma_large), attr,
                                 large_mfma_lds(dp))) != hipSuccess)
        return e;
    if ((e = hipFuncSetAttribute(reinterpret_cast<const void*>(&k_hist_large), attr, 4 * k)) != hipSuccess)
        return e;
    if ((e = hipFuncSetAttribute(reinterpret_cast<const void*>(&k_scatter_large), attr, 4 * k)) != hipSuccess)
        return e;
    return hipFuncSetAttribute(reinterpret_cast<const void*>(&k_centroid_table_tiled), attr,
                               large_table_lds(d));
}

hipError_t launch_large_table(const Dev& dv, int force, hipStream_t s) {
    hipLaunchKernelGGL(k_centroid_table_tiled, dim3((dv.k + kTiTile - 1) / kTiTile), dim3(256),
                       large_table_lds(dv.d), s, dv, force);
    return hipGetLastError();
}

}  // namespace km
