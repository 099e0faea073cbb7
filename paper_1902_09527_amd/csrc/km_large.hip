// Global-memory path of the MTI k-means hot path for gfx950 (MI355X), used
// when the centroids or the per-cluster sums do not fit in LDS (large k*d,
// e.g. k = 1000, d = 256).  One iteration (one ||Lloyd's MM step, paper
// section III-B) is:
//   k_bound_large       drift-updated bound and Clause 1 (section III-C) for
//                       every point; survivors compacted into a global list;
//   k_mfma_large        float32 MFMA distances of the survivors to all
//                       centroids (128-centroid x 128-survivor tiles over
//                       double-buffered 16-dimension chunks, expanded form), a
//                       top-4 candidate list per survivor, direct-form
//                       refinement of the candidates within the expanded
//                       form's error bound, float64 near-tie rule;
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

// The same insertion when j is larger than every index in the list (the
// centroids arrive in increasing index order): a tie keeps the earlier,
// lower index, so only strict comparisons are needed.
__device__ __forceinline__ void top4_insert_next(float (&L)[4], int (&J)[4], float v, int j) {
    if (!(v < L[3])) return;
    L[3] = v;
    J[3] = j;
#pragma unroll
    for (int q = 3; q > 0; --q) {
        if (L[q] < L[q - 1]) {
            const float tv = L[q];
            L[q] = L[q - 1];
            L[q - 1] = tv;
            const int tj = J[q];
            J[q] = J[q - 1];
            J[q - 1] = tj;
        }
    }
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

// Refinement of survivor c of a tile (entry s0 + c of the survivor list) by
// a thread pair (part 0 and 1, each over half of the dimensions) from the
// survivor's 16 candidate slots (candD, candJ: 4 lists of 4) and its squared
// norm x2: the candidates within twice the expanded form's error bound of the
// smallest are re-evaluated in the direct form, followed by the float64
// near-tie rule; the point's assignment and bound are written.
template <bool VEC>
__device__ __forceinline__ void refine_survivor(const Dev& P, const Large& Lg, const float* candD, const int* candJ,
                                                int s0, int c, int part, bool first, float x2, float cnmax,
                                                float gexp, float ecm, float gamma, uint64_t& my_changed,
                                                uint64_t& my_comp, uint64_t& my_rc) {
    const int k = P.k, d = P.d;
    constexpr bool vec = VEC;
    float T[4];
    int TJ[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        T[q] = INFINITY;
        TJ[q] = INT_MAX;
    }
    for (int q = 0; q < 16; ++q) top4_insert(T, TJ, candD[c * 16 + q], candJ[c * 16 + q]);
    const int64_t i = Lg.surv[s0 + c];
    const float* xr = P.X + i * d;
    const int inc = first ? -1 : P.a[i];
    const int hd = (d + 1) / 2, m0 = part * hd, m1 = min(d, m0 + hd);
    const float R = sqrtf(fmaxf(x2, 0.f)) * kUp + cnmax;
    const float thr = T[0] + 2.f * (gexp * R * R + 4.f * R * ecm + 2.f * ecm * ecm);
    // Only centroids whose expanded distance lies within thr of the
    // smallest can be the nearest: any other one is certified
    // farther than the smallest's centroid.  A fourth candidate
    // inside the bound means more may lie outside the list: all
    // centroids are decided in float64 then.
    const bool full = T[3] <= thr;
    int nq = 0;
    while (nq < 3 && T[nq] <= thr && TJ[nq] < k) ++nq;   // uniform in the pair
    // Direct-form distance of x to centroid j over this thread's half
    // of the dimensions, both halves added (equal in the pair).
    auto dist32 = [&](int j) {
        const float* cr = P.C32 + (int64_t)j * d;
        float accd = 0.f;
        if (vec && (m0 & 3) == 0) {
            int m = m0;
            for (; m + 4 <= m1; m += 4) {
                const f32x4 xv = *reinterpret_cast<const f32x4*>(xr + m);
                const f32x4 cv = *reinterpret_cast<const f32x4*>(cr + m);
                const float t0 = xv.x - cv.x, t1 = xv.y - cv.y, t2 = xv.z - cv.z, t3 = xv.w - cv.w;
                accd = fmaf(t0, t0, accd);
                accd = fmaf(t1, t1, accd);
                accd = fmaf(t2, t2, accd);
                accd = fmaf(t3, t3, accd);
            }
            for (; m < m1; ++m) {
                const float t = xr[m] - cr[m];
                accd = fmaf(t, t, accd);
            }
        } else {
            for (int m = m0; m < m1; ++m) {
                const float t = xr[m] - cr[m];
                accd = fmaf(t, t, accd);
            }
        }
        return accd + __shfl_xor(accd, 1);
    };
    auto dist64 = [&](int j) {
        const double* cr = P.C64 + (int64_t)j * d;
        double accd = 0.0;
        for (int m = m0; m < m1; ++m) {
            const double t = (double)xr[m] - cr[m];
            accd = fma(t, t, accd);
        }
        return accd + __shfl_xor(accd, 1);
    };
    bool re = full;
    float d1 = INFINITY, d2 = INFINITY;
    int rk1 = INT_MAX, j1 = 0;
    // One candidate is the nearest centroid (every other one is
    // certified farther): as on the LDS paths, its bound then comes
    // from its expanded value and the error bound, without the
    // direct form (kept when statistics are gathered).
    const bool single = !full && nq == 1 && !(P.flags & KM_FLAG_STATS);
    if (!full && !single) {
        for (int q = 0; q < nq; ++q) {
            const int j = TJ[q];
            const float Dd = dist32(j);
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
    float ub;
    if (single) {
        const float e1b = gexp * R * R + 4.f * R * ecm + 2.f * ecm * ecm;
        b = TJ[0];
        ub = __builtin_amdgcn_sqrtf(fmaxf(T[0] + e1b, 0.f)) * (1.0f + 0x1p-20f) * kUp;
    } else {
        ub = upper_bound(d1, P.ec[j1], gamma);
    }
    if (re) {
        // float64 decision against the master centroids with the
        // oracle's rule (smaller distance, then the incumbent, then
        // the lower index): among the candidates inside the bound, or
        // among all centroids when the list may be incomplete.
        double Dbb = INFINITY;
        int bb = -1, kb = INT_MAX;
        auto consider = [&](int j) {
            const double Dj = dist64(j);
            const int rk = j == inc ? -1 : j;
            if (Dj < Dbb || (Dj == Dbb && rk < kb)) {
                Dbb = Dj;
                bb = j;
                kb = rk;
            }
        };
        if (full) {
            for (int j = 0; j < k; ++j) consider(j);
        } else {
            for (int q = 0; q < nq; ++q) consider(TJ[q]);
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

// ---------------------------------------------------------------------------
// Dense survivor distances on the matrix cores, as a tiled product of the
// centroids (rows) and the survivors (columns) over the dimensions.  Block
// tile: kLgN = 128 centroids x kLgM = 128 survivors; wave (wr, wc) owns
// centroid rows 64 wr .. 64 wr + 63 and survivor columns 64 wc .. 64 wc + 63,
// four 32x32 float32 accumulators.  The dimensions stream in chunks
// of kLgK through double-buffered LDS (row-major, 16-byte rows: one 16-byte
// store per thread and row piece, two 16-byte reads per lane and operand);
// the next chunk's global loads are issued before the current chunk's
// products.  Within a chunk, product step s sums dimensions s (lanes 0-31)
// and 8 + s (lanes 32-63), so each lane's operands for the whole chunk are 8
// consecutive floats of one row.  Each lane
// keeps, for its two survivor columns, the four smallest expanded-form
// distances |x|^2 + |c|^2 - 2 x.c with their centroids; the 4 lists of a
// survivor (2 waves x 2 half-waves) are merged in LDS, and the candidates
// within the expanded form's error bound of the smallest are re-evaluated in
// the direct form, followed by the float64 near-tie rule.

template <bool VEC>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(2))) void k_mfma_large(Dev P, Large Lg) {
    IterState* st = P.st;
    if (!st->active) return;
    const int k = P.k, d = P.d;
    const bool first = st->t == 0;
    const uint32_t ns = *Lg.nsurv;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, col = lane & 31, half = lane >> 5;
    const int wr = wave >> 1, wc = wave & 1;   // the wave's 64-centroid row block and 64-survivor column block
    extern __shared__ __align__(16) unsigned char smem[];
    constexpr int kBufBytes = 2 * (kLgN + kLgM) * kLgRS * 4;
    constexpr int kCandBytes = kLgM * 16 * 8;
    float* Ab = reinterpret_cast<float*>(smem);                    // [2][kLgN][kLgRS]
    float* Bb = Ab + 2 * kLgN * kLgRS;                             // [2][kLgM][kLgRS]
    float* candD = reinterpret_cast<float*>(smem);                 // [kLgM][16], after the products
    int* candJ = reinterpret_cast<int*>(candD + kLgM * 16);
    float* x2s = reinterpret_cast<float*>(smem + (kBufBytes > kCandBytes ? kBufBytes : kCandBytes));   // [kLgM]
    float* red = x2s + kLgM;                                       // [4]
    float* cnt = red + 4;                                          // [kLgN]: the centroid tile's |c|^2

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
    const int ntiles = (int)((ns + kLgM - 1) / kLgM);
    const int nct = (k + kLgN - 1) / kLgN;
    const int nch = (d + kLgK - 1) / kLgK;
    constexpr bool vec = VEC;   // d % 4 == 0: 16-byte row chunks (every chunk start is then aligned)
    const f32x4* C4 = reinterpret_cast<const f32x4*>(P.C32);
    const f32x4* X4 = reinterpret_cast<const f32x4*>(P.X);

    // Chunk loads, two 4-float pieces per thread for each operand: centroid
    // row n0 + 64i + tid / 4 and survivor 64i + tid / 4, dimensions
    // 4 (tid % 4) .. +3 of the chunk; zero outside k, the survivors and d.
    f32x4 ra[2], rb[2];
    float x2p[2] = {0.f, 0.f};   // partial squared norms of this thread's two survivors (first centroid tile)
    int srow[2];                 // this thread's two survivors' point indices (-1: none)
    const int q4 = tid & 3, r4 = tid >> 2;
    auto load_chunk = [&](int n0, int c) __attribute__((always_inline)) {
        const int m0 = c * kLgK + 4 * q4;
#pragma unroll
        for (int i = 0; i < 2; ++i) {
            const int j = n0 + 64 * i + r4;
            f32x4 v = {0.f, 0.f, 0.f, 0.f};
            if (j < k) {
                if (vec) {
                    if (m0 < d) v = C4[((int64_t)j * d + m0) >> 2];
                } else {
#pragma unroll
                    for (int e = 0; e < 4; ++e)
                        if (m0 + e < d) v[e] = P.C32[(int64_t)j * d + m0 + e];
                }
            }
            ra[i] = v;
        }
#pragma unroll
        for (int i = 0; i < 2; ++i) {
            f32x4 v = {0.f, 0.f, 0.f, 0.f};
            if (srow[i] >= 0) {
                if (vec) {
                    if (m0 < d) v = X4[((int64_t)srow[i] * d + m0) >> 2];   // cached: re-read per centroid tile
                } else {
#pragma unroll
                    for (int e = 0; e < 4; ++e)
                        if (m0 + e < d) v[e] = P.X[(int64_t)srow[i] * d + m0 + e];
                }
            }
            rb[i] = v;
        }
    };
    auto store_chunk = [&](int buf) __attribute__((always_inline)) {
        float* A = Ab + buf * kLgN * kLgRS;
        float* B = Bb + buf * kLgM * kLgRS;
#pragma unroll
        for (int i = 0; i < 2; ++i) *reinterpret_cast<f32x4*>(A + (64 * i + r4) * kLgRS + 4 * q4) = ra[i];
#pragma unroll
        for (int i = 0; i < 2; ++i) *reinterpret_cast<f32x4*>(B + (64 * i + r4) * kLgRS + 4 * q4) = rb[i];
    };

    for (int tile = blockIdx.x; tile < ntiles; tile += gridDim.x) {
        const int s0 = tile * kLgM;
        const int rows = min(kLgM, (int)ns - s0);
#pragma unroll
        for (int i = 0; i < 2; ++i) {
            const int sl = 64 * i + r4;
            srow[i] = sl < rows ? Lg.surv[s0 + sl] : -1;
            x2p[i] = 0.f;
        }
        float L[2][4];
        int J[2][4];
#pragma unroll
        for (int cb = 0; cb < 2; ++cb)
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                L[cb][q] = INFINITY;
                J[cb][q] = INT_MAX;
            }
        for (int ct = 0; ct < nct; ++ct) {
            const int n0 = ct * kLgN;
            f32x16 acc[2][2];
#pragma unroll
            for (int a = 0; a < 2; ++a)
#pragma unroll
                for (int b = 0; b < 2; ++b)
#pragma unroll
                    for (int e = 0; e < 16; ++e) acc[a][b][e] = 0.f;
            __syncthreads();   // the previous tile's buffers and lists are consumed
            load_chunk(n0, 0);
            if (tid < kLgN) cnt[tid] = n0 + tid < k ? P.cn2[n0 + tid] : INFINITY;
            store_chunk(0);
            if (ct == 0)
#pragma unroll
                for (int i = 0; i < 2; ++i) x2p[i] += rb[i].x * rb[i].x + rb[i].y * rb[i].y + rb[i].z * rb[i].z + rb[i].w * rb[i].w;
            __syncthreads();
            for (int c = 0; c < nch; ++c) {
                const bool more = c + 1 < nch;
                if (more) load_chunk(n0, c + 1);
                // Lane (col, half): rows 64 wr + col (+ 32) of the centroid
                // chunk and 64 wc + col (+ 32) of the survivor chunk,
                // dimensions 8 half .. 8 half + 7.
                const float* A = Ab + (c & 1) * kLgN * kLgRS + (64 * wr + col) * kLgRS + 8 * half;
                const float* B = Bb + (c & 1) * kLgM * kLgRS + (64 * wc + col) * kLgRS + 8 * half;
                float a0[8], a1[8], b0[8], b1[8];
#pragma unroll
                for (int h = 0; h < 2; ++h) {
                    const f32x4 va0 = *reinterpret_cast<const f32x4*>(A + 4 * h);
                    const f32x4 va1 = *reinterpret_cast<const f32x4*>(A + 32 * kLgRS + 4 * h);
                    const f32x4 vb0 = *reinterpret_cast<const f32x4*>(B + 4 * h);
                    const f32x4 vb1 = *reinterpret_cast<const f32x4*>(B + 32 * kLgRS + 4 * h);
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        a0[4 * h + e] = va0[e];
                        a1[4 * h + e] = va1[e];
                        b0[4 * h + e] = vb0[e];
                        b1[4 * h + e] = vb1[e];
                    }
                }
#pragma unroll
                for (int s = 0; s < kLgK / 2; ++s) {
                    acc[0][0] = __builtin_amdgcn_mfma_f32_32x32x2f32(a0[s], b0[s], acc[0][0], 0, 0, 0);
                    acc[0][1] = __builtin_amdgcn_mfma_f32_32x32x2f32(a0[s], b1[s], acc[0][1], 0, 0, 0);
                    acc[1][0] = __builtin_amdgcn_mfma_f32_32x32x2f32(a1[s], b0[s], acc[1][0], 0, 0, 0);
                    acc[1][1] = __builtin_amdgcn_mfma_f32_32x32x2f32(a1[s], b1[s], acc[1][1], 0, 0, 0);
                }
                if (more) {
                    store_chunk((c + 1) & 1);
                    if (ct == 0)
#pragma unroll
                        for (int i = 0; i < 2; ++i)
                            x2p[i] += rb[i].x * rb[i].x + rb[i].y * rb[i].y + rb[i].z * rb[i].z + rb[i].w * rb[i].w;
                }
                __syncthreads();
            }
            if (ct == 0) {   // squared norms of the survivors: the 4 lanes of each row
#pragma unroll
                for (int i = 0; i < 2; ++i) {
                    float v = x2p[i];
                    v += __shfl_xor(v, 1);
                    v += __shfl_xor(v, 2);
                    if (q4 == 0) x2s[64 * i + r4] = v;
                }
                __syncthreads();
            }
            // Register e of accumulator [a][cb]: centroid n0 + 64 wr + 32 a + 8 (e / 4) + 4 half + e % 4,
            // survivor column 64 wc + 32 cb + col.
#pragma unroll
            for (int cb = 0; cb < 2; ++cb) {
                const float xa = x2s[64 * wc + 32 * cb + col];
#pragma unroll
                for (int a = 0; a < 2; ++a)
#pragma unroll
                    for (int g = 0; g < 4; ++g) {
                        const int jl = 64 * wr + 32 * a + 8 * g + 4 * half;   // 4 consecutive centroids
                        const f32x4 cn = *reinterpret_cast<const f32x4*>(cnt + jl);
#pragma unroll
                        for (int e = 0; e < 4; ++e)
                            top4_insert_next(L[cb], J[cb], xa + cn[e] - 2.f * acc[a][cb][4 * g + e], n0 + jl + e);
                    }
            }
        }
        // Merge the 4 lists of each survivor (2 waves x 2 half-waves).
        __syncthreads();   // the chunk buffers are no longer read
#pragma unroll
        for (int cb = 0; cb < 2; ++cb)
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const int slot = (wr * 2 + half) * 4 + q;
                candD[(64 * wc + 32 * cb + col) * 16 + slot] = L[cb][q];
                candJ[(64 * wc + 32 * cb + col) * 16 + slot] = J[cb][q];
            }
        __syncthreads();

        // Refinement: 2 threads per survivor, each half of the dimensions.
        const int c = tid >> 1, part = tid & 1;
        if (c < rows)
            refine_survivor<VEC>(P, Lg, candD, candJ, s0, c, part, first, x2s[c], cnmax, gexp, ecm, gamma,
                                 my_changed, my_comp, my_rc);
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
__global__ __launch_bounds__(256) void k_segsum_large(Dev P_, Large Lg) {
    const Dev P = with_scales(P_);
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

const void* large_mfma_symbol(int d) {
    return (d & 3) == 0 ? reinterpret_cast<const void*>(&k_mfma_large<true>)
                        : reinterpret_cast<const void*>(&k_mfma_large<false>);
}

hipError_t launch_large_assign(const Dev& dv, const Large& lg, int gb, hipStream_t s) {
    hipLaunchKernelGGL(k_bound_large, dim3(gb), dim3(256), 0, s, dv, lg);
    if ((dv.d & 3) == 0)
        hipLaunchKernelGGL(k_mfma_large<true>, dim3(lg.Gm), dim3(256), large_mfma_lds(), s, dv, lg);
    else
        hipLaunchKernelGGL(k_mfma_large<false>, dim3(lg.Gm), dim3(256), large_mfma_lds(), s, dv, lg);
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

hipError_t large_set_attributes(int k, int d) {
    hipError_t e;
    const auto attr = hipFuncAttributeMaxDynamicSharedMemorySize;
    if ((e = hipFuncSetAttribute(large_mfma_symbol(d), attr, large_mfma_lds())) != hipSuccess) return e;
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
