// HIP kernels of the MTI k-means hot path for gfx950 (MI355X).
//
// One iteration (one merged ||Lloyd's MM step, paper section III-B) is four
// stream-ordered launches, none of which needs the host:
//   k_assign          Clause-1 test on the drift-updated bound, fused float32
//                     distance + argmin for the surviving points with the
//                     per-centroid Clause 2/3 skips, and the per-block
//                     fixed-point partial sums/counts of ALL points
//                     (section III-C; section V "per-thread local centroids");
//   k_reduce          sums the per-block partial rows (integer, exact);
//   k_update          new centroids (member means, empty clusters kept; for
//                     spherical k-means projected to the unit sphere),
//                     drift f(c) (Table I), loop counters and the stop test;
//   k_centroid_table  half centroid-to-centroid distances h and
//                     s(c) = min_{c' != c} h(c, c') for the next step.
// Every kernel first reads the device loop state and returns at once when
// the run has stopped, so a whole run can be enqueued up front.
#include <float.h>
#include <limits.h>
#include <math.h>

#include "kmeans_mti.h"
#include "km_device.h"
#include "km_internal.h"

namespace km {

// Dynamic LDS of the assignment kernels.  Declared once at namespace scope so
// that device functions index it directly and every access stays an LDS
// (ds_*) instruction.
extern __shared__ __align__(16) unsigned char km_smem[];

namespace {

template <int D>
struct Row {
    float v[D > 0 ? D : 1];
};

// Squared float32 distance of a register row to an LDS centroid row.
template <int D>
__device__ inline float sqd_reg(const Row<D>& x, const float* c) {
    float acc = 0.f;
#pragma unroll
    for (int m = 0; m < D; m += 4) {
        const float4 cv = *reinterpret_cast<const float4*>(c + m);
        float t0 = x.v[m] - cv.x, t1 = x.v[m + 1] - cv.y, t2 = x.v[m + 2] - cv.z, t3 = x.v[m + 3] - cv.w;
        acc = fmaf(t0, t0, acc);
        acc = fmaf(t1, t1, acc);
        acc = fmaf(t2, t2, acc);
        acc = fmaf(t3, t3, acc);
    }
    return acc;
}

// Generic-d form: both rows in LDS.
__device__ inline float sqd_lds(const float* x, const float* c, int d) {
    float acc = 0.f;
    for (int m = 0; m < d; ++m) {
        float t = x[m] - c[m];
        acc = fmaf(t, t, acc);
    }
    return acc;
}

}  // namespace

// ---------------------------------------------------------------------------
// Init helpers

// Largest |value| (as float bits: non-negative floats order as their bits;
// NaN ignored, an infinite value counted as the largest float) and whether
// any value is not finite.
__device__ __forceinline__ void absmax_take(float v, uint32_t& m, uint32_t& bad) {
    const uint32_t u = __float_as_uint(v) & 0x7fffffffu;
    bad |= u >= 0x7f800000u ? 1u : 0u;
    const uint32_t c = u > 0x7f800000u ? 0u : (u < 0x7f7fffffu ? u : 0x7f7fffffu);
    m = c > m ? c : m;
}

// absmax_take over one array: 16-byte loads when it is 16-byte aligned,
// kAbsLoads in flight per lane, then the scalar tail.
constexpr int kAbsLoads = 8;
constexpr int kAbsBlocksPerCU = 1;
constexpr int kAbsSampleChunks = 16;
__device__ __forceinline__ void absmax_range(const float* __restrict__ p, int64_t count, int64_t t0,
                                             int64_t stride, uint32_t& m, uint32_t& bad) {
    auto take = [&](float v) __attribute__((always_inline)) { absmax_take(v, m, bad); };
    const int64_t nq = (reinterpret_cast<uintptr_t>(p) & 15) == 0 ? count / 4 : 0;
    const f32x4* __restrict__ q = reinterpret_cast<const f32x4*>(p);
    int64_t i = t0;
    for (; i + (kAbsLoads - 1) * stride < nq; i += kAbsLoads * stride) {
        f32x4 v[kAbsLoads];
#pragma unroll
        for (int r = 0; r < kAbsLoads; ++r) v[r] = __builtin_nontemporal_load(q + i + r * stride);
#pragma unroll
        for (int r = 0; r < kAbsLoads; ++r) {
            take(v[r].x);
            take(v[r].y);
            take(v[r].z);
            take(v[r].w);
        }
    }
    for (; i < nq; i += stride) {
        const f32x4 v = __builtin_nontemporal_load(q + i);
        take(v.x);
        take(v.y);
        take(v.z);
        take(v.w);
    }
    for (int64_t j = 4 * nq + t0; j < count; j += stride) take(p[j]);
}

// Three roles in one launch: blocks [0, blocks_a) scan a (out[kAmaxX],
// out[kAmaxXBad]), the next blocks_b scan b (out[kAmaxC], out[kAmaxCBad]),
// and the last blocks one chunk each of the sample of x: rows
// [c n / C, c n / C + max(1, 1024 / d)) of chunk c < C = kAbsSampleChunks,
// cut at n (out[kAmaxSample]).  whole: the sample holds every row (n <= C
// times the rows per chunk) and a is x: no sample blocks, the scan of a
// writes both words.  All words zero before the launch.
__global__ __launch_bounds__(256) void k_absmax(const float* __restrict__ a, int64_t na, const float* __restrict__ b,
                                               int64_t nb, int blocks_a, int blocks_b, const float* __restrict__ x,
                                               int64_t n, int32_t d, int whole, uint32_t* out) {
    const int bi = (int)blockIdx.x;
    const int role = bi < blocks_a ? 0 : (bi < blocks_a + blocks_b ? 1 : 2);
    uint32_t m = 0, bad = 0;
    if (role < 2) {
        const int blk = role == 0 ? bi : bi - blocks_a;
        const int nblk = role == 0 ? blocks_a : blocks_b;
        absmax_range(role == 0 ? a : b, role == 0 ? na : nb, (int64_t)blk * blockDim.x + threadIdx.x,
                     (int64_t)nblk * blockDim.x, m, bad);
    } else {
        const int64_t c = bi - blocks_a - blocks_b;
        const int64_t r0 = c * n / kAbsSampleChunks;
        const int64_t rows = d >= 1024 ? 1 : 1024 / d;
        const int64_t r1 = r0 + rows < n ? r0 + rows : n;
        // four loads per lane in flight, then their values
        for (int64_t j0 = r0 * d; j0 < r1 * d; j0 += 4 * (int64_t)blockDim.x) {
            float v[4];
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const int64_t j = j0 + threadIdx.x + (int64_t)u * blockDim.x;
                v[u] = j < r1 * d ? x[j] : 0.f;
            }
#pragma unroll
            for (int u = 0; u < 4; ++u) absmax_take(v[u], m, bad);
        }
    }
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) {
        const uint32_t o = __shfl_xor(m, off);
        m = o > m ? o : m;
    }
    const bool any_bad = __any(bad);
    if ((threadIdx.x & 63) == 0) {
        atomicMax(out + (role == 0 ? kAmaxX : (role == 1 ? kAmaxC : kAmaxSample)), m);
        if (role == 0 && whole) atomicMax(out + kAmaxSample, m);
        if (any_bad && role < 2) atomicOr(out + (role == 0 ? kAmaxXBad : kAmaxCBad), 1u);
    }
}

// Set-up of a context's device state in one launch: the listed ranges are
// cleared (16-byte stores, then the 4-byte tail; every range starts 16-byte
// aligned and is a whole number of 4-byte words) and the loop state is
// written.
__global__ __launch_bounds__(256) void k_init_buffers(ZeroRanges z) {
    const int64_t t0 = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int r = 0; r < z.n; ++r) {
        uint4* q = reinterpret_cast<uint4*>(z.p[r]);
        const int64_t n16 = (int64_t)(z.bytes[r] / 16);
        for (int64_t i = t0; i < n16; i += stride) q[i] = make_uint4(0u, 0u, 0u, 0u);
        uint32_t* w = reinterpret_cast<uint32_t*>(z.p[r]);
        const int64_t nw = (int64_t)(z.bytes[r] / 4);
        for (int64_t i = 4 * n16 + t0; i < nw; i += stride) w[i] = 0u;
    }
    if (t0 == 0 && z.st) {
        IterState st{};
        st.max_iters = z.max_iters;
        st.tol_n = z.tol_n;
        st.host = z.host;
        *z.st = st;
    }
}

// Fixed-point scales (put_scales) from the set-up magnitude words.  When the
// first step scans X itself, the X word is still zero here: the scales are
// those of the sample's bound, and the end of the first step sets them again
// from the word that step wrote (its sums corrected first when X exceeded
// the bound).
__global__ void k_set_scales(IterState* st, const uint32_t* absmax, int64_t n, int32_t d, int unit) {
    if (threadIdx.x != 0) return;
    put_scales(st, sum_exp(absmax), unit ? 1.0f : __uint_as_float(absmax[kAmaxC]), n, d);
}

__global__ void k_set_centroids(const float* __restrict__ C0, double* C64, float* C32, float* ec,
                                int64_t kd, int32_t k) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i < kd) {
        const float v = C0[i];
        C64[i] = (double)v;
        C32[i] = v;
    }
    if (i < k) ec[i] = 0.f;
}

// Spherical k-means (the paper's sk-means application): row i of X projected
// to the unit sphere, x / |x| with the norm and the quotient in float64
// (a zero row stays zero).
__global__ void k_normalize_rows(const float* __restrict__ X, int64_t n, int32_t d, float* __restrict__ Xn) {
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride) {
        const float* x = X + i * d;
        double s = 0.0;
        for (int m = 0; m < d; ++m) s = fma((double)x[m], (double)x[m], s);
        const double r = sqrt(s);
        float* o = Xn + i * d;
        for (int m = 0; m < d; ++m) o[m] = r > 0.0 ? (float)((double)x[m] / r) : 0.f;
    }
}

// Unit centroids from C0 (one thread per row): float64 master, its float32
// copy and that copy's rounding error; *zero is set for a zero row.
__global__ void k_set_centroids_unit(const float* __restrict__ C0, double* C64, float* C32, float* ec, int32_t k,
                                     int32_t d, int32_t* zero) {
    const int j = blockIdx.x * blockDim.x + threadIdx.x;
    if (j >= k) return;
    const float* c = C0 + (int64_t)j * d;
    double s = 0.0;
    for (int m = 0; m < d; ++m) s = fma((double)c[m], (double)c[m], s);
    if (!(s > 0.0)) {
        atomicOr(zero, 1);
        s = 1.0;
    }
    const double r = sqrt(s);
    double e2 = 0.0;
    for (int m = 0; m < d; ++m) {
        const double v = (double)c[m] / r;
        const float v32 = (float)v;
        C64[(int64_t)j * d + m] = v;
        C32[(int64_t)j * d + m] = v32;
        e2 = fma((double)v32 - v, (double)v32 - v, e2);
    }
    ec[j] = f32_up(sqrt(e2) * (1.0 + 0x1p-40));
}

// ---------------------------------------------------------------------------
// Centroid table: h[i][j] = d(c_i, c_j) / 2 rounded down, s[i] = min_{j != i}
// h[i][j] (paper section III-C, with the factor 1/2 of Elkan's lemma), and
// ec_max for the recheck band.  One block per row i.

__global__ __launch_bounds__(256) void k_centroid_table(Dev P, int force) {
    if (!force && !P.st->active) return;
    const int i = blockIdx.x, k = P.k, d = P.d;
    const double* ci = P.C64 + (int64_t)i * d;
    float mn = INFINITY;
    for (int j = threadIdx.x; j < k; j += blockDim.x) {
        float hv = 0.f;
        if (j != i) {
            const double* cj = P.C64 + (int64_t)j * d;
            double acc = 0.0;
            for (int m = 0; m < d; ++m) {
                double t = ci[m] - cj[m];
                acc = fma(t, t, acc);
            }
            // float64 rounding of the sum and the square root stays far below 2^-40
            hv = f32_down(0.5 * sqrt(acc) * (1.0 - 0x1p-40));
            mn = fminf(mn, hv);
        }
        P.h[(int64_t)i * k + j] = hv;
    }
    if (P.hm) {   // incremental path (k <= 128): min of row i over each 32-centroid block
        __shared__ float hrow[kIMMaxK];
        for (int j = threadIdx.x; j < k; j += blockDim.x) hrow[j] = P.h[(int64_t)i * k + j];
        __syncthreads();
        if ((int)threadIdx.x < 4) {
            const int cb = threadIdx.x, j1 = min(32 * cb + 32, k);
            float m = INFINITY;
            for (int j = 32 * cb; j < j1; ++j) m = fminf(m, hrow[j]);   // h[i][i] = 0
            P.hm[4 * i + cb] = m;
        }
    }
    if (threadIdx.x == 0) {   // ||c32_i||^2 for the expansion form of the matrix-core path
        const float* c = P.C32 + (int64_t)i * d;
        double n2 = 0.0;
        for (int m = 0; m < d; ++m) n2 = fma((double)c[m], (double)c[m], n2);
        P.cn2[i] = (float)n2;
    }
    __shared__ float red[256];
    __shared__ float redm[256];
    red[threadIdx.x] = mn;
    float em = 0.f;
    if (i == 0)
        for (int j = threadIdx.x; j < k; j += blockDim.x) em = fmaxf(em, P.ec[j]);
    redm[threadIdx.x] = em;
    __syncthreads();
    for (int w = blockDim.x / 2; w > 0; w >>= 1) {
        if ((int)threadIdx.x < w) {
            red[threadIdx.x] = fminf(red[threadIdx.x], red[threadIdx.x + w]);
            redm[threadIdx.x] = fmaxf(redm[threadIdx.x], redm[threadIdx.x + w]);
        }
        __syncthreads();
    }
    if (threadIdx.x == 0) {
        P.s[i] = red[0];
        if (i == 0) P.st->ec_max = redm[0];
    }
}

// ---------------------------------------------------------------------------
// Grouped survivor scan (d = 16 or 32, vector units): the survivors of a tile
// are spread over the whole block, L lanes per point, each lane holding D/L of
// the point's coordinates.  Partial distances are combined with xor
// butterflies, which give bitwise equal totals in every lane of a group, so
// all lanes of a group take the same pruning branches; the scan is the same
// MTI scan (incumbent first, then ascending index, running best) as the
// one-lane form.

namespace {

template <int L>
__device__ inline float group_sum(float v) {
#pragma unroll
    for (int o = 1; o < L; o <<= 1) v += __shfl_xor(v, o);
    return v;
}

struct ScanCtx {
    const float* Cs;
    int h_off;          // byte offset of the LDS copy of h (when it is in LDS)
    const float* hg;    // h in global memory (when it is not)
    const float* ss;
    const float* ecs;
    const double* C64;
    const float* Xs;
    int* sa;
    float* su;
    float* sD;
    const int* sq;
    int k;
    bool prune;
    float gamma, ecmax;
};

template <int D, int L, bool HL>
__device__ inline void grouped_survivors(const ScanCtx& W, int ns, int tid, int tp, uint64_t& comp,
                                         uint64_t& rechecks) {
    const float* hl = reinterpret_cast<const float*>(km_smem + W.h_off);
    auto hval = [&](int i) -> float {
        if constexpr (HL) return hl[i];
        else return W.hg[i];
    };
    constexpr int XS = ((D + 3) / 4) * 4 + 4;
    constexpr int DL = D / L;   // coordinates per lane
    const int per = tp / L;     // survivors per pass
    const int g = tid / L, sub = tid % L;
    const int k = W.k;
    for (int p0 = 0; p0 < ns; p0 += per) {
        const int slot = p0 + g;
        const bool act = slot < ns;
        const int r = W.sq[act ? slot : p0];
        const float* xrow = W.Xs + r * XS;
        float xp[DL];
        if constexpr (DL % 4 == 0) {
#pragma unroll
            for (int q = 0; q < DL; q += 4) {
                const f32x4 v = *reinterpret_cast<const f32x4*>(xrow + sub * DL + q);
                xp[q] = v.x;
                xp[q + 1] = v.y;
                xp[q + 2] = v.z;
                xp[q + 3] = v.w;
            }
        } else {
#pragma unroll
            for (int q = 0; q < DL; ++q) xp[q] = xrow[sub * DL + q];
        }
        auto dist = [&](int j) -> float {
            const float* c = W.Cs + j * D + sub * DL;
            float acc = 0.f;
#pragma unroll
            for (int q = 0; q < DL; ++q) {
                const float t = xp[q] - c[q];
                acc = fmaf(t, t, acc);
            }
            return group_sum<L>(acc);
        };
        const int inc = W.sa[r];
        int b = -1;
        float Db = INFINITY, D2 = INFINITY, ub = 0.f;
        uint64_t nc = 0;
        if (inc >= 0) {   // tighten: exact distance to the incumbent (U(u))
            Db = dist(inc);
            b = inc;
            nc = 1;
            ub = upper_bound(Db, W.ecs[inc], W.gamma);
        }
        const bool skip_all = W.prune && inc >= 0 && ub <= W.ss[inc];
        if (!skip_all) {
            for (int j = 0; j < k; ++j) {
                if (j == inc) continue;
                if (W.prune && b >= 0 && ub <= hval(b * k + j)) continue;   // Clause 2/3
                const float Dj = dist(j);
                nc += 1;
                if (Dj < Db) {
                    D2 = Db;
                    Db = Dj;
                    b = j;
                    ub = upper_bound(Db, W.ecs[j], W.gamma);
                } else if (Dj < D2) {
                    D2 = Dj;
                }
            }
        }
        bool re = false;
        if (D2 != INFINITY) {
            const float band = 2.f * W.gamma * (Db + D2) + 4.f * (sqrtf(Db) + sqrtf(D2)) * W.ecmax +
                               8.f * W.ecmax * W.ecmax;
            re = D2 - Db <= band;
        }
        if (act && sub == 0) {
            if (re) {   // float64 decision against the master centroids, oracle's tie rule
                int bb = -1;
                double Dbb = INFINITY;
                if (inc >= 0) {
                    Dbb = sqd64(xrow, W.C64 + (int64_t)inc * D, D);
                    bb = inc;
                }
                for (int j = 0; j < k; ++j) {
                    if (j == inc) continue;
                    const double Dj = sqd64(xrow, W.C64 + (int64_t)j * D, D);
                    if (Dj < Dbb) {
                        Dbb = Dj;
                        bb = j;
                    }
                }
                b = bb;
                Db = (float)Dbb;
                ub = f32_up(sqrt(Dbb) * (1.0 + 0x1p-40));
                rechecks += 1;
            }
            if (b < 0) b = 0;   // only for non-finite rows
            W.sa[r] = b;
            W.su[r] = ub;
            W.sD[r] = Db;
            comp += nc;
        }
    }
}

// Survivor scan for k <= 16 (d = 16 or 32): a group of G >= k lanes per
// survivor, lane j evaluates centroid j in the direct form unless Clause 2
// skips it (loose bound u <= h(a, j)); the group then takes the minimum
// with the oracle's tie rule and the second-best value with DPP row
// reductions.  All k distances of a survivor are in flight at once instead
// of one after another.

// All-reduce within rows of G lanes (G = 4, 8 or 16) on DPP row operations.
template <int G>
__device__ inline uint32_t dpp_min_u32(uint32_t v) {
    v = min(v, (uint32_t)__builtin_amdgcn_update_dpp((int)v, (int)v, 0xB1, 0xF, 0xF, false));   // xor 1
    v = min(v, (uint32_t)__builtin_amdgcn_update_dpp((int)v, (int)v, 0x4E, 0xF, 0xF, false));   // xor 2
    if constexpr (G >= 8)
        v = min(v, (uint32_t)__builtin_amdgcn_update_dpp((int)v, (int)v, 0x141, 0xF, 0xF, false));   // half mirror
    if constexpr (G >= 16)
        v = min(v, (uint32_t)__builtin_amdgcn_update_dpp((int)v, (int)v, 0x140, 0xF, 0xF, false));   // mirror
    return v;
}

template <int D, int G>
__device__ inline void klane_survivors(const ScanCtx& W, const float* hl, int ns, int tid, int tp,
                                       uint64_t& comp, uint64_t& rechecks) {
    constexpr int XS = ((D + 3) / 4) * 4 + 4;
    const int per = tp / G;            // survivors per pass
    const int g = tid / G, j = tid % G;
    const int k = W.k;
    const int lane = tid & 63;
    for (int p0 = 0; p0 < ns; p0 += per) {
        const int slot = p0 + g;
        const bool act = slot < ns;
        const int r = W.sq[act ? slot : p0];
        const float* xrow = W.Xs + r * XS;
        const int inc = W.sa[r];
        const float u = W.su[r];
        // Clause 2 with the loose bound: centroid j cannot beat the incumbent.
        const bool want = act && j < k &&
                          !(W.prune && inc >= 0 && j != inc && u <= hl[inc * k + j]);
        float Dj = INFINITY;
        if (want) {
            const float* c = W.Cs + j * D;
            float acc = 0.f;
#pragma unroll
            for (int m = 0; m < D; m += 4) {
                const f32x4 xv = *reinterpret_cast<const f32x4*>(xrow + m);
                const f32x4 cv = *reinterpret_cast<const f32x4*>(c + m);
                float t0 = xv.x - cv.x, t1 = xv.y - cv.y, t2 = xv.z - cv.z, t3 = xv.w - cv.w;
                acc = fmaf(t0, t0, acc);
                acc = fmaf(t1, t1, acc);
                acc = fmaf(t2, t2, acc);
                acc = fmaf(t3, t3, acc);
            }
            Dj = acc;
        }
        // D >= 0, so float order equals the order of the bit patterns.
        const uint32_t dbits = __float_as_uint(Dj);
        const uint32_t m1 = dpp_min_u32<G>(dbits);
        // Among the minimal lanes the incumbent wins, then the lowest index.
        const uint32_t key = dbits == m1 && want ? (j == inc ? 0u : (uint32_t)j + 1u) : 0xFFFFFFFFu;
        const uint32_t kmin = dpp_min_u32<G>(key);
        const int b = kmin == 0u ? inc : (int)kmin - 1;
        const uint32_t m2 = dpp_min_u32<G>(want && j != b ? dbits : 0x7F800000u);
        const float Db = __uint_as_float(m1), D2 = __uint_as_float(m2);
        const uint64_t wm = __ballot(want);
        const int gbase = lane - j;
        const uint64_t gm = G == 64 ? ~0ull : (((1ull << G) - 1ull) << gbase);
        if (act && j == 0) {
            int bb = b < 0 ? 0 : b;
            float Dbb = Db;
            float ub = upper_bound(Db, W.ecs[bb], W.gamma);
            if (D2 != INFINITY) {
                const float band = 2.f * W.gamma * (Db + D2) + 4.f * (sqrtf(Db) + sqrtf(D2)) * W.ecmax +
                                   8.f * W.ecmax * W.ecmax;
                if (D2 - Db <= band) {   // float64 decision, oracle's tie rule
                    int b64 = -1;
                    double D64 = INFINITY;
                    if (inc >= 0) {
                        D64 = sqd64(xrow, W.C64 + (int64_t)inc * D, D);
                        b64 = inc;
                    }
                    for (int q = 0; q < k; ++q) {
                        if (q == inc) continue;
                        const double Dq = sqd64(xrow, W.C64 + (int64_t)q * D, D);
                        if (Dq < D64) {
                            D64 = Dq;
                            b64 = q;
                        }
                    }
                    bb = b64 < 0 ? 0 : b64;
                    Dbb = (float)D64;
                    ub = f32_up(sqrt(D64) * (1.0 + 0x1p-40));
                    rechecks += 1;
                }
            }
            W.sa[r] = bb;
            W.su[r] = ub;
            W.sD[r] = Dbb;
            comp += (uint64_t)__popcll(wm & gm);
        }
    }
}

}  // namespace

// ---------------------------------------------------------------------------
// Assignment + partial sums.  Block = tp threads = one tile of tp points;
// blocks stride over tiles.  D > 0: the row lives in registers (D % 4 == 0);
// D == 0: any d, rows read from LDS.  KB == 0: the survivors run the
// per-point MTI scan on the vector units.  KB == 8: Elkan's triangle
// inequality scan (one lane per survivor) with a lower bound per point and
// centroid in addition to MTI's tests.  KB = 1, 2, 4 (D = 16 or 32, k <= 32*KB):
// the survivors' distances to all centroids come from float32 MFMA tiles
// (X . C^T in the expanded form |x|^2 + |c|^2 - 2 x.c), and every centroid
// within the expanded form's error bound of the best is re-evaluated in the
// direct form before the decision, so the result is the same as the vector
// path's.

template <int D, int KB>
__global__ __launch_bounds__(KB == 4 ? 512 : 256) __attribute__((amdgpu_waves_per_eu(2))) void k_assign(Dev P_) {
    const Dev P = with_scales(P_);
    constexpr bool ELK = KB == 8;          // Elkan's lower bounds, vector scan
    constexpr int MB = ELK ? 0 : KB;       // 32-centroid blocks of the matrix-core path
    constexpr bool WIDE = KB == 4;         // 512 threads, centroid operands in LDS
    IterState* st = P.st;
    if (st->done) {
        if (blockIdx.x == 0 && threadIdx.x == 0) st->active = 0;
        return;
    }
    if (blockIdx.x == 0 && threadIdx.x == 0) st->active = 1;

    const int d = D > 0 ? D : P.d;
    const int k = P.k;
    const int tp = blockDim.x;
    const int tid = threadIdx.x;
    const bool first = st->t == 0;
    const bool prune = !(P.flags & KM_FLAG_NO_PRUNE);
    const bool want_inertia = (P.flags & KM_FLAG_STATS) != 0;
    const float ecmax = st->ec_max;
    const float gamma = P.gamma;
    const int xs = xs_stride(d);

    const bool h_lds = assign_h_lds(KB, k);
    const AssignLds lay = assign_lds(d, k, tp, h_lds, WIDE);
    unsigned char* smem = km_smem;
    uint64_t* acc = reinterpret_cast<uint64_t*>(smem + lay.off_acc);
    uint32_t* cnt = reinterpret_cast<uint32_t*>(smem + lay.off_cnt);
    float* Cs = reinterpret_cast<float*>(smem + lay.off_c);
    float* fs = reinterpret_cast<float*>(smem + lay.off_f);
    float* ss = reinterpret_cast<float*>(smem + lay.off_s);
    float* ecs = reinterpret_cast<float*>(smem + lay.off_ec);
    float* Xs = reinterpret_cast<float*>(smem + lay.off_x);
    int* sa = reinterpret_cast<int*>(smem + lay.off_sa);
    float* su = reinterpret_cast<float*>(smem + lay.off_su);
    float* sD = reinterpret_cast<float*>(smem + lay.off_sd);
    int* sq = reinterpret_cast<int*>(smem + lay.off_sq);
    int* qlen = reinterpret_cast<int*>(smem + lay.off_misc);
    uint64_t* bst = reinterpret_cast<uint64_t*>(smem + lay.off_misc + 16);
    float* cn2s = reinterpret_cast<float*>(smem + lay.off_cn);
    if (h_lds) {   // half-distance table: LDS copy for small k
        float* hl = reinterpret_cast<float*>(smem + lay.off_h);
        for (int i = tid; i < k * k; i += tp) hl[i] = P.h[i];
    }

    for (int i = tid; i < k * d; i += tp) {
        Cs[i] = P.C32[i];
        acc[i] = 0;
    }
    for (int i = tid; i < k; i += tp) {
        cnt[i] = 0;
        fs[i] = P.f[i];
        ss[i] = P.s[i];
        ecs[i] = P.ec[i];
        if constexpr (ELK) cn2s[i] = P.dupf[i];   // the matrix-core norms' slot holds the drifts
    }
    if (tid < kNumStat) bst[tid] = 0;

    // Matrix-core path: this lane's A operands (centroid rows) for the whole
    // kernel.  Lane l feeds row (32*cb + l%32) and dimension half l/32; the
    // MFMA k-step s pairs dimension s with dimension D/2 + s.
    constexpr int kCb = MB > 0 ? MB : 1;
    constexpr int kHalf = D > 0 ? D / 2 : 1;
    float creg[WIDE ? 1 : kCb][WIDE ? 1 : kHalf];
    float* ca = reinterpret_cast<float*>(smem + lay.off_ca);   // WIDE: operand (cb, q) of lane l at (cb*kHalf + q)*64 + l
    float cnmax = 0.f;
    if constexpr (MB > 0) {
        static_assert(D == 16 || D == 32, "matrix-core path needs d = 16 or 32");
        const int lane = tid & 63, half = lane >> 5;
        if constexpr (WIDE) {
            for (int i = tid; i < MB * kHalf * 64; i += tp) {
                const int l = i & 63, q = (i >> 6) % kHalf, cb = i / (64 * kHalf);
                const int j = cb * 32 + (l & 31);
                ca[i] = j < k ? P.C32[(int64_t)j * D + (l >> 5) * kHalf + q] : 0.f;
            }
        } else {
#pragma unroll
            for (int cb = 0; cb < MB; ++cb) {
                const int j = cb * 32 + (lane & 31);
#pragma unroll
                for (int q = 0; q < kHalf; ++q)
                    creg[cb][q] = j < k ? P.C32[(int64_t)j * D + half * kHalf + q] : 0.f;
            }
        }
        for (int i = tid; i < MB * 32; i += tp) cn2s[i] = i < k ? P.cn2[i] : INFINITY;
        __syncthreads();
        float m2 = 0.f;
        for (int i = lane; i < k; i += 64) m2 = fmaxf(m2, cn2s[i]);
#pragma unroll
        for (int off = 32; off > 0; off >>= 1) m2 = fmaxf(m2, __shfl_xor(m2, off));
        cnmax = sqrtf(m2) * kUp;
    }
    // Error bound factor of an expanded-form float32 squared distance,
    // relative to (|x| + |c|)^2.
    const float gexp = (float)(D + 8) * 0x1p-24f;

    uint64_t my_changed = 0, my_comp = 0, my_c1 = 0, my_rc = 0, my_iq = 0;
    const int64_t ntiles = (P.n + tp - 1) / tp;

    // Register prefetch of the next tile: its X rows (coalesced 16-byte
    // chunks, specialised d only) and this thread's point state.  The loads
    // are branch-free (addresses clamped into the tile, so a short last tile
    // reads valid memory and ignores the extra values) so that the compiler
    // can keep them in flight across the whole tile body.
    constexpr int kChunks = D > 0 ? D / 4 : 1;   // 16-byte chunks per thread per tile
    f32x4 xbuf[kChunks];
    int abuf = 0;
    float ubuf = 0.f;
    auto prefetch = [&](int64_t tl) {
        const int64_t b = tl * tp;
        const int r = (int)((P.n - b) < tp ? (P.n - b) : tp);
        if constexpr (D > 0) {
            const f32x4* s4 = reinterpret_cast<const f32x4*>(P.X + b * D);
            const int last = r * kChunks - 1;
#pragma unroll
            for (int i = 0; i < kChunks; ++i) xbuf[i] = __builtin_nontemporal_load(s4 + min(tid + i * tp, last));
        }
        const int64_t q = b + min(tid, r - 1);
        abuf = P.a[q];   // unset before the first step: read but not used then
        ubuf = P.u[q];
    };
    if ((int64_t)blockIdx.x < ntiles) prefetch(blockIdx.x);
    if (tid < 2) qlen[tid] = 0;   // visible behind the first tile's barrier
    int it = 0;

    for (int64_t tile = blockIdx.x; tile < ntiles; tile += gridDim.x, ++it) {
        const int64_t base = tile * tp;
        const int rows = (int)((P.n - base) < tp ? (P.n - base) : tp);
        __syncthreads();   // the previous tile is fully consumed
        // Two survivor counters alternate: this tile's was cleared during the
        // previous one (behind the barrier above); clear the next tile's now.
        if (tid == 0) qlen[(it + 1) & 1] = 0;
        int* qn = qlen + (it & 1);

        // Bound update and Clause 1 on the prefetched state (before the next
        // prefetch reuses its registers).
        const bool valid = tid < rows;
        const int64_t p = base + tid;
        int a_old = -1;
        float u_cur = 0.f;
        bool surv = false;
        if (valid) {
            if (first) {
                surv = true;
            } else {
                a_old = abuf;
                u_cur = (ubuf + fs[a_old]) * kUp;
                if (!prune || u_cur > ss[a_old]) surv = true;
                else my_c1 += 1;
            }
        }

        // Stage the tile in LDS.
        if constexpr (D > 0) {
#pragma unroll
            for (int i = 0; i < kChunks; ++i) {
                const int c = tid + i * tp;
                if (c < rows * kChunks) {
                    const int r = c / kChunks, q = c - r * kChunks;
                    *reinterpret_cast<f32x4*>(Xs + r * xs + 4 * q) = xbuf[i];
                }
            }
        } else {
            const float* src = P.X + base * d;
            const int ne = rows * d;
            for (int e = tid; e < ne; e += tp) {
                const int r = e / d;
                Xs[r * xs + (e - r * d)] = src[e];
            }
        }
        if (tile + gridDim.x < ntiles) prefetch(tile + gridDim.x);

        if (valid) {
            sa[tid] = a_old;
            su[tid] = u_cur;
        }
        {   // compaction: one LDS atomic per wave, ranks from the ballot
            const uint64_t bm = __ballot(surv);
            const int lane = tid & 63;
            int wbase = 0;
            if (lane == 0 && bm) wbase = atomicAdd(qn, __popcll(bm));
            wbase = __shfl(wbase, 0);
            if (surv) sq[wbase + __popcll(bm & ((1ull << lane) - 1ull))] = tid;
        }
        __syncthreads();

        // Survivors, compacted into sq[0, nq).
        const int nq = *qn;
        if constexpr (MB > 0) {
            // Matrix cores: one wave per block of 32 survivors.  Lanes l and
            // l + 32 serve survivor l % 32 and hold 16 of its centroid
            // distances per 32-centroid block.
            const int lane = tid & 63, col = lane & 31, half = lane >> 5;
            const int nwaves = tp >> 6;
            for (int blk = tid >> 6; blk * 32 < nq; blk += nwaves) {
                const int qi = blk * 32 + col;
                const bool live = qi < nq;
                const int r = sq[live ? qi : blk * 32];
                const float* xr = Xs + r * xs;
                float xh[kHalf];
#pragma unroll
                for (int q = 0; q < kHalf; q += 4) {
                    const f32x4 v = *reinterpret_cast<const f32x4*>(xr + half * kHalf + q);
                    xh[q] = v.x;
                    xh[q + 1] = v.y;
                    xh[q + 2] = v.z;
                    xh[q + 3] = v.w;
                }
                float x2 = 0.f;
#pragma unroll
                for (int q = 0; q < kHalf; ++q) x2 = fmaf(xh[q], xh[q], x2);
                x2 += __shfl_xor(x2, 32);
                f32x16 dot[kCb];
#pragma unroll
                for (int cb = 0; cb < MB; ++cb)
#pragma unroll
                    for (int e = 0; e < 16; ++e) dot[cb][e] = 0.f;
#pragma unroll
                for (int q = 0; q < kHalf; ++q)
#pragma unroll
                    for (int cb = 0; cb < MB; ++cb)
                        dot[cb] = __builtin_amdgcn_mfma_f32_32x32x2f32(
                            WIDE ? ca[(cb * kHalf + q) * 64 + lane] : creg[WIDE ? 0 : cb][WIDE ? 0 : q], xh[q],
                            dot[cb], 0, 0, 0);
                // Register e of block cb holds centroid 32*cb + 8*(e/4) + 4*half + e%4.
                auto cent = [&](int cb, int e) { return cb * 32 + 8 * (e >> 2) + 4 * half + (e & 3); };
                float e1 = INFINITY;
#pragma unroll
                for (int cb = 0; cb < MB; ++cb)
#pragma unroll
                    for (int e = 0; e < 16; ++e)
                        e1 = fminf(e1, x2 + cn2s[cent(cb, e)] - 2.f * dot[cb][e]);
                e1 = fminf(e1, __shfl_xor(e1, 32));
                // Every centroid whose expanded-form value is within twice the
                // error bound of the smallest one is a candidate; the others
                // are certified farther than the true nearest centroid.
                const float R = sqrtf(fmaxf(x2, 0.f)) * kUp + cnmax;
                const float thr = e1 + 2.f * (gexp * R * R + 4.f * R * ecmax + 2.f * ecmax * ecmax);
                // Candidate bitmask (bit 16*cb + e), then direct-form distances
                // of the candidates from the LDS rows.
                uint64_t cmask = 0;
#pragma unroll
                for (int cb = 0; cb < MB; ++cb)
#pragma unroll
                    for (int e = 0; e < 16; ++e)
                        if (x2 + cn2s[cent(cb, e)] - 2.f * dot[cb][e] <= thr) cmask |= 1ull << (16 * cb + e);
                const int inc = live ? sa[r] : -1;
                const uint64_t cmask0 = cmask;
                // A single candidate over both half-waves is the nearest
                // centroid: its bound comes from its expanded value and the
                // error bound, without the direct form (kept with inertia).
                const int own = __popcll(cmask0);
                const bool single = !want_inertia && own + __shfl_xor(own, 32) == 1;
                const int jown = own ? cent(__builtin_ctzll(cmask0) >> 4, __builtin_ctzll(cmask0) & 15) : -1;
                const int jsingle = max(jown, __shfl_xor(jown, 32));
                if (single) cmask = 0;
                float d1 = INFINITY, d2 = INFINITY;
                int rk1 = INT_MAX, j1 = 0, ncand = 0;
                while (cmask) {
                    const int bit = __builtin_ctzll(cmask);
                    cmask &= cmask - 1;
                    const int j = cent(bit >> 4, bit & 15);
                    const float Dd = sqd_lds_fixed<D>(xr, Cs + j * D);
                    const int rk = j == inc ? -1 : j;   // incumbent wins a tie, then lowest index
                    ncand += 1;
                    if (Dd < d1 || (Dd == d1 && rk < rk1)) {
                        d2 = d1;
                        d1 = Dd;
                        rk1 = rk;
                        j1 = j;
                    } else if (Dd < d2) {
                        d2 = Dd;
                    }
                }
                const float od1 = __shfl_xor(d1, 32), od2 = __shfl_xor(d2, 32);
                const int ork = __shfl_xor(rk1, 32), oj = __shfl_xor(j1, 32);
                ncand += __shfl_xor(ncand, 32);
                if (od1 < d1 || (od1 == d1 && ork < rk1)) {
                    d2 = fminf(d1, fminf(d2, od2));
                    d1 = od1;
                    j1 = oj;
                } else {
                    d2 = fminf(d2, fminf(od1, od2));
                }
                // Near tie: float64 decision among the candidates (the only
                // centroids that can be nearest), each half-wave over its own,
                // then the smaller (distance, incumbent first, lower index).
                bool re = false;
                if (d2 != INFINITY) {
                    const float band = 2.f * gamma * (d1 + d2) +
                                       4.f * (sqrtf(d1) + sqrtf(d2)) * ecmax + 8.f * ecmax * ecmax;
                    re = live && d2 - d1 <= band;
                }
                double Dbb = INFINITY;
                int kb = INT_MAX, bb = -1;
                if (re) {
                    uint64_t cm = cmask0;
                    while (cm) {
                        const int bit = __builtin_ctzll(cm);
                        cm &= cm - 1;
                        const int j = cent(bit >> 4, bit & 15);
                        const double Dj = sqd64(xr, P.C64 + (int64_t)j * d, d);
                        const int rk = j == inc ? -1 : j;
                        if (Dj < Dbb || (Dj == Dbb && rk < kb)) {
                            Dbb = Dj;
                            kb = rk;
                            bb = j;
                        }
                    }
                }
                {
                    const double oD = __shfl_xor(Dbb, 32);
                    const int okb = __shfl_xor(kb, 32), obb = __shfl_xor(bb, 32);
                    if (oD < Dbb || (oD == Dbb && okb < kb)) {
                        Dbb = oD;
                        kb = okb;
                        bb = obb;
                    }
                }
                if (live && half == 0) {
                    int b = j1;
                    float Db = d1;
                    float ub = upper_bound(Db, ecs[b], gamma);
                    if (single) {
                        const float e1b = gexp * R * R + 4.f * R * ecmax + 2.f * ecmax * ecmax;
                        b = jsingle;
                        Db = e1;
                        ub = __builtin_amdgcn_sqrtf(fmaxf(e1 + e1b, 0.f)) * (1.0f + 0x1p-20f) * kUp;
                    }
                    if (re) {
                        b = bb < 0 ? 0 : bb;
                        Db = (float)Dbb;
                        ub = f32_up(sqrt(Dbb) * (1.0 + 0x1p-40));
                        my_rc += 1;
                    }
                    sa[r] = b;
                    su[r] = ub;
                    sD[r] = Db;
                    my_comp += (uint64_t)k;   // the dense pairs; refinements re-evaluate some
                }
            }
        } else if constexpr (D > 0 && !ELK) {
            ScanCtx W{Cs, lay.off_h, P.h, ss, ecs, P.C64, Xs, sa, su, sD, sq, k, prune, gamma, ecmax};
            const float* hl = reinterpret_cast<const float*>(km_smem + lay.off_h);
            if (k <= 4) {
                klane_survivors<D, 4>(W, hl, nq, tid, tp, my_comp, my_rc);
            } else if (k <= 8) {
                klane_survivors<D, 8>(W, hl, nq, tid, tp, my_comp, my_rc);
            } else if (k <= 16) {
                klane_survivors<D, 16>(W, hl, nq, tid, tp, my_comp, my_rc);
            } else if (h_lds) {
                grouped_survivors<D, 1, true>(W, nq, tid, tp, my_comp, my_rc);
            } else {
                grouped_survivors<D, 1, false>(W, nq, tid, tp, my_comp, my_rc);
            }
        } else {
            for (int qi = tid; qi < nq; qi += tp) {
                const int r = sq[qi];
                const float* xr = Xs + r * xs;
                Row<D> x;
                if constexpr (D > 0) {
    #pragma unroll
                    for (int m = 0; m < D; m += 4) {
                        const float4 v = *reinterpret_cast<const float4*>(xr + m);
                        x.v[m] = v.x;
                        x.v[m + 1] = v.y;
                        x.v[m + 2] = v.z;
                        x.v[m + 3] = v.w;
                    }
                }
                auto dist = [&](int j) -> float {
                    if constexpr (D > 0) return sqd_reg<D>(x, Cs + j * D);
                    else return sqd_lds(xr, Cs + j * d, d);
                };
                const int inc = sa[r];
                int b = -1;
                float Db = INFINITY, D2 = INFINITY, ub = 0.f;
                uint64_t nc = 0;
                if constexpr (ELK) {
                    // Elkan: skip c_j when the bound is within h(b, j) or
                    // within the lower bound l(x, c_j); the incumbent's
                    // distance is computed only when a centroid passes both
                    // tests with the loose bound.  Lower bounds are stored
                    // offset by the cumulative drift D_j of their centroid
                    // (l' = l + D_j then; l = l' - D_j now, rounded down).
                    float* lbp = P.lb + (base + r);
                    auto hv_of = [&](int bb, int j) -> float {
                        return h_lds ? reinterpret_cast<const float*>(smem + lay.off_h)[bb * k + j]
                                     : P.h[(int64_t)bb * k + j];
                    };
                    auto store_lb = [&](int j, float Dq) {
                        const double lo = ((double)sqrtf(Dq) * (1.0 - (double)gamma) - (double)ecs[j]) *
                                          (1.0 - 0x1p-20);
                        const double v = ((lo > 0.0 ? lo : 0.0) + P.dlo[j]) * (1.0 - 0x1p-50);
                        lbp[(int64_t)j * P.n] = f32_down(v);
                    };
                    bool tight = inc < 0;
                    if (inc >= 0) {
                        b = inc;
                        ub = su[r];
                    }
                    // ub <= l(x, c_j) = l' - D_j, tested as ub + D_j <= l' with
                    // the sum rounded up (D_j rounded up in dups).
                    const float* dups = cn2s;
                    auto below_lb = [&](float lp, int j) -> bool {
                        return !first && (ub + dups[j]) * (1.0f + 0x1p-22f) <= lp;
                    };
                    // Chunks of centroids: their lower bounds are loaded at
                    // once and tested against the bound at the chunk's start
                    // (tests only get stronger as the best improves); the
                    // candidates are then visited in ascending order and
                    // tested again with the current best and bound.
                    constexpr int kCh = D >= 32 ? 16 : 32;
                    for (int j0 = 0; j0 < k; j0 += kCh) {
                        float lv[kCh];
#pragma unroll
                        for (int q = 0; q < kCh; ++q)
                            lv[q] = (!first && j0 + q < k) ? lbp[(int64_t)(j0 + q) * P.n] : 0.f;
                        uint32_t m = 0;
#pragma unroll
                        for (int q = 0; q < kCh; ++q) {
                            const int j = j0 + q;
                            if (j < k && j != inc) {
                                const bool cut = prune && b >= 0 && (ub <= hv_of(b, j) || below_lb(lv[q], j));
                                m |= (cut ? 0u : 1u) << q;
                            }
                        }
                        while (m) {
                            const int q = __builtin_ctz(m);
                            m &= m - 1u;
                            const int j = j0 + q;
                            float lp = 0.f;
                            if (prune && b >= 0) {
                                if (ub <= hv_of(b, j)) continue;
                                if (!first) {
                                    lp = lbp[(int64_t)j * P.n];
                                    if (below_lb(lp, j)) continue;
                                }
                            }
                            if (!tight) {   // tighten: exact distance to the incumbent (U(u))
                                Db = dist(inc);
                                nc += 1;
                                tight = true;
                                ub = upper_bound(Db, ecs[inc], gamma);
                                store_lb(inc, Db);
                                if (prune && (ub <= hv_of(b, j) || below_lb(lp, j))) continue;
                            }
                            const float Dj = dist(j);
                            nc += 1;
                            store_lb(j, Dj);
                            if (Dj < Db) {
                                D2 = Db;
                                Db = Dj;
                                b = j;
                                ub = upper_bound(Db, ecs[j], gamma);
                            } else if (Dj < D2) {
                                D2 = Dj;
                            }
                        }
                    }
                    if (!tight) Db = -1.f;   // incumbent kept on the loose bound; distance not formed
                } else {
                if (inc >= 0) {   // tighten: exact distance to the incumbent (U(u))
                    Db = dist(inc);
                    b = inc;
                    nc += 1;
                    ub = upper_bound(Db, ecs[inc], gamma);
                }
                // Tightened bound within s(a): every other centroid is skipped.
                const bool skip_all = prune && inc >= 0 && ub <= ss[inc];
                if (!skip_all) {
                    for (int j = 0; j < k; ++j) {
                        if (j == inc) continue;
                        const float hv = h_lds ? reinterpret_cast<const float*>(smem + lay.off_h)[b * k + j]
                                           : P.h[(int64_t)b * k + j];
                    if (prune && b >= 0 && ub <= hv) continue;   // Clause 2/3
                        const float Dj = dist(j);
                        nc += 1;
                        if (Dj < Db) {
                            D2 = Db;
                            Db = Dj;
                            b = j;
                            ub = upper_bound(Db, ecs[j], gamma);
                        } else if (Dj < D2) {
                            D2 = Dj;
                        }
                    }
                }
                }
                // Near tie within the float32 error bound: decide in float64
                // against the master centroids with the oracle's tie rule.
                if (D2 != INFINITY) {
                    const float band = 2.f * gamma * (Db + D2) +
                                       4.f * (sqrtf(Db) + sqrtf(D2)) * ecmax + 8.f * ecmax * ecmax;
                    if (D2 - Db <= band) {
                        int bb = -1;
                        double Dbb = INFINITY;
                        if (inc >= 0) {
                            Dbb = sqd64(xr, P.C64 + (int64_t)inc * d, d);
                            bb = inc;
                        }
                        for (int j = 0; j < k; ++j) {
                            if (j == inc) continue;
                            const double Dj = sqd64(xr, P.C64 + (int64_t)j * d, d);
                            if (Dj < Dbb) {
                                Dbb = Dj;
                                bb = j;
                            }
                        }
                        b = bb;
                        Db = (float)Dbb;
                        ub = f32_up(sqrt(Dbb) * (1.0 + 0x1p-40));
                        my_rc += 1;
                    }
                }
                if (b < 0) b = 0;   // only for non-finite rows (no comparison succeeded)
                sa[r] = b;
                su[r] = ub;
                sD[r] = Db;
                my_comp += nc;
            }
        }
        __syncthreads();

        // Write back the point state; count members.
        if (valid) {
            const int a_new = sa[tid];
            if (a_new != a_old) {
                P.a[p] = a_new;
                my_changed += 1;
            }
            P.u[p] = su[tid];
            if (want_inertia) {
                float Dv;
                if (surv && sD[tid] >= 0.f) {
                    Dv = sD[tid];
                } else if constexpr (D > 0) {
                    Row<D> x;
#pragma unroll
                    for (int m = 0; m < D; ++m) x.v[m] = Xs[tid * xs + m];
                    Dv = sqd_reg<D>(x, Cs + a_new * D);
                } else {
                    Dv = sqd_lds(Xs + tid * xs, Cs + a_new * d, d);
                }
                my_iq += fixed_bits((double)Dv, P.iscale) - kMagicBits;
            }
            atomicAdd(&cnt[a_new], 1u);
        }

        // Per-cluster coordinate sums of every point of the tile (pruned or
        // not), as exact fixed-point integers in LDS.  Thread t adds
        // coordinate t % d of rows t / d, t / d + tp / d, ...
        if constexpr (D > 0) {
            if (tp % D == 0) {
                const int m = tid % D, r0 = tid / D, rstep = tp / D;
                const int nr = (rows - r0 + rstep - 1) / rstep;
                for (int i = 0; i < nr; ++i) {
                    const int r = r0 + i * rstep;
                    const uint64_t bits = fixed_bits((double)Xs[r * xs + m], P.qscale);
                    const uint32_t slot = (uint32_t)sa[r] * (uint32_t)D + (uint32_t)m;
                    atomicAdd(reinterpret_cast<unsigned long long*>(&acc[slot]), (unsigned long long)bits);
                }
            }
        } else {
            const int ne = rows * d;
            for (int e = tid; e < ne; e += tp) {
                const int r = e / d, m = e - r * d;
                const uint64_t bits = fixed_bits((double)Xs[r * xs + m], P.qscale);
                atomicAdd(reinterpret_cast<unsigned long long*>(&acc[sa[r] * d + m]),
                          (unsigned long long)bits);
            }
        }
    }
    __syncthreads();

    // Block counters, then the block's partial row.
    my_changed = wave_sum_u64(my_changed);
    my_comp = wave_sum_u64(my_comp);
    my_c1 = wave_sum_u64(my_c1);
    my_rc = wave_sum_u64(my_rc);
    my_iq = wave_sum_u64(my_iq);
    if ((tid & 63) == 0) {
        atomicAdd(reinterpret_cast<unsigned long long*>(&bst[kStChanged]), my_changed);
        atomicAdd(reinterpret_cast<unsigned long long*>(&bst[kStComputed]), my_comp);
        atomicAdd(reinterpret_cast<unsigned long long*>(&bst[kStClause1]), my_c1);
        atomicAdd(reinterpret_cast<unsigned long long*>(&bst[kStRecheck]), my_rc);
        atomicAdd(reinterpret_cast<unsigned long long*>(&bst[kStInertia]), my_iq);
    }
    __syncthreads();
    uint64_t* row = P.part + (int64_t)blockIdx.x * P.L;
    for (int i = tid; i < k * d; i += tp) row[i] = acc[i];
    for (int i = tid; i < k; i += tp) row[k * d + i] = cnt[i];
    if (tid < kNumStat) row[k * d + k + tid] = bst[tid];
}

// ---------------------------------------------------------------------------
// Second pass: total[col] = sum over blocks of part[g][col].  Integer, so the
// order of the additions does not matter.  Grid: (ceil(L/64), slices).

constexpr int kReduceRows = 64;   // partial rows per slice

__global__ __launch_bounds__(256) void k_reduce(Dev P) {
    if (!P.st->active) return;
    const int col = blockIdx.x * 64 + (threadIdx.x & 63);
    const int sub = threadIdx.x >> 6;
    const int g0 = blockIdx.y * kReduceRows;
    const int g1 = min(P.G, g0 + kReduceRows);
    uint64_t v = 0;
    if (col < P.L)
        for (int g = g0 + sub; g < g1; g += 4) v += P.part[(int64_t)g * P.L + col];
    __shared__ uint64_t red[256];
    red[threadIdx.x] = v;
    __syncthreads();
    if (sub == 0 && col < P.L) {
        v = red[threadIdx.x] + red[threadIdx.x + 64] + red[threadIdx.x + 128] + red[threadIdx.x + 192];
        atomicAdd(reinterpret_cast<unsigned long long*>(&P.total[col]), (unsigned long long)v);
    }
}

// ---------------------------------------------------------------------------
// Update: one wave per cluster j.  c_j = sum / count (an empty cluster keeps
// c_j), drift f_j = ||c_j^{t+1} - c_j^t|| rounded up, float32 copy and its
// rounding error.  Block 0 also closes the iteration: counters, history
// record, step count and the stop test.  Leaves total[] zero.

__global__ __launch_bounds__(64) void k_update(Dev P_) {
    const Dev P = with_scales(P_);
    IterState* st = P.st;
    if (!st->active) return;
    const int j = blockIdx.x, d = P.d, k = P.k;
    // The exact sums of the step: the reduced row, or on the incremental
    // path the running sums plus the reduced moves (wrap-around integers).
    auto total = [&](int64_t o) { return P.sums ? P.sums[o] + P.total[o] : P.total[o]; };
    const uint64_t count = total((int64_t)k * d + j);
    auto mean = [&](uint64_t v) {
        const int64_t q = (int64_t)(v - count * kMagicBits);
        return ((double)q * P.qinv) / (double)count;
    };
    // Spherical k-means: the mean is projected to the unit sphere (a zero
    // mean keeps the centroid).
    double scale = 1.0;
    bool keep = count == 0;
    if ((P.flags & KM_FLAG_SPHERICAL) && count > 0) {
        double s = 0.0;
        for (int m = threadIdx.x; m < d; m += 64) {
            const double v = mean(total((int64_t)j * d + m));
            s = fma(v, v, s);
        }
#pragma unroll
        for (int off = 32; off > 0; off >>= 1) s += __shfl_xor(s, off);
        if (s > 0.0) scale = sqrt(s);
        else keep = true;
    }
    double dr = 0.0, de = 0.0;
    for (int m = threadIdx.x; m < d; m += 64) {
        const int64_t o = (int64_t)j * d + m;
        const double cold = P.C64[o];
        const uint64_t tv = total(o);
        const double cnew = keep ? cold : mean(tv) / scale;
        if (P.sums) P.sums[o] = tv;
        P.total[o] = 0;
        const double df = cnew - cold;
        dr = fma(df, df, dr);
        const float c32 = (float)cnew;
        const double e = (double)c32 - cnew;
        de = fma(e, e, de);
        P.C64[o] = cnew;
        P.C32[o] = c32;
    }
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) {
        dr += __shfl_xor(dr, off);
        de += __shfl_xor(de, off);
    }
    if (threadIdx.x == 0) {
        P.f[j] = f32_up(sqrt(dr) * (1.0 + 0x1p-40));
        P.ec[j] = f32_up(sqrt(de) * (1.0 + 0x1p-40));
        if (P.sums) P.sums[(int64_t)k * d + j] = count;
        P.total[(int64_t)k * d + j] = 0;
        if (P.dhi) {   // cumulative drift, bracketed (Elkan lower bounds, incremental bounds)
            const double fd = sqrt(dr);
            const double hi = (P.dhi[j] + fd * (1.0 + 0x1p-40)) * (1.0 + 0x1p-50);
            const double lo = (P.dlo[j] + fd * (1.0 - 0x1p-40)) * (1.0 - 0x1p-50);
            P.dhi[j] = hi;
            P.dlo[j] = lo;
            P.dupf[j] = f32_up(hi);
            if (P.ddnf) P.ddnf[j] = f32_down(lo);
        }
    }
    if (j == 0 && threadIdx.x == 0) {
        uint64_t* sc = P.total + (int64_t)k * d + k;
        const int64_t changed = (int64_t)sc[kStChanged];
        const int64_t computed = (int64_t)sc[kStComputed];
        const int64_t c1 = (int64_t)sc[kStClause1];
        const int64_t rc = (int64_t)sc[kStRecheck];
        const int64_t iq = (int64_t)sc[kStInertia];
        for (int c = 0; c < kNumStat; ++c) sc[c] = 0;
        const double inertia = (P.flags & KM_FLAG_STATS) ? (double)iq * P.iinv : NAN;
        const int t = st->t;
        IterRec& r = P.rec[t % kHistCap];
        r.changed = changed;
        r.computed = computed;
        r.clause1 = c1;
        r.rechecks = rc;
        r.inertia = inertia;
        st->changed_last = changed;
        st->tot_computed += computed;
        st->tot_clause1 += c1;
        st->tot_rechecks += rc;
        st->inertia_last = inertia;
        st->t = t + 1;
        const bool tol_hit = (double)changed < st->tol_n;
        if (tol_hit || t + 1 >= st->max_iters) {
            st->done = 1;
            st->converged = tol_hit ? 1 : 0;
        }
        report_step(st, t, tol_hit || t + 1 >= st->max_iters);
    }
}

// ---------------------------------------------------------------------------
// Launchers

int assign_variant(int d, int k, bool aligned, bool vector_only, bool elkan) {
    const int D = aligned && (d == 16 || d == 32) ? d : 0;
    if (elkan) return 16 * D + 8;
    int KB = 0;
    if (D > 0 && !vector_only && k > 16 && k <= 128) KB = k <= 32 ? 1 : (k <= 64 ? 2 : 4);
    return 16 * D + KB;
}

#define KM_ASSIGN_VARIANTS(X) \
    X(0, 0) X(16, 0) X(32, 0) X(16, 1) X(16, 2) X(16, 4) X(32, 1) X(32, 2) X(32, 4) X(0, 8) X(16, 8) X(32, 8)

const void* assign_kernel_symbol(int variant) {
    switch (variant) {
#define KM_SYM(D_, KB_) \
    case 16 * D_ + KB_: return reinterpret_cast<const void*>(&k_assign<D_, KB_>);
        KM_ASSIGN_VARIANTS(KM_SYM)
#undef KM_SYM
        default: return nullptr;
    }
}

hipError_t launch_absmax(const float* a, int64_t na, const float* b, int64_t nb, const float* x, int64_t n,
                         int32_t d, int cus, uint32_t* out, hipStream_t s) {
    if (na < 0 || nb < 1 || n < 1 || d < 1) return hipErrorInvalidValue;
    // a (X): up to kAbsBlocksPerCU blocks per CU (none when na = 0); b (C0):
    // a few blocks; then the sample's chunks.
    int64_t ba = (na + 4 * 4 * 256 - 1) / (4 * 4 * 256);
    if (ba > kAbsBlocksPerCU * (int64_t)cus) ba = kAbsBlocksPerCU * (int64_t)cus;
    int64_t bb = (nb + 4 * 4 * 256 - 1) / (4 * 4 * 256);
    if (bb > 64) bb = 64;
    if (bb < 1) bb = 1;
    const int64_t rows = d >= 1024 ? 1 : 1024 / d;
    const int whole = na == n * d && a == x && n <= kAbsSampleChunks * rows ? 1 : 0;
    hipLaunchKernelGGL(k_absmax, dim3((unsigned)(ba + bb + (whole ? 0 : kAbsSampleChunks))), dim3(256), 0, s, a, na,
                       b, nb, (int)ba, (int)bb, x, n, d, whole, out);
    return hipGetLastError();
}

hipError_t launch_set_scales(IterState* st, const uint32_t* absmax, int64_t n, int32_t d, int unit, hipStream_t s) {
    hipLaunchKernelGGL(k_set_scales, dim3(1), dim3(64), 0, s, st, absmax, n, d, unit);
    return hipGetLastError();
}

hipError_t launch_init_buffers(const ZeroRanges& z, int cus, hipStream_t s) {
    if (z.overflow || z.n < 0 || z.n > ZeroRanges::kMax) return hipErrorInvalidValue;
    uint64_t total = 0;
    for (int r = 0; r < z.n; ++r) {
        if ((reinterpret_cast<uintptr_t>(z.p[r]) & 15) || (z.bytes[r] & 3)) return hipErrorInvalidValue;
        total += z.bytes[r];
    }
    int64_t blocks = (int64_t)(total / (16 * 256 * 4)) + 1;
    if (blocks > 8 * (int64_t)cus) blocks = 8 * (int64_t)cus;
    hipLaunchKernelGGL(k_init_buffers, dim3((unsigned)blocks), dim3(256), 0, s, z);
    return hipGetLastError();
}

hipError_t launch_normalize_rows(const float* X, int64_t n, int32_t d, float* Xn, hipStream_t s) {
    int64_t blocks = (n + 255) / 256;
    if (blocks > 16384) blocks = 16384;
    hipLaunchKernelGGL(k_normalize_rows, dim3((unsigned)blocks), dim3(256), 0, s, X, n, d, Xn);
    return hipGetLastError();
}

hipError_t launch_set_centroids_unit(const float* C0, double* C64, float* C32, float* ec, int32_t k, int32_t d,
                                     int32_t* zero, hipStream_t s) {
    hipLaunchKernelGGL(k_set_centroids_unit, dim3((unsigned)((k + 255) / 256)), dim3(256), 0, s, C0, C64, C32, ec,
                       k, d, zero);
    return hipGetLastError();
}

hipError_t launch_set_centroids(const float* C0, double* C64, float* C32, float* ec, int64_t kd,
                                int32_t k, hipStream_t s) {
    int64_t m = kd > k ? kd : k;
    hipLaunchKernelGGL(k_set_centroids, dim3((unsigned)((m + 255) / 256)), dim3(256), 0, s, C0, C64,
                       C32, ec, kd, k);
    return hipGetLastError();
}

hipError_t launch_assign(const Dev& dv, int variant, int tp, int lds_bytes, hipStream_t s) {
    switch (variant) {
#define KM_LAUNCH(D_, KB_)                                                              \
    case 16 * D_ + KB_:                                                                 \
        hipLaunchKernelGGL((k_assign<D_, KB_>), dim3(dv.G), dim3(tp), lds_bytes, s, dv); \
        break;
        KM_ASSIGN_VARIANTS(KM_LAUNCH)
#undef KM_LAUNCH
        default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

hipError_t launch_reduce(const Dev& dv, hipStream_t s) {
    dim3 grid((unsigned)((dv.L + 63) / 64), (unsigned)((dv.G + kReduceRows - 1) / kReduceRows));
    hipLaunchKernelGGL(k_reduce, grid, dim3(256), 0, s, dv);
    return hipGetLastError();
}

hipError_t launch_update(const Dev& dv, hipStream_t s) {
    hipLaunchKernelGGL(k_update, dim3(dv.k), dim3(64), 0, s, dv);
    return hipGetLastError();
}

hipError_t launch_centroid_table(const Dev& dv, int force, hipStream_t s) {
    hipLaunchKernelGGL(k_centroid_table, dim3(dv.k), dim3(256), 0, s, dv, force);
    return hipGetLastError();
}

}  // namespace km
