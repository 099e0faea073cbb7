// k-means++ seeding (paper section IV-C: each new seed is a data point drawn
// with probability D(v)^2 / sum D(v)^2, D the distance to the nearest seed
// so far).  The caller supplies the uniform numbers, so a seeding is a pure
// function of (X, k, u) and is reproduced bit for bit by any implementation
// of the same arithmetic:
//   - D^2 of a row to a seed in float64, coordinate differences summed in
//     index order by fused multiply-add; one lane owns a row, so the order
//     is the sequential one;
//   - the draw uses integer weights w_i = floor(D2_i * 2^S) (exact sums in any
//     order; S from the maximum of the current D2), T = floor(u * W) and the
//     smallest i whose inclusive prefix exceeds T.
//
// Kernels, per seed t (t = 0 first):
//   k_pp_step    one pass over the points: D2 = min(D2, ||x - c_t||^2) (all
//                points for t = 0) and the block's max of D2 (atomic max into
//                the slot of seed t);
//                with pruning a point is skipped when its nearest seed a is
//                at least twice as far from c_t as the point (triangle
//                inequality, Elkan's lemma; margins cover the float64
//                rounding, so D2 is unchanged by construction);
//   k_pp_weights the block sums of the next draw's weights, with the scale of
//                the maximum the pass before it left in its slot;
//   k_pp_select  one workgroup: scans the block sums, finds the block and
//                then the point of the draw, writes the seed index and row;
//   k_pp_dcc     the distances from the new seed to the earlier seeds (the
//                pruning table of the next pass), spread over the chip.
#include <math.h>
#include <stdint.h>

#include "km_device.h"
#include "km_internal.h"

namespace km {
namespace {

constexpr int kPPThreads = 256;
constexpr int kPPPer = kPPChunk / kPPThreads;   // points per thread in a pass
constexpr int kPPSelThreads = 1024;             // select kernel: 2 points per thread of a chunk
static_assert(kPPChunk == 2 * kPPSelThreads, "the select kernel covers one chunk with 2 points per thread");

// Seed draw from a uniform u in [0, 1) over n rows.
__device__ __forceinline__ int64_t uniform_index(double u, int64_t n) {
    const int64_t i = (int64_t)(u * (double)n);
    return i < n - 1 ? i : n - 1;
}

// Weight scale: S = 62 - e - L with M < 2^e (M > 0) and n <= 2^L.
__device__ __forceinline__ int weight_scale(double M, int L) {
    if (!(M > 0.0)) return 0;
    int e = 0;
    (void)frexp(M, &e);
    return 62 - e - L;
}

__device__ __forceinline__ uint64_t weight_of(double d2, int S) {
    return (uint64_t)floor(ldexp(d2, S));
}

__device__ __forceinline__ uint64_t wave_max_u64(uint64_t v) {
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) {
        const uint64_t o = __shfl_xor(v, off);
        v = o > v ? o : v;
    }
    return v;
}

// Inclusive scan of v over the block (blockDim.x multiple of 64, <= 1024);
// *total receives the block's sum.  lds: 16 words.  Contains barriers.
__device__ __forceinline__ uint64_t block_scan_u64(uint64_t v, uint64_t* lds, uint64_t* total) {
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, nw = blockDim.x >> 6;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
        const uint64_t o = __shfl_up(v, off);
        if (lane >= off) v += o;
    }
    if (lane == 63) lds[w] = v;
    __syncthreads();
    uint64_t pre = 0, tot = 0;
    for (int j = 0; j < nw; ++j) {
        const uint64_t s = lds[j];
        pre += j < w ? s : 0;
        tot += s;
    }
    __syncthreads();
    *total = tot;
    return v + pre;
}

// Two rows' squared distances to c at once (independent chains, so their
// loads are in flight together).  Each is ||x - c||^2 in float64 with the
// coordinate differences summed in index order by fused multiply-add.
template <int VW>
__device__ __forceinline__ void dist2_pair(const float* __restrict__ x0, const float* __restrict__ x1,
                                           const float* __restrict__ c, int d, double& r0, double& r1) {
    double a0 = 0.0, a1 = 0.0;
    auto quad = [&](int m) __attribute__((always_inline)) {
        const f32x4 u0 = *reinterpret_cast<const f32x4*>(x0 + m);
        const f32x4 u1 = *reinterpret_cast<const f32x4*>(x1 + m);
        const f32x4 cv = *reinterpret_cast<const f32x4*>(c + m);
        double e0 = (double)u0.x - (double)cv.x, e1 = (double)u1.x - (double)cv.x;
        a0 = fma(e0, e0, a0);
        a1 = fma(e1, e1, a1);
        e0 = (double)u0.y - (double)cv.y;
        e1 = (double)u1.y - (double)cv.y;
        a0 = fma(e0, e0, a0);
        a1 = fma(e1, e1, a1);
        e0 = (double)u0.z - (double)cv.z;
        e1 = (double)u1.z - (double)cv.z;
        a0 = fma(e0, e0, a0);
        a1 = fma(e1, e1, a1);
        e0 = (double)u0.w - (double)cv.w;
        e1 = (double)u1.w - (double)cv.w;
        a0 = fma(e0, e0, a0);
        a1 = fma(e1, e1, a1);
    };
    if (VW == 2) {   // d a multiple of 32: a 128-byte line of each row per step
        for (int m = 0; m < d; m += 32) {
#pragma unroll
            for (int q = 0; q < 32; q += 4) quad(m + q);
        }
    } else if (VW == 1) {
#pragma unroll 4
        for (int m = 0; m < d; m += 4) quad(m);
    } else {
#pragma unroll 4
        for (int m = 0; m < d; ++m) {
            const double cm = (double)c[m];
            const double e0 = (double)x0[m] - cm, e1 = (double)x1[m] - cm;
            a0 = fma(e0, e0, a0);
            a1 = fma(e1, e1, a1);
        }
    }
    r0 = a0;
    r1 = a1;
}

// One pass with seed t over a chunk of kPPChunk rows.  FIRST: D2 starts as
// the distance to seed 0.  PRUNE: skip test against the seed-to-seed table.
//   1. every row's D2 (and nearest seed) read with coalesced loads, the skip
//      test, and the rows that must be computed appended to an LDS list;
//   2. the listed rows spread over all lanes, two per lane at a time;
//   3. the max of the chunk's D2 values kept in LDS.
template <bool FIRST, bool PRUNE, int VW>
__global__ __launch_bounds__(kPPThreads) void k_pp_step(PPArgs P, int t) {
    __shared__ double sD[kPPChunk];
    __shared__ uint16_t sL[kPPChunk];
    __shared__ int sN;
    __shared__ uint64_t red[3][kPPThreads / 64];
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const int64_t base = (int64_t)blockIdx.x * kPPChunk;
    const int nloc = P.n - base < kPPChunk ? (int)(P.n - base) : kPPChunk;
    const int d = P.d;
    const float* __restrict__ c = P.C + (int64_t)t * d;
    constexpr bool kAll = FIRST || !PRUNE;   // every row is computed
    if (tid == 0) sN = 0;
    if (!FIRST) {
        double Dq[kPPPer];
        int32_t Aq[kPPPer];
#pragma unroll
        for (int q = 0; q < kPPPer; ++q) {
            const int j = q * kPPThreads + tid;
            Dq[q] = j < nloc ? P.D2[base + j] : 0.0;
            if (PRUNE) Aq[q] = j < nloc ? P.A[base + j] : 0;
        }
#pragma unroll
        for (int q = 0; q < kPPPer; ++q) {
            const int j = q * kPPThreads + tid;
            if (j < nloc) sD[j] = Dq[q];
        }
        if (PRUNE) {
            double Bq[kPPPer];
#pragma unroll
            for (int q = 0; q < kPPPer; ++q) Bq[q] = P.dcc[Aq[q]];
            __syncthreads();   // sN = 0 is visible
#pragma unroll
            for (int q = 0; q < kPPPer; ++q) {
                const int j = q * kPPThreads + tid;
                const bool surv = j < nloc && !(Bq[q] >= 4.0 * Dq[q] * (1.0 + 0x1p-26));
                const uint64_t bm = __ballot(surv);
                int wbase = 0;
                if (lane == 0 && bm) wbase = atomicAdd(&sN, __popcll(bm));
                wbase = __shfl(wbase, 0);
                if (surv) sL[wbase + __popcll(bm & ((1ull << lane) - 1ull))] = (uint16_t)j;
            }
        }
    }
    __syncthreads();
    const int ns = kAll ? nloc : sN;
    uint64_t ncomp = 0, nimp = 0;
    auto settle = [&](int j, double v) __attribute__((always_inline)) {
        const int64_t i = base + j;
        ++ncomp;
        if (FIRST) {
            P.D2[i] = v;
            if (PRUNE) P.A[i] = 0;
            sD[j] = v;
        } else if (v < sD[j]) {
            P.D2[i] = v;
            if (PRUNE) P.A[i] = t;
            sD[j] = v;
            ++nimp;
        }
    };
    for (int s0 = tid; s0 < ns; s0 += 2 * kPPThreads) {
        const int s1 = s0 + kPPThreads;
        const int j0 = kAll ? s0 : (int)sL[s0];
        const int j1 = s1 < ns ? (kAll ? s1 : (int)sL[s1]) : j0;
        double v0, v1;
        dist2_pair<VW>(P.X + (base + j0) * d, P.X + (base + j1) * d, c, d, v0, v1);
        settle(j0, v0);
        if (s1 < ns) settle(j1, v1);
    }
    __syncthreads();
    uint64_t dmax = 0;
#pragma unroll
    for (int q = 0; q < kPPPer; ++q) {
        const int j = q * kPPThreads + tid;
        if (j < nloc) {
            const uint64_t db = (uint64_t)__double_as_longlong(sD[j]);   // D >= 0: bits order as values
            dmax = db > dmax ? db : dmax;
        }
    }
    dmax = wave_max_u64(dmax);
    if (P.cnt) {
        ncomp = wave_sum_u64(ncomp);
        nimp = wave_sum_u64(nimp);
    }
    if (lane == 0) {
        red[0][w] = dmax;
        red[1][w] = ncomp;
        red[2][w] = nimp;
    }
    __syncthreads();
    if (tid == 0) {
        uint64_t b = 0, cc = 0, ci = 0;
#pragma unroll
        for (int j = 0; j < kPPThreads / 64; ++j) {
            b = red[0][j] > b ? red[0][j] : b;
            cc += red[1][j];
            ci += red[2][j];
        }
        atomicMax(reinterpret_cast<unsigned long long*>(P.Mb + t), (unsigned long long)b);
        if (P.cnt) {   // counters of the pass: distances computed, rows improved
            atomicAdd(reinterpret_cast<unsigned long long*>(P.cnt + 2 * t), (unsigned long long)cc);
            atomicAdd(reinterpret_cast<unsigned long long*>(P.cnt + 2 * t + 1), (unsigned long long)ci);
        }
    }
}

// Block sums of the weights of the draw after the pass with seed t (scale
// from that pass's maximum of D2).
__global__ __launch_bounds__(kPPThreads) void k_pp_weights(PPArgs P, int t) {
    __shared__ uint64_t red[kPPThreads / 64];
    const int tid = threadIdx.x;
    const int64_t base = (int64_t)blockIdx.x * kPPChunk;
    const int S = weight_scale(__longlong_as_double((long long)P.Mb[t]), P.L);
    uint64_t wsum = 0;
#pragma unroll
    for (int q = 0; q < kPPPer; ++q) {
        const int64_t i = base + q * kPPThreads + tid;
        if (i < P.n) wsum += weight_of(P.D2[i], S);
    }
    wsum = wave_sum_u64(wsum);
    if ((tid & 63) == 0) red[tid >> 6] = wsum;
    __syncthreads();
    if (tid == 0) {
        uint64_t a = 0;
#pragma unroll
        for (int j = 0; j < kPPThreads / 64; ++j) a += red[j];
        P.bs[blockIdx.x] = a;
    }
}

// Set-up: seed 0 (drawn on the host), the per-step max slots and counters.
__global__ __launch_bounds__(256) void k_pp_init(PPArgs P, int64_t i0) {
    const int tid = threadIdx.x;
    if (tid == 0) P.idx[0] = i0;
    for (int m = tid; m < P.d; m += blockDim.x) P.C[m] = P.X[i0 * P.d + m];
    for (int j = tid; j < P.k; j += blockDim.x) {
        P.Mb[j] = 0;
        if (P.cnt) P.cnt[2 * j] = P.cnt[2 * j + 1] = 0;
    }
}

// Draw of seed t + 1 from the weights after the pass with seed t.
__global__ __launch_bounds__(kPPSelThreads) void k_pp_select(PPArgs P, int t, int table) {
    __shared__ uint64_t scan_lds[16];
    __shared__ int64_t s_pick;
    __shared__ int64_t s_blk;
    __shared__ uint64_t s_rem;
    const int tid = threadIdx.x;
    const int G = P.G;
    const int per = (G + kPPSelThreads - 1) / kPPSelThreads;
    const int b0 = min(tid * per, G), b1 = min(b0 + per, G);
    uint64_t part = 0;
    for (int b = b0; b < b1; ++b) part += P.bs[b];
    uint64_t W = 0;
    const uint64_t incl = block_scan_u64(part, scan_lds, &W);
    const double u = P.u[t + 1];
    if (tid == 0) {
        s_pick = uniform_index(u, P.n);   // W = 0: every point lies on a seed
        s_blk = -1;
        s_rem = 0;
    }
    __syncthreads();
    if (W > 0) {
        uint64_t T = (uint64_t)(u * (double)W);
        if (T >= W) T = W - 1;
        const uint64_t excl = incl - part;
        if (part > 0 && excl <= T && T < incl) {   // exactly one thread
            uint64_t run = excl;
            for (int b = b0; b < b1; ++b) {
                const uint64_t nx = run + P.bs[b];
                if (nx > T) {
                    s_blk = b;
                    s_rem = T - run;
                    break;
                }
                run = nx;
            }
        }
        __syncthreads();
        const int64_t blk = s_blk;
        if (blk >= 0) {   // always, as the block sums add up to W
            const int S = weight_scale(__longlong_as_double((long long)P.Mb[t]), P.L);
            const int64_t i0 = blk * kPPChunk + 2 * tid;
            const uint64_t w0 = i0 < P.n ? weight_of(P.D2[i0], S) : 0;
            const uint64_t w1 = i0 + 1 < P.n ? weight_of(P.D2[i0 + 1], S) : 0;
            uint64_t tot = 0;
            const uint64_t inc2 = block_scan_u64(w0 + w1, scan_lds, &tot);
            const uint64_t ex2 = inc2 - (w0 + w1);
            const uint64_t R = s_rem;
            if (w0 + w1 > 0 && ex2 <= R && R < inc2) s_pick = ex2 + w0 > R ? i0 : i0 + 1;
        }
    }
    __syncthreads();
    const int64_t pick = s_pick;
    const int d = P.d;
    if (tid == 0) P.idx[t + 1] = pick;
    const float* __restrict__ xp = P.X + pick * d;
    for (int m = tid; m < d; m += kPPSelThreads) P.C[(int64_t)(t + 1) * d + m] = xp[m];
    // Small seed-to-seed tables are formed here (one thread per earlier
    // seed; as in k_pp_dcc), larger ones by k_pp_dcc over the chip.
    if (!table) return;
    for (int a = tid; a <= t; a += kPPSelThreads) {
        const float* __restrict__ ca = P.C + (int64_t)a * d;
        double acc = 0.0;
        for (int m = 0; m < d; ++m) {
            const double e = (double)ca[m] - (double)xp[m];
            acc = fma(e, e, acc);
        }
        P.dcc[a] = acc * (1.0 - 0x1p-28);
    }
}

// Seed-to-seed table for the pass with seed t + 1: a lower bound of
// ||c_a - c_{t+1}||^2 for every a <= t (any summation order; margin 2^-28
// over the float64 rounding).  G lanes (a power of two) share one earlier
// seed; the grid covers t + 1 seeds.
__global__ __launch_bounds__(256) void k_pp_dcc(PPArgs P, int t, int G, int vec4) {
    const int gid = blockIdx.x * 256 + threadIdx.x;
    const int a = gid / G, r = gid % G;
    const int d = P.d;
    const float* __restrict__ cn = P.C + (int64_t)(t + 1) * d;
    double acc = 0.0;
    if (a <= t) {
        const float* __restrict__ ca = P.C + (int64_t)a * d;
        if (vec4) {
#pragma unroll 4
            for (int m = 4 * r; m < d; m += 4 * G) {
                const f32x4 av = *reinterpret_cast<const f32x4*>(ca + m);
                const f32x4 pv = *reinterpret_cast<const f32x4*>(cn + m);
                double e = (double)av.x - (double)pv.x;
                acc = fma(e, e, acc);
                e = (double)av.y - (double)pv.y;
                acc = fma(e, e, acc);
                e = (double)av.z - (double)pv.z;
                acc = fma(e, e, acc);
                e = (double)av.w - (double)pv.w;
                acc = fma(e, e, acc);
            }
        } else {
#pragma unroll 4
            for (int m = r; m < d; m += G) {
                const double e = (double)ca[m] - (double)cn[m];
                acc = fma(e, e, acc);
            }
        }
    }
    for (int off = G >> 1; off > 0; off >>= 1) acc += __shfl_xor(acc, off);
    if (a <= t && r == 0) P.dcc[a] = acc * (1.0 - 0x1p-28);
}

template <bool FIRST, bool PRUNE>
hipError_t step_vec(const PPArgs& P, int t, int vw, hipStream_t s) {
    const dim3 grid((unsigned)P.G), block(kPPThreads);
    if (vw == 2)
        hipLaunchKernelGGL((k_pp_step<FIRST, PRUNE, 2>), grid, block, 0, s, P, t);
    else if (vw == 1)
        hipLaunchKernelGGL((k_pp_step<FIRST, PRUNE, 1>), grid, block, 0, s, P, t);
    else
        hipLaunchKernelGGL((k_pp_step<FIRST, PRUNE, 0>), grid, block, 0, s, P, t);
    return hipGetLastError();
}

}  // namespace

// The seed-to-seed table of the pass with seed t + 1 is formed inside the
// draw kernel when it is small ((t + 1) * d <= kPPTableInline), else by its
// own kernel.
constexpr int64_t kPPTableInline = 4096;

int pp_launches(int k, int d, bool prune) {
    if (k == 1) return 2;
    int n = 3 + 3 * (k - 1) - 1;   // set-up, first pass, weights; per draw: select, pass, weights (not after the last)
    if (prune)
        for (int t = 0; t + 1 < k; ++t) n += (int64_t)(t + 1) * d > kPPTableInline;
    return n;
}

hipError_t launch_pp_seed(const PPArgs& P, int64_t i0, int vw, hipEvent_t* ev, int8_t* kind, hipStream_t s) {
    hipError_t e;
    int j = 0;
    // kind of the launch just enqueued: 0 first pass, 1 later pass, 2 other
    auto mark = [&](int8_t kd) {
        if (!ev) return hipSuccess;
        if (j > 0) kind[j - 1] = kd;
        return hipEventRecord(ev[j++], s);
    };
    if ((e = mark(2)) != hipSuccess) return e;
    hipLaunchKernelGGL(k_pp_init, dim3(1), dim3(256), 0, s, P, i0);
    if ((e = hipGetLastError()) != hipSuccess || (e = mark(2)) != hipSuccess) return e;
    e = P.prune ? step_vec<true, true>(P, 0, vw, s) : step_vec<true, false>(P, 0, vw, s);
    if (e != hipSuccess || (e = mark(0)) != hipSuccess) return e;
    if (P.k == 1) return hipSuccess;
    hipLaunchKernelGGL(k_pp_weights, dim3((unsigned)P.G), dim3(kPPThreads), 0, s, P, 0);
    if ((e = hipGetLastError()) != hipSuccess || (e = mark(2)) != hipSuccess) return e;
    int G = 1;   // lanes per earlier seed in k_pp_dcc
    while (G < 64 && 16 * G < P.d) G *= 2;
    for (int t = 0; t + 1 < P.k; ++t) {
        const bool own = P.prune && (int64_t)(t + 1) * P.d > kPPTableInline;
        hipLaunchKernelGGL(k_pp_select, dim3(1), dim3(kPPSelThreads), 0, s, P, t, (P.prune && !own) ? 1 : 0);
        if ((e = hipGetLastError()) != hipSuccess || (e = mark(2)) != hipSuccess) return e;
        if (own) {
            const int64_t thr = (int64_t)(t + 1) * G;
            hipLaunchKernelGGL(k_pp_dcc, dim3((unsigned)((thr + 255) / 256)), dim3(256), 0, s, P, t, G,
                               vw > 0 ? 1 : 0);
            if ((e = hipGetLastError()) != hipSuccess || (e = mark(2)) != hipSuccess) return e;
        }
        const int tn = t + 1;   // pass with the new seed, then the weights of the next draw
        e = P.prune ? step_vec<false, true>(P, tn, vw, s) : step_vec<false, false>(P, tn, vw, s);
        if (e != hipSuccess || (e = mark(1)) != hipSuccess) return e;
        if (tn + 1 < P.k) {
            hipLaunchKernelGGL(k_pp_weights, dim3((unsigned)P.G), dim3(kPPThreads), 0, s, P, tn);
            if ((e = hipGetLastError()) != hipSuccess || (e = mark(2)) != hipSuccess) return e;
        }
    }
    return hipSuccess;
}

}  // namespace km
