// k-means++ seeding (paper section IV-C: each new seed is a data point drawn
// with probability D(v)^2 / sum D(v)^2, D the distance to the nearest seed
// so far).  The caller supplies the uniform numbers, so a seeding is a pure
// function of (X, k, u) and is reproduced bit for bit by any implementation
// of the same arithmetic:
//   - D^2 of a row to a seed in float64, coordinate differences summed in
//     index order by fused multiply-add; one lane owns a row, so the order
//     is the sequential one;
//   - the draw uses integer weights w_i = floor(D2_i * 2^S) (exact sums in any
//     order; S from a bound of max D2 known before the pass, so the weights
//     are formed in the same pass that updates D2), T = floor(u * W) and the
//     smallest i whose inclusive prefix exceeds T.
//
// Kernels, per seed t (t = 0 first):
//   k_pp_step    one pass over the points: D2 = min(D2, ||x - c_t||^2) (all
//                points for t = 0), the block's weight sum for the next draw
//                and the block's max of D2 (atomic max into a per-step slot);
//                with pruning a point is skipped when its nearest seed a is
//                at least twice as far from c_t as the point (triangle
//                inequality, Elkan's lemma; margins cover the float64
//                rounding, so D2 is unchanged by construction);
//   k_pp_weights the weight sums of the first draw (its scale needs the max
//                of the first pass);
//   k_pp_select  one workgroup: scans the block sums, finds the block and
//                then the point of the draw, writes the seed index and row,
//                and the distances from the new seed to the earlier seeds
//                (the pruning table of the next pass).
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

// ||x - c||^2 in float64, index order, fused (the oracle's definition).
template <bool VEC4>
__device__ __forceinline__ double dist2_seq(const float* __restrict__ x, const float* __restrict__ c, int d) {
    double acc = 0.0;
    if (VEC4) {
        for (int m = 0; m < d; m += 4) {
            const f32x4 xv = *reinterpret_cast<const f32x4*>(x + m);
            const f32x4 cv = *reinterpret_cast<const f32x4*>(c + m);
            double df = (double)xv.x - (double)cv.x;
            acc = fma(df, df, acc);
            df = (double)xv.y - (double)cv.y;
            acc = fma(df, df, acc);
            df = (double)xv.z - (double)cv.z;
            acc = fma(df, df, acc);
            df = (double)xv.w - (double)cv.w;
            acc = fma(df, df, acc);
        }
    } else {
        for (int m = 0; m < d; ++m) {
            const double df = (double)x[m] - (double)c[m];
            acc = fma(df, df, acc);
        }
    }
    return acc;
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

// One pass with seed t.  FIRST: D2 starts as the distance to seed 0.
// WEIGHTS: block sums of the next draw's weights with the scale from
// Mb[s_slot].  PRUNE: skip test against the seed-to-seed table.
template <bool FIRST, bool WEIGHTS, bool PRUNE, bool VEC4>
__global__ __launch_bounds__(kPPThreads) void k_pp_step(PPArgs P, int t, int s_slot) {
    __shared__ uint64_t red[3][kPPThreads / 64];
    const int tid = threadIdx.x;
    const int64_t base = (int64_t)blockIdx.x * kPPChunk;
    const int d = P.d;
    const float* __restrict__ c = P.C + (int64_t)t * d;
    const int S = WEIGHTS ? weight_scale(__longlong_as_double((long long)P.Mb[s_slot]), P.L) : 0;
    uint64_t wsum = 0, dmax = 0, ncomp = 0;
#pragma unroll
    for (int q = 0; q < kPPPer; ++q) {
        const int64_t i = base + q * kPPThreads + tid;
        if (i < P.n) {
            const float* __restrict__ x = P.X + i * d;
            double D;
            if (FIRST) {
                D = dist2_seq<VEC4>(x, c, d);
                P.D2[i] = D;
                if (PRUNE) P.A[i] = 0;
                ++ncomp;
            } else {
                D = P.D2[i];
                bool skip = false;
                if (PRUNE) skip = P.dcc[P.A[i]] >= 4.0 * D * (1.0 + 0x1p-26);
                if (!skip) {
                    const double v = dist2_seq<VEC4>(x, c, d);
                    ++ncomp;
                    if (v < D) {
                        D = v;
                        P.D2[i] = v;
                        if (PRUNE) P.A[i] = t;
                    }
                }
            }
            const uint64_t db = (uint64_t)__double_as_longlong(D);   // D >= 0: bits order as values
            dmax = db > dmax ? db : dmax;
            if (WEIGHTS) wsum += weight_of(D, S);
        }
    }
    const int lane = tid & 63, w = tid >> 6;
    wsum = wave_sum_u64(wsum);
    dmax = wave_max_u64(dmax);
    ncomp = wave_sum_u64(ncomp);
    if (lane == 0) {
        red[0][w] = wsum;
        red[1][w] = dmax;
        red[2][w] = ncomp;
    }
    __syncthreads();
    if (tid == 0) {
        uint64_t a = 0, b = 0, cc = 0;
#pragma unroll
        for (int j = 0; j < kPPThreads / 64; ++j) {
            a += red[0][j];
            b = red[1][j] > b ? red[1][j] : b;
            cc += red[2][j];
        }
        if (WEIGHTS) P.bs[blockIdx.x] = a;
        atomicMax(reinterpret_cast<unsigned long long*>(P.Mb + t), (unsigned long long)b);
        if (P.cnt) atomicAdd(reinterpret_cast<unsigned long long*>(P.cnt + t), (unsigned long long)cc);
    }
}

// Weight sums of the first draw (scale from the max of the first pass).
__global__ __launch_bounds__(kPPThreads) void k_pp_weights(PPArgs P) {
    __shared__ uint64_t red[kPPThreads / 64];
    const int tid = threadIdx.x;
    const int64_t base = (int64_t)blockIdx.x * kPPChunk;
    const int S = weight_scale(__longlong_as_double((long long)P.Mb[0]), P.L);
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
        if (P.cnt) P.cnt[j] = 0;
    }
}

// Draw of seed t + 1 from the weights after the pass with seed t.
__global__ __launch_bounds__(kPPSelThreads) void k_pp_select(PPArgs P, int t, int s_slot) {
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
            const int S = weight_scale(__longlong_as_double((long long)P.Mb[s_slot]), P.L);
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
    if (!P.prune) return;
    // Seed-to-seed table for the next pass: a lower bound of
    // ||c_a - c_{t+1}||^2 for a <= t (any summation order, margin 2^-28).
    if (d <= 64) {
        for (int a = tid; a <= t; a += kPPSelThreads) {
            const float* ca = P.C + (int64_t)a * d;
            double acc = 0.0;
            for (int m = 0; m < d; ++m) {
                const double df = (double)ca[m] - (double)xp[m];
                acc = fma(df, df, acc);
            }
            P.dcc[a] = acc * (1.0 - 0x1p-28);
        }
    } else {
        const int lane = tid & 63;
        for (int a = tid >> 6; a <= t; a += kPPSelThreads / 64) {
            const float* ca = P.C + (int64_t)a * d;
            double acc = 0.0;
            for (int m = lane; m < d; m += 64) {
                const double df = (double)ca[m] - (double)xp[m];
                acc = fma(df, df, acc);
            }
#pragma unroll
            for (int off = 32; off > 0; off >>= 1) acc += __shfl_xor(acc, off);
            if (lane == 0) P.dcc[a] = acc * (1.0 - 0x1p-28);
        }
    }
}

template <bool FIRST, bool WEIGHTS, bool PRUNE>
hipError_t step_vec(const PPArgs& P, int t, int s_slot, bool vec4, hipStream_t s) {
    const dim3 grid((unsigned)P.G), block(kPPThreads);
    if (vec4)
        hipLaunchKernelGGL((k_pp_step<FIRST, WEIGHTS, PRUNE, true>), grid, block, 0, s, P, t, s_slot);
    else
        hipLaunchKernelGGL((k_pp_step<FIRST, WEIGHTS, PRUNE, false>), grid, block, 0, s, P, t, s_slot);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_pp_seed(const PPArgs& P, int64_t i0, bool vec4, hipStream_t s) {
    hipError_t e;
    hipLaunchKernelGGL(k_pp_init, dim3(1), dim3(256), 0, s, P, i0);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    e = P.prune ? step_vec<true, false, true>(P, 0, 0, vec4, s) : step_vec<true, false, false>(P, 0, 0, vec4, s);
    if (e != hipSuccess) return e;
    if (P.k == 1) return hipSuccess;
    hipLaunchKernelGGL(k_pp_weights, dim3((unsigned)P.G), dim3(kPPThreads), 0, s, P);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    for (int t = 0; t + 1 < P.k; ++t) {
        hipLaunchKernelGGL(k_pp_select, dim3(1), dim3(kPPSelThreads), 0, s, P, t, t == 0 ? 0 : t - 1);
        if ((e = hipGetLastError()) != hipSuccess) return e;
        const int tn = t + 1;   // pass with the new seed; its weights serve the next draw
        const bool weights = tn + 1 < P.k;
        if (P.prune)
            e = weights ? step_vec<false, true, true>(P, tn, tn - 1, vec4, s)
                        : step_vec<false, false, true>(P, tn, 0, vec4, s);
        else
            e = weights ? step_vec<false, true, false>(P, tn, tn - 1, vec4, s)
                        : step_vec<false, false, false>(P, tn, 0, vec4, s);
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

}  // namespace km
