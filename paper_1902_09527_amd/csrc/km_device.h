// Device helpers shared by the kernel translation units: directed float32
// rounding of float64 values, the upper bound of a distance from a float32
// squared distance, the split-bf16 operands of the matrix-core distances,
// and the exact fixed-point image of a coordinate.
#pragma once

#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include "km_internal.h"

namespace km {

constexpr float kUp = 1.0f + 0x1p-22f;   // covers one float32 rounding, upward

typedef float f32x4 __attribute__((ext_vector_type(4)));    // native 16-byte vector
typedef float f32x16 __attribute__((ext_vector_type(16)));  // 32x32 MFMA accumulator slice
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));    // a bf16 matrix-core operand (16 bytes)

// Split operands of two float32 values: hi = bf16(x) (rounded to nearest),
// returned packed, and the residuals x - hi (exact in float32); split_lo
// packs bf16 of the two residuals.  x.c is then formed as hi.hi + hi.lo +
// lo.hi on the bf16 matrix cores.
__device__ __forceinline__ uint32_t split_hi(float a, float b, float& ra, float& rb) {
    const f32x2 v = {a, b};
    const uint32_t h = __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2));
    ra = a - __uint_as_float(h << 16);
    rb = b - __uint_as_float(h & 0xffff0000u);
    return h;
}

__device__ __forceinline__ uint32_t split_lo(float a, float b) {
    const f32x2 v = {a, b};
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2));
}

// Largest float <= v and smallest float >= v.
__device__ inline float f32_down(double v) {
    float r = (float)v;
    if ((double)r > v) r = nextafterf(r, -INFINITY);
    return r;
}
__device__ inline float f32_up(double v) {
    float r = (float)v;
    if ((double)r < v) r = nextafterf(r, INFINITY);
    return r;
}

// Upper bound on the exact distance to the float64 centroid from a float32
// squared distance D (relative error <= gamma) and the centroid's float32
// rounding error ec.
__device__ inline float upper_bound(float D, float ec, float gamma) {
    return (sqrtf(D) * (1.0f + gamma) + ec) * kUp;
}

// Exact integer image of v * scale (|v * scale| < 2^51), offset by kMagicBits.
__device__ inline uint64_t fixed_bits(double v, double scale) {
    return (uint64_t)__double_as_longlong(fma(v, scale, kMagic));
}

// Set-up magnitude words (uint32 float bits of non-negative values): the
// largest |x| over all of X (written by the first step itself when that step
// is the first to read X), whether X or C0 holds a non-finite value, the
// largest |c| of C0, a zero C0 row (spherical k-means), and the largest |x|
// over a fixed sample of X.
constexpr int kAmaxX = 0, kAmaxXBad = 1, kAmaxC = 2, kAmaxCBad = 3, kAmaxZeroRow = 4, kAmaxSample = 5;

// The e with v <= 2^e (frexp's exponent; 0 for v = 0).
__device__ inline int bound_exp(double v) {
    int e = 0;
    if (v > 0.0) (void)frexp(v, &e);
    return e;
}

// Exponent of the bound on |x| that the exact sums are scaled for: 16 times
// the sample's bound, unless X exceeds it.  A fixed sample and margin make
// it known before X is read in nearly every case.
__device__ inline int sum_exp(const uint32_t* amax) {
    const int es = bound_exp((double)__uint_as_float(amax[kAmaxSample])) + 4;
    const int ex = bound_exp((double)__uint_as_float(amax[kAmaxX]));
    return ex <= es ? es : ex;
}

// Shift S of the coordinate sums for |x| <= 2^ex and n points:
// |x 2^S| <= 2^50 per value and n 2^ex 2^S <= 2^61 overall, so every image
// is exact and no sum can overflow.
__device__ inline int sum_shift(int ex, int64_t n) {
    int lgn = 0;
    while (lgn < 64 && (1ull << lgn) < (uint64_t)n) ++lgn;
    const int S = 61 - lgn - ex;
    return S < 50 - ex ? S : 50 - ex;
}

// The scales for |x| <= 2^ex and |c| <= cmax: coordinate sums as above,
// inertia the same for squared distances up to d (2 max(2^ex, cmax))^2.
__device__ inline void put_scales(IterState* st, int ex, float cmax, int64_t n, int32_t d) {
    const int S = sum_shift(ex, n);
    const double xb = ldexp(1.0, ex);
    const double am = xb > (double)cmax ? xb : (double)cmax;
    const int SI = sum_shift(bound_exp((double)d * 4.0 * am * am), n);
    st->qscale = ldexp(1.0, S);
    st->qinv = ldexp(1.0, -S);
    st->iscale = ldexp(1.0, SI);
    st->iinv = ldexp(1.0, -SI);
}

// x subtracted from a 64-bit word in LDS, modulo 2^64 (one LDS subtract: no
// negation of x first).
__device__ __forceinline__ void lds_sub64(uint64_t* p, uint64_t x) {
    __hip_atomic_fetch_sub(p, x, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
}

// The end of step t (one thread): the progress word of a run's host loop, if
// any, becomes t + 1, negated when the run stops (a system-scope store to
// pinned host memory).
__device__ inline void report_step(const IterState* st, int t, bool done) {
    if (st->host) __hip_atomic_store(st->host, done ? -(t + 1) : t + 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
}

// The kernel's Dev with the fixed-point scales the set-up kernel left in the
// loop state (the host does not wait for them).
__device__ inline Dev with_scales(Dev P) {
    const IterState* st = P.st;
    P.qscale = st->qscale;
    P.qinv = st->qinv;
    P.iscale = st->iscale;
    P.iinv = st->iinv;
    return P;
}

// Squared float32 distance (direct-difference form, coordinates in order) of
// two rows, compile-time D (16-byte aligned rows).
template <int D>
__device__ inline float sqd_lds_fixed(const float* x, const float* c) {
    float acc = 0.f;
#pragma unroll
    for (int m = 0; m < D; m += 4) {
        const float4 xv = *reinterpret_cast<const float4*>(x + m);
        const float4 cv = *reinterpret_cast<const float4*>(c + m);
        float t0 = xv.x - cv.x, t1 = xv.y - cv.y, t2 = xv.z - cv.z, t3 = xv.w - cv.w;
        acc = fmaf(t0, t0, acc);
        acc = fmaf(t1, t1, acc);
        acc = fmaf(t2, t2, acc);
        acc = fmaf(t3, t3, acc);
    }
    return acc;
}

// Squared float64 distance (direct-difference form) of a float row to a
// float64 centroid row.
__device__ inline double sqd64(const float* x, const double* c, int d) {
    double acc = 0.0;
    for (int m = 0; m < d; ++m) {
        double t = (double)x[m] - c[m];
        acc = fma(t, t, acc);
    }
    return acc;
}

// Clause-1 threshold on a bound kept relative to the cumulative drift: when
// Clause 1 holds for v + D_a <= s(a) (D_a rounded up, s(a) rounded down), thr
// is the largest float with thr + D_a <= s(a), so that the test is v <= thr
// (+inf when k = 1).
__device__ inline float clause1_thr(float s, double dhi) {
    const double x = (double)s - dhi;
    return isinf(x) ? (float)x : f32_down(x - fabs(x) * 0x1p-50);
}

// Set bits of a wave mask below the calling lane.
__device__ inline int lanes_below(uint64_t m) {
    return (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
}

__device__ inline uint64_t wave_sum_u64(uint64_t v) {
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off);
    return v;
}

}  // namespace km
