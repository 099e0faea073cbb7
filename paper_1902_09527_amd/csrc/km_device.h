// Device helpers shared by the kernel translation units (km_kernels.hip,
// km_large.hip): directed float32 rounding of float64 values, the upper
// bound of a distance from a float32 squared distance, and the exact
// fixed-point image of a coordinate.
#pragma once

#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include "km_internal.h"

namespace km {

constexpr float kUp = 1.0f + 0x1p-22f;   // covers one float32 rounding, upward

typedef float f32x4 __attribute__((ext_vector_type(4)));    // native 16-byte vector
typedef float f32x16 __attribute__((ext_vector_type(16)));  // 32x32 MFMA accumulator slice

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

__device__ inline uint64_t wave_sum_u64(uint64_t v) {
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off);
    return v;
}

}  // namespace km
