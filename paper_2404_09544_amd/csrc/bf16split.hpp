// fp32 values as three bf16 parts, for fp32-accurate products on the bf16
// matrix cores (the bf16x6 scheme of Henry, Tang and Heinecke, "Leveraging
// the bfloat16 artificial intelligence datatype for higher-precision
// computations", ARITH 2019).  x = x1 + x2 + x3 + e with |e| < 2^-23 |x|:
// x1 is the top 16 bits of x (truncation), x2 those of x - x1, x3 those of
// x - x1 - x2; both differences are exact in fp32.  A product a b then takes
// the six part products a1 b1, a1 b2, a2 b1, a1 b3, a3 b1, a2 b2; the three
// it drops are below 2^-30 |a b|.  Part products are exact in fp32.
#pragma once
#include <hip/hip_runtime.h>
#include <cstdint>

namespace gnnav {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

__device__ __forceinline__ uint32_t hi16_pair(uint32_t a, uint32_t b) { return (a >> 16) | (b & 0xffff0000u); }

// x[0..7] (consecutive k) -> the three parts as MFMA k-fragments
__device__ __forceinline__ void split3(const float (&x)[8], bf16x8 &p1, bf16x8 &p2, bf16x8 &p3) {
    typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
    u32x4 q1, q2, q3;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        const float x0 = x[2 * e], x1 = x[2 * e + 1];
        const uint32_t u0 = __float_as_uint(x0), u1 = __float_as_uint(x1);
        const float r0 = x0 - __uint_as_float(u0 & 0xffff0000u), r1 = x1 - __uint_as_float(u1 & 0xffff0000u);
        const uint32_t v0 = __float_as_uint(r0), v1 = __float_as_uint(r1);
        const float s0 = r0 - __uint_as_float(v0 & 0xffff0000u), s1 = r1 - __uint_as_float(v1 & 0xffff0000u);
        q1[e] = hi16_pair(u0, u1);
        q2[e] = hi16_pair(v0, v1);
        q3[e] = hi16_pair(__float_as_uint(s0), __float_as_uint(s1));
    }
    p1 = __builtin_bit_cast(bf16x8, q1);
    p2 = __builtin_bit_cast(bf16x8, q2);
    p3 = __builtin_bit_cast(bf16x8, q3);
}

// The three bf16 parts of one value (bit patterns).
__device__ __forceinline__ void split3_bits(float x, uint16_t &p1, uint16_t &p2, uint16_t &p3) {
    const uint32_t u = __float_as_uint(x);
    const float r = x - __uint_as_float(u & 0xffff0000u);
    const uint32_t v = __float_as_uint(r);
    const float t = r - __uint_as_float(v & 0xffff0000u);
    p1 = (uint16_t)(u >> 16);
    p2 = (uint16_t)(v >> 16);
    p3 = (uint16_t)(__float_as_uint(t) >> 16);
}

// acc += the six part products of a and b (smallest first)
typedef float f32x16_split __attribute__((ext_vector_type(16)));
__device__ __forceinline__ f32x16_split mfma_split6(const bf16x8 &a1, const bf16x8 &a2, const bf16x8 &a3,
                                                    const bf16x8 &b1, const bf16x8 &b2, const bf16x8 &b3,
                                                    f32x16_split c) {
    c = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a2, b2, c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a3, b1, c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a1, b3, c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a2, b1, c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a1, b2, c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a1, b1, c, 0, 0, 0);
    return c;
}

}  // namespace gnnav
