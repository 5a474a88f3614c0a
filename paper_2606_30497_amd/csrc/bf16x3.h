// bf16x3.h -- fp32 products on the bf16 matrix cores: three-part bf16 splits
// of fp32 values and the bf16 MFMA that multiplies them (deep.hip, forward.hip).
//
// A value x splits exactly into x0 + x1 + x2, each part the bf16 rounding (to
// nearest even) of what the earlier parts leave; |x1| <= 2^-8 (1 + 2^-8) |x|,
// |x2| <= 2^-16 |x|. A product a b is then the sum of the six part products
// a_i b_j with i + j <= 2, each exact in fp32; the three dropped ones are at
// most 2.01 u |a b| together (u = 2^-24). An operand within 2^-8 of the fp32
// maximum rounds to infinity in its first part, and its products become NaN.
#pragma once

#include <hip/hip_runtime.h>

#include <stdint.h>

#include "lanes.h"

namespace mlp {

typedef uint32_t u2v __attribute__((ext_vector_type(2)));
typedef uint32_t u4v __attribute__((ext_vector_type(4)));
typedef float f2v __attribute__((ext_vector_type(2)));
typedef __bf16 bf2v __attribute__((ext_vector_type(2)));
typedef __bf16 bf8v __attribute__((ext_vector_type(8)));

// bf16 roundings (to nearest even) of a and b, packed (a in the low half)
__device__ __forceinline__ uint32_t bf16_pair(float a, float b) {
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(f2v{a, b}, bf2v));
}

// The three bf16 parts of a and of b, part i of both in word i (a in the low
// half): part 0 rounds the value, part 1 what part 0 leaves, part 2 what parts
// 0 and 1 leave; every difference is exact in fp32, and the last remainder has
// at most eight significant bits, so the parts sum to the value exactly.
__device__ __forceinline__ void split_pair(float a, float b, uint32_t (&w)[3]) {
#pragma unroll
    for (int i = 0; i < 3; ++i) {
        w[i] = bf16_pair(a, b);
        a -= __uint_as_float(w[i] << 16);
        b -= __uint_as_float(w[i] & 0xFFFF0000u);
    }
}

__device__ __forceinline__ f4 mfma_bf16(u4v a, u4v b, f4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf8v, a),
                                                   __builtin_bit_cast(bf8v, b), c, 0, 0, 0);
}

}  // namespace mlp
