// lanes.h -- cross-lane sums of a 64-wide wavefront on gfx950, on the VALU
// (DPP row operations and the permlane swaps), with no LDS round trips.
#pragma once

#include <hip/hip_runtime.h>

namespace mlp {

typedef float f4 __attribute__((ext_vector_type(4)));

// Cross-lane sums on the VALU (DPP and lane-swap instructions, no LDS round
// trips). Each pairs lanes symmetrically, so both lanes of a pair compute the
// same sum bitwise (a + b == b + a): every lane of a group ends with the same
// total, summed in a fixed order.
template <int CTRL>
__device__ __forceinline__ float dppf(float v) {
    return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), CTRL, 0xF, 0xF, false));
}
// v + (v of lane l ^ 8), within each row of 16 lanes (row_ror:8)
__device__ __forceinline__ float xadd8(float v) { return v + dppf<0x128>(v); }
// v + (v of lane l ^ 16)
__device__ __forceinline__ float xadd16(float v) {
    const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}
// v + (v of lane l ^ 32)
__device__ __forceinline__ float xadd32(float v) {
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}
// sum over each row of 16 lanes, in every lane of the row: pairs (i, i^8),
// (i, 7-i within 8), (i, i^2), (i, i^1)
__device__ __forceinline__ float rsum16(float v) {
    v += dppf<0x128>(v);   // row_ror:8
    v += dppf<0x141>(v);   // row_half_mirror
    v += dppf<0x4E>(v);    // quad_perm [2,3,0,1]
    v += dppf<0xB1>(v);    // quad_perm [1,0,3,2]
    return v;
}
__device__ __forceinline__ float sum64(float v) { return xadd32(xadd16(rsum16(v))); }
// Row sums of four values per lane over each row of 16 lanes, by a transposing
// butterfly: the lane pairs of rsum16 (li ^ 8, 7 - li within 8, li ^ 2, li ^ 1),
// but each exchange hands over only the values the partner keeps. Lane li ends
// with the sum of y[li >> 2] over its row (the same in the four lanes li >> 2
// share).
__device__ __forceinline__ float rsum16x4(const float (&y)[4], int li) {
    const bool b3 = (li & 8) != 0, b2 = (li & 4) != 0;
    const float k0 = b3 ? y[2] : y[0], k1 = b3 ? y[3] : y[1];   // kept
    const float g0 = b3 ? y[0] : y[2], g1 = b3 ? y[1] : y[3];   // handed over
    const float t0 = k0 + dppf<0x128>(g0);                       // row_ror:8
    const float t1 = k1 + dppf<0x128>(g1);
    const float kk = b2 ? t1 : t0, gg = b2 ? t0 : t1;
    float r = kk + dppf<0x141>(gg);                              // row_half_mirror
    r += dppf<0x4E>(r);                                          // lanes li, li ^ 2
    r += dppf<0xB1>(r);                                          // lanes li, li ^ 1
    return r;
}

}  // namespace mlp
