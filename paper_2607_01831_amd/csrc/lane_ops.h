// Wavefront-level helpers shared by the matrix-core attention kernels:
// operand vector types and cross-lane reductions on VALU permute paths (DPP
// inside a 16-lane row, permlane16/32 swaps across rows), no LDS traffic.
// Not part of the public ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace lynx {

typedef __attribute__((__vector_size__(4 * sizeof(float)))) float f32x4_t;
typedef __attribute__((__vector_size__(4 * sizeof(uint32_t)))) uint32_t u32x4_t;
typedef __attribute__((__vector_size__(2 * sizeof(int)))) int intx2_t;

template <int CTRL>
__device__ __forceinline__ float dpp(float v) {
    return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), CTRL, 0xF, 0xF, false));
}
__device__ __forceinline__ float row16_sum(float v) {  // over the 16 lanes of a row
    v += dpp<0xB1>(v);   // quad_perm [1,0,3,2]
    v += dpp<0x4E>(v);   // quad_perm [2,3,0,1]
    v += dpp<0x141>(v);  // row_half_mirror
    return v + dpp<0x140>(v);  // row_mirror
}
// Over lanes l, l^16, l^32, l^48 (the four rows of one column).
__device__ __forceinline__ float sum_kg(float v) {
    auto r = __builtin_amdgcn_permlane16_swap(__float_as_int(v), __float_as_int(v), false, false);
    v = __int_as_float(r[0]) + __int_as_float(r[1]);
    r = __builtin_amdgcn_permlane32_swap(__float_as_int(v), __float_as_int(v), false, false);
    return __int_as_float(r[0]) + __int_as_float(r[1]);
}
// Maximum of values that are finite or -inf (never NaN), without the NaN
// canonicalisation the compiler adds around fmaxf.
__device__ __forceinline__ float fmax2(float a, float b) {
    float r;
    asm("v_max_f32 %0, %1, %2" : "=v"(r) : "v"(a), "v"(b));
    return r;
}
__device__ __forceinline__ float fmax3(float a, float b, float c) {
    float r;
    asm("v_max3_f32 %0, %1, %2, %3" : "=v"(r) : "v"(a), "v"(b), "v"(c));
    return r;
}
__device__ __forceinline__ float row16_max(float v) {  // over the 16 lanes of a row
    v = fmax2(v, dpp<0xB1>(v));
    v = fmax2(v, dpp<0x4E>(v));
    v = fmax2(v, dpp<0x141>(v));
    return fmax2(v, dpp<0x140>(v));
}
__device__ __forceinline__ float max_kg(float v) {
    auto r = __builtin_amdgcn_permlane16_swap(__float_as_int(v), __float_as_int(v), false, false);
    v = fmax2(__int_as_float(r[0]), __int_as_float(r[1]));
    r = __builtin_amdgcn_permlane32_swap(__float_as_int(v), __float_as_int(v), false, false);
    return fmax2(__int_as_float(r[0]), __int_as_float(r[1]));
}

}  // namespace lynx
