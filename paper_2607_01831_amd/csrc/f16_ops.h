// fp16 matrix-core operands over 8-bit codes (gfx950): shared by the
// verification kernel and the anchor decode over split-width anchors.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "lane_ops.h"
#include "lynx_internal.h"

namespace lynx {

typedef _Float16 f16x8_t __attribute__((ext_vector_type(8)));

__device__ __forceinline__ f32x4_t mfma_f16(u32x4_t a, u32x4_t b, f32x4_t c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(f16x8_t, a),
                                                 __builtin_bit_cast(f16x8_t, b), c, 0, 0, 0);
}

// Eight code bytes (two words, byte e = element e) -> eight fp16 values
// 1024 + c in element order.
__device__ __forceinline__ u32x4_t codes_to_f16(uint32_t w0, uint32_t w1) {
    const uint32_t c = 0x64646464u;
    u32x4_t r;
    r[0] = __builtin_amdgcn_perm(c, w0, 0x04010400u);
    r[1] = __builtin_amdgcn_perm(c, w0, 0x04030402u);
    r[2] = __builtin_amdgcn_perm(c, w1, 0x04010400u);
    r[3] = __builtin_amdgcn_perm(c, w1, 0x04030402u);
    return r;
}

// Two floats -> two fp16 in one word, a in the low half.  pack_f16 rounds
// toward zero (the split of bounded query values into hi + lo);
// pack_f16_rne rounds to nearest and overflows to infinity, so a softmax
// weight too large for fp16 cannot saturate unnoticed.
__device__ __forceinline__ uint32_t pack_f16(float a, float b) {
    return __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_pkrtz(a, b));
}
typedef float f32x2_t __attribute__((ext_vector_type(2)));
typedef _Float16 f16x2_t __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint32_t pack_f16_rne(float a, float b) {
    return __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2_t){a, b}, f16x2_t));
}
__device__ __forceinline__ float f16_lo(uint32_t w) {
    return (float)__builtin_bit_cast(_Float16, (uint16_t)(w & 0xffffu));
}
__device__ __forceinline__ float f16_hi(uint32_t w) {
    return (float)__builtin_bit_cast(_Float16, (uint16_t)(w >> 16));
}
__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// Byte offset of 16-byte chunk q of V-tile row t (rows of 128 code bytes) in
// an LDS tile.  The XOR swizzle spreads the 8 rows one transposed read
// (ds_read_b64_tr_b8) touches over all 32 banks.
__device__ __forceinline__ uint32_t v_slot(int t, int q) {
    const int sw = (t & 7) ^ ((t >> 4) << 2);
    return (uint32_t)t * kCodeRow + (uint32_t)((q ^ sw) * 16);
}

}  // namespace lynx
