// Wavefront-level helpers shared by the matrix-core attention kernels:
// operand vector types, cross-lane reductions on VALU permute paths (DPP
// inside a 16-lane row, permlane16/32 swaps across rows, no LDS traffic),
// and global-to-LDS copies.  Not part of the public ABI.
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
// Minimum / maximum without the NaN canonicalisation the compiler adds around
// fminf / fmaxf (for values that are never NaN, or where a NaN's result does
// not matter).
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
__device__ __forceinline__ float fmin2(float a, float b) {
    float r;
    asm("v_min_f32 %0, %1, %2" : "=v"(r) : "v"(a), "v"(b));
    return r;
}
__device__ __forceinline__ float fmin3(float a, float b, float c) {
    float r;
    asm("v_min3_f32 %0, %1, %2, %3" : "=v"(r) : "v"(a), "v"(b), "v"(c));
    return r;
}
__device__ __forceinline__ float row16_min(float v) {  // over the 16 lanes of a row
    v = fmin2(v, dpp<0xB1>(v));
    v = fmin2(v, dpp<0x4E>(v));
    v = fmin2(v, dpp<0x141>(v));
    return fmin2(v, dpp<0x140>(v));
}
__device__ __forceinline__ float min_kg(float v) {  // over lanes l, l^16, l^32, l^48
    auto r = __builtin_amdgcn_permlane16_swap(__float_as_int(v), __float_as_int(v), false, false);
    v = fmin2(__int_as_float(r[0]), __int_as_float(r[1]));
    r = __builtin_amdgcn_permlane32_swap(__float_as_int(v), __float_as_int(v), false, false);
    return fmin2(__int_as_float(r[0]), __int_as_float(r[1]));
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

// ---- Buffer accesses with a cache policy ----
// A buffer resource over [base, base + bytes): an access at an offset past the
// end reads 0 and writes nothing.  `base` and `bytes` must be uniform.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t buffer_rsrc(const void *base, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), 0, (int)bytes, 0x00020000);
}
// Cache-policy bits of the buffer builtins: sc1 makes an access coherent
// across the XCDs' L2 caches (agent scope): stores write through, loads do
// not return another XCD's stale copy.
constexpr int kAgentCoherent = 16;
__device__ __forceinline__ void store16_agent(__amdgpu_buffer_rsrc_t r, uint32_t off, float4 v) {
    __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4_t, v), r, (int)off, 0, kAgentCoherent);
}
__device__ __forceinline__ void store8_agent(__amdgpu_buffer_rsrc_t r, uint32_t off, float2 v) {
    __builtin_amdgcn_raw_buffer_store_b64(__builtin_bit_cast(intx2_t, v), r, (int)off, 0, kAgentCoherent);
}
__device__ __forceinline__ float4 load16_agent(__amdgpu_buffer_rsrc_t r, uint32_t off) {
    return __builtin_bit_cast(float4, __builtin_amdgcn_raw_buffer_load_b128(r, (int)off, 0, kAgentCoherent));
}
__device__ __forceinline__ float2 load8_agent(__amdgpu_buffer_rsrc_t r, uint32_t off) {
    return __builtin_bit_cast(float2, __builtin_amdgcn_raw_buffer_load_b64(r, (int)off, 0, kAgentCoherent));
}

// ---- Global-to-LDS copies (global_load_lds), issued as inline assembly ----
// The 16-byte copies carry the nontemporal hint: the attention kernels read
// each K/V byte once (32K decode 16.9 -> 15.8-16.2 us, 128K verification
// 67.8 -> 63.1-63.4 us, paged batch decode 156.7 -> 146-149 us).
// One instruction moves 16 (or 4) bytes per lane from each lane's global
// address into LDS at M0 + 16 * lane (4 * lane): a wavefront fills one
// contiguous 1 KB (256 B) LDS run, and the lanes' global addresses choose
// which source chunk lands where.  The copies count in vmcnt like loads, in
// issue order.  They are written as assembly so that the compiler, which
// cannot tell which LDS bytes they fill, does not drain every copy in flight
// before each LDS read: a kernel using them waits explicitly with
// wait_vmcnt<N>() before reading the bytes, keeps its own global loads out
// of the stretches where copies are in flight (their compiler-placed waits
// would also drain the copies), and waits for vmcnt(0) before reusing the
// LDS for anything else or exiting.

// LDS byte address of a __shared__ object (low 32 bits of its flat address).
__device__ __forceinline__ uint32_t lds_addr(const void *p) { return (uint32_t)(uintptr_t)p; }

// The LDS address (and a base address) must be the same in every lane; they
// are read from the first lane, since the compiler cannot always prove it.
__device__ __forceinline__ uint32_t uniform(uint32_t v) { return __builtin_amdgcn_readfirstlane(v); }
__device__ __forceinline__ const void *uniform(const void *p) {
    const uint64_t v = (uint64_t)(uintptr_t)p;
    return (const void *)(uintptr_t)(((uint64_t)uniform((uint32_t)(v >> 32)) << 32) | uniform((uint32_t)v));
}
// The global-to-LDS copies take their LDS address in M0, which they set
// themselves and list as clobbered, so the compiler never assumes a value of
// its own survives them (it re-initialises M0 before any use and inserts the
// hazard waits).  M0 is a reserved register to the compiler, which warns that
// such a clobber is not preserved: that is the intent, and the warning is
// silenced for these three functions only.
#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
// 16 bytes per lane from sbase + voff (sbase uniform) to LDS at lds + 16 lane.
__device__ __forceinline__ void lds_copy16(const void *sbase, uint32_t voff, uint32_t lds) {
    asm volatile("s_mov_b32 m0, %2\n\tglobal_load_lds_dwordx4 %0, %1 nt" ::"v"(voff), "s"(uniform(sbase)),
                 "s"(uniform(lds))
                 : "memory", "m0");
}
// 16 bytes per lane from the lane's own address.
__device__ __forceinline__ void lds_copy16(const void *addr, uint32_t lds) {
    asm volatile("s_mov_b32 m0, %1\n\tglobal_load_lds_dwordx4 %0, off nt" ::"v"(addr), "s"(uniform(lds))
                 : "memory", "m0");
}
// 4 bytes per lane from the lane's own address to LDS at lds + 4 lane.
__device__ __forceinline__ void lds_copy4(const void *addr, uint32_t lds) {
    asm volatile("s_mov_b32 m0, %1\n\tglobal_load_lds_dword %0, off" ::"v"(addr), "s"(uniform(lds))
                 : "memory", "m0");
}
#pragma clang diagnostic pop
// Wait until at most N vector-memory operations of this wavefront are in flight.
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
    static_assert(N >= 0 && N < 64, "vmcnt range");
    asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}
// The same for a count the compiler folds to a constant (an unrolled loop's
// arithmetic); a count above 31 waits for all.
__device__ __forceinline__ void wait_vmcnt_folded(int n) {
    switch (n) {
#define LYNX_WAIT_CASE(N) \
    case N:               \
        wait_vmcnt<N>();  \
        break;
        LYNX_WAIT_CASE(1) LYNX_WAIT_CASE(2) LYNX_WAIT_CASE(3) LYNX_WAIT_CASE(4) LYNX_WAIT_CASE(5)
        LYNX_WAIT_CASE(6) LYNX_WAIT_CASE(7) LYNX_WAIT_CASE(8) LYNX_WAIT_CASE(9) LYNX_WAIT_CASE(10)
        LYNX_WAIT_CASE(11) LYNX_WAIT_CASE(12) LYNX_WAIT_CASE(13) LYNX_WAIT_CASE(14) LYNX_WAIT_CASE(15)
        LYNX_WAIT_CASE(16) LYNX_WAIT_CASE(17) LYNX_WAIT_CASE(18) LYNX_WAIT_CASE(19) LYNX_WAIT_CASE(20)
        LYNX_WAIT_CASE(21) LYNX_WAIT_CASE(22) LYNX_WAIT_CASE(23) LYNX_WAIT_CASE(24) LYNX_WAIT_CASE(25)
        LYNX_WAIT_CASE(26) LYNX_WAIT_CASE(27) LYNX_WAIT_CASE(28) LYNX_WAIT_CASE(29) LYNX_WAIT_CASE(30)
        LYNX_WAIT_CASE(31)
#undef LYNX_WAIT_CASE
    default:
        wait_vmcnt<0>();
        break;
    }
}

}  // namespace lynx
