// Split-stream KV codec kernels for gfx950: encode (quantize, split, pack),
// merge (anchor + residual -> 8-bit codes), and the deserializer's scatter of
// transmission buffers into the pages (Sec. 4.2 Anchor and Residual phases).
//
// Encode follows the grouped linear quantization of Sec. 2.3 (zero = group
// minimum, scale = range / 255) and the split-stream construction of Alg. 1
// stage 4 (anchor = the 4 most significant bits, residual = the 4 least
// significant bits), packing two 4-bit values per byte as the Compression
// Kernel of Sec. 5 does.  Merge is the Residual phase of Sec. 4.2.
//
// The fp32 arithmetic that decides a code is spelled out operation by
// operation (sub, mul, round-half-even, clamp; one IEEE division per group)
// so that every code is the one the definition gives.
#include "lane_ops.h"
#include "lynx_internal.h"

#include <float.h>

namespace lynx {
namespace {

constexpr int kEncodeThreads = 256;

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// Eight BF16 values held in a uint4 -> floats.
__device__ __forceinline__ void unpack8(const uint4 &u, float *x) {
    x[0] = bf16_lo(u.x); x[1] = bf16_hi(u.x);
    x[2] = bf16_lo(u.y); x[3] = bf16_hi(u.y);
    x[4] = bf16_lo(u.z); x[5] = bf16_hi(u.z);
    x[6] = bf16_lo(u.w); x[7] = bf16_hi(u.w);
}

// Group statistics from the group's min and max: zero, scale, inverse range.
__device__ __forceinline__ void group_params(float mn, float mx, float &zero, float &scale,
                                             float &inv) {
    if (mn == 0.0f) mn = 0.0f;  // -0 -> +0
    if (mx == 0.0f) mx = 0.0f;
    const float range = mx - mn;
    const float r = 255.0f / range;  // correctly rounded IEEE division
    if (!(range > 0.0f) || !(range <= FLT_MAX) || !(r <= FLT_MAX)) {
        scale = 0.0f;
        inv = 0.0f;
    } else {
        scale = range / 255.0f;
        inv = r;
    }
    zero = mn;
}

// (Min / max and the cross-lane reductions come from lane_ops.h; non-finite
// inputs give unspecified codes.)

// Eight values -> eight codes clamp(rint((x - zero) * inv), 0, 255), then
// the anchor word (nibble j = code_j >> 4) and the residual word (nibble j =
// code_j & 15).  v_cvt_pk_u8_f32 rounds half to even and saturates to
// [0, 255] (NaN -> 0), which is exactly the clamp-of-rint of the definition.
__device__ __forceinline__ void quantize_split8(const float *x, const float *zero, const float *inv,
                                                uint32_t &anc, uint32_t &res) {
    uint32_t w[2] = {0u, 0u};
#pragma unroll
    for (int j = 0; j < 8; ++j) {
        const float y = (x[j] - zero[j]) * inv[j];
        w[j >> 2] = __builtin_amdgcn_cvt_pk_u8_f32(y, (uint32_t)(j & 3), w[j >> 2]);
    }
    // bytes (c0, c1, c2, c3) -> nibble pairs c0 | c1 << 4 in byte 0, c2 | c3 << 4 in byte 2
    const uint32_t a0 = (w[0] >> 4) & 0x0F0F0F0Fu, a1 = (w[1] >> 4) & 0x0F0F0F0Fu;
    const uint32_t r0 = w[0] & 0x0F0F0F0Fu, r1 = w[1] & 0x0F0F0F0Fu;
    anc = __builtin_amdgcn_perm(a1 | (a1 >> 4), a0 | (a0 >> 4), 0x06040200u);
    res = __builtin_amdgcn_perm(r1 | (r1 >> 4), r0 | (r0 >> 4), 0x06040200u);
}

typedef unsigned int u32v4 __attribute__((ext_vector_type(4)));

// Eight values -> eight codes (bytes 0..7 of the result), as quantize_split8.
__device__ __forceinline__ uint64_t quantize8(const float *x, const float *zero, const float *inv) {
    uint32_t w[2] = {0u, 0u};
#pragma unroll
    for (int j = 0; j < 8; ++j) {
        const float y = (x[j] - zero[j]) * inv[j];
        w[j >> 2] = __builtin_amdgcn_cvt_pk_u8_f32(y, (uint32_t)(j & 3), w[j >> 2]);
    }
    return (uint64_t)w[0] | ((uint64_t)w[1] << 32);
}

// Codes of 8 dims (8 m .. 8 m + 7) of one plane row, split A + (8 - A):
// the A-bit anchors and the R-bit residuals as little-endian bit strings
// (A and R bytes), stored at byte A m of the anchor row (16 A bytes) and
// R m of the residual row.  A = 4 is the nibble path of quantize_split8.
template <int A>
__device__ __forceinline__ void store_split(const float *x, const float *zero, const float *inv,
                                            uint8_t *anc, uint8_t *res, size_t row, int m) {
    if constexpr (A == 4) {
        uint32_t a, r;
        quantize_split8(x, zero, inv, a, r);
        __builtin_nontemporal_store(a, reinterpret_cast<uint32_t *>(anc + row * kNibbleRow + 4 * m));
        __builtin_nontemporal_store(r, reinterpret_cast<uint32_t *>(res + row * kNibbleRow + 4 * m));
    } else {
        constexpr int R = 8 - A;
        const uint64_t c = quantize8(x, zero, inv);
        uint64_t an = 0, rs = 0;
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            const uint64_t cj = (c >> (8 * j)) & 0xFFu;
            an |= (cj >> R) << (A * j);
            rs |= (cj & ((1u << R) - 1u)) << (R * j);
        }
        uint16_t *ap = reinterpret_cast<uint16_t *>(anc + row * (16 * A) + A * m);
        uint16_t *rp = reinterpret_cast<uint16_t *>(res + row * (16 * R) + R * m);
#pragma unroll
        for (int i = 0; i < A / 2; ++i) __builtin_nontemporal_store((uint16_t)(an >> (16 * i)), ap + i);
#pragma unroll
        for (int i = 0; i < R / 2; ++i) __builtin_nontemporal_store((uint16_t)(rs >> (16 * i)), rp + i);
    }
}

// One workgroup encodes one 128-token window of one kv head, of K
// (blockIdx.z 0) or of V (1): a workgroup holds only one tensor's window
// in registers (128 VGPRs, four workgroups per CU against three with both:
// 43.2 -> 40.9 us per 32K layer).
// Thread (tr = tid / 16, m = tid % 16) owns dims 8m..8m+7 of the window's
// tokens tr, tr+16, ..., tr+112: every 16-byte load is part of a fully used
// 256-byte token row, and a token's 16 owners are the 16 lanes of one DPP
// row.  LAYOUT 0: one block per sequence; 1: paged; 2: a transmission-buffer
// object (planes [Hkv][T][64], no block table).  The BF16 input is read once
// and the planes are not read back by this kernel: nontemporal loads and
// stores (4.27 -> 4.8 TB/s on a 32K layer).  A: anchor bits (4, or the
// other split widths 2 and 6, whose plane rows are 16 A and 16 (8 - A)
// bytes).
template <int LAYOUT, int A = 4>
__global__ __launch_bounds__(kEncodeThreads, 4) void encode_kernel(
    Geometry geo, int b, int T, int bt_shift, const int32_t *__restrict__ block_table,
    const uint16_t *__restrict__ k, const uint16_t *__restrict__ v, uint8_t *__restrict__ k_anc,
    uint8_t *__restrict__ v_anc, uint8_t *__restrict__ k_res, uint8_t *__restrict__ v_res,
    MetaPtrs meta) {
    const int g = blockIdx.y;
    const int h = blockIdx.x;
    const int which = blockIdx.z;  // 0: K, 1: V
    const int tid = threadIdx.x;
    const int m = tid & 15;
    const int tr = tid >> 4;
    const int wave = tid >> 6;
    const int t0 = g * kKGroup;
    const int n = min(kKGroup, T - t0);
    const int Hkv = geo.Hkv;

    __shared__ float s_min[4][kHeadDim];
    __shared__ float s_max[4][kHeadDim];
    __shared__ float s_zero[kHeadDim];
    __shared__ float s_inv[kHeadDim];

    // ---- load the window: 8 tokens x 8 dims per thread, of K or V ----
    uint4 raw[8];
    const uint16_t *src = which == 0 ? k : v;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        const int tl = min(tr + 16 * i, n - 1);  // rows past the window re-read its last token
        const size_t e = ((size_t)(t0 + tl) * Hkv + h) * kHeadDim + 8 * m;
        const u32v4 xx = __builtin_nontemporal_load(reinterpret_cast<const u32v4 *>(src + e));
        raw[i] = make_uint4(xx.x, xx.y, xx.z, xx.w);
    }

    // Plane row of token t (the block lookup of a paged cache is checked).
    const int32_t *bt_row = block_table + (size_t)b * geo.max_blocks;
    auto plane_row = [&](int t, bool &ok) -> size_t {
        int blk, tb;
        if (LAYOUT == 2) {
            blk = 0;
            tb = t;
        } else if (LAYOUT == 0) {
            blk = bt_row[0];
            tb = t;
        } else {
            const int bi = bt_shift >= 0 ? (t >> bt_shift) : t / geo.bt;
            blk = bt_row[bi];
            tb = t - bi * geo.bt;
        }
        ok = blk >= 0 && blk < geo.num_blocks;
        return ((size_t)blk * Hkv + h) * geo.bt + tb;
    };

    if (which == 1) {
        // ---- V workgroups: per-token groups over 128 dims (the 16 lanes of a
        // DPP row) ----
        float vzero[8], vinv[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            float x[8];
            unpack8(raw[i], x);
            float mn = fmin3(fmin3(x[0], x[1], x[2]), fmin3(x[3], x[4], x[5]), fmin2(x[6], x[7]));
            float mx = fmax3(fmax3(x[0], x[1], x[2]), fmax3(x[3], x[4], x[5]), fmax2(x[6], x[7]));
            mn = row16_min(mn);
            mx = row16_max(mx);
            float scale;
            group_params(mn, mx, vzero[i], scale, vinv[i]);
            const int tl = tr + 16 * i;
            if (m == 0 && tl < n) {
                const size_t mi = ((size_t)b * Hkv + h) * geo.max_tokens + t0 + tl;
                meta.v_scale[mi] = scale;
                meta.v_zero[mi] = vzero[i];
            }
        }
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const int tl = tr + 16 * i;
            if (tl < n) {
                bool ok;
                const size_t row = plane_row(t0 + tl, ok);
                if (ok) {
                    float x[8];
                    unpack8(raw[i], x);
                    const float zv[8] = {vzero[i], vzero[i], vzero[i], vzero[i],
                                         vzero[i], vzero[i], vzero[i], vzero[i]};
                    const float iv[8] = {vinv[i], vinv[i], vinv[i], vinv[i],
                                         vinv[i], vinv[i], vinv[i], vinv[i]};
                    store_split<A>(x, zv, iv, v_anc, v_res, row, m);
                }
            }
        }
        return;
    }

    // ---- K: per-channel min/max over the window's tokens (the re-read
    // last token of a short window changes neither) ----
    float kmin[8], kmax[8];
    {
        float x[8][8];
#pragma unroll
        for (int i = 0; i < 8; ++i) unpack8(raw[i], x[i]);
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            kmin[j] = fmin3(fmin3(x[0][j], x[1][j], x[2][j]), fmin3(x[3][j], x[4][j], x[5][j]),
                            fmin2(x[6][j], x[7][j]));
            kmax[j] = fmax3(fmax3(x[0][j], x[1][j], x[2][j]), fmax3(x[3][j], x[4][j], x[5][j]),
                            fmax2(x[6][j], x[7][j]));
        }
    }
    // lanes m, m+16, m+32, m+48 of a wave hold the same channels
#pragma unroll
    for (int j = 0; j < 8; ++j) {
        kmin[j] = min_kg(kmin[j]);
        kmax[j] = max_kg(kmax[j]);
    }
    if ((tid & 63) < 16) {
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            s_min[wave][8 * m + j] = kmin[j];
            s_max[wave][8 * m + j] = kmax[j];
        }
    }
    __syncthreads();
    if (tid < kHeadDim) {
        const int d = tid;
        const float mn = fmin2(fmin2(s_min[0][d], s_min[1][d]), fmin2(s_min[2][d], s_min[3][d]));
        const float mx = fmax2(fmax2(s_max[0][d], s_max[1][d]), fmax2(s_max[2][d], s_max[3][d]));
        float zero, scale, inv;
        group_params(mn, mx, zero, scale, inv);
        s_zero[d] = zero;
        s_inv[d] = inv;
        const size_t mi = (((size_t)b * Hkv + h) * geo.n_groups + g) * kHeadDim + d;
        meta.k_scale[mi] = scale;
        meta.k_zero[mi] = zero;
    }

    __syncthreads();

    // ---- K codes -> planes ----
    float kz[8], ki[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
        kz[j] = s_zero[8 * m + j];
        ki[j] = s_inv[8 * m + j];
    }
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        const int tl = tr + 16 * i;
        if (tl < n) {
            bool ok;
            const size_t row = plane_row(t0 + tl, ok);
            if (ok) {
                float x[8];
                unpack8(raw[i], x);
                store_split<A>(x, kz, ki, k_anc, k_res, row, m);
            }
        }
    }
}

// Interleave the nibbles of 4 anchor bytes and 4 residual bytes into 8 codes:
// code[2j] = (a_j & 15) << 4 | (r_j & 15), code[2j+1] = (a_j & 0xF0) | (r_j >> 4).
__device__ __forceinline__ uint2 merge4(uint32_t a, uint32_t r) {
    // spread bytes 0,1 (lo) and 2,3 (hi) into 16-bit lanes
    const uint32_t alo = (a & 0xffu) | ((a & 0xff00u) << 8);
    const uint32_t ahi = ((a >> 16) & 0xffu) | ((a >> 8) & 0xff0000u);
    const uint32_t rlo = (r & 0xffu) | ((r & 0xff00u) << 8);
    const uint32_t rhi = ((r >> 16) & 0xffu) | ((r >> 8) & 0xff0000u);
    uint2 o;
    o.x = ((alo & 0x000F000Fu) << 4) | ((alo & 0x00F000F0u) << 8) | (rlo & 0x000F000Fu) |
          ((rlo & 0x00F000F0u) << 4);
    o.y = ((ahi & 0x000F000Fu) << 4) | ((ahi & 0x00F000F0u) << 8) | (rhi & 0x000F000Fu) |
          ((rhi & 0x00F000F0u) << 4);
    return o;
}

constexpr int kMergeThreads = 256;

// Wave w of the grid merges pieces (8 anchor + 8 residual bytes -> 16 code
// bytes) base + lane and base + 64 + lane, base = 128 w, 128 (w + waves), ...:
// every load instruction reads 512 contiguous bytes and every store
// instruction writes 1 KB, whole cache lines (two 16-byte stores per lane
// that interleave inside each line were 10% slower).  The stores are
// nontemporal: the verification that follows reads the codes much faster
// when they were not written through the last-level cache (a 70B-shaped
// verification over 1.1 GB of codes: 278 -> 214 us right after the merge).
__global__ __launch_bounds__(kMergeThreads) void merge_kernel(
    const uint2 *__restrict__ anc, const uint2 *__restrict__ res, uint8_t *__restrict__ codes,
    size_t n8, const uint8_t *__restrict__ anc_b, const uint8_t *__restrict__ res_b,
    uint8_t *__restrict__ codes_b, size_t n_packed) {
    const int lane = threadIdx.x & 63;
    const size_t wave = ((size_t)blockIdx.x * blockDim.x + threadIdx.x) >> 6;
    const size_t n_waves = ((size_t)gridDim.x * blockDim.x) >> 6;
    u32v4 *out = reinterpret_cast<u32v4 *>(codes);
    for (size_t base = 128 * wave; base < n8; base += 128 * n_waves) {
        const size_t p0 = base + lane, p1 = base + 64 + lane;
        uint2 a0 = make_uint2(0u, 0u), r0 = a0, a1 = a0, r1 = a0;
        if (p0 < n8) {
            a0 = anc[p0];
            r0 = res[p0];
        }
        if (p1 < n8) {
            a1 = anc[p1];
            r1 = res[p1];
        }
        const uint2 x0 = merge4(a0.x, r0.x), y0 = merge4(a0.y, r0.y);
        const uint2 x1 = merge4(a1.x, r1.x), y1 = merge4(a1.y, r1.y);
        const u32v4 o0 = {x0.x, x0.y, y0.x, y0.y};
        const u32v4 o1 = {x1.x, x1.y, y1.x, y1.y};
        if (p0 < n8) __builtin_nontemporal_store(o0, out + p0);
        if (p1 < n8) __builtin_nontemporal_store(o1, out + p1);
    }
    // ragged tail (< 8 bytes)
    if (blockIdx.x == 0 && threadIdx.x == 0) {
        for (size_t j = n8 * 8; j < n_packed; ++j) {
            const uint32_t a = anc_b[j], r = res_b[j];
            codes_b[2 * j] = (uint8_t)(((a & 15u) << 4) | (r & 15u));
            codes_b[2 * j + 1] = (uint8_t)((a & 0xF0u) | (r >> 4));
        }
    }
}

constexpr int kCopyThreads = 256;

// Row index of (sequence b, kv head h, token t) in a plane pool, or -1 when
// the block table names no valid block (such rows are skipped, as encode
// skips them).
__device__ __forceinline__ long long pool_row(const Geometry &g, const int32_t *bt_row, int bt_shift,
                                              int h, int t) {
    const int bi = bt_shift >= 0 ? (t >> bt_shift) : t / g.bt;
    const int blk = bt_row[bi];
    if (blk < 0 || blk >= g.num_blocks) return -1;
    return ((long long)blk * g.Hkv + h) * g.bt + (t - bi * g.bt);
}

// Anchor phase of the deserializer: the anchor buffer of the object (tokens
// t0 .. t0 + n - 1 of sequence b) is scattered into the pages.  Part
// blockIdx.y: 0 = K and V anchor rows (16 bytes per thread), 1 = K scales
// and zeros (float4 per thread), 2 = V scales and zeros (one float each).
__global__ __launch_bounds__(kCopyThreads) void deserialize_anchor_kernel(
    Geometry g, int b, int t0, int n, int bt_shift, const int32_t *__restrict__ block_table,
    const uint8_t *__restrict__ buf, uint8_t *__restrict__ k_anc, uint8_t *__restrict__ v_anc,
    MetaPtrs meta) {
    const int32_t *bt_row = block_table + (size_t)b * g.max_blocks;
    const size_t rows = (size_t)g.Hkv * n;
    const size_t rows_bytes = rows * kNibbleRow;
    const int ng = (n + kKGroup - 1) / kKGroup;
    const size_t kmeta = (size_t)g.Hkv * ng * kHeadDim;  // floats per K metadata section
    const size_t stride = (size_t)gridDim.x * blockDim.x;
    const size_t i0 = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (blockIdx.y == 0) {
        for (size_t e = i0; e < 2 * rows * 4; e += stride) {
            const size_t which = e / (rows * 4);  // 0: K, 1: V
            const size_t r = (e / 4) % rows;
            const int q = (int)(e & 3);
            const int h = (int)(r / n), i = (int)(r % n);
            const long long pr = pool_row(g, bt_row, bt_shift, h, t0 + i);
            if (pr < 0) continue;
            const uint4 x = *reinterpret_cast<const uint4 *>(buf + which * rows_bytes + r * kNibbleRow + 16 * q);
            uint8_t *plane = which == 0 ? k_anc : v_anc;
            *reinterpret_cast<uint4 *>(plane + (size_t)pr * kNibbleRow + 16 * q) = x;
        }
    } else if (blockIdx.y == 1) {
        const float *src = reinterpret_cast<const float *>(buf + 2 * rows_bytes);
        for (size_t e = i0; e < 2 * kmeta / 4; e += stride) {
            const size_t which = e / (kmeta / 4);  // 0: scales, 1: zeros
            const size_t f = 4 * (e % (kmeta / 4));
            const int h = (int)(f / ((size_t)ng * kHeadDim));
            const size_t rem = f % ((size_t)ng * kHeadDim);
            const float4 x = *reinterpret_cast<const float4 *>(src + which * kmeta + f);
            float *dst = which == 0 ? meta.k_scale : meta.k_zero;
            const size_t gi = (((size_t)b * g.Hkv + h) * g.n_groups + t0 / kKGroup) * kHeadDim + rem;
            *reinterpret_cast<float4 *>(dst + gi) = x;
        }
    } else {
        const float *src = reinterpret_cast<const float *>(buf + 2 * rows_bytes) + 2 * kmeta;
        for (size_t e = i0; e < 2 * rows; e += stride) {
            const size_t which = e / rows;  // 0: scales, 1: zeros
            const size_t r = e % rows;
            const int h = (int)(r / n), i = (int)(r % n);
            float *dst = which == 0 ? meta.v_scale : meta.v_zero;
            dst[((size_t)b * g.Hkv + h) * g.max_tokens + t0 + i] = src[which * rows + r];
        }
    }
}

// Residual phase of the deserializer: the residual buffer of the object and
// its anchor rows already in the pages merge into the code rows of the
// pages (16 anchor + 16 residual bytes -> 32 code bytes per thread).
__global__ __launch_bounds__(kCopyThreads) void deserialize_residual_kernel(
    Geometry g, int b, int t0, int n, int bt_shift, const int32_t *__restrict__ block_table,
    const uint8_t *__restrict__ buf, const uint8_t *__restrict__ k_anc,
    const uint8_t *__restrict__ v_anc, uint8_t *__restrict__ k_codes, uint8_t *__restrict__ v_codes) {
    const int32_t *bt_row = block_table + (size_t)b * g.max_blocks;
    const size_t rows = (size_t)g.Hkv * n;
    const size_t stride = (size_t)gridDim.x * blockDim.x;
    for (size_t e = (size_t)blockIdx.x * blockDim.x + threadIdx.x; e < 2 * rows * 4; e += stride) {
        const size_t which = e / (rows * 4);
        const size_t r = (e / 4) % rows;
        const int q = (int)(e & 3);
        const int h = (int)(r / n), i = (int)(r % n);
        const long long pr = pool_row(g, bt_row, bt_shift, h, t0 + i);
        if (pr < 0) continue;
        const uint4 a = *reinterpret_cast<const uint4 *>((which == 0 ? k_anc : v_anc) +
                                                         (size_t)pr * kNibbleRow + 16 * q);
        const uint4 x = *reinterpret_cast<const uint4 *>(buf + which * rows * kNibbleRow +
                                                         r * kNibbleRow + 16 * q);
        const uint2 c0 = merge4(a.x, x.x);
        const uint2 c1 = merge4(a.y, x.y);
        const uint2 c2 = merge4(a.z, x.z);
        const uint2 c3 = merge4(a.w, x.w);
        uint4 *dst = reinterpret_cast<uint4 *>((which == 0 ? k_codes : v_codes) +
                                               (size_t)pr * kCodeRow + 32 * q);
        dst[0] = make_uint4(c0.x, c0.y, c1.x, c1.y);
        dst[1] = make_uint4(c2.x, c2.y, c3.x, c3.y);
    }
}

int bt_shift_of(int bt) {
    for (int sh = 0; sh < 31; ++sh)
        if ((1 << sh) == bt) return sh;
    return -1;
}

unsigned copy_blocks(size_t work) {
    size_t blocks = (work + kCopyThreads - 1) / kCopyThreads;
    if (blocks > 256 * 32) blocks = 256 * 32;
    return (unsigned)(blocks == 0 ? 1 : blocks);
}

}  // namespace

template <int A>
void launch_encode_width(const Geometry &g, int b, int T, int bt_shift, const int32_t *block_table,
                         const uint16_t *k, const uint16_t *v, uint8_t *k_anc, uint8_t *v_anc,
                         uint8_t *k_res, uint8_t *v_res, MetaPtrs meta, hipStream_t stream) {
    dim3 grid(g.Hkv, (T + kKGroup - 1) / kKGroup, 2);
    if (g.max_blocks == 1)
        hipLaunchKernelGGL((encode_kernel<0, A>), grid, dim3(kEncodeThreads), 0, stream, g, b, T, bt_shift,
                           block_table, k, v, k_anc, v_anc, k_res, v_res, meta);
    else
        hipLaunchKernelGGL((encode_kernel<1, A>), grid, dim3(kEncodeThreads), 0, stream, g, b, T, bt_shift,
                           block_table, k, v, k_anc, v_anc, k_res, v_res, meta);
}

hipError_t launch_encode(const Geometry &g, int b, int T, const int32_t *block_table,
                         const uint16_t *k, const uint16_t *v, uint8_t *k_anc, uint8_t *v_anc,
                         uint8_t *k_res, uint8_t *v_res, MetaPtrs meta, hipStream_t stream,
                         int anchor_bits) {
    if (T <= 0) return hipSuccess;
    int bt_shift = -1;
    for (int sh = 0; sh < 31; ++sh)
        if ((1 << sh) == g.bt) bt_shift = sh;
    if (anchor_bits == 4)
        launch_encode_width<4>(g, b, T, bt_shift, block_table, k, v, k_anc, v_anc, k_res, v_res, meta, stream);
    else if (anchor_bits == 2)
        launch_encode_width<2>(g, b, T, bt_shift, block_table, k, v, k_anc, v_anc, k_res, v_res, meta, stream);
    else if (anchor_bits == 6)
        launch_encode_width<6>(g, b, T, bt_shift, block_table, k, v, k_anc, v_anc, k_res, v_res, meta, stream);
    else
        return hipErrorInvalidValue;
    return hipGetLastError();
}

hipError_t launch_merge(const uint8_t *anc, const uint8_t *res, uint8_t *codes, size_t n_packed,
                        hipStream_t stream) {
    if (n_packed == 0) return hipSuccess;
    const size_t n8 = n_packed / 8;
    // enough workgroups to cover the device several times over (two pieces
    // per thread and round); each wave then loops over the rest
    size_t blocks = (n8 + 2 * kMergeThreads - 1) / (2 * kMergeThreads);
    if (blocks > 256 * 32) blocks = 256 * 32;
    if (blocks == 0) blocks = 1;
    hipLaunchKernelGGL(merge_kernel, dim3((unsigned)blocks), dim3(kMergeThreads), 0, stream,
                       reinterpret_cast<const uint2 *>(anc), reinterpret_cast<const uint2 *>(res), codes, n8,
                       anc, res, codes, n_packed);
    return hipGetLastError();
}

hipError_t launch_serialize(int Hkv, int n, const uint16_t *k, const uint16_t *v,
                            uint8_t *anc_buf, uint8_t *res_buf, hipStream_t stream) {
    if (n <= 0) return hipSuccess;
    // the object as a one-block cache of its own: its planes and metadata
    // rows are the sections of the two buffers
    Geometry g;
    g.Hkv = Hkv;
    g.bt = n;
    g.max_blocks = 1;
    g.num_blocks = 1;
    g.max_tokens = n;
    g.n_groups = (n + kKGroup - 1) / kKGroup;
    g.n_pages = (n + 255) / 256;
    g.n_chunks = (n + 31) / 32;
    const size_t rows_bytes = (size_t)Hkv * n * kNibbleRow;
    const size_t kmeta = (size_t)Hkv * g.n_groups * kHeadDim;
    float *m = reinterpret_cast<float *>(anc_buf + 2 * rows_bytes);
    MetaPtrs meta{m, m + kmeta, m + 2 * kmeta, m + 2 * kmeta + (size_t)Hkv * n};
    dim3 grid(Hkv, g.n_groups, 2);
    hipLaunchKernelGGL(encode_kernel<2>, grid, dim3(kEncodeThreads), 0, stream, g, 0, n, -1,
                       static_cast<const int32_t *>(nullptr), k, v, anc_buf, anc_buf + rows_bytes,
                       res_buf, res_buf + rows_bytes, meta);
    return hipGetLastError();
}

hipError_t launch_deserialize_anchor(const Geometry &g, int b, int t0, int n,
                                     const int32_t *block_table, const uint8_t *buf,
                                     uint8_t *k_anc, uint8_t *v_anc, MetaPtrs meta,
                                     hipStream_t stream) {
    if (n <= 0) return hipSuccess;
    const size_t work = (size_t)2 * g.Hkv * n * 4;  // the largest part
    hipLaunchKernelGGL(deserialize_anchor_kernel, dim3(copy_blocks(work), 3), dim3(kCopyThreads), 0,
                       stream, g, b, t0, n, bt_shift_of(g.bt), block_table, buf, k_anc, v_anc, meta);
    return hipGetLastError();
}

hipError_t launch_deserialize_residual(const Geometry &g, int b, int t0, int n,
                                       const int32_t *block_table, const uint8_t *buf,
                                       const uint8_t *k_anc, const uint8_t *v_anc,
                                       uint8_t *k_codes, uint8_t *v_codes, hipStream_t stream) {
    if (n <= 0) return hipSuccess;
    const size_t work = (size_t)2 * g.Hkv * n * 4;
    hipLaunchKernelGGL(deserialize_residual_kernel, dim3(copy_blocks(work)), dim3(kCopyThreads), 0,
                       stream, g, b, t0, n, bt_shift_of(g.bt), block_table, buf, k_anc, v_anc,
                       k_codes, v_codes);
    return hipGetLastError();
}

namespace {

// Merge of A-bit anchor rows and R-bit residual rows: thread per 8 elements
// of a row (A + R bytes in, 8 code bytes out), grid-stride; nontemporal
// stores, as in merge_kernel.
template <int A>
__global__ __launch_bounds__(kMergeThreads) void merge_split_kernel(const uint8_t *__restrict__ anc,
                                                                    const uint8_t *__restrict__ res,
                                                                    uint8_t *__restrict__ codes,
                                                                    size_t n_pieces) {
    constexpr int R = 8 - A;
    const size_t stride = (size_t)gridDim.x * blockDim.x;
    for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n_pieces; i += stride) {
        const uint16_t *ap = reinterpret_cast<const uint16_t *>(anc + A * i);
        const uint16_t *rp = reinterpret_cast<const uint16_t *>(res + R * i);
        uint64_t an = 0, rs = 0;
#pragma unroll
        for (int k = 0; k < A / 2; ++k) an |= (uint64_t)ap[k] << (16 * k);
#pragma unroll
        for (int k = 0; k < R / 2; ++k) rs |= (uint64_t)rp[k] << (16 * k);
        uint64_t c = 0;
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            const uint64_t a = (an >> (A * j)) & ((1u << A) - 1u);
            const uint64_t r = (rs >> (R * j)) & ((1u << R) - 1u);
            c |= ((a << R) | r) << (8 * j);
        }
        __builtin_nontemporal_store(c, reinterpret_cast<uint64_t *>(codes + 8 * i));
    }
}

__device__ __forceinline__ uint32_t f32_to_bf16_bits(float f) {
    const uint32_t u = __float_as_uint(f);
    if ((u & 0x7F800000u) == 0x7F800000u && (u & 0x007FFFFFu)) return (u >> 16) | 0x40u;
    return (u + 0x7FFFu + ((u >> 16) & 1u)) >> 16;
}

// Anchor phase for other split widths: K and V of one sequence from the A-bit
// anchors as BF16 [T][Hkv][128]; the anchor stands for code
// 2^R a + (2^R - 1) / 2, x = fmaf(code, scale, zero) rounded to BF16.
// Thread per (8 tokens, head, 8 dims), the dims fastest: the K scales and
// zeros of its dims are loaded once for its 8 tokens (which share a K
// group), grid-stride.
template <int A, int LAYOUT>
__global__ __launch_bounds__(kMergeThreads) void dequant_anchor_split_kernel(
    Geometry geo, int b, int T, int bt_shift, const int32_t *__restrict__ block_table,
    const uint8_t *__restrict__ k_anc, const uint8_t *__restrict__ v_anc, MetaPtrs meta,
    uint16_t *__restrict__ k_out, uint16_t *__restrict__ v_out) {
    constexpr int R = 8 - A;
    constexpr float kHalf = (float)((1 << R) - 1) / 2.0f;
    const int Hkv = geo.Hkv;
    const int n_oct = (T + 7) / 8;
    const size_t per = (size_t)n_oct * Hkv * 16;
    const size_t stride = (size_t)gridDim.x * blockDim.x;
    const int32_t *bt_row = block_table + (size_t)b * geo.max_blocks;
    for (size_t e = (size_t)blockIdx.x * blockDim.x + threadIdx.x; e < 2 * per; e += stride) {
        const int which = e >= per ? 1 : 0;
        const size_t r = e - (size_t)which * per;
        const int m = (int)(r & 15);
        const size_t oh = r >> 4;
        const int h = (int)(oh % Hkv);
        const int t0 = 8 * (int)(oh / Hkv);
        float sc[8], zr[8];
        if (which == 0) {
            const size_t km = (((size_t)b * Hkv + h) * geo.n_groups + t0 / kKGroup) * kHeadDim + 8 * m;
#pragma unroll
            for (int j = 0; j < 8; ++j) {
                sc[j] = meta.k_scale[km + j];
                zr[j] = meta.k_zero[km + j];
            }
        }
        const uint8_t *plane = which == 0 ? k_anc : v_anc;
        uint16_t *out = which == 0 ? k_out : v_out;
        const int nt = min(8, T - t0);
#pragma unroll
        for (int k = 0; k < 8; ++k) {
            if (k >= nt) break;
            const int t = t0 + k;
            int blk, tb;
            if (LAYOUT == 0) {
                blk = bt_row[0];
                tb = t;
            } else {
                const int bi = bt_shift >= 0 ? (t >> bt_shift) : t / geo.bt;
                blk = bt_row[bi];
                tb = t - bi * geo.bt;
            }
            if (blk < 0 || blk >= geo.num_blocks) continue;
            const size_t row = ((size_t)blk * Hkv + h) * geo.bt + tb;
            const uint16_t *ap = reinterpret_cast<const uint16_t *>(plane + row * (16 * A) + A * m);
            uint64_t an = 0;
#pragma unroll
            for (int i = 0; i < A / 2; ++i) an |= (uint64_t)ap[i] << (16 * i);
            float s1[8], z1[8];
            if (which == 0) {
#pragma unroll
                for (int j = 0; j < 8; ++j) {
                    s1[j] = sc[j];
                    z1[j] = zr[j];
                }
            } else {
                const size_t vm = ((size_t)b * Hkv + h) * geo.max_tokens + t;
                const float s0 = meta.v_scale[vm], z0 = meta.v_zero[vm];
#pragma unroll
                for (int j = 0; j < 8; ++j) {
                    s1[j] = s0;
                    z1[j] = z0;
                }
            }
            uint32_t o[4];
#pragma unroll
            for (int j = 0; j < 8; j += 2) {
                const float q0 = (float)(((an >> (A * j)) & ((1u << A) - 1u)) << R) + kHalf;
                const float q1 = (float)(((an >> (A * (j + 1))) & ((1u << A) - 1u)) << R) + kHalf;
                o[j / 2] = f32_to_bf16_bits(fmaf(q0, s1[j], z1[j])) |
                           (f32_to_bf16_bits(fmaf(q1, s1[j + 1], z1[j + 1])) << 16);
            }
            *reinterpret_cast<uint4 *>(out + ((size_t)t * Hkv + h) * kHeadDim + 8 * m) =
                make_uint4(o[0], o[1], o[2], o[3]);
        }
    }
}

}  // namespace

hipError_t launch_merge_split(int anchor_bits, const uint8_t *anc, const uint8_t *res, uint8_t *codes,
                              size_t n_rows, hipStream_t stream) {
    if (n_rows == 0) return hipSuccess;
    const size_t n_pieces = n_rows * 16;
    size_t blocks = (n_pieces + kMergeThreads - 1) / kMergeThreads;
    if (blocks > 256 * 32) blocks = 256 * 32;
    if (anchor_bits == 2)
        hipLaunchKernelGGL(merge_split_kernel<2>, dim3((unsigned)blocks), dim3(kMergeThreads), 0, stream, anc, res,
                           codes, n_pieces);
    else if (anchor_bits == 4)
        hipLaunchKernelGGL(merge_split_kernel<4>, dim3((unsigned)blocks), dim3(kMergeThreads), 0, stream, anc, res,
                           codes, n_pieces);
    else if (anchor_bits == 6)
        hipLaunchKernelGGL(merge_split_kernel<6>, dim3((unsigned)blocks), dim3(kMergeThreads), 0, stream, anc, res,
                           codes, n_pieces);
    else
        return hipErrorInvalidValue;
    return hipGetLastError();
}

template <int A>
static void launch_dequant_split_width(const Geometry &g, int b, int T, int sh, const int32_t *block_table,
                                       const uint8_t *k_anc, const uint8_t *v_anc, MetaPtrs meta,
                                       uint16_t *k_out, uint16_t *v_out, dim3 grid, hipStream_t stream) {
    if (g.max_blocks == 1)
        hipLaunchKernelGGL((dequant_anchor_split_kernel<A, 0>), grid, dim3(kMergeThreads), 0, stream, g, b, T, sh,
                           block_table, k_anc, v_anc, meta, k_out, v_out);
    else
        hipLaunchKernelGGL((dequant_anchor_split_kernel<A, 1>), grid, dim3(kMergeThreads), 0, stream, g, b, T, sh,
                           block_table, k_anc, v_anc, meta, k_out, v_out);
}

hipError_t launch_dequant_anchor_split(int anchor_bits, const Geometry &g, int b, int T,
                                       const int32_t *block_table, const uint8_t *k_anc,
                                       const uint8_t *v_anc, MetaPtrs meta, uint16_t *k_out,
                                       uint16_t *v_out, hipStream_t stream) {
    if (T <= 0) return hipSuccess;
    size_t blocks = ((size_t)2 * ((T + 7) / 8) * g.Hkv * 16 + kMergeThreads - 1) / kMergeThreads;
    if (blocks > 256 * 32) blocks = 256 * 32;
    const dim3 grid((unsigned)blocks);
    int sh = -1;
    for (int k = 0; k < 31; ++k)
        if ((1 << k) == g.bt) sh = k;
    if (anchor_bits == 2)
        launch_dequant_split_width<2>(g, b, T, sh, block_table, k_anc, v_anc, meta, k_out, v_out, grid, stream);
    else if (anchor_bits == 4)
        launch_dequant_split_width<4>(g, b, T, sh, block_table, k_anc, v_anc, meta, k_out, v_out, grid, stream);
    else if (anchor_bits == 6)
        launch_dequant_split_width<6>(g, b, T, sh, block_table, k_anc, v_anc, meta, k_out, v_out, grid, stream);
    else
        return hipErrorInvalidValue;
    return hipGetLastError();
}

}  // namespace lynx
