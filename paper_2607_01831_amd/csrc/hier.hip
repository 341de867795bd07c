// The hierarchical non-linear codec of Alg. 1 (Sec. 4.1) for gfx950:
// encode (page normalization, chunk isolation, alpha-law transform, split
// into a signed 4-bit anchor and a signed 4-bit correction) and the
// deserializer's dequantization of the anchor alone or of the merged codes
// into BF16 pages (Sec. 4.2 Anchor and Residual phases).
//
// Per channel of a kv head (K and V alike), pages of 256 tokens, chunks of
// 32 (Sec. 6.1):
//   1. gmin = min x, gscale = max x - gmin over the page; X = (x - gmin) *
//      (1 / gscale);
//   2. mu = the chunk's mean of X (fp32 sum in token order / count),
//      Xc = X - mu, sigma = max |Xc|, Xf = Xc * (1 / sigma);
//   3. I = Round(M ln(1 + a|Xf|) / ln(1 + a)): the number of decision
//      thresholds theta_k <= |Xf|, found from the transform evaluated in
//      fp32 (within one of the count) and one exact step against the two
//      thresholds around it; S = sign(Xc); M = 127, or 7 for the 4-bit code;
//   4. by variant, with the sign-aware anchor Q_anc = V, or -V - 1 for S < 0:
//      biased:  V = min((I + 7) >> 4, 7), Q_res = clamp(16 V - I, -8, 7);
//      centred: V = I >> 4, Q_res = I - 16 V - 8 (every code kept);
//      4-bit:   V = I, no correction.
// A range whose reciprocal is not finite and positive normalizes to 0.  Every
// fp32 product that an add follows is rounded on its own (mul_rn), so no
// fused multiply-add changes a result.
#include "lynx_internal.h"

#include <float.h>
#include <math.h>

namespace lynx {
namespace {

constexpr int kPage = 256;
constexpr int kChunk = 32;
constexpr int kHThreads = 256;

__device__ __forceinline__ float bf16_to_f32(uint32_t bits16) { return __uint_as_float(bits16 << 16); }

// An fp32 product rounded on its own.  HIP contracts a product into a
// following add (an FMA, one rounding fewer) even across statements; the
// empty asm hands the rounded product over, so the sum that follows is a
// separate IEEE add, as the definition has it.
__device__ __forceinline__ float mul_rn(float a, float b) {
    float p = a * b;
    asm volatile("" : "+v"(p));
    return p;
}

__device__ __forceinline__ float range_recip(float r) {
    const float v = 1.0f / r;  // IEEE division (correctly rounded)
    return (r > 0.0f && v <= FLT_MAX) ? v : 0.0f;
}

__device__ __forceinline__ uint32_t bf16_rne(float f) {
    const uint32_t u = __float_as_uint(f);
    if ((u & 0x7F800000u) == 0x7F800000u && (u & 0x007FFFFFu)) return (u >> 16) | 0x40u;
    return (u + 0x7FFFu + ((u >> 16) & 1u)) >> 16;
}

// Stage 4 of every variant in one branch-free form: V = min((I + bias) >> sh,
// 7), Q_res = clamp(sgn (16 V - I) - off, -8, 7), with (bias, sh, sgn, off)
// = (7, 4, 1, 0) for the biased split, (0, 4, -1, 8) for the centred one
// (V = I >> 4, Q_res = I - 16 V - 8, never clamped) and (0, 0, 1, 0) for the
// 4-bit code (V = I; no residual is written).
struct SplitRule {
    int bias, sh, sgn, off;
};
__device__ __forceinline__ SplitRule split_rule(int variant) {
    if (variant == kHBiased) return {7, 4, 1, 0};
    if (variant == kHCentred) return {0, 4, -1, 8};
    return {0, 0, 1, 0};
}
// The byte-ready nibbles of the anchor and residual of one code.
__device__ __forceinline__ void split(const SplitRule &sr, int I, float xc, uint32_t &qa, uint32_t &qr) {
    const int V = min((I + sr.bias) >> sr.sh, 7);
    const int r = min(max(sr.sgn * (16 * V - I) - sr.off, -8), 7);
    qa = (uint32_t)(xc < 0.0f ? -V - 1 : V) & 15u;
    qr = (uint32_t)r & 15u;
}

// Workgroup (kv head, page, K or V).  Thread (quarter q = tid / 64, channel
// pair cp = tid % 64) owns channels 2 cp, 2 cp + 1 of the page's tokens
// 64 q .. 64 q + 63 (chunks 2 q, 2 q + 1): a wavefront reads whole 256-byte
// token rows and writes whole 64-byte plane rows.  LAYOUT 0: one block per
// sequence; 1: paged.  The 4-bit variant writes the anchor planes only.
template <int LAYOUT>
__global__ __launch_bounds__(kHThreads, 3) void hencode_kernel(
    Geometry geo, int b, int T, int bt_shift, const int32_t *__restrict__ block_table,
    const uint16_t *__restrict__ k, const uint16_t *__restrict__ v, uint8_t *__restrict__ k_anc,
    uint8_t *__restrict__ v_anc, uint8_t *__restrict__ k_res, uint8_t *__restrict__ v_res,
    HMetaPtrs meta, HTables tab, int variant) {
    const int h = blockIdx.x;
    const int p = blockIdx.y;
    const int which = blockIdx.z;
    const int tid = threadIdx.x;
    const int cp = tid & 63;
    const int q = tid >> 6;
    const int Hkv = geo.Hkv;
    const int t0 = p * kPage;
    const int n = min(kPage, T - t0);
    const SplitRule sr = split_rule(variant);
    const bool has_res = variant != kHInt4;
    const uint16_t *src = which == 0 ? k : v;
    uint8_t *anc = which == 0 ? k_anc : v_anc;
    uint8_t *res = which == 0 ? k_res : v_res;
    float *gmin_a = which == 0 ? meta.k_gmin : meta.v_gmin;
    float *gsc_a = which == 0 ? meta.k_gscale : meta.v_gscale;
    float *mu_a = which == 0 ? meta.k_mu : meta.v_mu;
    float *sig_a = which == 0 ? meta.k_sigma : meta.v_sigma;

    __shared__ float s_theta[130];  // -inf, theta[0..127], +inf
    __shared__ float s_lo[4][kHeadDim], s_hi[4][kHeadDim];
    if (tid < 130) s_theta[tid] = tid == 0 ? -INFINITY : (tid <= 128 ? tab.theta[tid - 1] : INFINITY);

    // the thread's 64 tokens x 2 channels (BF16 pairs)
    uint32_t raw[64];
#pragma unroll
    for (int i = 0; i < 64; ++i) {
        const int tl = min(64 * q + i, n - 1);  // rows past the page re-read its last token
        raw[i] = *reinterpret_cast<const uint32_t *>(src + ((size_t)(t0 + tl) * Hkv + h) * kHeadDim + 2 * cp);
    }
    const int mine = max(0, min(64, n - 64 * q));  // valid tokens of the thread

    // ---- stage 1: page min / max per channel (rows past the page repeat
    // its last token, which leaves a minimum or maximum unchanged) ----
    float lo0 = INFINITY, hi0 = -INFINITY, lo1 = INFINITY, hi1 = -INFINITY;
#pragma unroll
    for (int i = 0; i < 64; ++i) {
        const float x0 = bf16_to_f32(raw[i] & 0xffffu), x1 = bf16_to_f32(raw[i] >> 16);
        lo0 = fminf(lo0, x0);
        hi0 = fmaxf(hi0, x0);
        lo1 = fminf(lo1, x1);
        hi1 = fmaxf(hi1, x1);
    }
    s_lo[q][2 * cp] = lo0;
    s_lo[q][2 * cp + 1] = lo1;
    s_hi[q][2 * cp] = hi0;
    s_hi[q][2 * cp + 1] = hi1;
    __syncthreads();
    float lo[2], hi[2], ig[2], gsc[2];
#pragma unroll
    for (int j = 0; j < 2; ++j) {
        const int d = 2 * cp + j;
        lo[j] = fminf(fminf(s_lo[0][d], s_lo[1][d]), fminf(s_lo[2][d], s_lo[3][d]));
        hi[j] = fmaxf(fmaxf(s_hi[0][d], s_hi[1][d]), fmaxf(s_hi[2][d], s_hi[3][d]));
        if (lo[j] == 0.0f) lo[j] = 0.0f;  // -0 -> +0
        if (hi[j] == 0.0f) hi[j] = 0.0f;
        gsc[j] = hi[j] - lo[j];
        ig[j] = range_recip(gsc[j]);
    }
    const size_t pm = (((size_t)b * Hkv + h) * geo.n_pages + p) * kHeadDim + 2 * cp;
    if (q == 0) {
        *reinterpret_cast<float2 *>(gmin_a + pm) = make_float2(lo[0], lo[1]);
        *reinterpret_cast<float2 *>(gsc_a + pm) = make_float2(gsc[0], gsc[1]);
    }

    const int32_t *bt_row = block_table + (size_t)b * geo.max_blocks;
    // LAYOUT 0: the thread's plane bytes for its first token; token i of
    // the quarter is i rows (64 bytes) further
    const int blk0 = bt_row[0];
    const bool ok0 = LAYOUT == 0 && blk0 >= 0 && blk0 < geo.num_blocks;
    const size_t off0 = (((size_t)blk0 * Hkv + h) * geo.bt + (size_t)(t0 + 64 * q)) * kNibbleRow + cp;

    // ---- stages 2-4, chunk by chunk ----
#pragma unroll
    for (int c = 0; c < 2; ++c) {
        const int i0 = 32 * c;
        const int cnt = max(0, min(kChunk, mine - i0));
        if (cnt == 0) continue;  // uniform within the wavefront
        float X[2][kChunk];
        float mu[2], sig[2], is[2];
#pragma unroll
        for (int j = 0; j < 2; ++j) {
#pragma unroll
            for (int i = 0; i < kChunk; ++i) {
                const uint32_t w = raw[i0 + i];
                const float x = bf16_to_f32(j == 0 ? (w & 0xffffu) : (w >> 16));
                X[j][i] = mul_rn(x - lo[j], ig[j]);
            }
            // the sum in token order over the chunk's tokens
            float sum = 0.0f;
            if (cnt == kChunk) {  // uniform
#pragma unroll
                for (int i = 0; i < kChunk; ++i) sum = sum + X[j][i];
            } else {
#pragma unroll
                for (int i = 0; i < kChunk; ++i)
                    if (i < cnt) sum = sum + X[j][i];
            }
            mu[j] = sum / (float)cnt;
            // rows past the page repeat its last token, inside this chunk
            float s = 0.0f;
#pragma unroll
            for (int i = 0; i < kChunk; ++i) s = fmaxf(s, fabsf(X[j][i] - mu[j]));
            sig[j] = s;
            is[j] = range_recip(s);
        }
        const size_t cm = (((size_t)b * Hkv + h) * geo.n_chunks + (size_t)t0 / kChunk + 2 * q + c) * kHeadDim + 2 * cp;
        *reinterpret_cast<float2 *>(mu_a + cm) = make_float2(mu[0], mu[1]);
        *reinterpret_cast<float2 *>(sig_a + cm) = make_float2(sig[0], sig[1]);
#pragma unroll
        for (int i = 0; i < kChunk; ++i) {
            if (i < cnt) {  // uniform within the wavefront
                uint32_t qa[2], qr[2];
#pragma unroll
                for (int j = 0; j < 2; ++j) {
                    const float xc = X[j][i] - mu[j];
                    float xf = fabsf(mul_rn(xc, is[j]));
                    xf = xf > 1.0f ? 1.0f : xf;
                    // the number of thresholds <= xf: the transform's own
                    // value rounded (within one of the count: its fp32 error
                    // is far below half a code), then one exact step against
                    // the thresholds on either side (a NaN counts none)
                    const float ye = tab.linear ? xf : __log2f(1.0f + tab.alpha * xf);
                    const float y = fminf(fmaxf(ye * tab.yscale + 0.5f, 0.0f), (float)tab.levels);
                    const int I0 = (int)y;
                    const int I = I0 - (s_theta[I0] > xf ? 1 : 0) + (s_theta[I0 + 1] <= xf ? 1 : 0);
                    split(sr, I, xc, qa[j], qr[j]);
                }
                const uint8_t ab = (uint8_t)(qa[0] | (qa[1] << 4)), rb = (uint8_t)(qr[0] | (qr[1] << 4));
                if (LAYOUT == 0) {
                    if (ok0) {
                        anc[off0 + (size_t)(i0 + i) * kNibbleRow] = ab;
                        if (has_res) res[off0 + (size_t)(i0 + i) * kNibbleRow] = rb;
                    }
                } else {
                    const int t = t0 + 64 * q + i0 + i;
                    const int bi = bt_shift >= 0 ? (t >> bt_shift) : t / geo.bt;
                    const int blk = bt_row[bi];
                    if (blk >= 0 && blk < geo.num_blocks) {
                        const size_t off = (((size_t)blk * Hkv + h) * geo.bt + (t - bi * geo.bt)) * kNibbleRow + cp;
                        anc[off] = ab;
                        if (has_res) res[off] = rb;
                    }
                }
            }
        }
    }
}

__device__ __forceinline__ int sext4(uint32_t nib) { return (int)nib >= 8 ? (int)nib - 16 : (int)nib; }

// Dequantization to BF16 [T][Hkv][128]: thread (8 tokens, 8 dims), per
// dimension the level of the code the variant names (biased: 16 V for the
// anchor, 16 V - Q_res for the merged code; centred: the bucket centre
// 16 V + 7.5, or 16 V + 8 + Q_res; 4-bit: V), x = ((+-level * sigma) + mu) *
// gscale + gmin in fp32, rounded to BF16 to nearest even.  FULL 0: anchor
// nibble planes; 1: code planes.
template <int FULL, int LAYOUT>
__global__ __launch_bounds__(kHThreads) void hdequant_kernel(
    Geometry geo, int b, int T, int bt_shift, const int32_t *__restrict__ block_table,
    const uint8_t *__restrict__ k_plane, const uint8_t *__restrict__ v_plane, HMetaPtrs meta,
    HTables tab, int variant, uint16_t *__restrict__ k_out, uint16_t *__restrict__ v_out) {
    __shared__ float s_level[128];
    __shared__ float s_alevel[8];
    if (threadIdx.x < 128) s_level[threadIdx.x] = tab.level[threadIdx.x];
    if (threadIdx.x < 8) s_alevel[threadIdx.x] = tab.alevel[threadIdx.x];
    __syncthreads();
    const int Hkv = geo.Hkv;
    // item (tensor, token octet, head, 8-dim piece), the piece fastest: a
    // thread loads the page and chunk scalars of its 8 dims once and
    // reconstructs 8 consecutive tokens (an octet never straddles a chunk)
    const int n_oct = (T + 7) / 8;
    const size_t per = (size_t)n_oct * Hkv * 16;
    const size_t stride = (size_t)gridDim.x * blockDim.x;
    const int32_t *bt_row = block_table + (size_t)b * geo.max_blocks;
    for (size_t e = (size_t)blockIdx.x * blockDim.x + threadIdx.x; e < 2 * per; e += stride) {
        const int which = e >= per ? 1 : 0;
        const size_t r = e - (size_t)which * per;
        const int d8 = (int)(r & 15);
        const size_t oh = r >> 4;  // octet * Hkv + h
        const int h = (int)(oh % Hkv);
        const int t0 = 8 * (int)(oh / Hkv);
        const size_t pm = (((size_t)b * Hkv + h) * geo.n_pages + t0 / kPage) * kHeadDim + 8 * d8;
        const size_t cm = (((size_t)b * Hkv + h) * geo.n_chunks + t0 / kChunk) * kHeadDim + 8 * d8;
        const float *gmin_a = which == 0 ? meta.k_gmin : meta.v_gmin;
        const float *gsc_a = which == 0 ? meta.k_gscale : meta.v_gscale;
        const float *mu_a = which == 0 ? meta.k_mu : meta.v_mu;
        const float *sig_a = which == 0 ? meta.k_sigma : meta.v_sigma;
        float gm[8], gs[8], mu[8], sg[8];
#pragma unroll
        for (int k4 = 0; k4 < 2; ++k4) {
            const float4 a = *reinterpret_cast<const float4 *>(gmin_a + pm + 4 * k4);
            const float4 s = *reinterpret_cast<const float4 *>(gsc_a + pm + 4 * k4);
            const float4 m = *reinterpret_cast<const float4 *>(mu_a + cm + 4 * k4);
            const float4 g = *reinterpret_cast<const float4 *>(sig_a + cm + 4 * k4);
            gm[4 * k4] = a.x; gm[4 * k4 + 1] = a.y; gm[4 * k4 + 2] = a.z; gm[4 * k4 + 3] = a.w;
            gs[4 * k4] = s.x; gs[4 * k4 + 1] = s.y; gs[4 * k4 + 2] = s.z; gs[4 * k4 + 3] = s.w;
            mu[4 * k4] = m.x; mu[4 * k4 + 1] = m.y; mu[4 * k4 + 2] = m.z; mu[4 * k4 + 3] = m.w;
            sg[4 * k4] = g.x; sg[4 * k4 + 1] = g.y; sg[4 * k4 + 2] = g.z; sg[4 * k4 + 3] = g.w;
        }
        const uint8_t *plane = which == 0 ? k_plane : v_plane;
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
            int qa[8], qr[8];
            if (FULL) {
                const uint2 cw = *reinterpret_cast<const uint2 *>(plane + row * kCodeRow + 8 * d8);
#pragma unroll
                for (int j = 0; j < 8; ++j) {
                    const uint32_t c = ((j < 4 ? cw.x : cw.y) >> (8 * (j & 3))) & 0xffu;
                    qa[j] = sext4(c >> 4);
                    qr[j] = sext4(c & 15u);
                }
            } else {
                const uint32_t w = *reinterpret_cast<const uint32_t *>(plane + row * kNibbleRow + 4 * d8);
#pragma unroll
                for (int j = 0; j < 8; ++j) {
                    qa[j] = sext4((w >> (4 * j)) & 15u);
                    qr[j] = 0;
                }
            }
            uint32_t o[4];
#pragma unroll
            for (int j = 0; j < 8; j += 2) {
                uint32_t hb[2];
#pragma unroll
                for (int u = 0; u < 2; ++u) {
                    const int a = qa[j + u];
                    const int V = a >= 0 ? a : -a - 1;
                    float lv;
                    if (variant == kHBiased) {
                        int Ip = 16 * V - qr[j + u];
                        Ip = Ip < 0 ? 0 : (Ip > 127 ? 127 : Ip);
                        lv = s_level[Ip];
                    } else if (variant == kHCentred) {
                        lv = FULL ? s_level[16 * V + 8 + qr[j + u]] : s_alevel[V];
                    } else {
                        lv = s_level[V];
                    }
                    const float m = a >= 0 ? lv : -lv;
                    const float xc = mul_rn(m, sg[j + u]);
                    const float X = xc + mu[j + u];
                    const float x = mul_rn(X, gs[j + u]) + gm[j + u];
                    hb[u] = bf16_rne(x);
                }
                o[j / 2] = hb[0] | (hb[1] << 16);
            }
            *reinterpret_cast<uint4 *>(out + ((size_t)t * Hkv + h) * kHeadDim + 8 * d8) =
                make_uint4(o[0], o[1], o[2], o[3]);
        }
    }
}

int shift_of(int bt) {
    for (int sh = 0; sh < 31; ++sh)
        if ((1 << sh) == bt) return sh;
    return -1;
}

}  // namespace

void make_htables(float alpha, int variant, HTables *t) {
    const double la = log1p((double)alpha);
    const int M = variant == kHInt4 ? 7 : 127;
    for (int k = 0; k < 128; ++k)
        t->theta[k] = k < M ? (float)(expm1(((k + 0.5) / M) * la) / (double)alpha) : INFINITY;
    for (int i = 0; i < 128; ++i)
        t->level[i] = (float)(expm1(((double)(i < M ? i : M) / M) * la) / (double)alpha);
    for (int v = 0; v < 8; ++v) t->alevel[v] = (float)(expm1(((16 * v + 7.5) / 127.0) * la) / (double)alpha);
    t->alpha = alpha;
    t->levels = M;
    t->linear = alpha < 1e-3f ? 1 : 0;
    t->yscale = t->linear ? (float)M : (float)(M / log2(1.0 + (double)alpha));
}

hipError_t launch_hencode(const Geometry &g, int b, int T, const int32_t *block_table,
                          const uint16_t *k, const uint16_t *v, uint8_t *k_anc, uint8_t *v_anc,
                          uint8_t *k_res, uint8_t *v_res, HMetaPtrs meta, const HTables &tab,
                          int variant, hipStream_t stream) {
    if (T <= 0) return hipSuccess;
    dim3 grid(g.Hkv, (T + kPage - 1) / kPage, 2);
    if (g.max_blocks == 1)
        hipLaunchKernelGGL(hencode_kernel<0>, grid, dim3(kHThreads), 0, stream, g, b, T, shift_of(g.bt),
                           block_table, k, v, k_anc, v_anc, k_res, v_res, meta, tab, variant);
    else
        hipLaunchKernelGGL(hencode_kernel<1>, grid, dim3(kHThreads), 0, stream, g, b, T, shift_of(g.bt),
                           block_table, k, v, k_anc, v_anc, k_res, v_res, meta, tab, variant);
    return hipGetLastError();
}

hipError_t launch_hdequant(bool full, const Geometry &g, int b, int T, const int32_t *block_table,
                           const uint8_t *k_plane, const uint8_t *v_plane, HMetaPtrs meta,
                           const HTables &tab, int variant, uint16_t *k_out, uint16_t *v_out,
                           hipStream_t stream) {
    if (T <= 0) return hipSuccess;
    size_t blocks = ((size_t)2 * ((T + 7) / 8) * g.Hkv * 16 + kHThreads - 1) / kHThreads;
    if (blocks > 256 * 32) blocks = 256 * 32;
    const dim3 grid((unsigned)blocks);
    const int sh = shift_of(g.bt);
    if (full) {
        if (g.max_blocks == 1)
            hipLaunchKernelGGL((hdequant_kernel<1, 0>), grid, dim3(kHThreads), 0, stream, g, b, T, sh,
                               block_table, k_plane, v_plane, meta, tab, variant, k_out, v_out);
        else
            hipLaunchKernelGGL((hdequant_kernel<1, 1>), grid, dim3(kHThreads), 0, stream, g, b, T, sh,
                               block_table, k_plane, v_plane, meta, tab, variant, k_out, v_out);
    } else {
        if (g.max_blocks == 1)
            hipLaunchKernelGGL((hdequant_kernel<0, 0>), grid, dim3(kHThreads), 0, stream, g, b, T, sh,
                               block_table, k_plane, v_plane, meta, tab, variant, k_out, v_out);
        else
            hipLaunchKernelGGL((hdequant_kernel<0, 1>), grid, dim3(kHThreads), 0, stream, g, b, T, sh,
                               block_table, k_plane, v_plane, meta, tab, variant, k_out, v_out);
    }
    return hipGetLastError();
}

}  // namespace lynx
