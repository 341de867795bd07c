// Anchor-phase decode over the anchors of the other split widths (gfx950,
// fp16 matrix cores).
//
// What it computes (Sec. 4.2 Anchor phase with the widths of Sec. 8): the
// uniform 8-bit code c of every K/V element split into an A-bit anchor
// a = c >> R and an R-bit residual (R = 8 - A, A in 2, 4, 6); before the
// residual arrives the anchor alone stands for code 2^R a + (2^R - 1) / 2,
// the middle of the codes it covers, so the cache reads
//   k = z + (2^R a + (2^R - 1) / 2) s,
// and one query per sequence attends it: o = softmax(q K^T / sqrt(128)) V.
// Planes hold a token's 128 anchors as a little-endian bit string of 16 A
// bytes (element e at bits e A .. e A + A - 1).
//
// The anchor value is a code dequantization with adjusted metadata:
// k = z' + a s' with s' = 2^R s and z' = z + (2^R - 1) / 2 s, so the
// attention is the code attention of the verification kernel over the
// A-bit values a < 64: the K scale s' is folded into the query rows (fp16
// hi + lo, exponent E per group and row), z' enters a per-(group, row) bias,
// and the V scale s' rides on the softmax weight with a 2^-Ev factor that
// keeps the fp16 weights at most 1.  The operands are the exact fp16 values
// of a (the byte trick 1024 + a, then one packed fp16 subtraction of 1024 per
// two values): with s' = 2^R s the fold's exponent grows by R, and an offset
// of 1024 carried through the fp32 accumulation would cost 2^R times the
// rounding of the code kernels in the scores.
//
// Work split: grid = (context split, kv head x chunk of 16 query heads,
// sequence); 4 wavefronts per workgroup, wavefront w owning the split's
// groups w, w + 4, ...  Per 32-token tile a wavefront loads (plain loads,
// the next tile's issued before the current one is attended) its lanes'
// K fields, unpacks them to bytes and straight into the MFMA operand
// registers (lane (col, kg) takes dims 32 kg .. + 31 of token col of each
// 16-token half: 4 A bytes), and unpacks the tile's V fields into byte rows
// of a per-wavefront LDS tile, read back transposed (ds_read_b64_tr_b8) as
// the P V operand.  The softmax keeps a running maximum (rescaling when a
// tile raises it).  The four wavefronts merge through LDS into one partial
// per split.  When the grid runs in one round the last workgroup of each
// (sequence, kv head, row chunk) merges the splits in the same launch (as
// the 4-bit decode does); otherwise the combine kernel merges them.
#include "f16_ops.h"
#include "lane_ops.h"
#include "lynx_internal.h"
#include "split_merge.h"

#include <math.h>

namespace lynx {

namespace {

constexpr int kThreads = 256;
constexpr int kWaves = 4;
constexpr int kTile = 32;
constexpr int kRows = 16;  // query rows (heads) per workgroup
constexpr float kLog2e = 1.4426950408889634f;
constexpr int kVTileBytes = kTile * kCodeRow;  // 32 V rows of 128 code bytes
constexpr int kKMetaFloats = 2 * kHeadDim;     // s' [128] | z' [128] of a group

// Bits [p, p + 32) of a little-endian bit string held in words w[0 .. n).
template <int N>
__device__ __forceinline__ uint32_t bits32(const uint32_t (&w)[N], int p) {
    const int i = p >> 5, sh = p & 31;
    const uint32_t lo = w[i];
    const uint32_t hi = i + 1 < N ? w[i + 1] : 0u;
    return sh == 0 ? lo : (lo >> sh) | (hi << (32 - sh));
}

// 32 A-bit fields (the bit string w, field e at bits e A ..) -> 32 bytes
// (8 words, byte e = field e).
template <int A, int N>
__device__ __forceinline__ void fields_to_bytes(const uint32_t (&w)[N], uint32_t (&b)[8]) {
    constexpr uint32_t mask = (1u << A) - 1u;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
        const uint32_t x = bits32(w, 4 * A * j);  // fields 4 j .. 4 j + 3
        b[j] = (x & mask) | (((x >> A) & mask) << 8) | (((x >> (2 * A)) & mask) << 16) |
               (((x >> (3 * A)) & mask) << 24);
    }
}

// Eight byte values a (two words, byte e = element e) -> eight exact fp16
// values a in element order: 1024 + a by byte permutes, less 1024.
__device__ __forceinline__ u32x4_t bytes_to_f16(uint32_t w0, uint32_t w1) {
    const u32x4_t r = codes_to_f16(w0, w1);
    const f16x2_t off = {(_Float16)-1024.0f, (_Float16)-1024.0f};
    u32x4_t o;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        // through a scalar copy: a bit cast of the vector element itself
        // compiles to element 0 for every i with this compiler
        const uint32_t ri = r[i];
        f16x2_t h;
        __builtin_memcpy(&h, &ri, 4);
        h = h + off;
        uint32_t oi;
        __builtin_memcpy(&oi, &h, 4);
        o[i] = oi;
    }
    return o;
}

// Loads of n consecutive words from a 4-byte-aligned address.
template <int N>
__device__ __forceinline__ void load_words(const uint8_t *p, uint32_t (&w)[N]) {
    const uint32_t *q = reinterpret_cast<const uint32_t *>(p);
    if constexpr (N % 4 == 0 && N > 0) {
#pragma unroll
        for (int i = 0; i < N; i += 4) {
            const uint4 v = *reinterpret_cast<const uint4 *>(q + i);
            w[i] = v.x;
            w[i + 1] = v.y;
            w[i + 2] = v.z;
            w[i + 3] = v.w;
        }
    } else {
#pragma unroll
        for (int i = 0; i < N; i += 2) {
            const uint2 v = *reinterpret_cast<const uint2 *>(q + i);
            w[i] = v.x;
            w[i + 1] = v.y;
        }
    }
}

// One tile's loads for one lane: K fields of tokens 16 r + col (r = 0, 1),
// dims 32 kg .. + 31; V fields of token lane / 2, dims 64 (lane % 2) .. + 63;
// V scale and zero of token lane % 32; with a group's first tile, K scale and
// zero of dims 2 lane, 2 lane + 1.
template <int A>
struct TileRegs {
    uint32_t k[2][A];
    uint32_t v[2 * A];
    float vs, vz;
    float2 ks, kz;
};

// LAYOUT 0: one block per sequence (contiguous); 1: any paging.
// SG: 128-token groups per split (4, 8 or 16).
template <int A, int LAYOUT, int SG>
__global__ __launch_bounds__(kThreads, 2) void anchor_split_decode_kernel(SplitDecodeArgs a) {
    constexpr int R = 8 - A;
    constexpr int kRowBytes = 16 * A;
    constexpr int kMaxGroups = SG / kWaves;
    static_assert(SG % kWaves == 0, "groups must split evenly over the wavefronts");
    const float centre = (float)((1 << R) - 1) * 0.5f;
    const int Hkv = a.geo.Hkv;
    const int split = blockIdx.x;
    const int hc = blockIdx.y;
    const int h = hc % Hkv;
    const int chunk = hc / Hkv;
    const int b = blockIdx.z;
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int w = tid >> 6;
    const int col = lane & 15;
    const int kg = lane >> 4;
    const int T = max(0, min(a.seq_lens[b], a.max_seq_len));
    const int g0 = split * SG;
    const int n_groups = max(0, min(SG, (T - g0 * kKGroup + kKGroup - 1) / kKGroup));
    const int row_base = chunk * kRows;
    const float kscore = kLog2e * rsqrtf((float)kHeadDim);
    auto partial_index = [&](int r) {
        return (((size_t)b * Hkv + h) * a.rows_total + r) * a.ws_splits + split;
    };
    const int heads = min(kRows, a.rows_total - row_base);  // live query rows of the chunk
    // splits holding tokens (one for an empty sequence)
    const int live = max(1, (T + SG * kKGroup - 1) / (SG * kKGroup));
    if (a.fused && split >= live) return;  // nothing to attend, nothing to merge
    if (n_groups == 0) {
        if (a.fused) {  // split 0 of an empty sequence: zero output, lse -inf
            const size_t orow0 = (size_t)b * a.Hq + (size_t)h * a.G + row_base;
            for (int idx = tid; idx < heads * (kHeadDim / 4); idx += kThreads)
                *reinterpret_cast<uint2 *>(a.out + (orow0 + idx / (kHeadDim / 4)) * kHeadDim +
                                           4 * (idx % (kHeadDim / 4))) = make_uint2(0u, 0u);
            if (a.lse && tid < heads) a.lse[orow0 + tid] = -INFINITY;
            return;
        }
        // a split past the context: (max, sum) = (-inf, 0)
        for (int r = tid; r < kRows; r += kThreads)
            if (row_base + r < a.rows_total) a.ws_ml[partial_index(row_base + r)] = make_float2(-INFINITY, 0.0f);
        return;
    }

    // LDS: query rows; per wavefront its V byte tile, the tile's V scales
    // and zeros, and its group's K scales and zeros; the epilogue reuses the
    // V tiles and metadata
    constexpr int kWaveBytes = kVTileBytes + 2 * kTile * 4 + kKMetaFloats * 4;
    constexpr int kEpilogueBytes = (kWaves * kRows * (kHeadDim + 4)) * 4;
    constexpr int kBufBytes = kWaves * kWaveBytes > kEpilogueBytes ? kWaves * kWaveBytes : kEpilogueBytes;
    __shared__ __attribute__((aligned(16))) uint8_t s_buf[kBufBytes];
    __shared__ __attribute__((aligned(16))) uint8_t s_q[kRows * kHeadDim * 2];
    __shared__ int s_ev[kWaves];
    __shared__ float s_ML[kRows][2];
    uint8_t *s_vt = s_buf + (size_t)w * kWaveBytes;                           // V byte rows
    float *s_vm = reinterpret_cast<float *>(s_vt + kVTileBytes);              // s' [32] | z' [32]
    float *s_km = s_vm + 2 * kTile;                                           // s' [128] | z' [128]

    bool bad = false;
    const int32_t *bt_row = a.block_table + (size_t)b * a.geo.max_blocks;
    const size_t vmeta = ((size_t)b * Hkv + h) * a.geo.max_tokens;
    const size_t kmeta = ((size_t)b * Hkv + h) * a.geo.n_groups * kHeadDim;
    const int blk0 = LAYOUT == 0 ? min(max(bt_row[0], 0), a.geo.num_blocks - 1) : 0;
    if (LAYOUT == 0 && (bt_row[0] < 0 || bt_row[0] >= a.geo.num_blocks)) bad = true;
    // plane row of token t (tokens past the context are clamped by the caller)
    auto row_of = [&](int t) -> size_t {
        if (LAYOUT == 0) return ((size_t)blk0 * Hkv + h) * a.geo.bt + (size_t)t;
        const int bi = t / a.geo.bt;
        int blk = bt_row[bi];
        if (blk < 0 || blk >= a.geo.num_blocks) {
            bad = true;
            blk = 0;
        }
        return ((size_t)blk * Hkv + h) * a.geo.bt + (size_t)(t - bi * a.geo.bt);
    };

    // this wavefront's tiles: tile j is tile j % 4 of its group j / 4, the
    // split's group w + 4 (j / 4)
    const int n_mine = n_groups > w ? (n_groups - w + kWaves - 1) / kWaves : 0;
    const int n_tiles = 4 * n_mine;
    auto tile_t0 = [&](int j) { return (g0 + w + kWaves * (j >> 2)) * kKGroup + kTile * (j & 3); };

    auto load_tile = [&](int j, TileRegs<A> &rg) {
        const int t0 = tile_t0(j);
#pragma unroll
        for (int r = 0; r < 2; ++r) {
            const int t = min(t0 + 16 * r + col, T - 1);
            load_words(a.k_anc + row_of(t) * kRowBytes + 4 * A * kg, rg.k[r]);
        }
        {
            const int t = min(t0 + (lane >> 1), T - 1);
            load_words(a.v_anc + row_of(t) * kRowBytes + 8 * A * (lane & 1), rg.v);
        }
        {
            const int t = min(t0 + (lane & 31), T - 1);
            rg.vs = a.meta.v_scale[vmeta + t];
            rg.vz = a.meta.v_zero[vmeta + t];
        }
        if ((j & 3) == 0) {
            const int g = g0 + w + kWaves * (j >> 2);
            rg.ks = reinterpret_cast<const float2 *>(a.meta.k_scale + kmeta + (size_t)g * kHeadDim)[lane];
            rg.kz = reinterpret_cast<const float2 *>(a.meta.k_zero + kmeta + (size_t)g * kHeadDim)[lane];
        }
    };

    // the first tile's loads, the query rows and the V scales go out together:
    // one round trip before the loop
    TileRegs<A> cur, nxt;
    if (n_tiles > 0) load_tile(0, cur);
    uint4 q4;
    {
        const int r = tid >> 4;  // 16 threads per 256-byte row (rows past the chunk's heads repeat the last)
        const int hh = min(row_base + r, a.rows_total - 1);
        const size_t qrow = (size_t)b * a.Hq + (size_t)h * a.G + hh;
        q4 = reinterpret_cast<const uint4 *>(a.q + qrow * kHeadDim)[tid & 15];
    }
    // ---- the largest adjusted V scale s' of the wavefront's tokens ----
    int Ev = 0;
    {
        float vm = 0.0f;
#pragma unroll
        for (int u = 0; u < kMaxGroups; ++u) {
#pragma unroll
            for (int k = 0; k < 2; ++k) {
                const int t = (g0 + w + kWaves * u) * kKGroup + 64 * k + lane;
                if (u < n_mine && t < T) vm = fmax2(vm, a.meta.v_scale[vmeta + t]);
            }
        }
        vm = max_kg(row16_max(vm)) * (float)(1 << R);
        if (vm > 0.0f) frexpf(vm, &Ev);
        Ev = max(Ev, -100);
    }

    reinterpret_cast<uint4 *>(s_q)[tid] = q4;
    __syncthreads();  // the query rows are in

    // ---- per-wavefront online-softmax state: lane (col = query row, kg);
    // the reference carries the 2^-Ev factor of the V weights ----
    float m_run = -INFINITY, m_ref = -INFINITY, l_part = 0.0f, ob_part = 0.0f;
    f32x4_t acc[8];
#pragma unroll
    for (int n = 0; n < 8; ++n) acc[n] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    const bool row_live = row_base + col < a.rows_total;

    // fold of a group from s' and z' in LDS: q''_d = q_d s'_d 2^-E as fp16
    // hi + lo, score scale 2^E kscore, bias kscore sum_d q_d z'_d
    u32x4_t bq[8];
    float bsc = 0.0f, bb = 0.0f;
    auto fold = [&]() {
        const float *ks = s_km + 32 * kg;
        const float *kz = s_km + kHeadDim + 32 * kg;
        const uint4 *qp = reinterpret_cast<const uint4 *>(s_q + col * (kHeadDim * 2) + 64 * kg);
        float mx = 0.0f, bias = 0.0f;
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            const uint4 u = qp[k];
            const float qv[8] = {bf16_lo(u.x), bf16_hi(u.x), bf16_lo(u.y), bf16_hi(u.y),
                                 bf16_lo(u.z), bf16_hi(u.z), bf16_lo(u.w), bf16_hi(u.w)};
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                const float sv = ks[8 * k + e], zv = kz[8 * k + e];
                mx = fmax2(mx, fabsf(qv[e] * sv));
                bias = fmaf(qv[e], zv, bias);
            }
        }
        mx = max_kg(mx);
        bias = sum_kg(bias);
        int E = 0;
        if (mx > 0.0f) frexpf(mx, &E);
#pragma unroll
        for (int kk = 0; kk < 4; ++kk) {
            const uint4 u = qp[kk];
            const float qv[8] = {bf16_lo(u.x), bf16_hi(u.x), bf16_lo(u.y), bf16_hi(u.y),
                                 bf16_lo(u.z), bf16_hi(u.z), bf16_lo(u.w), bf16_hi(u.w)};
            u32x4_t hi, lo;
#pragma unroll
            for (int e = 0; e < 8; e += 2) {
                const float y0 = row_live ? ldexpf(qv[e] * ks[8 * kk + e], -E) : 0.0f;
                const float y1 = row_live ? ldexpf(qv[e + 1] * ks[8 * kk + e + 1], -E) : 0.0f;
                const uint32_t hp = pack_f16(y0, y1);
                hi[e / 2] = hp;
                lo[e / 2] = pack_f16(y0 - f16_lo(hp), y1 - f16_hi(hp));
            }
            bq[2 * kk] = hi;
            bq[2 * kk + 1] = lo;
        }
        bsc = ldexpf(kscore, E);
        bb = row_live ? bias * kscore : 0.0f;
    };

    const int tr = 16 * ((col >> 1) >> 2) + 4 * kg + ((col >> 1) & 3);
    const int half = col & 1;

    for (int j = 0; j < n_tiles; ++j) {
        if (j + 1 < n_tiles) load_tile(j + 1, nxt);  // in flight while tile j is attended
        const int t0 = tile_t0(j);
        // V fields -> byte rows of the LDS tile; s', z' of the tile's tokens;
        // with a group's first tile its K s', z'
        {
            uint32_t bytes[2][8];
            uint32_t wv[A];
#pragma unroll
            for (int p = 0; p < 2; ++p) {
#pragma unroll
                for (int i = 0; i < A; ++i) wv[i] = cur.v[p * A + i];
                fields_to_bytes<A>(wv, bytes[p]);
            }
            const int t = lane >> 1;
#pragma unroll
            for (int p = 0; p < 2; ++p)
#pragma unroll
                for (int q2 = 0; q2 < 2; ++q2)
                    *reinterpret_cast<uint4 *>(s_vt + v_slot(t, 4 * (lane & 1) + 2 * p + q2)) =
                        make_uint4(bytes[p][4 * q2], bytes[p][4 * q2 + 1], bytes[p][4 * q2 + 2], bytes[p][4 * q2 + 3]);
            // lane l < 32: s' of token l; lane l >= 32: z' of token l - 32
            s_vm[lane] = lane < 32 ? ldexpf(cur.vs, R) : fmaf(centre, cur.vs, cur.vz);
            if ((j & 3) == 0) {
                s_km[2 * lane] = ldexpf(cur.ks.x, R);
                s_km[2 * lane + 1] = ldexpf(cur.ks.y, R);
                s_km[kHeadDim + 2 * lane] = fmaf(centre, cur.ks.x, cur.kz.x);
                s_km[kHeadDim + 2 * lane + 1] = fmaf(centre, cur.ks.y, cur.kz.y);
            }
        }
        asm volatile("" ::: "memory");  // the LDS writes above precede the reads below
        if ((j & 3) == 0) fold();

        // scores (log2 units): lane (col, kg) gets token t0 + 16 r + 4 kg + i
        // of query row col in x[4 r + i]
        float x[8];
        {
            f32x4_t sc[2];
#pragma unroll
            for (int r = 0; r < 2; ++r) {
                uint32_t kb[8];
                fields_to_bytes<A>(cur.k[r], kb);
                sc[r] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int kk = 0; kk < 4; ++kk) {
                    const u32x4_t av = bytes_to_f16(kb[2 * kk], kb[2 * kk + 1]);
                    sc[r] = mfma_f16(av, bq[2 * kk + 0], sc[r]);
                    sc[r] = mfma_f16(av, bq[2 * kk + 1], sc[r]);
                }
            }
#pragma unroll
            for (int i = 0; i < 8; ++i) x[i] = fmaf(sc[i >> 2][i & 3], bsc, bb);
            if (t0 + kTile > T) {
#pragma unroll
                for (int i = 0; i < 8; ++i) {
                    const int t = t0 + 16 * (i >> 2) + 4 * kg + (i & 3);
                    x[i] = t < T ? x[i] : -INFINITY;
                }
            }
        }
        // running maximum per row; rescale when the tile raises it
        {
            const float mx = max_kg(fmax3(fmax3(x[0], x[1], x[2]), fmax3(x[3], x[4], x[5]), fmax2(x[6], x[7])));
            if (__any(mx > m_run)) {
                const float m_new = fmaxf(mx, m_run);
                const float alpha = (m_run == -INFINITY) ? 0.0f : exp2f(m_run - m_new);
                m_run = m_new;
                m_ref = m_new + (float)Ev;
                l_part *= alpha;
                ob_part *= alpha;
                float af[4];
#pragma unroll
                for (int i = 0; i < 4; ++i) af[i] = __shfl(alpha, 4 * kg + i);
#pragma unroll
                for (int n = 0; n < 8; ++n)
#pragma unroll
                    for (int i = 0; i < 4; ++i) acc[n][i] *= af[i];
            }
        }
        // weights and P V
        {
            const float4 vs0 = *reinterpret_cast<const float4 *>(s_vm + 4 * kg);
            const float4 vs1 = *reinterpret_cast<const float4 *>(s_vm + 16 + 4 * kg);
            const float4 vz0 = *reinterpret_cast<const float4 *>(s_vm + kTile + 4 * kg);
            const float4 vz1 = *reinterpret_cast<const float4 *>(s_vm + kTile + 16 + 4 * kg);
            const float vsv[8] = {vs0.x, vs0.y, vs0.z, vs0.w, vs1.x, vs1.y, vs1.z, vs1.w};
            const float vzv[8] = {vz0.x, vz0.y, vz0.z, vz0.w, vz1.x, vz1.y, vz1.z, vz1.w};
            float pw[8];
#pragma unroll
            for (int i = 0; i < 8; ++i) {
                const float p = __builtin_amdgcn_exp2f(x[i] - m_ref);
                l_part += p;
                ob_part = fmaf(p, vzv[i], ob_part);
                pw[i] = p * vsv[i];
            }
            u32x4_t pa;
#pragma unroll
            for (int e = 0; e < 4; ++e) pa[e] = pack_f16_rne(pw[2 * e], pw[2 * e + 1]);
#pragma unroll
            for (int c = 0; c < 8; ++c) {
                const intx2_t vt = __builtin_amdgcn_ds_read_tr8_b64_v2i32(
                    (__attribute__((address_space(3))) intx2_t *)(s_vt + v_slot(tr, c) + 8 * half));
                acc[c] = mfma_f16(pa, bytes_to_f16((uint32_t)vt[0], (uint32_t)vt[1]), acc[c]);
            }
        }
        // the LDS tile and metadata are rewritten for the next tile: their
        // reads must be done
        asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
        if (j + 1 < n_tiles) cur = nxt;
    }

    // ---- per-wavefront totals -> LDS (still scaled by 2^-Ev) ----
    __syncthreads();  // every wavefront is done with its LDS tile
    float *s_o = reinterpret_cast<float *>(s_buf);
    float(*s_m)[kRows] = reinterpret_cast<float(*)[kRows]>(s_o + kWaves * kRows * kHeadDim);
    float(*s_l)[kRows] = s_m + kWaves;
    float(*s_ob)[kRows] = s_l + kWaves;
    float(*s_f)[kRows] = s_ob + kWaves;
    static_assert((kWaves * kRows * kHeadDim + 4 * kWaves * kRows) * 4 <= kBufBytes,
                  "the epilogue's arrays must fit");
    {
        const float l = sum_kg(l_part);
        const float ob = sum_kg(ob_part);
        if (kg == 0) {
            s_m[w][col] = m_run;
            s_l[w][col] = l;
            s_ob[w][col] = ob;
        }
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int c = 0; c < 8; ++c)
                s_o[(w * kRows + 4 * kg + i) * kHeadDim + 16 * c + col] = acc[c][i];
    }
    if (lane == 0) s_ev[w] = Ev;
    const bool any_bad = __syncthreads_or(bad);
    if (tid < kRows) {
        float M = -INFINITY;
#pragma unroll
        for (int ww = 0; ww < kWaves; ++ww) M = fmaxf(M, s_m[ww][tid]);
        float L = 0.0f;
#pragma unroll
        for (int ww = 0; ww < kWaves; ++ww) {
            const float f = (M == -INFINITY || s_m[ww][tid] == -INFINITY)
                                ? 0.0f
                                : exp2f(s_m[ww][tid] - M) * ldexpf(1.0f, s_ev[ww]);
            s_f[ww][tid] = f;
            L = fmaf(s_l[ww][tid], f, L);
        }
        s_ML[tid][0] = M;
        s_ML[tid][1] = any_bad ? NAN : L;
    }
    __syncthreads();
    // the chunk's partials: rows row_base .. + heads - 1 of (b, h)
    const size_t prow0 = ((size_t)b * Hkv + h) * a.rows_total + row_base;
    const __amdgpu_buffer_rsrc_t pair_o =
        buffer_rsrc(a.ws_o + prow0 * a.ws_splits * kHeadDim, (uint32_t)heads * a.ws_splits * kHeadDim * 4);
    const __amdgpu_buffer_rsrc_t pair_ml = buffer_rsrc(a.ws_ml + prow0 * a.ws_splits, (uint32_t)heads * a.ws_splits * 8);
    for (int idx = tid; idx < kRows * (kHeadDim / 4); idx += kThreads) {
        const int rr = idx / (kHeadDim / 4);
        const int d4 = idx % (kHeadDim / 4);
        const int row = row_base + rr;
        if (row >= a.rows_total) continue;
        float4 O = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
        for (int ww = 0; ww < kWaves; ++ww) {
            const float f = s_f[ww][rr];
            const float ob = s_ob[ww][rr];
            const float4 o = reinterpret_cast<const float4 *>(s_o + (ww * kRows + rr) * kHeadDim)[d4];
            O.x = fmaf(o.x + ob, f, O.x);
            O.y = fmaf(o.y + ob, f, O.y);
            O.z = fmaf(o.z + ob, f, O.z);
            O.w = fmaf(o.w + ob, f, O.w);
        }
        if (any_bad) O = make_float4(NAN, NAN, NAN, NAN);
        if (a.fused) {
            const uint32_t sp = (uint32_t)rr * a.ws_splits + split;  // within the chunk's rows
            store16_agent(pair_o, (sp * kHeadDim + 4 * d4) * 4, O);
            if (d4 == 0) store8_agent(pair_ml, sp * 8, make_float2(s_ML[rr][0], s_ML[rr][1]));
        } else {
            const size_t pi = partial_index(row);
            reinterpret_cast<float4 *>(a.ws_o + pi * kHeadDim)[d4] = O;
            if (d4 == 0) a.ws_ml[pi] = make_float2(s_ML[rr][0], s_ML[rr][1]);
        }
    }
    if (!a.fused) return;

    // ---- split merge: count in; the chunk's last workgroup merges ----
    __shared__ int s_last;
    unsigned *ctr = a.counters + (((size_t)b * Hkv + h) * a.row_chunks + chunk) * kCounterStride;
    if (!last_to_arrive(ctr, live, &s_last)) return;
    const size_t orow0 = (size_t)b * a.Hq + (size_t)h * a.G + row_base;
    if (heads <= 4)
        merge_pair<4>(a, pair_o, pair_ml, orow0, heads, live, s_buf);
    else if (heads <= 8)
        merge_pair<8>(a, pair_o, pair_ml, orow0, heads, live, s_buf);
    else
        merge_pair<16>(a, pair_o, pair_ml, orow0, heads, live, s_buf);
}

template <int A, int LAYOUT>
hipError_t launch_sg(const SplitDecodeArgs &args, dim3 grid, hipStream_t stream) {
    switch (args.groups_per_split) {
        case 4:
            hipLaunchKernelGGL((anchor_split_decode_kernel<A, LAYOUT, 4>), grid, dim3(kThreads), 0, stream, args);
            break;
        case 8:
            hipLaunchKernelGGL((anchor_split_decode_kernel<A, LAYOUT, 8>), grid, dim3(kThreads), 0, stream, args);
            break;
        case 16:
            hipLaunchKernelGGL((anchor_split_decode_kernel<A, LAYOUT, 16>), grid, dim3(kThreads), 0, stream, args);
            break;
        default:
            return hipErrorInvalidValue;
    }
    return hipSuccess;
}

template <int A>
hipError_t launch_a(const SplitDecodeArgs &args, dim3 grid, hipStream_t stream) {
    return args.geo.max_blocks == 1 ? launch_sg<A, 0>(args, grid, stream) : launch_sg<A, 1>(args, grid, stream);
}

}  // namespace

hipError_t launch_anchor_split_decode(const SplitDecodeArgs &args, hipStream_t stream) {
    const int chunks = (args.rows_total + kRows - 1) / kRows;
    const dim3 grid(args.n_splits, (unsigned)(args.geo.Hkv * chunks), args.B);
    hipError_t e;
    switch (args.anchor_bits) {
        case 2:
            e = launch_a<2>(args, grid, stream);
            break;
        case 4:
            e = launch_a<4>(args, grid, stream);
            break;
        case 6:
            e = launch_a<6>(args, grid, stream);
            break;
        default:
            return hipErrorInvalidValue;
    }
    if (e != hipSuccess) return e;
    return hipGetLastError();
}

}  // namespace lynx
