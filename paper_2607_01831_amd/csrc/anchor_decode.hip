// Anchor-phase decode attention on matrix cores (gfx950 MFMA).
//
// What it computes (Sec. 4.2 Anchor phase; attention of Sec. 2): for one
// query token per sequence and every query head, O = softmax(q K^T/sqrt(128)) V
// where K and V are reconstructed from the 4-bit anchor nibbles alone as
// zero + (16 a + 7.5) scale.
//
// Why matrix cores: with G query heads per kv head every token costs 2 x 128 x G
// multiply-adds but only 144 bytes, so plain fp32 vector arithmetic cannot keep
// up with HBM once G >= 4.  The contraction is a real dense product
// (G x 128 x tokens), so it runs as v_mfma_f32_16x16x32_bf16; the vector units
// only unpack nibbles and run the softmax.
//
// Exactness of the operands:
//  * a nibble n becomes the bf16 value 128 + n (bit pattern 0x4300 | n), one
//    v_perm per two values; the 128 offset is removed after the product.
//  * the K scale is folded into the query: q'_d = 16 c q_d s_d per 128-token
//    group (c = log2(e) / sqrt(128), so the products come out as softmax
//    exponents in log2 units), carried as bf16 hi + bf16 lo (two MFMAs, ~16
//    significant bits); zero, the 7.5 bucket centre and the 128 offset enter
//    a per-group bias c sum_d q_d (z_d - 2040.5 s_d), the accumulator's
//    initial value.
//  * the V scale is folded into the softmax weight: p'_t = p_t s_t (bf16);
//    the zero/centre term sum_t p_t (z_t + 7.5 s_t) is a per-head scalar and
//    the 128 offset is measured by one extra MFMA against a constant operand.
//
// Work split: grid = (context split of NG 128-token groups, kv head x head
// chunk, sequence); 4 wavefronts per workgroup, two workgroups per CU.
// Wavefront w owns the groups w, w + 4, ... of the split: it folds each
// group's K scales into its own MFMA operand lanes of the query (registers)
// and attends the group's four 32-token tiles with its own online softmax,
// so the loop has no barrier.  Tiles stream into a private 2-slot LDS ring
// by global-to-LDS copies, one tile ahead of the one being attended (no
// registers held by loads in flight), each with its V metadata; a group's K
// metadata rides with its first tile.  At the end the wavefronts are merged
// through LDS into one partial (max, sum, output) per head.
//
// Split merge in the same launch: each workgroup stores its partial with
// agent-coherent stores, waits for them and counts in on its (sequence, kv
// head, head chunk) counter; the last to arrive merges the splits' partials,
// writes the output and lse, and resets the counter.  A second, dependent
// launch costs 4 us on this part (8 us while a copy engine streams the
// residual).  With a BF16 tail the combine kernel of attention.hip merges
// instead.
#include "lane_ops.h"
#include "split_merge.h"
#include "lynx_internal.h"

#include <float.h>
#include <math.h>

namespace lynx {

namespace {

typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8_t;

constexpr int kThreads = 256;
constexpr int kWaves = 4;
constexpr int kTile = 32;  // tokens per wavefront step
constexpr float kLog2e = 1.4426950408889634f;

__device__ __forceinline__ f32x4_t mfma(u32x4_t a, u32x4_t b, f32x4_t c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, a),
                                                  __builtin_bit_cast(bf16x8_t, b), c, 0, 0, 0);
}

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }
typedef float f32x2_t __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
// Two floats -> two bf16 (round to nearest even) in one word, a in the low half.
__device__ __forceinline__ uint32_t pack2(float a, float b) {
    return __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2_t){a, b}, bf16x2_t));
}

// Eight nibbles of one 32-bit word (nibble j = element j) -> eight bf16
// values 128 + n in MFMA k-order (j = 0, 2, 4, 6, 1, 3, 5, 7).
__device__ __forceinline__ u32x4_t nibbles_to_bf16(uint32_t w) {
    const uint32_t lo = w & 0x0F0F0F0Fu;
    const uint32_t hi = (w >> 4) & 0x0F0F0F0Fu;
    const uint32_t c = 0x43434343u;
    u32x4_t r;
    r[0] = __builtin_amdgcn_perm(c, lo, 0x04010400u);
    r[1] = __builtin_amdgcn_perm(c, lo, 0x04030402u);
    r[2] = __builtin_amdgcn_perm(c, hi, 0x04010400u);
    r[3] = __builtin_amdgcn_perm(c, hi, 0x04030402u);
    return r;
}

// Ring slot of one tile: K rows (32 x 64 B), V rows (32 x 64 B), then the
// tile's V scales [32] and zeros [32].  Two slots per wavefront: a third
// (two tiles ahead) puts more requests in flight at the start, and every
// wavefront's first tile arrives later (32K layer 15.3 -> 15.8 us per call,
// paged batch 148 -> 154 us, 70B batch 114.7 -> 115.9 us).
constexpr int kDepth = 2;
constexpr int kPlaneTile = kTile * kNibbleRow;           // 2 KB
constexpr int kVMetaOff = 2 * kPlaneTile;
constexpr int kSlotBytes = kVMetaOff + 2 * kTile * 4;    // 4.25 KB
constexpr int kKMetaBytes = 2 * kHeadDim * 4;            // K scales [128], zeros [128]

// K rows in LDS: 16-byte chunk q of row t sits at chunk q ^ ((t >> 1) & 3),
// so the 8 lanes of one ds_read_b128 phase (rows t..t+7, same chunk) touch 8
// different bank groups.  V rows keep their natural layout for the
// transposed reads.
__device__ __forceinline__ uint32_t k_slot(int t, int q) {
    return (uint32_t)t * kNibbleRow + (uint32_t)((q ^ ((t >> 1) & 3)) * 16);
}

// LAYOUT 0: one block per sequence (contiguous cache, max_blocks_per_seq == 1)
// LAYOUT 1: paged, block_tokens a multiple of 16 (a 16-token run is in one block)
// LAYOUT 2: any other paging (per-token block lookups)
// GP: heads per chunk, padded (4, 8 or 16); NG: 128-token groups per split.
template <int GP, int LAYOUT, int NG>
__global__ __launch_bounds__(kThreads, 2) void anchor_decode_kernel(DecodeArgs a) {
    constexpr int kMaxGroups = NG / kWaves;  // groups per wavefront
    static_assert(NG % kWaves == 0, "groups must split evenly over the wavefronts");
    const int Hkv = a.geo.Hkv;
    // Grid (split, kv head x chunk, sequence) for the contiguous layout.  A
    // paged block holds the rows of every kv head for its tokens side by side,
    // so paged layouts make the kv head the fastest grid index: workgroups
    // reading the same blocks run together and share DRAM pages.
    const int split = LAYOUT == 0 ? blockIdx.x : blockIdx.y;
    const int hc = LAYOUT == 0 ? blockIdx.y : blockIdx.x;
    const int h = hc % Hkv;
    const int chunk = hc / Hkv;
    const int b = blockIdx.z;
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int w = tid >> 6;
    const int col = lane & 15;  // MFMA column (head) / 16-lane row index
    const int kg = lane >> 4;   // MFMA row group
    const int heads = min(a.chunk_heads, a.G - chunk * a.chunk_heads);
    const int T = max(0, min(a.seq_lens[b], a.max_seq_len));
    const int g0 = split * NG;
    // groups of this split that hold tokens (uniform across the workgroup)
    const int n_groups = max(0, min(NG, (T - g0 * kKGroup + kKGroup - 1) / kKGroup));
    const size_t q_row0 = (size_t)b * a.Hq + (size_t)h * a.G + (size_t)chunk * a.chunk_heads;

    // splits holding tokens (one for an empty sequence)
    const int live = max(1, (T + NG * kKGroup - 1) / (NG * kKGroup));
    if (a.fused && split >= live) return;  // nothing to attend, nothing to merge
    if (n_groups == 0 && a.fused) {
        // split 0 of an empty sequence: zero output, lse -inf
        const size_t orow0 = (size_t)b * a.Hq + (size_t)h * a.G + (size_t)chunk * a.chunk_heads;
        for (int idx = tid; idx < heads * (kHeadDim / 4); idx += kThreads)
            *reinterpret_cast<uint2 *>(a.out + (orow0 + idx / (kHeadDim / 4)) * kHeadDim +
                                       4 * (idx % (kHeadDim / 4))) = make_uint2(0u, 0u);
        if (a.lse && tid < heads) a.lse[orow0 + tid] = -INFINITY;
        return;
    }
    if (n_groups == 0) {
        // a split past the context: (max, sum) = (-inf, 0), no output
        for (int hh = tid; hh < heads; hh += kThreads) {
            const size_t pi =
                (((size_t)b * Hkv + h) * a.rows_total + chunk * a.chunk_heads + hh) * a.ws_splits + split;
            a.ws_ml[pi] = make_float2(-INFINITY, 0.0f);
        }
        return;
    }

    // LDS: 39-43 KB, two workgroups per CU; the epilogue reuses the ring
    __shared__ __attribute__((aligned(16))) uint8_t s_ring[kWaves * kDepth * kSlotBytes];
    __shared__ __attribute__((aligned(16))) uint8_t s_km[kWaves][kKMetaBytes];
    __shared__ __attribute__((aligned(16))) uint8_t s_q[GP * kHeadDim * 2];  // BF16 query rows
    static_assert((kWaves * GP * (kHeadDim + 4) + 2 * GP) * 4 <= kWaves * kDepth * kSlotBytes,
                  "the epilogue's arrays must fit in the ring");

    bool bad = false;
    const int32_t *bt_row = a.block_table + (size_t)b * a.geo.max_blocks;
    const size_t vmeta = ((size_t)b * Hkv + h) * a.geo.max_tokens;
    const size_t kmeta = ((size_t)b * Hkv + h) * a.geo.n_groups * kHeadDim;
    const size_t blk0_rows =
        LAYOUT == 0 ? ((size_t)min(max(bt_row[0], 0), a.geo.num_blocks - 1) * Hkv + h) * a.geo.bt : 0;
    if (LAYOUT == 0 && (bt_row[0] < 0 || bt_row[0] >= a.geo.num_blocks)) bad = true;

    // Row index (not bytes) of token t in the nibble planes.
    auto row_of = [&](int t) -> size_t {
        if (LAYOUT == 0) return blk0_rows + (size_t)t;
        const int bi = a.bt_shift >= 0 ? (t >> a.bt_shift) : t / a.geo.bt;
        int blk = bt_row[bi];
        if (blk < 0 || blk >= a.geo.num_blocks) {
            bad = true;
            blk = 0;
        }
        return ((size_t)blk * Hkv + h) * a.geo.bt + (size_t)(t - bi * a.geo.bt);
    };

    // This wavefront's tiles: tile j is tile j % 4 of its group j / 4, the
    // split's group w + 4 (j / 4).
    const int n_mine = n_groups > w ? (n_groups - w + kWaves - 1) / kWaves : 0;
    auto tile_t0 = [&](int j) { return (g0 + w + kWaves * (j >> 2)) * kKGroup + kTile * (j & 3); };
    auto tile_valid = [&](int j) { return (j >> 2) < n_mine && tile_t0(j) < T; };

    const float kscore = kLog2e * rsqrtf((float)kHeadDim);

    // ---- copies into the ring ----
    // Lane l of a 1 KB tile copy fills row 16 i + l / 4, physical chunk l % 4
    // of the plane's 32 rows (i = instruction 0 or 1).
    const int crow = lane >> 2;
    const int kq = (lane & 3) ^ ((lane >> 3) & 3);  // logical K chunk of that slot
    const uint32_t ring = lds_addr(s_ring) + (uint32_t)w * kDepth * kSlotBytes;
    const uint8_t *ring_p = s_ring + (size_t)w * kDepth * kSlotBytes;
    const uint32_t km = lds_addr(&s_km[w][0]);
    // copies per tile: 2 K + 2 V + 1 V metadata, + 1 K metadata (into the
    // wavefront's K-metadata buffer) for a group's first tile

    // LAYOUT 1: the block of every 16-token run the wavefront attends (lane
    // 8 u + r: run r of its group u), looked up once before any copy is in
    // flight; a full tile's copies then take their blocks by readlane
    // instead of waiting on a block-table load each.  Lanes past the
    // wavefront's groups read a clamped, unused entry.
    int run_blk = 0;
    if (LAYOUT == 1) {
        const int u = lane >> 3;
        if (u < kMaxGroups) {
            const int tr = (g0 + w + kWaves * u) * kKGroup + 16 * (lane & 7);
            const int bi = a.bt_shift >= 0 ? (tr >> a.bt_shift) : tr / a.geo.bt;
            run_blk = bt_row[min(bi, a.geo.max_blocks - 1)];
        }
        // the compiler places its wait for the load before this use: ahead of
        // every copy, whose waits it does not see
        asm volatile("" : "+v"(run_blk));
    }

    // Tile j of this wavefront into ring slot j % kDepth.
    auto issue_tile = [&](int j) {
        const int t0 = __builtin_amdgcn_readfirstlane(tile_t0(j));
        const uint32_t slot = ring + (uint32_t)(j % kDepth) * kSlotBytes;
        if (LAYOUT != 2 && t0 + kTile <= T) {
            // two 16-token runs, each inside one block
#pragma unroll
            for (int i = 0; i < 2; ++i) {
                size_t row0;
                if (LAYOUT == 0) {
                    row0 = blk0_rows + (size_t)(t0 + 16 * i);
                } else {
                    const int tr = t0 + 16 * i;
                    const int bi = a.bt_shift >= 0 ? (tr >> a.bt_shift) : tr / a.geo.bt;
                    // run 2 (j % 4) + i of the wavefront's group j / 4
                    int blk = __builtin_amdgcn_readlane(run_blk, 8 * (j >> 2) + 2 * (j & 3) + i);
                    if (blk < 0 || blk >= a.geo.num_blocks) {
                        bad = true;
                        blk = 0;
                    }
                    row0 = ((size_t)blk * Hkv + h) * a.geo.bt + (size_t)(tr - bi * a.geo.bt);
                }
                const size_t rb = row0 * kNibbleRow;
                const uint32_t off = (uint32_t)crow * kNibbleRow;
                lds_copy16(a.k_anc + rb, off + 16u * kq, slot + 1024u * i);
                lds_copy16(a.v_anc + rb, off + 16u * (lane & 3), slot + kPlaneTile + 1024u * i);
            }
        } else {
            // per-lane rows; rows past the context repeat the last token
#pragma unroll
            for (int i = 0; i < 2; ++i) {
                const int t = min(t0 + 16 * i + crow, T - 1);
                const size_t rb = row_of(t) * kNibbleRow;
                lds_copy16(a.k_anc + rb + 16 * kq, slot + 1024u * i);
                lds_copy16(a.v_anc + rb + 16 * (lane & 3), slot + kPlaneTile + 1024u * i);
            }
        }
        // V scale (lanes 0..31) and zero (lanes 32..63) of the tile's tokens;
        // tokens past the context repeat the last one
        {
            const int t = min(t0 + (lane & 31), T - 1);
            lds_copy4((lane < 32 ? a.meta.v_scale : a.meta.v_zero) + vmeta + t, slot + kVMetaOff);
        }
        // K scale (lanes 0..31) and zero (lanes 32..63) of the group
        if ((j & 3) == 0) {
            const int g = g0 + min(w + kWaves * (j >> 2), n_groups - 1);
            const float *src = (lane < 32 ? a.meta.k_scale : a.meta.k_zero) + kmeta + (size_t)g * kHeadDim;
            lds_copy16(src + 4 * (lane & 31), km);
        }
    };

    // The query rows of the chunk (GP / 4 copies of four 256-byte rows; heads
    // past the chunk repeat the last), fetched by wavefront 0 before its
    // first tiles.
    if (w == 0) {
#pragma unroll
        for (int k = 0; k < GP / 4; ++k) {
            const int hh = min(4 * k + (lane >> 4), heads - 1);
            lds_copy16(a.q + (q_row0 + hh) * kHeadDim + 8 * (lane & 15), lds_addr(s_q) + 1024u * k);
        }
    }
    // this lane's query values: head col, dims 32 kg .. + 31 (the dims of its
    // MFMA operand pieces), times 16 c
    float q16[32];
    auto load_query = [&]() {
        const uint4 *qp = reinterpret_cast<const uint4 *>(s_q + min(col, GP - 1) * (kHeadDim * 2) + 64 * kg);
        const bool live = col < heads;
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            const uint4 u = qp[k];
            const uint32_t wv[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                q16[8 * k + 2 * e] = live ? (16.0f * kscore) * bf16_lo(wv[e]) : 0.0f;
                q16[8 * k + 2 * e + 1] = live ? (16.0f * kscore) * bf16_hi(wv[e]) : 0.0f;
            }
        }
    };

    // ---- per-wave online-softmax state (lane: column col, token group kg) ----
    float m_run = -INFINITY, l_part = 0.0f, ob_part = 0.0f;
    f32x4_t acc[8], acc_off;
    auto reset_state = [&]() {
        m_run = -INFINITY;
        l_part = ob_part = 0.0f;
#pragma unroll
        for (int n = 0; n < 8; ++n) acc[n] = f32x4_t{0.f, 0.f, 0.f, 0.f};
        acc_off = f32x4_t{0.f, 0.f, 0.f, 0.f};
    };
    reset_state();
    const u32x4_t c128 = {0x43004300u, 0x43004300u, 0x43004300u, 0x43004300u};

    // Fold of a group (K scales and zeros from the K-metadata buffer):
    // q'_d = 16 c q_d s_d as bf16 hi + lo operands in k-order
    // (0, 2, 4, 6, 1, 3, 5, 7) within each 8 dims, and the bias
    // c sum_d q_d (z_d - 2040.5 s_d) of head col, the scores' initial value.
    u32x4_t bq[8];
    f32x4_t bk4;
    auto fold = [&]() {
        const float *ks = reinterpret_cast<const float *>(&s_km[w][0]) + 32 * kg;
        const float *kz = ks + kHeadDim;
        float bias = 0.0f;
#pragma unroll
        for (int kk = 0; kk < 4; ++kk) {
            const float4 s0 = reinterpret_cast<const float4 *>(ks)[2 * kk];
            const float4 s1 = reinterpret_cast<const float4 *>(ks)[2 * kk + 1];
            const float4 z0 = reinterpret_cast<const float4 *>(kz)[2 * kk];
            const float4 z1 = reinterpret_cast<const float4 *>(kz)[2 * kk + 1];
            const float sv[8] = {s0.x, s0.y, s0.z, s0.w, s1.x, s1.y, s1.z, s1.w};
            const float zv[8] = {z0.x, z0.y, z0.z, z0.w, z1.x, z1.y, z1.z, z1.w};
            float x[8];
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                x[e] = q16[8 * kk + e] * sv[e];
                bias = fmaf(q16[8 * kk + e], fmaf(-2040.5f, sv[e], zv[e]), bias);
            }
            // k-order pairs: dims (0, 2), (4, 6), (1, 3), (5, 7)
            const int ord[8] = {0, 2, 4, 6, 1, 3, 5, 7};
            u32x4_t hi, lo;
#pragma unroll
            for (int e = 0; e < 8; e += 2) {
                const float y0 = x[ord[e]], y1 = x[ord[e + 1]];
                const uint32_t hp = pack2(y0, y1);
                hi[e / 2] = hp;
                lo[e / 2] = pack2(y0 - bf16_lo(hp), y1 - bf16_hi(hp));
            }
            bq[2 * kk] = hi;
            bq[2 * kk + 1] = lo;
        }
        const float bk = sum_kg(bias) * 0.0625f;  // q16 carries 16 c
        bk4 = f32x4_t{bk, bk, bk, bk};
    };
    // Scores of tile j (log2 units): lane (col, kg) gets token
    // t0 + 16 r + 4 kg + i in x[4 r + i]; tokens past the context get -inf.
    auto tile_scores = [&](const uint8_t *slot_p, int j, float (&x)[8]) {
        f32x4_t sc[2];
#pragma unroll
        for (int r = 0; r < 2; ++r) {
            sc[r] = bk4;  // the bias enters as the initial accumulator
            const uint4 u = *reinterpret_cast<const uint4 *>(slot_p + k_slot(16 * r + col, kg));
            const uint32_t kw[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
            for (int kk = 0; kk < 4; ++kk) {
                const u32x4_t av = nibbles_to_bf16(kw[kk]);
                sc[r] = mfma(av, bq[2 * kk + 0], sc[r]);
                sc[r] = mfma(av, bq[2 * kk + 1], sc[r]);
            }
        }
#pragma unroll
        for (int i = 0; i < 8; ++i) x[i] = sc[i >> 2][i & 3];
        const int t0 = tile_t0(j);
        if (t0 + kTile > T) {
            asm volatile("" ::: "memory");  // keep the masking out of full tiles
#pragma unroll
            for (int i = 0; i < 8; ++i) {
                const int t = t0 + 16 * (i >> 2) + 4 * kg + (i & 3);
                x[i] = t < T ? x[i] : -INFINITY;
            }
        }
    };
    auto tile_max = [&](const float (&x)[8]) {
        return max_kg(fmax3(fmax3(x[0], x[1], x[2]), fmax3(x[3], x[4], x[5]), fmax2(x[6], x[7])));
    };
    // LDS transpose-read offset of the V rows for the PV operands.  Lane
    // (col, kg) names row col of its 16-lane group: token
    // tau(kg, col % 8) = 16 (col % 8 / 4) + 4 kg + col % 4 of the tile, 8-byte
    // chunk (col / 8) of dims; ds_read_b64_tr_b4 then hands lane (col, kg)
    // nibble col of the group's 16 rows = dim 16 c + col of 8 tokens (first
    // dword) and dim 16 (c + 1) + col (second dword) for chunk pair c.
    const uint32_t v_tr =
        (uint32_t)(16 * ((col & 7) >> 2) + 4 * kg + (col & 3)) * kNibbleRow + 8u * (col >> 3);
    // Softmax weights against the reference m_run, then P V for the tile.
    auto tile_accumulate = [&](const uint8_t *slot_p, const float (&x)[8]) {
        const float *vsm = reinterpret_cast<const float *>(slot_p + kVMetaOff) + 4 * kg;
        const float4 vs0 = *reinterpret_cast<const float4 *>(vsm);
        const float4 vs1 = *reinterpret_cast<const float4 *>(vsm + 16);
        const float4 vz0 = *reinterpret_cast<const float4 *>(vsm + kTile);
        const float4 vz1 = *reinterpret_cast<const float4 *>(vsm + kTile + 16);
        const float vsv[8] = {vs0.x, vs0.y, vs0.z, vs0.w, vs1.x, vs1.y, vs1.z, vs1.w};
        const float vzv[8] = {vz0.x, vz0.y, vz0.z, vz0.w, vz1.x, vz1.y, vz1.z, vz1.w};
        float pw[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const float p = __builtin_amdgcn_exp2f(x[i] - m_run);
            l_part += p;
            ob_part = fmaf(p, vzv[i], ob_part);
            pw[i] = p * vsv[i];
        }
        // softmax weights as the A operand, k-order (0, 2, 4, 6, 1, 3, 5, 7)
        u32x4_t pa;
        pa[0] = pack2(pw[0], pw[2]);
        pa[1] = pack2(pw[4], pw[6]);
        pa[2] = pack2(pw[1], pw[3]);
        pa[3] = pack2(pw[5], pw[7]);
        // values: transposed nibbles straight from the ring slot
        const uint8_t *vl = slot_p + kPlaneTile + v_tr;
#pragma unroll
        for (int c = 0; c < 8; c += 2) {
            const intx2_t vt = __builtin_amdgcn_ds_read_tr4_b64_v2i32(
                (__attribute__((address_space(3))) intx2_t *)(vl + 8 * c));
            acc[c] = mfma(pa, nibbles_to_bf16((uint32_t)vt[0]), acc[c]);
            acc[c + 1] = mfma(pa, nibbles_to_bf16((uint32_t)vt[1]), acc[c + 1]);
        }
        acc_off = mfma(pa, c128, acc_off);
    };

    // Fast path: the softmax reference of each head is the maximum of the
    // wavefront's first tile and stays fixed, so the loop carries no rescale.
    // Weights of later, larger scores exceed 1; if any sum leaves the safe
    // range the wavefront redoes its tiles below with a running maximum.
    // The next tile is in flight while one is attended; no barriers.
    // copies of a tile at position c of its group: 5, and 6 for a group's first
    auto copies_at = [](int c) { return (c & 3) == 0 ? 6 : 5; };
    static_assert(kDepth - 1 <= 4, "the ring reaches at most into the next group");
    if (n_mine > 0) {
#pragma unroll
        for (int c = 0; c < kDepth - 1; ++c) issue_tile(c);  // all in the first group
    }
    if (w == 0) {
        // the query rows are in once only the first tiles' copies remain
        int later = 0;
#pragma unroll
        for (int c = 0; c < kDepth - 1; ++c) later += copies_at(c);
        wait_vmcnt_folded(later);
    }
    __syncthreads();  // the query rows are visible to every wavefront
    load_query();
    for (int u = 0; u < kMaxGroups; ++u) {
        if (u >= n_mine) break;  // wavefront-uniform
        const bool next_group = u + 1 < n_mine;
#pragma unroll
        for (int c = 0; c < 4; ++c) {
            const int j = 4 * u + c;
            // tile j + kDepth - 1: inside this group, or in the next one
            if (c + kDepth - 1 < 4 || next_group) issue_tile(j + kDepth - 1);
            // tile j is in once only the later tiles' copies may remain in
            // flight (counts the unrolled loop folds to constants)
            int later_here = 0, later_next = 0;
#pragma unroll
            for (int k = 1; k < kDepth; ++k) {
                later_next += copies_at(c + k);
                if (c + k < 4) later_here += copies_at(c + k);
            }
            if (next_group) {
                wait_vmcnt_folded(later_next);
            } else {
                wait_vmcnt_folded(later_here);
            }
            const uint8_t *slot_p = ring_p + (j % kDepth) * kSlotBytes;
            if (c == 0) fold();
            if (tile_valid(j)) {
                float x[8];
                tile_scores(slot_p, j, x);
                if (j == 0) m_run = tile_max(x);
                tile_accumulate(slot_p, x);
            }
            // the slot and the K-metadata buffer are rewritten by later
            // copies: their reads must be done
            asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
        }
    }
    bool unsafe = !(l_part < 1e30f) || !(fabsf(ob_part) < 1e30f);
#pragma unroll
    for (int n = 0; n < 8; ++n)
#pragma unroll
        for (int i = 0; i < 4; ++i) unsafe |= !(fabsf(acc[n][i]) < 1e30f);
#pragma unroll
    for (int i = 0; i < 4; ++i) unsafe |= !(fabsf(acc_off[i]) < 1e30f);
    if (__any(unsafe)) {
        // Slow path (this wavefront only): running maximum with rescaling,
        // one tile fetched and waited for at a time.
        reset_state();
        for (int j = 0; j < 4 * n_mine; ++j) {
            issue_tile(j);
            wait_vmcnt<0>();
            const uint8_t *slot_p = ring_p + (j % kDepth) * kSlotBytes;
            if ((j & 3) == 0) fold();
            if (tile_valid(j)) {
                float x[8];
                tile_scores(slot_p, j, x);
                const float mx = tile_max(x);
                if (__any(mx > m_run)) {
                    const float m_new = fmaxf(mx, m_run);
                    const float alpha = (m_run == -INFINITY) ? 0.0f : exp2f(m_run - m_new);
                    m_run = m_new;
                    l_part *= alpha;
                    ob_part *= alpha;
                    float af[4];
#pragma unroll
                    for (int i = 0; i < 4; ++i) af[i] = __shfl(alpha, 4 * kg + i);
#pragma unroll
                    for (int n = 0; n < 8; ++n)
#pragma unroll
                        for (int i = 0; i < 4; ++i) acc[n][i] *= af[i];
#pragma unroll
                    for (int i = 0; i < 4; ++i) acc_off[i] *= af[i];
                }
                tile_accumulate(slot_p, x);
            }
            asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
        }
    }
    wait_vmcnt<0>();  // no copy may land in the ring once it is reused below

    // ---- per-wavefront totals -> LDS ----
    // o = sum_t p_t z_t + 16 sum_t pw_t a_t + 7.5 sum_t pw_t, with
    // acc = sum pw (128 + a) and acc_off = 128 sum pw.
    l_part = sum_kg(l_part);
    ob_part = sum_kg(ob_part);
    __syncthreads();  // every wavefront is done with its ring
    // ring reused: o [wave][GP][128], then max, sum, sum p z and merge
    // factors [wave][GP], and (M, L) per head
    float *s_o = reinterpret_cast<float *>(s_ring);
    float(*s_m)[GP] = reinterpret_cast<float(*)[GP]>(s_o + kWaves * GP * kHeadDim);
    float(*s_l)[GP] = s_m + kWaves;
    float(*s_ob)[GP] = s_l + kWaves;
    float(*s_f)[GP] = s_ob + kWaves;
    float(*s_ML)[2] = reinterpret_cast<float(*)[2]>(s_f + kWaves);
    if (kg == 0 && col < heads) {
        s_m[w][col] = m_run;
        s_l[w][col] = l_part;
        s_ob[w][col] = ob_part;
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int hh = 4 * kg + i;
        if (hh < heads && hh < GP) {
#pragma unroll
            for (int c = 0; c < 8; ++c)
                s_o[(w * GP + hh) * kHeadDim + 16 * c + col] = 16.0f * acc[c][i] - (16.0f - 7.5f / 128.0f) * acc_off[i];
        }
    }
    const bool any_bad = __syncthreads_or(bad);

    // ---- merge the wavefronts, write this split's partial: per-head
    // factors first, then float4 multiply-adds ----
    if (tid < heads) {
        const int hh = tid;
        float M = -INFINITY;
#pragma unroll
        for (int ww = 0; ww < kWaves; ++ww) M = fmaxf(M, s_m[ww][hh]);
        float L = 0.0f;
#pragma unroll
        for (int ww = 0; ww < kWaves; ++ww) {
            const float f = (M == -INFINITY || s_m[ww][hh] == -INFINITY) ? 0.0f : exp2f(s_m[ww][hh] - M);
            s_f[ww][hh] = f;
            L = fmaf(s_l[ww][hh], f, L);
        }
        s_ML[hh][0] = M;
        s_ML[hh][1] = any_bad ? NAN : L;
    }
    __syncthreads();
    // the pair's partials: rows chunk * chunk_heads .. + heads - 1 of (b, h)
    const size_t prow0 = ((size_t)b * Hkv + h) * a.rows_total + (size_t)chunk * a.chunk_heads;
    const __amdgpu_buffer_rsrc_t pair_o =
        buffer_rsrc(a.ws_o + prow0 * a.ws_splits * kHeadDim, (uint32_t)heads * a.ws_splits * kHeadDim * 4);
    const __amdgpu_buffer_rsrc_t pair_ml = buffer_rsrc(a.ws_ml + prow0 * a.ws_splits, (uint32_t)heads * a.ws_splits * 8);
    for (int idx = tid; idx < heads * (kHeadDim / 4); idx += kThreads) {
        const int hh = idx / (kHeadDim / 4);
        const int d4 = idx % (kHeadDim / 4);
        float4 O = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
        for (int ww = 0; ww < kWaves; ++ww) {
            const float f = s_f[ww][hh];
            const float ob = s_ob[ww][hh];
            const float4 o = reinterpret_cast<const float4 *>(s_o + (ww * GP + hh) * kHeadDim)[d4];
            O.x = fmaf(o.x + ob, f, O.x);
            O.y = fmaf(o.y + ob, f, O.y);
            O.z = fmaf(o.z + ob, f, O.z);
            O.w = fmaf(o.w + ob, f, O.w);
        }
        if (any_bad) O = make_float4(NAN, NAN, NAN, NAN);
        const int gr = chunk * a.chunk_heads + hh;  // row = head within the kv group
        const size_t pi = (((size_t)b * Hkv + h) * a.rows_total + gr) * a.ws_splits + split;
        if (a.fused) {
            const uint32_t sp = (uint32_t)hh * a.ws_splits + split;  // within the pair's rows
            store16_agent(pair_o, (sp * kHeadDim + 4 * d4) * 4, O);
            if (d4 == 0) store8_agent(pair_ml, sp * 8, make_float2(s_ML[hh][0], s_ML[hh][1]));
        } else {
            reinterpret_cast<float4 *>(a.ws_o + pi * kHeadDim)[d4] = O;
            if (d4 == 0) a.ws_ml[pi] = make_float2(s_ML[hh][0], s_ML[hh][1]);
        }
    }
    if (!a.fused) return;

    // ---- fused merge: count in; the pair's last workgroup merges ----
    __shared__ int s_last;
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");  // this thread's partial stores are done
    __syncthreads();                                    // ... and every other thread's
    unsigned *ctr = a.counters + (((size_t)b * Hkv + h) * a.row_chunks + chunk) * kCounterStride;
    if (tid == 0)
        s_last = __hip_atomic_fetch_add(ctr, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) ==
                 (unsigned)(live - 1);
    __syncthreads();
    if (!s_last) return;
    if (tid == 0) __hip_atomic_store(ctr, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    const size_t orow0 = (size_t)b * a.Hq + (size_t)h * a.G + (size_t)chunk * a.chunk_heads;
    merge_pair<GP>(a, pair_o, pair_ml, orow0, heads, live, s_ring);
}

template <int LAYOUT, int NG>
void launch_layout(const DecodeArgs &args, dim3 grid, hipStream_t stream) {
    if (args.chunk_heads <= 4) {
        hipLaunchKernelGGL((anchor_decode_kernel<4, LAYOUT, NG>), grid, dim3(kThreads), 0, stream, args);
    } else if (args.chunk_heads <= 8) {
        hipLaunchKernelGGL((anchor_decode_kernel<8, LAYOUT, NG>), grid, dim3(kThreads), 0, stream, args);
    } else {
        hipLaunchKernelGGL((anchor_decode_kernel<16, LAYOUT, NG>), grid, dim3(kThreads), 0, stream, args);
    }
}

template <int NG>
void launch_groups(const DecodeArgs &args, dim3 grid, hipStream_t stream) {
    if (args.geo.max_blocks == 1) {
        launch_layout<0, NG>(args, grid, stream);
    } else if (args.geo.bt % 16 == 0) {
        launch_layout<1, NG>(args, grid, stream);
    } else {
        launch_layout<2, NG>(args, grid, stream);
    }
}

}  // namespace

hipError_t launch_anchor_decode_mfma(const DecodeArgs &args, int chunks, hipStream_t stream) {
    // kv head fastest for paged layouts (the kernel reads the grid the same way)
    if (args.geo.max_blocks != 1 && args.n_splits > 65535) return hipErrorInvalidValue;
    const unsigned hc = (unsigned)(args.geo.Hkv * chunks);
    const dim3 grid = args.geo.max_blocks == 1 ? dim3(args.n_splits, hc, args.B) : dim3(hc, args.n_splits, args.B);
    if (args.groups_per_split == 4) {
        launch_groups<4>(args, grid, stream);
    } else if (args.groups_per_split == 8) {
        launch_groups<8>(args, grid, stream);
    } else if (args.groups_per_split == 16) {
        launch_groups<16>(args, grid, stream);
    } else if (args.groups_per_split == 32 && args.geo.max_blocks == 1) {
        // the long splits of one-round contiguous batches (plan_attention)
        launch_layout<0, 32>(args, grid, stream);
    } else if (args.groups_per_split == 64 && args.geo.max_blocks == 1) {
        launch_layout<0, 64>(args, grid, stream);
    } else {
        return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

}  // namespace lynx
