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
// Work split: grid = (context split, kv head x head chunk, sequence).  A
// workgroup (4 wavefronts) walks its split one 128-token K group at a time:
// the workgroup folds the group's scales into the query (shared through
// LDS), then each wavefront takes one 32-token tile of the group, keeping
// its own online softmax.  At the end the wavefronts are merged through LDS
// into one partial (max, sum, output) per head, which the combine kernel of
// attention.hip merges across splits.
#include "lane_ops.h"
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

__device__ __forceinline__ uint32_t bf16_bits(float x) {
    return (uint32_t)__builtin_bit_cast(unsigned short, (__bf16)x);
}
__device__ __forceinline__ float bf16_val(uint32_t bits16) { return __uint_as_float(bits16 << 16); }
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

// One wavefront's registers for one 32-token tile: 16-byte pieces of the K
// and V nibble rows (row col and col + 16 of the tile, dims 32 kg..32 kg+31).
struct Tile {
    uint4 k[2];
    uint4 v[2];
};

constexpr int kPrefetch = 3;  // tiles in flight ahead of the one being computed

// LAYOUT 0: one block per sequence (contiguous cache, max_blocks_per_seq == 1)
// LAYOUT 1: paged, block_tokens a multiple of 16 (a 16-token run is in one block)
// LAYOUT 2: any other paging (per-token block lookups)
// GP: heads per chunk, padded (4, 8 or 16); NG: 128-token groups per split.
template <int GP, int LAYOUT, int NG>
__global__ __launch_bounds__(kThreads, 2) void anchor_decode_kernel(DecodeArgs a) {
    const int Hkv = a.geo.Hkv;
    const int split = blockIdx.x;
    const int h = blockIdx.y % Hkv;
    const int chunk = blockIdx.y / Hkv;
    const int b = blockIdx.z;
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int w = tid >> 6;
    const int col = lane & 15;  // MFMA column / 16-lane row index
    const int kg = lane >> 4;   // MFMA row group
    const int heads = min(a.chunk_heads, a.G - chunk * a.chunk_heads);
    const int T = max(0, min(a.seq_lens[b], a.max_seq_len));
    const int g0 = split * NG;
    // groups of this split that hold tokens (uniform across the workgroup)
    const int n_groups = max(0, min(NG, (T - g0 * kKGroup + kKGroup - 1) / kKGroup));

    // The split is walked in rounds of 4 groups, one group per wavefront.
    // Folded query operands of a round: one 16-byte MFMA operand piece per
    // (group, kk, hi/lo, row group kg, head), double-buffered across rounds;
    // a trailing zero piece feeds the columns past the chunk's heads.
    constexpr int kRounds = NG / 4;
    constexpr int kBufs = kRounds > 1 ? 2 : 1;
    constexpr int kRoundPieces = 4 * 8 * 4 * GP;
    constexpr int kZeroPiece = kBufs * kRoundPieces;
    __shared__ u32x4_t s_b[kZeroPiece + 1];
    __shared__ float s_bias[kBufs][kWaves][4][GP];  // per-wavefront partial biases
    __shared__ __attribute__((aligned(16))) float s_vs[kBufs][4 * kKGroup];
    __shared__ __attribute__((aligned(16))) float s_vz[kBufs][4 * kKGroup];
    __shared__ __attribute__((aligned(16))) uint8_t s_v[kWaves][kTile * kNibbleRow];
    __shared__ __attribute__((aligned(16))) float s_o[kWaves][GP][kHeadDim];
    __shared__ float s_m[kWaves][GP], s_l[kWaves][GP], s_ob[kWaves][GP];

    const size_t vmeta = ((size_t)b * Hkv + h) * a.geo.max_tokens;
    const size_t kmeta = ((size_t)b * Hkv + h) * a.geo.n_groups * kHeadDim;
    const size_t q_row0 = (size_t)b * a.Hq + (size_t)h * a.G + (size_t)chunk * a.chunk_heads;
    const float kscore = kLog2e * rsqrtf((float)kHeadDim);

  if (n_groups > 0) {
    bool bad = false;
    const int32_t *bt_row = a.block_table + (size_t)b * a.geo.max_blocks;
    const u32x4_t c128 = {0x43004300u, 0x43004300u, 0x43004300u, 0x43004300u};

    // block of a contiguous cache (LAYOUT 0)
    const size_t blk0_rows =
        LAYOUT == 0 ? ((size_t)min(max(bt_row[0], 0), a.geo.num_blocks - 1) * Hkv + h) * a.geo.bt
                    : 0;
    if (LAYOUT == 0 && (bt_row[0] < 0 || bt_row[0] >= a.geo.num_blocks)) bad = true;

    // Row index (not bytes) of token t in the plane, generic form.
    auto row_generic = [&](int t) -> size_t {
        if (LAYOUT == 0) return blk0_rows + (size_t)t;
        const int bi = a.bt_shift >= 0 ? (t >> a.bt_shift) : t / a.geo.bt;
        int blk = bt_row[bi];
        if (blk < 0 || blk >= a.geo.num_blocks) {
            bad = true;
            blk = 0;
        }
        return ((size_t)blk * Hkv + h) * a.geo.bt + (size_t)(t - bi * a.geo.bt);
    };

    // ---- per-round metadata, loaded one round ahead into registers ----
    const int n_rounds = (n_groups + 3) / 4;
    // V metadata of a round's tokens (zero past the context)
    constexpr int kVmPer = 4 * kKGroup / kThreads;
    float vs_r[kVmPer], vz_r[kVmPer];
    // K scales and query pieces of the fold: piece (gl, kk, dg, hh) covers
    // dims 32 dg + 8 kk .. + 7 of head hh and group gl of the round.  Indices
    // are clamped into range; pieces past the heads or groups are zeroed.
    constexpr int kFoldPieces = 4 * 4 * 4 * GP;
    constexpr int kFoldPer = kFoldPieces / kThreads;
    static_assert(kFoldPieces % kThreads == 0, "fold pieces must tile the workgroup");
    float4 fs0[kFoldPer], fs1[kFoldPer];
    uint4 fq[kFoldPer];  // the query pieces are the same in every round
#pragma unroll
    for (int k = 0; k < kFoldPer; ++k) {
        const int pidx = tid + k * kThreads;
        const int hh = min(pidx % GP, heads - 1);
        const int d0 = 32 * ((pidx / GP) % 4) + 8 * ((pidx / (4 * GP)) % 4);
        fq[k] = *reinterpret_cast<const uint4 *>(a.q + (q_row0 + hh) * kHeadDim + d0);
    }
    // bias operands: query of head col, K scale/zero of group col of the round,
    // dims 32 w + 8 kg ..
    const uint4 bqw = *reinterpret_cast<const uint4 *>(
        a.q + (q_row0 + min(col, heads - 1)) * kHeadDim + 32 * w + 8 * kg);
    float4 bs0, bs1, bz0, bz1;
    auto load_round_meta = [&](int r) {
#pragma unroll
        for (int k = 0; k < kVmPer; ++k) {
            const int t = (g0 + 4 * r) * kKGroup + tid + k * kThreads;
            const size_t ti = vmeta + (size_t)min(t, T - 1);
            vs_r[k] = a.meta.v_scale[ti];
            vz_r[k] = a.meta.v_zero[ti];
            if (t >= T) vs_r[k] = vz_r[k] = 0.0f;
        }
#pragma unroll
        for (int k = 0; k < kFoldPer; ++k) {
            const int pidx = tid + k * kThreads;
            const int gl = min(4 * r + pidx / (16 * GP), n_groups - 1);
            const int d0 = 32 * ((pidx / GP) % 4) + 8 * ((pidx / (4 * GP)) % 4);
            const float *sp = a.meta.k_scale + kmeta + (size_t)(g0 + gl) * kHeadDim + d0;
            fs0[k] = *reinterpret_cast<const float4 *>(sp);
            fs1[k] = *reinterpret_cast<const float4 *>(sp + 4);
        }
        const int gc = min(4 * r + min(col, 3), n_groups - 1);
        const size_t mo = kmeta + (size_t)(g0 + gc) * kHeadDim + 32 * w + 8 * kg;
        bs0 = *reinterpret_cast<const float4 *>(a.meta.k_scale + mo);
        bs1 = *reinterpret_cast<const float4 *>(a.meta.k_scale + mo + 4);
        bz0 = *reinterpret_cast<const float4 *>(a.meta.k_zero + mo);
        bz1 = *reinterpret_cast<const float4 *>(a.meta.k_zero + mo + 4);
    };
    load_round_meta(0);

    // ---- this wavefront's tiles: groups w, w+4, ..; 4 tiles of 32 tokens each ----
    constexpr int kTilesPerWave = NG;  // (NG / 4) groups x 4 tiles
    auto tile_t0 = [&](int j) { return (g0 + w + 4 * (j >> 2)) * kKGroup + kTile * (j & 3); };
    auto tile_valid = [&](int j) { return (w + 4 * (j >> 2)) < n_groups && tile_t0(j) < T; };
    const uint32_t kv_lane = (uint32_t)col * kNibbleRow + 16u * kg;

    // Issue the K and V loads of tile j.  Full tiles address through a
    // uniform base plus constant lane offsets; a partial tile clamps its rows
    // to the last token (its scores are masked later).
    auto load_tile = [&](int j, Tile &tl) {
        const int t0 = __builtin_amdgcn_readfirstlane(tile_t0(j));
        if (LAYOUT != 2 && t0 + kTile <= T) {
#pragma unroll
            for (int r = 0; r < 2; ++r) {
                size_t row;
                if (LAYOUT == 0) {
                    row = blk0_rows + (size_t)(t0 + 16 * r);
                } else {
                    const int tr = t0 + 16 * r;
                    const int bi = a.bt_shift >= 0 ? (tr >> a.bt_shift) : tr / a.geo.bt;
                    int blk = bt_row[bi];
                    if (blk < 0 || blk >= a.geo.num_blocks) {
                        bad = true;
                        blk = 0;
                    }
                    row = ((size_t)blk * Hkv + h) * a.geo.bt + (size_t)(tr - bi * a.geo.bt);
                }
                tl.k[r] = *reinterpret_cast<const uint4 *>(a.k_anc + row * kNibbleRow + kv_lane);
                tl.v[r] = *reinterpret_cast<const uint4 *>(a.v_anc + row * kNibbleRow + kv_lane);
            }
        } else {
#pragma unroll
            for (int r = 0; r < 2; ++r) {
                const size_t row = row_generic(min(t0 + 16 * r + col, T - 1));
                tl.k[r] = *reinterpret_cast<const uint4 *>(a.k_anc + row * kNibbleRow + 16 * kg);
                tl.v[r] = *reinterpret_cast<const uint4 *>(a.v_anc + row * kNibbleRow + 16 * kg);
            }
        }
    };

    // Put the first tiles in flight before the fold below.
    // Loads of tiles past the context read clamped rows and are never used;
    // issuing them unconditionally keeps the wait counts exact.
    Tile tiles[kPrefetch + 1];
#pragma unroll
    for (int j = 0; j < kPrefetch; ++j)
        if (j < kTilesPerWave) load_tile(j, tiles[j]);

    // ---- fold of one round (whole workgroup): the groups' K scales into
    // the query, per-wavefront bias partials, V metadata into LDS ----
    auto fold_round = [&](int buf, int r) {
        // (a) Folded operands, one 16-byte piece (8 dims) at a time: piece
        // (gl, kk, dg, hh) holds q'_d = 16 c q_d s_d of dims 32 dg + 8 kk +
        // pi(e), as bf16 hi in s_b and bf16 lo 4 GP pieces further.
#pragma unroll
        for (int k = 0; k < kFoldPer; ++k) {
            const int pidx = tid + k * kThreads;
            const int hh = pidx % GP;
            const int dg = (pidx / GP) % 4;
            const int kk = (pidx / (4 * GP)) % 4;
            const int gl = pidx / (16 * GP);
            const bool live = hh < heads && 4 * r + gl < n_groups;
            const uint4 qw = fq[k];
            // dims d0 + (0, 2, 4, 6, 1, 3, 5, 7)
            const float qv[8] = {bf16_val(qw.x & 0xffffu), bf16_val(qw.y & 0xffffu),
                                 bf16_val(qw.z & 0xffffu), bf16_val(qw.w & 0xffffu),
                                 __uint_as_float(qw.x & 0xffff0000u), __uint_as_float(qw.y & 0xffff0000u),
                                 __uint_as_float(qw.z & 0xffff0000u), __uint_as_float(qw.w & 0xffff0000u)};
            const float4 s0 = fs0[k], s1 = fs1[k];
            const float sv[8] = {s0.x, s0.z, s1.x, s1.z, s0.y, s0.w, s1.y, s1.w};
            u32x4_t hi, lo;
#pragma unroll
            for (int e = 0; e < 8; e += 2) {
                const float q0 = live ? (16.0f * kscore) * qv[e] * sv[e] : 0.0f;
                const float q1 = live ? (16.0f * kscore) * qv[e + 1] * sv[e + 1] : 0.0f;
                const uint32_t hp = pack2(q0, q1);
                hi[e / 2] = hp;
                lo[e / 2] = pack2(q0 - bf16_val(hp & 0xffffu), q1 - __uint_as_float(hp & 0xffff0000u));
            }
            const int piece = buf * kRoundPieces + ((gl * 8 + kk * 2) * 4 + dg) * GP + hh;
            s_b[piece] = hi;
            s_b[piece + 4 * GP] = lo;
        }
        // (b) Biases bias[gl][hh] = c sum_d q_d (z_d - 2040.5 s_d) as a small
        // matrix product on the matrix cores: rows = heads, columns = the
        // round's groups, wavefront w contracting dims 32 w..32 w+31 (zc
        // carried as bf16 hi + lo); the four wavefront partials are summed
        // when a group's operands are loaded.
        {
            u32x4_t qa = {0u, 0u, 0u, 0u};
            if (col < heads) qa = u32x4_t{bqw.x, bqw.y, bqw.z, bqw.w};
            u32x4_t zh = {0u, 0u, 0u, 0u}, zl = {0u, 0u, 0u, 0u};
            if (col < 4 && 4 * r + col < n_groups) {
                const float zc[8] = {bz0.x - 2040.5f * bs0.x, bz0.y - 2040.5f * bs0.y,
                                     bz0.z - 2040.5f * bs0.z, bz0.w - 2040.5f * bs0.w,
                                     bz1.x - 2040.5f * bs1.x, bz1.y - 2040.5f * bs1.y,
                                     bz1.z - 2040.5f * bs1.z, bz1.w - 2040.5f * bs1.w};
#pragma unroll
                for (int e = 0; e < 8; e += 2) {
                    const uint32_t hp = pack2(zc[e], zc[e + 1]);
                    zh[e / 2] = hp;
                    zl[e / 2] = pack2(zc[e] - bf16_val(hp & 0xffffu), zc[e + 1] - __uint_as_float(hp & 0xffff0000u));
                }
            }
            f32x4_t cb = {0.f, 0.f, 0.f, 0.f};
            cb = mfma(qa, zh, cb);
            cb = mfma(qa, zl, cb);
            // lane (group col, row group kg) holds heads 4 kg + i
            if (col < 4) {
#pragma unroll
                for (int i = 0; i < 4; ++i)
                    if (4 * kg + i < GP) s_bias[buf][w][col][4 * kg + i] = cb[i] * kscore;
            }
        }
        // (c) V metadata
#pragma unroll
        for (int k = 0; k < kVmPer; ++k) {
            s_vs[buf][tid + k * kThreads] = vs_r[k];
            s_vz[buf][tid + k * kThreads] = vz_r[k];
        }
    };
    fold_round(0, 0);
    if (tid == 0) s_b[kZeroPiece] = u32x4_t{0u, 0u, 0u, 0u};
    if (n_rounds > 1) load_round_meta(1);
    __syncthreads();  // the first round's operands, biases and V metadata are ready

    // ---- per-wave online-softmax state (lane: column col, token group kg) ----
    float m_run = -INFINITY, l_part = 0.0f, ob_part = 0.0f;
    f32x4_t acc[8], acc_off;
#pragma unroll
    for (int n = 0; n < 8; ++n) acc[n] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    acc_off = f32x4_t{0.f, 0.f, 0.f, 0.f};

    // LDS transpose-read addresses of the V tile for the PV operands.  Lane
    // (col, kg) names row col of its 16-lane group: token
    // tau(kg, col % 8) = 16 (col % 8 / 4) + 4 kg + col % 4 of the tile, 8-byte
    // chunk (col / 8) of dims; ds_read_b64_tr_b4 then hands lane (col, kg)
    // nibble col of the group's 16 rows = dim 16 c + col of 8 tokens (first
    // dword) and dim 16 (c + 1) + col (second dword) for chunk pair c.
    const uint32_t v_tr_addr =
        (uint32_t)(16 * ((col & 7) >> 2) + 4 * kg + (col & 3)) * kNibbleRow + 8u * (col >> 3);
    const uint32_t v_wr_addr = (uint32_t)col * kNibbleRow + 16u * kg;  // + 1024 for run 1
    auto *vlds = &s_v[w][0];
    const int b_piece = col < GP ? kg * GP + col : -1;

    u32x4_t bq[8];
    float bk = 0.0f;
    f32x4_t bk4 = {0.f, 0.f, 0.f, 0.f};
    // Folded query operands and bias of this wavefront's group of a round.
    auto load_group_operands = [&](int buf) {
#pragma unroll
        for (int i = 0; i < 8; ++i)
            bq[i] = b_piece >= 0 ? s_b[buf * kRoundPieces + (w * 8 + i) * 4 * GP + b_piece]
                                 : s_b[kZeroPiece];
        bk = col < heads ? (s_bias[buf][0][w][col] + s_bias[buf][1][w][col]) +
                               (s_bias[buf][2][w][col] + s_bias[buf][3][w][col])
                         : 0.0f;
        bk4 = f32x4_t{bk, bk, bk, bk};
    };
    // Scores of tile j (log2 units): lane (col, kg) gets token
    // t0 + 16 r + 4 kg + i in x[4 r + i]; tokens past the context get -inf.
    // Also stages the tile's V rows in the wavefront's LDS slot.
    auto tile_scores = [&](const Tile &cur, int j, float (&x)[8]) {
        *reinterpret_cast<uint4 *>(vlds + v_wr_addr) = cur.v[0];
        *reinterpret_cast<uint4 *>(vlds + v_wr_addr + 16 * kNibbleRow) = cur.v[1];
        f32x4_t sc[2];
#pragma unroll
        for (int r = 0; r < 2; ++r) sc[r] = bk4;  // the bias enters as the initial accumulator
#pragma unroll
        for (int kk = 0; kk < 4; ++kk) {
#pragma unroll
            for (int r = 0; r < 2; ++r) {
                const uint32_t kw = kk == 0 ? cur.k[r].x : kk == 1 ? cur.k[r].y
                                  : kk == 2 ? cur.k[r].z : cur.k[r].w;
                const u32x4_t av = nibbles_to_bf16(kw);
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
    // Softmax weights against reference m_ref, then P V for tile j.
    auto tile_accumulate = [&](int buf, int j, const float (&x)[8]) {
        const int tl = w * kKGroup + kTile * (j & 3) + 4 * kg;
        const float4 vs0 = *reinterpret_cast<const float4 *>(&s_vs[buf][tl]);
        const float4 vs1 = *reinterpret_cast<const float4 *>(&s_vs[buf][tl + 16]);
        const float4 vz0 = *reinterpret_cast<const float4 *>(&s_vz[buf][tl]);
        const float4 vz1 = *reinterpret_cast<const float4 *>(&s_vz[buf][tl + 16]);
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
        // values: transposed nibbles straight from LDS
#pragma unroll
        for (int c = 0; c < 8; c += 2) {
            const intx2_t vt = __builtin_amdgcn_ds_read_tr4_b64_v2i32(
                (__attribute__((address_space(3))) intx2_t *)(vlds + v_tr_addr + 8 * c));
            acc[c] = mfma(pa, nibbles_to_bf16((uint32_t)vt[0]), acc[c]);
            acc[c + 1] = mfma(pa, nibbles_to_bf16((uint32_t)vt[1]), acc[c + 1]);
        }
        acc_off = mfma(pa, c128, acc_off);
    };

    // Fast path: the softmax reference of each head is the maximum of the
    // wavefront's first tile and stays fixed, so the loop carries no rescale.
    // Weights of later, larger scores exceed 1; if any sum leaves the safe
    // range the workgroup redoes the split below with a running maximum.
    // Each round ends with a barrier, after the next round's fold.
#pragma unroll
    for (int r = 0; r < kRounds; ++r) {
        if (r >= n_rounds) break;  // uniform across the workgroup
        const int buf = kBufs > 1 ? (r & 1) : 0;
        load_group_operands(buf);
#pragma unroll
        for (int jj = 0; jj < 4; ++jj) {
            const int j = 4 * r + jj;
            if (j + kPrefetch < kTilesPerWave)
                load_tile(j + kPrefetch, tiles[(j + kPrefetch) % (kPrefetch + 1)]);
            if (tile_valid(j)) {  // wavefront-uniform
                float x[8];
                tile_scores(tiles[j % (kPrefetch + 1)], j, x);
                if (j == 0) m_run = tile_max(x);
                tile_accumulate(buf, j, x);
            }
        }
        if (kRounds > 1) {
            if (r + 1 < n_rounds) {
                fold_round(buf ^ 1, r + 1);
                if (r + 2 < n_rounds) load_round_meta(r + 2);
            }
            __syncthreads();  // next round's operands in place; this round's buffer is free
        }
    }
    bool unsafe = !(l_part < 1e30f) || !(fabsf(ob_part) < 1e30f);
#pragma unroll
    for (int n = 0; n < 8; ++n)
#pragma unroll
        for (int i = 0; i < 4; ++i) unsafe |= !(fabsf(acc[n][i]) < 1e30f);
#pragma unroll
    for (int i = 0; i < 4; ++i) unsafe |= !(fabsf(acc_off[i]) < 1e30f);
    if (__syncthreads_or(unsafe)) {
        // Slow path (scores far above the first tile's): running maximum
        // with rescaling, one round and tile at a time.
        m_run = -INFINITY;
        l_part = ob_part = 0.0f;
#pragma unroll
        for (int n = 0; n < 8; ++n) acc[n] = f32x4_t{0.f, 0.f, 0.f, 0.f};
        acc_off = f32x4_t{0.f, 0.f, 0.f, 0.f};
        for (int r = 0; r < n_rounds; ++r) {
            load_round_meta(r);
            fold_round(0, r);
            __syncthreads();
            load_group_operands(0);
            for (int jj = 0; jj < 4; ++jj) {
                const int j = 4 * r + jj;
                if (!tile_valid(j)) continue;
                Tile cur;
                load_tile(j, cur);
                float x[8];
                tile_scores(cur, j, x);
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
                tile_accumulate(0, j, x);
            }
            __syncthreads();
        }
    }

    // ---- per-wavefront totals -> LDS ----
    // o = sum_t p_t z_t + 16 sum_t pw_t a_t + 7.5 sum_t pw_t, with
    // acc = sum pw (128 + a) and acc_off = 128 sum pw.
    l_part = sum_kg(l_part);
    ob_part = sum_kg(ob_part);
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
                s_o[w][hh][16 * c + col] = 16.0f * acc[c][i] - (16.0f - 7.5f / 128.0f) * acc_off[i];
        }
    }
    const bool any_bad = __syncthreads_or(bad);

    // ---- merge the wavefronts, write this split's partial: per-head
    // factors first, then float4 multiply-adds ----
    __shared__ float s_f[kWaves][GP], s_ML[GP][2];
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
    for (int idx = tid; idx < heads * (kHeadDim / 4); idx += kThreads) {
        const int hh = idx / (kHeadDim / 4);
        const int d4 = idx % (kHeadDim / 4);
        float4 O = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
        for (int ww = 0; ww < kWaves; ++ww) {
            const float f = s_f[ww][hh];
            const float ob = s_ob[ww][hh];
            const float4 o = reinterpret_cast<const float4 *>(&s_o[ww][hh][0])[d4];
            O.x = fmaf(o.x + ob, f, O.x);
            O.y = fmaf(o.y + ob, f, O.y);
            O.z = fmaf(o.z + ob, f, O.z);
            O.w = fmaf(o.w + ob, f, O.w);
        }
        if (any_bad) O = make_float4(NAN, NAN, NAN, NAN);
        const int gr = chunk * a.chunk_heads + hh;  // row = head within the kv group
        const size_t pi = (((size_t)b * Hkv + h) * a.rows_total + gr) * a.ws_splits + split;
        reinterpret_cast<float4 *>(a.ws_o + pi * kHeadDim)[d4] = O;
        if (d4 == 0) a.ws_ml[pi] = make_float2(s_ML[hh][0], s_ML[hh][1]);
    }
  } else {
    // a split past the context: (max, sum) = (-inf, 0), no output
    for (int hh = tid; hh < heads; hh += kThreads) {
        const size_t pi =
            (((size_t)b * Hkv + h) * a.rows_total + chunk * a.chunk_heads + hh) * a.ws_splits + split;
        a.ws_ml[pi] = make_float2(-INFINITY, 0.0f);
    }
  }
}

template <int LAYOUT, int NG>
void launch_layout(const DecodeArgs &args, dim3 grid, hipStream_t stream) {
    if (args.chunk_heads <= 4) {
        hipLaunchKernelGGL((anchor_decode_kernel<4, LAYOUT, NG>), grid, dim3(kThreads), 0, stream, args);
    } else if (args.chunk_heads <= 8) {
        hipLaunchKernelGGL((anchor_decode_kernel<8, LAYOUT, NG>), grid, dim3(kThreads), 0, stream, args);
    } else {
        // 16 heads per chunk keep the split at 4 groups (LDS budget)
        hipLaunchKernelGGL((anchor_decode_kernel<16, LAYOUT, 4>), grid, dim3(kThreads), 0, stream, args);
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
    dim3 grid(args.n_splits, args.geo.Hkv * chunks, args.B);
    if (args.groups_per_split == 4) {
        launch_groups<4>(args, grid, stream);
    } else if (args.groups_per_split == 8) {
        launch_groups<8>(args, grid, stream);
    } else if (args.groups_per_split == 16) {
        launch_groups<16>(args, grid, stream);
    } else {
        return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

}  // namespace lynx
