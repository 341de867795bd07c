// Verification attention on matrix cores (gfx950 MFMA, fp16 operands).
//
// What it computes (Sec. 4.3; attention of Sec. 2): the k draft queries of a
// sequence attend, in one pass, over the merged 8-bit cache, with K and V
// reconstructed as zero + code * scale.  This kernel covers the context
// tokens; the combine kernel of attention.hip merges its splits and attends
// the drafts' own BF16 K/V (the causal tail) as one more partial.
//
// Why matrix cores: with k * G query rows per kv head (32 for 8 drafts and
// G = 4) every context token costs 2 x 128 x 32 multiply-adds against 272
// bytes, above what fp32 vector arithmetic sustains at HBM speed; the
// contraction is dense, so Q K^T and P V run as v_mfma_f32_16x16x32_f16.
//
// Exactness of the operands:
//  * a code byte c becomes the fp16 value 1024 + c (bit pattern 0x6400 | c),
//    one v_perm per two values; the 1024 offset is removed after the product.
//  * per 128-token group the K scale is folded into the query rows:
//    q''_d = q_d s_d 2^-E (E per group and row, so |q''| < 1), carried as fp16
//    hi + lo through two MFMAs; zero and offset enter a per-(group, row) bias
//    sum_d q_d (z_d - 1024 s_d).
//  * the V scale is folded into the softmax weight, pw_t = p_t s_t 2^-Ev
//    (fp16, rounded to nearest; Ev per wavefront from the largest V scale of
//    its tokens, so pw <= 1 while p <= 1, and a weight beyond the fp16 range
//    becomes infinite and sends the wavefront to the running-maximum path);
//    sum_t p_t z_t is summed in fp32 and the offset is measured by one MFMA
//    against the constant 1024.  The 2^-Ev factor rides on the softmax
//    reference, so l, sum p z and the products all carry it and one multiply
//    restores it when the wavefronts are merged.
//
// Work split: grid = (context split of SG 128-token groups, kv head x chunk
// of 16 RT query rows, sequence); 4 wavefronts per workgroup, two
// workgroups per CU.  Wavefront w owns the groups w, w + 4, ... of the split
// and serves all RT row tiles from each of their 32-token tiles, so every
// K/V byte is fetched once per workgroup and the query fold of a group
// (q'' for the wavefront's own MFMA operand lanes) lives in its registers:
// no barrier inside the loop.  Tiles, each with its V metadata, stream
// into a private 2-slot LDS ring by global-to-LDS copies, one tile ahead
// of the one being attended (no registers held by loads in flight); a
// group's K metadata rides with its first tile, and the query rows are
// copied into LDS once.  At the end the four wavefronts merge through LDS
// into one partial per row and split.
#include "f16_ops.h"
#include "lane_ops.h"
#include "lynx_internal.h"

#include <math.h>

namespace lynx {

namespace {

constexpr int kThreads = 256;
constexpr int kWaves = 4;
constexpr int kTile = 32;      // tokens per wavefront step
constexpr float kLog2e = 1.4426950408889634f;

constexpr int kDepth = 2;                          // ring slots per wavefront
constexpr int kTileBytes = kTile * kCodeRow;       // one plane's 32 rows: 4 KB
constexpr int kVMetaOff = 2 * kTileBytes;          // V scale[32] | V zero[32] of the tile
constexpr int kSlotBytes = kVMetaOff + 2 * kTile * 4;  // 8.25 KB
constexpr int kKMetaBytes = 2 * kHeadDim * 4;      // K scale[128] | K zero[128] of a group

// K tile rows in LDS: 16-byte chunk q of row t sits at chunk q ^ (t & 7), so
// the 8 lanes of one ds_read_b128 phase (8 consecutive rows, same chunk)
// touch 8 different bank groups.
__device__ __forceinline__ uint32_t k_slot(int t, int q) {
    return (uint32_t)t * kCodeRow + (uint32_t)((q ^ (t & 7)) * 16);
}

// LAYOUT 0: one block per sequence; 1: paged, block_tokens a multiple of 16;
// 2: any other paging.  RT: 16-row query tiles per workgroup (1 or 2), all
// served by every wavefront.  SG: 128-token groups per split (4, 8 or 16).
template <int RT, int LAYOUT, int SG>
__global__ __launch_bounds__(kThreads, 2) void verify_kernel(VerifyArgs a) {
    constexpr int kRows = RT * 16;
    constexpr int NQ = kWaves;             // wavefront w takes groups w, w + 4, ...
    constexpr int kMaxGroups = SG / NQ;    // groups per wavefront
    static_assert(SG % NQ == 0, "groups must split evenly over the wavefronts");
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
    const int col = lane & 15;
    const int kg = lane >> 4;
    const int gq = w;  // this wavefront's groups: gq, gq + NQ, ...
    const int T = max(0, min(a.seq_lens[b], a.max_seq_len));
    const int g0 = split * SG;
    const int n_groups = max(0, min(SG, (T - g0 * kKGroup + kKGroup - 1) / kKGroup));
    const int row_base = chunk * kRows;  // first query row of the workgroup
    const float kscore = kLog2e * rsqrtf((float)kHeadDim);

    // query row r <-> (draft r / G, head r % G); its partial-output row
    auto partial_index = [&](int r) {
        return (((size_t)b * Hkv + h) * a.rows_total + r) * a.ws_splits + split;
    };

    if (n_groups == 0) {  // a split past the context: (max, sum) = (-inf, 0)
        for (int r = tid; r < kRows; r += kThreads)
            if (row_base + r < a.rows_total) a.ws_ml[partial_index(row_base + r)] = make_float2(-INFINITY, 0.0f);
        return;
    }

    // LDS: under 80 KB for RT = 2, so two workgroups share a CU; the
    // epilogue reuses the ring
    __shared__ __attribute__((aligned(16))) uint8_t s_ring[kWaves * kDepth * kSlotBytes];
    __shared__ __attribute__((aligned(16))) uint8_t s_km[kWaves][kKMetaBytes];
    __shared__ __attribute__((aligned(16))) uint8_t s_q[kRows * kHeadDim * 2];  // BF16 query rows
    __shared__ int s_ev[kWaves];
    __shared__ float s_ML[kRows][2];
    static_assert(kWaves * kRows * (kHeadDim + 4) * 4 <= kWaves * kDepth * kSlotBytes,
                  "the epilogue's arrays must fit in the ring");

    bool bad = false;
    const int32_t *bt_row = a.block_table + (size_t)b * a.geo.max_blocks;
    const size_t vmeta = ((size_t)b * Hkv + h) * a.geo.max_tokens;
    const size_t kmeta = ((size_t)b * Hkv + h) * a.geo.n_groups * kHeadDim;
    const size_t blk0_rows =
        LAYOUT == 0 ? ((size_t)min(max(bt_row[0], 0), a.geo.num_blocks - 1) * Hkv + h) * a.geo.bt : 0;
    if (LAYOUT == 0 && (bt_row[0] < 0 || bt_row[0] >= a.geo.num_blocks)) bad = true;

    // Row index (not bytes) of token t in the code planes.
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
    // split's group gq + NQ (j / 4).
    const int n_mine = n_groups > gq ? (n_groups - gq + NQ - 1) / NQ : 0;  // its groups
    auto group_of = [&](int j) { return gq + NQ * (j >> 2); };
    auto tile_t0 = [&](int j) { return (g0 + group_of(j)) * kKGroup + kTile * (j & 3); };
    auto tile_valid = [&](int j) { return (j >> 2) < n_mine && tile_t0(j) < T; };

    // ---- the largest V scale of the wavefront's tokens (plain loads, all
    // consumed before the first copy) ----
    int Ev = 0;
    {
        float vm = 0.0f;
#pragma unroll 4
        for (int u = 0; u < kMaxGroups; ++u) {
#pragma unroll
            for (int k = 0; k < 2; ++k) {
                const int t = (g0 + gq + NQ * u) * kKGroup + 64 * k + lane;
                if (u < n_mine && t < T) vm = fmax2(vm, a.meta.v_scale[vmeta + t]);
            }
        }
        vm = max_kg(row16_max(vm));
        if (vm > 0.0f) frexpf(vm, &Ev);
        // V scales below 2^-100 contribute below 255 * 2^-100 per token; the
        // clamp keeps 2^-Ev, and so the weights p 2^-Ev, finite
        Ev = max(Ev, -100);
    }
    // LAYOUT 1: the block of every 16-token run the wavefront attends (lane
    // 8 u + r: run r of its group u), looked up here so that a full tile's
    // copies take their blocks by readlane instead of waiting on a
    // block-table load each.  Lanes past the wavefront's groups read a
    // clamped, unused entry.
    int run_blk = 0;
    if (LAYOUT == 1) {
        const int u = lane >> 3;
        if (u < kMaxGroups) {
            const int tr = (g0 + gq + NQ * u) * kKGroup + 16 * (lane & 7);
            const int bi = a.bt_shift >= 0 ? (tr >> a.bt_shift) : tr / a.geo.bt;
            run_blk = bt_row[min(bi, a.geo.max_blocks - 1)];
        }
    }
    // every plain load has been consumed (Ev and run_blk depend on all of
    // them): nothing of the compiler's own is in flight once the copies start
    asm volatile("" ::"v"(Ev), "v"(run_blk) : "memory");
    wait_vmcnt<0>();

    // ---- copies into the ring ----
    // Lane l of a 1 KB tile copy fills row 8 i + l / 8, physical chunk l % 8
    // of the slot (i = instruction); these are the logical chunks it fetches.
    const int crow = lane >> 3;
    const int kq = (lane & 7) ^ crow;  // K, and V rows 0..15
    const uint32_t ring = lds_addr(s_ring) + (uint32_t)w * kDepth * kSlotBytes;
    const uint8_t *ring_p = s_ring + (size_t)w * kDepth * kSlotBytes;
    // copies per tile: 4 K + 4 V + 1 V metadata, + 1 K metadata (into the
    // wavefront's K-metadata buffer) for a group's first tile
    const uint32_t km = lds_addr(&s_km[w][0]);

    // Tile j of this wavefront into ring slot j % kDepth.
    auto issue_tile = [&](int j) {
        const int t0 = __builtin_amdgcn_readfirstlane(tile_t0(j));
        const uint32_t slot = ring + (uint32_t)(j % kDepth) * kSlotBytes;
        if (LAYOUT != 2 && t0 + kTile <= T) {
            // two 16-token runs, each inside one block
#pragma unroll
            for (int run = 0; run < 2; ++run) {
                size_t row0;
                if (LAYOUT == 0) {
                    row0 = blk0_rows + (size_t)(t0 + 16 * run);
                } else {
                    const int tr = t0 + 16 * run;
                    const int bi = a.bt_shift >= 0 ? (tr >> a.bt_shift) : tr / a.geo.bt;
                    // run 2 (j % 4) + run of the wavefront's group j / 4
                    int blk = __builtin_amdgcn_readlane(run_blk, 8 * (j >> 2) + 2 * (j & 3) + run);
                    if (blk < 0 || blk >= a.geo.num_blocks) {
                        bad = true;
                        blk = 0;
                    }
                    row0 = ((size_t)blk * Hkv + h) * a.geo.bt + (size_t)(tr - bi * a.geo.bt);
                }
                const uint32_t vq = (uint32_t)(kq ^ (run << 2));
#pragma unroll
                for (int i2 = 0; i2 < 2; ++i2) {
                    const int i = 2 * run + i2;
                    const size_t rb = (row0 + 8 * i2) * kCodeRow;
                    const uint32_t off = (uint32_t)crow * kCodeRow;
                    lds_copy16(a.k_codes + rb, off + 16u * kq, slot + 1024u * i);
                    lds_copy16(a.v_codes + rb, off + 16u * vq, slot + kTileBytes + 1024u * i);
                }
            }
        } else {
            // per-lane rows; rows past the context repeat the last token
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int t = min(t0 + 8 * i + crow, T - 1);
                const size_t rb = row_of(t) * kCodeRow;
                lds_copy16(a.k_codes + rb + 16 * kq, slot + 1024u * i);
                lds_copy16(a.v_codes + rb + 16 * (kq ^ ((i >> 1) << 2)), slot + kTileBytes + 1024u * i);
            }
        }
        // V scale (lanes 0..31) and zero (lanes 32..63) of the tile's tokens;
        // tokens past the context repeat the last one
        {
            const int t = min(t0 + (lane & 31), T - 1);
            lds_copy4((lane < 32 ? a.meta.v_scale : a.meta.v_zero) + vmeta + t, slot + kVMetaOff);
        }
        // K scale (lanes 0..31) and zero (lanes 32..63) of the group; the
        // previous group's values were consumed by its fold three tiles ago
        if ((j & 3) == 0) {
            const int g = g0 + min(group_of(j), n_groups - 1);
            const float *src = (lane < 32 ? a.meta.k_scale : a.meta.k_zero) + kmeta + (size_t)g * kHeadDim;
            lds_copy16(src + 4 * (lane & 31), km);
        }
    };

    // query rows of the workgroup into LDS: copy m holds rows 4 m .. 4 m + 3
    // (RT copies per wavefront; rows past the last repeat it)
#pragma unroll
    for (int k = 0; k < RT; ++k) {
        const int m = w + 4 * k;
        const int r = min(row_base + 4 * m + (lane >> 4), a.rows_total - 1);
        const size_t qrow = ((size_t)b * a.nq + r / a.G) * a.Hq + (size_t)h * a.G + r % a.G;
        lds_copy16(a.q + qrow * kHeadDim + 8 * (lane & 15), lds_addr(s_q) + 1024u * m);
    }

    // ---- per-wavefront online-softmax state: lane (col = query row of the
    // row tile, kg); the reference carries the 2^-Ev factor of the V weights ----
    float m_run[RT], m_ref[RT], l_part[RT], ob_part[RT];
    f32x4_t acc[RT][8], acc_off[RT];
    auto reset_state = [&]() {
#pragma unroll
        for (int rt = 0; rt < RT; ++rt) {
            m_run[rt] = m_ref[rt] = -INFINITY;
            l_part[rt] = ob_part[rt] = 0.0f;
#pragma unroll
            for (int n = 0; n < 8; ++n) acc[rt][n] = f32x4_t{0.f, 0.f, 0.f, 0.f};
            acc_off[rt] = f32x4_t{0.f, 0.f, 0.f, 0.f};
        }
    };
    reset_state();
    const u32x4_t c1024 = {0x64006400u, 0x64006400u, 0x64006400u, 0x64006400u};

    // Fold of a group (K scales and zeros from the wavefront's K-metadata
    // buffer, query rows from LDS), per row tile: q''_d = q_d s_d 2^-E as fp16
    // hi + lo MFMA operands, score scale 2^E kscore and bias
    // kscore sum_d q_d (z_d - 1024 s_d), E per row.  Lane (col, kg) holds
    // dims 32 kg .. + 31 of row col, the dims of its MFMA operand pieces.
    u32x4_t bq[RT][8];
    float bsc[RT], bb[RT];
    auto fold = [&]() {
        const float *ks = reinterpret_cast<const float *>(&s_km[w][0]) + 32 * kg;
        const float *kz = ks + kHeadDim;
#pragma unroll
        for (int rt = 0; rt < RT; ++rt) {
            const int rl = rt * 16 + col;
            const bool row_live = row_base + rl < a.rows_total;
            const uint4 *qp = reinterpret_cast<const uint4 *>(s_q + rl * (kHeadDim * 2) + 64 * kg);
            // pass 1: row maximum of |q s| and the bias
            float mx = 0.0f, bias = 0.0f;
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                const uint4 u = qp[k];
                const float qv[8] = {bf16_lo(u.x), bf16_hi(u.x), bf16_lo(u.y), bf16_hi(u.y),
                                     bf16_lo(u.z), bf16_hi(u.z), bf16_lo(u.w), bf16_hi(u.w)};
                const float4 s0 = reinterpret_cast<const float4 *>(ks)[2 * k];
                const float4 s1 = reinterpret_cast<const float4 *>(ks)[2 * k + 1];
                const float4 z0 = reinterpret_cast<const float4 *>(kz)[2 * k];
                const float4 z1 = reinterpret_cast<const float4 *>(kz)[2 * k + 1];
                const float sv[8] = {s0.x, s0.y, s0.z, s0.w, s1.x, s1.y, s1.z, s1.w};
                const float zv[8] = {z0.x, z0.y, z0.z, z0.w, z1.x, z1.y, z1.z, z1.w};
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    mx = fmax2(mx, fabsf(qv[e] * sv[e]));
                    bias = fmaf(qv[e], fmaf(-1024.0f, sv[e], zv[e]), bias);
                }
            }
            mx = max_kg(mx);
            bias = sum_kg(bias);
            int E = 0;
            if (mx > 0.0f) frexpf(mx, &E);  // mx = f 2^E, f in [0.5, 1)
            // pass 2: the scaled products (the same roundings as pass 1)
#pragma unroll
            for (int kk = 0; kk < 4; ++kk) {
                const uint4 u = qp[kk];
                const float qv[8] = {bf16_lo(u.x), bf16_hi(u.x), bf16_lo(u.y), bf16_hi(u.y),
                                     bf16_lo(u.z), bf16_hi(u.z), bf16_lo(u.w), bf16_hi(u.w)};
                const float4 s0 = reinterpret_cast<const float4 *>(ks)[2 * kk];
                const float4 s1 = reinterpret_cast<const float4 *>(ks)[2 * kk + 1];
                const float sv[8] = {s0.x, s0.y, s0.z, s0.w, s1.x, s1.y, s1.z, s1.w};
                u32x4_t hi, lo;
#pragma unroll
                for (int e = 0; e < 8; e += 2) {
                    const float y0 = row_live ? ldexpf(qv[e] * sv[e], -E) : 0.0f;
                    const float y1 = row_live ? ldexpf(qv[e + 1] * sv[e + 1], -E) : 0.0f;
                    const uint32_t hp = pack_f16(y0, y1);
                    hi[e / 2] = hp;
                    lo[e / 2] = pack_f16(y0 - f16_lo(hp), y1 - f16_hi(hp));
                }
                bq[rt][2 * kk] = hi;
                bq[rt][2 * kk + 1] = lo;
            }
            bsc[rt] = ldexpf(kscore, E);
            bb[rt] = row_live ? bias * kscore : 0.0f;
        }
    };
    // Scores of tile j in log2 units: lane (col, kg) gets token
    // t0 + 16 r + 4 kg + i in x[4 r + i]; tokens past the context get -inf.
    auto tile_scores = [&](const uint8_t *slot_p, int j, float (&x)[RT][8]) {
        f32x4_t sc[RT][2];
#pragma unroll
        for (int r = 0; r < 2; ++r) {
            const int t = 16 * r + col;
            const uint4 u0 = *reinterpret_cast<const uint4 *>(slot_p + k_slot(t, 2 * kg));
            const uint4 u1 = *reinterpret_cast<const uint4 *>(slot_p + k_slot(t, 2 * kg + 1));
#pragma unroll
            for (int rt = 0; rt < RT; ++rt) sc[rt][r] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int kk = 0; kk < 4; ++kk) {
                const uint4 &u = (kk >> 1) ? u1 : u0;
                const u32x4_t av = (kk & 1) ? codes_to_f16(u.z, u.w) : codes_to_f16(u.x, u.y);
#pragma unroll
                for (int rt = 0; rt < RT; ++rt) {
                    sc[rt][r] = mfma_f16(av, bq[rt][2 * kk + 0], sc[rt][r]);
                    sc[rt][r] = mfma_f16(av, bq[rt][2 * kk + 1], sc[rt][r]);
                }
            }
        }
#pragma unroll
        for (int rt = 0; rt < RT; ++rt)
#pragma unroll
            for (int i = 0; i < 8; ++i) x[rt][i] = fmaf(sc[rt][i >> 2][i & 3], bsc[rt], bb[rt]);
        const int t0 = tile_t0(j);
        if (t0 + kTile > T) {
            asm volatile("" ::: "memory");
#pragma unroll
            for (int i = 0; i < 8; ++i) {
                const int t = t0 + 16 * (i >> 2) + 4 * kg + (i & 3);
#pragma unroll
                for (int rt = 0; rt < RT; ++rt) x[rt][i] = t < T ? x[rt][i] : -INFINITY;
            }
        }
    };
    auto tile_max = [&](const float (&x)[8]) {
        return max_kg(fmax3(fmax3(x[0], x[1], x[2]), fmax3(x[3], x[4], x[5]), fmax2(x[6], x[7])));
    };
    // Weights against m_ref, then P V for the tile (V rows from the slot,
    // transposed on read).
    auto tile_accumulate = [&](const uint8_t *slot_p, const float (&x)[RT][8]) {
        const float *vsm = reinterpret_cast<const float *>(slot_p + kVMetaOff) + 4 * kg;
        const float4 vs0 = *reinterpret_cast<const float4 *>(vsm);
        const float4 vs1 = *reinterpret_cast<const float4 *>(vsm + 16);
        const float4 vz0 = *reinterpret_cast<const float4 *>(vsm + kTile);
        const float4 vz1 = *reinterpret_cast<const float4 *>(vsm + kTile + 16);
        const float vsv[8] = {vs0.x, vs0.y, vs0.z, vs0.w, vs1.x, vs1.y, vs1.z, vs1.w};
        const float vzv[8] = {vz0.x, vz0.y, vz0.z, vz0.w, vz1.x, vz1.y, vz1.z, vz1.w};
        u32x4_t pa[RT];
#pragma unroll
        for (int rt = 0; rt < RT; ++rt) {
            float pw[8];
#pragma unroll
            for (int i = 0; i < 8; ++i) {
                const float p = __builtin_amdgcn_exp2f(x[rt][i] - m_ref[rt]);
                l_part[rt] += p;
                ob_part[rt] = fmaf(p, vzv[i], ob_part[rt]);
                pw[i] = p * vsv[i];
            }
#pragma unroll
            for (int e = 0; e < 4; ++e) pa[rt][e] = pack_f16_rne(pw[2 * e], pw[2 * e + 1]);
        }
        // V values of the 8 tokens tau(kg, e) = 16 (e / 4) + 4 kg + e % 4 for
        // dims 16 c + col, read transposed from LDS
        const uint8_t *vl = slot_p + kTileBytes;
        const int tr = 16 * ((col >> 1) >> 2) + 4 * kg + ((col >> 1) & 3);
        const int half = col & 1;
#pragma unroll
        for (int c = 0; c < 8; ++c) {
            const intx2_t vt = __builtin_amdgcn_ds_read_tr8_b64_v2i32(
                (__attribute__((address_space(3))) intx2_t *)(vl + v_slot(tr, c) + 8 * half));
            const u32x4_t bv = codes_to_f16((uint32_t)vt[0], (uint32_t)vt[1]);
#pragma unroll
            for (int rt = 0; rt < RT; ++rt) acc[rt][c] = mfma_f16(pa[rt], bv, acc[rt][c]);
        }
#pragma unroll
        for (int rt = 0; rt < RT; ++rt) acc_off[rt] = mfma_f16(pa[rt], c1024, acc_off[rt]);
    };

    // Fast path: the softmax reference of each row is the maximum of the
    // wavefront's first tile and stays fixed.  If any sum leaves the safe
    // range the wavefront redoes its tiles below with a running maximum.
    // Tile j + 1 is in flight while tile j is attended; no barriers.
    if (n_mine > 0) issue_tile(0);
    // the query rows are in once only tile 0's copies may remain in flight
    if (n_mine > 0) {
        wait_vmcnt<10>();
    } else {
        wait_vmcnt<0>();
    }
    __syncthreads();
    for (int u = 0; u < kMaxGroups; ++u) {
        if (u >= n_mine) break;  // wavefront-uniform
#pragma unroll
        for (int c = 0; c < 4; ++c) {
            const int j = 4 * u + c;
            // the next tile: inside this group, or the next group's first
            const bool more = c < 3 || u + 1 < n_mine;
            if (more) issue_tile(j + 1);
            // tile j is in once only tile j + 1's copies may remain in flight
            if (!more) {
                wait_vmcnt<0>();
            } else if (c == 3) {
                wait_vmcnt<10>();
            } else {
                wait_vmcnt<9>();
            }
            const uint8_t *slot_p = ring_p + (c % kDepth) * kSlotBytes;
            if (c == 0) fold();
            if (tile_valid(j)) {
                float x[RT][8];
                tile_scores(slot_p, j, x);
                if (j == 0) {
#pragma unroll
                    for (int rt = 0; rt < RT; ++rt) {
                        m_run[rt] = tile_max(x[rt]);
                        m_ref[rt] = m_run[rt] + (float)Ev;
                    }
                }
                tile_accumulate(slot_p, x);
            }
            // the slot and the K-metadata buffer are rewritten by later
            // copies: their reads must be done
            asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
        }
    }
    bool unsafe = false;
#pragma unroll
    for (int rt = 0; rt < RT; ++rt) {
        unsafe |= !(l_part[rt] < 1e30f) || !(fabsf(ob_part[rt]) < 1e30f);
#pragma unroll
        for (int n = 0; n < 8; ++n)
#pragma unroll
            for (int i = 0; i < 4; ++i) unsafe |= !(fabsf(acc[rt][n][i]) < 1e30f);
#pragma unroll
        for (int i = 0; i < 4; ++i) unsafe |= !(fabsf(acc_off[rt][i]) < 1e30f);
    }
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
                float x[RT][8];
                tile_scores(slot_p, j, x);
#pragma unroll
                for (int rt = 0; rt < RT; ++rt) {
                    const float mx = tile_max(x[rt]);
                    if (__any(mx > m_run[rt])) {
                        const float m_new = fmaxf(mx, m_run[rt]);
                        const float alpha = (m_run[rt] == -INFINITY) ? 0.0f : exp2f(m_run[rt] - m_new);
                        m_run[rt] = m_new;
                        m_ref[rt] = m_new + (float)Ev;
                        l_part[rt] *= alpha;
                        ob_part[rt] *= alpha;
                        float af[4];
#pragma unroll
                        for (int i = 0; i < 4; ++i) af[i] = __shfl(alpha, 4 * kg + i);
#pragma unroll
                        for (int n = 0; n < 8; ++n)
#pragma unroll
                            for (int i = 0; i < 4; ++i) acc[rt][n][i] *= af[i];
#pragma unroll
                        for (int i = 0; i < 4; ++i) acc_off[rt][i] *= af[i];
                    }
                }
                tile_accumulate(slot_p, x);
            }
            asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
        }
    }
    wait_vmcnt<0>();  // no copy may land in the ring once it is reused below

    // ---- per-wavefront totals -> LDS (still scaled by 2^-Ev) ----
    // o' = sum p' z + sum pw (1024 + c) - 1024 sum pw
    __syncthreads();  // every wavefront is done with its ring
    // ring reused: o [wave][kRows][128], then max, sum, sum p z and merge
    // factors [wave][kRows]
    float *s_o = reinterpret_cast<float *>(s_ring);
    float(*s_m)[kRows] = reinterpret_cast<float(*)[kRows]>(s_o + kWaves * kRows * kHeadDim);
    float(*s_l)[kRows] = s_m + kWaves;
    float(*s_ob)[kRows] = s_l + kWaves;
    float(*s_f)[kRows] = s_ob + kWaves;
#pragma unroll
    for (int rt = 0; rt < RT; ++rt) {
        const float l = sum_kg(l_part[rt]);
        const float ob = sum_kg(ob_part[rt]);
        if (kg == 0) {
            s_m[w][rt * 16 + col] = m_run[rt];
            s_l[w][rt * 16 + col] = l;
            s_ob[w][rt * 16 + col] = ob;
        }
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int c = 0; c < 8; ++c)
                s_o[(w * kRows + rt * 16 + 4 * kg + i) * kHeadDim + 16 * c + col] = acc[rt][c][i] - acc_off[rt][i];
    }
    if (lane == 0) s_ev[w] = Ev;
    const bool any_bad = __syncthreads_or(bad);

    // ---- merge the four wavefronts, write this split's partial: per-row
    // factors first, then float4 multiply-adds ----
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
    for (int idx = tid; idx < kRows * (kHeadDim / 4); idx += kThreads) {
        const int rr = idx / (kHeadDim / 4);  // row within the workgroup
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
        // nontemporal: the combine kernel reads the partials back faster when
        // they did not go through the last-level cache (32K layer 30.3 ->
        // 29.8 us per call, 128K 65.2 -> 63.9 us)
        const size_t pi = partial_index(row);
        const f32x4_t ov = {O.x, O.y, O.z, O.w};
        __builtin_nontemporal_store(ov, reinterpret_cast<f32x4_t *>(a.ws_o + pi * kHeadDim) + d4);
        if (d4 == 0) {
            const f32x2_t mlv = {s_ML[rr][0], s_ML[rr][1]};
            __builtin_nontemporal_store(mlv, reinterpret_cast<f32x2_t *>(a.ws_ml + pi));
        }
    }
}

template <int RT, int LAYOUT>
void launch_rt(const VerifyArgs &args, int split_groups, dim3 grid, hipStream_t stream) {
    if (split_groups == 4)
        hipLaunchKernelGGL((verify_kernel<RT, LAYOUT, 4>), grid, dim3(kThreads), 0, stream, args);
    else if (LAYOUT == 0 && split_groups == 32)
        hipLaunchKernelGGL((verify_kernel<RT, 0, 32>), grid, dim3(kThreads), 0, stream, args);
    else if (LAYOUT == 0 && split_groups == 64)
        hipLaunchKernelGGL((verify_kernel<RT, 0, 64>), grid, dim3(kThreads), 0, stream, args);
    else if (split_groups == 8)
        hipLaunchKernelGGL((verify_kernel<RT, LAYOUT, 8>), grid, dim3(kThreads), 0, stream, args);
    else
        hipLaunchKernelGGL((verify_kernel<RT, LAYOUT, 16>), grid, dim3(kThreads), 0, stream, args);
}

template <int RT>
void launch_layout(const VerifyArgs &args, int split_groups, dim3 grid, hipStream_t stream) {
    if (args.geo.max_blocks == 1)
        launch_rt<RT, 0>(args, split_groups, grid, stream);
    else if (args.geo.bt % 16 == 0)
        launch_rt<RT, 1>(args, split_groups, grid, stream);
    else
        launch_rt<RT, 2>(args, split_groups, grid, stream);
}

}  // namespace

hipError_t launch_verify_mfma(const VerifyArgs &args, int split_groups, hipStream_t stream) {
    if (split_groups != 4 && split_groups != 8 && split_groups != 16 &&
        !(args.geo.max_blocks == 1 && (split_groups == 32 || split_groups == 64)))
        return hipErrorInvalidValue;
    if (args.rows_total < 1) return hipErrorInvalidValue;
    const int rt = args.rows_total <= 16 ? 1 : 2;
    const int chunks = (args.rows_total + 16 * rt - 1) / (16 * rt);
    // kv head fastest for paged layouts (the kernel reads the grid the same way)
    if (args.geo.max_blocks != 1 && args.n_ctx_splits > 65535) return hipErrorInvalidValue;
    const unsigned hc = (unsigned)(args.geo.Hkv * chunks);
    const dim3 grid = args.geo.max_blocks == 1 ? dim3(args.n_ctx_splits, hc, args.B) : dim3(hc, args.n_ctx_splits, args.B);
    if (rt == 1)
        launch_layout<1>(args, split_groups, grid, stream);
    else
        launch_layout<2>(args, split_groups, grid, stream);
    return hipGetLastError();
}

}  // namespace lynx
