// Verification attention on matrix cores (gfx950 MFMA, fp16 operands).
//
// What it computes (Sec. 4.3; attention of Sec. 2): the k draft queries of a
// sequence attend, in one pass, over the merged 8-bit cache, with K and V
// reconstructed as zero + code * scale.  This kernel covers the context
// tokens.  The drafts' own BF16 K/V (the causal tail) form one more split,
// handled by the vector kernel of attention.hip, and the combine kernel
// merges all splits.
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
//    (fp16; Ev per split, so pw <= 1 while p <= 1); sum_t p_t z_t is summed
//    in fp32 and the offset is measured by one MFMA against the constant 1024.
//    The 2^-Ev factor rides on the softmax reference, so l, sum p z and the
//    products all carry it and one multiply restores it at the end.
//
// Work split: grid = (context split of SG 128-token groups, kv head x chunk
// of 16 RT query rows, sequence).  A workgroup has 4 wavefronts; wavefront w
// serves row tile w % RT and every (4 / RT)-th 32-token tile of each group.
// The query fold of group g + 1 goes to the other half of a double buffer
// while group g is attended, one barrier per group.  At the end the
// wavefronts of a row tile merge through LDS into one partial per split.
#include "lane_ops.h"
#include "lynx_internal.h"

#include <math.h>

namespace lynx {

namespace {

typedef _Float16 f16x8_t __attribute__((ext_vector_type(8)));

constexpr int kThreads = 256;
constexpr int kWaves = 4;
constexpr int kTile = 32;      // tokens per wavefront step
constexpr float kLog2e = 1.4426950408889634f;

__device__ __forceinline__ f32x4_t mfma(u32x4_t a, u32x4_t b, f32x4_t c) {
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

__device__ __forceinline__ uint32_t pack_f16(float a, float b) {
    return __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_pkrtz(a, b));
}
__device__ __forceinline__ float f16_lo(uint32_t w) {
    return (float)__builtin_bit_cast(_Float16, (uint16_t)(w & 0xffffu));
}
__device__ __forceinline__ float f16_hi(uint32_t w) {
    return (float)__builtin_bit_cast(_Float16, (uint16_t)(w >> 16));
}
__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// Byte offset of 16-byte chunk q of V-tile row t in a wavefront's LDS slot.
// The XOR swizzle spreads the 8 rows one transposed read touches over all
// 32 banks.
__device__ __forceinline__ uint32_t v_slot(int t, int q) {
    const int sw = (t & 7) ^ ((t >> 4) << 2);
    return (uint32_t)t * kCodeRow + (uint32_t)((q ^ sw) * 16);
}

// One wavefront's registers for one 32-token tile: the 32-byte segment
// (dims 32 kg .. 32 kg + 31) of K and V rows col and col + 16.
struct Tile {
    uint4 k[2][2];
    uint4 v[2][2];
};

// LAYOUT 0: one block per sequence; 1: paged, block_tokens a multiple of 16;
// 2: any other paging.  RT: 16-row query tiles per workgroup (1 or 2).
// SG: 128-token groups per split (4 or 8).
template <int RT, int LAYOUT, int SG>
__global__ __launch_bounds__(kThreads, 2) void verify_kernel(VerifyArgs a) {
    constexpr int NP = kWaves / RT;  // wavefronts sharing one row tile
    constexpr int TPG = 4 / NP;      // tiles of a group per wavefront
    constexpr int kTilesPerWave = SG * TPG;
    // tiles in flight ahead of the one being computed (one for two row tiles:
    // registers; each wavefront then still has 8 KB of K/V loads in flight)
    constexpr int kPrefetch = RT == 1 ? 2 : 1;
    const int Hkv = a.geo.Hkv;
    const int split = blockIdx.x;
    const int h = blockIdx.y % Hkv;
    const int chunk = blockIdx.y / Hkv;
    const int b = blockIdx.z;
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int w = tid >> 6;
    const int col = lane & 15;
    const int kg = lane >> 4;
    const int rt = w % RT;
    const int part = w / RT;
    const int T = max(0, min(a.seq_lens[b], a.max_seq_len));
    const int g0 = split * SG;
    const int n_groups = max(0, min(SG, (T - g0 * kKGroup + kKGroup - 1) / kKGroup));
    const int row_base = chunk * RT * 16;  // first query row of the workgroup
    const float kscore = kLog2e * rsqrtf((float)kHeadDim);

    // query row r <-> (draft r / G, head r % G); its partial-output row
    auto partial_index = [&](int r) {
        return (((size_t)b * Hkv + h) * a.rows_total + r) * a.ws_splits + split;
    };

    if (n_groups == 0) {  // a split past the context: (max, sum) = (-inf, 0)
        for (int r = tid; r < RT * 16; r += kThreads)
            if (row_base + r < a.rows_total) a.ws_ml[partial_index(row_base + r)] = make_float2(-INFINITY, 0.0f);
        return;
    }

    // Folded query operands of two groups: [buffer][row tile][kk, hi/lo][lane]
    constexpr int kFoldBytes = 2 * RT * 8 * 64 * 16;
    constexpr int kMergeBytes = kWaves * 16 * kHeadDim * 4;
    __shared__ __attribute__((aligned(16))) uint8_t s_raw[kFoldBytes > kMergeBytes ? kFoldBytes : kMergeBytes];
    u32x4_t *s_b = reinterpret_cast<u32x4_t *>(s_raw);
    __shared__ float s_sc[2][RT * 16], s_bias[2][RT * 16];
    __shared__ __attribute__((aligned(16))) float s_vs[SG * kKGroup];
    __shared__ __attribute__((aligned(16))) float s_vz[SG * kKGroup];
    __shared__ __attribute__((aligned(16))) uint8_t s_v[kWaves][kTile * kCodeRow];
    __shared__ float s_vmax[kWaves];
    __shared__ float s_m[kWaves][16], s_l[kWaves][16], s_ob[kWaves][16];

    bool bad = false;
    const int32_t *bt_row = a.block_table + (size_t)b * a.geo.max_blocks;
    const size_t vmeta = ((size_t)b * Hkv + h) * a.geo.max_tokens;
    const size_t kmeta = ((size_t)b * Hkv + h) * a.geo.n_groups * kHeadDim;
    const size_t blk0_rows =
        LAYOUT == 0 ? ((size_t)min(max(bt_row[0], 0), a.geo.num_blocks - 1) * Hkv + h) * a.geo.bt : 0;
    if (LAYOUT == 0 && (bt_row[0] < 0 || bt_row[0] >= a.geo.num_blocks)) bad = true;

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

    // ---- fold operands held by this thread: rows fr = pass * 16 + tid / 16,
    // dims 32 fkg + 8 fkk .. + 7 ----
    const int frow = tid >> 4;
    const int fkg = (tid & 15) >> 2;
    const int fkk = tid & 3;
    const int fd0 = 32 * fkg + 8 * fkk;
    uint4 fq[RT];
#pragma unroll
    for (int p = 0; p < RT; ++p) {
        const int r = min(row_base + p * 16 + frow, a.rows_total - 1);
        const size_t qrow = ((size_t)b * a.nq + r / a.G) * a.Hq + (size_t)h * a.G + r % a.G;
        fq[p] = *reinterpret_cast<const uint4 *>(a.q + qrow * kHeadDim + fd0);
        if (row_base + p * 16 + frow >= a.rows_total) fq[p] = make_uint4(0u, 0u, 0u, 0u);
    }
    // V metadata of the split (zero past the context)
    constexpr int kVmPer = SG * kKGroup / kThreads;
    float vs_r[kVmPer], vz_r[kVmPer];
#pragma unroll
    for (int k = 0; k < kVmPer; ++k) {
        const int t = g0 * kKGroup + tid + k * kThreads;
        const size_t ti = vmeta + (size_t)min(t, T - 1);
        vs_r[k] = a.meta.v_scale[ti];
        vz_r[k] = a.meta.v_zero[ti];
        if (t >= T) vs_r[k] = vz_r[k] = 0.0f;
    }
    // K metadata of one group for this thread's dims
    float4 ks0, ks1, kz0, kz1;
    auto load_kmeta = [&](int gl) {
        const size_t mo = kmeta + (size_t)(g0 + gl) * kHeadDim + fd0;
        ks0 = *reinterpret_cast<const float4 *>(a.meta.k_scale + mo);
        ks1 = *reinterpret_cast<const float4 *>(a.meta.k_scale + mo + 4);
        kz0 = *reinterpret_cast<const float4 *>(a.meta.k_zero + mo);
        kz1 = *reinterpret_cast<const float4 *>(a.meta.k_zero + mo + 4);
    };
    load_kmeta(0);

    // ---- this wavefront's tiles: tile j of group j / TPG, position
    // part + NP (j % TPG) within the group ----
    auto tile_t0 = [&](int j) { return (g0 + j / TPG) * kKGroup + kTile * (part + NP * (j % TPG)); };
    auto tile_valid = [&](int j) { return j / TPG < n_groups && tile_t0(j) < T; };
    const uint32_t kv_lane = (uint32_t)col * kCodeRow + 32u * kg;
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
                const uint8_t *kp = a.k_codes + row * kCodeRow + kv_lane;
                const uint8_t *vp = a.v_codes + row * kCodeRow + kv_lane;
                tl.k[r][0] = *reinterpret_cast<const uint4 *>(kp);
                tl.k[r][1] = *reinterpret_cast<const uint4 *>(kp + 16);
                tl.v[r][0] = *reinterpret_cast<const uint4 *>(vp);
                tl.v[r][1] = *reinterpret_cast<const uint4 *>(vp + 16);
            }
        } else {
#pragma unroll
            for (int r = 0; r < 2; ++r) {
                const size_t row = row_generic(min(max(t0 + 16 * r + col, 0), T - 1));
                const uint8_t *kp = a.k_codes + row * kCodeRow + 32u * kg;
                const uint8_t *vp = a.v_codes + row * kCodeRow + 32u * kg;
                tl.k[r][0] = *reinterpret_cast<const uint4 *>(kp);
                tl.k[r][1] = *reinterpret_cast<const uint4 *>(kp + 16);
                tl.v[r][0] = *reinterpret_cast<const uint4 *>(vp);
                tl.v[r][1] = *reinterpret_cast<const uint4 *>(vp + 16);
            }
        }
    };

    // Fold group gl into buffer buf: q''_d = q_d s_d 2^-E as fp16 hi + lo,
    // per-row score scale 2^E kscore and bias sum_d q_d (z_d - 1024 s_d) kscore.
    // Every thread takes part (the row reductions run over 16 lanes).
    auto fold = [&](int buf, int gl) {
        const bool live = gl < n_groups;
        const float sv[8] = {ks0.x, ks0.y, ks0.z, ks0.w, ks1.x, ks1.y, ks1.z, ks1.w};
        const float zv[8] = {kz0.x, kz0.y, kz0.z, kz0.w, kz1.x, kz1.y, kz1.z, kz1.w};
#pragma unroll
        for (int p = 0; p < RT; ++p) {
            const uint4 qw = fq[p];
            const float qv[8] = {bf16_lo(qw.x), bf16_hi(qw.x), bf16_lo(qw.y), bf16_hi(qw.y),
                                 bf16_lo(qw.z), bf16_hi(qw.z), bf16_lo(qw.w), bf16_hi(qw.w)};
            float x[8], mx = 0.0f, bias = 0.0f;
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                x[e] = live ? qv[e] * sv[e] : 0.0f;
                mx = fmax2(mx, fabsf(x[e]));
                bias = fmaf(qv[e], fmaf(-1024.0f, sv[e], zv[e]), bias);
            }
            mx = row16_max(mx);
            bias = live ? row16_sum(bias) : 0.0f;
            int E = 0;
            if (mx > 0.0f) frexpf(mx, &E);  // mx = f 2^E, f in [0.5, 1)
            u32x4_t hi, lo;
#pragma unroll
            for (int e = 0; e < 8; e += 2) {
                const float y0 = ldexpf(x[e], -E), y1 = ldexpf(x[e + 1], -E);
                const uint32_t hp = pack_f16(y0, y1);
                hi[e / 2] = hp;
                lo[e / 2] = pack_f16(y0 - f16_lo(hp), y1 - f16_hi(hp));
            }
            const int base = ((buf * RT + p) * 8 + fkk * 2) * 64 + fkg * 16 + frow;
            s_b[base] = hi;
            s_b[base + 64] = lo;
            if ((tid & 15) == 0) {
                s_sc[buf][p * 16 + frow] = ldexpf(kscore, E);
                s_bias[buf][p * 16 + frow] = bias * kscore;
            }
        }
    };

    // ---- prologue ----
    Tile tiles[kPrefetch + 1];
#pragma unroll
    for (int j = 0; j < kPrefetch; ++j)
        if (j < kTilesPerWave) load_tile(j, tiles[j]);
    {
        float vm = 0.0f;
#pragma unroll
        for (int k = 0; k < kVmPer; ++k) {
            s_vs[tid + k * kThreads] = vs_r[k];
            s_vz[tid + k * kThreads] = vz_r[k];
            vm = fmax2(vm, vs_r[k]);
        }
        vm = max_kg(row16_max(vm));
        if (lane == 0) s_vmax[w] = vm;
    }
    fold(0, 0);
    if (n_groups > 1) load_kmeta(1);
    __syncthreads();
    int Ev = 0;
    {
        const float vm = fmax2(fmax2(s_vmax[0], s_vmax[1]), fmax2(s_vmax[2], s_vmax[3]));
        if (vm > 0.0f) frexpf(vm, &Ev);
        // V scales below 2^-100 contribute below 255 * 2^-100 per token; the
        // clamp keeps 2^-Ev, and so the weights p 2^-Ev, finite
        Ev = max(Ev, -100);
    }

    // ---- per-wave online-softmax state: lane (col = query row of the tile,
    // kg); the reference carries the 2^-Ev factor of the V weights ----
    float m_run = -INFINITY, m_ref = -INFINITY, l_part = 0.0f, ob_part = 0.0f;
    f32x4_t acc[8], acc_off;
#pragma unroll
    for (int n = 0; n < 8; ++n) acc[n] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    acc_off = f32x4_t{0.f, 0.f, 0.f, 0.f};
    const u32x4_t c1024 = {0x64006400u, 0x64006400u, 0x64006400u, 0x64006400u};
    auto *vlds = &s_v[w][0];

    u32x4_t bq[8];
    float bsc = 0.0f, bb = 0.0f;
    auto load_group_operands = [&](int buf) {
#pragma unroll
        for (int i = 0; i < 8; ++i) bq[i] = s_b[((buf * RT + rt) * 8 + i) * 64 + lane];
        bsc = s_sc[buf][rt * 16 + col];
        bb = s_bias[buf][rt * 16 + col];
    };
    // Scores of tile j in log2 units: lane (col, kg) gets token
    // t0 + 16 r + 4 kg + i in x[4 r + i]; tokens past the context get -inf.
    // Also stages the tile's V rows in the wavefront's LDS slot.
    auto tile_scores = [&](const Tile &cur, int j, float (&x)[8]) {
#pragma unroll
        for (int r = 0; r < 2; ++r) {
            const int t = 16 * r + col;
            *reinterpret_cast<uint4 *>(vlds + v_slot(t, 2 * kg)) = cur.v[r][0];
            *reinterpret_cast<uint4 *>(vlds + v_slot(t, 2 * kg + 1)) = cur.v[r][1];
        }
        f32x4_t sc[2];
#pragma unroll
        for (int r = 0; r < 2; ++r) {
            sc[r] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int kk = 0; kk < 4; ++kk) {
                const uint4 &u = cur.k[r][kk >> 1];
                const u32x4_t av = (kk & 1) ? codes_to_f16(u.z, u.w) : codes_to_f16(u.x, u.y);
                sc[r] = mfma(av, bq[2 * kk + 0], sc[r]);
                sc[r] = mfma(av, bq[2 * kk + 1], sc[r]);
            }
        }
#pragma unroll
        for (int i = 0; i < 8; ++i) x[i] = fmaf(sc[i >> 2][i & 3], bsc, bb);
        const int t0 = tile_t0(j);
        if (t0 + kTile > T) {
            asm volatile("" ::: "memory");
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
    // Weights against m_ref, then P V for tile j.
    auto tile_accumulate = [&](int j, const float (&x)[8]) {
        const int tl = (j / TPG) * kKGroup + kTile * (part + NP * (j % TPG)) + 4 * kg;
        const float4 vs0 = *reinterpret_cast<const float4 *>(&s_vs[tl]);
        const float4 vs1 = *reinterpret_cast<const float4 *>(&s_vs[tl + 16]);
        const float4 vz0 = *reinterpret_cast<const float4 *>(&s_vz[tl]);
        const float4 vz1 = *reinterpret_cast<const float4 *>(&s_vz[tl + 16]);
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
        for (int e = 0; e < 4; ++e) pa[e] = pack_f16(pw[2 * e], pw[2 * e + 1]);
        // V values of the 8 tokens tau(kg, e) = 16 (e / 4) + 4 kg + e % 4 for
        // dims 16 c + col, read transposed from LDS
        const int tr = 16 * ((col >> 1) >> 2) + 4 * kg + ((col >> 1) & 3);
        const int half = col & 1;
#pragma unroll
        for (int c = 0; c < 8; ++c) {
            const intx2_t vt = __builtin_amdgcn_ds_read_tr8_b64_v2i32(
                (__attribute__((address_space(3))) intx2_t *)(vlds + v_slot(tr, c) + 8 * half));
            acc[c] = mfma(pa, codes_to_f16((uint32_t)vt[0], (uint32_t)vt[1]), acc[c]);
        }
        acc_off = mfma(pa, c1024, acc_off);
    };

    // Fast path: each row's softmax reference is the maximum of the
    // wavefront's first tile and stays fixed.  If any sum leaves the safe
    // range the workgroup redoes the split below with a running maximum.
#pragma unroll
    for (int gi = 0; gi < SG; ++gi) {
        if (gi >= n_groups) break;  // uniform across the workgroup
        if (gi + 1 < n_groups) {
            fold((gi + 1) & 1, gi + 1);
            if (gi + 2 < n_groups) load_kmeta(gi + 2);
        }
        load_group_operands(gi & 1);
#pragma unroll
        for (int jj = 0; jj < TPG; ++jj) {
            const int j = gi * TPG + jj;
            if (j + kPrefetch < kTilesPerWave)
                load_tile(j + kPrefetch, tiles[(j + kPrefetch) % (kPrefetch + 1)]);
            if (tile_valid(j)) {
                float x[8];
                tile_scores(tiles[j % (kPrefetch + 1)], j, x);
                if (j == 0) {
                    m_run = tile_max(x);
                    m_ref = m_run + (float)Ev;
                }
                tile_accumulate(j, x);
            }
        }
        __syncthreads();  // the next group's fold is in place; this group's buffer is free
    }
    bool unsafe = !(l_part < 1e30f) || !(fabsf(ob_part) < 1e30f);
#pragma unroll
    for (int n = 0; n < 8; ++n)
#pragma unroll
        for (int i = 0; i < 4; ++i) unsafe |= !(fabsf(acc[n][i]) < 1e30f);
#pragma unroll
    for (int i = 0; i < 4; ++i) unsafe |= !(fabsf(acc_off[i]) < 1e30f);
    if (__syncthreads_or(unsafe)) {
        // Slow path: running maximum with rescaling, one group and tile at a time.
        m_run = m_ref = -INFINITY;
        l_part = ob_part = 0.0f;
#pragma unroll
        for (int n = 0; n < 8; ++n) acc[n] = f32x4_t{0.f, 0.f, 0.f, 0.f};
        acc_off = f32x4_t{0.f, 0.f, 0.f, 0.f};
        for (int gi = 0; gi < n_groups; ++gi) {
            load_kmeta(gi);
            fold(0, gi);
            __syncthreads();
            load_group_operands(0);
            for (int jj = 0; jj < TPG; ++jj) {
                const int j = gi * TPG + jj;
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
#pragma unroll
                    for (int i = 0; i < 4; ++i) acc_off[i] *= af[i];
                }
                tile_accumulate(j, x);
            }
            __syncthreads();
        }
    }

    // ---- per-wavefront totals -> LDS (still scaled by 2^-Ev) ----
    // o' = sum p' z + sum pw (1024 + c) - 1024 sum pw
    l_part = sum_kg(l_part);
    ob_part = sum_kg(ob_part);
    if (kg == 0) {
        s_m[w][col] = m_run;
        s_l[w][col] = l_part;
        s_ob[w][col] = ob_part;
    }
    float *s_o = reinterpret_cast<float *>(s_raw);  // [wave][16 rows][128]
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int c = 0; c < 8; ++c)
            s_o[(w * 16 + 4 * kg + i) * kHeadDim + 16 * c + col] = acc[c][i] - acc_off[i];
    const bool any_bad = __syncthreads_or(bad);

    // ---- merge the wavefronts of each row tile, write this split's partial:
    // per-row factors first, then float4 multiply-adds ----
    __shared__ float s_f[kWaves][16], s_ML[RT * 16][2];
    if (tid < RT * 16) {
        const int rtile = tid / 16, r16 = tid % 16;
        float M = -INFINITY;
#pragma unroll
        for (int p = 0; p < NP; ++p) M = fmaxf(M, s_m[p * RT + rtile][r16]);
        const float ev_scale = ldexpf(1.0f, Ev);
        float L = 0.0f;
#pragma unroll
        for (int p = 0; p < NP; ++p) {
            const int ww = p * RT + rtile;
            const float f = (M == -INFINITY || s_m[ww][r16] == -INFINITY) ? 0.0f
                                                                           : exp2f(s_m[ww][r16] - M) * ev_scale;
            s_f[ww][r16] = f;
            L = fmaf(s_l[ww][r16], f, L);
        }
        s_ML[tid][0] = M;
        s_ML[tid][1] = any_bad ? NAN : L;
    }
    __syncthreads();
    for (int idx = tid; idx < RT * 16 * (kHeadDim / 4); idx += kThreads) {
        const int rr = idx / (kHeadDim / 4);  // row within the workgroup
        const int d4 = idx % (kHeadDim / 4);
        const int rtile = rr / 16, r16 = rr % 16;
        const int row = row_base + rr;
        if (row >= a.rows_total) continue;
        float4 O = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
        for (int p = 0; p < NP; ++p) {
            const int ww = p * RT + rtile;
            const float f = s_f[ww][r16];
            const float ob = s_ob[ww][r16];
            const float4 o = reinterpret_cast<const float4 *>(s_o + (ww * 16 + r16) * kHeadDim)[d4];
            O.x = fmaf(o.x + ob, f, O.x);
            O.y = fmaf(o.y + ob, f, O.y);
            O.z = fmaf(o.z + ob, f, O.z);
            O.w = fmaf(o.w + ob, f, O.w);
        }
        if (any_bad) O = make_float4(NAN, NAN, NAN, NAN);
        const size_t pi = partial_index(row);
        reinterpret_cast<float4 *>(a.ws_o + pi * kHeadDim)[d4] = O;
        if (d4 == 0) a.ws_ml[pi] = make_float2(s_ML[rr][0], s_ML[rr][1]);
    }
}

template <int RT, int LAYOUT>
void launch_rt(const VerifyArgs &args, int split_groups, dim3 grid, hipStream_t stream) {
    if (split_groups == 4)
        hipLaunchKernelGGL((verify_kernel<RT, LAYOUT, 4>), grid, dim3(kThreads), 0, stream, args);
    else
        hipLaunchKernelGGL((verify_kernel<RT, LAYOUT, 8>), grid, dim3(kThreads), 0, stream, args);
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
    if (split_groups != 4 && split_groups != 8) return hipErrorInvalidValue;
    const int rt = args.rows_total <= 16 ? 1 : 2;
    const int chunks = (args.rows_total + 16 * rt - 1) / (16 * rt);
    dim3 grid(args.n_ctx_splits, args.geo.Hkv * chunks, args.B);
    if (rt == 1)
        launch_layout<1>(args, split_groups, grid, stream);
    else
        launch_layout<2>(args, split_groups, grid, stream);
    return hipGetLastError();
}

}  // namespace lynx
