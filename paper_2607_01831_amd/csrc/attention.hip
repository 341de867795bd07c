// Attention over the split-stream KV cache for gfx950: planning and launch of
// the anchor-only decode (Sec. 4.2 Anchor phase; anchor_decode.hip) and of
// the verification pass over the merged 8-bit cache (Sec. 4.3; verify.hip),
// both O = softmax(q K^T / sqrt(128)) V (Sec. 2) split along the context,
// and the combine kernel that merges their per-split partials (max, sum,
// unnormalised output) and attends the BF16 tail: the drafts, causal among
// themselves, in verification, and the generated tokens in decode.
#include "lynx_internal.h"

#include <float.h>
#include <math.h>

#include <mutex>

namespace lynx {
namespace {

constexpr int kWaves = 4;  // wavefronts per decode / verification workgroup
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

struct AttnArgs {
    Geometry geo;
    int B, Hq, nq, G, max_seq_len;
    int rows_total, n_ctx_splits, n_splits, split_tokens;
    int split_base;  // split index of blockIdx.x == 0
    int tail_in_combine;  // the combine kernel attends the BF16 tail itself
    int tail_count;       // tokens of the tail every query sees; -1: query i sees i + 1 (drafts)
    int tail_stride;      // tail tokens stored per sequence in k_new / v_new
    const int32_t *seq_lens;
    const int32_t *block_table;
    const uint8_t *k_plane;
    const uint8_t *v_plane;
    MetaPtrs meta;
    const uint16_t *q;
    const uint16_t *k_new;
    const uint16_t *v_new;
    float *ws_o;    // [B][Hkv][rows_total][n_splits][128]
    float2 *ws_ml;  // [B][Hkv][rows_total][n_splits]
};

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

__device__ __forceinline__ void unpack8_bf16(const uint4 &u, float *x) {
    x[0] = bf16_lo(u.x); x[1] = bf16_hi(u.x);
    x[2] = bf16_lo(u.y); x[3] = bf16_hi(u.y);
    x[4] = bf16_lo(u.z); x[5] = bf16_hi(u.z);
    x[6] = bf16_lo(u.w); x[7] = bf16_hi(u.w);
}

// fp32 -> BF16 bits, round to nearest even (NaN -> a quiet NaN).
__device__ __forceinline__ uint16_t f32_to_bf16_rne(float f) {
    uint32_t u = __float_as_uint(f);
    if ((u & 0x7fffffffu) > 0x7f800000u) return 0x7fc0;  // NaN
    u += 0x7fffu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
}

constexpr int kCombineThreads = 256;

// One workgroup per (row, kv head, sequence): merge the partials of all
// splits and the BF16 tail tokens, normalise, round to BF16, write lse.
// Thread (split group sg, float4 column d4) folds every 8th split into a
// running (max, sum, output), loading kBatch splits' partial outputs and
// (max, sum) pairs together (8 when 64 splits or fewer, so no load is a
// clamped repeat; 16 above), then every 8th tail token the same way, as a
// partial of weight 1.  The 8 running triples meet in LDS.  Every load the
// kernel needs first (the first kBatch splits' partials, the tail's values,
// and the query and tail keys for the tail scores) is issued before any of
// them is used, so the kernel waits for memory once for up to 8 kBatch
// splits.
template <int kBatch>
__global__ __launch_bounds__(kCombineThreads) void attn_combine_kernel(AttnArgs a, uint16_t *out,
                                                                       float *lse) {
    const int gr = blockIdx.x;
    const int h = blockIdx.y;
    const int b = blockIdx.z;
    const int tid = threadIdx.x;
    const int Hkv = a.geo.Hkv;
    const size_t base = (((size_t)b * Hkv + h) * a.rows_total + gr) * a.n_splits;
    // splits with partials: every split, or the context ones when this kernel
    // attends the tail itself
    const int n = a.tail_in_combine ? a.n_ctx_splits : a.n_splits;
    constexpr int kGroups = kCombineThreads / (kHeadDim / 4);  // 8 split groups
    constexpr int kTailMax = 64;                   // tail tokens attended at most
    constexpr int kTailPer = kTailMax / kGroups;   // per split group
    __shared__ float4 s_acc[kGroups][kHeadDim / 4];
    __shared__ float s_m[kGroups][kHeadDim / 4], s_l[kGroups][kHeadDim / 4];
    __shared__ float s_ts[kTailMax];  // tail scores (log2 units)

    // query row gr <-> (query qi, head qg); with a tail, query qi also sees
    // the BF16 tokens of the tail: drafts 0..qi in verification (causal among
    // the drafts), all tail_count generated tokens in decode
    const int qi = gr / a.G;
    const int qg = gr % a.G;
    const size_t qrow = ((size_t)b * a.nq + qi) * a.Hq + (size_t)h * a.G + qg;
    const int n_tail = a.tail_in_combine ? (a.tail_count < 0 ? qi + 1 : a.tail_count) : 0;

    const int d4 = tid % (kHeadDim / 4);
    const int sg = tid / (kHeadDim / 4);
    const float4 *o4 = reinterpret_cast<const float4 *>(a.ws_o) + base * (kHeadDim / 4) + d4;
    // a batch of partials: splits s0, s0 + 8, ... (clamped to the last split)
    float4 v[kBatch];
    float2 ml[kBatch];
    bool live[kBatch];
    auto load_batch = [&](int s0) {
#pragma unroll
        for (int u = 0; u < kBatch; ++u) {
            const int s = min(s0 + kGroups * u, n - 1);
            v[u] = o4[(size_t)s * (kHeadDim / 4)];
            ml[u] = a.ws_ml[base + s];
            live[u] = s0 + kGroups * u < n;
        }
    };
    load_batch(sg);
    // this thread's tail values: tokens sg, sg + 8, ... (dims 4 d4 .. + 3)
    uint2 tvw[kTailPer];
    if (n_tail > 0) {
#pragma unroll
        for (int u = 0; u < kTailPer; ++u) {
            const int j = min(sg + kGroups * u, n_tail - 1);
            tvw[u] = *reinterpret_cast<const uint2 *>(
                a.v_new + (((size_t)b * a.tail_stride + j) * Hkv + h) * kHeadDim + 4 * d4);
        }
    }
    if (n_tail > 0) {
        // tail scores, 16 tokens per pass: thread (token tid / 16, dims
        // 8 (tid % 16) .. + 7), summed over the 16 lanes of a token
        const int piece = tid & 15;
        float qv[8];
        unpack8_bf16(*reinterpret_cast<const uint4 *>(a.q + qrow * kHeadDim + 8 * piece), qv);
        const float sm = kLog2e * rsqrtf((float)kHeadDim);
        uint4 kw[kTailMax / 16];
#pragma unroll
        for (int p = 0; p < kTailMax / 16; ++p) {
            const int j = min(16 * p + (tid >> 4), n_tail - 1);
            kw[p] = *reinterpret_cast<const uint4 *>(
                a.k_new + (((size_t)b * a.tail_stride + j) * Hkv + h) * kHeadDim + 8 * piece);
        }
#pragma unroll
        for (int p = 0; p < kTailMax / 16; ++p) {
            const int j = 16 * p + (tid >> 4);
            float kv[8];
            unpack8_bf16(kw[p], kv);
            float d = 0.0f;
#pragma unroll
            for (int e = 0; e < 8; ++e) d = fmaf(qv[e], kv[e], d);
#pragma unroll
            for (int off = 8; off > 0; off >>= 1) d += __shfl_xor(d, off);
            if (piece == 0 && j < n_tail) s_ts[j] = d * sm;
        }
        __syncthreads();
    }

    float m_t = -INFINITY, l_t = 0.0f;
    float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
    bool nan = false;
    // fold N partials (max mlv.x, sum mlv.y, output vv) into the running triple
    auto fold = [&](const auto &vv, auto &mlv, const auto &lv) {
        constexpr int N = sizeof(lv) / sizeof(lv[0]);
        float mb = m_t;
#pragma unroll
        for (int u = 0; u < N; ++u) {
            if (!lv[u]) mlv[u] = make_float2(-INFINITY, 0.0f);
            mb = fmaxf(mb, mlv[u].x);
        }
        const float sc = m_t == -INFINITY ? 0.0f : exp2f(m_t - mb);
        acc.x *= sc;
        acc.y *= sc;
        acc.z *= sc;
        acc.w *= sc;
        l_t *= sc;
#pragma unroll
        for (int u = 0; u < N; ++u) {
            const float e = mlv[u].x == -INFINITY ? 0.0f : exp2f(mlv[u].x - mb);
            nan |= isnan(mlv[u].y);
            l_t = fmaf(mlv[u].y, e, l_t);
            // a split with weight 0 may hold no partial output at all
            const float4 x = e != 0.0f ? vv[u] : make_float4(0.f, 0.f, 0.f, 0.f);
            acc.x = fmaf(x.x, e, acc.x);
            acc.y = fmaf(x.y, e, acc.y);
            acc.z = fmaf(x.z, e, acc.z);
            acc.w = fmaf(x.w, e, acc.w);
        }
        m_t = mb;
    };
    for (int s0 = sg; s0 < n; s0 += kGroups * kBatch) {
        if (s0 != sg) load_batch(s0);
        fold(v, ml, live);
    }
    // the tail tokens: partials (score, 1, value)
    if (n_tail > 0) {
        float4 tv[kTailPer];
        float2 tml[kTailPer];
        bool tlive[kTailPer];
#pragma unroll
        for (int u = 0; u < kTailPer; ++u) {
            const int j = sg + kGroups * u;
            tlive[u] = j < n_tail;
            tv[u] = make_float4(bf16_lo(tvw[u].x), bf16_hi(tvw[u].x), bf16_lo(tvw[u].y), bf16_hi(tvw[u].y));
            tml[u] = make_float2(tlive[u] ? s_ts[j] : -INFINITY, 1.0f);
        }
        fold(tv, tml, tlive);
    }
    s_acc[sg][d4] = acc;
    s_m[sg][d4] = m_t;
    s_l[sg][d4] = nan ? NAN : l_t;
    __syncthreads();
    if (sg == 0) {
        float M = -INFINITY;
#pragma unroll
        for (int g = 0; g < kGroups; ++g) M = fmaxf(M, s_m[g][d4]);
        float4 O = make_float4(0.f, 0.f, 0.f, 0.f);
        float L = 0.0f;
        bool any_nan = false;
#pragma unroll
        for (int g = 0; g < kGroups; ++g) {
            const float f = s_m[g][d4] == -INFINITY ? 0.0f : exp2f(s_m[g][d4] - M);
            const float4 o = s_acc[g][d4];
            O.x = fmaf(o.x, f, O.x);
            O.y = fmaf(o.y, f, O.y);
            O.z = fmaf(o.z, f, O.z);
            O.w = fmaf(o.w, f, O.w);
            any_nan |= isnan(s_l[g][d4]);
            L = fmaf(s_l[g][d4], f, L);
        }
        float r[4] = {O.x, O.y, O.z, O.w};
#pragma unroll
        for (int i = 0; i < 4; ++i) r[i] = any_nan ? NAN : (L > 0.0f ? r[i] / L : 0.0f);
        const size_t row = qrow;
        const uint32_t lo = f32_to_bf16_rne(r[0]) | ((uint32_t)f32_to_bf16_rne(r[1]) << 16);
        const uint32_t hi = f32_to_bf16_rne(r[2]) | ((uint32_t)f32_to_bf16_rne(r[3]) << 16);
        *reinterpret_cast<uint2 *>(out + row * kHeadDim + 4 * d4) = make_uint2(lo, hi);
        if (lse && d4 == 0)
            lse[row] = any_nan ? NAN : (L > 0.0f ? (M + log2f(L)) * kLn2 : -INFINITY);
    }
}

// Compute units of the current device (0 if unknown), queried once per device.
int compute_units() {
    constexpr int kMaxDevices = 64;
    static std::once_flag once[kMaxDevices];
    static int cus[kMaxDevices];
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return 0;
    std::call_once(once[dev], [dev]() {
        int n = 0;
        cus[dev] = hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess ? n : 0;
    });
    return cus[dev];
}

}  // namespace

AttnPlan plan_attention(const Geometry &g, int B, int Hq, int nq, int max_seq_len, bool tail) {
    AttnPlan p{};
    const int G = Hq / g.Hkv;
    p.rows_total = nq * G;
    // Context tokens per split: 512, doubled while the launch still fills
    // the chip (>= 1024 decode workgroups, two per CU; >= 512 verification
    // workgroups, also two per CU), so long contexts write fewer partials
    // and workgroups live longer: up to 2048 tokens (512 for decode when
    // 16-head chunks leave no LDS for more groups).
    p.split_tokens = kWaves * kKGroup;
    const int max_split = nq == 1 && G > 8 ? 512 : 2048;
    const int min_workgroups = nq == 1 ? 1024 : 512;
    while (p.split_tokens < max_split) {
        const long long next = ((long long)max_seq_len + 2 * p.split_tokens - 1) / (2 * p.split_tokens);
        if (next * g.Hkv * B < min_workgroups) break;
        p.split_tokens *= 2;
    }
    if (nq > 1 && g.max_blocks == 1) {
        // The same for verification of a contiguous batch (its combine kernel
        // still attends the draft tail, over fewer splits): 70B-shaped batch,
        // k = 4, 2048 workgroups of 2048 tokens 231 us, 512 of 8192 212 us.
        const int cus = compute_units();
        const int rt = p.rows_total <= 16 ? 1 : 2;
        const long long chunks = (p.rows_total + 16 * rt - 1) / (16 * rt);
        for (int st = p.split_tokens; cus > 0 && st <= 8192; st *= 2) {
            const long long splits = max_seq_len > 0 ? (max_seq_len + st - 1) / st : 1;
            if (splits * g.Hkv * chunks * B <= 2LL * cus) {
                p.split_tokens = st;
                break;
            }
        }
    }
    if (nq == 1 && !tail && g.max_blocks == 1 && G <= 8) {
        // A contiguous decode batch that fits one round of workgroups (two per
        // CU) with longer splits, up to 8192 tokens, takes them: the split
        // merge then runs in the same launch, and no workgroup waits for a
        // second round (70B-shaped batch, 4 x 128K tokens: 2048 workgroups of
        // 2048 tokens and the combine kernel, 112 us; 512 of 8192, 104 us).
        const int cus = compute_units();
        for (int st = p.split_tokens; cus > 0 && st <= 8192; st *= 2) {
            const long long splits = max_seq_len > 0 ? (max_seq_len + st - 1) / st : 1;
            if (splits * g.Hkv * B <= 2LL * cus) {
                p.split_tokens = st;
                break;
            }
        }
    }
    // at least one split, so that empty sequences still get (zero) outputs
    p.n_ctx_splits = max_seq_len > 0 ? (max_seq_len + p.split_tokens - 1) / p.split_tokens : 1;
    p.n_splits = p.n_ctx_splits + (tail ? 1 : 0);
    const size_t parts = (size_t)B * g.Hkv * p.rows_total * p.n_splits;
    p.o_bytes = parts * kHeadDim * sizeof(float);
    p.ml_bytes = parts * sizeof(float2);
    p.row_chunks = (p.rows_total + 15) / 16;
    p.counters_fit = (long long)B * g.Hkv * p.row_chunks <= kCounters;
    return p;
}

hipError_t launch_attention(KvMode mode, const Geometry &g, const AttnPlan &plan, int B, int Hq,
                            int nq, int max_seq_len, const int32_t *seq_lens,
                            const int32_t *block_table, const uint8_t *k_plane,
                            const uint8_t *v_plane, MetaPtrs meta, const uint16_t *q,
                            const uint16_t *k_new, const uint16_t *v_new, int tail_count,
                            uint16_t *out,
                            float *lse, void *workspace, hipStream_t stream, int anchor_bits) {
    if (B == 0 || plan.n_splits == 0) return hipSuccess;
    AttnArgs a;
    a.geo = g;
    a.B = B;
    a.Hq = Hq;
    a.nq = nq;
    a.G = Hq / g.Hkv;
    a.max_seq_len = max_seq_len;
    a.rows_total = plan.rows_total;
    a.n_ctx_splits = plan.n_ctx_splits;
    a.n_splits = plan.n_splits;
    a.split_tokens = plan.split_tokens;
    a.split_base = 0;
    // the matrix-core paths leave the BF16 tail to the combine kernel:
    // causal drafts in verification, tail_count generated tokens in decode
    const bool mfma_path = mode == KvMode::kCodes || nq == 1;
    a.tail_in_combine = (mfma_path && k_new != nullptr) ? 1 : 0;
    a.tail_count = mode == KvMode::kCodes ? -1 : tail_count;
    a.tail_stride = mode == KvMode::kCodes ? nq : tail_count;
    a.seq_lens = seq_lens;
    a.block_table = block_table;
    a.k_plane = k_plane;
    a.v_plane = v_plane;
    a.meta = meta;
    a.q = q;
    a.k_new = k_new;
    a.v_new = v_new;
    a.ws_o = reinterpret_cast<float *>(reinterpret_cast<char *>(workspace) + kCounterBytes);
    a.ws_ml = reinterpret_cast<float2 *>(reinterpret_cast<char *>(workspace) + kCounterBytes +
                                         plan.o_bytes);
    if (mode == KvMode::kAnchor && nq == 1) {
        // matrix-core decode over the anchor nibbles
        DecodeArgs d;
        d.geo = g;
        d.B = B;
        d.Hq = Hq;
        d.G = a.G;
        d.max_seq_len = max_seq_len;
        d.n_splits = plan.n_ctx_splits;
        d.groups_per_split = plan.split_tokens / kKGroup;
        d.chunk_heads = a.G < 16 ? a.G : 16;
        d.bt_shift = -1;
        for (int sh = 0; sh < 31; ++sh)
            if ((1 << sh) == g.bt) d.bt_shift = sh;
        d.meta_vec4 = (g.max_tokens % 4 == 0) ? 1 : 0;
        d.seq_lens = seq_lens;
        d.block_table = block_table;
        d.k_anc = k_plane;
        d.v_anc = v_plane;
        d.meta = meta;
        d.q = q;
        d.ws_o = a.ws_o;
        d.ws_ml = a.ws_ml;
        d.rows_total = plan.rows_total;
        d.ws_splits = plan.n_splits;
        // without a tail the last workgroup of each (sequence, kv head, head
        // chunk) merges the splits itself: no second launch
        // The in-kernel merge costs every workgroup a wait for its partial's
        // stores and an atomic (about 1.2 us), during which it holds its CU
        // slot: a win when the whole grid runs in one round (two workgroups
        // per CU), a loss over several rounds, where the combine kernel
        // merges instead (70B batch: 126 us per step with the combine, 133
        // fused; 32K layer: 17.7 us with the combine, 15.9 fused).  The merge
        // holds up to two splits' (max, sum) per thread: 256 / GP threads per
        // row, GP = 4, 8 or 16 rows padded.
        const int gp = d.chunk_heads <= 4 ? 4 : d.chunk_heads <= 8 ? 8 : 16;
        const int chunks_ = (a.G + d.chunk_heads - 1) / d.chunk_heads;
        const long long wgs = (long long)plan.n_ctx_splits * g.Hkv * chunks_ * B;
        const bool one_round = wgs <= 2LL * compute_units();
        d.fused = (k_new == nullptr && plan.counters_fit && plan.n_ctx_splits <= 2 * (256 / gp) &&
                   one_round) ? 1 : 0;
        d.row_chunks = plan.row_chunks;
        d.counters = reinterpret_cast<unsigned *>(workspace);
        d.out = out;
        d.lse = lse;
        const int chunks = (a.G + d.chunk_heads - 1) / d.chunk_heads;
        hipError_t e = launch_anchor_decode_mfma(d, chunks, stream);
        if (e != hipSuccess) return e;
        if (d.fused) return hipSuccess;
    } else if (mode == KvMode::kAnchorSplit && nq == 1 && k_new == nullptr) {
        // matrix-core decode over A-bit anchors; the combine kernel below
        // merges its splits
        SplitDecodeArgs d;
        d.geo = g;
        d.B = B;
        d.Hq = Hq;
        d.G = a.G;
        d.max_seq_len = max_seq_len;
        d.anchor_bits = anchor_bits;
        d.n_splits = plan.n_ctx_splits;
        d.groups_per_split = plan.split_tokens / kKGroup;
        d.rows_total = plan.rows_total;
        d.ws_splits = plan.n_splits;
        d.seq_lens = seq_lens;
        d.block_table = block_table;
        d.k_anc = k_plane;
        d.v_anc = v_plane;
        d.meta = meta;
        d.q = q;
        d.ws_o = a.ws_o;
        d.ws_ml = a.ws_ml;
        // the split merge in the same launch, under the rule of the 4-bit
        // decode: one round of workgroups, and at most 2 * 256 / GP splits
        // for the merging workgroup (GP: the chunk's rows, padded)
        const int gp = a.G <= 4 ? 4 : a.G <= 8 ? 8 : 16;
        const long long wgs = (long long)plan.n_ctx_splits * g.Hkv * plan.row_chunks * B;
        d.fused = (plan.counters_fit && plan.n_ctx_splits <= 2 * (256 / gp) &&
                   wgs <= 2LL * compute_units()) ? 1 : 0;
        d.row_chunks = plan.row_chunks;
        d.counters = reinterpret_cast<unsigned *>(workspace);
        d.out = out;
        d.lse = lse;
        hipError_t e = launch_anchor_split_decode(d, stream);
        if (e != hipSuccess) return e;
        if (d.fused) return hipSuccess;
    } else if (mode == KvMode::kCodes) {
        // matrix-core verification over the context splits ...
        VerifyArgs v;
        v.geo = g;
        v.B = B;
        v.Hq = Hq;
        v.G = a.G;
        v.nq = nq;
        v.max_seq_len = max_seq_len;
        v.rows_total = plan.rows_total;
        v.n_ctx_splits = plan.n_ctx_splits;
        v.ws_splits = plan.n_splits;
        v.bt_shift = -1;
        for (int sh = 0; sh < 31; ++sh)
            if ((1 << sh) == g.bt) v.bt_shift = sh;
        v.seq_lens = seq_lens;
        v.block_table = block_table;
        v.k_codes = k_plane;
        v.v_codes = v_plane;
        v.meta = meta;
        v.q = q;
        v.ws_o = a.ws_o;
        v.ws_ml = a.ws_ml;
        hipError_t e = launch_verify_mfma(v, plan.split_tokens / kKGroup, stream);
        if (e != hipSuccess) return e;
        // the BF16 draft tail is attended by the combine kernel below
    } else {
        return hipErrorInvalidValue;  // anchor attention with several queries: no entry point asks for it
    }
    const int n_merged = a.tail_in_combine ? a.n_ctx_splits : a.n_splits;
    if (n_merged <= 64)
        hipLaunchKernelGGL(attn_combine_kernel<8>, dim3(plan.rows_total, g.Hkv, B), dim3(kCombineThreads),
                           0, stream, a, out, lse);
    else
        hipLaunchKernelGGL(attn_combine_kernel<16>, dim3(plan.rows_total, g.Hkv, B), dim3(kCombineThreads),
                           0, stream, a, out, lse);
    return hipGetLastError();
}

}  // namespace lynx
