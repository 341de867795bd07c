// Internal declarations shared by the HIP translation units of liblynx.so.
// Not part of the public ABI (include/lynx.h is).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace lynx {

constexpr int kHeadDim = 128;    // D
constexpr int kKGroup = 128;     // tokens per K quantization group
constexpr int kNibbleRow = 64;   // bytes per token row of a nibble plane
constexpr int kCodeRow = 128;    // bytes per token row of a code plane

// Geometry of a plane pool as the kernels see it.
struct Geometry {
    int Hkv;
    int bt;            // tokens per block
    int max_blocks;    // block_table row stride
    int num_blocks;    // valid block ids are [0, num_blocks)
    int max_tokens;    // metadata token stride
    int n_groups;      // ceil(max_tokens / 128): K metadata group stride
    int n_pages;       // ceil(max_tokens / 256): hierarchical page stride
    int n_chunks;      // ceil(max_tokens / 32): hierarchical chunk stride
};

struct MetaPtrs {
    float *k_scale, *k_zero, *v_scale, *v_zero;
};

// ---- encode / merge (codec.hip) ---------------------------------------------
hipError_t launch_encode(const Geometry &g, int b, int T, const int32_t *block_table,
                         const uint16_t *k, const uint16_t *v, uint8_t *k_anc, uint8_t *v_anc,
                         uint8_t *k_res, uint8_t *v_res, MetaPtrs meta, hipStream_t stream,
                         int anchor_bits = 4);
// Split widths other than 4 + 4: rows of 16 A-bit anchors per 16 A bytes
// (little-endian bit strings) and 16 (8 - A) residual bytes.
hipError_t launch_merge_split(int anchor_bits, const uint8_t *anc, const uint8_t *res, uint8_t *codes,
                              size_t n_rows, hipStream_t stream);
hipError_t launch_dequant_anchor_split(int anchor_bits, const Geometry &g, int b, int T,
                                       const int32_t *block_table, const uint8_t *k_anc,
                                       const uint8_t *v_anc, MetaPtrs meta, uint16_t *k_out,
                                       uint16_t *v_out, hipStream_t stream);
hipError_t launch_merge(const uint8_t *anc, const uint8_t *res, uint8_t *codes, size_t n_packed,
                        hipStream_t stream);

// ---- hierarchical codec of Alg. 1 (hier.hip) ----------------------------------
struct HMetaPtrs {
    float *k_gmin, *k_gscale, *k_mu, *k_sigma;  // [B][Hkv][n_pages][128], [B][Hkv][n_chunks][128]
    float *v_gmin, *v_gscale, *v_mu, *v_sigma;
};
// Codec variants (the values of lynx.h's LYNX_HQ_*).
constexpr int kHBiased = 0;
constexpr int kHCentred = 1;
constexpr int kHInt4 = 2;
// Per-(alpha, variant) tables, with M = 127 (7 for the 4-bit code): decision
// thresholds theta[k] = expm1((k + 0.5) / M * log1p(alpha)) / alpha for
// k < M, +inf beyond; levels level[i] = expm1(i / M * log1p(alpha)) / alpha
// (i <= M); the centred split's anchor-only levels alevel[V] at code
// 16 V + 7.5 of 127.  Each the fp32 value of the double expression.
// The encode's first guess at a code: yscale * log2(1 + alpha |Xf|), or
// yscale * |Xf| when `linear` (alpha < 1e-3), with yscale = M / log2(1 + alpha)
// (or M), is within one of the count the thresholds decide.
struct HTables {
    float theta[128];
    float level[128];
    float alevel[8];
    float alpha, yscale;
    int linear, levels;
};
void make_htables(float alpha, int variant, HTables *t);
hipError_t launch_hencode(const Geometry &g, int b, int T, const int32_t *block_table,
                          const uint16_t *k, const uint16_t *v, uint8_t *k_anc, uint8_t *v_anc,
                          uint8_t *k_res, uint8_t *v_res, HMetaPtrs meta, const HTables &tab,
                          int variant, hipStream_t stream);
hipError_t launch_hdequant(bool full, const Geometry &g, int b, int T, const int32_t *block_table,
                           const uint8_t *k_plane, const uint8_t *v_plane, HMetaPtrs meta,
                           const HTables &tab, int variant, uint16_t *k_out, uint16_t *v_out,
                           hipStream_t stream);

// ---- serializer / deserializer (codec.hip) -----------------------------------
// Object: tokens t0 .. t0 + n - 1 of one sequence, all kv heads.  Anchor
// buffer: K, V anchor rows [Hkv][n][64], K scales, K zeros [Hkv][ceil(n/128)][128],
// V scales, V zeros [Hkv][n]; residual buffer: K, V residual rows.
hipError_t launch_serialize(int Hkv, int n, const uint16_t *k, const uint16_t *v,
                            uint8_t *anc_buf, uint8_t *res_buf, hipStream_t stream);
hipError_t launch_deserialize_anchor(const Geometry &g, int b, int t0, int n,
                                     const int32_t *block_table, const uint8_t *buf,
                                     uint8_t *k_anc, uint8_t *v_anc, MetaPtrs meta,
                                     hipStream_t stream);
hipError_t launch_deserialize_residual(const Geometry &g, int b, int t0, int n,
                                       const int32_t *block_table, const uint8_t *buf,
                                       const uint8_t *k_anc, const uint8_t *v_anc,
                                       uint8_t *k_codes, uint8_t *v_codes, hipStream_t stream);

// ---- attention (attention.hip) ----------------------------------------------
// Arrival counters at the head of every attention workspace (the value of
// lynx.h's LYNX_ATTN_COUNTER_BYTES): zero before a workspace's first use,
// left zero by every call.
// One counter per 256 bytes: arrivals on one cache line serialise (512
// workgroups counting in on one line took 5 us, 64 per line 0.4 us).
constexpr size_t kCounterBytes = 262144;
constexpr int kCounterStride = 64;  // uint32 slots between counters
constexpr int kCounters = (int)(kCounterBytes / (kCounterStride * sizeof(unsigned)));
enum class KvMode : int { kAnchor = 0, kCodes = 1, kAnchorSplit = 2 };

struct AttnPlan {
    int rows_total;   // nq * G query rows per (sequence, kv head)
    int split_tokens; // context tokens per split
    int n_ctx_splits; // ceil(max_seq_len / split_tokens)
    int n_splits;     // n_ctx_splits (+1 when a BF16 draft tail is attended)
    int row_chunks;   // ceil(rows_total / 16): arrival counters per (sequence, kv head)
    bool counters_fit;  // B * Hkv * row_chunks <= kCounters
    size_t o_bytes;   // workspace bytes for the partial outputs
    size_t ml_bytes;  // workspace bytes for the partial (max, sum) pairs
    // [arrival counters, kCounterBytes][outputs][(max, sum)]: the counters sit
    // at the same place for every call shape, so calls of different shapes
    // can share a workspace without one's partials landing on the counters
    size_t workspace_bytes() const { return kCounterBytes + o_bytes + ml_bytes; }
};

// Arguments of the matrix-core anchor decode kernel (anchor_decode.hip).
struct DecodeArgs {
    Geometry geo;
    int B, Hq, G, max_seq_len;
    int n_splits, groups_per_split, chunk_heads;
    int bt_shift;   // log2(block_tokens) when it is a power of two, else -1
    int meta_vec4;  // max_tokens % 4 == 0: V metadata loads may be 16 bytes
    const int32_t *seq_lens;
    const int32_t *block_table;
    const uint8_t *k_anc;
    const uint8_t *v_anc;
    MetaPtrs meta;
    const uint16_t *q;
    float *ws_o;    // split partials, same layout as the attention workspace
    float2 *ws_ml;
    int rows_total, ws_splits;
    // Fused split merge: the last workgroup of a (sequence, kv head, head
    // chunk) to finish merges its splits' partials and writes out / lse.
    // Arrival counters uint32 [B][Hkv][row_chunks], zero on entry, left zero.
    int fused;
    int row_chunks;
    unsigned *counters;
    uint16_t *out;  // BF16 [B][Hq][128]
    float *lse;     // fp32 [B][Hq] or nullptr
};

hipError_t launch_anchor_decode_mfma(const DecodeArgs &args, int chunks, hipStream_t stream);

// Arguments of the matrix-core verification kernel (verify.hip): context
// splits only; the combine kernel attends the BF16 draft tail.
struct VerifyArgs {
    Geometry geo;
    int B, Hq, G, nq, max_seq_len;
    int rows_total;    // nq * G query rows per (sequence, kv head)
    int n_ctx_splits;  // grid.x
    int ws_splits;     // partial-row stride (context splits + tail)
    int bt_shift;      // log2(block_tokens) when it is a power of two, else -1
    const int32_t *seq_lens;
    const int32_t *block_table;
    const uint8_t *k_codes;
    const uint8_t *v_codes;
    MetaPtrs meta;
    const uint16_t *q;  // BF16 [B][nq][Hq][128]
    float *ws_o;
    float2 *ws_ml;
};

hipError_t launch_verify_mfma(const VerifyArgs &args, int split_groups, hipStream_t stream);

// Arguments of the anchor decode over split-width anchors (anchor_split.hip):
// one query per sequence over A-bit anchor planes (rows of 16 A bytes);
// context splits only, merged by the combine kernel.
struct SplitDecodeArgs {
    Geometry geo;
    int B, Hq, G, max_seq_len;
    int anchor_bits;      // A: 2, 4 or 6
    int n_splits;         // grid.x
    int groups_per_split; // 4, 8 or 16
    int rows_total;       // G query rows per (sequence, kv head)
    int ws_splits;        // partial-row stride
    const int32_t *seq_lens;
    const int32_t *block_table;
    const uint8_t *k_anc;
    const uint8_t *v_anc;
    MetaPtrs meta;
    const uint16_t *q;    // BF16 [B][Hq][128]
    float *ws_o;
    float2 *ws_ml;
    // split merge in the same launch (as DecodeArgs): arrival counters
    // uint32 [B][Hkv][row_chunks], zero on entry, left zero
    int fused;
    int row_chunks;
    unsigned *counters;
    uint16_t *out;        // BF16 [B][Hq][128]
    float *lse;           // fp32 [B][Hq] or nullptr
};

hipError_t launch_anchor_split_decode(const SplitDecodeArgs &args, hipStream_t stream);

AttnPlan plan_attention(const Geometry &g, int B, int Hq, int nq, int max_seq_len, bool tail);

// k_new / v_new: the BF16 tail, or nullptr.  Verification (kCodes): k drafts
// per sequence, causal among the drafts.  Decode (kAnchor, nq == 1):
// tail_count generated tokens per sequence, all visible to the query.
hipError_t launch_attention(KvMode mode, const Geometry &g, const AttnPlan &plan, int B, int Hq,
                            int nq, int max_seq_len, const int32_t *seq_lens,
                            const int32_t *block_table, const uint8_t *k_plane,
                            const uint8_t *v_plane, MetaPtrs meta, const uint16_t *q,
                            const uint16_t *k_new, const uint16_t *v_new, int tail_count,
                            uint16_t *out, float *lse, void *workspace, hipStream_t stream,
                            int anchor_bits = 4);

// ---- acceptance of drafts (spec.hip) ------------------------------------------
// Sampled acceptance workspace: B * (k + 1) * spec_accept_chunks(vocab) pairs of
// uint64 chunk sums.
hipError_t launch_spec_accept_sample(int B, int k, int vocab, const float *p, const float *q,
                                     const int32_t *drafts, const float *u, int32_t *accepted,
                                     int32_t *next_token, void *workspace, hipStream_t stream);
// greedy acceptance
// Workspace: B * (k + 1) * spec_accept_chunks(vocab) (score, index) pairs.
int spec_accept_chunks(int vocab);
hipError_t launch_spec_accept_greedy(int B, int k, int vocab, const float *logits,
                                     const int32_t *drafts, int32_t *accepted,
                                     int32_t *next_token, void *workspace, hipStream_t stream);

}  // namespace lynx
