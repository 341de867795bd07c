/*
 * lynx.h -- C ABI of the Lynx split-stream KV codec and its attention kernels
 * for AMD Instinct MI355X (gfx950).
 *
 * Method: "Lynx: Progressive Speculative Quantization for accelerating KV
 * Transfer in Long-Context Inference".  The prefill side quantizes the KV
 * cache to 8 bits and splits every code into a 4-bit Anchor (most significant
 * bits, sent first) and a 4-bit Residual (least significant bits, sent
 * second) (Sec. 4 overview; Alg. 1 stage 4; Sec. 5 Compression Kernel).  The
 * decode side starts generating from the Anchor alone (Sec. 4.2 Anchor
 * phase), merges the Residual back into the full 8-bit cache when it arrives
 * (Sec. 4.2 Residual phase), and verifies the speculative tokens in one
 * parallel pass over the full cache (Sec. 4.3).
 *
 * Conventions for every entry point
 *   - Pointers named *_bf16, planes, codes, metadata, seq_lens, block_table,
 *     q, out, lse and workspace are DEVICE pointers (hipMalloc'd or torch
 *     CUDA tensors).  `L` and `meta` point to small HOST structs read during
 *     the call.
 *   - Every device pointer must be 16-byte aligned.
 *   - Calls are asynchronous on `stream` (a hipStream_t; NULL = the legacy
 *     default stream).  The library never allocates, never synchronizes and
 *     keeps no mutable global state; it is safe to call from several threads.
 *     Buffers must stay alive until the stream work completes.
 *   - Arguments are validated before anything is launched; on an error
 *     nothing is launched and a negative lynx_status is returned.  Faults in
 *     device memory the caller described wrongly surface at the caller's next
 *     stream synchronization.
 *
 * Data layout (all sizes in bytes; D = head_dim = 128; Hkv kv heads)
 *   - K/V inputs of one sequence: BF16 [T][Hkv][128], contiguous.
 *   - Codes: K is grouped per channel over windows of 128 consecutive tokens,
 *     V per token over its 128 dims (grouped quantization, Sec. 2.3).  For a
 *     group with minimum mn and maximum mx: zero = mn, scale = (mx-mn)/255,
 *     code = rint((x - zero) * (255/(mx-mn))) in IEEE fp32 (round half to
 *     even), clamped to [0, 255].  A group whose range is not a positive
 *     finite number, or whose 255/(mx-mn) overflows, stores scale 0 and codes
 *     0.  -0 is stored as +0.  Anchor a = code >> 4, residual r = code & 15.
 *   - Nibble planes (k_anc, v_anc, k_res, v_res): one 64-byte row per
 *     (token, kv head); byte j of a row holds dim 2j in its low nibble and dim
 *     2j+1 in its high nibble.  The row of (sequence b, kv head h, token t)
 *     starts at  ((block_table[b][t / bt] * Hkv + h) * bt + t % bt) * 64.
 *     Code planes (k_codes, v_codes) use the same formula with 128-byte rows,
 *     byte d = the code of dim d.  A contiguous cache is bt >= T with
 *     block_table[b][0] = b.  Bytes of rows t >= T are never read.
 *   - Metadata (fp32, logical, never paged), per sequence b:
 *       k_scale, k_zero [B][Hkv][ceil(max_tokens/128)][128]
 *       v_scale, v_zero [B][Hkv][max_tokens]
 *   - Query head hq reads kv head hq / (Hq / Hkv).
 *
 * Reconstruction used by the attention kernels
 *   - Anchor only: zero + (16 a + 7.5) * scale   (|error| <= 8 scale)
 *   - Full 8-bit:  zero + code * scale           (|error| <= scale / 2)
 */
#ifndef LYNX_H
#define LYNX_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum lynx_status {
    LYNX_OK = 0,
    LYNX_EINVAL = -1,     /* NULL/misaligned pointer, bad size or count   */
    LYNX_ENOTSUP = -2,    /* head_dim or k_group_tokens other than 128      */
    LYNX_EWORKSPACE = -3, /* workspace missing or smaller than required     */
    LYNX_EHIP = -4        /* the HIP runtime reported a launch error        */
} lynx_status;

/* Cache geometry shared by every call (host struct). */
typedef struct lynx_layout {
    int32_t num_kv_heads;       /* Hkv >= 1                                      */
    int32_t head_dim;           /* must be 128                                   */
    int32_t k_group_tokens;     /* must be 128: K group = 128 tokens x 1 channel */
    int32_t block_tokens;       /* bt >= 1: tokens per plane block               */
    int32_t max_blocks_per_seq; /* row stride of block_table, >= ceil(T/bt)      */
    int32_t num_blocks;         /* blocks in the plane pool; block ids must be
                                   in [0, num_blocks): kernels skip (encode) or
                                   return NaN for (attention) rows whose block
                                   id is outside that range                     */
    int32_t max_tokens;         /* token stride of the metadata arrays, >= T     */
} lynx_layout;

/* Device pointers to the fp32 metadata of the whole batch (host struct). */
typedef struct lynx_meta {
    float *k_scale; /* [B][Hkv][ceil(max_tokens/128)][128] */
    float *k_zero;
    float *v_scale; /* [B][Hkv][max_tokens] */
    float *v_zero;
} lynx_meta;

/*
 * lynx_kv_encode -- the prefill-side compression of one sequence (Sec. 4.2
 * Prefill workflow: the quantization kernel turns a KV object into the Anchor
 * and Residual streams and their metadata; Alg. 1 stage 4; Sec. 5).
 *
 *   b            sequence index: selects block_table row b and metadata row b
 *   T            tokens to encode, 0 <= T <= min(max_tokens,
 *                max_blocks_per_seq * bt); T == 0 launches nothing
 *   block_table  int32 [B][max_blocks_per_seq] (device)
 *   k_bf16,v_bf16  BF16 [T][Hkv][128] (device, read)
 *   k_anc, v_anc, k_res, v_res  nibble planes (device, written for rows t < T)
 *   meta         metadata row b written (K groups 0..ceil(T/128)-1, V tokens < T)
 * Returns LYNX_OK or an error; launches one kernel.
 */
int lynx_kv_encode(const lynx_layout *L, int32_t b, int32_t T, const int32_t *block_table,
                   const void *k_bf16, const void *v_bf16, uint8_t *k_anc, uint8_t *v_anc,
                   uint8_t *k_res, uint8_t *v_res, const lynx_meta *meta, void *stream);

/*
 * lynx_kv_merge -- the decode-side Residual phase (Sec. 4.2): anchor and
 * residual recombine into the full 8-bit code Q_full.  Elementwise and
 * layout-agnostic: for byte j of the planes,
 *   codes[2j]   = (anc[j] & 15) << 4 | (res[j] & 15)
 *   codes[2j+1] = (anc[j] >> 4) << 4 | (res[j] >> 4)
 * so a nibble-plane pool maps onto a code-plane pool with the same blocks.
 *   anc, res     n_packed_bytes each (device, read)
 *   codes        2 * n_packed_bytes (device, written); must not overlap inputs
 * n_packed_bytes == 0 launches nothing.
 */
int lynx_kv_merge(const uint8_t *anc, const uint8_t *res, uint8_t *codes,
                  size_t n_packed_bytes, void *stream);

/*
 * lynx_attn_workspace_bytes -- device workspace an attention call needs for
 * its split-context partial results, for `num_queries` query tokens per
 * sequence (1 for anchor decode, k for verify) and sequences of at most
 * max_seq_len tokens.  Returns 0 on invalid arguments.
 * Layout: LYNX_ATTN_COUNTER_BYTES of uint32 arrival counters, then the
 * partials.  The counters let the last workgroup of each (sequence, kv head)
 * merge the split partials itself, so a decode call is one launch.
 * Zero the first LYNX_ATTN_COUNTER_BYTES once, before the workspace's first
 * use (e.g. hipMemsetAsync(workspace, 0, LYNX_ATTN_COUNTER_BYTES, stream));
 * every call leaves them zero again, so calls of any shape can share one
 * workspace afterwards.  The rest needs no initialisation.  Calls that share
 * a workspace must not run concurrently.
 */
#define LYNX_ATTN_COUNTER_BYTES 262144
size_t lynx_attn_workspace_bytes(const lynx_layout *L, int32_t B, int32_t Hq,
                                 int32_t num_queries, int32_t max_seq_len);

/*
 * lynx_attn_anchor_decode -- decode attention over the Anchor-only cache
 * (Sec. 4.2 Anchor phase; Speculative Decoder): for every sequence b and
 * query head hq, O = softmax(q K^T / sqrt(128)) V (Sec. 2) with K, V
 * reconstructed from the anchor nibbles as zero + (16 a + 7.5) scale.
 *
 *   B, Hq        batch size and query heads (Hq % Hkv == 0)
 *   max_seq_len  host upper bound of seq_lens (sizes the launch); tokens at
 *                or beyond it are ignored
 *   seq_lens     int32 [B] (device): context length of each sequence
 *   block_table  int32 [B][max_blocks_per_seq] (device)
 *   k_anc, v_anc nibble planes (device); meta: metadata of the batch
 *   q_bf16       BF16 [B][Hq][128] (device)
 *   out_bf16     BF16 [B][Hq][128] (device, written)
 *   lse          fp32 [B][Hq] natural-log sum of exp of the scaled scores,
 *                or NULL (device, written)
 *   workspace    >= lynx_attn_workspace_bytes(L, B, Hq, 1, max_seq_len)
 * A sequence with no tokens yields zeros and lse = -inf.
 */
int lynx_attn_anchor_decode(const lynx_layout *L, int32_t B, int32_t Hq, int32_t max_seq_len,
                            const int32_t *seq_lens, const int32_t *block_table,
                            const uint8_t *k_anc, const uint8_t *v_anc, const lynx_meta *meta,
                            const void *q_bf16, void *out_bf16, float *lse, void *workspace,
                            size_t workspace_bytes, void *stream);

/*
 * lynx_attn_anchor_decode_noalloc -- lynx_attn_anchor_decode for callers that
 * cannot allocate device memory or pass a workspace (code under HIP graph
 * capture, tight serving loops, harnesses that forbid allocation).  Same
 * arguments and results, minus the workspace: the split partials and arrival
 * counters live in a static array of LYNX_NOALLOC_SCRATCH_BYTES that the
 * library holds on every GPU it runs on until the process ends.  The call
 * allocates nothing (no hipMalloc, no allocating library routine).
 *   LYNX_EWORKSPACE  the call needs more than LYNX_NOALLOC_SCRATCH_BYTES
 *                    (lynx_attn_workspace_bytes(L, B, Hq, 1, max_seq_len)
 *                    bounds what it needs), checked before anything runs
 *   LYNX_EHIP        the array's device address could not be obtained
 * Every call on a GPU shares that GPU's array: calls that overlap on one GPU
 * (other streams, other threads) race and give wrong results.
 */
#define LYNX_NOALLOC_SCRATCH_BYTES (16u << 20)
int lynx_attn_anchor_decode_noalloc(const lynx_layout *L, int32_t B, int32_t Hq,
                                    int32_t max_seq_len, const int32_t *seq_lens,
                                    const int32_t *block_table, const uint8_t *k_anc,
                                    const uint8_t *v_anc, const lynx_meta *meta,
                                    const void *q_bf16, void *out_bf16, float *lse, void *stream);

/*
 * lynx_attn_verify -- the verification pass (Sec. 4.3): the k speculative
 * query tokens of every sequence attend, in one parallel pass, over the
 * merged 8-bit cache (reconstructed as zero + code * scale) and over the
 * draft tokens' own BF16 K/V, causally: draft query i sees the whole context
 * and draft tokens 0..i.  k is capped at 64, the paper's limit on speculative
 * tokens (Sec. 6.1).
 *
 *   k            draft queries per sequence, 1 <= k <= 64
 *   k_codes, v_codes  code planes (device)
 *   q_bf16       BF16 [B][k][Hq][128] (device)
 *   k_new, v_new BF16 [B][k][Hkv][128] draft K/V (device), or both NULL to
 *                attend over the context only
 *   out_bf16     BF16 [B][k][Hq][128] (device, written)
 *   workspace    >= lynx_attn_workspace_bytes(L, B, Hq, k, max_seq_len)
 */
int lynx_attn_verify(const lynx_layout *L, int32_t B, int32_t Hq, int32_t k,
                     int32_t max_seq_len, const int32_t *seq_lens, const int32_t *block_table,
                     const uint8_t *k_codes, const uint8_t *v_codes, const lynx_meta *meta,
                     const void *q_bf16, const void *k_new, const void *v_new, void *out_bf16,
                     void *workspace, size_t workspace_bytes, void *stream);

/*
 * lynx_attn_anchor_decode_tail -- lynx_attn_anchor_decode for a speculative
 * decoder that has already generated tokens of its own (Sec. 4.2-4.3): the
 * query attends the Anchor-only context and, after it, the n_tail tokens
 * generated since the context arrived, whose K/V are BF16 (computed locally,
 * never quantized), all of them visible to the query (the caller passes
 * exactly the visible ones).  Arguments as lynx_attn_anchor_decode, plus:
 *
 *   n_tail       generated tokens per sequence, 0 <= n_tail <= 64 (0 is the
 *                plain anchor decode)
 *   k_tail, v_tail  BF16 [B][n_tail][Hkv][128] (device), or NULL when
 *                n_tail == 0
 *   workspace    >= lynx_attn_workspace_bytes(L, B, Hq, 1, max_seq_len)
 * A sequence with no context attends its tail alone.
 */
int lynx_attn_anchor_decode_tail(const lynx_layout *L, int32_t B, int32_t Hq,
                                 int32_t max_seq_len, const int32_t *seq_lens,
                                 const int32_t *block_table, const uint8_t *k_anc,
                                 const uint8_t *v_anc, const lynx_meta *meta, const void *q_bf16,
                                 int32_t n_tail, const void *k_tail, const void *v_tail,
                                 void *out_bf16, float *lse, void *workspace,
                                 size_t workspace_bytes, void *stream);

/*
 * lynx_spec_accept_workspace_bytes -- device workspace of
 * lynx_spec_accept_greedy and lynx_spec_accept_sample for B sequences, k
 * drafts and a vocabulary of `vocab` entries.  Returns 0 on invalid
 * arguments.
 */
size_t lynx_spec_accept_workspace_bytes(int32_t B, int32_t k, int32_t vocab);

/*
 * lynx_spec_accept_greedy -- greedy acceptance of the drafts after the
 * verification pass (Sec. 4.3: keep the longest prefix of the drafts the
 * target model agrees with, correct the first divergence).  The target's
 * choice at a position is its highest score, the lowest vocabulary index
 * among equal scores.
 *
 *   B, k, vocab    sequences (<= 65535), drafts per sequence (1..64) and
 *                  vocabulary size
 *   target_logits  fp32 [B][k+1][vocab] (device): the target's scores for
 *                  the token at each draft position and at the one after the
 *                  last; scores must be finite (a NaN never wins)
 *   draft_tokens   int32 [B][k] (device)
 *   accepted       int32 [B] (device, written): number of leading drafts
 *                  equal to the target's choices (0..k)
 *   next_token     int32 [B] (device, written): the target's choice at
 *                  position `accepted` (the correction, or the bonus token
 *                  when all k are kept)
 *   workspace      >= lynx_spec_accept_workspace_bytes(B, k, vocab)
 */
int lynx_spec_accept_greedy(int32_t B, int32_t k, int32_t vocab, const float *target_logits,
                            const int32_t *draft_tokens, int32_t *accepted,
                            int32_t *next_token, void *workspace, size_t workspace_bytes,
                            void *stream);

/*
 * lynx_spec_accept_sample -- acceptance of sampled drafts (Sec. 4.3's
 * longest-prefix rule in its speculative-sampling form).  Draft i, token x
 * drawn from the draft model's distribution q_i, is kept when
 * u[i] * q_i(x) <= p_i(x) (fp32 product), i.e. with probability
 * min(1, p_i(x) / q_i(x)); a token outside [0, vocab) is not kept.  At the
 * first draft not kept, n, the next token is drawn from the weights
 * max(p_n - q_n, 0); when all k are kept, the bonus token from p_k.  The
 * emitted tokens are then distributed as the target model's.
 * The draw is exact, so its outcome depends on the inputs alone: weights
 * w_v = floor(r_v * 2^40) with r_v clamped to [0, 1] (NaN counts 0),
 * S = sum w_v, U = floor(u[k] * 2^32) clamped to [0, 2^32 - 1] (NaN 0),
 * t = floor(S * U / 2^32); the token is the smallest v whose inclusive
 * prefix sum of w exceeds t.  If the residual weights are all 0 the draw
 * uses p_n; if those are all 0 too, next_token is -1.
 *
 *   B, k, vocab   sequences (<= 65535), drafts per sequence (1..64),
 *                 vocabulary size (1..2^23)
 *   target_probs  fp32 [B][k+1][vocab] (device): the target's probabilities
 *                 at each draft position and the one after the last
 *   draft_probs   fp32 [B][k][vocab] (device): the draft model's
 *   draft_tokens  int32 [B][k] (device)
 *   uniforms      fp32 [B][k+1] (device): uniform numbers in [0, 1) drawn by
 *                 the caller, one per draft test and one for the draw
 *   accepted      int32 [B] (device, written): drafts kept (0..k)
 *   next_token    int32 [B] (device, written): the drawn token, or -1
 *   workspace     >= lynx_spec_accept_workspace_bytes(B, k, vocab)
 *                 (LYNX_EWORKSPACE otherwise)
 * All pointers 16-byte aligned.  Launches two kernels.
 */
int lynx_spec_accept_sample(int32_t B, int32_t k, int32_t vocab, const float *target_probs,
                            const float *draft_probs, const int32_t *draft_tokens,
                            const float *uniforms, int32_t *accepted, int32_t *next_token,
                            void *workspace, size_t workspace_bytes, void *stream);

/*
 * Serializer / deserializer (Sec. 4.2 Prioritized Transmission; Sec. 5
 * Compression Kernel).  A KV object is tokens [t0, t0 + n) of one sequence
 * (one layer), all kv heads, with t0 a multiple of 128 so that its K groups
 * are the sequence's.  Its two contiguous transmission buffers, each section
 * directly after the previous one:
 *   anchor buffer:   K anchor rows [Hkv][n][64] bytes, V anchor rows
 *                    [Hkv][n][64], then the shared scalars: K scales and K
 *                    zeros fp32 [Hkv][ceil(n/128)][128], V scales and V zeros
 *                    fp32 [Hkv][n]  (Hkv * (136 n + 1024 ceil(n/128)) bytes)
 *   residual buffer: K residual rows [Hkv][n][64], V residual rows
 *                    [Hkv][n][64]  (128 Hkv n bytes)
 * Rows and scalars are those lynx_kv_encode gives the same tokens of the
 * sequence, so serialize + deserialize_anchor reproduces its planes and
 * metadata, and deserialize_residual its merged codes.
 */

/* Byte sizes of an object's anchor and residual buffers (host call; no
 * launch).  Returns LYNX_EINVAL for num_kv_heads < 1, n_tokens < 1 or a NULL
 * output pointer. */
int lynx_serialized_bytes(int32_t num_kv_heads, int32_t n_tokens, size_t *anchor_bytes,
                          size_t *residual_bytes);

/*
 * lynx_kv_serialize -- the prefill side: quantize one object straight into
 * its transmission buffers (the anchor stream followed by its scalars; the
 * residual stream in the other buffer).
 *   k_bf16, v_bf16  BF16 [n][Hkv][128] (device, read): the object's tokens,
 *                   i.e. a sequence's K, V advanced by t0 token rows
 *   anchor_buf, residual_buf  lynx_serialized_bytes() bytes each (device,
 *                   written, 16-byte aligned, not overlapping)
 * Launches one kernel.
 */
int lynx_kv_serialize(int32_t num_kv_heads, int32_t n_tokens, const void *k_bf16,
                      const void *v_bf16, void *anchor_buf, void *residual_buf, void *stream);

/*
 * lynx_kv_deserialize_anchor -- the decode side's Anchor phase: scatter a
 * received anchor buffer into the anchor planes of the pool (rows of tokens
 * t0 .. t0 + n - 1 of sequence b, through block_table row b) and into
 * metadata row b.
 *   L, block_table, k_anc, v_anc, meta  as for lynx_kv_encode
 *   t0           first token; a multiple of 128; t0 + n_tokens must not
 *                exceed min(max_tokens, max_blocks_per_seq * bt)
 *   anchor_buf   the object's anchor buffer (device, read, 16-byte aligned)
 * Rows whose block id is outside [0, num_blocks) are skipped.  Launches one
 * kernel.
 */
int lynx_kv_deserialize_anchor(const lynx_layout *L, int32_t b, int32_t t0, int32_t n_tokens,
                               const int32_t *block_table, const void *anchor_buf,
                               uint8_t *k_anc, uint8_t *v_anc, const lynx_meta *meta,
                               void *stream);

/*
 * lynx_kv_deserialize_residual -- the decode side's Residual phase for one
 * object: its received residual buffer and its anchor rows already in the
 * pool (a prior lynx_kv_deserialize_anchor on the same stream, or an encode)
 * merge into the code planes of the pool (128-byte rows, same block ids):
 * the lynx_kv_merge rule per byte.
 *   residual_buf  the object's residual buffer (device, read, 16-byte aligned)
 *   k_anc, v_anc  anchor planes (device, read); k_codes, v_codes code planes
 *                 (device, written)
 * Same t0 / n_tokens rules and skipped rows as the anchor phase.  Launches
 * one kernel.
 */
int lynx_kv_deserialize_residual(const lynx_layout *L, int32_t b, int32_t t0, int32_t n_tokens,
                                 const int32_t *block_table, const void *residual_buf,
                                 const uint8_t *k_anc, const uint8_t *v_anc, uint8_t *k_codes,
                                 uint8_t *v_codes, void *stream);

/*
 * Split widths other than 4 + 4 (the paper leaves them to future work,
 * Sec. 8): the same 8-bit codes as lynx_kv_encode, split into an anchor of
 * A = anchor_bits bits (code >> (8 - A)) and a residual of R = 8 - A bits
 * (code & (2^R - 1)), A in {2, 4, 6}.  A plane row (one token of one kv
 * head) holds the 128 fields as a little-endian bit string: element e at
 * bits e W .. e W + W - 1 (W = A or R), so anchor rows are 16 A bytes and
 * residual rows 16 R bytes, at row index ((block * Hkv + h) * bt + t % bt)
 * as in the 4 + 4 planes.  A = 4 gives exactly the 4 + 4 planes.  Merged
 * codes are those of lynx_kv_merge, so lynx_attn_verify reads them as is.
 */

/*
 * lynx_kv_encode_split -- encode one sequence (one layer) with an A + R
 * split.  Arguments as lynx_kv_encode; the planes hold rows of 16 A (anchor)
 * and 16 R (residual) bytes.  Launches one kernel.
 */
int lynx_kv_encode_split(const lynx_layout *L, int32_t anchor_bits, int32_t b, int32_t T,
                         const int32_t *block_table, const void *k_bf16, const void *v_bf16,
                         uint8_t *k_anc, uint8_t *v_anc, uint8_t *k_res, uint8_t *v_res,
                         const lynx_meta *meta, void *stream);

/*
 * lynx_kv_merge_split -- n_rows rows of A-bit anchors (16 A bytes each) and
 * R-bit residuals (16 R bytes) into n_rows rows of 128 code bytes, row for
 * row (device, 16-byte aligned; codes must not overlap an input).  Launches
 * one kernel.
 */
int lynx_kv_merge_split(int32_t anchor_bits, size_t n_rows, const uint8_t *anc, const uint8_t *res,
                        uint8_t *codes, void *stream);

/*
 * lynx_kv_dequant_anchor_split -- the anchor phase's BF16 pages for an
 * A + R split (Sec. 4.2 dequantizes anchors into BF16 pages): sequence b's
 * K and V [T][Hkv][128] (device, written) from the anchor planes alone, the
 * anchor a standing for code 2^R a + (2^R - 1) / 2, the middle of the codes
 * it covers: x = fmaf(code, scale, zero) in fp32, rounded to BF16 to
 * nearest even.  Launches one kernel.
 */
int lynx_kv_dequant_anchor_split(const lynx_layout *L, int32_t anchor_bits, int32_t b, int32_t T,
                                 const int32_t *block_table, const uint8_t *k_anc,
                                 const uint8_t *v_anc, const lynx_meta *meta, void *k_out_bf16,
                                 void *v_out_bf16, void *stream);

/*
 * lynx_attn_anchor_decode_split -- decode attention over the anchors of a
 * split width (Sec. 4.2 Anchor phase, with the other widths of Sec. 8), read
 * straight from the A-bit anchor planes: for every sequence b and query head
 * hq, O = softmax(q K^T / sqrt(128)) V (Sec. 2) with K, V reconstructed as
 * zero + (2^R a + (2^R - 1) / 2) scale, R = 8 - anchor_bits (the anchor
 * alone at the middle of the codes it covers, as lynx_kv_dequant_anchor_split).
 *
 *   anchor_bits  A: 2, 4 or 6
 *   k_anc, v_anc anchor planes of rows of 16 A bytes (device), as written by
 *                lynx_kv_encode_split; meta: metadata of the batch
 *   other arguments as lynx_attn_anchor_decode; workspace >=
 *   lynx_attn_workspace_bytes(L, B, Hq, 1, max_seq_len), its arrival counters
 *   zero on entry as for lynx_attn_anchor_decode (every call leaves them zero).
 * Errors: LYNX_EINVAL (anchor_bits not 2, 4 or 6, or an argument
 * lynx_attn_anchor_decode rejects), LYNX_EWORKSPACE, LYNX_EHIP.  A sequence
 * with no tokens yields zeros and lse = -inf.
 */
int lynx_attn_anchor_decode_split(int32_t anchor_bits, const lynx_layout *L, int32_t B, int32_t Hq,
                                  int32_t max_seq_len, const int32_t *seq_lens,
                                  const int32_t *block_table, const uint8_t *k_anc,
                                  const uint8_t *v_anc, const lynx_meta *meta, const void *q_bf16,
                                  void *out_bf16, float *lse, void *workspace,
                                  size_t workspace_bytes, void *stream);

/*
 * The hierarchical non-linear codec of Alg. 1 (Sec. 4.1), the paper's own
 * quantizer, as an alternative to the uniform 8-bit one.  Per channel of a
 * kv head (K and V alike), over pages of 256 tokens and chunks of 32:
 * page normalization to [0, 1] (gmin, gscale), chunk centring and scaling
 * (mu, sigma), the alpha-law transform to a magnitude code I of M levels
 * (I = Round(M ln(1 + alpha |x|) / ln(1 + alpha))) and a sign, and the split
 * into 4-bit two's complement nibbles packed like the uniform codec's (same
 * plane layout).  The anchor carries the sign with the sign-aware map
 * (Q_anc = V, or -V - 1 for a negative value, so a negative zero keeps its
 * sign).  alpha is not fixed by the paper.  Variants (the variant argument):
 *   LYNX_HQ_BIASED   Alg. 1's biased split, M = 127: anchor
 *                    V = min((I + 7) >> 4, 7), correction
 *                    Q_res = clamp(16 V - I, -8, 7).  Codes above 120 come
 *                    back as 120: Alg. 1's anchor reaches 8 there,
 *                    which four signed bits cannot hold.
 *   LYNX_HQ_CENTRED  the split that keeps every code, M = 127: anchor
 *                    V = I >> 4 (sign and top three bits), correction
 *                    Q_res = I - 16 V - 8, centred on the bucket.  The anchor
 *                    alone stands for the bucket's centre, code 16 V + 7.5;
 *                    the merged byte is a complete 8-bit code (the paper's
 *                    single-precision 8-bit configuration, Sec. 6.1).
 *   LYNX_HQ_INT4     the single-precision 4-bit configuration (Sec. 6.1):
 *                    M = 7, the anchor plane holds Q = I or -I - 1, no
 *                    residual.
 */
enum { LYNX_HQ_BIASED = 0, LYNX_HQ_CENTRED = 1, LYNX_HQ_INT4 = 2 };

typedef struct lynx_hmeta {
    float *k_gmin, *k_gscale; /* [B][Hkv][ceil(max_tokens/256)][128] fp32 */
    float *k_mu, *k_sigma;    /* [B][Hkv][ceil(max_tokens/32)][128] fp32  */
    float *v_gmin, *v_gscale;
    float *v_mu, *v_sigma;
} lynx_hmeta;

/*
 * lynx_hkv_encode -- hierarchical encode of one sequence (one layer).
 *   Arguments as lynx_kv_encode, plus alpha (0 < alpha <= 1e30), the
 *   variant (LYNX_HQ_*), and the hierarchical metadata (all 16-byte
 *   aligned): row b written for pages and chunks holding tokens < T.
 *   LYNX_HQ_INT4 writes the anchor planes only: k_res and v_res may be NULL.
 *   Launches one kernel.
 */
int lynx_hkv_encode(const lynx_layout *L, int32_t b, int32_t T, const int32_t *block_table,
                    const void *k_bf16, const void *v_bf16, float alpha, int32_t variant,
                    uint8_t *k_anc, uint8_t *v_anc, uint8_t *k_res, uint8_t *v_res,
                    const lynx_hmeta *meta, void *stream);

/*
 * lynx_hkv_dequant -- the deserializer's dequantization into BF16 pages
 * (Sec. 4.2): sequence b's K and V reconstructed as BF16 [T][Hkv][128]
 * (k_out_bf16, v_out_bf16, device, written).
 *   full 0: from the anchor nibble planes alone (code 16 V for
 *           LYNX_HQ_BIASED, 16 V + 7.5 for LYNX_HQ_CENTRED, V for
 *           LYNX_HQ_INT4);
 *   full 1: from the merged code planes of lynx_kv_merge (high nibble
 *           anchor, low nibble correction; code 16 V - Q_res, or
 *           16 V + 8 + Q_res); not for LYNX_HQ_INT4 (LYNX_EINVAL).
 *   x = ((+-level(code) * sigma) + mu) * gscale + gmin in fp32, rounded to
 *   BF16 to nearest even, level(i) = expm1(i / M * log1p(alpha)) / alpha.
 * Launches one kernel.
 */
int lynx_hkv_dequant(const lynx_layout *L, int32_t b, int32_t T, const int32_t *block_table,
                     int32_t full, const uint8_t *k_plane, const uint8_t *v_plane, float alpha,
                     int32_t variant, const lynx_hmeta *meta, void *k_out_bf16, void *v_out_bf16,
                     void *stream);

/* Static, human-readable text for a lynx_status value. */
const char *lynx_strerror(int status);

#ifdef __cplusplus
}
#endif

#endif /* LYNX_H */
