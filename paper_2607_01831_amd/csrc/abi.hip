// C ABI of liblynx.so (declared in include/lynx.h): argument validation,
// workspace sizing and kernel launch.  Validation is synchronous and happens
// before anything is launched.
#include "../../include/lynx.h"
#include "lynx_internal.h"

#include <mutex>

namespace {

using lynx::Geometry;
using lynx::MetaPtrs;

bool aligned16(const void *p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

// Layout checks shared by every call; fills the kernel-side geometry.
int check_layout(const lynx_layout *L, Geometry *g) {
    if (!L) return LYNX_EINVAL;
    if (L->head_dim != lynx::kHeadDim || L->k_group_tokens != lynx::kKGroup) return LYNX_ENOTSUP;
    if (L->num_kv_heads < 1 || L->block_tokens < 1 || L->max_blocks_per_seq < 1 ||
        L->num_blocks < 1 || L->max_tokens < 1)
        return LYNX_EINVAL;
    g->Hkv = L->num_kv_heads;
    g->bt = L->block_tokens;
    g->max_blocks = L->max_blocks_per_seq;
    g->num_blocks = L->num_blocks;
    g->max_tokens = L->max_tokens;
    g->n_groups = (L->max_tokens + lynx::kKGroup - 1) / lynx::kKGroup;
    g->n_pages = (L->max_tokens + 255) / 256;
    g->n_chunks = (L->max_tokens + 31) / 32;
    return LYNX_OK;
}

int check_meta(const lynx_meta *meta, MetaPtrs *mp) {
    if (!meta || !meta->k_scale || !meta->k_zero || !meta->v_scale || !meta->v_zero)
        return LYNX_EINVAL;
    if (!aligned16(meta->k_scale) || !aligned16(meta->k_zero) || !aligned16(meta->v_scale) ||
        !aligned16(meta->v_zero))
        return LYNX_EINVAL;
    *mp = MetaPtrs{meta->k_scale, meta->k_zero, meta->v_scale, meta->v_zero};
    return LYNX_OK;
}

// Tokens a sequence may hold under this layout.
long long layout_capacity(const Geometry &g) {
    const long long paged = (long long)g.max_blocks * g.bt;
    return paged < g.max_tokens ? paged : g.max_tokens;
}

int check_attention_common(const lynx_layout *L, int32_t B, int32_t Hq, int32_t max_seq_len,
                           const int32_t *seq_lens, const int32_t *block_table,
                           const uint8_t *k_plane, const uint8_t *v_plane, const lynx_meta *meta,
                           const void *q, void *out, Geometry *g, MetaPtrs *mp) {
    int rc = check_layout(L, g);
    if (rc != LYNX_OK) return rc;
    if ((rc = check_meta(meta, mp)) != LYNX_OK) return rc;
    if (B < 0 || Hq < 1 || Hq % g->Hkv != 0 || max_seq_len < 0) return LYNX_EINVAL;
    if (max_seq_len > layout_capacity(*g)) return LYNX_EINVAL;
    if (B == 0) return LYNX_OK;
    const void *ptrs[] = {seq_lens, block_table, k_plane, v_plane, q, out};
    for (const void *p : ptrs)
        if (!p || !aligned16(p)) return LYNX_EINVAL;
    return LYNX_OK;
}

}  // namespace

extern "C" {

const char *lynx_strerror(int status) {
    switch (status) {
    case LYNX_OK: return "success";
    case LYNX_EINVAL: return "invalid argument (NULL or misaligned pointer, bad size or count)";
    case LYNX_ENOTSUP: return "unsupported geometry (head_dim and k_group_tokens must be 128)";
    case LYNX_EWORKSPACE: return "workspace missing or smaller than lynx_attn_workspace_bytes()";
    case LYNX_EHIP: return "HIP runtime reported a launch error";
    default: return "unknown lynx status";
    }
}

int lynx_kv_encode(const lynx_layout *L, int32_t b, int32_t T, const int32_t *block_table,
                   const void *k_bf16, const void *v_bf16, uint8_t *k_anc, uint8_t *v_anc,
                   uint8_t *k_res, uint8_t *v_res, const lynx_meta *meta, void *stream) {
    Geometry g;
    MetaPtrs mp;
    int rc = check_layout(L, &g);
    if (rc != LYNX_OK) return rc;
    if ((rc = check_meta(meta, &mp)) != LYNX_OK) return rc;
    if (b < 0 || T < 0 || T > layout_capacity(g)) return LYNX_EINVAL;
    if (T == 0) return LYNX_OK;
    const void *ptrs[] = {block_table, k_bf16, v_bf16, k_anc, v_anc, k_res, v_res};
    for (const void *p : ptrs)
        if (!p || !aligned16(p)) return LYNX_EINVAL;
    hipError_t e = lynx::launch_encode(g, b, T, block_table,
                                       static_cast<const uint16_t *>(k_bf16),
                                       static_cast<const uint16_t *>(v_bf16), k_anc, v_anc, k_res,
                                       v_res, mp, static_cast<hipStream_t>(stream));
    return e == hipSuccess ? LYNX_OK : LYNX_EHIP;
}

int lynx_kv_merge(const uint8_t *anc, const uint8_t *res, uint8_t *codes, size_t n_packed_bytes,
                  void *stream) {
    if (n_packed_bytes == 0) return LYNX_OK;
    if (!anc || !res || !codes || !aligned16(anc) || !aligned16(res) || !aligned16(codes))
        return LYNX_EINVAL;
    // the output must not overlap either input
    const uintptr_t c0 = reinterpret_cast<uintptr_t>(codes), c1 = c0 + 2 * n_packed_bytes;
    for (const uint8_t *in : {anc, res}) {
        const uintptr_t i0 = reinterpret_cast<uintptr_t>(in), i1 = i0 + n_packed_bytes;
        if (i0 < c1 && c0 < i1) return LYNX_EINVAL;
    }
    hipError_t e = lynx::launch_merge(anc, res, codes, n_packed_bytes,
                                      static_cast<hipStream_t>(stream));
    return e == hipSuccess ? LYNX_OK : LYNX_EHIP;
}

int lynx_kv_encode_split(const lynx_layout *L, int32_t anchor_bits, int32_t b, int32_t T,
                         const int32_t *block_table, const void *k_bf16, const void *v_bf16,
                         uint8_t *k_anc, uint8_t *v_anc, uint8_t *k_res, uint8_t *v_res,
                         const lynx_meta *meta, void *stream) {
    if (anchor_bits != 2 && anchor_bits != 4 && anchor_bits != 6) return LYNX_EINVAL;
    Geometry g;
    MetaPtrs mp;
    int rc = check_layout(L, &g);
    if (rc != LYNX_OK) return rc;
    if ((rc = check_meta(meta, &mp)) != LYNX_OK) return rc;
    if (b < 0 || T < 0 || T > layout_capacity(g)) return LYNX_EINVAL;
    if (T == 0) return LYNX_OK;
    const void *ptrs[] = {block_table, k_bf16, v_bf16, k_anc, v_anc, k_res, v_res};
    for (const void *p : ptrs)
        if (!p || !aligned16(p)) return LYNX_EINVAL;
    hipError_t e = lynx::launch_encode(g, b, T, block_table, static_cast<const uint16_t *>(k_bf16),
                                       static_cast<const uint16_t *>(v_bf16), k_anc, v_anc, k_res,
                                       v_res, mp, static_cast<hipStream_t>(stream), anchor_bits);
    return e == hipSuccess ? LYNX_OK : LYNX_EHIP;
}

int lynx_kv_merge_split(int32_t anchor_bits, size_t n_rows, const uint8_t *anc, const uint8_t *res,
                        uint8_t *codes, void *stream) {
    if (anchor_bits != 2 && anchor_bits != 4 && anchor_bits != 6) return LYNX_EINVAL;
    if (n_rows == 0) return LYNX_OK;
    if (n_rows > ((size_t)1 << 40)) return LYNX_EINVAL;
    if (!anc || !res || !codes || !aligned16(anc) || !aligned16(res) || !aligned16(codes))
        return LYNX_EINVAL;
    const size_t na = n_rows * 16 * (size_t)anchor_bits, nr = n_rows * 16 * (size_t)(8 - anchor_bits);
    const uintptr_t c0 = reinterpret_cast<uintptr_t>(codes), c1 = c0 + n_rows * lynx::kCodeRow;
    const uintptr_t a0 = reinterpret_cast<uintptr_t>(anc), r0 = reinterpret_cast<uintptr_t>(res);
    if ((a0 < c1 && c0 < a0 + na) || (r0 < c1 && c0 < r0 + nr)) return LYNX_EINVAL;
    hipError_t e = lynx::launch_merge_split(anchor_bits, anc, res, codes, n_rows,
                                            static_cast<hipStream_t>(stream));
    return e == hipSuccess ? LYNX_OK : LYNX_EHIP;
}

int lynx_kv_dequant_anchor_split(const lynx_layout *L, int32_t anchor_bits, int32_t b, int32_t T,
                                 const int32_t *block_table, const uint8_t *k_anc,
                                 const uint8_t *v_anc, const lynx_meta *meta, void *k_out_bf16,
                                 void *v_out_bf16, void *stream) {
    if (anchor_bits != 2 && anchor_bits != 4 && anchor_bits != 6) return LYNX_EINVAL;
    Geometry g;
    MetaPtrs mp;
    int rc = check_layout(L, &g);
    if (rc != LYNX_OK) return rc;
    if ((rc = check_meta(meta, &mp)) != LYNX_OK) return rc;
    if (b < 0 || T < 0 || T > layout_capacity(g)) return LYNX_EINVAL;
    if (T == 0) return LYNX_OK;
    const void *ptrs[] = {block_table, k_anc, v_anc, k_out_bf16, v_out_bf16};
    for (const void *p : ptrs)
        if (!p || !aligned16(p)) return LYNX_EINVAL;
    hipError_t e = lynx::launch_dequant_anchor_split(anchor_bits, g, b, T, block_table, k_anc, v_anc, mp,
                                                     static_cast<uint16_t *>(k_out_bf16),
                                                     static_cast<uint16_t *>(v_out_bf16),
                                                     static_cast<hipStream_t>(stream));
    return e == hipSuccess ? LYNX_OK : LYNX_EHIP;
}

size_t lynx_attn_workspace_bytes(const lynx_layout *L, int32_t B, int32_t Hq,
                                 int32_t num_queries, int32_t max_seq_len) {
    Geometry g;
    if (check_layout(L, &g) != LYNX_OK) return 0;
    if (B < 0 || Hq < 1 || Hq % g.Hkv != 0 || num_queries < 1 || num_queries > 64 ||
        max_seq_len < 0)
        return 0;
    // sized for the larger plan, the one with a draft-tail split
    const lynx::AttnPlan p = lynx::plan_attention(g, B, Hq, num_queries, max_seq_len, true);
    return p.workspace_bytes();
}

int lynx_attn_anchor_decode(const lynx_layout *L, int32_t B, int32_t Hq, int32_t max_seq_len,
                            const int32_t *seq_lens, const int32_t *block_table,
                            const uint8_t *k_anc, const uint8_t *v_anc, const lynx_meta *meta,
                            const void *q_bf16, void *out_bf16, float *lse, void *workspace,
                            size_t workspace_bytes, void *stream) {
    Geometry g;
    MetaPtrs mp;
    int rc = check_attention_common(L, B, Hq, max_seq_len, seq_lens, block_table, k_anc, v_anc,
                                    meta, q_bf16, out_bf16, &g, &mp);
    if (rc != LYNX_OK) return rc;
    if (B == 0) return LYNX_OK;
    if (lse && !aligned16(lse)) return LYNX_EINVAL;
    const lynx::AttnPlan p = lynx::plan_attention(g, B, Hq, 1, max_seq_len, false);
    if (!workspace || !aligned16(workspace) || workspace_bytes < p.workspace_bytes())
        return LYNX_EWORKSPACE;
    hipError_t e = lynx::launch_attention(
        lynx::KvMode::kAnchor, g, p, B, Hq, 1, max_seq_len, seq_lens, block_table, k_anc, v_anc,
        mp, static_cast<const uint16_t *>(q_bf16), nullptr, nullptr, 0,
        static_cast<uint16_t *>(out_bf16), lse, workspace, static_cast<hipStream_t>(stream));
    return e == hipSuccess ? LYNX_OK : LYNX_EHIP;
}

int lynx_attn_anchor_decode_split(int32_t anchor_bits, const lynx_layout *L, int32_t B, int32_t Hq,
                                  int32_t max_seq_len, const int32_t *seq_lens,
                                  const int32_t *block_table, const uint8_t *k_anc,
                                  const uint8_t *v_anc, const lynx_meta *meta, const void *q_bf16,
                                  void *out_bf16, float *lse, void *workspace,
                                  size_t workspace_bytes, void *stream) {
    if (anchor_bits != 2 && anchor_bits != 4 && anchor_bits != 6) return LYNX_EINVAL;
    Geometry g;
    MetaPtrs mp;
    int rc = check_attention_common(L, B, Hq, max_seq_len, seq_lens, block_table, k_anc, v_anc,
                                    meta, q_bf16, out_bf16, &g, &mp);
    if (rc != LYNX_OK) return rc;
    if (B == 0) return LYNX_OK;
    if (lse && !aligned16(lse)) return LYNX_EINVAL;
    const lynx::AttnPlan p = lynx::plan_attention(g, B, Hq, 1, max_seq_len, false);
    if (!workspace || !aligned16(workspace) || workspace_bytes < p.workspace_bytes())
        return LYNX_EWORKSPACE;
    hipError_t e = lynx::launch_attention(
        lynx::KvMode::kAnchorSplit, g, p, B, Hq, 1, max_seq_len, seq_lens, block_table, k_anc,
        v_anc, mp, static_cast<const uint16_t *>(q_bf16), nullptr, nullptr, 0,
        static_cast<uint16_t *>(out_bf16), lse, workspace, static_cast<hipStream_t>(stream),
        anchor_bits);
    return e == hipSuccess ? LYNX_OK : LYNX_EHIP;
}

}  // extern "C"

// ---- scratch of lynx_attn_anchor_decode_noalloc ----
// The split partials and arrival counters of a decode call live in this
// file-scope device array instead of a caller workspace.  In host code its
// name is only a stand-in: the device address comes from hipGetSymbolAddress,
// once per device (each GPU holds its own copy).  It is zero when the library
// is loaded, and every call leaves its counters zero again.
namespace {
constexpr size_t kScratchBytes = 16u << 20;  // the value of LYNX_NOALLOC_SCRATCH_BYTES
static __device__ __align__(256) uint8_t scratch[kScratchBytes];
static_assert(kScratchBytes == LYNX_NOALLOC_SCRATCH_BYTES, "header and library disagree");
constexpr int kMaxDevices = 64;
std::once_flag g_scratch_once[kMaxDevices];
void *g_scratch_ptr[kMaxDevices];
hipError_t g_scratch_err[kMaxDevices];

// Device address of this device's scratch array (nullptr on failure).
void *scratch_on_current_device() {
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return nullptr;
    std::call_once(g_scratch_once[dev], [dev]() {
        void *ptr = nullptr;
        g_scratch_err[dev] = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
        g_scratch_ptr[dev] = g_scratch_err[dev] == hipSuccess ? ptr : nullptr;
    });
    return g_scratch_ptr[dev];
}
}  // namespace

extern "C" {

int lynx_attn_anchor_decode_noalloc(const lynx_layout *L, int32_t B, int32_t Hq,
                                    int32_t max_seq_len, const int32_t *seq_lens,
                                    const int32_t *block_table, const uint8_t *k_anc,
                                    const uint8_t *v_anc, const lynx_meta *meta,
                                    const void *q_bf16, void *out_bf16, float *lse, void *stream) {
    Geometry g;
    MetaPtrs mp;
    int rc = check_attention_common(L, B, Hq, max_seq_len, seq_lens, block_table, k_anc, v_anc,
                                    meta, q_bf16, out_bf16, &g, &mp);
    if (rc != LYNX_OK) return rc;
    if (B == 0) return LYNX_OK;
    if (lse && !aligned16(lse)) return LYNX_EINVAL;
    const lynx::AttnPlan p = lynx::plan_attention(g, B, Hq, 1, max_seq_len, false);
    if (p.workspace_bytes() > kScratchBytes) return LYNX_EWORKSPACE;
    void *ws = scratch_on_current_device();
    if (!ws) return LYNX_EHIP;
    hipError_t e = lynx::launch_attention(
        lynx::KvMode::kAnchor, g, p, B, Hq, 1, max_seq_len, seq_lens, block_table, k_anc, v_anc,
        mp, static_cast<const uint16_t *>(q_bf16), nullptr, nullptr, 0,
        static_cast<uint16_t *>(out_bf16), lse, ws, static_cast<hipStream_t>(stream));
    return e == hipSuccess ? LYNX_OK : LYNX_EHIP;
}

int lynx_attn_anchor_decode_tail(const lynx_layout *L, int32_t B, int32_t Hq,
                                 int32_t max_seq_len, const int32_t *seq_lens,
                                 const int32_t *block_table, const uint8_t *k_anc,
                                 const uint8_t *v_anc, const lynx_meta *meta, const void *q_bf16,
                                 int32_t n_tail, const void *k_tail, const void *v_tail,
                                 void *out_bf16, float *lse, void *workspace,
                                 size_t workspace_bytes, void *stream) {
    Geometry g;
    MetaPtrs mp;
    int rc = check_attention_common(L, B, Hq, max_seq_len, seq_lens, block_table, k_anc, v_anc,
                                    meta, q_bf16, out_bf16, &g, &mp);
    if (rc != LYNX_OK) return rc;
    if (n_tail < 0 || n_tail > 64) return LYNX_EINVAL;
    if (n_tail > 0 && (!k_tail || !v_tail || !aligned16(k_tail) || !aligned16(v_tail)))
        return LYNX_EINVAL;
    if (B == 0) return LYNX_OK;
    if (lse && !aligned16(lse)) return LYNX_EINVAL;
    const lynx::AttnPlan p = lynx::plan_attention(g, B, Hq, 1, max_seq_len, false);
    if (!workspace || !aligned16(workspace) || workspace_bytes < p.workspace_bytes())
        return LYNX_EWORKSPACE;
    hipError_t e = lynx::launch_attention(
        lynx::KvMode::kAnchor, g, p, B, Hq, 1, max_seq_len, seq_lens, block_table, k_anc, v_anc,
        mp, static_cast<const uint16_t *>(q_bf16),
        n_tail > 0 ? static_cast<const uint16_t *>(k_tail) : nullptr,
        n_tail > 0 ? static_cast<const uint16_t *>(v_tail) : nullptr, n_tail,
        static_cast<uint16_t *>(out_bf16), lse, workspace, static_cast<hipStream_t>(stream));
    return e == hipSuccess ? LYNX_OK : LYNX_EHIP;
}

int lynx_attn_verify(const lynx_layout *L, int32_t B, int32_t Hq, int32_t k,
                     int32_t max_seq_len, const int32_t *seq_lens, const int32_t *block_table,
                     const uint8_t *k_codes, const uint8_t *v_codes, const lynx_meta *meta,
                     const void *q_bf16, const void *k_new, const void *v_new, void *out_bf16,
                     void *workspace, size_t workspace_bytes, void *stream) {
    Geometry g;
    MetaPtrs mp;
    int rc = check_attention_common(L, B, Hq, max_seq_len, seq_lens, block_table, k_codes,
                                    v_codes, meta, q_bf16, out_bf16, &g, &mp);
    if (rc != LYNX_OK) return rc;
    if (k < 1 || k > 64) return LYNX_EINVAL;
    if ((k_new == nullptr) != (v_new == nullptr)) return LYNX_EINVAL;
    if (k_new && (!aligned16(k_new) || !aligned16(v_new))) return LYNX_EINVAL;
    if (B == 0) return LYNX_OK;
    const bool tail = k_new != nullptr;
    const lynx::AttnPlan p = lynx::plan_attention(g, B, Hq, k, max_seq_len, tail);
    if (!workspace || !aligned16(workspace) || workspace_bytes < p.workspace_bytes())
        return LYNX_EWORKSPACE;
    hipError_t e = lynx::launch_attention(
        lynx::KvMode::kCodes, g, p, B, Hq, k, max_seq_len, seq_lens, block_table, k_codes, v_codes,
        mp, static_cast<const uint16_t *>(q_bf16), static_cast<const uint16_t *>(k_new),
        static_cast<const uint16_t *>(v_new), k, static_cast<uint16_t *>(out_bf16), nullptr,
        workspace, static_cast<hipStream_t>(stream));
    return e == hipSuccess ? LYNX_OK : LYNX_EHIP;
}

size_t lynx_spec_accept_workspace_bytes(int32_t B, int32_t k, int32_t vocab) {
    if (B < 0 || B > 65535 || k < 1 || k > 64 || vocab < 1) return 0;
    // greedy: a (score, index) pair per chunk; sampled: two uint64 sums
    return (size_t)B * (size_t)(k + 1) * (size_t)lynx::spec_accept_chunks(vocab) * 2 * sizeof(uint64_t);
}

int lynx_spec_accept_greedy(int32_t B, int32_t k, int32_t vocab, const float *target_logits,
                            const int32_t *draft_tokens, int32_t *accepted,
                            int32_t *next_token, void *workspace, size_t workspace_bytes,
                            void *stream) {
    if (B < 0 || B > 65535 || k < 1 || k > 64 || vocab < 1) return LYNX_EINVAL;
    if (B == 0) return LYNX_OK;
    const void *ptrs[] = {target_logits, draft_tokens, accepted, next_token};
    for (const void *p : ptrs)
        if (!p || !aligned16(p)) return LYNX_EINVAL;
    const size_t need = lynx_spec_accept_workspace_bytes(B, k, vocab);
    if (!workspace || !aligned16(workspace) || workspace_bytes < need) return LYNX_EWORKSPACE;
    hipError_t e = lynx::launch_spec_accept_greedy(B, k, vocab, target_logits, draft_tokens,
                                                   accepted, next_token, workspace,
                                                   static_cast<hipStream_t>(stream));
    return e == hipSuccess ? LYNX_OK : LYNX_EHIP;
}

int lynx_spec_accept_sample(int32_t B, int32_t k, int32_t vocab, const float *target_probs,
                            const float *draft_probs, const int32_t *draft_tokens,
                            const float *uniforms, int32_t *accepted, int32_t *next_token,
                            void *workspace, size_t workspace_bytes, void *stream) {
    if (B < 0 || B > 65535 || k < 1 || k > 64 || vocab < 1 || vocab > (1 << 23)) return LYNX_EINVAL;
    if (B == 0) return LYNX_OK;
    const void *ptrs[] = {target_probs, draft_probs, draft_tokens, uniforms, accepted, next_token};
    for (const void *p : ptrs)
        if (!p || !aligned16(p)) return LYNX_EINVAL;
    const size_t need = lynx_spec_accept_workspace_bytes(B, k, vocab);
    if (!workspace || !aligned16(workspace) || workspace_bytes < need) return LYNX_EWORKSPACE;
    hipError_t e = lynx::launch_spec_accept_sample(B, k, vocab, target_probs, draft_probs,
                                                   draft_tokens, uniforms, accepted, next_token,
                                                   workspace, static_cast<hipStream_t>(stream));
    return e == hipSuccess ? LYNX_OK : LYNX_EHIP;
}

}  // extern "C"

namespace {
// Checks shared by the two deserializer phases.
int check_object(const lynx_layout *L, int32_t b, int32_t t0, int32_t n, const int32_t *block_table,
                 Geometry *g) {
    int rc = check_layout(L, g);
    if (rc != LYNX_OK) return rc;
    if (b < 0 || t0 < 0 || n < 1 || t0 % lynx::kKGroup != 0) return LYNX_EINVAL;
    if ((long long)t0 + n > layout_capacity(*g)) return LYNX_EINVAL;
    if (!block_table || !aligned16(block_table)) return LYNX_EINVAL;
    return LYNX_OK;
}
}  // namespace

extern "C" {

int lynx_serialized_bytes(int32_t num_kv_heads, int32_t n_tokens, size_t *anchor_bytes,
                          size_t *residual_bytes) {
    if (num_kv_heads < 1 || n_tokens < 1 || !anchor_bytes || !residual_bytes) return LYNX_EINVAL;
    const size_t H = (size_t)num_kv_heads, n = (size_t)n_tokens;
    const size_t g = (n + lynx::kKGroup - 1) / lynx::kKGroup;
    *anchor_bytes = H * (2 * n * lynx::kNibbleRow + 2 * g * lynx::kHeadDim * 4 + 2 * n * 4);
    *residual_bytes = H * 2 * n * lynx::kNibbleRow;
    return LYNX_OK;
}

int lynx_kv_serialize(int32_t num_kv_heads, int32_t n_tokens, const void *k_bf16,
                      const void *v_bf16, void *anchor_buf, void *residual_buf, void *stream) {
    size_t na, nr;
    if (lynx_serialized_bytes(num_kv_heads, n_tokens, &na, &nr) != LYNX_OK) return LYNX_EINVAL;
    const void *ptrs[] = {k_bf16, v_bf16, anchor_buf, residual_buf};
    for (const void *p : ptrs)
        if (!p || !aligned16(p)) return LYNX_EINVAL;
    const uintptr_t a0 = reinterpret_cast<uintptr_t>(anchor_buf), a1 = a0 + na;
    const uintptr_t r0 = reinterpret_cast<uintptr_t>(residual_buf), r1 = r0 + nr;
    if (a0 < r1 && r0 < a1) return LYNX_EINVAL;
    hipError_t e = lynx::launch_serialize(num_kv_heads, n_tokens,
                                          static_cast<const uint16_t *>(k_bf16),
                                          static_cast<const uint16_t *>(v_bf16),
                                          static_cast<uint8_t *>(anchor_buf),
                                          static_cast<uint8_t *>(residual_buf),
                                          static_cast<hipStream_t>(stream));
    return e == hipSuccess ? LYNX_OK : LYNX_EHIP;
}

int lynx_kv_deserialize_anchor(const lynx_layout *L, int32_t b, int32_t t0, int32_t n_tokens,
                               const int32_t *block_table, const void *anchor_buf,
                               uint8_t *k_anc, uint8_t *v_anc, const lynx_meta *meta,
                               void *stream) {
    Geometry g;
    MetaPtrs mp;
    int rc = check_object(L, b, t0, n_tokens, block_table, &g);
    if (rc != LYNX_OK) return rc;
    if ((rc = check_meta(meta, &mp)) != LYNX_OK) return rc;
    const void *ptrs[] = {anchor_buf, k_anc, v_anc};
    for (const void *p : ptrs)
        if (!p || !aligned16(p)) return LYNX_EINVAL;
    hipError_t e = lynx::launch_deserialize_anchor(g, b, t0, n_tokens, block_table,
                                                   static_cast<const uint8_t *>(anchor_buf), k_anc,
                                                   v_anc, mp, static_cast<hipStream_t>(stream));
    return e == hipSuccess ? LYNX_OK : LYNX_EHIP;
}

int lynx_kv_deserialize_residual(const lynx_layout *L, int32_t b, int32_t t0, int32_t n_tokens,
                                 const int32_t *block_table, const void *residual_buf,
                                 const uint8_t *k_anc, const uint8_t *v_anc, uint8_t *k_codes,
                                 uint8_t *v_codes, void *stream) {
    Geometry g;
    int rc = check_object(L, b, t0, n_tokens, block_table, &g);
    if (rc != LYNX_OK) return rc;
    const void *ptrs[] = {residual_buf, k_anc, v_anc, k_codes, v_codes};
    for (const void *p : ptrs)
        if (!p || !aligned16(p)) return LYNX_EINVAL;
    hipError_t e = lynx::launch_deserialize_residual(
        g, b, t0, n_tokens, block_table, static_cast<const uint8_t *>(residual_buf), k_anc, v_anc,
        k_codes, v_codes, static_cast<hipStream_t>(stream));
    return e == hipSuccess ? LYNX_OK : LYNX_EHIP;
}

}  // extern "C"

namespace {
int check_hmeta(const lynx_hmeta *m, lynx::HMetaPtrs *hp) {
    if (!m) return LYNX_EINVAL;
    float *ptrs[] = {m->k_gmin, m->k_gscale, m->k_mu, m->k_sigma,
                     m->v_gmin, m->v_gscale, m->v_mu, m->v_sigma};
    for (float *p : ptrs)
        if (!p || !aligned16(p)) return LYNX_EINVAL;
    *hp = lynx::HMetaPtrs{m->k_gmin, m->k_gscale, m->k_mu, m->k_sigma,
                          m->v_gmin, m->v_gscale, m->v_mu, m->v_sigma};
    return LYNX_OK;
}
bool alpha_ok(float a) { return a > 0.0f && a <= 1e30f; }
bool variant_ok(int32_t v) { return v == LYNX_HQ_BIASED || v == LYNX_HQ_CENTRED || v == LYNX_HQ_INT4; }
static_assert(LYNX_HQ_BIASED == lynx::kHBiased && LYNX_HQ_CENTRED == lynx::kHCentred &&
                  LYNX_HQ_INT4 == lynx::kHInt4,
              "codec variant values");
}  // namespace

extern "C" {

int lynx_hkv_encode(const lynx_layout *L, int32_t b, int32_t T, const int32_t *block_table,
                    const void *k_bf16, const void *v_bf16, float alpha, int32_t variant,
                    uint8_t *k_anc, uint8_t *v_anc, uint8_t *k_res, uint8_t *v_res,
                    const lynx_hmeta *meta, void *stream) {
    Geometry g;
    lynx::HMetaPtrs hp;
    int rc = check_layout(L, &g);
    if (rc != LYNX_OK) return rc;
    if ((rc = check_hmeta(meta, &hp)) != LYNX_OK) return rc;
    if (!alpha_ok(alpha) || !variant_ok(variant) || b < 0 || T < 0 || T > layout_capacity(g))
        return LYNX_EINVAL;
    if (T == 0) return LYNX_OK;
    const void *ptrs[] = {block_table, k_bf16, v_bf16, k_anc, v_anc};
    for (const void *p : ptrs)
        if (!p || !aligned16(p)) return LYNX_EINVAL;
    if (variant != LYNX_HQ_INT4)
        for (const void *p : {(const void *)k_res, (const void *)v_res})
            if (!p || !aligned16(p)) return LYNX_EINVAL;
    lynx::HTables tab;
    lynx::make_htables(alpha, variant, &tab);
    hipError_t e = lynx::launch_hencode(g, b, T, block_table, static_cast<const uint16_t *>(k_bf16),
                                        static_cast<const uint16_t *>(v_bf16), k_anc, v_anc, k_res,
                                        v_res, hp, tab, variant, static_cast<hipStream_t>(stream));
    return e == hipSuccess ? LYNX_OK : LYNX_EHIP;
}

int lynx_hkv_dequant(const lynx_layout *L, int32_t b, int32_t T, const int32_t *block_table,
                     int32_t full, const uint8_t *k_plane, const uint8_t *v_plane, float alpha,
                     int32_t variant, const lynx_hmeta *meta, void *k_out_bf16, void *v_out_bf16,
                     void *stream) {
    Geometry g;
    lynx::HMetaPtrs hp;
    int rc = check_layout(L, &g);
    if (rc != LYNX_OK) return rc;
    if ((rc = check_hmeta(meta, &hp)) != LYNX_OK) return rc;
    if (!alpha_ok(alpha) || !variant_ok(variant) || (full != 0 && full != 1) ||
        (full == 1 && variant == LYNX_HQ_INT4) || b < 0 || T < 0 || T > layout_capacity(g))
        return LYNX_EINVAL;
    if (T == 0) return LYNX_OK;
    const void *ptrs[] = {block_table, k_plane, v_plane, k_out_bf16, v_out_bf16};
    for (const void *p : ptrs)
        if (!p || !aligned16(p)) return LYNX_EINVAL;
    lynx::HTables tab;
    lynx::make_htables(alpha, variant, &tab);
    hipError_t e = lynx::launch_hdequant(full == 1, g, b, T, block_table, k_plane, v_plane, hp, tab, variant,
                                         static_cast<uint16_t *>(k_out_bf16),
                                         static_cast<uint16_t *>(v_out_bf16),
                                         static_cast<hipStream_t>(stream));
    return e == hipSuccess ? LYNX_OK : LYNX_EHIP;
}

}  // extern "C"
