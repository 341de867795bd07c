/*
 * Lynx CPU oracle -- TEST INFRASTRUCTURE ONLY.
 *
 * A plain, slow, deliberately unoptimised CPU statement of what the Lynx hot
 * path computes.  Only the test suite, the smoke check and the benchmark's CPU
 * baseline leg load this library; the product path never does.  It shares no
 * code, header, table or helper with the HIP implementation.
 *
 * What it implements (paper: "Lynx: Progressive Speculative Quantization for
 * accelerating KV Transfer in Long-Context Inference"):
 *
 *   encode  -- grouped linear quantization to 8-bit codes (Sec. 2.3, the
 *              linear map Q(X) = round(X/S + Z) with S taken from the group's
 *              [x_min, x_max], and grouped quantization), then the
 *              split-stream construction of Alg. 1 stage 4 / Sec. 4.1: the 4
 *              most significant bits form the Anchor stream, the 4 least
 *              significant bits the Residual stream, two 4-bit values packed
 *              per byte (Sec. 5, Compression Kernel).
 *   merge   -- the Residual phase of Sec. 4.2: Anchor and Residual recombine
 *              into the full 8-bit code Q_full.
 *   dequant -- value reconstruction from the 8-bit code, or from the Anchor
 *              alone (Anchor phase of Sec. 4.2).
 *   attention -- O = softmax(Q K^T / sqrt(d_k)) V (Sec. 2, attention
 *              equation): decode of one query over the Anchor-only cache
 *              (Sec. 4.2 Anchor phase, Speculative Decoder) and the single
 *              parallel verification pass of k draft queries over the merged
 *              cache, causal among the drafts (Sec. 4.3); the decode may also
 *              attend the BF16 tokens generated since the context arrived
 *              (the speculative decoder's own KV, Sec. 4.2-4.3);
 *              the decode over the A-bit anchors of the other split widths
 *              (Sec. 8) as well.
 *
 * Readings where the paper is silent (each listed in the design notes):
 *   - K is grouped per channel over 128 consecutive tokens, V per token over
 *     its 128 dims.
 *   - zero = group minimum (the value of code 0); scale = (max - min) / 255;
 *     the code is rint((x - zero) * inv) with inv = 255 / (max - min), all in
 *     IEEE fp32, rint = round half to even, clamped to [0, 255].
 *   - A group whose range is not a positive finite number, or whose inverse
 *     range overflows, gets scale = inv = 0 and all codes 0.
 *   - -0 in a group's min/max is stored as +0.
 *   - Split: anchor a = code >> 4, residual r = code & 15, so code = a*16 + r.
 *   - Anchor-only reconstruction: zero + (16 a + 7.5) * scale (the centre of
 *     the 16 codes an anchor value stands for).
 *   - Packing: within a byte the low nibble holds the even element (dim 2j),
 *     the high nibble the odd one (dim 2j+1).
 *   - Plane layout: a token row of a nibble plane is 64 bytes; the row of
 *     (sequence b, kv head h, token t) starts at
 *        ((block_table[b][t / bt] * Hkv + h) * bt + t % bt) * 64.
 *     Code planes use the same formula with 128-byte rows.
 *   - Metadata is logical (never paged): k_scale/k_zero are
 *     [B][Hkv][ceil(max_tokens/128)][128], v_scale/v_zero [B][Hkv][max_tokens].
 *   - Query head hq reads kv head hq / (Hq / Hkv).
 *   - Verification: draft query i sees the whole context plus draft tokens
 *     0..i, whose K/V are BF16 and never quantized.
 *   - Decode with a tail: the query sees the whole context plus all n_tail
 *     BF16 tokens passed with it (the caller passes exactly the visible ones).
 *
 * Precision: the codec runs in fp32 because fp32 arithmetic decides the
 * integer codes and the GPU path must take the same decision; attention runs
 * in fp64 from the fp32 metadata and exact BF16->fp64 inputs.
 *
 * Build: gcc -O2 -ffp-contract=off -fno-fast-math -shared -fPIC -pthread.
 */
#include <float.h>
#include <math.h>
#include <pthread.h>
#include <stddef.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define HEAD_DIM 128
#define K_GROUP 128
#define NIBBLE_ROW 64
#define CODE_ROW 128

/* ------------------------------------------------------------------------ */
/* Scalar helpers                                                            */
/* ------------------------------------------------------------------------ */

/* BF16 is the top half of an IEEE fp32; widening is exact. */
static float bf16_bits_to_float(uint16_t bits)
{
    uint32_t u = (uint32_t)bits << 16;
    float f;
    memcpy(&f, &u, sizeof f);
    return f;
}

/* Byte offset of token row (b, h, t) in a plane with `row_bytes` per row. */
static size_t plane_row_offset(const int32_t *block_table_row, int Hkv, int bt,
                               int h, int t, int row_bytes)
{
    size_t block = (size_t)block_table_row[t / bt];
    return ((block * (size_t)Hkv + (size_t)h) * (size_t)bt + (size_t)(t % bt)) *
           (size_t)row_bytes;
}

/* Group statistics of Sec. 2.3: zero = min, scale = (max-min)/255, and the
 * reciprocal inv = 255/(max-min) used to map values onto 0..255. */
static void group_stats(const float *x, int n, float *scale, float *zero,
                        float *inv)
{
    float mn = x[0], mx = x[0];
    for (int i = 1; i < n; ++i) {
        if (x[i] < mn) mn = x[i];
        if (x[i] > mx) mx = x[i];
    }
    if (mn == 0.0f) mn = 0.0f; /* store -0 as +0 */
    if (mx == 0.0f) mx = 0.0f;
    float range = mx - mn;
    float r = 255.0f / range;
    if (!(range > 0.0f) || !(range <= FLT_MAX) || !(r <= FLT_MAX)) {
        *scale = 0.0f;
        *inv = 0.0f;
    } else {
        *scale = range / 255.0f;
        *inv = r;
    }
    *zero = mn;
}

/* Linear quantization of one value to an unsigned 8-bit code. */
static int quantize(float x, float zero, float inv)
{
    float y = (x - zero) * inv;
    float c = rintf(y);
    if (!(c >= 0.0f)) c = 0.0f; /* also maps NaN to 0 */
    if (c > 255.0f) c = 255.0f;
    return (int)c;
}

/* Put 4-bit value `nib` as element `e` of a packed row (low nibble = even e). */
static void put_nibble(uint8_t *row, int e, int nib)
{
    int j = e / 2;
    int shift = (e % 2) * 4;
    row[j] = (uint8_t)((row[j] & ~(0xF << shift)) | ((nib & 0xF) << shift));
}

static int get_nibble(const uint8_t *row, int e)
{
    return (row[e / 2] >> ((e % 2) * 4)) & 0xF;
}

/* ------------------------------------------------------------------------ */
/* Encode (quantize, split, pack) for one sequence b of one layer            */
/* ------------------------------------------------------------------------ */

/*
 * k, v: BF16 bits [T][Hkv][128].  Writes the four nibble planes for rows
 * t < T of sequence b and metadata row b.  Returns 0, or -1 on bad sizes.
 */
int oracle_encode(int Hkv, int bt, int max_blocks, int max_tokens, int b, int T,
                  const int32_t *block_table, const uint16_t *k,
                  const uint16_t *v, uint8_t *k_anc, uint8_t *v_anc,
                  uint8_t *k_res, uint8_t *v_res, float *k_scale,
                  float *k_zero, float *v_scale, float *v_zero)
{
    if (Hkv < 1 || bt < 1 || T < 0 || T > max_tokens ||
        (size_t)(T + bt - 1) / (size_t)bt > (size_t)max_blocks)
        return -1;
    const int32_t *bt_row = block_table + (size_t)b * (size_t)max_blocks;
    const int n_groups_max = (max_tokens + K_GROUP - 1) / K_GROUP;
    float vals[K_GROUP > HEAD_DIM ? K_GROUP : HEAD_DIM];

    for (int h = 0; h < Hkv; ++h) {
        /* K: one group per (128-token window g, channel d). */
        for (int g = 0; g * K_GROUP < T; ++g) {
            int t0 = g * K_GROUP;
            int t1 = t0 + K_GROUP < T ? t0 + K_GROUP : T;
            for (int d = 0; d < HEAD_DIM; ++d) {
                for (int t = t0; t < t1; ++t)
                    vals[t - t0] = bf16_bits_to_float(
                        k[((size_t)t * Hkv + h) * HEAD_DIM + d]);
                float scale, zero, inv;
                group_stats(vals, t1 - t0, &scale, &zero, &inv);
                for (int t = t0; t < t1; ++t) {
                    int c = quantize(vals[t - t0], zero, inv);
                    size_t off = plane_row_offset(bt_row, Hkv, bt, h, t, NIBBLE_ROW);
                    put_nibble(k_anc + off, d, c >> 4);
                    put_nibble(k_res + off, d, c & 15);
                }
                size_t m = (((size_t)b * Hkv + h) * n_groups_max + g) * HEAD_DIM + d;
                k_scale[m] = scale;
                k_zero[m] = zero;
            }
        }
        /* V: one group per token, over its 128 dims. */
        for (int t = 0; t < T; ++t) {
            for (int d = 0; d < HEAD_DIM; ++d)
                vals[d] = bf16_bits_to_float(v[((size_t)t * Hkv + h) * HEAD_DIM + d]);
            float scale, zero, inv;
            group_stats(vals, HEAD_DIM, &scale, &zero, &inv);
            size_t off = plane_row_offset(bt_row, Hkv, bt, h, t, NIBBLE_ROW);
            for (int d = 0; d < HEAD_DIM; ++d) {
                int c = quantize(vals[d], zero, inv);
                put_nibble(v_anc + off, d, c >> 4);
                put_nibble(v_res + off, d, c & 15);
            }
            size_t m = ((size_t)b * Hkv + h) * (size_t)max_tokens + t;
            v_scale[m] = scale;
            v_zero[m] = zero;
        }
    }
    return 0;
}

/* ------------------------------------------------------------------------ */
/* Merge (Residual phase): code = anchor * 16 + residual, element by element */
/* ------------------------------------------------------------------------ */

/* n_packed bytes of each nibble plane -> 2 * n_packed code bytes. */
void oracle_merge(const uint8_t *anc, const uint8_t *res, uint8_t *codes,
                  size_t n_packed)
{
    for (size_t e = 0; e < 2 * n_packed; ++e) {
        int a = (anc[e / 2] >> ((e % 2) * 4)) & 0xF;
        int r = (res[e / 2] >> ((e % 2) * 4)) & 0xF;
        codes[e] = (uint8_t)(a * 16 + r);
    }
}

/* ------------------------------------------------------------------------ */
/* Dequantization                                                            */
/* ------------------------------------------------------------------------ */

/* One reconstructed element (b, h, t, d), fp64.
 * mode 0: anchor-only, planes are nibble planes:  x = zero + (16 a + 7.5) scale
 * mode 1: full 8-bit, planes are code planes:     x = zero + c * scale      */
static int get_field(const uint8_t *row, int e, int w);

/* mode 0: 4-bit anchors (16 a + 7.5); mode 1: 8-bit codes; mode 2: A-bit
 * anchors of a split width (rows of 16 A bytes, the anchor standing for code
 * 2^R a + (2^R - 1) / 2 with R = 8 - A). */
static void dequant_element(int mode, int A, int Hkv, int bt, int max_tokens,
                            const int32_t *bt_row, int b, int h, int t, int d,
                            const uint8_t *k_plane, const uint8_t *v_plane,
                            const float *k_scale, const float *k_zero,
                            const float *v_scale, const float *v_zero,
                            double *k_out, double *v_out)
{
    const int n_groups_max = (max_tokens + K_GROUP - 1) / K_GROUP;
    const int row_bytes = mode == 0 ? NIBBLE_ROW : mode == 1 ? CODE_ROW : 16 * A;
    size_t off = plane_row_offset(bt_row, Hkv, bt, h, t, row_bytes);
    size_t km = (((size_t)b * Hkv + h) * n_groups_max + t / K_GROUP) * HEAD_DIM + d;
    size_t vm = ((size_t)b * Hkv + h) * (size_t)max_tokens + t;
    double kq, vq;
    if (mode == 0) {
        kq = 16.0 * get_nibble(k_plane + off, d) + 7.5;
        vq = 16.0 * get_nibble(v_plane + off, d) + 7.5;
    } else if (mode == 2) {
        const int R = 8 - A;
        const double w = (double)(1 << R), half = ((double)(1 << R) - 1.0) / 2.0;
        kq = w * get_field(k_plane + off, d, A) + half;
        vq = w * get_field(v_plane + off, d, A) + half;
    } else {
        kq = (double)k_plane[off + d];
        vq = (double)v_plane[off + d];
    }
    *k_out = (double)k_zero[km] + kq * (double)k_scale[km];
    *v_out = (double)v_zero[vm] + vq * (double)v_scale[vm];
}

/*
 * Fills k_hat, v_hat [T][Hkv][128] (fp64) for sequence b; mode as above.
 * Returns 0 or -1.
 */
int oracle_dequant(int mode, int Hkv, int bt, int max_blocks, int max_tokens,
                   int b, int T, const int32_t *block_table,
                   const uint8_t *k_plane, const uint8_t *v_plane,
                   const float *k_scale, const float *k_zero,
                   const float *v_scale, const float *v_zero, double *k_hat,
                   double *v_hat)
{
    if ((mode != 0 && mode != 1) || T < 0 || T > max_tokens) return -1;
    const int32_t *bt_row = block_table + (size_t)b * (size_t)max_blocks;
    for (int t = 0; t < T; ++t)
        for (int h = 0; h < Hkv; ++h)
            for (int d = 0; d < HEAD_DIM; ++d) {
                size_t o = ((size_t)t * Hkv + h) * HEAD_DIM + d;
                dequant_element(mode, 0, Hkv, bt, max_tokens, bt_row, b, h, t, d,
                                k_plane, v_plane, k_scale, k_zero, v_scale,
                                v_zero, &k_hat[o], &v_hat[o]);
            }
    return 0;
}

/* ------------------------------------------------------------------------ */
/* Attention: O = softmax(q K^T / sqrt(d)) V, fp64                           */
/* ------------------------------------------------------------------------ */

/* One query row over n key/value rows (row stride `stride` doubles).
 * Writes o[128] and the log-sum-exp of the scaled scores. */
static void attend(const double *q, const double *keys, const double *vals,
                   size_t stride, int n, double *o, double *lse)
{
    const double sm_scale = 1.0 / sqrt((double)HEAD_DIM);
    double *s = (double *)malloc(sizeof(double) * (size_t)(n > 0 ? n : 1));
    double m = -INFINITY;
    for (int t = 0; t < n; ++t) {
        double acc = 0.0;
        for (int d = 0; d < HEAD_DIM; ++d) acc += q[d] * keys[(size_t)t * stride + d];
        s[t] = acc * sm_scale;
        if (s[t] > m) m = s[t];
    }
    double l = 0.0;
    for (int t = 0; t < n; ++t) {
        s[t] = exp(s[t] - m);
        l += s[t];
    }
    for (int d = 0; d < HEAD_DIM; ++d) {
        double acc = 0.0;
        for (int t = 0; t < n; ++t) acc += s[t] * vals[(size_t)t * stride + d];
        o[d] = n > 0 ? acc / l : 0.0;
    }
    if (lse) *lse = n > 0 ? m + log(l) : -INFINITY;
    free(s);
}

typedef struct {
    int mode; /* 0 anchor decode, 1 verify, 2 anchor decode over A-bit anchors */
    int anchor_bits; /* mode 2: A */
    int Hkv, bt, max_blocks, max_tokens, B, Hq, nq;
    int n_tail; /* anchor decode: BF16 tail tokens per sequence, all visible */
    const int32_t *seq_lens, *block_table;
    const uint8_t *k_plane, *v_plane;
    const float *k_scale, *k_zero, *v_scale, *v_zero;
    const uint16_t *q, *k_new, *v_new;
    const uint8_t *unit_mask;
    double *out, *lse;
    int nthreads;
    int thread_id;
    int status;
} attn_job;

/* Work unit u = b * Hkv + kvh: all G query heads of one kv head. */
static void attention_unit(const attn_job *J, int u, double *keys, double *vals)
{
    const int Hkv = J->Hkv, G = J->Hq / J->Hkv;
    const int b = u / Hkv, kvh = u % Hkv;
    const int T = J->seq_lens[b];
    const int32_t *bt_row = J->block_table + (size_t)b * (size_t)J->max_blocks;
    for (int t = 0; t < T; ++t)
        for (int d = 0; d < HEAD_DIM; ++d)
            dequant_element(J->mode, J->anchor_bits, Hkv, J->bt, J->max_tokens, bt_row, b, kvh, t,
                            d, J->k_plane, J->v_plane, J->k_scale, J->k_zero,
                            J->v_scale, J->v_zero, &keys[(size_t)t * HEAD_DIM + d],
                            &vals[(size_t)t * HEAD_DIM + d]);
    double qd[HEAD_DIM];
    for (int i = 0; i < J->nq; ++i) {
        int n = T;
        if (J->k_new) {
            /* BF16 tokens follow the context: in verification drafts 0..i
               (causal among the drafts); in decode all n_tail tokens generated
               since the context was transferred. */
            const int n_new = J->mode == 1 ? i + 1 : J->n_tail;
            const int stride = J->mode == 1 ? J->nq : J->n_tail;
            for (int j = 0; j < n_new; ++j)
                for (int d = 0; d < HEAD_DIM; ++d) {
                    size_t src = ((((size_t)b * stride + j) * Hkv) + kvh) * HEAD_DIM + d;
                    keys[(size_t)(T + j) * HEAD_DIM + d] = bf16_bits_to_float(J->k_new[src]);
                    vals[(size_t)(T + j) * HEAD_DIM + d] = bf16_bits_to_float(J->v_new[src]);
                }
            n = T + n_new;
        }
        for (int g = 0; g < G; ++g) {
            int hq = kvh * G + g;
            size_t row = (((size_t)b * J->nq + i) * J->Hq + hq);
            for (int d = 0; d < HEAD_DIM; ++d)
                qd[d] = bf16_bits_to_float(J->q[row * HEAD_DIM + d]);
            attend(qd, keys, vals, HEAD_DIM, n, J->out + row * HEAD_DIM,
                   J->lse ? J->lse + row : NULL);
        }
    }
}

static void *attention_worker(void *arg)
{
    attn_job *J = (attn_job *)arg;
    int max_T = 0;
    for (int b = 0; b < J->B; ++b)
        if (J->seq_lens[b] > max_T) max_T = J->seq_lens[b];
    size_t one = (size_t)(max_T + J->nq + J->n_tail + 1) * HEAD_DIM;
    double *keys = (double *)malloc(one * sizeof(double));
    double *vals = (double *)malloc(one * sizeof(double));
    if (!keys || !vals) {
        J->status = -2;
    } else {
        int units = J->B * J->Hkv;
        for (int u = J->thread_id; u < units; u += J->nthreads)
            if (!J->unit_mask || J->unit_mask[u]) attention_unit(J, u, keys, vals);
    }
    free(keys);
    free(vals);
    return NULL;
}

static int run_attention(attn_job *base)
{
    if (base->Hkv < 1 || base->Hq < 1 || base->Hq % base->Hkv != 0 || base->B < 0 ||
        base->nq < 1 || base->n_tail < 0)
        return -1;
    for (int b = 0; b < base->B; ++b)
        if (base->seq_lens[b] < 0 || base->seq_lens[b] > base->max_tokens) return -1;
    int nt = base->nthreads < 1 ? 1 : base->nthreads;
    attn_job *jobs = (attn_job *)calloc((size_t)nt, sizeof(attn_job));
    pthread_t *th = (pthread_t *)calloc((size_t)nt, sizeof(pthread_t));
    if (!jobs || !th) {
        free(jobs);
        free(th);
        return -2;
    }
    for (int i = 0; i < nt; ++i) {
        jobs[i] = *base;
        jobs[i].nthreads = nt;
        jobs[i].thread_id = i;
        jobs[i].status = 0;
    }
    for (int i = 1; i < nt; ++i) pthread_create(&th[i], NULL, attention_worker, &jobs[i]);
    attention_worker(&jobs[0]);
    int status = jobs[0].status;
    for (int i = 1; i < nt; ++i) {
        pthread_join(th[i], NULL);
        if (jobs[i].status) status = jobs[i].status;
    }
    free(jobs);
    free(th);
    return status;
}

/*
 * Anchor-phase decode: one query per sequence over the Anchor-only cache.
 * q: BF16 bits [B][Hq][128]; out: fp64 [B][Hq][128]; lse: fp64 [B][Hq] or NULL.
 * unit_mask: NULL, or B*Hkv flags selecting which (b, kv head) units to compute.
 */
int oracle_anchor_decode(int Hkv, int bt, int max_blocks, int max_tokens, int B,
                         int Hq, const int32_t *seq_lens,
                         const int32_t *block_table, const uint8_t *k_anc,
                         const uint8_t *v_anc, const float *k_scale,
                         const float *k_zero, const float *v_scale,
                         const float *v_zero, const uint16_t *q, double *out,
                         double *lse, const uint8_t *unit_mask, int nthreads)
{
    attn_job J;
    memset(&J, 0, sizeof J);
    J.mode = 0;
    J.Hkv = Hkv; J.bt = bt; J.max_blocks = max_blocks; J.max_tokens = max_tokens;
    J.B = B; J.Hq = Hq; J.nq = 1;
    J.seq_lens = seq_lens; J.block_table = block_table;
    J.k_plane = k_anc; J.v_plane = v_anc;
    J.k_scale = k_scale; J.k_zero = k_zero; J.v_scale = v_scale; J.v_zero = v_zero;
    J.q = q; J.out = out; J.lse = lse; J.unit_mask = unit_mask;
    J.nthreads = nthreads;
    return run_attention(&J);
}

/*
 * Anchor-phase decode with the tokens generated since the context arrived:
 * one query per sequence over the Anchor-only cache followed by n_tail BF16
 * tokens (k_new, v_new: BF16 bits [B][n_tail][Hkv][128]), all visible to the
 * query.  n_tail = 0 is the plain anchor decode.
 */
int oracle_anchor_decode_tail(int Hkv, int bt, int max_blocks, int max_tokens, int B,
                              int Hq, const int32_t *seq_lens,
                              const int32_t *block_table, const uint8_t *k_anc,
                              const uint8_t *v_anc, const float *k_scale,
                              const float *k_zero, const float *v_scale,
                              const float *v_zero, const uint16_t *q, int n_tail,
                              const uint16_t *k_new, const uint16_t *v_new,
                              double *out, double *lse, const uint8_t *unit_mask,
                              int nthreads)
{
    if (n_tail < 0 || (n_tail > 0 && (!k_new || !v_new))) return -1;
    attn_job J;
    memset(&J, 0, sizeof J);
    J.mode = 0;
    J.Hkv = Hkv; J.bt = bt; J.max_blocks = max_blocks; J.max_tokens = max_tokens;
    J.B = B; J.Hq = Hq; J.nq = 1; J.n_tail = n_tail;
    J.seq_lens = seq_lens; J.block_table = block_table;
    J.k_plane = k_anc; J.v_plane = v_anc;
    J.k_scale = k_scale; J.k_zero = k_zero; J.v_scale = v_scale; J.v_zero = v_zero;
    J.q = q; J.k_new = n_tail > 0 ? k_new : NULL; J.v_new = n_tail > 0 ? v_new : NULL;
    J.out = out; J.lse = lse; J.unit_mask = unit_mask;
    J.nthreads = nthreads;
    return run_attention(&J);
}

/*
 * Verification pass: nq draft queries per sequence over the merged 8-bit
 * cache, plus (if k_new != NULL) the BF16 draft tokens, causal among drafts.
 * q: BF16 bits [B][nq][Hq][128]; k_new, v_new: BF16 bits [B][nq][Hkv][128]
 * or NULL; out: fp64 [B][nq][Hq][128]; lse: fp64 [B][nq][Hq] or NULL.
 */
int oracle_verify(int Hkv, int bt, int max_blocks, int max_tokens, int B, int Hq,
                  int nq, const int32_t *seq_lens, const int32_t *block_table,
                  const uint8_t *k_codes, const uint8_t *v_codes,
                  const float *k_scale, const float *k_zero,
                  const float *v_scale, const float *v_zero, const uint16_t *q,
                  const uint16_t *k_new, const uint16_t *v_new, double *out,
                  double *lse, const uint8_t *unit_mask, int nthreads)
{
    if ((k_new == NULL) != (v_new == NULL)) return -1;
    attn_job J;
    memset(&J, 0, sizeof J);
    J.mode = 1;
    J.Hkv = Hkv; J.bt = bt; J.max_blocks = max_blocks; J.max_tokens = max_tokens;
    J.B = B; J.Hq = Hq; J.nq = nq;
    J.seq_lens = seq_lens; J.block_table = block_table;
    J.k_plane = k_codes; J.v_plane = v_codes;
    J.k_scale = k_scale; J.k_zero = k_zero; J.v_scale = v_scale; J.v_zero = v_zero;
    J.q = q; J.k_new = k_new; J.v_new = v_new;
    J.out = out; J.lse = lse; J.unit_mask = unit_mask;
    J.nthreads = nthreads;
    return run_attention(&J);
}

/* ------------------------------------------------------------------------ */
/* Hierarchical non-linear quantization (Alg. 1, Sec. 4.1)                   */
/* ------------------------------------------------------------------------ */
/*
 * Per channel of one kv head (K and V alike), over pages of 256 tokens and
 * chunks of 32 tokens (the configuration of Sec. 6.1), in the order of the
 * four stages of Alg. 1:
 *   1. page normalization: gmin = min x and gscale = max x - gmin over the
 *      page's tokens; X = (x - gmin) * (1 / gscale), so X lies in [0, 1];
 *   2. chunk isolation: mu = the mean of X over the chunk's tokens (an fp32
 *      sum in token order divided by the count), Xc = X - mu,
 *      sigma = max |Xc|, Xf = Xc * (1 / sigma), so |Xf| <= 1;
 *   3. non-linear transform: I = Round(M ln(1 + a |Xf|) / ln(1 + a)), the
 *      sign S of Xc, with M = 127 (seven magnitude bits and a sign);
 *   4. split into a signed 4-bit anchor and a signed 4-bit residual, both
 *      kept as two's complement nibbles; the anchor is the magnitude's
 *      bucket V with the sign-aware map Q_anc = V for S >= 0 and -V - 1 for
 *      S < 0, so a zero magnitude keeps its sign.
 * Three variants of stage 4 (the variant argument):
 *   0 (biased): Alg. 1's split: V = (I + 7) >> 4, the magnitude rounded
 *     half down to a multiple of 16, Q_res = 16 V - I.  V reaches 8 for
 *     I >= 121, which 4 bits cannot hold with a sign: V is clamped to 7 and
 *     Q_res to [-8, 7], so codes above 120 come back as 120.  The anchor
 *     alone reconstructs code 16 V; anchor and residual 16 V - Q_res.
 *   1 (centred): the lossless split that keeps all 128 magnitudes: V = I >> 4
 *     (the top three magnitude bits: the anchor is the sign and the top
 *     bits of the 8-bit code), Q_res = I - 16 V - 8, a correction centred on
 *     the bucket's middle.  The anchor alone reconstructs code 16 V + 7.5,
 *     the bucket's centre; anchor and residual 16 V + 8 + Q_res = I.  The
 *     merged byte is then a complete 8-bit code: the single-precision 8-bit
 *     configuration of Sec. 6.1.
 *   2 (4-bit): the single-precision 4-bit configuration of Sec. 6.1: stage 3
 *     with M = 7 (three magnitude bits and a sign), the anchor holding
 *     Q = I or -I - 1 and no residual.
 * Readings where Alg. 1 is garbled or at odds with the 4-bit streams:
 *   - the sign is that of the centred value Xc (Alg. 1's X_view is
 *     non-negative after stage 1);
 *   - no epsilon: a page (chunk) whose range (sigma) has no finite positive
 *     reciprocal normalizes to 0;
 *   - Round(Y) is decided as the number of decision thresholds theta_k
 *     (k = 0..M-1) with theta_k <= |Xf|, theta_k being the fp32 value of
 *     expm1(((k + 0.5) / M) * log1p(a)) / a in IEEE double: the point
 *     where the transform equals k + 1/2;
 *   - reconstruction maps a code index i to the level
 *     expm1((i / M) * log1p(a)) / a (fp32 of the double value), then
 *     x = ((+-level * sigma) + mu) * gscale + gmin, each step an fp32
 *     operation, rounded to BF16 to nearest even.
 */
#define H_PAGE 256
#define H_CHUNK 32

#define H_BIASED 0
#define H_CENTRED 1
#define H_INT4 2

/* Magnitude levels M of stage 3: 127 (8-bit code), 7 (4-bit code). */
static int h_levels(int variant) { return variant == H_INT4 ? 7 : 127; }

/* Decision thresholds theta[0..M-1], levels level[0..M] and the centred
 * split's anchor-only levels alevel[V] (code 16 V + 7.5, V = 0..7). */
static void h_tables(float alpha, int variant, float *theta, float *level, float *alevel)
{
    const double la = log1p((double)alpha);
    const int M = h_levels(variant);
    for (int k = 0; k < M; ++k)
        theta[k] = (float)(expm1(((k + 0.5) / M) * la) / (double)alpha);
    for (int i = 0; i <= M; ++i)
        level[i] = (float)(expm1(((double)i / M) * la) / (double)alpha);
    for (int v = 0; v < 8; ++v)
        alevel[v] = (float)(expm1(((16 * v + 7.5) / 127.0) * la) / (double)alpha);
}

/* The reciprocal of a range, or 0 when it is not a finite positive value. */
static float range_recip(float r)
{
    float v = 1.0f / r;
    return (r > 0.0f && v <= FLT_MAX) ? v : 0.0f;
}

/* Stage 4: the anchor and residual nibble values of (I, S).  Returns 0, or
 * -1 for an unknown variant or a code out of range. */
int oracle_hsplit(int variant, int I, int S, int *q_anc, int *q_res)
{
    if (variant < H_BIASED || variant > H_INT4 || I < 0 || I > h_levels(variant)) return -1;
    int V, r;
    if (variant == H_BIASED) {
        V = (I + 7) >> 4;
        if (V > 7) V = 7;
        r = 16 * V - I;
        if (r < -8) r = -8;
        if (r > 7) r = 7;
    } else if (variant == H_CENTRED) {
        V = I >> 4;
        r = I - 16 * V - 8;
    } else {
        V = I;
        r = 0;
    }
    *q_anc = S < 0 ? -V - 1 : V;
    *q_res = r;
    return 0;
}

/* Exposes the decision thresholds (M), reconstruction levels (M + 1) and the
 * centred split's anchor-only levels (8).  Returns M, or -1. */
int oracle_htables(float alpha, int variant, float *theta, float *level, float *alevel)
{
    if (variant < H_BIASED || variant > H_INT4) return -1;
    h_tables(alpha, variant, theta, level, alevel);
    return h_levels(variant);
}

static int sext4(int nib) { return nib >= 8 ? nib - 16 : nib; }

static uint16_t float_to_bf16_rne(float f)
{
    uint32_t u;
    memcpy(&u, &f, sizeof u);
    if ((u & 0x7F800000u) == 0x7F800000u && (u & 0x007FFFFFu)) return (uint16_t)((u >> 16) | 0x40);
    u += 0x7FFFu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
}

/*
 * k, v: BF16 bits [T][Hkv][128] of sequence b.  Writes its rows of the
 * anchor and residual nibble planes (variant 2: the anchor plane only; the
 * residual planes are not touched) and its metadata rows: gmin, gscale
 * [B][Hkv][ceil(max_tokens/256)][128], mu, sigma
 * [B][Hkv][ceil(max_tokens/32)][128], for K and V.  Returns 0, or -1.
 */
int oracle_hencode(int Hkv, int bt, int max_blocks, int max_tokens, int b, int T,
                   const int32_t *block_table, const uint16_t *k, const uint16_t *v, float alpha,
                   int variant, uint8_t *k_anc, uint8_t *v_anc, uint8_t *k_res, uint8_t *v_res,
                   float *k_gmin, float *k_gscale, float *k_mu, float *k_sigma,
                   float *v_gmin, float *v_gscale, float *v_mu, float *v_sigma)
{
    if (Hkv < 1 || bt < 1 || T < 0 || T > max_tokens || !(alpha > 0.0f)) return -1;
    if (variant < H_BIASED || variant > H_INT4) return -1;
    float theta[127], level[128], alevel[8];
    h_tables(alpha, variant, theta, level, alevel);
    const int M = h_levels(variant);
    const int n_pages = (max_tokens + H_PAGE - 1) / H_PAGE;
    const int n_chunks = (max_tokens + H_CHUNK - 1) / H_CHUNK;
    const int32_t *bt_row = block_table + (size_t)b * max_blocks;
    for (int which = 0; which < 2; ++which) {
        const uint16_t *src = which == 0 ? k : v;
        uint8_t *anc = which == 0 ? k_anc : v_anc;
        uint8_t *res = which == 0 ? k_res : v_res;
        float *gmin_a = which == 0 ? k_gmin : v_gmin, *gsc_a = which == 0 ? k_gscale : v_gscale;
        float *mu_a = which == 0 ? k_mu : v_mu, *sig_a = which == 0 ? k_sigma : v_sigma;
        for (int h = 0; h < Hkv; ++h)
            for (int p = 0; p * H_PAGE < T; ++p) {
                const int t0 = p * H_PAGE;
                const int n = T - t0 < H_PAGE ? T - t0 : H_PAGE;
                for (int d = 0; d < HEAD_DIM; ++d) {
                    float x[H_PAGE] = {0.0f}, X[H_PAGE];
                    for (int i = 0; i < n; ++i)
                        x[i] = bf16_bits_to_float(src[((size_t)(t0 + i) * Hkv + h) * HEAD_DIM + d]);
                    /* stage 1 */
                    float lo = x[0], hi = x[0];
                    for (int i = 1; i < n; ++i) {
                        if (x[i] < lo) lo = x[i];
                        if (x[i] > hi) hi = x[i];
                    }
                    if (lo == 0.0f) lo = 0.0f;
                    if (hi == 0.0f) hi = 0.0f;
                    const float gscale = hi - lo;
                    const float ig = range_recip(gscale);
                    for (int i = 0; i < n; ++i) X[i] = (x[i] - lo) * ig;
                    const size_t pm = (((size_t)b * Hkv + h) * n_pages + p) * HEAD_DIM + d;
                    gmin_a[pm] = lo;
                    gsc_a[pm] = gscale;
                    /* stages 2-4, chunk by chunk */
                    for (int c = 0; c * H_CHUNK < n; ++c) {
                        const int i0 = c * H_CHUNK;
                        const int cnt = n - i0 < H_CHUNK ? n - i0 : H_CHUNK;
                        float sum = 0.0f;
                        for (int i = i0; i < i0 + cnt; ++i) sum += X[i];
                        const float mu = sum / (float)cnt;
                        float sigma = 0.0f;
                        for (int i = i0; i < i0 + cnt; ++i) {
                            const float a = fabsf(X[i] - mu);
                            if (a > sigma) sigma = a;
                        }
                        const float is = range_recip(sigma);
                        const size_t cm = (((size_t)b * Hkv + h) * n_chunks + (size_t)t0 / H_CHUNK + c) * HEAD_DIM + d;
                        mu_a[cm] = mu;
                        sig_a[cm] = sigma;
                        for (int i = i0; i < i0 + cnt; ++i) {
                            const float xc = X[i] - mu;
                            float xf = fabsf(xc * is);
                            if (xf > 1.0f) xf = 1.0f;
                            int I = 0;
                            while (I < M && theta[I] <= xf) ++I;
                            const int S = xc > 0.0f ? 1 : (xc < 0.0f ? -1 : 0);
                            int qa, qr;
                            oracle_hsplit(variant, I, S, &qa, &qr);
                            const int t = t0 + i;
                            if (bt_row[t / bt] < 0) return -1;
                            const size_t row = plane_row_offset(bt_row, Hkv, bt, h, t, NIBBLE_ROW);
                            put_nibble(anc + row, d, qa & 0xF);
                            if (variant != H_INT4) put_nibble(res + row, d, qr & 0xF);
                        }
                    }
                }
            }
    }
    return 0;
}

/*
 * Reconstruction of sequence b's K and V as BF16 bits [T][Hkv][128]:
 * mode 0 from the anchor nibble planes alone, mode 1 from the merged code
 * planes (byte of element e: anchor nibble << 4 | residual nibble; not for
 * variant 2).  The code index is, by variant: 0: 16 V (anchor),
 * 16 V - Q_res (merged); 1: 16 V + 7.5 (anchor), 16 V + 8 + Q_res (merged);
 * 2: V.  Returns 0, or -1.
 */
int oracle_hdequant(int mode, int variant, int Hkv, int bt, int max_blocks, int max_tokens, int b, int T,
                    const int32_t *block_table, const uint8_t *k_plane, const uint8_t *v_plane,
                    float alpha, const float *k_gmin, const float *k_gscale, const float *k_mu,
                    const float *k_sigma, const float *v_gmin, const float *v_gscale,
                    const float *v_mu, const float *v_sigma, uint16_t *k_out, uint16_t *v_out)
{
    if ((mode != 0 && mode != 1) || Hkv < 1 || T < 0 || T > max_tokens || !(alpha > 0.0f)) return -1;
    if (variant < H_BIASED || variant > H_INT4 || (variant == H_INT4 && mode == 1)) return -1;
    float theta[127], level[128], alevel[8];
    h_tables(alpha, variant, theta, level, alevel);
    const int n_pages = (max_tokens + H_PAGE - 1) / H_PAGE;
    const int n_chunks = (max_tokens + H_CHUNK - 1) / H_CHUNK;
    const int32_t *bt_row = block_table + (size_t)b * max_blocks;
    for (int which = 0; which < 2; ++which) {
        const uint8_t *plane = which == 0 ? k_plane : v_plane;
        const float *gmin_a = which == 0 ? k_gmin : v_gmin, *gsc_a = which == 0 ? k_gscale : v_gscale;
        const float *mu_a = which == 0 ? k_mu : v_mu, *sig_a = which == 0 ? k_sigma : v_sigma;
        uint16_t *out = which == 0 ? k_out : v_out;
        for (int t = 0; t < T; ++t)
            for (int h = 0; h < Hkv; ++h) {
                if (bt_row[t / bt] < 0) return -1;
                const uint8_t *row = plane + plane_row_offset(bt_row, Hkv, bt, h, t,
                                                              mode == 0 ? NIBBLE_ROW : CODE_ROW);
                for (int d = 0; d < HEAD_DIM; ++d) {
                    int qa, Ip;
                    if (mode == 0) {
                        qa = sext4(get_nibble(row, d));
                    } else {
                        qa = sext4(row[d] >> 4);
                    }
                    const int V = qa >= 0 ? qa : -qa - 1;
                    float lv;
                    if (variant == H_BIASED) {
                        Ip = 16 * V;
                        if (mode == 1) Ip -= sext4(row[d] & 0xF);
                        if (Ip < 0) Ip = 0;
                        if (Ip > 127) Ip = 127;
                        lv = level[Ip];
                    } else if (variant == H_CENTRED) {
                        if (mode == 1) {
                            Ip = 16 * V + 8 + sext4(row[d] & 0xF);
                            lv = level[Ip];
                        } else {
                            lv = alevel[V];
                        }
                    } else {
                        lv = level[V];
                    }
                    const float m = qa >= 0 ? lv : -lv;
                    const size_t pm = (((size_t)b * Hkv + h) * n_pages + t / H_PAGE) * HEAD_DIM + d;
                    const size_t cm = (((size_t)b * Hkv + h) * n_chunks + t / H_CHUNK) * HEAD_DIM + d;
                    const float xc = m * sig_a[cm];
                    const float X = xc + mu_a[cm];
                    const float y = X * gsc_a[pm];
                    const float x = y + gmin_a[pm];
                    out[((size_t)t * Hkv + h) * HEAD_DIM + d] = float_to_bf16_rne(x);
                }
            }
    }
    return 0;
}

/* ------------------------------------------------------------------------ */
/* Acceptance of drafts by sampling (Sec. 4.3)                               */
/* ------------------------------------------------------------------------ */
/*
 * Sec. 4.3 keeps the longest prefix of the drafts the target model agrees
 * with and corrects the first divergence.  With sampled drafts the agreement
 * test is the standard speculative-sampling rule: draft i (token x, drawn
 * from the draft distribution q_i) is kept with probability
 * min(1, p_i(x) / q_i(x)), p_i the target's distribution; at the first draft
 * not kept, n, the next token is drawn from the residual weights
 * max(p_n - q_n, 0); when all k are kept, the bonus token is drawn from
 * p_k.  The emitted tokens are then distributed as the target's.
 * Readings (the paper fixes none of the mechanics):
 *   - the random numbers are inputs: u[b][i] (i < k) for the test of draft
 *     i, u[b][k] for the draw;
 *   - draft i is kept when u[b][i] * q_i(x) <= p_i(x), the fp32 product
 *     rounded once; a token outside [0, V) is not kept;
 *   - each weight is clamped to [0, 1] (NaN counts 0); if every residual
 *     weight is 0 the draw uses p_n, and if that is all 0 too, next_token is
 *     -1;
 *   - the draw is inverse-CDF sampling with every step exact: weights
 *     w_v = floor(r_v * 2^40), S = sum w_v, U = floor(u[b][k] * 2^32) clamped
 *     to [0, 2^32 - 1] (NaN -> 0), t = floor(S * U / 2^32), and the token is
 *     the smallest v whose inclusive prefix sum of w exceeds t.
 */
static uint64_t sample_weight(float r)
{
    r = r > 0.0f ? r : 0.0f; /* NaN and negatives count 0 */
    r = r < 1.0f ? r : 1.0f;
    return (uint64_t)(r * 1099511627776.0f); /* 2^40: an exact scaling, then truncation */
}

static uint32_t sample_uniform(float u)
{
    const float s = u * 4294967296.0f; /* 2^32 */
    if (!(s > 0.0f)) return 0u;
    if (s >= 4294967296.0f) return 0xFFFFFFFFu;
    return (uint32_t)s;
}

/* Residual weight of token v: p_v - q_v (q != NULL) or p_v. */
static float sample_residual(const float *p, const float *q, int v)
{
    return q ? p[v] - q[v] : p[v];
}

/* The draw over the residual weights; -1 if S = 0. */
static int32_t sample_draw(int V, const float *p, const float *q, float u)
{
    uint64_t S = 0;
    for (int v = 0; v < V; ++v) S += sample_weight(sample_residual(p, q, v));
    if (S == 0) return -1;
    const unsigned __int128 prod = (unsigned __int128)S * sample_uniform(u);
    const uint64_t t = (uint64_t)(prod >> 32);
    uint64_t acc = 0;
    for (int v = 0; v < V; ++v) {
        acc += sample_weight(sample_residual(p, q, v));
        if (acc > t) return v;
    }
    return -1; /* not reached: t < S */
}

/*
 * p: [B][k+1][V] target probabilities, q: [B][k][V] draft probabilities,
 * drafts: int32 [B][k], u: [B][k+1] uniforms.  Writes accepted[B] (0..k)
 * and next_token[B].  Returns 0, or -1 on bad sizes.
 */
int oracle_accept_sample(int B, int k, int V, const float *p, const float *q,
                         const int32_t *drafts, const float *u, int32_t *accepted,
                         int32_t *next_token)
{
    if (B < 0 || k < 1 || V < 1) return -1;
    for (int b = 0; b < B; ++b) {
        const float *pb = p + (size_t)b * (k + 1) * V;
        const float *qb = q + (size_t)b * k * V;
        const float *ub = u + (size_t)b * (k + 1);
        int n = 0;
        while (n < k) {
            const int32_t x = drafts[(size_t)b * k + n];
            if (x < 0 || x >= V) break;
            const float prod = ub[n] * qb[(size_t)n * V + x];
            if (!(prod <= pb[(size_t)n * V + x])) break;
            ++n;
        }
        accepted[b] = n;
        int32_t tok = -1;
        if (n < k) tok = sample_draw(V, pb + (size_t)n * V, qb + (size_t)n * V, ub[k]);
        if (tok < 0) tok = sample_draw(V, pb + (size_t)n * V, NULL, ub[k]);
        next_token[b] = tok;
    }
    return 0;
}

/* ------------------------------------------------------------------------ */
/* Split widths other than 4 + 4 (the paper's future work, Sec. 8)           */
/* ------------------------------------------------------------------------ */
/*
 * The uniform codec's 8-bit code c split into an anchor of A bits, c >> R,
 * and a residual of R = 8 - A bits, c & (2^R - 1), for A in {2, 4, 6}.
 * A plane row holds the 128 elements of one token and kv head as a
 * little-endian bit string: element e at bits e W .. e W + W - 1 (W = A or
 * R), byte j holding bits 8 j .. 8 j + 7, so a row is 16 W bytes.  W = 4 is
 * the nibble layout of the 4 + 4 planes.  Merging gives back c = (a << R) | r.
 * The anchor alone stands for code 2^R a + (2^R - 1) / 2, the middle of the
 * codes it covers, dequantized as the fp32 fmaf(code, scale, zero) rounded
 * to BF16 to nearest even (the BF16 pages of the paper's anchor phase).
 */
static void put_field(uint8_t *row, int e, int w, int val)
{
    for (int i = 0; i < w; ++i) {
        const int bit = e * w + i;
        const uint8_t m = (uint8_t)(1u << (bit % 8));
        if ((val >> i) & 1)
            row[bit / 8] |= m;
        else
            row[bit / 8] &= (uint8_t)~m;
    }
}

static int get_field(const uint8_t *row, int e, int w)
{
    int v = 0;
    for (int i = 0; i < w; ++i) {
        const int bit = e * w + i;
        v |= ((row[bit / 8] >> (bit % 8)) & 1) << i;
    }
    return v;
}

static int split_ok(int A) { return A == 2 || A == 4 || A == 6; }

/* As oracle_encode, with anchor rows of 16 A bytes and residual rows of
 * 16 (8 - A) bytes.  Returns 0, or -1. */
int oracle_encode_split(int A, int Hkv, int bt, int max_blocks, int max_tokens, int b, int T,
                        const int32_t *block_table, const uint16_t *k, const uint16_t *v,
                        uint8_t *k_anc, uint8_t *v_anc, uint8_t *k_res, uint8_t *v_res,
                        float *k_scale, float *k_zero, float *v_scale, float *v_zero)
{
    if (!split_ok(A) || Hkv < 1 || bt < 1 || T < 0 || T > max_tokens ||
        (size_t)(T + bt - 1) / (size_t)bt > (size_t)max_blocks)
        return -1;
    const int R = 8 - A;
    const int32_t *bt_row = block_table + (size_t)b * (size_t)max_blocks;
    const int n_groups_max = (max_tokens + K_GROUP - 1) / K_GROUP;
    float vals[K_GROUP > HEAD_DIM ? K_GROUP : HEAD_DIM];
    for (int h = 0; h < Hkv; ++h) {
        for (int g = 0; g * K_GROUP < T; ++g) {
            const int t0 = g * K_GROUP;
            const int t1 = t0 + K_GROUP < T ? t0 + K_GROUP : T;
            for (int d = 0; d < HEAD_DIM; ++d) {
                for (int t = t0; t < t1; ++t)
                    vals[t - t0] = bf16_bits_to_float(k[((size_t)t * Hkv + h) * HEAD_DIM + d]);
                float scale, zero, inv;
                group_stats(vals, t1 - t0, &scale, &zero, &inv);
                for (int t = t0; t < t1; ++t) {
                    const int c = quantize(vals[t - t0], zero, inv);
                    put_field(k_anc + plane_row_offset(bt_row, Hkv, bt, h, t, 16 * A), d, A, c >> R);
                    put_field(k_res + plane_row_offset(bt_row, Hkv, bt, h, t, 16 * R), d, R,
                              c & ((1 << R) - 1));
                }
                const size_t km = (((size_t)b * Hkv + h) * n_groups_max + g) * HEAD_DIM + d;
                k_scale[km] = scale;
                k_zero[km] = zero;
            }
        }
        for (int t = 0; t < T; ++t) {
            for (int d = 0; d < HEAD_DIM; ++d)
                vals[d] = bf16_bits_to_float(v[((size_t)t * Hkv + h) * HEAD_DIM + d]);
            float scale, zero, inv;
            group_stats(vals, HEAD_DIM, &scale, &zero, &inv);
            for (int d = 0; d < HEAD_DIM; ++d) {
                const int c = quantize(vals[d], zero, inv);
                put_field(v_anc + plane_row_offset(bt_row, Hkv, bt, h, t, 16 * A), d, A, c >> R);
                put_field(v_res + plane_row_offset(bt_row, Hkv, bt, h, t, 16 * R), d, R,
                          c & ((1 << R) - 1));
            }
            const size_t vm = ((size_t)b * Hkv + h) * (size_t)max_tokens + t;
            v_scale[vm] = scale;
            v_zero[vm] = zero;
        }
    }
    return 0;
}

/* n_rows rows of anchors (16 A bytes each) and residuals (16 (8 - A)) ->
 * n_rows rows of 128 codes.  Returns 0, or -1. */
int oracle_merge_split(int A, size_t n_rows, const uint8_t *anc, const uint8_t *res, uint8_t *codes)
{
    if (!split_ok(A)) return -1;
    const int R = 8 - A;
    for (size_t r = 0; r < n_rows; ++r)
        for (int e = 0; e < HEAD_DIM; ++e)
            codes[r * HEAD_DIM + e] = (uint8_t)((get_field(anc + r * 16 * A, e, A) << R) |
                                                get_field(res + r * 16 * R, e, R));
    return 0;
}

/* Sequence b's K and V from the anchors alone as BF16 bits [T][Hkv][128].
 * Returns 0, or -1. */
int oracle_dequant_anchor_split(int A, int Hkv, int bt, int max_blocks, int max_tokens, int b, int T,
                                const int32_t *block_table, const uint8_t *k_anc,
                                const uint8_t *v_anc, const float *k_scale, const float *k_zero,
                                const float *v_scale, const float *v_zero, uint16_t *k_out,
                                uint16_t *v_out)
{
    if (!split_ok(A) || Hkv < 1 || T < 0 || T > max_tokens) return -1;
    const int R = 8 - A;
    const float half = (float)((1 << R) - 1) / 2.0f;
    const int32_t *bt_row = block_table + (size_t)b * (size_t)max_blocks;
    const int n_groups_max = (max_tokens + K_GROUP - 1) / K_GROUP;
    for (int t = 0; t < T; ++t)
        for (int h = 0; h < Hkv; ++h) {
            const size_t off = plane_row_offset(bt_row, Hkv, bt, h, t, 16 * A);
            const size_t vm = ((size_t)b * Hkv + h) * (size_t)max_tokens + t;
            for (int d = 0; d < HEAD_DIM; ++d) {
                const size_t km = (((size_t)b * Hkv + h) * n_groups_max + t / K_GROUP) * HEAD_DIM + d;
                const float qk = (float)(get_field(k_anc + off, d, A) << R) + half;
                const float qv = (float)(get_field(v_anc + off, d, A) << R) + half;
                const size_t o = ((size_t)t * Hkv + h) * HEAD_DIM + d;
                k_out[o] = float_to_bf16_rne(fmaf(qk, k_scale[km], k_zero[km]));
                v_out[o] = float_to_bf16_rne(fmaf(qv, v_scale[vm], v_zero[vm]));
            }
        }
    return 0;
}

/*
 * Anchor-phase decode over the A-bit anchors of a split width (Sec. 4.2
 * Anchor phase with the widths of Sec. 8): one query per sequence, as
 * oracle_anchor_decode, with each anchor standing for code 2^R a + (2^R - 1)/2
 * (R = 8 - A) dequantized in fp64 with the group's scale and zero.  Planes of
 * rows of 16 A bytes (the layout of oracle_encode_split).  A = 4 is the plain
 * anchor decode.  Returns 0, or -1.
 */
int oracle_anchor_decode_split(int A, int Hkv, int bt, int max_blocks, int max_tokens, int B,
                               int Hq, const int32_t *seq_lens,
                               const int32_t *block_table, const uint8_t *k_anc,
                               const uint8_t *v_anc, const float *k_scale,
                               const float *k_zero, const float *v_scale,
                               const float *v_zero, const uint16_t *q, double *out,
                               double *lse, const uint8_t *unit_mask, int nthreads)
{
    if (!split_ok(A)) return -1;
    attn_job J;
    memset(&J, 0, sizeof J);
    J.mode = 2;
    J.anchor_bits = A;
    J.Hkv = Hkv; J.bt = bt; J.max_blocks = max_blocks; J.max_tokens = max_tokens;
    J.B = B; J.Hq = Hq; J.nq = 1;
    J.seq_lens = seq_lens; J.block_table = block_table;
    J.k_plane = k_anc; J.v_plane = v_anc;
    J.k_scale = k_scale; J.k_zero = k_zero; J.v_scale = v_scale; J.v_zero = v_zero;
    J.q = q; J.out = out; J.lse = lse; J.unit_mask = unit_mask;
    J.nthreads = nthreads;
    return run_attention(&J);
}
