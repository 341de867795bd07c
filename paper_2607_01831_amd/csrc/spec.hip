// Greedy acceptance of speculative tokens (Sec. 4.3): the verification pass
// gives the target model's scores at the k draft positions and the one after
// them; the drafts are kept up to the first position where the target's own
// choice (its highest score, the lowest vocabulary index among equal scores)
// differs, and that choice corrects the divergence (or, when all k drafts are
// kept, is the bonus token).
//
// Two passes, both HBM-bound on the (k + 1) x V scores of a sequence:
//  1. argmax_chunk_kernel -- grid (vocabulary chunk, position, sequence): the
//     best (score, index) of 4096 vocabulary entries, 16-byte loads when the
//     rows allow it, a shuffle tree inside each wavefront and LDS across the
//     four;
//  2. accept_kernel -- one wavefront per sequence: positions in order, each
//     reducing its chunks' partials, until the first disagreement.
//
// Acceptance of sampled drafts (the speculative-sampling form of the same
// rule): draft i, token x, is kept when u_i q_i(x) <= p_i(x) (kept with
// probability min(1, p/q)); at the first draft not kept, n, the next token is
// drawn from max(p_n - q_n, 0), and when all are kept the bonus from p_k.
// The draw is an exact inverse-CDF draw: weights w_v = floor(r_v 2^40) with
// r_v clamped to [0, 1] (NaN 0), S = sum w, U = floor(u_k 2^32),
// t = floor(S U / 2^32), the token the first whose inclusive prefix of w
// exceeds t; a zero residual falls back to p_n, and an all-zero p_n gives
// -1.
// Two passes, like the greedy one: sample_chunk_kernel sums the integer
// weights of every (chunk, position) of the rows, sample_pick_kernel tests
// the drafts and locates t through the chunk sums and then one chunk.
#include "lynx_internal.h"

#include <limits.h>
#include <math.h>

namespace lynx {
namespace {

constexpr int kThreads = 256;
constexpr int kChunk = 4096;  // vocabulary entries per workgroup of pass 1

// (v, i) beats (bv, bi): a higher score, or the same score at a lower index.
// A NaN score never wins.
__device__ __forceinline__ bool better(float v, int i, float bv, int bi) {
    return v > bv || (v == bv && i < bi);
}

__device__ __forceinline__ void wave_best(float &bv, int &bi) {
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) {
        const float ov = __shfl_xor(bv, off);
        const int oi = __shfl_xor(bi, off);
        if (better(ov, oi, bv, bi)) {
            bv = ov;
            bi = oi;
        }
    }
}

__global__ __launch_bounds__(kThreads) void argmax_chunk_kernel(const float *__restrict__ logits,
                                                                int V, int n_chunks, int vec4,
                                                                float *part_v, int *part_i) {
    const int chunk = blockIdx.x;
    const int pos = blockIdx.y;
    const int b = blockIdx.z;
    const int tid = threadIdx.x;
    const float *row = logits + ((size_t)b * gridDim.y + pos) * (size_t)V;
    const int lo = chunk * kChunk;
    const int hi = min(V, lo + kChunk);
    float bv = -INFINITY;
    int bi = INT_MAX;
    if (vec4) {
        // V % 4 == 0 and 16-byte rows: every float4 lies inside [lo, hi)
        for (int e = lo + 4 * tid; e < hi; e += 4 * kThreads) {
            const float4 x = *reinterpret_cast<const float4 *>(row + e);
            if (better(x.x, e, bv, bi)) { bv = x.x; bi = e; }
            if (better(x.y, e + 1, bv, bi)) { bv = x.y; bi = e + 1; }
            if (better(x.z, e + 2, bv, bi)) { bv = x.z; bi = e + 2; }
            if (better(x.w, e + 3, bv, bi)) { bv = x.w; bi = e + 3; }
        }
    } else {
        for (int e = lo + tid; e < hi; e += kThreads) {
            const float x = row[e];
            if (better(x, e, bv, bi)) { bv = x; bi = e; }
        }
    }
    wave_best(bv, bi);
    __shared__ float s_v[kThreads / 64];
    __shared__ int s_i[kThreads / 64];
    if ((tid & 63) == 0) {
        s_v[tid >> 6] = bv;
        s_i[tid >> 6] = bi;
    }
    __syncthreads();
    if (tid == 0) {
        for (int w = 1; w < kThreads / 64; ++w)
            if (better(s_v[w], s_i[w], bv, bi)) {
                bv = s_v[w];
                bi = s_i[w];
            }
        const size_t p = ((size_t)b * gridDim.y + pos) * n_chunks + chunk;
        part_v[p] = bv;
        part_i[p] = bi;
    }
}

__global__ __launch_bounds__(64) void accept_kernel(const float *part_v, const int *part_i, int k,
                                                    int n_chunks, const int32_t *drafts,
                                                    int32_t *accepted, int32_t *next_token) {
    const int b = blockIdx.x;
    const int lane = threadIdx.x;
    int n = k, next = 0;
    for (int pos = 0; pos <= k; ++pos) {
        const size_t p0 = ((size_t)b * (k + 1) + pos) * n_chunks;
        float bv = -INFINITY;
        int bi = INT_MAX;
        for (int c = lane; c < n_chunks; c += 64)
            if (better(part_v[p0 + c], part_i[p0 + c], bv, bi)) {
                bv = part_v[p0 + c];
                bi = part_i[p0 + c];
            }
        wave_best(bv, bi);  // every lane holds the position's choice
        if (pos == k || bi != drafts[(size_t)b * k + pos]) {
            n = pos;
            next = bi;
            break;  // uniform across the wavefront
        }
    }
    if (lane == 0) {
        accepted[b] = n;
        next_token[b] = next;
    }
}

__device__ __forceinline__ uint64_t sample_weight(float r) {
    r = r > 0.0f ? r : 0.0f;  // NaN and negatives count 0
    r = r < 1.0f ? r : 1.0f;
    return (uint64_t)(r * 1099511627776.0f);  // 2^40: exact scaling, then truncation
}

__device__ __forceinline__ uint32_t sample_uniform(float u) {
    const float s = u * 4294967296.0f;  // 2^32
    if (!(s > 0.0f)) return 0u;
    if (s >= 4294967296.0f) return 0xFFFFFFFFu;
    return (uint32_t)s;
}

__device__ __forceinline__ uint64_t block_sum_u64(uint64_t x, uint64_t *s_wave) {
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) x += __shfl_xor(x, off);
    const int w = threadIdx.x >> 6;
    __syncthreads();  // s_wave may still be read from a previous use
    if ((threadIdx.x & 63) == 0) s_wave[w] = x;
    __syncthreads();
    uint64_t t = 0;
    for (int j = 0; j < kThreads / 64; ++j) t += s_wave[j];
    return t;
}

// Exclusive prefix of x over the workgroup's threads in thread order, and the
// total.
__device__ __forceinline__ uint64_t block_scan_u64(uint64_t x, uint64_t *s_wave, uint64_t &total) {
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    uint64_t incl = x;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
        const uint64_t y = __shfl_up(incl, off);
        if (lane >= off) incl += y;
    }
    __syncthreads();
    if (lane == 63) s_wave[w] = incl;
    __syncthreads();
    uint64_t pre = incl - x;
    total = 0;
    for (int j = 0; j < kThreads / 64; ++j) {
        if (j < w) pre += s_wave[j];
        total += s_wave[j];
    }
    return pre;
}

// Pass 1 of the sampled acceptance: per (chunk of 4096 entries, position,
// sequence) the sums of the integer weights of the residual p_i - q_i
// (p_k at the last position) and of p_i alone (the fall-back draw).  Sums are
// integers, so the order of the additions does not matter.
__global__ __launch_bounds__(kThreads) void sample_chunk_kernel(const float *__restrict__ p,
                                                                const float *__restrict__ q, int k,
                                                                int V, int n_chunks, int vec4,
                                                                uint64_t *ws) {
    const int chunk = blockIdx.x, i = blockIdx.y, b = blockIdx.z;
    const int tid = threadIdx.x;
    const float *prow = p + ((size_t)b * (k + 1) + i) * V;
    const float *qrow = i < k ? q + ((size_t)b * k + i) * V : nullptr;
    const int lo = chunk * kChunk, hi = min(V, lo + kChunk);
    uint64_t sr = 0, sp = 0;
    if (vec4) {
        for (int e = lo + 4 * tid; e < hi; e += 4 * kThreads) {
            const float4 a = *reinterpret_cast<const float4 *>(prow + e);
            float4 c = make_float4(0.f, 0.f, 0.f, 0.f);
            if (qrow) c = *reinterpret_cast<const float4 *>(qrow + e);
            sp += sample_weight(a.x) + sample_weight(a.y) + sample_weight(a.z) + sample_weight(a.w);
            if (qrow)
                sr += sample_weight(a.x - c.x) + sample_weight(a.y - c.y) + sample_weight(a.z - c.z) +
                      sample_weight(a.w - c.w);
        }
    } else {
        for (int e = lo + tid; e < hi; e += kThreads) {
            const float a = prow[e];
            sp += sample_weight(a);
            if (qrow) sr += sample_weight(a - qrow[e]);
        }
    }
    __shared__ uint64_t s_wave[kThreads / 64];
    sp = block_sum_u64(sp, s_wave);
    sr = block_sum_u64(sr, s_wave);
    if (tid == 0) {
        const size_t o = (((size_t)b * (k + 1) + i) * n_chunks + chunk) * 2;
        ws[o] = qrow ? sr : sp;
        ws[o + 1] = sp;
    }
}

// Pass 2: one workgroup per sequence.  Wavefront 0 tests the drafts (one
// ballot per 64); the row of the first draft not kept (or the bonus row)
// gives S from its chunk sums, falling back to the p-only sums when the
// residual is all 0; a scan over the chunk sums finds the chunk that holds
// t, and a scan over that chunk's 16-entry thread slices the slice; its
// thread walks it.
__global__ __launch_bounds__(kThreads) void sample_pick_kernel(
    const float *__restrict__ p, const float *__restrict__ q, const int32_t *__restrict__ drafts,
    const float *__restrict__ u, int k, int V, int n_chunks, const uint64_t *__restrict__ ws,
    int32_t *accepted, int32_t *next_token) {
    const int b = blockIdx.x;
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    __shared__ int s_n, s_tok, s_chunk, s_fallback;
    __shared__ uint64_t s_t;
    __shared__ uint64_t s_wave[kThreads / 64];
    const float *pb = p + (size_t)b * (k + 1) * V;
    const float *qb = q + (size_t)b * k * V;
    const float *ub = u + (size_t)b * (k + 1);
    if (tid < 64) {
        int n = k;
        for (int i0 = 0; i0 < k; i0 += 64) {
            const int i = i0 + lane;
            bool stop = false;
            if (i < k) {
                const int x = drafts[(size_t)b * k + i];
                stop = x < 0 || x >= V || !(ub[i] * qb[(size_t)i * V + x] <= pb[(size_t)i * V + x]);
            }
            const uint64_t m = __ballot(stop);
            if (m) {  // uniform across the wavefront
                n = i0 + __ffsll((long long)m) - 1;
                break;
            }
        }
        if (lane == 0) {
            s_n = n;
            s_tok = -1;
            s_chunk = -1;
        }
    }
    __syncthreads();
    const int n = s_n;
    const uint64_t *cs = ws + ((size_t)b * (k + 1) + n) * n_chunks * 2;
    // thread slices of the chunk sums: ceil(n_chunks / 256) chunks each
    const int cper = (n_chunks + kThreads - 1) / kThreads;
    const int c0 = min(n_chunks, tid * cper), c1 = min(n_chunks, c0 + cper);
    for (int alt = 0; alt < 2; ++alt) {  // residual sums, then the p-only ones
        uint64_t mine = 0;
        for (int c = c0; c < c1; ++c) mine += cs[2 * c + alt];
        uint64_t S;
        const uint64_t pre = block_scan_u64(mine, s_wave, S);
        if (S > 0) {  // uniform
            const uint32_t U = sample_uniform(ub[k]);
            const uint64_t t = (S >> 32) * U + (((S & 0xFFFFFFFFull) * U) >> 32);
            if (mine > 0 && pre <= t && t - pre < mine) {
                uint64_t acc = pre;
                for (int c = c0; c < c1; ++c) {
                    const uint64_t x = cs[2 * c + alt];
                    if (t - acc < x) {
                        s_chunk = c;
                        s_t = t - acc;
                        s_fallback = alt;
                        break;
                    }
                    acc += x;
                }
            }
            break;
        }
        if (n == k) break;  // the bonus row's two sums are the same
    }
    __syncthreads();
    const int chunk = s_chunk;
    if (chunk >= 0) {  // uniform
        const uint64_t t = s_t;
        const float *prow = pb + (size_t)n * V;
        const float *qrow = (n < k && !s_fallback) ? qb + (size_t)n * V : nullptr;
        const int lo = chunk * kChunk, hi = min(V, lo + kChunk);
        constexpr int kSlice = kChunk / kThreads;  // 16 entries per thread, in order
        const int v0 = min(hi, lo + kSlice * tid), v1 = min(hi, v0 + kSlice);
        uint64_t mine = 0;
        for (int v = v0; v < v1; ++v) mine += sample_weight(qrow ? prow[v] - qrow[v] : prow[v]);
        uint64_t tot;
        const uint64_t pre = block_scan_u64(mine, s_wave, tot);
        if (mine > 0 && pre <= t && t - pre < mine) {
            uint64_t acc = pre;
            for (int v = v0; v < v1; ++v) {
                acc += sample_weight(qrow ? prow[v] - qrow[v] : prow[v]);
                if (acc > t) {
                    s_tok = v;
                    break;
                }
            }
        }
    }
    __syncthreads();
    if (tid == 0) {
        accepted[b] = n;
        next_token[b] = s_tok;
    }
}

}  // namespace

int spec_accept_chunks(int vocab) { return (vocab + kChunk - 1) / kChunk; }

hipError_t launch_spec_accept_sample(int B, int k, int vocab, const float *p, const float *q,
                                     const int32_t *drafts, const float *u, int32_t *accepted,
                                     int32_t *next_token, void *workspace, hipStream_t stream) {
    const int n_chunks = spec_accept_chunks(vocab);
    uint64_t *ws = reinterpret_cast<uint64_t *>(workspace);
    const int vec4 = (vocab % 4 == 0 && (reinterpret_cast<uintptr_t>(p) & 15u) == 0 &&
                      (reinterpret_cast<uintptr_t>(q) & 15u) == 0) ? 1 : 0;
    hipLaunchKernelGGL(sample_chunk_kernel, dim3(n_chunks, k + 1, B), dim3(kThreads), 0, stream, p, q, k,
                       vocab, n_chunks, vec4, ws);
    hipLaunchKernelGGL(sample_pick_kernel, dim3(B), dim3(kThreads), 0, stream, p, q, drafts, u, k, vocab,
                       n_chunks, ws, accepted, next_token);
    return hipGetLastError();
}

hipError_t launch_spec_accept_greedy(int B, int k, int vocab, const float *logits,
                                     const int32_t *drafts, int32_t *accepted,
                                     int32_t *next_token, void *workspace, hipStream_t stream) {
    const int n_chunks = spec_accept_chunks(vocab);
    float *part_v = reinterpret_cast<float *>(workspace);
    int *part_i = reinterpret_cast<int *>(part_v + (size_t)B * (k + 1) * n_chunks);
    const int vec4 = (vocab % 4 == 0 && (reinterpret_cast<uintptr_t>(logits) & 15u) == 0) ? 1 : 0;
    hipLaunchKernelGGL(argmax_chunk_kernel, dim3(n_chunks, k + 1, B), dim3(kThreads), 0, stream,
                       logits, vocab, n_chunks, vec4, part_v, part_i);
    hipLaunchKernelGGL(accept_kernel, dim3(B), dim3(64), 0, stream, part_v, part_i, k, n_chunks,
                       drafts, accepted, next_token);
    return hipGetLastError();
}

}  // namespace lynx
