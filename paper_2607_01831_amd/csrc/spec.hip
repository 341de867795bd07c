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

}  // namespace

int spec_accept_chunks(int vocab) { return (vocab + kChunk - 1) / kChunk; }

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
