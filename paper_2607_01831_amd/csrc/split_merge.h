// Split merge in the launch that produced the splits (gfx950): the last
// workgroup of a (sequence, kv head, row chunk) to store its partial merges
// every split's partial.  Shared by the decode kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include "lane_ops.h"
#include "lynx_internal.h"

namespace lynx {

constexpr int kMergeThreads = 256;  // threads of the merging workgroup that take part

// ---- fused split merge ----
// A workgroup stores its partial with agent-coherent (sc1) stores, waits for
// them, then counts in on its pair's counter; the pair's last arrival reads
// every partial back with agent-coherent loads.  Neither side needs a fence
// that writes back or invalidates a whole L2.
__device__ __forceinline__ uint16_t f32_to_bf16_rne(float f) {
    uint32_t u = __float_as_uint(f);
    if ((u & 0x7fffffffu) > 0x7f800000u) return 0x7fc0;  // NaN
    u += 0x7fffu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
}

// Reductions over the kP lanes of one row (kP = 64, 32 or 16 lanes aligned
// in the wavefront), on the permute paths (DPP, permlane swaps).
template <int kP>
__device__ __forceinline__ float row_max(float v) {
    v = row16_max(v);
    if (kP >= 32) {
        const auto r = __builtin_amdgcn_permlane16_swap(__float_as_int(v), __float_as_int(v), false, false);
        v = fmax2(__int_as_float(r[0]), __int_as_float(r[1]));
    }
    if (kP >= 64) {
        const auto r = __builtin_amdgcn_permlane32_swap(__float_as_int(v), __float_as_int(v), false, false);
        v = fmax2(__int_as_float(r[0]), __int_as_float(r[1]));
    }
    return v;
}
template <int kP>
__device__ __forceinline__ float row_sum(float v) {
    v = row16_sum(v);
    if (kP >= 32) {
        const auto r = __builtin_amdgcn_permlane16_swap(__float_as_int(v), __float_as_int(v), false, false);
        v = __int_as_float(r[0]) + __int_as_float(r[1]);
    }
    if (kP >= 64) {
        const auto r = __builtin_amdgcn_permlane32_swap(__float_as_int(v), __float_as_int(v), false, false);
        v = __int_as_float(r[0]) + __int_as_float(r[1]);
    }
    return v;
}

// Merge of the `live` split partials of `heads` query rows by one workgroup.
// ro / rml: buffer resources over the pair's partial outputs [heads][ws_splits]
// [128] and (max, sum) pairs [heads][ws_splits]; output row orow0 + r.
// Threads (row r, u < kP): thread u holds the (max, sum) of splits u and
// u + kP (live <= 2 kP), and as (split group sg, float4 column d4) the partial
// outputs of splits sg, sg + groups, ...  Every load of the first round is
// issued before any is used, without branches: a slot past the live splits
// or rows reads at an offset past the resource, which returns zeros.  The
// row's maximum and sum meet on the permute paths, the split weights (zero
// past the live splits) go through LDS, the groups' sums meet in LDS; the
// result is normalised, rounded to BF16 and written with the lse.
template <int GP, typename Args>
__device__ void merge_pair(const Args &a, __amdgpu_buffer_rsrc_t ro, __amdgpu_buffer_rsrc_t rml,
                           size_t orow0, int heads, int live, uint8_t *lds) {
    constexpr int kP = kMergeThreads / GP;           // threads per row: 64, 32, 16
    constexpr int kGroups = kP >= 32 ? kP / 32 : 1;  // split groups per row
    constexpr int kCols = kP >= 32 ? 1 : 32 / kP;    // float4 columns per thread
    constexpr int kRound = 32 / kCols;               // partial outputs per column and round
    constexpr uint32_t kPast = 0x80000000u;          // an offset past any resource
    const int tid = threadIdx.x;
    const int r = tid / kP, u = tid % kP;
    const int sg = kP >= 32 ? u / 32 : 0;
    const bool row_live = r < heads;
    const uint32_t prow = (uint32_t)r * a.ws_splits;
    float *s_f = reinterpret_cast<float *>(lds);                     // [GP][2 kP] split weights
    float4 *s_acc = reinterpret_cast<float4 *>(s_f + GP * 2 * kP);   // [GP][kGroups][32]
    auto o_off = [&](int sp, int d4) {
        return (row_live && sp < live) ? ((prow + sp) * kHeadDim + 4 * d4) * 4 : kPast;
    };

    // round 0: (max, sum) of splits u, u + kP and the first partial outputs
    float2 ml[2];
#pragma unroll
    for (int j = 0; j < 2; ++j) {
        const int sp = u + j * kP;
        ml[j] = load8_agent(rml, (row_live && sp < live) ? (prow + sp) * 8 : kPast);
    }
    float4 v[kCols][kRound];
#pragma unroll
    for (int c = 0; c < kCols; ++c) {
        const int d4 = kP >= 32 ? u % 32 : u + kP * c;
#pragma unroll
        for (int i = 0; i < kRound; ++i) v[c][i] = load16_agent(ro, o_off(sg + kGroups * i, d4));
    }
    // the row's maximum, the split weights (zero past the live splits) and
    // the row's sum
    float m[2];
#pragma unroll
    for (int j = 0; j < 2; ++j) m[j] = u + j * kP < live ? ml[j].x : -INFINITY;
    const float M = row_max<kP>(fmax2(m[0], m[1]));
    float L = 0.0f;
#pragma unroll
    for (int j = 0; j < 2; ++j) {
        // a split with weight 0 contributes nothing (its output may be unset)
        const float f = m[j] == -INFINITY ? 0.0f : __builtin_amdgcn_exp2f(m[j] - M);
        L = fmaf(u + j * kP < live ? ml[j].y : 0.0f, f, L);  // a NaN sum (bad block id) stays NaN
        if (r < GP) s_f[r * 2 * kP + u + j * kP] = f;
    }
    L = row_sum<kP>(L);
    __syncthreads();
#pragma unroll
    for (int c = 0; c < kCols; ++c) {
        const int d4 = kP >= 32 ? u % 32 : u + kP * c;
        float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
        const float *fr = s_f + min(r, GP - 1) * 2 * kP;
        for (int i0 = 0; i0 * kGroups < live; i0 += kRound) {
            if (i0 > 0) {  // a later round (more than kRound splits per group)
#pragma unroll
                for (int i = 0; i < kRound; ++i) v[c][i] = load16_agent(ro, o_off(sg + kGroups * (i0 + i), d4));
            }
#pragma unroll
            for (int i = 0; i < kRound; ++i) {
                const int sp = min(sg + kGroups * (i0 + i), 2 * kP - 1);
                const float f = fr[sp];  // zero past the live splits
                acc.x = fmaf(v[c][i].x, f, acc.x);
                acc.y = fmaf(v[c][i].y, f, acc.y);
                acc.z = fmaf(v[c][i].z, f, acc.z);
                acc.w = fmaf(v[c][i].w, f, acc.w);
            }
        }
        if (r < GP) s_acc[(r * kGroups + sg) * 32 + d4] = acc;
    }
    __syncthreads();
#pragma unroll
    for (int c = 0; c < kCols; ++c) {
        const int d4 = kP >= 32 ? u % 32 : u + kP * c;
        if (row_live && sg == 0) {
            float4 O = s_acc[(r * kGroups) * 32 + d4];
#pragma unroll
            for (int g = 1; g < kGroups; ++g) {
                const float4 o = s_acc[(r * kGroups + g) * 32 + d4];
                O.x += o.x;
                O.y += o.y;
                O.z += o.z;
                O.w += o.w;
            }
            const bool nan = isnan(L);
            float res[4] = {O.x, O.y, O.z, O.w};
#pragma unroll
            for (int i = 0; i < 4; ++i) res[i] = nan ? NAN : (L > 0.0f ? res[i] / L : 0.0f);
            const uint32_t lo = f32_to_bf16_rne(res[0]) | ((uint32_t)f32_to_bf16_rne(res[1]) << 16);
            const uint32_t hi = f32_to_bf16_rne(res[2]) | ((uint32_t)f32_to_bf16_rne(res[3]) << 16);
            *reinterpret_cast<uint2 *>(a.out + (orow0 + r) * kHeadDim + 4 * d4) = make_uint2(lo, hi);
            if (a.lse && d4 == 0)
                a.lse[orow0 + r] = nan ? NAN : (L > 0.0f ? (M + log2f(L)) * 0.6931471805599453f : -INFINITY);
        }
    }
}

// Count in after this workgroup's partial stores (agent-coherent) are done:
// true in every thread of the last of `live` workgroups to arrive, which also
// resets the counter for the next call.  *flag is a __shared__ int.
__device__ __forceinline__ bool last_to_arrive(unsigned *ctr, int live, int *flag) {
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");  // this thread's partial stores are done
    __syncthreads();                                    // ... and every other thread's
    if (threadIdx.x == 0)
        *flag = __hip_atomic_fetch_add(ctr, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) ==
                (unsigned)(live - 1);
    __syncthreads();
    if (!*flag) return false;
    if (threadIdx.x == 0) __hip_atomic_store(ctr, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    return true;
}

}  // namespace lynx
