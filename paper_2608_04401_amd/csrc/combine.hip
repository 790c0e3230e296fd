// Weighted combine of the expert outputs back to token order (the MoE output is the
// routing-weighted sum over the token's selected experts, Section 2):
//   y[t] = [residual[t] +] sum_{j < k_t} w[t, j] * Y[inv[t, j]]   (no inv: Y[t K + j])
// summed in rank order j = 0, 1, ... with fp32 accumulation (deterministic; no atomics).
// y may alias residual (each element is read, then written, by the same thread).
// One block per token; each thread owns 8 (bf16) or 4 (fp32) consecutive columns, so every
// expert row is read with 16-byte coalesced loads.  The token's slots are taken eight at a
// time: their rows and weights first, then all eight row loads at once, then the FMAs in rank
// order, so a block waits for memory once per eight experts instead of twice per expert.
#include "common.h"

namespace elb {

namespace {

// Slots j0 .. j0 + 7 of token t: the row of Y each one adds (-1 past k_t) and its weight.
// t and K are block-uniform, so these are scalar loads; a whole group of eight is loaded
// with two 32-byte loads at once (no per-slot branch between dependent loads), and only a
// group that would run past the token's K slots is loaded slot by slot.
__device__ __forceinline__ void slot_group(const int* __restrict__ inv,
                                           const float* __restrict__ w, int64_t t, int K, int j0,
                                           int kt, int64_t (&r)[8], float (&wj)[8]) {
    const int64_t base = t * K + j0;
    int iv[8];
    float wv[8];
    if (j0 + 8 <= K) {
        if (inv) {
#pragma unroll
            for (int q = 0; q < 8; ++q) iv[q] = inv[base + q];
        }
#pragma unroll
        for (int q = 0; q < 8; ++q) wv[q] = w[base + q];
    } else {
#pragma unroll
        for (int q = 0; q < 8; ++q) {
            const bool in = j0 + q < K;
            iv[q] = (inv && in) ? inv[base + q] : 0;
            wv[q] = in ? w[base + q] : 0.f;
        }
    }
#pragma unroll
    for (int q = 0; q < 8; ++q) {
        const bool use = j0 + q < kt;
        r[q] = use ? (inv ? (int64_t)iv[q] : base + q) : -1;
        wj[q] = use ? wv[q] : 0.f;
    }
}

// NT: the rows are loaded with the non-temporal hint (chosen when Y is larger than the
// last-level cache, so that it streams from HBM; a smaller Y that the down GEMM has just
// written is read faster with plain loads)
template <bool NT>
__global__ __launch_bounds__(256) void combine_bf16(const bf16_t* __restrict__ Y,
                                                    const int* __restrict__ k,
                                                    const int* __restrict__ inv,
                                                    const float* __restrict__ w,
                                                    const bf16_t* residual,
                                                    int64_t T, int d, int K, bf16_t* y) {
    const int64_t t = blockIdx.x;
    const int kt = k[t] < K ? k[t] : K;  // block-uniform
    for (int c = threadIdx.x * 8; c < d; c += 256 * 8) {
        float acc[8];
        if (residual) {
            const uint4 q = *reinterpret_cast<const uint4*>(residual + t * d + c);
            const bf16_t* h = reinterpret_cast<const bf16_t*>(&q);
#pragma unroll
            for (int i = 0; i < 8; ++i) acc[i] = bf16_to_f32(h[i]);
        } else {
#pragma unroll
            for (int i = 0; i < 8; ++i) acc[i] = 0.f;
        }
        for (int j0 = 0; j0 < kt; j0 += 8) {
            int64_t r[8];
            float wj[8];
            slot_group(inv, w, t, K, j0, kt, r, wj);
            u32x4_t yq[8];
#pragma unroll
            for (int q = 0; q < 8; ++q) {
                const u32x4_t* const src = reinterpret_cast<const u32x4_t*>(Y + r[q] * d + c);
                yq[q] = r[q] < 0 ? u32x4_t{0u, 0u, 0u, 0u}
                        : NT     ? __builtin_nontemporal_load(src)
                                 : *src;
            }
#pragma unroll
            for (int q = 0; q < 8; ++q) {
                if (r[q] < 0) continue;  // slots past k_t, and dropped ones, add nothing
                const bf16_t* h = reinterpret_cast<const bf16_t*>(&yq[q]);
#pragma unroll
                for (int i = 0; i < 8; ++i) acc[i] = fmaf(wj[q], bf16_to_f32(h[i]), acc[i]);
            }
        }
        uint4 o;
        bf16_t* ob = reinterpret_cast<bf16_t*>(&o);
#pragma unroll
        for (int i = 0; i < 8; ++i) ob[i] = f32_to_bf16(acc[i]);
        *reinterpret_cast<uint4*>(y + t * d + c) = o;
    }
}

__global__ __launch_bounds__(256) void combine_f32(const float* __restrict__ Y,
                                                   const int* __restrict__ k,
                                                   const int* __restrict__ inv,
                                                   const float* __restrict__ w,
                                                   const float* residual,
                                                   int64_t T, int d, int K, float* y) {
    const int64_t t = blockIdx.x;
    const int kt = k[t] < K ? k[t] : K;  // block-uniform
    for (int c = threadIdx.x * 4; c < d; c += 256 * 4) {
        float4 acc = residual ? *reinterpret_cast<const float4*>(residual + t * d + c)
                              : make_float4(0.f, 0.f, 0.f, 0.f);
        for (int j0 = 0; j0 < kt; j0 += 8) {
            int64_t r[8];
            float wj[8];
            slot_group(inv, w, t, K, j0, kt, r, wj);
            float4 yq[8];
#pragma unroll
            for (int q = 0; q < 8; ++q)
                yq[q] = r[q] >= 0 ? *reinterpret_cast<const float4*>(Y + r[q] * d + c)
                                  : make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
            for (int q = 0; q < 8; ++q) {
                if (r[q] < 0) continue;
                acc.x = fmaf(wj[q], yq[q].x, acc.x);
                acc.y = fmaf(wj[q], yq[q].y, acc.y);
                acc.z = fmaf(wj[q], yq[q].z, acc.z);
                acc.w = fmaf(wj[q], yq[q].w, acc.w);
            }
        }
        *reinterpret_cast<float4*>(y + t * d + c) = acc;
    }
}

}  // namespace

hipError_t launch_combine(const void* Y, const int* k, const int* inv, const float* w,
                          const void* residual, int64_t T, int d, int K, int dtype, void* y,
                          hipStream_t s) {
    if (T == 0) return hipSuccess;
    if (dtype == ELB_BF16) {
        ProfileScope prof("combine_bf16", s);
        // Y holds at most T K rows of d bf16 values
        const bool nt = (double)T * K * d * 2 > (double)kLastLevelCacheBytes;
        if (nt)
            ELB_LAUNCH(combine_bf16<true>, dim3((unsigned)T), dim3(256), 0, s, (const bf16_t*)Y,
                       k, inv, w, (const bf16_t*)residual, T, d, K, (bf16_t*)y);
        else
            ELB_LAUNCH(combine_bf16<false>, dim3((unsigned)T), dim3(256), 0, s,
                       (const bf16_t*)Y, k, inv, w, (const bf16_t*)residual, T, d, K,
                       (bf16_t*)y);
    } else {
        ProfileScope prof("combine_f32", s);
        ELB_LAUNCH(combine_f32, dim3((unsigned)T), dim3(256), 0, s, (const float*)Y, k,
                           inv, w, (const float*)residual, T, d, K, (float*)y);
    }
    return hipGetLastError();
}

}  // namespace elb
