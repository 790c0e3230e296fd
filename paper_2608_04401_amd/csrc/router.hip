// Router logits l = x W_r^T (Section 2: a learned router produces logits l(x) in R^N),
// fp32 accumulation and fp32 output.
//
// bf16: one block of 4 waves per 16 tokens; wave w owns experts [16w, 16w + 16) and runs
// v_mfma_f32_16x16x32_bf16 over the full d, reading its fragments straight from global
// memory (the 16 x d slice of x is shared by the 4 waves through L1/L2; W_r (N x d) stays in
// L2 across blocks).  N <= 64.
// fp32: one thread per (token, expert) dot product (the small fp32 configuration).
#include "common.h"

namespace elb {

namespace {

__global__ __launch_bounds__(256) void router_bf16(const bf16_t* __restrict__ x,
                                                   const bf16_t* __restrict__ Wr, int64_t T,
                                                   int d, int N, float* __restrict__ logits) {
    const int lane = threadIdx.x & 63;
    const int w = threadIdx.x >> 6;
    const int64_t t0 = (int64_t)blockIdx.x * 16;
    const int n0 = w * 16;
    if (n0 >= N) return;  // no barriers in this kernel
    const int l16 = lane & 15;
    const int kq = (lane >> 4) * 8;
    const int64_t ta = t0 + l16;
    const bool arow = ta < T;
    const bool brow = n0 + l16 < N;
    const bf16_t* ap = x + (arow ? ta : 0) * d + kq;
    const bf16_t* bp = Wr + (int64_t)(brow ? n0 + l16 : 0) * d + kq;
    const bf16x8_t zero = {};
    f32x4_t acc0 = {0.f, 0.f, 0.f, 0.f}, acc1 = {0.f, 0.f, 0.f, 0.f};
    int k0 = 0;
    for (; k0 + 64 <= d; k0 += 64) {
        bf16x8_t a0 = *reinterpret_cast<const bf16x8_t*>(ap + k0);
        bf16x8_t b0 = *reinterpret_cast<const bf16x8_t*>(bp + k0);
        bf16x8_t a1 = *reinterpret_cast<const bf16x8_t*>(ap + k0 + 32);
        bf16x8_t b1 = *reinterpret_cast<const bf16x8_t*>(bp + k0 + 32);
        if (!arow) { a0 = zero; a1 = zero; }
        if (!brow) { b0 = zero; b1 = zero; }
        acc0 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a0, b0, acc0, 0, 0, 0);
        acc1 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a1, b1, acc1, 0, 0, 0);
    }
    for (; k0 < d; k0 += 32) {
        bf16x8_t a0 = *reinterpret_cast<const bf16x8_t*>(ap + k0);
        bf16x8_t b0 = *reinterpret_cast<const bf16x8_t*>(bp + k0);
        if (!arow) a0 = zero;
        if (!brow) b0 = zero;
        acc0 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a0, b0, acc0, 0, 0, 0);
    }
    const int rq = (lane >> 4) * 4;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
        const int64_t t = t0 + rq + r;
        if (t < T && brow) logits[t * N + n0 + l16] = acc0[r] + acc1[r];
    }
}

__global__ __launch_bounds__(256) void router_f32(const float* __restrict__ x,
                                                  const float* __restrict__ Wr, int64_t T,
                                                  int d, int N, float* __restrict__ logits) {
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i >= T * N) return;
    const int64_t t = i / N;
    const int n = (int)(i - t * N);
    const float* a = x + t * d;
    const float* b = Wr + (int64_t)n * d;
    float acc = 0.f;
    for (int c = 0; c < d; ++c) acc = fmaf(a[c], b[c], acc);
    logits[i] = acc;
}

}  // namespace

hipError_t launch_router(const void* x, const void* Wr, int64_t T, int d, int N, int dtype,
                         float* logits, hipStream_t s) {
    if (T == 0) return hipSuccess;
    if (dtype == ELB_BF16) {
        ProfileScope prof("router_bf16", s);
        hipLaunchKernelGGL(router_bf16, dim3((unsigned)((T + 15) / 16)), dim3(256), 0, s,
                           (const bf16_t*)x, (const bf16_t*)Wr, T, d, N, logits);
    } else {
        ProfileScope prof("router_f32", s);
        hipLaunchKernelGGL(router_f32, dim3((unsigned)((T * N + 255) / 256)), dim3(256), 0, s,
                           (const float*)x, (const float*)Wr, T, d, N, logits);
    }
    return hipGetLastError();
}

}  // namespace elb
