// Router logits l = x W_r^T (Section 2: a learned router produces logits l(x) in R^N),
// fp32 accumulation and fp32 output; and the router fused with the routing of its logits.
//
// bf16: one block of 4 waves per 16 tokens.  The 32-deep k-steps are dealt round-robin to
// the waves, so each wave reads a distinct quarter of the 16 x d slice of x (x is read once)
// and the matching columns of all N rows of W_r (which stays in L2 across blocks); each wave
// runs 4 v_mfma_f32_16x16x32_bf16 chains (16 experts each) with its loads four steps ahead
// of their use, and the 4 partial 16 x N tiles are summed in LDS in a fixed order.
// N <= 64, d % 32 == 0.
// fp32: one thread per (token, expert) dot product (the small fp32 configuration).
#include "route_lane.h"

namespace elb {

namespace {

constexpr int RW = 4;  // waves per router block

// The logits of tokens [t0, t0 + 16) and experts [16 g0, 16 (g0 + NG)) (NG groups of 16):
// each wave's partial sums over its k-steps go to part[w] (lane rows, expert columns
// 16 g + ..., g < NG); the caller sums the RW partial tiles.  Every logit is computed the same
// way whatever NG and g0 are (its own MFMA column, the same k-steps per wave, the same sum).
template <int NG>
__device__ __forceinline__ void router_partials(const bf16_t* __restrict__ x,
                                                const bf16_t* __restrict__ Wr, int64_t T,
                                                int d, int N, int64_t t0, int g0,
                                                float (&part)[RW][16][65]) {
    const int lane = threadIdx.x & 63;
    const int w = threadIdx.x >> 6;
    const int l16 = lane & 15;
    const int kq = (lane >> 4) * 8;
    const int64_t ta = t0 + l16;
    const bool arow = ta < T;
    const bf16_t* ap = x + (arow ? ta : 0) * d + kq;
    const bf16_t* bp[NG];
#pragma unroll
    for (int g = 0; g < NG; ++g) {
        const int n = 16 * (g0 + g) + l16;
        bp[g] = Wr + (int64_t)(n < N ? n : 0) * d + kq;
    }
    f32x4_t acc[NG];
#pragma unroll
    for (int g = 0; g < NG; ++g) acc[g] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    // wave w takes the 32-deep k-steps w, w + RW, w + 2 RW, ... (its steps j = 0, 1, ...).  A
    // ring of R register slots keeps R - 1 steps in flight: step j lives in slot j % R, and
    // while step j is multiplied, step j + R - 1 is loaded into the slot step j - 1 has just
    // freed.  Unrolled by R, so every slot index is a constant.
    constexpr int R = 5;
    const int nsteps = d / 32;
    const int mine = (nsteps - w + RW - 1) / RW;  // steps of this wave
    bf16x8_t ra[R], rb[R][NG];
    auto load = [&](int slot_j, bf16x8_t& a, bf16x8_t (&bb)[NG]) {
        const int k0 = (slot_j < mine ? w + RW * slot_j : 0) * 32;  // past the end: step 0
        a = *reinterpret_cast<const bf16x8_t*>(ap + k0);
#pragma unroll
        for (int g = 0; g < NG; ++g) bb[g] = *reinterpret_cast<const bf16x8_t*>(bp[g] + k0);
    };
    // rows past T and experts past N read row 0 and give logits that are never written
    auto mma = [&](const bf16x8_t& a, const bf16x8_t (&bb)[NG]) {
#pragma unroll
        for (int g = 0; g < NG; ++g)
            acc[g] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, bb[g], acc[g], 0, 0, 0);
    };
#pragma unroll
    for (int p = 0; p < R - 1; ++p) load(p, ra[p], rb[p]);
    int i = 0;
    for (; i + R <= mine; i += R) {
#pragma unroll
        for (int p = 0; p < R; ++p) {
            const int q = (p + R - 1) % R;
            load(i + p + R - 1, ra[q], rb[q]);
            mma(ra[p], rb[p]);
        }
    }
#pragma unroll
    for (int p = 0; p < R; ++p) {  // the last steps (fewer than R)
        if (i + p < mine) {
            const int q = (p + R - 1) % R;
            load(i + p + R - 1, ra[q], rb[q]);
            mma(ra[p], rb[p]);
        }
    }
    const int rq = (lane >> 4) * 4;
#pragma unroll
    for (int g = 0; g < NG; ++g)
#pragma unroll
        for (int r = 0; r < 4; ++r) part[w][rq + r][16 * g + l16] = acc[g][r];
}

// logit of output o of the block (token o / 64, expert o % 64): the RW partials summed in a
// fixed order (deterministic, the same bits in every kernel that uses it)
__device__ __forceinline__ float router_sum(const float (&part)[RW][16][65], int tr, int n) {
    float v = part[0][tr][n];
#pragma unroll
    for (int ww = 1; ww < RW; ++ww) v += part[ww][tr][n];
    return v;
}

// NG = 4: a block computes all N <= 64 experts of its 16 tokens; NG = 1 (few tokens): one
// block per (16 tokens, 16 experts) — blockIdx.y is the expert group — so the reads of W_r
// are spread over N / 16 times more compute units
template <int NG>
__global__ __launch_bounds__(64 * RW) void router_bf16(const bf16_t* __restrict__ x,
                                                      const bf16_t* __restrict__ Wr, int64_t T,
                                                      int d, int N, float* __restrict__ logits) {
    __shared__ float part[RW][16][65];  // per-wave partial logits (padded rows)
    const int64_t t0 = (int64_t)blockIdx.x * 16;
    const int g0 = (NG == 4) ? 0 : (int)blockIdx.y;
    router_partials<NG>(x, Wr, T, d, N, t0, g0, part);
    __syncthreads();
#pragma unroll
    for (int q = 0; q < 256 * NG / (64 * RW); ++q) {
        const int o = threadIdx.x + 64 * RW * q;
        const int tr = o / (16 * NG), nl = o % (16 * NG);
        const int64_t t = t0 + tr;
        const int n = 16 * g0 + nl;
        if (t < T && n < N) logits[t * N + n] = router_sum(part, tr, nl);
    }
}

// Router GEMM and routing fused: the block's 16 x N logits are summed into LDS and routed
// there, so the logits need not travel through HBM; they are written out only when `logits`
// is not null.  N = 64: 16 lanes per token (route_token_x16); otherwise one lane per token
// (route_token, the routing kernel's own per-token code).  Both give the routing kernel's
// bits.
template <int NP, bool FULL, int KMAX>
__global__ __launch_bounds__(64 * RW) void router_route_bf16(
    const bf16_t* __restrict__ x, const bf16_t* __restrict__ Wr, int64_t T, int d, int N,
    int K, float eps, int mode, int renorm, XTable xt, float* __restrict__ logits,
    int* __restrict__ kout, int* __restrict__ ids, float* __restrict__ wout) {
    __shared__ float part[RW][16][65];
    const int64_t t0 = (int64_t)blockIdx.x * 16;
    router_partials<4>(x, Wr, T, d, N, t0, 0, part);
    __syncthreads();
#pragma unroll
    for (int q = 0; q < 1024 / (64 * RW); ++q) {
        const int o = threadIdx.x + 64 * RW * q;
        const int tr = o >> 6, n = o & 63;
        const int64_t t = t0 + tr;
        const float v = router_sum(part, tr, n);
        part[0][tr][n] = v;  // the summed tile replaces partial 0 (same thread, same word)
        if (logits && t < T && n < N) logits[t * N + n] = v;
    }
    __syncthreads();
    if constexpr (NP == 64 && FULL) {
        // 16 lanes per token: wave w routes the block's tokens 4 w .. 4 w + 3
        const int tr = threadIdx.x >> 4;
        route_token_x16<KMAX>(&part[0][tr][0], K, eps, mode, renorm, xt, t0 + tr,
                              t0 + tr < T, kout, ids, wout);
    } else {
        if (threadIdx.x < 16 && t0 + threadIdx.x < T)
            route_token<NP, FULL, KMAX>(&part[0][threadIdx.x][0], N, K, eps, mode, renorm,
                                        xt, t0 + threadIdx.x, kout, ids, wout);
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

template <int NP, bool FULL, int KMAX>
void launch_rr(const void* x, const void* Wr, int64_t T, int d, int N,
               const elb_route_params& p, float* logits, int* k, int* ids, float* w,
               hipStream_t s) {
    hipLaunchKernelGGL((router_route_bf16<NP, FULL, KMAX>), dim3((unsigned)((T + 15) / 16)),
                       dim3(64 * RW), 0, s, (const bf16_t*)x, (const bf16_t*)Wr, T, d, N, p.K,
                       p.eps, p.mode, p.renormalize, make_xtable(N), logits, k, ids, w);
}

template <int KMAX>
void launch_rr_n(const void* x, const void* Wr, int64_t T, int d, int N,
                 const elb_route_params& p, float* logits, int* k, int* ids, float* w,
                 hipStream_t s) {
    switch (N) {
        case 8: return launch_rr<8, true, KMAX>(x, Wr, T, d, N, p, logits, k, ids, w, s);
        case 16: return launch_rr<16, true, KMAX>(x, Wr, T, d, N, p, logits, k, ids, w, s);
        case 32: return launch_rr<32, true, KMAX>(x, Wr, T, d, N, p, logits, k, ids, w, s);
        case 64: return launch_rr<64, true, KMAX>(x, Wr, T, d, N, p, logits, k, ids, w, s);
        default: break;
    }
    if (N < 8) return launch_rr<8, false, KMAX>(x, Wr, T, d, N, p, logits, k, ids, w, s);
    if (N < 16) return launch_rr<16, false, KMAX>(x, Wr, T, d, N, p, logits, k, ids, w, s);
    if (N < 32) return launch_rr<32, false, KMAX>(x, Wr, T, d, N, p, logits, k, ids, w, s);
    return launch_rr<64, false, KMAX>(x, Wr, T, d, N, p, logits, k, ids, w, s);
}

}  // namespace

bool router_route_fusable(int dtype, int K) { return dtype == ELB_BF16 && K <= kLaneMaxK; }

hipError_t launch_router_route(const void* x, const void* Wr, int64_t T, int d, int N,
                               const elb_route_params& p, float* logits, int* k, int* ids,
                               float* w, hipStream_t s) {
    if (T == 0) return hipSuccess;
    ProfileScope prof("router_route_bf16", s);
    if (p.K <= 8) launch_rr_n<8>(x, Wr, T, d, N, p, logits, k, ids, w, s);
    else launch_rr_n<kLaneMaxK>(x, Wr, T, d, N, p, logits, k, ids, w, s);
    return hipGetLastError();
}

hipError_t launch_router(const void* x, const void* Wr, int64_t T, int d, int N, int dtype,
                         float* logits, hipStream_t s) {
    if (T == 0) return hipSuccess;
    if (dtype == ELB_BF16) {
        ProfileScope prof("router_bf16", s);
        if (T <= kSmallBatch)
            hipLaunchKernelGGL(router_bf16<1>, dim3((unsigned)((T + 15) / 16), (unsigned)((N + 15) / 16)),
                               dim3(64 * RW), 0, s, (const bf16_t*)x, (const bf16_t*)Wr, T, d,
                               N, logits);
        else
            hipLaunchKernelGGL(router_bf16<4>, dim3((unsigned)((T + 15) / 16)), dim3(64 * RW), 0,
                               s, (const bf16_t*)x, (const bf16_t*)Wr, T, d, N, logits);
    } else {
        ProfileScope prof("router_f32", s);
        hipLaunchKernelGGL(router_f32, dim3((unsigned)((T * N + 255) / 256)), dim3(256), 0, s,
                           (const float*)x, (const float*)Wr, T, d, N, logits);
    }
    return hipGetLastError();
}

}  // namespace elb
