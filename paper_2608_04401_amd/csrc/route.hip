// Routing kernel: softmax, per-token descending sort, Kneedle elbow, cap, weights (the
// per-token arithmetic and its reading of Section 2, Section 2.1 and Appendix A.1
// Algorithm 1 are in route_lane.h).
//
// GPU design (CDNA4, wave64): one LANE per token.  A wave stages its 64 tokens' logits
// (64 * N contiguous floats) through LDS with coalesced loads, then every lane routes its
// token from its staged row.
#include "route_lane.h"

namespace elb {

namespace {

// FULL: N == NP, so every "position < N" test is static; KM: a bound on K (8 or 16)
template <int NP, bool FULL, int KMAX>
__global__ __launch_bounds__(256) void route_kernel(const float* __restrict__ logits, int64_t T,
                                                    int N, int K, float eps, int mode,
                                                    int renorm, int vec4, XTable xt,
                                                    int* __restrict__ kout,
                                                    int* __restrict__ ids,
                                                    float* __restrict__ wout) {
    constexpr int LD = NP + 1;  // padded row: lane t reads word t*LD + c, banks (t + c) % 64
    __shared__ float lds[4 * kWave * LD];
    const int lane = threadIdx.x & (kWave - 1);
    const int wv = threadIdx.x >> 6;
    const int64_t t0 = ((int64_t)blockIdx.x * 4 + wv) * kWave;
    float* tile = lds + wv * kWave * LD;
    int rows = 0;
    if (t0 < T) rows = (int)((T - t0) < kWave ? (T - t0) : kWave);

    stage_rows<NP, FULL>(logits + t0 * N, N, rows, vec4, tile, lane);
    __syncthreads();
    if (lane >= rows) return;  // no barrier follows

    route_token<NP, FULL, KMAX>(tile + lane * LD, N, K, eps, mode, renorm, xt, t0 + lane, kout,
                                ids, wout);
}

template <int NP, bool FULL, int KMAX>
hipError_t launch_np(const float* logits, int64_t T, int N, const elb_route_params& p, int* k,
                     int* ids, float* w, hipStream_t s) {
    const XTable xt = make_xtable(N);
    const int64_t waves = (T + kWave - 1) / kWave;
    const unsigned blocks = (unsigned)((waves + 3) / 4);
    const int vec4 = ((uintptr_t)logits % 16) == 0;
    ProfileScope prof("route", s);
    hipLaunchKernelGGL((route_kernel<NP, FULL, KMAX>), dim3(blocks), dim3(256), 0, s, logits, T, N, p.K,
                       p.eps, p.mode, p.renormalize, vec4, xt, k, ids, w);
    return hipGetLastError();
}

template <int KMAX>
hipError_t launch_k(const float* logits, int64_t T, int N, const elb_route_params& p, int* k,
                   int* ids, float* w, hipStream_t s) {
    switch (N) {
        case 8: return launch_np<8, true, KMAX>(logits, T, N, p, k, ids, w, s);
        case 16: return launch_np<16, true, KMAX>(logits, T, N, p, k, ids, w, s);
        case 32: return launch_np<32, true, KMAX>(logits, T, N, p, k, ids, w, s);
        case 64: return launch_np<64, true, KMAX>(logits, T, N, p, k, ids, w, s);
        default: break;
    }
    if (N < 8) return launch_np<8, false, KMAX>(logits, T, N, p, k, ids, w, s);
    if (N < 16) return launch_np<16, false, KMAX>(logits, T, N, p, k, ids, w, s);
    if (N < 32) return launch_np<32, false, KMAX>(logits, T, N, p, k, ids, w, s);
    return launch_np<64, false, KMAX>(logits, T, N, p, k, ids, w, s);
}

}  // namespace

hipError_t launch_route(const float* logits, int64_t T, int N, const elb_route_params& p,
                        int* k, int* ids, float* w, hipStream_t s) {
    if (T == 0) return hipSuccess;
    if (p.K <= 8) return launch_k<8>(logits, T, N, p, k, ids, w, s);
    if (p.K <= kLaneMaxK) return launch_k<kLaneMaxK>(logits, T, N, p, k, ids, w, s);
    return launch_route_pair(logits, nullptr, T, N, p, k, ids, w, nullptr, nullptr, s);
}

}  // namespace elb
