// Routing kernel: softmax, per-token descending sort, Kneedle elbow, cap, weights.
//
// Method (Section 2, Section 2.1 and Appendix A.1 Algorithm 1 of the paper): per token,
// p = softmax(l); sort p in descending order; normalise the sorted curve to the unit square;
// D_i = deviation of point i from the reference line; e = argmax D; k = min(e + 1, K).
// The normalised curve runs from (0,0) to (1,1), as in the elbow-angle definition of
// Section 2.3: p'_i = (p_(0) - p_(i)) / (p_(0) - p_(N-1) + eps), x'_i = i / (N - 1).
//
// GPU design (CDNA4, wave64): one LANE per token.  A wave stages its 64 tokens' logits
// (64 * N contiguous floats) through LDS with coalesced loads, then every lane holds its
// token's N values in registers and sorts them with a compile-time odd-even merge network
// (all register indices are constants), so no cross-lane traffic is needed.
//
// Arithmetic differs from the definition only by positive scaling and the sum's
// cancellation, which leave the argmax unchanged:
//   u_i = exp(l_(i) - l_(0)) (so p_(i) = u_i / S, S = sum u), and
//   D_i * (p_max - p_min + eps) * S = (1 - u_i) - x'_i * (1 - u_min + eps * S).
// The sort key is the fp32 logit itself (softmax is strictly increasing), with ties broken
// by the lower expert id, so the ids and their order never depend on exp/division rounding.
#include <utility>

#include "common.h"
#include "sortnet.h"

namespace elb {

namespace {

struct XTable {
    float x[ELB_MAX_EXPERTS];  // x'_i = i / (N - 1), correctly rounded; x[N - 1] == 1
};

constexpr float kLog2e = 1.4426950408889634f;

template <int NP>
struct NetHolder {
    static constexpr OddEvenMergeNet<NP> net{};
};

// One comparator of the network: (v, id) pairs ordered by larger logit, then lower id.
template <int NP, int Q>
__device__ __forceinline__ void compare_exchange(float* v, int* id) {
    constexpr int a = NetHolder<NP>::net.a[Q];
    constexpr int b = NetHolder<NP>::net.b[Q];
    const bool sw = (v[b] > v[a]) || (v[b] == v[a] && id[b] < id[a]);
    const float va = sw ? v[b] : v[a];
    const float vb = sw ? v[a] : v[b];
    const int ia = sw ? id[b] : id[a];
    const int ib = sw ? id[a] : id[b];
    v[a] = va;
    v[b] = vb;
    id[a] = ia;
    id[b] = ib;
}

// The whole network as straight-line code (a fold over the comparator indices), so every
// register index is a compile-time constant regardless of loop-unrolling heuristics.
template <int NP, int... Q>
__device__ __forceinline__ void sort_desc(float* v, int* id, std::integer_sequence<int, Q...>) {
    (compare_exchange<NP, Q>(v, id), ...);
}

template <int NP>
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

    // ---- stage the wave's rows (contiguous in memory) through LDS, coalesced ----
    const float* src = logits + t0 * N;
    if (N == NP && vec4) {
        const int total4 = rows * (NP / 4);
        for (int i = lane; i < total4; i += kWave) {
            const float4 q = reinterpret_cast<const float4*>(src)[i];
            const int r = i / (NP / 4);
            const int c = (i % (NP / 4)) * 4;
            float* dst = tile + r * LD + c;
            dst[0] = q.x;
            dst[1] = q.y;
            dst[2] = q.z;
            dst[3] = q.w;
        }
    } else {
        const int total = rows * N;
        for (int i = lane; i < total; i += kWave) {
            const int r = i / N;
            tile[r * LD + (i - r * N)] = src[i];
        }
    }
    __syncthreads();
    if (lane >= rows) return;  // no barrier follows

    // ---- load the token's logits; pads (c >= N) sort last ----
    float v[NP];
    int id[NP];
#pragma unroll
    for (int c = 0; c < NP; ++c) {
        v[c] = (c < N) ? tile[lane * LD + c] : -INFINITY;
        id[c] = c;
    }

    // ---- descending sort of (logit, id): larger logit first, then lower id ----
    sort_desc<NP>(v, id, std::make_integer_sequence<int, NetHolder<NP>::net.n>{});

    // ---- u_i = exp(l_(i) - l_(0)) in place; S = sum u; u_min = u_(N-1) ----
    const float lmax = v[0];
    float S = 0.f;
    float umin = 0.f;
#pragma unroll
    for (int i = 0; i < NP; ++i) {
        if (i < N) {
            const float u = __builtin_amdgcn_exp2f((v[i] - lmax) * kLog2e);
            v[i] = u;
            S += u;
            if (i == N - 1) umin = u;
        }
    }

    int k = K;
    if (mode == ELB_MODE_ELBOW) {
        // scaled deviation: (1 - u_i) - x'_i * (1 - u_min + eps * S); D_0 == 0 exactly
        const float Rp = (1.0f - umin) + eps * S;
        float best = 0.f;
        int e = 0;
#pragma unroll
        for (int i = 1; i < NP; ++i) {
            if (i < N) {
                const float Di = fmaf(-xt.x[i], Rp, 1.0f - v[i]);
                if (Di > best) {  // strict: the first index wins ties
                    best = Di;
                    e = i;
                }
            }
        }
        k = e + 1 < K ? e + 1 : K;
    }

    float denom = S;
    if (renorm) {
        float sel = 0.f;
#pragma unroll
        for (int j = 0; j < ELB_MAX_K && j < NP; ++j)
            if (j < k) sel += v[j];
        denom = sel;
    }
    const float inv = 1.0f / denom;
    const int64_t t = t0 + lane;
    kout[t] = k;
#pragma unroll
    for (int j = 0; j < ELB_MAX_K && j < NP; ++j) {
        if (j < K) {
            const bool on = j < k;
            ids[t * K + j] = on ? id[j] : -1;
            wout[t * K + j] = on ? v[j] * inv : 0.f;
        }
    }
}

template <int NP>
hipError_t launch_np(const float* logits, int64_t T, int N, const elb_route_params& p, int* k,
                     int* ids, float* w, hipStream_t s) {
    XTable xt;
    for (int i = 0; i < ELB_MAX_EXPERTS; ++i)
        xt.x[i] = (i < N) ? (float)((double)i / (double)(N - 1)) : 0.f;
    const int64_t waves = (T + kWave - 1) / kWave;
    const unsigned blocks = (unsigned)((waves + 3) / 4);
    const int vec4 = ((uintptr_t)logits % 16) == 0;
    ProfileScope prof("route", s);
    hipLaunchKernelGGL(route_kernel<NP>, dim3(blocks), dim3(256), 0, s, logits, T, N, p.K,
                       p.eps, p.mode, p.renormalize, vec4, xt, k, ids, w);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_route(const float* logits, int64_t T, int N, const elb_route_params& p,
                        int* k, int* ids, float* w, hipStream_t s) {
    if (T == 0) return hipSuccess;
    if (N <= 8) return launch_np<8>(logits, T, N, p, k, ids, w, s);
    if (N <= 16) return launch_np<16>(logits, T, N, p, k, ids, w, s);
    if (N <= 32) return launch_np<32>(logits, T, N, p, k, ids, w, s);
    return launch_np<64>(logits, T, N, p, k, ids, w, s);
}

}  // namespace elb
