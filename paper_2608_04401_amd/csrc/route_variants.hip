// Routing variants: one WAVE per token, one lane per expert.
//
// Serves what the lane-per-token routing kernel does not: caps above 16 up to N (the
// uncapped "Elbow-N" routing is K = N), tail randomisation (Section 2.2: the experts after
// the elbow are replaced by experts drawn from outside the elbow's selection) and the elbow
// angle of Section 2.3.  Every lane knows its expert's exact rank in the order (logit
// descending, expert id ascending) -- the number of experts ahead of it, counted against
// the 64 logits broadcast one by one -- so the whole permutation is available and each
// output is written by the lane that owns it.
//
// Same arithmetic as the main routing kernel: u_i = exp(l_(i) - l_(0)), S = sum u, and the
// scaled deviation D_i = (1 - u_i) - x'_i (1 - u_min + eps S), whose first argmax over all
// ranks is the elbow index e (the definition's D times the positive (p_max - p_min + eps) S).
// The elbow point is (x'_e, p'_e) with p'_e = (1 - u_e) / (1 - u_min + eps S).
#include "common.h"

namespace elb {

namespace {

constexpr float kLog2eV = 1.4426950408889634f;

__device__ __forceinline__ float wave_sum(float x) {
#pragma unroll
    for (int o = 1; o < kWave; o <<= 1) x += __shfl_xor(x, o);
    return x;  // every lane: the same bits (each step adds two equal-order partial sums)
}

// (value, index) pair reductions over the wave; ties: lower index
__device__ __forceinline__ void wave_argmax(float& v, int& i) {
#pragma unroll
    for (int o = 1; o < kWave; o <<= 1) {
        const float pv = __shfl_xor(v, o);
        const int pi = __shfl_xor(i, o);
        const bool take = pv > v || (pv == v && pi < i);
        v = take ? pv : v;
        i = take ? pi : i;
    }
}
__device__ __forceinline__ void wave_argmin(float& v, int& i) {
#pragma unroll
    for (int o = 1; o < kWave; o <<= 1) {
        const float pv = __shfl_xor(v, o);
        const int pi = __shfl_xor(i, o);
        const bool take = pv < v || (pv == v && pi < i);
        v = take ? pv : v;
        i = take ? pi : i;
    }
}

// value of lane `src` (wave-uniform)
__device__ __forceinline__ float lane_value(float x, int src) {
    return __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, x), src));
}

// first lane whose predicate holds (0 if none, which finite inputs never give)
__device__ __forceinline__ int first_lane(bool pred) {
    const uint64_t b = __ballot(pred);
    return b ? __builtin_ctzll(b) : 0;
}

__global__ __launch_bounds__(256) void route_wave_kernel(
    const float* __restrict__ logits, const float* __restrict__ rand, int64_t T, int N, int K,
    float eps, int mode, int renorm, int* __restrict__ kout, int* __restrict__ ids,
    float* __restrict__ wout, int* __restrict__ eout, float* __restrict__ thout) {
    const int lane = threadIdx.x & (kWave - 1);
    const int64_t t = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    if (t >= T) return;  // wave-uniform; no barriers in this kernel
    const bool real = lane < N;
    // canonical key (x + 0 turns -0 into +0); pads sort last
    const float key = real ? logits[t * N + lane] + 0.0f : -INFINITY;

    // rank of this expert in (key descending, id ascending)
    int rank = 0;
    for (int q = 0; q < N; ++q) {
        const float kq = lane_value(key, q);
        rank += (kq > key || (kq == key && q < lane)) ? 1 : 0;
    }
    if (!real) rank = kWave;  // never selected, never the elbow

    // u = exp(l - l_(0)); S; u_min = u of rank N - 1
    const float lmax = lane_value(key, first_lane(rank == 0));
    const float u = real ? __builtin_amdgcn_exp2f((key - lmax) * kLog2eV) : 0.f;
    const float S = wave_sum(u);
    const float umin = lane_value(u, first_lane(rank == N - 1));
    const float Rp = (1.0f - umin) + eps * S;
    const float xr = real ? (float)((double)rank / (double)(N - 1)) : INFINITY;
    // elbow: first argmax over the ranks of the scaled deviation (D_0 == 0 exactly)
    float D = real ? fmaf(-xr, Rp, 1.0f - u) : -INFINITY;
    int e = real ? rank : kWave;
    wave_argmax(D, e);
    const int k = (mode == ELB_MODE_TOPK) ? K : (e + 1 < K ? e + 1 : K);

    if (eout && lane == 0) eout[t] = e;
    if (thout && rank == e) {  // the elbow's lane: angle between (0,0), the point, (1,1)
        float th = 180.0f;  // no point below the chord: e = 0, taken as a straight line
        if (e > 0) {
            // atan2(|v1 x v2|, v1 . v2): well conditioned near 90 and 180 degrees, unlike acos
            const float pe = (1.0f - u) / Rp;
            const float v1x = -xr, v1y = -pe, v2x = 1.0f - xr, v2y = 1.0f - pe;
            const float dot = fmaf(v1x, v2x, v1y * v2y);
            const float crs = fmaf(v1x, v2y, -(v1y * v2x));
            th = atan2f(fabsf(crs), dot) * (180.0f / 3.14159265358979323846f);
        }
        thout[t] = th;
    }
    if (kout && lane == 0) kout[t] = k;
    if (!ids) return;

    // selection: ranks < k, then (tail randomisation) K - k experts from outside them,
    // those with the smallest draws in increasing order (ties: lower id)
    const bool sel = real && rank < k;
    int slot = sel ? rank : -1;
    if (rand) {
        const float draw = real ? rand[t * N + lane] : INFINITY;
        for (int j = k; j < K; ++j) {
            float v = (real && slot < 0) ? draw : INFINITY;
            int who = (real && slot < 0) ? lane : kWave;
            wave_argmin(v, who);
            if (lane == who) slot = j;
        }
    }
    float denom = S;
    if (renorm) denom = wave_sum(slot >= 0 ? u : 0.f);
    if (slot >= 0) {
        ids[t * K + slot] = lane;
        wout[t * K + slot] = u / denom;
    }
    if (!rand && lane >= k && lane < K) {  // empty slots
        ids[t * K + lane] = -1;
        wout[t * K + lane] = 0.f;
    }
}

}  // namespace

hipError_t launch_route_wave(const float* logits, const float* rand, int64_t T, int N,
                             const elb_route_params& p, int* k, int* ids, float* w, int* e,
                             float* theta, hipStream_t s) {
    if (T == 0) return hipSuccess;
    ProfileScope prof("route_wave", s);
    hipLaunchKernelGGL(route_wave_kernel, dim3((unsigned)((T + 3) / 4)), dim3(256), 0, s, logits,
                       rand, T, N, p.K, p.eps, p.mode, p.renormalize, k, ids, w, e, theta);
    return hipGetLastError();
}

}  // namespace elb
