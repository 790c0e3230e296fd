// Routing kernel: softmax, per-token descending sort, Kneedle elbow, cap, weights (the
// per-token arithmetic and its reading of Section 2, Section 2.1 and Appendix A.1
// Algorithm 1 are in route_lane.h).
//
// GPU design (CDNA4, wave64): one LANE per token; a wave owns 64 consecutive tokens.
//  - route_dma_kernel (N = 16, 32, 64, 16-byte aligned logits): the wave's 64 N logits are
//    copied straight from HBM into its LDS tile (global_load_lds_dwordx4, no registers) in
//    two parts of N / 2 columns each (whole 128-byte lines of every row), issued at once;
//    each lane sorts its row's first half as soon as it has landed (the sorting network run
//    in part order, sortnet.h PhasedNet) while the second is still in flight.  The tile is
//    swizzled so that 16 lanes reading their own rows hit 16 distinct bank groups.  Each
//    lane keeps its ids and w in registers and stores them itself (16-byte stores when K is
//    the template cap).  This file is built without NaN semantics (the
//    inputs are finite or -inf), so the raw logits are sort keys as they are.
//  - route_kernel (any N <= 64): the rows staged through registers into a padded LDS tile;
//    every lane routes its token from its row and stores its own outputs.
//  - route_x16_kernel (N = 64, batches of at most kSmallBatch tokens): 16 lanes per token
//    (route_token_x16: a bitonic sort across the 16 lanes), 16 tokens per block, so that a
//    small batch still spreads over many compute units.  The same bits as the other two.
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

// ---- route_dma_kernel ----

template <int NP, int P, int G, int... I>
__device__ __forceinline__ void sort_group(float* key, std::integer_sequence<int, I...>) {
    (compare_exchange<NP, PhasedHolder<NP, P>::net.idx[G][I]>(key), ...);
}

// read part p of row `lane` into key[p B .. p B + B) (and okey), then sort that part
template <int NP, int G>
__device__ __forceinline__ void load_sort_part(const float* tile, int lane, float* key,
                                               float* okey) {
    using L = DmaTile<NP>;
#pragma unroll
    for (int cc = 0; cc < L::CP; ++cc) {
        const float4 v = *reinterpret_cast<const float4*>(
            tile + ((G * 64 * L::CP + lane * L::CP + (cc ^ L::swz(lane))) << 2));
        const int c0 = G * L::B + cc * 4;
        okey[c0 + 0] = v.x;  // raw logits: this file is built without NaN semantics, so
        okey[c0 + 1] = v.y;  // min/max need no canonicalisation, and -0 / +0 compare and
        okey[c0 + 2] = v.z;  // subtract as equals, so the order and every value derived
        okey[c0 + 3] = v.w;  // from the keys are those of the canonical keys
#pragma unroll
        for (int q = 0; q < 4; ++q) key[c0 + q] = okey[c0 + q];
    }
    sort_group<NP, L::P, G>(
        key, std::make_integer_sequence<int, PhasedHolder<NP, L::P>::net.cnt[G]>{});
}

// N == NP in {16, 32, 64}; logits 16-byte aligned.  vst: ids and w 16-byte aligned (the
// output stores are then 16 bytes wide).
template <int NP, int KMAX>
__global__ __launch_bounds__(256) void route_dma_kernel(const float* __restrict__ logits,
                                                        int64_t T, int K, float eps, int mode,
                                                        int renorm, int vst, XTable xt,
                                                        int* __restrict__ kout,
                                                        int* __restrict__ ids,
                                                        float* __restrict__ wout) {
    using L = DmaTile<NP>;
    constexpr int WS = 64 * NP;  // floats of a wave's logit tile
    __shared__ __attribute__((aligned(1024))) float lds[4 * WS];
    const int lane = threadIdx.x & (kWave - 1);
    const int wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);  // uniform: scalar bases
    const int64_t t0 = ((int64_t)blockIdx.x * 4 + wv) * kWave;
    if (t0 >= T) return;  // wave-uniform; the kernel has no block barrier
    const int rows = (int)((T - t0) < kWave ? (T - t0) : kWave);
    float* tile = lds + wv * WS;

    // ---- copy the tile: part p, instruction j of CP; lane -> (row, slot) of its 16 bytes ----
    const float* src = logits + t0 * NP;
    const uint32_t lds0 = (uint32_t)(uintptr_t)(lds_void_t*)tile;
#pragma unroll
    for (int p = 0; p < L::P; ++p)
#pragma unroll
        for (int j = 0; j < L::CP; ++j) {
            const int local = j * 64 + lane;
            const int r = local / L::CP;
            const int cc = (local % L::CP) ^ L::swz(r);
            const int rs = r < rows ? r : rows - 1;  // rows past T: a valid row, never used
            const uint32_t va = (uint32_t)(rs * NP + (p * L::CP + cc) * 4) * 4u;
            const uint32_t la =
                __builtin_amdgcn_readfirstlane(lds0 + (p * 64 * L::CP + j * 64) * 16);
            // non-temporal: the logits are read once (measured: -3 % at T = 65536 and 2^20)
            asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dwordx4 %1, %2 nt"
                         :: "s"(la), "v"(va), "s"(src) : "memory", "m0");
        }

    // ---- each part: wait for its copies (they complete in order), read the row's part, sort
    float key[NP], okey[NP];
#define ELB_PART(G)                                                                      \
    if constexpr (G < L::P) {                                                            \
        __builtin_amdgcn_sched_barrier(0);                                               \
        ELB_WAIT_VMCNT((L::P - 1 - (G)) * L::CP);                                     \
        __builtin_amdgcn_sched_barrier(0);                                               \
        load_sort_part<NP, G>(tile, lane, key, okey);                                    \
    }
    ELB_PART(0)
    ELB_PART(1)
    ELB_PART(2)
    ELB_PART(3)
#undef ELB_PART
    sort_group<NP, L::P, L::P>(
        key, std::make_integer_sequence<int, PhasedHolder<NP, L::P>::net.cnt[L::P]>{});

    float u[NP], S;
    const int k = sorted_elbow<NP, true, KMAX>(key, NP, K, eps, mode, xt, u, S);
    if (lane < rows) kout[t0 + lane] = k;

    // ---- select; each lane's outputs go to registers: the common path emits rank j with j a
    // compile-time constant, so the unrolled select below is a plain move (the rare tie path
    // gets a select chain), and the lane stores its own row without staging it in LDS ----
    int oid[KMAX];
    float ow[KMAX];
#pragma unroll
    for (int q = 0; q < KMAX; ++q) {
        oid[q] = -1;
        ow[q] = 0.f;
    }
    select_emit<NP, true, KMAX>(
        key, [&](int c) { return okey[c]; },
        [&](int c) { return order_key(tile[L::at(lane, c)]); }, NP, K, k, u, S, renorm,
        [&](int j, int id, float w) {
#pragma unroll
            for (int q = 0; q < KMAX; ++q)
                if (q == j) {
                    oid[q] = id;
                    ow[q] = w;
                }
        });
    if (lane >= rows) return;
    int* const gi = ids + (t0 + lane) * K;
    float* const gw = wout + (t0 + lane) * K;
    if (vst && K == KMAX) {  // rows of KMAX values, 16-byte aligned: KMAX / 4 stores each
#pragma unroll
        for (int q = 0; q < KMAX; q += 4) {
            *reinterpret_cast<int4*>(gi + q) =
                make_int4(oid[q], oid[q + 1], oid[q + 2], oid[q + 3]);
            *reinterpret_cast<float4*>(gw + q) =
                make_float4(ow[q], ow[q + 1], ow[q + 2], ow[q + 3]);
        }
    } else {
#pragma unroll
        for (int q = 0; q < KMAX; ++q)
            if (q < K) {
                gi[q] = oid[q];
                gw[q] = ow[q];
            }
    }
}

template <int NP, bool FULL, int KMAX>
hipError_t launch_np(const float* logits, int64_t T, int N, const elb_route_params& p, int* k,
                     int* ids, float* w, hipStream_t s) {
    const XTable xt = make_xtable(N);
    const int64_t waves = (T + kWave - 1) / kWave;
    const unsigned blocks = (unsigned)((waves + 3) / 4);
    const int vec4 = ((uintptr_t)logits % 16) == 0;
    ProfileScope prof("route", s);
    if constexpr (FULL && NP >= 16) {
        if (vec4) {
            const int vst = ((uintptr_t)ids % 16) == 0 && ((uintptr_t)w % 16) == 0;
            ELB_LAUNCH((route_dma_kernel<NP, KMAX>), dim3(blocks), dim3(256), 0, s,
                               logits, T, p.K, p.eps, p.mode, p.renormalize, vst, xt, k, ids, w);
            return hipGetLastError();
        }
    }
    ELB_LAUNCH((route_kernel<NP, FULL, KMAX>), dim3(blocks), dim3(256), 0, s, logits, T, N, p.K,
                       p.eps, p.mode, p.renormalize, vec4, xt, k, ids, w);
    return hipGetLastError();
}

// ---- route_x16_kernel: small batches with N = 64, 16 lanes per token (route_token_x16),
// 16 tokens per block ----
template <int KMAX>
__global__ __launch_bounds__(256) void route_x16_kernel(const float* __restrict__ logits,
                                                        int64_t T, int K, float eps, int mode,
                                                        int renorm, XTable xt,
                                                        int* __restrict__ kout,
                                                        int* __restrict__ ids,
                                                        float* __restrict__ wout) {
    __shared__ float rows[16][65];
    const int64_t t0 = (int64_t)blockIdx.x * 16;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        const int i = threadIdx.x + 256 * q;
        const int r = i >> 6, c = i & 63;
        const int64_t t = t0 + r;
        rows[r][c] = (t < T) ? logits[t * 64 + c] : 0.f;  // rows past T: finite, never stored
    }
    __syncthreads();
    const int tr = threadIdx.x >> 4;
    route_token_x16<KMAX>(&rows[tr][0], K, eps, mode, renorm, xt, t0 + tr, t0 + tr < T, kout,
                          ids, wout);
}

template <int KMAX>
hipError_t launch_k(const float* logits, int64_t T, int N, const elb_route_params& p, int* k,
                   int* ids, float* w, hipStream_t s) {
    if (N == 64 && T <= kSmallBatch) {
        ProfileScope prof("route", s);
        ELB_LAUNCH((route_x16_kernel<KMAX>), dim3((unsigned)((T + 15) / 16)), dim3(256),
                           0, s, logits, T, p.K, p.eps, p.mode, p.renormalize, make_xtable(N), k,
                           ids, w);
        return hipGetLastError();
    }
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
