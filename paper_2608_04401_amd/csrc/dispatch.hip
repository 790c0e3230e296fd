// Variable-k dispatch: per-expert token lists from a routing (k_t experts per token).
//
// Three launches, deterministic, no atomics:
//   count   one lane per token; a wave ORs each token's selected experts into a 64-bit mask
//           and, per expert, counts the wave's tokens with one ballot + popcount.  The
//           per-wave counts form a [groups, N] histogram.
//   scan    one block: for every expert, an exclusive prefix over groups (the base of each
//           group inside the expert's list), the expert totals, their exclusive prefix
//           (list offsets) and the grouped GEMM's M-tile offsets.
//   scatter one lane per token again: the rank of a token inside its group's share of
//           expert e is the popcount of the expert's ballot below the lane; the row is
//           offsets[e] + base[group, e] + rank.  Rows within an expert are therefore in
//           increasing token order.
// Requires N <= 64 (one mask bit per expert).
#include "common.h"

namespace elb {

namespace {

__device__ __forceinline__ uint64_t token_mask(const int* __restrict__ k,
                                               const int* __restrict__ ids, int64_t t, int N,
                                               int K, bool valid) {
    uint64_t mask = 0;
    if (valid) {
        const int kt = k[t];
        for (int j = 0; j < K; ++j) {
            const int e = ids[t * K + j];
            if (j < kt && (unsigned)e < (unsigned)N) mask |= 1ull << e;
        }
    }
    return mask;
}

__global__ __launch_bounds__(256) void dispatch_count(const int* __restrict__ k,
                                                      const int* __restrict__ ids, int64_t T,
                                                      int N, int K, int* __restrict__ hist) {
    const int lane = threadIdx.x & (kWave - 1);
    const int64_t g = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    const int64_t t = g * kWave + lane;
    const int64_t groups = (T + kWave - 1) / kWave;
    if (g >= groups) return;  // wave-uniform
    const uint64_t mask = token_mask(k, ids, t, N, K, t < T);
    int mine = 0;
    for (int e = 0; e < N; ++e) {
        const uint64_t b = __ballot((mask >> e) & 1ull);
        const int c = __popcll(b);
        if (lane == e) mine = c;
    }
    if (lane < N) hist[g * N + lane] = mine;
}

// one block of 1024 threads: thread (e = tid % 64, part = tid / 64)
__global__ __launch_bounds__(1024) void dispatch_scan(int* __restrict__ hist, int64_t groups,
                                                     int N, int* __restrict__ counts,
                                                     int* __restrict__ offsets,
                                                     int* __restrict__ tile_off,
                                                     int tile_rows) {
    constexpr int kParts = 16;
    __shared__ int part_sum[kParts][64];
    __shared__ int part_base[kParts][64];
    __shared__ int tot[64];
    const int e = threadIdx.x & 63;
    const int part = threadIdx.x >> 6;
    const int64_t per = (groups + kParts - 1) / kParts;
    const int64_t g0 = part * per;
    const int64_t g1 = (g0 + per < groups) ? g0 + per : groups;
    int s = 0;
    if (e < N)
        for (int64_t g = g0; g < g1; ++g) s += hist[g * N + e];
    part_sum[part][e] = s;
    __syncthreads();
    if (part == 0) {
        int run = 0;
        for (int p = 0; p < kParts; ++p) {
            part_base[p][e] = run;
            run += part_sum[p][e];
        }
        tot[e] = (e < N) ? run : 0;
    }
    __syncthreads();
    if (e < N) {
        int run = part_base[part][e];
        for (int64_t g = g0; g < g1; ++g) {
            const int c = hist[g * N + e];
            hist[g * N + e] = run;  // exclusive base of group g inside expert e's list
            run += c;
        }
    }
    if (threadIdx.x < 64) {  // wave 0: offsets and tile offsets over experts
        const int c = tot[e];
        const int tiles = (c + tile_rows - 1) / tile_rows;
        int incl = c, tincl = tiles;
        for (int d = 1; d < 64; d <<= 1) {
            const int o = __shfl_up(incl, d);
            const int to = __shfl_up(tincl, d);
            if (e >= d) {
                incl += o;
                tincl += to;
            }
        }
        if (e < N) {
            counts[e] = c;
            offsets[e] = incl - c;
            tile_off[e] = tincl - tiles;
        }
        if (e == N - 1) {
            offsets[N] = incl;
            tile_off[N] = tincl;
        }
    }
}

__global__ __launch_bounds__(256) void dispatch_scatter(const int* __restrict__ k,
                                                        const int* __restrict__ ids, int64_t T,
                                                        int N, int K,
                                                        const int* __restrict__ hist,
                                                        const int* __restrict__ offsets,
                                                        int* __restrict__ row_token,
                                                        int* __restrict__ inv) {
    __shared__ int pos[4][kWave][kWave + 1];
    const int lane = threadIdx.x & (kWave - 1);
    const int wv = threadIdx.x >> 6;
    const int64_t g = (int64_t)blockIdx.x * 4 + wv;
    const int64_t t = g * kWave + lane;
    const int64_t groups = (T + kWave - 1) / kWave;
    if (g >= groups) return;  // wave-uniform; no block barrier in this kernel
    const bool valid = t < T;
    const uint64_t mask = token_mask(k, ids, t, N, K, valid);
    // lane e holds the first row of expert e that belongs to this group
    const int base_mine = (lane < N) ? offsets[lane] + hist[g * N + lane] : 0;
    const uint64_t below = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
    for (int e = 0; e < N; ++e) {
        const bool has = (mask >> e) & 1ull;
        const uint64_t b = __ballot(has);
        const int base = __shfl(base_mine, e);
        if (has) {
            const int r = base + __popcll(b & below);
            row_token[r] = (int)t;
            pos[wv][lane][e] = r;
        }
    }
    if (!valid) return;
    const int kt = k[t];
    for (int j = 0; j < K; ++j) {
        const int e = ids[t * K + j];
        int r = -1;
        if (j < kt && (unsigned)e < (unsigned)N) r = pos[wv][lane][e];
        inv[t * K + j] = r;
    }
}

}  // namespace

hipError_t launch_dispatch(const int* k, const int* ids, int64_t T, int N, int K, int* counts,
                           int* offsets, int* row_token, int* inv, int* hist, int* tile_off,
                           int tile_rows, hipStream_t s) {
    const int64_t groups = dispatch_groups(T);
    const unsigned blocks = (unsigned)((groups + 3) / 4);
    {
        ProfileScope prof("dispatch_count", s);
        if (T > 0)
            hipLaunchKernelGGL(dispatch_count, dim3(blocks), dim3(256), 0, s, k, ids, T, N, K,
                               hist);
    }
    {
        ProfileScope prof("dispatch_scan", s);
        hipLaunchKernelGGL(dispatch_scan, dim3(1), dim3(1024), 0, s, hist, groups, N, counts,
                           offsets, tile_off, tile_rows);
    }
    {
        ProfileScope prof("dispatch_scatter", s);
        if (T > 0)
            hipLaunchKernelGGL(dispatch_scatter, dim3(blocks), dim3(256), 0, s, k, ids, T, N, K,
                               hist, offsets, row_token, inv);
    }
    return hipGetLastError();
}

}  // namespace elb
