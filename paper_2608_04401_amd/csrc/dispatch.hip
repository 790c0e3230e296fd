// Variable-k dispatch: per-expert token lists from a routing (k_t experts per token).
//
// Deterministic, no atomics.  Three launches for large batches:
//   count   one lane per token; a wave ORs each token's selected experts into a 64-bit mask
//           and, per expert, counts the wave's tokens with one ballot + popcount.  The
//           per-wave counts form an expert-major [N, groups] histogram (row stride ld, a
//           multiple of 4), or a group-major one (row g: the N counts of group g) when the
//           scatter reads it itself.
//   scan    one block per expert: an exclusive prefix over groups (the base of each group
//           inside the expert's list) and the expert's total.
//   scatter one block of 4 waves per 64-token group, one lane per token.  Each wave forms
//           the exclusive prefix of the expert totals (list offsets) and of their M-tile
//           counts with a wave scan (block 0 also writes them out); the rank of a token inside
//           its group's share of expert e is the popcount of the expert's ballot below the
//           lane, and its row is offsets[e] + base[e, group] + rank (each wave takes a quarter
//           of the experts).  Rows within an expert are therefore in increasing token order.
// Up to kDirectGroups groups (T <= 8192) the scan launch is skipped: every scatter wave reads
// the whole group-major histogram (lane e: entry e of every group's row, so that each load is
// one contiguous row; all in flight at once) and forms the expert totals and its own group's
// base itself.  When the split router's routing wrote one histogram per quarter of each group
// (kHistSubs of them), wave w reads histogram w and the four waves add their sums through
// LDS.  One launch (dispatch_small) for T <= 256.  All three forms give the same rows.
// Requires N <= 64 (one mask bit per expert).
#include "common.h"

namespace elb {

namespace {

// waves (64-token groups) per block of the count and scatter kernels
constexpr int kDispWaves = 1;

// slots j0 .. j0 + 7 of token t's ids (-1 past K): eight independent loads, so a lane waits
// for memory once per eight slots rather than once per slot
__device__ __forceinline__ void load_ids8(const int* __restrict__ ids, int64_t t, int K, int j0,
                                          int (&e8)[8]) {
#pragma unroll
    for (int q = 0; q < 8; ++q) e8[q] = (j0 + q < K) ? ids[t * K + j0 + q] : -1;
}

// the mask of token t's first kt experts from its slots: the first eight already loaded
// (e8), the rest (K > 8) loaded here
__device__ __forceinline__ uint64_t token_mask_pre(int kt, const int (&e8)[8],
                                                   const int* __restrict__ ids, int64_t t,
                                                   int N, int K, bool valid) {
    uint64_t mask = 0;
    if (valid) {
#pragma unroll
        for (int q = 0; q < 8; ++q) {
            const int e = e8[q];
            if (q < kt && (unsigned)e < (unsigned)N) mask |= 1ull << e;
        }
        for (int j0 = 8; j0 < K; j0 += 8) {
            int f8[8];
            load_ids8(ids, t, K, j0, f8);
#pragma unroll
            for (int q = 0; q < 8; ++q) {
                const int e = f8[q];
                if (j0 + q < kt && (unsigned)e < (unsigned)N) mask |= 1ull << e;
            }
        }
    }
    return mask;
}

__device__ __forceinline__ uint64_t token_mask(const int* __restrict__ k,
                                               const int* __restrict__ ids, int64_t t, int N,
                                               int K, bool valid) {
    uint64_t mask = 0;
    if (valid) {
        const int kt = k[t];
        for (int j0 = 0; j0 < K; j0 += 8) {
            int e8[8];
            load_ids8(ids, t, K, j0, e8);
#pragma unroll
            for (int q = 0; q < 8; ++q) {
                const int e = e8[q];
                if (j0 + q < kt && (unsigned)e < (unsigned)N) mask |= 1ull << e;
            }
        }
    }
    return mask;
}

// The M-tile count of expert `lane` (c rows) under the plan; on the whole wave (lane e < N
// holds expert e), so that the tail decision sees every expert.  tail_mine: the expert's
// remainder goes to the tail kernel; n_tail: how many experts do.
__device__ __forceinline__ int plan_tiles(int c, int lane, int N, const TilePlan& tp,
                                          bool& tail_mine, int& n_tail) {
    const int full = c / tp.tile_rows;
    const int rem = c - full * tp.tile_rows;
    const int tiles = full + (rem > 0 ? 1 : 0);
    const bool cand = tp.tail_rows > 0 && lane < N && full >= 1 && rem > 0 &&
                      rem <= tp.tail_rows;
    int sum = lane < N ? tiles : 0;
#pragma unroll
    for (int o = 1; o < kWave; o <<= 1) sum += __shfl_xor(sum, o);
    const int nc = __popcll(__ballot(cand));
    const int r_all = (sum + tp.tiles_per_round - 1) / tp.tiles_per_round;
    const int r_tail = (sum - nc + tp.tiles_per_round - 1) / tp.tiles_per_round;
    const bool use = nc > 0 && nc <= tp.tail_max && r_tail < r_all;
    tail_mine = use && cand;
    n_tail = use ? nc : 0;
    return tail_mine ? full : tiles;
}

// the compact list of tail experts (by wave 0 of block 0)
__device__ __forceinline__ void write_tail_list(bool tail_mine, int n_tail, int lane,
                                                int* __restrict__ tail_list) {
    const uint64_t b = __ballot(tail_mine);
    const uint64_t below = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
    if (tail_mine) tail_list[1 + __popcll(b & below)] = lane;
    if (lane == 0) tail_list[0] = n_tail;
}

// gmajor: write the group-major histogram the scatter reads itself (row g of N counts), else
// the expert-major one the scan launch takes
__global__ __launch_bounds__(64 * kDispWaves) void dispatch_count(
    const int* __restrict__ k, const int* __restrict__ ids, int64_t T, int N, int K, int64_t ld,
    int gmajor, int* __restrict__ hist) {
    const int lane = threadIdx.x & (kWave - 1);
    const int64_t g = (int64_t)blockIdx.x * kDispWaves + (threadIdx.x >> 6);
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
    if (lane < N) hist[gmajor ? g * N + lane : (int64_t)lane * ld + g] = mine;
}

// one block per expert e: exclusive prefix of hist[e, :] over the groups, in place
__global__ __launch_bounds__(1024) void dispatch_scan(int* __restrict__ hist, int64_t groups,
                                                     int64_t ld, int* __restrict__ counts) {
    __shared__ int wsum[16];
    const int e = blockIdx.x;
    const int tid = threadIdx.x;
    const int lane = tid & (kWave - 1);
    const int wv = tid >> 6;
    int* h = hist + (int64_t)e * ld;
    const int64_t chunk = (groups + 1023) / 1024;  // consecutive groups per thread
    const int64_t g0 = tid * chunk;
    const int64_t g1 = (g0 + chunk < groups) ? g0 + chunk : groups;
    int s = 0;
    for (int64_t g = g0; g < g1; ++g) s += h[g];
    // block-wide exclusive scan of s: within the wave, then over the 16 wave totals
    int incl = s;
    for (int dd = 1; dd < kWave; dd <<= 1) {
        const int o = __shfl_up(incl, dd);
        if (lane >= dd) incl += o;
    }
    if (lane == kWave - 1) wsum[wv] = incl;
    __syncthreads();
    int wbase = 0, total = 0;
    for (int q = 0; q < 16; ++q) {
        const int v = wsum[q];
        wbase += (q < wv) ? v : 0;
        total += v;
    }
    int run = wbase + incl - s;
    for (int64_t g = g0; g < g1; ++g) {
        const int c = h[g];
        h[g] = run;  // exclusive base of group g inside expert e's list
        run += c;
    }
    if (tid == 0) counts[e] = total;
}

constexpr int kScatterWaves = 4;  // waves per 64-token group in the scatter
static_assert(kScatterWaves == kHistSubs, "one scatter wave per sub-histogram");

// One block per 64-token group g; its kScatterWaves waves each place the group's tokens in the
// lists of N / kScatterWaves experts, then each writes a share of the group's inv slots.
// DIRECT: hist holds the raw per-group counts (no scan launch) and counts is written here;
// subs (DIRECT only): the number of histograms (kHistSubs: one per quarter of each group,
// sub_stride ints apart, summed here; 1: every wave reads the one histogram)
template <bool DIRECT>
__global__ __launch_bounds__(64 * kScatterWaves) void dispatch_scatter(
    const int* __restrict__ k, const int* __restrict__ ids, int64_t T, int N, int K, int64_t ld,
    const int* __restrict__ hist, int subs, int64_t sub_stride, int* __restrict__ counts,
    int* __restrict__ offsets, int* __restrict__ tile_off, int* __restrict__ tail_list,
    TilePlan plan, int* __restrict__ row_token, int* __restrict__ inv) {
    __shared__ int pos[kWave][kWave + 1];  // [token lane][expert]: the token's row
    __shared__ int red[2][kScatterWaves][kWave];  // per-wave sums of the sub-histograms
    const int lane = threadIdx.x & (kWave - 1);
    const int wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);  // wave-uniform
    const int64_t g = blockIdx.x;
    const int64_t t = g * kWave + lane;
    const int64_t groups = (T + kWave - 1) / kWave;
    // the lane's token: k and its first eight slots, loaded before the histogram (both in
    // flight together) and kept for the inverse map.  No per-lane branch around the loads (a
    // lane past T reads token T - 1 and drops it): behind a divergent branch the compiler
    // cannot tell the loads have landed and waits for every memory operation, the row stores
    // below included, before each later use.
    const bool valid = t < T;  // false for every lane of a block past the groups (T == 0)
    int kt = 0, e8[8];
#pragma unroll
    for (int q = 0; q < 8; ++q) e8[q] = -1;
    if (T > 0) {  // uniform
        const int64_t tc = valid ? t : T - 1;
        kt = valid ? k[tc] : 0;
        load_ids8(ids, tc, K, 0, e8);
    }
    // expert list offsets and M-tile offsets: exclusive prefixes over the experts (lane e),
    // formed by every wave.  c: expert e's total; hist_mine: the base of this group inside
    // expert e's list.
    int c = 0, hist_mine = 0;
    if (DIRECT) {
        // lane e sums expert e's counts of the raw histogram: over every group (the total)
        // and over the groups below g (the base), in group order; pad rows past `groups` are
        // not read
        const int sub = subs > 1 ? wv : 0;  // wave wv reads histogram wv (or the only one)
        {
            // group-major: lane e reads entry e of every group's row (each load one contiguous
            // row of N counts); lanes past N read entry N - 1 and drop it (no per-lane branch
            // around the loads)
            const int* const hb = hist + sub * sub_stride + (lane < N ? lane : N - 1);
            const int ng = (int)groups, gg = (int)g;
            int v[kDirectGroups];
#pragma unroll
            for (int q = 0; q < kDirectGroups; ++q) v[q] = (q < ng) ? hb[(int64_t)q * N] : 0;
#pragma unroll
            for (int q = 0; q < kDirectGroups; ++q) {
                c += v[q];
                hist_mine += q < gg ? v[q] : 0;
            }
            if (lane >= N) c = hist_mine = 0;
        }
        if (subs > 1) {  // block-uniform: every wave takes the sums over the histograms
            red[0][wv][lane] = c;
            red[1][wv][lane] = hist_mine;
            __syncthreads();
            c = 0;
            hist_mine = 0;
#pragma unroll
            for (int q = 0; q < kScatterWaves; ++q) {
                c += red[0][q][lane];
                hist_mine += red[1][q][lane];
            }
        }
    } else {
        // the group's (scanned) histogram entry is loaded together with the totals (one
        // memory round trip for both)
        c = (lane < N) ? counts[lane] : 0;
        hist_mine = (lane < N) ? hist[(int64_t)lane * ld + (g < groups ? g : 0)] : 0;
    }
    bool tail_mine;
    int n_tail;
    const int tiles = plan_tiles(c, lane, N, plan, tail_mine, n_tail);  // whole wave
    int incl = c, tincl = tiles;
    for (int dd = 1; dd < kWave; dd <<= 1) {
        const int o = __shfl_up(incl, dd);
        const int to = __shfl_up(tincl, dd);
        if (lane >= dd) {
            incl += o;
            tincl += to;
        }
    }
    const int off_mine = incl - c;
    if (blockIdx.x == 0 && wv == 0) {
        if (lane < N) {
            offsets[lane] = off_mine;
            tile_off[lane] = tincl - tiles;
            if (DIRECT) counts[lane] = c;
        }
        if (lane == N - 1) {
            offsets[N] = incl;
            tile_off[N] = tincl;
        }
        write_tail_list(tail_mine, n_tail, lane, tail_list);
    }
    if (g >= groups) return;  // block-uniform (T == 0: the one block only writes the offsets)
    const uint64_t mask = token_mask_pre(kt, e8, ids, t, N, K, valid);
    // lane e holds the first row of expert e that belongs to this group
    const int base_mine = (lane < N) ? off_mine + hist_mine : 0;
    const uint64_t below = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
    const int per = (N + kScatterWaves - 1) / kScatterWaves;
    const int e0 = wv * per, e1 = e0 + per < N ? e0 + per : N;
    // a fixed trip count (N <= 64), unrolled, so that the experts' ballots and lane reads
    // overlap instead of forming one dependent chain
#pragma unroll
    for (int i = 0; i < kWave / kScatterWaves; ++i) {
        const int e = e0 + i;
        if (e < e1) {  // wave-uniform
            const bool has = (mask >> e) & 1ull;
            const uint64_t b = __ballot(has);
            const int base = __builtin_amdgcn_readlane(base_mine, e);
            if (has) {
                const int r = base + __popcll(b & below);
                row_token[r] = (int)t;
                pos[lane][e] = r;
            }
        }
    }
    __syncthreads();
    if (!valid) return;  // no barrier follows
#pragma unroll
    for (int j = 0; j < 8; ++j) {
        if (j < K && j % kScatterWaves == wv) {  // wave-uniform
            const int e = e8[j];
            int r = -1;
            if (j < kt && (unsigned)e < (unsigned)N) r = pos[lane][e];
            inv[t * K + j] = r;
        }
    }
    for (int j = 8 + wv; j < K; j += kScatterWaves) {
        const int e = ids[t * K + j];
        int r = -1;
        if (j < kt && (unsigned)e < (unsigned)N) r = pos[lane][e];
        inv[t * K + j] = r;
    }
}

// Small batches (T <= 256, decode): the three steps in ONE block of 4 waves, one lane per
// token.  The per-wave expert counts go to LDS; wave 0 turns them into per-wave bases inside
// each expert's list and, with a wave scan over the experts, into the list and M-tile
// offsets; then every wave places its tokens exactly as dispatch_scatter does.  Same rows,
// same order, as the three-launch path.
__global__ __launch_bounds__(256) void dispatch_small(const int* __restrict__ k,
                                                      const int* __restrict__ ids, int T, int N,
                                                      int K, int* __restrict__ counts,
                                                      int* __restrict__ offsets,
                                                      int* __restrict__ tile_off,
                                                      int* __restrict__ tail_list,
                                                      TilePlan plan,
                                                      int* __restrict__ row_token,
                                                      int* __restrict__ inv) {
    __shared__ int base[4][kWave];  // per-wave counts, then each wave's base in the list
    __shared__ int offs[kWave];
    __shared__ int pos[4][kWave][kWave + 1];
    const int lane = threadIdx.x & (kWave - 1);
    const int wv = threadIdx.x >> 6;
    const int t = wv * kWave + lane;
    const bool valid = t < T;
    const uint64_t mask = token_mask(k, ids, t, N, K, valid);
    int mine = 0;
    for (int e = 0; e < N; ++e) {
        const int c = __popcll(__ballot((mask >> e) & 1ull));
        if (lane == e) mine = c;
    }
    base[wv][lane] = mine;
    __syncthreads();
    if (wv == 0) {
        int c = 0;
#pragma unroll
        for (int w = 0; w < 4; ++w) {  // lane e: exclusive prefix over the waves
            const int cw = base[w][lane];
            base[w][lane] = c;
            c += cw;
        }
        if (lane >= N) c = 0;
        bool tail_mine;
        int n_tail;
        const int tiles = plan_tiles(c, lane, N, plan, tail_mine, n_tail);
        int incl = c, tincl = tiles;
        for (int dd = 1; dd < kWave; dd <<= 1) {
            const int o = __shfl_up(incl, dd);
            const int to = __shfl_up(tincl, dd);
            if (lane >= dd) {
                incl += o;
                tincl += to;
            }
        }
        offs[lane] = incl - c;
        if (lane < N) {
            counts[lane] = c;
            offsets[lane] = incl - c;
            tile_off[lane] = tincl - tiles;
        }
        if (lane == N - 1) {
            offsets[N] = incl;
            tile_off[N] = tincl;
        }
        write_tail_list(tail_mine, n_tail, lane, tail_list);
    }
    __syncthreads();
    const int base_mine = (lane < N) ? offs[lane] + base[wv][lane] : 0;
    const uint64_t below = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
    for (int e = 0; e < N; ++e) {
        const bool has = (mask >> e) & 1ull;
        const uint64_t b = __ballot(has);
        const int bse = __builtin_amdgcn_readlane(base_mine, e);  // e is wave-uniform
        if (has) {
            const int r = bse + __popcll(b & below);
            row_token[r] = t;
            pos[wv][lane][e] = r;
        }
    }
    if (!valid) return;  // no barrier follows
    const int kt = k[t];
    for (int j0 = 0; j0 < K; j0 += 8) {
        int e8[8];
        load_ids8(ids, t, K, j0, e8);
#pragma unroll
        for (int q = 0; q < 8; ++q) {
            const int j = j0 + q, e = e8[q];
            if (j >= K) break;
            int r = -1;
            if (j < kt && (unsigned)e < (unsigned)N) r = pos[wv][lane][e];
            inv[(int64_t)t * K + j] = r;
        }
    }
}

}  // namespace

hipError_t launch_dispatch(const int* k, const int* ids, int64_t T, int N, int K, int* counts,
                           int* offsets, int* row_token, int* inv, int* hist, int* tile_off,
                           int* tail_list, const TilePlan& plan, hipStream_t s,
                           bool hist_ready, int hist_subs) {
    if (T <= 256 && !hist_ready) {
        ProfileScope prof("dispatch_small", s);
        ELB_LAUNCH(dispatch_small, dim3(1), dim3(256), 0, s, k, ids, (int)T, N, K,
                           counts, offsets, tile_off, tail_list, plan, row_token, inv);
        return hipGetLastError();
    }
    const int64_t groups = dispatch_groups(T);
    const int64_t ld = dispatch_hist_ld(T);
    const bool direct = groups <= kDirectGroups;
    if (hist_subs != 1 && !(hist_ready && direct && hist_subs == kHistSubs))
        return hipErrorInvalidValue;  // sub-histograms come from the split router, T <= 8192
    // at least one scatter block, which also writes offsets and tile_off (also when T == 0)
    const int64_t nb = (groups + kDispWaves - 1) / kDispWaves;
    const unsigned blocks = (unsigned)(nb > 0 ? nb : 1);
    if (T > 0 && !hist_ready) {
        ProfileScope prof("dispatch_count", s);
        ELB_LAUNCH(dispatch_count, dim3(blocks), dim3(64 * kDispWaves), 0, s, k, ids, T,
                           N, K, ld, (int)direct, hist);
    }
    if (!direct) {
        ProfileScope prof("dispatch_scan", s);
        ELB_LAUNCH(dispatch_scan, dim3((unsigned)N), dim3(1024), 0, s, hist, groups, ld,
                           counts);
    }
    {
        ProfileScope prof("dispatch_scatter", s);
        const unsigned sblocks = (unsigned)(groups > 0 ? groups : 1);
        if (direct)
            ELB_LAUNCH(dispatch_scatter<true>, dim3(sblocks), dim3(64 * kScatterWaves), 0, s,
                       k, ids, T, N, K, ld, hist, hist_subs, ld * N, counts, offsets,
                       tile_off, tail_list, plan, row_token, inv);
        else
            ELB_LAUNCH(dispatch_scatter<false>, dim3(sblocks), dim3(64 * kScatterWaves), 0, s,
                       k, ids, T, N, K, ld, hist, 1, ld * N, counts, offsets, tile_off,
                       tail_list, plan, row_token, inv);
    }
    return hipGetLastError();
}

}  // namespace elb
