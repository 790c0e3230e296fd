// Router logits l = x W_r^T (Section 2: a learned router produces logits l(x) in R^N),
// fp32 accumulation and fp32 output; and the router fused with the routing of its logits.
//
// bf16: one block of 4 waves per 16 tokens.  Wave w takes the w-th contiguous quarter of the
// 32-deep k-steps (router_slice), so it reads a distinct quarter of the 16 x d slice of x (x
// is read once) and the matching columns of all N rows of W_r (which stays in L2 across
// blocks); each wave runs 4 v_mfma_f32_16x16x32_bf16 chains (16 experts each) with its loads
// four steps ahead of their use, and the 4 partial 16 x N tiles are summed in LDS in order.
// N <= 64, d % 32 == 0.
// fp32: one thread per (token, expert) dot product (the small fp32 configuration).
#include "route_lane.h"

namespace elb {

namespace {

constexpr int RW = 4;  // waves per router block

// The order in which every router kernel accumulates a logit (so that all of them give the same
// bits): the d / 32 k-steps of 32 are cut into RW contiguous slices, slice s holding steps
// [s n / RW, (s + 1) n / RW); each slice is one chain of MFMAs over its steps in order,
// starting from zero, and the logit is ((P_0 + P_1) + P_2) + P_3 in fp32.
__device__ __forceinline__ void router_slice(int d, int s, int& first, int& count) {
    const int n = d / 32;
    first = s * n / RW;
    count = (s + 1) * n / RW - first;
}

// The logits of tokens [t0, t0 + 16) and experts [16 g0, 16 (g0 + NG)) (NG groups of 16):
// each wave's partial sums over its k-steps go to part[w] (lane rows, expert columns
// 16 g + ..., g < NG); the caller sums the RW partial tiles.  Every logit is computed the same
// way whatever NG and g0 are (its own MFMA column, the same k-steps per wave, the same sum).
// w: the slice (by default the wave's index in the block).
template <int NG>
__device__ __forceinline__ void router_partials(const bf16_t* __restrict__ x,
                                                const bf16_t* __restrict__ Wr, int64_t T,
                                                int d, int N, int64_t t0, int g0,
                                                float (&part)[RW][16][65],
                                                int w = threadIdx.x >> 6) {
    const int lane = threadIdx.x & 63;
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
    // wave w takes the w-th quarter of the 32-deep k-steps (router_slice), in order.  A ring
    // of R register slots keeps R - 1 steps in flight: step j lives in slot j % R, and while
    // step j is multiplied, step j + R - 1 is loaded into the slot step j - 1 has just freed.
    // Unrolled by R, so every slot index is a constant.
    constexpr int R = 5;
    int first, mine;
    router_slice(d, w, first, mine);
    bf16x8_t ra[R], rb[R][NG];
    auto load = [&](int slot_j, bf16x8_t& a, bf16x8_t (&bb)[NG]) {
        const int k0 = (slot_j < mine ? first + slot_j : 0) * 32;  // past the end: step 0
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

// Batches of at most kSmallBatch tokens with N = 64 (decode): one wave per (16 tokens, 16
// experts, slice s of the contraction), so that the x and W_r reads spread over four times as
// many compute units as in router_bf16<1> (32 KB per block instead of 128 KB); the partial
// tile goes to part [4, T, 64], and route_split_sum_x16 sums the four slices in order and
// routes them (the same bits as router_bf16's LDS sum and every other router path).
__global__ __launch_bounds__(64) void router_slice_bf16(const bf16_t* __restrict__ x,
                                                        const bf16_t* __restrict__ Wr,
                                                        int64_t T, int d,
                                                        float* __restrict__ part) {
    __shared__ float tile[RW][16][65];  // only row blockIdx.z is used
    const int64_t t0 = (int64_t)blockIdx.x * 16;
    const int g0 = (int)blockIdx.y, s = (int)blockIdx.z;
    router_partials<1>(x, Wr, T, d, 64, t0, g0, tile, s);
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        const int o = threadIdx.x + 64 * q;
        const int tr = o >> 4, nl = o & 15;
        const int64_t t = t0 + tr;
        if (t < T) part[((int64_t)s * T + t) * 64 + 16 * g0 + nl] = tile[s][tr][nl];
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

// ---- split router: the layer's router and routing for large batches (N = 64) ----
//
// router_split_bf16: block (64-token group, slice s) computes partial logit P_s of its 64
// tokens x 64 experts over slice s of the contraction (router_slice), in the same MFMA
// chains as the one-block kernels, so P_s has the same bits.  Both operands go through LDS:
// per 64-column chunk, the block copies its 64 x rows and the 64 W_r rows (128 bytes, one
// cache line, per row) straight into LDS with global_load_lds_dwordx4 (8 rows per
// instruction, 16-byte chunks XOR-swizzled by row so that the MFMA operand reads of 16
// consecutive rows spread over the banks), up to seven chunks ahead in a ring of eight (at
// d = 2048 a slice is eight chunks, all in flight at once).  A block reads
// 64 KB of x and 64 KB of W_r at d = 2048, instead of the 256 KB of W_r that every 16-token
// block of the one-block kernel streams.  Wave w multiplies tokens [16 w, 16 w + 16) by all
// 64 experts.  The partials go to part[s][t][n] (workspace).
// route_split_sum: one wave per 64 tokens, one lane per token: the four partials summed in
// order (the logit), then the routing kernel's per-lane code; the wave also writes its
// group's per-expert assignment counts (the dispatch histogram column of these 64 tokens).
// Requires N == 64 and d % 256 == 0 (every slice a whole number of 64-column chunks).
constexpr int kSplitRing = 8;                // chunks in the ring (128 KB of LDS)
constexpr int kSplitSlot = 2 * 64 * 128;     // bytes per chunk: 64 W_r rows, then 64 x rows

__global__ __launch_bounds__(256) void router_split_bf16(const bf16_t* __restrict__ x,
                                                         const bf16_t* __restrict__ Wr,
                                                         int64_t T, int d,
                                                         float* __restrict__ part) {
    __shared__ __attribute__((aligned(1024))) char sm[kSplitRing * kSplitSlot];
    const int s = blockIdx.y;
    const int64_t t0 = (int64_t)blockIdx.x * 64;
    const int lane = threadIdx.x & 63;
    const int w = threadIdx.x >> 6;
    int first, steps;
    router_slice(d, s, first, steps);  // d % 256 == 0: first and steps are even
    const int c0 = first / 2, nc = steps / 2;
    const bf16_t* const xb = x + t0 * d;  // the block's first token row
    // copy sources: wave w copies rows [16 w, 16 w + 16) of W_r and of x, 8 rows (1 KB) per
    // instruction; lane l fills physical chunk l & 7 of row 16 w + 8 i + (l >> 3), i.e. it
    // fetches that row's logical chunk (l & 7) ^ (row & 7)
    uint32_t woff[2], xoff[2];
#pragma unroll
    for (int i = 0; i < 2; ++i) {
        const int r = 16 * w + 8 * i + (lane >> 3);
        const int q = (lane & 7) ^ (r & 7);
        const int tr = (t0 + r < T) ? r : (int)(T - 1 - t0);  // rows past T: never stored
        woff[i] = ((uint32_t)r * (uint32_t)d + c0 * 64 + q * 8) * 2u;
        xoff[i] = ((uint32_t)tr * (uint32_t)d + c0 * 64 + q * 8) * 2u;
    }
    const uint32_t lds0 = (uint32_t)(uintptr_t)(lds_void_t*)sm;
    auto issue = [&](int c, int slot) {  // chunk c of the slice into ring slot `slot`
#pragma unroll
        for (int i = 0; i < 2; ++i) {
            const uint32_t lw = __builtin_amdgcn_readfirstlane(
                lds0 + slot * kSplitSlot + (2 * w + i) * 1024);
            const uint32_t lx = lw + 64 * 128;
            const uint32_t vw = woff[i] + c * 128, vx = xoff[i] + c * 128;
            asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dwordx4 %1, %2"
                         :: "s"(lw), "v"(vw), "s"(Wr) : "memory", "m0");
            asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dwordx4 %1, %2"
                         :: "s"(lx), "v"(vx), "s"(xb) : "memory", "m0");
        }
    };
    f32x4_t acc[4];
#pragma unroll
    for (int g = 0; g < 4; ++g) acc[g] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    const int l16 = lane & 15, hq = lane >> 4;
    const int arow = 16 * w + l16;  // the A operand's row (token) of this lane
#pragma unroll
    for (int p = 0; p < kSplitRing - 1; ++p)
        if (p < nc) issue(p, p);
    for (int c = 0; c < nc; ++c) {
        // this wave's copies of chunk c are done when at most those of the chunks issued
        // after it (at most kSplitRing - 2, four instructions each) are in flight; the barrier
        // then makes every wave's copies of chunk c visible and frees the slot of chunk c - 1,
        // whose reads every wave has completed
        const int left = nc - 1 - c;
        switch (left < kSplitRing - 2 ? left : kSplitRing - 2) {
            case 0: ELB_WAIT_VMCNT(0); break;
            case 1: ELB_WAIT_VMCNT(4); break;
            case 2: ELB_WAIT_VMCNT(8); break;
            case 3: ELB_WAIT_VMCNT(12); break;
            case 4: ELB_WAIT_VMCNT(16); break;
            case 5: ELB_WAIT_VMCNT(20); break;
            default: ELB_WAIT_VMCNT(24); break;
        }
        asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
        if (c + kSplitRing - 1 < nc) issue(c + kSplitRing - 1, (c + kSplitRing - 1) % kSplitRing);
        const char* const sl = sm + (c % kSplitRing) * kSplitSlot;
#pragma unroll
        for (int j = 0; j < 2; ++j) {  // the chunk's two 32-deep k-steps
            const int q = 4 * j + hq;  // logical 16-byte chunk of this lane's 8 k values
            const bf16x8_t a = *reinterpret_cast<const bf16x8_t*>(
                sl + 64 * 128 + arow * 128 + ((q ^ (arow & 7)) << 4));
            bf16x8_t b[4];
#pragma unroll
            for (int g = 0; g < 4; ++g) {
                const int n = 16 * g + l16;
                b[g] = *reinterpret_cast<const bf16x8_t*>(sl + n * 128 + ((q ^ (n & 7)) << 4));
            }
#pragma unroll
            for (int g = 0; g < 4; ++g)
                acc[g] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b[g], acc[g], 0, 0, 0);
        }
    }
    // lane: tokens 16 w + 4 hq + r (r < 4), expert 16 g + l16
    float* const pp = part + ((int64_t)s * T + t0) * 64;
#pragma unroll
    for (int g = 0; g < 4; ++g)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int tr = 16 * w + 4 * hq + r;
            if (t0 + tr < T) pp[(int64_t)tr * 64 + 16 * g + l16] = acc[g][r];
        }
}

// route_split_sum: one wave per 64-token group, one lane per token.  The group's four partial
// tiles (64 x 64 fp32 each) are copied into LDS with global_load_lds (the routing kernel's
// swizzled tile layout), each lane sums its token's four rows in order -- the logits -- and
// routes them with the routing kernel's own per-lane code (the same bits), then the group's
// per-expert assignment counts are written to its histogram column.
template <int KMAX>
__global__ __launch_bounds__(64) void route_split_sum(const float* __restrict__ part,
                                                      int64_t T, int K, float eps, int mode,
                                                      int renorm, XTable xt,
                                                      float* __restrict__ logits,
                                                      int* __restrict__ kout,
                                                      int* __restrict__ ids,
                                                      float* __restrict__ wout,
                                                      int* __restrict__ hist,
                                                      int64_t hist_ld) {
    using L = DmaTile<64>;
    constexpr int NP = 64, TILE = 64 * 64;
    __shared__ __attribute__((aligned(1024))) float lds[4 * TILE];
    __shared__ int h[64];
    const int lane = threadIdx.x;
    const int64_t t0 = (int64_t)blockIdx.x * 64;
    const int rows = (int)((T - t0) < 64 ? (T - t0) : 64);
    h[lane] = 0;
#pragma unroll
    for (int q = 0; q < 4; ++q) dma_tile<NP>(part + ((int64_t)q * T + t0) * NP, rows,
                                             lds + q * TILE, lane);
    ELB_WAIT_VMCNT(0);
    __builtin_amdgcn_s_barrier();  // one wave: orders the copies' LDS writes before the reads
    // the token's logits: ((P0 + P1) + P2) + P3, element by element
    auto logit = [&](int c) {
        const int a = L::at(lane, c);
        return ((lds[a] + lds[TILE + a]) + lds[2 * TILE + a]) + lds[3 * TILE + a];
    };
    float key[NP], okey[NP];
#pragma unroll
    for (int c = 0; c < NP; ++c) okey[c] = logit(c);
    const bool valid = lane < rows;
    const int64_t t = t0 + lane;
    if (logits && valid) {  // the sums as they are (the one-block kernels write the same)
#pragma unroll
        for (int c = 0; c < NP; ++c) logits[t * NP + c] = okey[c];
    }
#pragma unroll
    for (int c = 0; c < NP; ++c) {
        okey[c] = order_key(okey[c]);
        key[c] = okey[c];
    }
    sort_desc<NP>(key, std::make_integer_sequence<int, NetHolder<NP>::net.n>{});
    float u[NP], S;
    const int k = sorted_elbow<NP, true, KMAX>(key, NP, K, eps, mode, xt, u, S);
    if (valid) kout[t] = k;
    // outputs in registers (the common path emits rank j with j a compile-time constant, so
    // the unrolled select is a plain move; the rare tie path gets a select chain)
    int oid[KMAX];
    float ow[KMAX];
#pragma unroll
    for (int q = 0; q < KMAX; ++q) {
        oid[q] = -1;
        ow[q] = 0.f;
    }
    select_emit<NP, true, KMAX>(
        key, [&](int c) { return okey[c]; }, [&](int c) { return order_key(logit(c)); }, NP, K,
        k, u, S, renorm, [&](int j, int id, float w) {
#pragma unroll
            for (int q = 0; q < KMAX; ++q)
                if (q == j) {
                    oid[q] = id;
                    ow[q] = w;
                }
            if (valid && id >= 0) atomicAdd(&h[id], 1);
        });
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    hist[lane * hist_ld + blockIdx.x] = h[lane];
    if (!valid) return;
#pragma unroll
    for (int q = 0; q < KMAX; ++q)
        if (q < K) {
            ids[t * K + q] = oid[q];
            wout[t * K + q] = ow[q];
        }
}

// route_split_sum_x16 (T <= 64 kDirectGroups, where one lane per token would leave most of
// the chip idle): one block per 16 tokens (a quarter of a 64-token group), 16 lanes per token.
// Lane sl of token r sums elements 4 sl .. 4 sl + 3 of the token's four partial rows in order,
// ((P0 + P1) + P2) + P3 -- the logits, the same sums as above -- and the token is routed by
// the 16-lane routing (route_token_x16, the same bits as the lane kernels).  The block's
// per-expert assignment counts go to histogram blockIdx.x % kHistSubs, row blockIdx.x /
// kHistSubs (the group-major layout the scatter reads: one contiguous row of 64 counts per
// group); the grid has kHistSubs blocks per group, so blocks past T write zero counts.
static_assert(16 * kHistSubs == kWave, "four 16-token blocks per 64-token group");
template <int KMAX>
__global__ __launch_bounds__(256) void route_split_sum_x16(const float* __restrict__ part,
                                                           int64_t T, int K, float eps,
                                                           int mode, int renorm, XTable xt,
                                                           float* __restrict__ logits,
                                                           int* __restrict__ kout,
                                                           int* __restrict__ ids,
                                                           float* __restrict__ wout,
                                                           int* __restrict__ hist,
                                                           int64_t hist_ld) {
    __shared__ float rows[16][65];
    __shared__ int h[64];
    const int tr = threadIdx.x >> 4, sl = threadIdx.x & 15;
    const int64_t t = (int64_t)blockIdx.x * 16 + tr;
    const bool valid = t < T;
    if (threadIdx.x < 64) h[threadIdx.x] = 0;
    float4 v[4];
#pragma unroll
    for (int q = 0; q < 4; ++q)
        v[q] = valid ? *reinterpret_cast<const float4*>(part + ((int64_t)q * T + t) * 64 + 4 * sl)
                     : make_float4(0.f, 0.f, 0.f, 0.f);  // rows past T: finite, never stored
    const float l0 = ((v[0].x + v[1].x) + v[2].x) + v[3].x;
    const float l1 = ((v[0].y + v[1].y) + v[2].y) + v[3].y;
    const float l2 = ((v[0].z + v[1].z) + v[2].z) + v[3].z;
    const float l3 = ((v[0].w + v[1].w) + v[2].w) + v[3].w;
    if (logits && valid) {
        float* const lt = logits + t * 64 + 4 * sl;
        lt[0] = l0;
        lt[1] = l1;
        lt[2] = l2;
        lt[3] = l3;
    }
    float* const row = &rows[tr][0];
    row[4 * sl + 0] = l0;
    row[4 * sl + 1] = l1;
    row[4 * sl + 2] = l2;
    row[4 * sl + 3] = l3;
    __syncthreads();  // h zeroed (and the rows written) before any count
    route_token_x16<KMAX>(row, K, eps, mode, renorm, xt, t, valid, kout, ids, wout, h);
    __syncthreads();
    if (threadIdx.x < 64) {
        const int64_t j = blockIdx.x % kHistSubs, g = blockIdx.x / kHistSubs;
        hist[(j * hist_ld + g) * 64 + threadIdx.x] = h[threadIdx.x];
    }
}

// ---- one launch for router + routing: N = 64, d % 256 == 0, T <= kRouteDmaMaxT ----
//
// router_route_dma: block b takes tokens [16 b, 16 b + 16) (quarter b % 4 of 64-token group
// b / 4), wave w quarter w of the contraction (router_slice), as router_split_bf16 does for
// 64 tokens -- but here the four quarters of a token are in one block, so no partial logits
// leave the chip and the routing follows in the same launch.  Per 64-column chunk of its
// quarter a wave copies the 64 W_r rows and the block's 16 x rows (one 128-byte line per row,
// 16-byte chunks XOR-swizzled by row) straight into its own LDS ring with
// global_load_lds_dwordx4, kDmaRing - 1 chunks ahead, and waits only for its own copies: the
// loop has no barrier.  The MFMA chains, the sum ((P0 + P1) + P2) + P3 and the 16-lane routing
// (route_token_x16) are those of router_split_bf16 + route_split_sum_x16, so the logits,
// k, ids and weights are the same bits.  hist (optional): the block's per-expert assignment
// counts go to histogram b % 4, row b / 4, as route_split_sum_x16 writes them (the grid has
// four blocks per 64-token group; blocks past the last token write zero counts).
constexpr int kDmaRing = 4;                // chunks in a wave's ring
constexpr int kDmaSlot = (64 + 16) * 128;  // bytes per chunk: 64 W_r rows, then 16 x rows
constexpr int kDmaWave = kDmaRing * kDmaSlot;

template <int KMAX>
__global__ __launch_bounds__(256) void router_route_dma(
    const bf16_t* __restrict__ x, const bf16_t* __restrict__ Wr, int64_t T, int d, int K,
    float eps, int mode, int renorm, XTable xt, float* __restrict__ logits,
    int* __restrict__ kout, int* __restrict__ ids, float* __restrict__ wout,
    int* __restrict__ hist, int64_t hist_ld) {
    // the four rings take all of LDS; after the loop a wave's partial tile [16][65] lies at the
    // start of its own ring, and the 64-bin histogram in wave 1's
    __shared__ __attribute__((aligned(1024))) char sm[RW * kDmaWave];
    const int64_t t0 = (int64_t)blockIdx.x * 16;
    if (t0 >= T) {  // a quarter past the last token of the last group: zero counts only
        if (hist && threadIdx.x < 64)
            hist[((int64_t)(blockIdx.x % kHistSubs) * hist_ld + blockIdx.x / kHistSubs) * 64 +
                 threadIdx.x] = 0;
        return;  // block-uniform, before any barrier
    }
    const int lane = threadIdx.x & 63;
    const int w = threadIdx.x >> 6;
    int first, steps;
    router_slice(d, w, first, steps);  // d % 256 == 0: first and steps are even
    const int c0 = first / 2, nc = steps / 2;
    const bf16_t* const xb = x + t0 * d;  // the block's first token row
    // copy sources: W_r rows 8 i + (lane >> 3) (i < 8) and x rows 8 i + (lane >> 3) (i < 2);
    // lane l fills physical chunk l & 7 of its row, i.e. it fetches logical chunk
    // (l & 7) ^ (row & 7).  Rows past T repeat the last token's row (never stored).
    uint32_t woff[8], xoff[2];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        const int r = 8 * i + (lane >> 3);
        const int q = (lane & 7) ^ (r & 7);
        woff[i] = ((uint32_t)r * (uint32_t)d + c0 * 64 + q * 8) * 2u;
    }
#pragma unroll
    for (int i = 0; i < 2; ++i) {
        const int r = 8 * i + (lane >> 3);
        const int q = (lane & 7) ^ (r & 7);
        const int tr = (t0 + r < T) ? r : (int)(T - 1 - t0);
        xoff[i] = ((uint32_t)tr * (uint32_t)d + c0 * 64 + q * 8) * 2u;
    }
    char* const ring = sm + w * kDmaWave;
    const uint32_t lds_ring =
        __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)(lds_void_t*)ring);
    auto issue = [&](int c, int slot) {  // chunk c of the quarter into ring slot `slot`
        const uint32_t base = lds_ring + slot * kDmaSlot;
#pragma unroll
        for (int i = 0; i < 8; ++i)
            asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dwordx4 %1, %2"
                         :: "s"(base + i * 1024), "v"(woff[i] + c * 128), "s"(Wr)
                         : "memory", "m0");
#pragma unroll
        for (int i = 0; i < 2; ++i)
            asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dwordx4 %1, %2"
                         :: "s"(base + 64 * 128 + i * 1024), "v"(xoff[i] + c * 128), "s"(xb)
                         : "memory", "m0");
    };
    f32x4_t acc[4];
#pragma unroll
    for (int g = 0; g < 4; ++g) acc[g] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    const int l16 = lane & 15, hq = lane >> 4;
#pragma unroll
    for (int p = 0; p < kDmaRing - 1; ++p)
        if (p < nc) issue(p, p);
    for (int c = 0; c < nc; ++c) {
        // chunk c is in when at most the copies of the chunks issued after it (at most
        // kDmaRing - 2 of them, ten instructions each) are in flight; its slot's previous
        // chunk (c - 1) was read before its MFMAs, so it is free for chunk c + kDmaRing - 1
        const int left = nc - 1 - c;
        static_assert(kDmaRing == 4, "wait counts below");
        if (left >= 2) ELB_WAIT_VMCNT(20);
        else if (left == 1) ELB_WAIT_VMCNT(10);
        else ELB_WAIT_VMCNT(0);
        // the copies write LDS behind the compiler's back: keep this chunk's reads below the wait
        asm volatile("" ::: "memory");
        if (c + kDmaRing - 1 < nc) issue(c + kDmaRing - 1, (c + kDmaRing - 1) % kDmaRing);
        const char* const sl = ring + (c % kDmaRing) * kDmaSlot;
#pragma unroll
        for (int j = 0; j < 2; ++j) {  // the chunk's two 32-deep k-steps
            const int q = 4 * j + hq;  // logical 16-byte chunk of this lane's 8 k values
            const bf16x8_t a = *reinterpret_cast<const bf16x8_t*>(
                sl + 64 * 128 + l16 * 128 + ((q ^ (l16 & 7)) << 4));
            bf16x8_t b[4];
#pragma unroll
            for (int g = 0; g < 4; ++g) {
                const int n = 16 * g + l16;
                b[g] = *reinterpret_cast<const bf16x8_t*>(sl + n * 128 + ((q ^ (n & 7)) << 4));
            }
#pragma unroll
            for (int g = 0; g < 4; ++g)
                acc[g] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b[g], acc[g], 0, 0, 0);
        }
    }
    // this wave's partial tile (lane: tokens 4 hq + r, expert 16 g + l16) at the start of its
    // own ring: every copy into the ring has landed and every read of it has been used
    float* const pw = reinterpret_cast<float*>(ring);
#pragma unroll
    for (int g = 0; g < 4; ++g)
#pragma unroll
        for (int r = 0; r < 4; ++r) pw[(4 * hq + r) * 65 + 16 * g + l16] = acc[g][r];
    __syncthreads();  // every wave is past its loop and its partial tile is written
    int* const h = reinterpret_cast<int*>(sm + kDmaWave + 16 * 65 * 4);  // in wave 1's ring
    if (threadIdx.x < 64) h[threadIdx.x] = 0;
    // the logits: lane sl of token tr sums elements 4 sl .. 4 sl + 3 of the four partials in
    // order; the sums replace partial 0 (each word read, then written, by one thread)
    const int tr = threadIdx.x >> 4, sl = threadIdx.x & 15;
    const int64_t t = t0 + tr;
    const bool valid = t < T;
    float* const row = reinterpret_cast<float*>(sm) + tr * 65;
    float l4[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int n = 4 * sl + i;
        const float* p0 = reinterpret_cast<const float*>(sm) + tr * 65 + n;
        float v = p0[0];
#pragma unroll
        for (int ww = 1; ww < RW; ++ww) v += p0[ww * (kDmaWave / 4)];
        l4[i] = v;
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) row[4 * sl + i] = l4[i];
    if (logits && valid) {
        float* const lt = logits + t * 64 + 4 * sl;
#pragma unroll
        for (int i = 0; i < 4; ++i) lt[i] = l4[i];
    }
    __syncthreads();  // the logit rows and the zeroed histogram before any count
    route_token_x16<KMAX>(row, K, eps, mode, renorm, xt, t, valid, kout, ids, wout, h);
    if (!hist) return;  // kernel-uniform
    __syncthreads();
    if (threadIdx.x < 64) {
        const int64_t j = blockIdx.x % kHistSubs, g = blockIdx.x / kHistSubs;
        hist[(j * hist_ld + g) * 64 + threadIdx.x] = h[threadIdx.x];
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
    ELB_LAUNCH((router_route_bf16<NP, FULL, KMAX>), dim3((unsigned)((T + 15) / 16)),
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

bool router_route_dma_usable(int dtype, int64_t T, int d, int N, int K) {
    // up to one 16-token block per compute unit (256 on MI355X): above that a second round
    // of blocks costs more than the split form's second launch (measured at 6144 tokens)
    return dtype == ELB_BF16 && N == 64 && K <= kLaneMaxK && T > 0 && T <= kRouteDmaMaxT &&
           d % 256 == 0 && d <= (1 << 20);
}

hipError_t launch_router_route_dma(const void* x, const void* Wr, int64_t T, int d,
                                   const elb_route_params& p, float* logits, int* k, int* ids,
                                   float* w, int* hist, int64_t hist_ld, hipStream_t s) {
    if (T == 0) return hipSuccess;
    ProfileScope prof("router_route_dma", s);
    const dim3 grid((unsigned)(dispatch_groups(T) * kHistSubs));  // every histogram quarter
    const XTable xt = make_xtable(64);
    if (p.K <= 8)
        ELB_LAUNCH(router_route_dma<8>, grid, dim3(256), 0, s, (const bf16_t*)x,
                   (const bf16_t*)Wr, T, d, p.K, p.eps, p.mode, p.renormalize, xt, logits, k,
                   ids, w, hist, hist_ld);
    else
        ELB_LAUNCH(router_route_dma<kLaneMaxK>, grid, dim3(256), 0, s, (const bf16_t*)x,
                   (const bf16_t*)Wr, T, d, p.K, p.eps, p.mode, p.renormalize, xt, logits, k,
                   ids, w, hist, hist_ld);
    return hipGetLastError();
}

bool router_split_usable(int dtype, int64_t T, int d, int N, int K) {
    return dtype == ELB_BF16 && N == 64 && K <= kLaneMaxK && T > kSmallBatch && d % 256 == 0 &&
           d <= (1 << 20);
}

hipError_t launch_router_split_route(const void* x, const void* Wr, int64_t T, int d,
                                     const elb_route_params& p, float* part, float* logits,
                                     int* k, int* ids, float* w, int* hist, int64_t hist_ld,
                                     hipStream_t s) {
    if (T == 0) return hipSuccess;
    const unsigned groups = (unsigned)((T + 63) / 64);
    {
        ProfileScope prof("router_split_bf16", s);
        ELB_LAUNCH(router_split_bf16, dim3(groups, RW), dim3(256), 0, s,
                           (const bf16_t*)x, (const bf16_t*)Wr, T, d, part);
    }
    ProfileScope prof("route_split_sum", s);
    const XTable xt = make_xtable(64);
    if (split_hist_subs(T) == kHistSubs) {  // 16 tokens per block, kHistSubs histograms
        const dim3 grid(groups * kHistSubs);
        if (p.K <= 8)
            ELB_LAUNCH(route_split_sum_x16<8>, grid, dim3(256), 0, s, part, T, p.K, p.eps,
                       p.mode, p.renormalize, xt, logits, k, ids, w, hist, hist_ld);
        else
            ELB_LAUNCH(route_split_sum_x16<kLaneMaxK>, grid, dim3(256), 0, s, part, T, p.K,
                       p.eps, p.mode, p.renormalize, xt, logits, k, ids, w, hist, hist_ld);
        return hipGetLastError();
    }
    if (p.K <= 8)
        ELB_LAUNCH(route_split_sum<8>, dim3(groups), dim3(64), 0, s, part, T, p.K, p.eps,
                   p.mode, p.renormalize, xt, logits, k, ids, w, hist, hist_ld);
    else
        ELB_LAUNCH(route_split_sum<kLaneMaxK>, dim3(groups), dim3(64), 0, s, part, T, p.K,
                   p.eps, p.mode, p.renormalize, xt, logits, k, ids, w, hist, hist_ld);
    return hipGetLastError();
}

bool router_slices_usable(int dtype, int64_t T, int N, int K) {
    return dtype == ELB_BF16 && N == 64 && K <= kLaneMaxK && T > 0 && T <= kSmallBatch;
}

hipError_t launch_router_slices_route(const void* x, const void* Wr, int64_t T, int d,
                                      const elb_route_params& p, float* part, float* logits,
                                      int* k, int* ids, float* w, int* hist, int64_t hist_ld,
                                      hipStream_t s) {
    if (T == 0) return hipSuccess;
    {
        ProfileScope prof("router_slice_bf16", s);
        ELB_LAUNCH(router_slice_bf16, dim3((unsigned)((T + 15) / 16), 4, RW), dim3(64), 0, s,
                   (const bf16_t*)x, (const bf16_t*)Wr, T, d, part);
    }
    ProfileScope prof("route_split_sum", s);
    const dim3 grid((unsigned)(dispatch_groups(T) * kHistSubs));
    const XTable xt = make_xtable(64);
    if (p.K <= 8)
        ELB_LAUNCH(route_split_sum_x16<8>, grid, dim3(256), 0, s, part, T, p.K, p.eps, p.mode,
                   p.renormalize, xt, logits, k, ids, w, hist, hist_ld);
    else
        ELB_LAUNCH(route_split_sum_x16<kLaneMaxK>, grid, dim3(256), 0, s, part, T, p.K, p.eps,
                   p.mode, p.renormalize, xt, logits, k, ids, w, hist, hist_ld);
    return hipGetLastError();
}

hipError_t launch_router(const void* x, const void* Wr, int64_t T, int d, int N, int dtype,
                         float* logits, hipStream_t s) {
    if (T == 0) return hipSuccess;
    if (dtype == ELB_BF16) {
        ProfileScope prof("router_bf16", s);
        if (T <= kSmallBatch)
            ELB_LAUNCH(router_bf16<1>, dim3((unsigned)((T + 15) / 16), (unsigned)((N + 15) / 16)),
                               dim3(64 * RW), 0, s, (const bf16_t*)x, (const bf16_t*)Wr, T, d,
                               N, logits);
        else
            ELB_LAUNCH(router_bf16<4>, dim3((unsigned)((T + 15) / 16)), dim3(64 * RW), 0,
                               s, (const bf16_t*)x, (const bf16_t*)Wr, T, d, N, logits);
    } else {
        ProfileScope prof("router_f32", s);
        ELB_LAUNCH(router_f32, dim3((unsigned)((T * N + 255) / 256)), dim3(256), 0, s,
                           (const float*)x, (const float*)Wr, T, d, N, logits);
    }
    return hipGetLastError();
}

}  // namespace elb
