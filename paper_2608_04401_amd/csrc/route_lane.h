// Routing of ONE token by ONE lane (Section 2, Section 2.1 and Appendix A.1 Algorithm 1):
// softmax, descending sort, Kneedle elbow, cap, weights, from the token's N logits in LDS.
// Shared by the routing kernel and the fused router + routing kernel, so both compute the
// same bits from the same logits.
//
// The normalised curve runs from (0,0) to (1,1), as in the elbow-angle definition of
// Section 2.3: p'_i = (p_(0) - p_(i)) / (p_(0) - p_(N-1) + eps), x'_i = i / (N - 1).
// Arithmetic differs from the definition only by positive scaling, a constant and the sum's
// cancellation, which leave the argmax unchanged:
//   u_i = exp(l_(i) - l_(0)) (so p_(i) = u_i / S, S = sum u), and
//   D_i * (p_max - p_min + eps) * S = 1 - E_i,  E_i = u_i + x'_i * (1 - u_min + eps * S),
// so the first argmax of D is the first argmin of E (one fma per point), with E_0 = 1.
// The sort key is the fp32 logit itself (softmax is strictly increasing), with ties broken
// by the lower expert id, so the ids and their order never depend on exp/division rounding.
// The lane holds the token's N values in registers and sorts them with a compile-time
// odd-even merge network (all register indices are constants): no cross-lane traffic.
#pragma once

#include <utility>

#include "common.h"
#include "sortnet.h"

namespace elb {

namespace {

struct XTable {
    float x[ELB_MAX_EXPERTS];  // x'_i = i / (N - 1), correctly rounded; x[N - 1] == 1
};

constexpr float kLog2e = 1.4426950408889634f;

// u = exp(l - l_max) = 2^(l log2(e) + nl) with the per-token constant nl = -(l_max log2(e)),
// the exponent one fma: every kernel computes a token's u values this way, so all of them
// give the same bits
__device__ __forceinline__ float neg_scaled(float lmax) { return -(lmax * kLog2e); }
__device__ __forceinline__ float rel_exp(float l, float nl) {
    return __builtin_amdgcn_exp2f(fmaf(l, kLog2e, nl));
}

template <int NP>
struct NetHolder {
    static constexpr OddEvenMergeNet<NP> net{};
};
template <int NP, int P>
struct PhasedHolder {
    static constexpr PhasedNet<NP, P> net{};
};

// Sort key of a logit: the value itself, made canonical by an add of +0 (which also turns
// -0 into +0), so that min/max compile to single v_min_f32/v_max_f32.  Non-NaN inputs.
__device__ __forceinline__ float order_key(float f) { return f + 0.0f; }

// One comparator of the network: larger value to the lower position (v_max_f32/v_min_f32).
template <int NP, int Q>
__device__ __forceinline__ void compare_exchange(float* key) {
    constexpr int a = NetHolder<NP>::net.a[Q];
    constexpr int b = NetHolder<NP>::net.b[Q];
    const float hi = fmaxf(key[a], key[b]);
    const float lo = fminf(key[a], key[b]);
    key[a] = hi;
    key[b] = lo;
}

// The whole network as straight-line code (a fold over the comparator indices), so every
// register index is a compile-time constant regardless of loop-unrolling heuristics.
template <int NP, int... Q>
__device__ __forceinline__ void sort_desc(float* key, std::integer_sequence<int, Q...>) {
    (compare_exchange<NP, Q>(key), ...);
}

// Balanced pairwise sum of v[0..n), n a power of two: ((v0 + v1) + (v2 + v3)) + ...  Every
// kernel sums S (and a renormalised denominator) over the ranks in this one order, so that
// all of them give the same bits: a lane that holds all n values adds them in this tree, and
// lanes holding 4 consecutive ranks each add their 4 as (v0 + v1) + (v2 + v3) and then
// combine with an XOR butterfly (partners 1, 2, 4, 8), which walks the same tree (IEEE addition
// is commutative, and adding the exact zeros of masked ranks changes nothing).
template <int n>
__device__ __forceinline__ float tree_sum(const float* v) {
    if constexpr (n == 1) return v[0];
    else return tree_sum<n / 2>(v) + tree_sum<n / 2>(v + n / 2);
}

// index of the lowest set bit of m | 2^top (m's lowest bit if it has one below top, else top)
__device__ __forceinline__ int lowest_bit_or(uint64_t m, int top) {
    return __builtin_ctzll(m | (1ull << top));
}

// x'_i = i / (N - 1), correctly rounded; +inf past N (pads never win the argmax)
inline XTable make_xtable(int N) {
    XTable xt;
    for (int i = 0; i < ELB_MAX_EXPERTS; ++i)
        xt.x[i] = (i < N) ? (float)((double)i / (double)(N - 1)) : INFINITY;
    return xt;
}

// Stage a wave's `rows` token rows (rows * N contiguous floats at src) into its LDS tile,
// row r at tile + r * (NP + 1), with coalesced loads: every load of the lane is issued before
// the first LDS write, so the wave waits for memory once.  vec4: src is 16-byte aligned.
template <int NP, bool FULL>
__device__ __forceinline__ void stage_rows(const float* __restrict__ src, int N, int rows,
                                           int vec4, float* tile, int lane) {
    constexpr int LD = NP + 1;
    if (FULL && vec4) {
        constexpr int PER = NP / 4;  // float4 per lane (64 rows x NP / 4 per wave)
        const int total4 = rows * (NP / 4);
        float4 q[PER];
#pragma unroll
        for (int it = 0; it < PER; ++it) {
            const int i = lane + it * kWave;
            if (rows == kWave || i < total4) q[it] = reinterpret_cast<const float4*>(src)[i];
        }
        __builtin_amdgcn_sched_barrier(0);  // keep every load ahead of the first write
#pragma unroll
        for (int it = 0; it < PER; ++it) {
            const int i = lane + it * kWave;
            const int r = i / (NP / 4);
            const int c = (i % (NP / 4)) * 4;
            if (rows == kWave || i < total4) {
                float* dst = tile + r * LD + c;
                dst[0] = q[it].x; dst[1] = q[it].y; dst[2] = q[it].z; dst[3] = q[it].w;
            }
        }
    } else {
        const int total = rows * N;
        for (int i = lane; i < total; i += kWave) {
            const int r = i / N;
            tile[r * LD + (i - r * N)] = src[i];
        }
    }
}

// LDS DMA layout of a wave's 64 x NP tile: P parts of CP 16-byte chunks per row; chunk cc of
// part p of row r sits at 16-byte slot p 64 CP + r CP + (cc ^ swz(r)), so that for a fixed
// chunk 16 consecutive rows fall in 16 distinct groups of 4 banks.
constexpr int kRouteParts = 2;  // parts of the copy (a power of two)

template <int NP>
struct DmaTile {
    static constexpr int C = NP / 4;              // 16-byte chunks per row
    static constexpr int P = C >= kRouteParts ? kRouteParts : C;  // parts
    static constexpr int CP = C / P;              // chunks per row per part
    static constexpr int B = NP / P;              // floats per row per part
    static constexpr int RPG = 16 / CP;           // rows per swizzle period
    __device__ static int swz(int r) { return (r / RPG) % CP; }
    // float index of value c (0 <= c < NP) of row r
    __device__ static int at(int r, int c) {
        const int p = c / B, cc = (c % B) / 4;
        return ((p * 64 * CP + r * CP + (cc ^ swz(r))) << 2) + (c & 3);
    }
};

// Copy rows [0, rows) of a row-major 64 x NP fp32 tile at src (rows past `rows` repeat row
// rows - 1, never used) into a wave's LDS tile in the DmaTile layout, with
// global_load_lds_dwordx4 (whole 128-byte lines of every row per instruction; no registers);
// part p of every row is issued before part p + 1.  The caller waits (vmcnt) before reading.
template <int NP>
__device__ __forceinline__ void dma_tile(const float* src, int rows, float* tile, int lane) {
    using L = DmaTile<NP>;
    const uint32_t lds0 = (uint32_t)(uintptr_t)(lds_void_t*)tile;
#pragma unroll
    for (int p = 0; p < L::P; ++p)
#pragma unroll
        for (int j = 0; j < L::CP; ++j) {
            const int local = j * 64 + lane;
            const int r = local / L::CP;
            const int cc = (local % L::CP) ^ L::swz(r);
            const int rs = r < rows ? r : rows - 1;
            const uint32_t va = (uint32_t)(rs * NP + (p * L::CP + cc) * 4) * 4u;
            const uint32_t la =
                __builtin_amdgcn_readfirstlane(lds0 + (p * 64 * L::CP + j * 64) * 16);
            asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dwordx4 %1, %2"
                         :: "s"(la), "v"(va), "s"(src) : "memory", "m0");
        }
}

// ---- the per-token steps, shared by every kernel that routes in one lane ----

// u_i = exp(l_(i) - l_(0)) in rank order (0 for pads), S = sum u over the ranks (tree_sum),
// and the elbow's k (K in top-K mode) from the sorted keys.
template <int NP, bool FULL, int KMAX>
__device__ __forceinline__ int sorted_elbow(const float (&key)[NP], int Nn, int K, float eps,
                                            int mode, const XTable& xt, float (&u)[NP],
                                            float& S) {
    constexpr int KM = NP < KMAX ? NP : KMAX;
    const float nl = neg_scaled(key[0]);
#pragma unroll
    for (int i = 0; i < NP; ++i) u[i] = rel_exp(key[i], nl);
    S = tree_sum<NP>(u);
    float umin = u[NP - 1];
    if (!FULL) {
#pragma unroll
        for (int i = 0; i < NP; ++i) umin = (i == Nn - 1) ? u[i] : umin;
    }
    int k = K;
    if (mode == ELB_MODE_ELBOW) {
        // E_i = u_i + x'_i (1 - u_min + eps S), E_0 = 1 (D_0 = 0).  The first argmin only
        // matters below K - 1 (beyond it k = K), so later points need only a min.  Pads have
        // x' = +inf and never win.
        const float Rp = (1.0f - umin) + eps * S;
        float best = 1.f;
        int e = 0;
        float tail = INFINITY;
#pragma unroll
        for (int i = 1; i < NP; ++i) {
            const float Ei = fmaf(xt.x[i], Rp, u[i]);
            if (i < KM - 1) {
                const bool head = i < K - 1;
                const bool better = head && (Ei < best);  // strict: first index wins ties
                best = better ? Ei : best;
                e = better ? i : e;
                tail = head ? tail : fminf(tail, Ei);
            } else {
                tail = fminf(tail, Ei);
            }
        }
        k = (tail < best) ? K : e + 1;
    }
    return k;
}

// The experts of the first k ranks of the sorted order (keys descending, equal keys by lower
// expert id), from the sorted keys: tau = the key at rank k - 1; every expert whose key is
// above tau, then the experts whose key equals tau, lowest ids first.  okey(c): expert c's
// key (c a compile-time constant).  Returns them as a 64-bit mask over expert ids.  Shared by
// every kernel that selects from sorted keys alone.
template <int NP, int KM, class OKey>
__device__ __forceinline__ uint64_t select_first_k(const float (&key)[NP], OKey&& okey,
                                                   int Nn, int k, float* tau_out = nullptr) {
    float tau = key[0];
#pragma unroll
    for (int i = 0; i < KM; ++i)
        if (i == k - 1) tau = key[i];
    if (tau_out) *tau_out = tau;
    // common case: exactly k experts have a key >= tau (no tie at the boundary).  okey(c) >= tau
    // exactly when okey(c) - tau' is not negative, tau' being tau with a zero made -0 (so that
    // the keys -0 and +0, equal as floats, both give +0; a finite difference keeps its sign
    // even when it underflows): one subtraction per expert, its sign bit shifted into a word
    // by v_alignbit, instead of a compare and a select.  tau = -inf selects every expert.
    const float tau2 = (tau == 0.f) ? -0.f : tau;
    constexpr int n0 = NP < 32 ? NP : 32;
    uint32_t w0 = 0;  // after the loop, bit n0 - 1 - c: okey(c) < tau
#pragma unroll
    for (int c = 0; c < n0; ++c)
        w0 = __builtin_amdgcn_alignbit(w0, __float_as_uint(okey(c) - tau2), 31);
    uint64_t neg = __builtin_bitreverse32(w0) >> (32 - n0);
    if constexpr (NP > 32) {
        uint32_t w1 = 0;
#pragma unroll
        for (int c = 32; c < NP; ++c)
            w1 = __builtin_amdgcn_alignbit(w1, __float_as_uint(okey(c) - tau2), 31);
        neg |= (uint64_t)(__builtin_bitreverse32(w1) >> (64 - NP)) << 32;
    }
    const uint64_t real = Nn >= 64 ? ~0ull : ((1ull << Nn) - 1);
    uint64_t sel = (tau == -INFINITY) ? real : (~neg & real);
    const bool tie = __popcll(sel) != k;
    if (__builtin_expect(__any(tie), 0)) {  // wave-uniform slow path: ties at tau
        int g = 0;  // ranks < k with a key above tau
#pragma unroll
        for (int i = 0; i < KM; ++i)
            if (i < k && key[i] > tau) ++g;
        uint64_t eq = 0;
        sel = 0;
#pragma unroll
        for (int c = 0; c < NP; ++c) {
            const bool real = c < Nn;
            if (real && okey(c) > tau) sel |= 1ull << c;
            if (real && okey(c) == tau) eq |= 1ull << c;
        }
        for (int r = 0; r < k - g; ++r) {
            const uint64_t low = eq & (~eq + 1);  // lowest set bit
            sel |= low;
            eq ^= low;
        }
    }
    return sel;
}

// The k selected experts (select_first_k) in increasing id order, with their keys: cid[r],
// ck[r] for r < k; ck = -inf (and cid a valid id) for k <= r < KM.  key_of(c): expert c's key
// re-read from memory (c is not a compile-time constant there).
template <int NP, int KM, class KeyOf>
__device__ __forceinline__ void selected_in_id_order(uint64_t sel, KeyOf&& key_of, int k,
                                                     int (&cid)[KM], float (&ck)[KM]) {
#pragma unroll
    for (int r = 0; r < KM; ++r) {
        const int b = lowest_bit_or(sel, NP - 1);  // r >= k: no bit left, a valid id
        const float kb = key_of(b);                // read on every lane: no branch
        cid[r] = b;
        ck[r] = r < k ? kb : -INFINITY;
        sel &= sel - 1;
    }
}

// The k selected experts (the k largest keys, equal keys by lower id) with their weights,
// handed to emit(rank, id, w) in no particular order of rank, then emit(j, -1, 0) for
// k <= j < K.  okey(c): expert c's key (c a compile-time constant); key_of(c): expert c's key
// re-read from memory (c is not a compile-time constant there).
template <int NP, bool FULL, int KMAX, class OKey, class KeyOf, class Emit>
__device__ __forceinline__ void select_emit(const float (&key)[NP], OKey&& okey,
                                            KeyOf&& key_of, int Nn, int K, int k,
                                            const float (&u)[NP], float S, int renorm,
                                            Emit&& emit) {
    constexpr int KM = NP < KMAX ? NP : KMAX;
    const float nl = neg_scaled(key[0]);
    float tau;
    const uint64_t sel = select_first_k<NP, KM>(key, okey, Nn, k, &tau);
    int cid[KM];
    float ck[KM];
    selected_in_id_order<NP, KM>(sel, key_of, k, cid, ck);
    float denom = S;
    if (renorm) {
        float sel_u[KM];
#pragma unroll
        for (int j = 0; j < KM; ++j) sel_u[j] = j < k ? u[j] : 0.f;
        denom = tree_sum<KM>(sel_u);
    }
    const float inv = 1.0f / denom;
    // Common case, wave-uniform: the k selected keys are distinct and finite.  Then rank j's
    // expert is the one selected expert whose key equals key[j], and its weight is u_j / S
    // (u_j is rel_exp(key[j], nl), the same bits as from the expert's own key).
    bool distinct = tau != -INFINITY;
#pragma unroll
    for (int j = 0; j + 1 < KM; ++j)
        if (j + 1 < k && key[j] == key[j + 1]) distinct = false;
    if (__builtin_expect(__all(distinct), 1)) {
#pragma unroll
        for (int j = 0; j < KM; ++j) {
            if (j < k) {
                int id = cid[0];
#pragma unroll
                for (int r = 0; r < KM; ++r) id = (ck[r] == key[j]) ? cid[r] : id;
                emit(j, id, u[j] * inv);
            }
        }
    } else {
        // rank of each in descending order (equal keys: lower id, i.e. lower r, first)
#pragma unroll
        for (int r = 0; r < KM; ++r) {
            if (r < k) {
                int rank = 0;
#pragma unroll
                for (int q = 0; q < KM; ++q) {
                    if (q < r) rank += (q < k && ck[q] >= ck[r]) ? 1 : 0;
                    if (q > r) rank += (q < k && ck[q] > ck[r]) ? 1 : 0;
                }
                emit(rank, cid[r], rel_exp(ck[r], nl) * inv);
            }
        }
    }
#pragma unroll
    for (int j = 0; j < KM; ++j)
        if (j >= k && j < K) emit(j, -1, 0.f);
}

// Token t's routing from row[0..N) (LDS).  FULL: N == NP, so every "position < N" test is
// static; KMAX: a bound on K (8 or 16).  Writes k[t], ids[t, 0..K), w[t, 0..K).
template <int NP, bool FULL, int KMAX>
__device__ __forceinline__ void route_token(const float* row, int N, int K, float eps,
                                            int mode, int renorm, const XTable& xt, int64_t t,
                                            int* __restrict__ kout, int* __restrict__ ids,
                                            float* __restrict__ wout) {
    const int Nn = FULL ? NP : N;
    // ---- keys of the token's logits (pads are -inf and sort last) ----
    float key[NP], okey[NP];
#pragma unroll
    for (int c = 0; c < NP; ++c) {
        okey[c] = (c < Nn) ? order_key(row[c]) : -INFINITY;
        key[c] = okey[c];
    }
    sort_desc<NP>(key, std::make_integer_sequence<int, NetHolder<NP>::net.n>{});
    float u[NP], S;
    const int k = sorted_elbow<NP, FULL, KMAX>(key, Nn, K, eps, mode, xt, u, S);
    kout[t] = k;
    select_emit<NP, FULL, KMAX>(
        key, [&](int c) { return okey[c]; }, [&](int c) { return order_key(row[c]); }, Nn, K,
        k, u, S, renorm,
        [&](int j, int id, float w) {
            ids[t * K + j] = id;
            wout[t * K + j] = w;
        });
}

// ---- one token by 16 lanes (N = 64): for latency, where few tokens are routed at once ----
//
// The same keys, u, S, deviations, first argmin and weights as route_token, bit for bit, with
// the work spread over 16 consecutive lanes of a wave, one 16-lane DPP row (lane sl holds
// ranks 4 sl .. 4 sl + 3): the (key, id) pairs are sorted by a bitonic network whose strides
// of 4 and more cross lanes (row exchanges by DPP); S (and the renormalised denominator) is
// the tree_sum order walked by an XOR butterfly; the first argmin of E and the tail minimum
// are exact reductions over the row.

// the order-preserving integer image of a canonical fp32 value, and its inverse
__device__ __forceinline__ int ord_flip32(int i) { return i ^ ((i >> 31) & 0x7fffffff); }

// The value of lane l ^ M (M = 1, 2, 4, 8) inside each 16-lane row, by DPP: a modifier of one
// VALU move, with no LDS round trip (a ds_bpermute costs one, and the 16-lane routing's
// exchanges form a dependent chain).  M = 1, 2: quad permutations; M = 8: rotation of the row
// by 8; M = 4: rotations by 4 and by 12, chosen by lane bit 2 (lane l takes lane (l - 4)
// mod 16 or (l - 12) mod 16, whichever is l ^ 4).
template <int M>
__device__ __forceinline__ int xor16(int v) {
    static_assert(M == 1 || M == 2 || M == 4 || M == 8, "row exchange");
    if constexpr (M == 1) return __builtin_amdgcn_update_dpp(0, v, 0xB1, 0xF, 0xF, false);
    else if constexpr (M == 2) return __builtin_amdgcn_update_dpp(0, v, 0x4E, 0xF, 0xF, false);
    else if constexpr (M == 8) return __builtin_amdgcn_update_dpp(0, v, 0x128, 0xF, 0xF, false);
    else {
        const int r4 = __builtin_amdgcn_update_dpp(0, v, 0x124, 0xF, 0xF, false);
        const int r12 = __builtin_amdgcn_update_dpp(0, v, 0x12C, 0xF, 0xF, false);
        return (threadIdx.x & 4) ? r4 : r12;
    }
}
template <int M>
__device__ __forceinline__ float xor16f(float v) {
    return __int_as_float(xor16<M>(__float_as_int(v)));
}
template <int M>
__device__ __forceinline__ int64_t xor16_64(int64_t v) {
    const int lo = xor16<M>((int)(uint32_t)v);
    const int hi = xor16<M>((int)(v >> 32));
    return ((int64_t)hi << 32) | (uint32_t)lo;
}
__device__ __forceinline__ int64_t xor16_64(int64_t v, int m) {  // m a constant after unrolling
    switch (m) {
        case 1: return xor16_64<1>(v);
        case 2: return xor16_64<2>(v);
        case 4: return xor16_64<4>(v);
        default: return xor16_64<8>(v);
    }
}
// lane 0 (first) or lane 15 (last) of each 16-lane row, by a swizzle (bit mode: lane & 0x10,
// or 0x0f)
__device__ __forceinline__ float row_first(float v) {
    return __int_as_float(__builtin_amdgcn_ds_swizzle(__float_as_int(v), 0x10));
}
__device__ __forceinline__ float row_last(float v) {
    return __int_as_float(__builtin_amdgcn_ds_swizzle(__float_as_int(v), 0x10 | (0x0f << 5)));
}

// row: the token's 64 logits in LDS; every lane of the group calls this (valid: the token
// exists; only valid groups write)
// lds_hist (optional): a 64-bin LDS histogram to which each selected expert of a valid token
// adds one (the dispatch's per-group counts).
template <int KMAX>
__device__ __forceinline__ void route_token_x16(float* row, int K, float eps, int mode,
                                                int renorm, const XTable& xt, int64_t t,
                                                bool valid, int* __restrict__ kout,
                                                int* __restrict__ ids,
                                                float* __restrict__ wout,
                                                int* lds_hist = nullptr) {
    constexpr int NP = 64;
    const int sl = threadIdx.x & 15;
    // ---- (key, id) pairs of positions 4 sl + i: key image high, 63 - id low ----
    int64_t v[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int c = 4 * sl + i;
        v[i] = ((int64_t)ord_flip32(__float_as_int(order_key(row[c]))) << 32) |
               (uint32_t)(NP - 1 - c);
    }
    // ---- bitonic sort, descending: position p = 4 sl + i ----
#pragma unroll
    for (int k = 2; k <= NP; k <<= 1) {
#pragma unroll
        for (int j = k >> 1; j >= 1; j >>= 1) {
            if (j >= 4) {
                const int m = j >> 2;  // partner lane sl ^ m, same i
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const int p = 4 * sl + i;
                    const int64_t w = xor16_64(v[i], m);
                    const bool desc = (p & k) == 0 || k == NP;
                    const bool lower = (p & j) == 0;
                    const bool take_max = lower == desc;
                    const bool gt = w > v[i];
                    v[i] = (gt == take_max) ? w : v[i];
                }
            } else {
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    if (i & j) continue;
                    const int p = 4 * sl + i;
                    const bool desc = (p & k) == 0 || k == NP;
                    const int64_t a = v[i], b = v[i | j];
                    const bool sw = desc ? (b > a) : (a > b);
                    v[i] = sw ? b : a;
                    v[i | j] = sw ? a : b;
                }
            }
        }
    }
    float key[4];
    int id[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        key[i] = __int_as_float(ord_flip32((int)(v[i] >> 32)));
        id[i] = NP - 1 - (int)(uint32_t)v[i];
    }
    const float nl = neg_scaled(row_first(key[0]));
    float u[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) u[i] = rel_exp(key[i], nl);
    // ---- S over the ranks (tree_sum by a butterfly), u_min = u of rank 63 ----
    float S = (u[0] + u[1]) + (u[2] + u[3]);
    S += xor16f<1>(S);
    S += xor16f<2>(S);
    S += xor16f<4>(S);
    S += xor16f<8>(S);
    const float umin = row_last(u[3]);
    int k = K;
    if (mode == ELB_MODE_ELBOW) {
        const float Rp = (1.0f - umin) + eps * S;
        float bd = (sl == 0) ? 1.f : INFINITY;  // E_0 = 1
        int be = (sl == 0) ? 0 : NP;
        float tail = INFINITY;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int r = 4 * sl + i;
            if (r == 0) continue;
            const float Ei = fmaf(xt.x[r], Rp, u[i]);
            if (r < K - 1) {
                if (Ei < bd) {  // strict: ranks rise with i, so the first index wins ties
                    bd = Ei;
                    be = r;
                }
            } else {
                tail = fminf(tail, Ei);
            }
        }
        auto step = [&](float obd, int obe, float ot) {
            if (obd < bd || (obd == bd && obe < be)) {
                bd = obd;
                be = obe;
            }
            tail = fminf(tail, ot);
        };
        step(xor16f<8>(bd), xor16<8>(be), xor16f<8>(tail));
        step(xor16f<4>(bd), xor16<4>(be), xor16f<4>(tail));
        step(xor16f<2>(bd), xor16<2>(be), xor16f<2>(tail));
        step(xor16f<1>(bd), xor16<1>(be), xor16f<1>(tail));
        k = (tail < bd) ? K : be + 1;
    }
    float denom = S;
    if (renorm) {  // the selected ranks' u, the others as exact zeros, in the same tree
        float m4[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) m4[i] = (4 * sl + i < k) ? u[i] : 0.f;
        denom = (m4[0] + m4[1]) + (m4[2] + m4[3]);
        denom += xor16f<1>(denom);
        denom += xor16f<2>(denom);
        denom += xor16f<4>(denom);
        denom += xor16f<8>(denom);
    }
    const float inv = 1.0f / denom;
    if (!valid) return;
    if (sl == 0) kout[t] = k;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int r = 4 * sl + i;
        if (r < K) {
            ids[t * K + r] = (r < k) ? id[i] : -1;
            wout[t * K + r] = (r < k) ? u[i] * inv : 0.f;
        }
        if (lds_hist && r < k) atomicAdd(&lds_hist[id[i]], 1);
    }
}

}  // namespace

}  // namespace elb
