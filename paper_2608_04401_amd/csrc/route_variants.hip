// Routing variants (Section 2.1, 2.2, 2.3): caps above 16 up to N (the uncapped elbow
// routing is K = N), tail randomisation (the experts after the elbow replaced by experts
// drawn from outside the elbow's selection) and the elbow angle with the uncapped elbow
// index.
//
// One LANE per token with the routing kernel's staging and arithmetic (route_lane.h), but the
// sorting network carries the expert ids along with the logits, so the id at every rank is
// known and any cap up to N costs the same.  Same bits as the routing kernel: the same keys,
// u_i = exp(l_(i) - l_(0)) in rank order (rel_exp), S as the same tree over the ranks
// (tree_sum), the same E_i and first argmin, w = u * (1 / denominator).  The elbow angle (no
// selection asked for) and tail randomisation with K <= 16 sort the keys only.
#include "route_lane.h"

namespace elb {

namespace {

// ---------------------------------------------------------------------------------------
// One LANE per token, (key, id) pairs sorted by a network: the same staging and arithmetic as
// the routing kernel, but the sort carries the expert ids, so every rank's id is known and
// any cap up to N costs no more than K = 1.  A pair is one 64-bit integer: the logit's
// order-preserving integer image in the high word and (NP - 1 - id) in the low word, so one
// signed 64-bit comparison orders by logit descending, then id ascending (pads, -inf with the
// largest ids, sort last).  Each comparator is one v_cmp_gt_i64 and four v_cndmask_b32.
// ---------------------------------------------------------------------------------------

// order-preserving signed integer image of a canonical (non-NaN, no -0) fp32 value; its
// own inverse
__device__ __forceinline__ int ord_flip(int i) { return i ^ ((i >> 31) & 0x7fffffff); }

template <int NP, int Q>
__device__ __forceinline__ void cx_pair(int64_t* v) {
    constexpr int a = NetHolder<NP>::net.a[Q];
    constexpr int b = NetHolder<NP>::net.b[Q];
    const bool sw = v[b] > v[a];
    const int64_t hi = sw ? v[b] : v[a];
    const int64_t lo = sw ? v[a] : v[b];
    v[a] = hi;
    v[b] = lo;
}
template <int NP, int... Q>
__device__ __forceinline__ void sort_pairs_desc(int64_t* v, std::integer_sequence<int, Q...>) {
    (cx_pair<NP, Q>(v), ...);
}

// The experts of the first k ranks from the sorted keys, by the routing kernel's rule
// (select_first_k): their mask `taken`, and up to KM of them in id order (cid) with their keys
// (ck, -inf past k; re-read from the token's LDS row, as the id is not a compile-time
// constant there).
template <int NP, int KM>
__device__ __forceinline__ void first_k_experts(const float (&key)[NP], const float (&okey)[NP],
                                                const float* row, int Nn, int k,
                                                uint64_t& taken, int (&cid)[KM],
                                                float (&ck)[KM]) {
    taken = select_first_k<NP, KM>(key, [&](int c) { return okey[c]; }, Nn, k);
    selected_in_id_order<NP, KM>(taken, [&](int c) { return order_key(row[c]); }, k, cid, ck);
}

// PAIRS: sort (key, id) pairs (a selection with any cap is asked for).  Otherwise the keys
// alone are sorted (the routing kernel's value network: the same sorted keys, so the same e
// and theta bits, at two instructions per comparator): for the elbow angle (no selection), and
// for tail randomisation with K <= kLaneMaxK, whose first k experts are then recovered by the
// routing kernel's selection rule.
template <int NP, bool FULL, bool PAIRS>
__global__ __launch_bounds__(256) void route_pair_kernel(
    const float* __restrict__ logits, const float* __restrict__ rand, int64_t T, int N, int K,
    float eps, int mode, int renorm, int vec4, XTable xt, int* __restrict__ kout,
    int* __restrict__ ids, float* __restrict__ wout, int* __restrict__ eout,
    float* __restrict__ thout) {
    constexpr int LD = NP + 1;
    __shared__ float lds[4 * kWave * LD];
    const int lane = threadIdx.x & (kWave - 1);
    const int wv = threadIdx.x >> 6;
    const int64_t t0 = ((int64_t)blockIdx.x * 4 + wv) * kWave;
    float* tile = lds + wv * kWave * LD;
    int rows = 0;
    if (t0 < T) rows = (int)((T - t0) < kWave ? (T - t0) : kWave);
    stage_rows<NP, FULL>(logits + t0 * N, N, rows, vec4, tile, lane);
    __syncthreads();
    // lanes past the last token route a copy of the first one and write nothing: every lane
    // takes part in the staged stores at the end (no barrier follows)
    const bool active = lane < rows;
    const float* row = tile + (active ? lane : 0) * LD;
    const int64_t t = t0 + (active ? lane : 0);
    const int Nn = FULL ? NP : N;

    // ---- sort (key, id) pairs: rank r holds key[r] and id[r] ----
    float key[NP];
    int id[NP];
    if (PAIRS) {
        int64_t v[NP];
#pragma unroll
        for (int c = 0; c < NP; ++c) {
            const float f = (c < Nn) ? order_key(row[c]) : -INFINITY;
            v[c] = ((int64_t)ord_flip(__float_as_int(f)) << 32) | (uint32_t)(NP - 1 - c);
        }
        sort_pairs_desc<NP>(v, std::make_integer_sequence<int, NetHolder<NP>::net.n>{});
#pragma unroll
        for (int r = 0; r < NP; ++r) {
            key[r] = __int_as_float(ord_flip((int)(v[r] >> 32)));
            id[r] = NP - 1 - (int)(uint32_t)v[r];
        }
    } else {
#pragma unroll
        for (int c = 0; c < NP; ++c) {
            key[c] = (c < Nn) ? order_key(row[c]) : -INFINITY;
            id[c] = 0;  // not used: no selection without PAIRS
        }
        sort_desc<NP>(key, std::make_integer_sequence<int, NetHolder<NP>::net.n>{});
    }

    // ---- u, S, u_min and the elbow: the routing kernel's arithmetic, in rank order ----
    const float nl = neg_scaled(key[0]);
    float u[NP];
#pragma unroll
    for (int i = 0; i < NP; ++i) u[i] = rel_exp(key[i], nl);
    const float S = tree_sum<NP>(u);
    float umin = u[NP - 1];
    if (!FULL) {
#pragma unroll
        for (int i = 0; i < NP; ++i) umin = (i == Nn - 1) ? u[i] : umin;
    }
    const float Rp = (1.0f - umin) + eps * S;
    float best = 1.f;  // E_0 = 1 (D_0 = 0)
    int e = 0;
#pragma unroll
    for (int i = 1; i < NP; ++i) {
        const float Ei = fmaf(xt.x[i], Rp, u[i]);  // pads: x' = +inf, never win
        const bool better = Ei < best;  // strict: the first index wins ties
        best = better ? Ei : best;
        e = better ? i : e;
    }
    if (eout && active) eout[t] = e;
    if (thout && active) {  // the angle at the elbow point (x'_e, p'_e) between (0,0) and (1,1)
        float th = 180.0f;  // e = 0: no point off the chord, a straight curve
        if (e > 0) {
            float xe = 0.f, ue = 0.f;
#pragma unroll
            for (int i = 1; i < NP; ++i) {
                xe = (i == e) ? xt.x[i] : xe;
                ue = (i == e) ? u[i] : ue;
            }
            const float pe = (1.0f - ue) / Rp;
            const float v1x = -xe, v1y = -pe, v2x = 1.0f - xe, v2y = 1.0f - pe;
            const float dot = fmaf(v1x, v2x, v1y * v2y);
            const float crs = fmaf(v1x, v2y, -(v1y * v2x));
            th = atan2f(fabsf(crs), dot) * (180.0f / 3.14159265358979323846f);
        }
        thout[t] = th;
    }
    if (!ids) return;
    const int k = (mode == ELB_MODE_TOPK) ? K : (e + 1 < K ? e + 1 : K);
    if (active) kout[t] = k;

    if (!PAIRS) {
        // tail randomisation with K <= kLaneMaxK from the sorted keys alone: the first k ranks'
        // experts by the routing kernel's selection rule, then the K - k untaken experts with
        // the smallest draws (equal draws: lower id), as below; the same ids and weight bits
        // as the pair path (an elbow expert's u is recomputed from its own key)
        constexpr int KM = NP < kLaneMaxK ? NP : kLaneMaxK;
        float okey[NP];
#pragma unroll
        for (int c = 0; c < NP; ++c) okey[c] = (c < Nn) ? order_key(row[c]) : -INFINITY;
        uint64_t taken;
        int cid[KM];
        float ck[KM];
        first_k_experts<NP, KM>(key, okey, row, Nn, k, taken, cid, ck);
        const float* rr = rand + t * N;
        float draw[NP];
#pragma unroll
        for (int c = 0; c < NP; ++c) draw[c] = (c < Nn) ? rr[c] : INFINITY;
        float denom = S;
        if (renorm) {
            float sel_u[KM];
#pragma unroll
            for (int j = 0; j < KM; ++j) sel_u[j] = j < k ? u[j] : 0.f;
            denom = tree_sum<KM>(sel_u);
        }
        for (int j = k; j < K; ++j) {
            float bv = INFINITY;
            int bc = -1;
#pragma unroll
            for (int c = 0; c < NP; ++c) {
                const bool ok = c < Nn && !((taken >> c) & 1ull) && (bc < 0 || draw[c] < bv);
                bv = ok ? draw[c] : bv;
                bc = ok ? c : bc;
            }
            taken |= 1ull << bc;
            const float ub = rel_exp(order_key(row[bc]), nl);
            if (active) {
                ids[t * K + j] = bc;
                wout[t * K + j] = ub;
            }
            if (renorm) denom += ub;
        }
        const float inv = 1.0f / denom;
        if (!active) return;
        // the elbow's experts at their ranks (descending key; equal keys: lower id first)
#pragma unroll
        for (int r = 0; r < KM; ++r) {
            if (r < k) {
                int rank = 0;
#pragma unroll
                for (int q = 0; q < KM; ++q) {
                    if (q < r) rank += (q < k && ck[q] >= ck[r]) ? 1 : 0;
                    if (q > r) rank += (q < k && ck[q] > ck[r]) ? 1 : 0;
                }
                ids[t * K + rank] = cid[r];
                wout[t * K + rank] = rel_exp(ck[r], nl) * inv;
            }
        }
        for (int j = k; j < K; ++j) wout[t * K + j] *= inv;  // this lane's own writes
        return;
    }

    if (rand) {
        // tail randomisation: K - k experts outside the first k ranks, smallest draws first
        // (equal draws: lower id); weights are the experts' own probabilities
        const float* rr = rand + t * N;
        float draw[NP];
#pragma unroll
        for (int c = 0; c < NP; ++c) draw[c] = (c < Nn) ? rr[c] : INFINITY;
        uint64_t taken = 0;
#pragma unroll
        for (int r = 0; r < NP; ++r)
            if (r < k) taken |= 1ull << id[r];

        float denom = S;
        if (renorm) {
            float sel_u[NP];
#pragma unroll
            for (int j = 0; j < NP; ++j) sel_u[j] = j < k ? u[j] : 0.f;
            denom = tree_sum<NP>(sel_u);
        }
        // pass 1: the tail's ids, with unnormalised weights u (the denominator needs them all)
        for (int j = k; j < K; ++j) {
            float bv = INFINITY;
            int bc = -1;
#pragma unroll
            for (int c = 0; c < NP; ++c) {
                const bool ok = c < Nn && !((taken >> c) & 1ull) && (bc < 0 || draw[c] < bv);
                bv = ok ? draw[c] : bv;
                bc = ok ? c : bc;
            }
            taken |= 1ull << bc;
            const float ub = rel_exp(order_key(row[bc]), nl);
            if (active) {
                ids[t * K + j] = bc;
                wout[t * K + j] = ub;
            }
            if (renorm) denom += ub;
        }
        const float inv = 1.0f / denom;
        if (!active) return;
#pragma unroll
        for (int r = 0; r < NP; ++r) {
            if (r < k) {
                ids[t * K + r] = id[r];
                wout[t * K + r] = u[r] * inv;
            }
        }
        for (int j = k; j < K; ++j) wout[t * K + j] *= inv;  // pass 2 (this lane's own writes)
        return;
    }
    float denom = S;
    if (renorm) {
        float sel_u[NP];
#pragma unroll
        for (int j = 0; j < NP; ++j) sel_u[j] = j < k ? u[j] : 0.f;
        denom = tree_sum<NP>(sel_u);
    }
    const float inv = 1.0f / denom;
    if (K <= 16) {  // few slots: direct stores
        if (!active) return;
#pragma unroll
        for (int r = 0; r < NP; ++r) {
            if (r < k) {
                ids[t * K + r] = id[r];
                wout[t * K + r] = u[r] * inv;
            } else if (r < K) {
                ids[t * K + r] = -1;
                wout[t * K + r] = 0.f;
            }
        }
        return;
    }
    // many slots: stage the wave's 64 output rows in its LDS tile (its logits have been read;
    // a wave's LDS operations complete in order), rows padded to K + 1 words, then store each
    // token's K contiguous values with the whole wave
    int* sti = reinterpret_cast<int*>(tile);
#pragma unroll
    for (int r = 0; r < NP; ++r)
        if (r < K) sti[lane * (K + 1) + r] = (r < k) ? id[r] : -1;
    for (int q = 0; q < rows; ++q)
        for (int c = lane; c < K; c += kWave) ids[(t0 + q) * K + c] = sti[q * (K + 1) + c];
#pragma unroll
    for (int r = 0; r < NP; ++r)
        if (r < K) tile[lane * (K + 1) + r] = (r < k) ? u[r] * inv : 0.f;
    for (int q = 0; q < rows; ++q)
        for (int c = lane; c < K; c += kWave) wout[(t0 + q) * K + c] = tile[q * (K + 1) + c];
}

template <int NP, bool FULL>
void launch_pair_np(const float* logits, const float* rand, int64_t T, int N,
                    const elb_route_params& p, int* k, int* ids, float* w, int* e, float* theta,
                    hipStream_t s) {
    const int64_t waves = (T + kWave - 1) / kWave;
    const int vec4 = ((uintptr_t)logits % 16) == 0;
    const dim3 grid((unsigned)((waves + 3) / 4));
    // keys only: the elbow angle (no ids), or tail randomisation with K <= kLaneMaxK
    const bool keys_only = !ids || (rand && p.K <= kLaneMaxK);
    if (!keys_only)
        ELB_LAUNCH((route_pair_kernel<NP, FULL, true>), grid, dim3(256), 0, s, logits,
                           rand, T, N, p.K, p.eps, p.mode, p.renormalize, vec4, make_xtable(N),
                           k, ids, w, e, theta);
    else
        ELB_LAUNCH((route_pair_kernel<NP, FULL, false>), grid, dim3(256), 0, s, logits,
                           rand, T, N, p.K, p.eps, p.mode, p.renormalize, vec4,
                           make_xtable(N), k, ids, w, e, theta);
}

}  // namespace

hipError_t launch_route_pair(const float* logits, const float* rand, int64_t T, int N,
                             const elb_route_params& p, int* k, int* ids, float* w, int* e,
                             float* theta, hipStream_t s) {
    if (T == 0) return hipSuccess;
    ProfileScope prof("route_pair", s);
    switch (N) {
        case 8: launch_pair_np<8, true>(logits, rand, T, N, p, k, ids, w, e, theta, s); break;
        case 16: launch_pair_np<16, true>(logits, rand, T, N, p, k, ids, w, e, theta, s); break;
        case 32: launch_pair_np<32, true>(logits, rand, T, N, p, k, ids, w, e, theta, s); break;
        case 64: launch_pair_np<64, true>(logits, rand, T, N, p, k, ids, w, e, theta, s); break;
        default:
            if (N < 8)
                launch_pair_np<8, false>(logits, rand, T, N, p, k, ids, w, e, theta, s);
            else if (N < 16)
                launch_pair_np<16, false>(logits, rand, T, N, p, k, ids, w, e, theta, s);
            else if (N < 32)
                launch_pair_np<32, false>(logits, rand, T, N, p, k, ids, w, e, theta, s);
            else
                launch_pair_np<64, false>(logits, rand, T, N, p, k, ids, w, e, theta, s);
    }
    return hipGetLastError();
}

}  // namespace elb
