// Grouped expert GEMMs for decode-sized batches: weight streaming (gemm_stream.h).
//
// With a few tokens per expert (T K / N of order 10) the expert GEMMs are matrix-vector
// products in disguise: every used expert's weights are read once from HBM and each weight
// is used for only a handful of FLOPs, so the kernels are bound by HBM bandwidth, not by the
// matrix cores.  The design follows from that:
//  - the weights are the streamed operand.  One wave owns a task (expert e, a slice of 64
//    weight rows) and walks the contraction dimension in 64-deep stages, loading each weight
//    row as whole 128-byte lines straight into MFMA operand registers (no LDS), two stages
//    in flight;
//  - the expert's token rows are the small operand (chunks of up to 32 rows, 2 tiles of
//    16), read from L2, where the expert's other waves also find them;
//  - v_mfma_f32_16x16x32_bf16 with the WEIGHTS as the first operand: the output tile is
//    (weight row) x (token), so a lane holds 4 consecutive output columns of one token row;
//  - experts without tokens cost nothing: their waves exit before any load;
//  - gate/up: a task is 32 H columns, i.e. its 32 gate rows and the 32 matching up rows, so
//    SwiGLU is applied in registers and H is written once (bf16); down: a task is 64 Y
//    columns.
// An expert with more than 32 rows is processed in chunks of 32 rows, re-reading its
// weights per chunk (rare where this path is chosen: at most 16 rows per expert on
// average).
//
// Block -> task mapping: 4 waves per block take 4 consecutive tasks of one expert; blocks
// are numbered expert-major and each of the 8 XCDs (block b runs on XCD b % 8) takes a
// contiguous range of them, so an expert's token rows are shared through one XCD's L2.
#include "gemm_stream.h"

namespace elb {

namespace {

constexpr int SK_MAXMT = 2;  // token tiles of 16 rows per chunk (32 rows)

// One chunk of up to 16 * MT token rows of a task over the whole contraction.
template <int MODE, int MT, bool PACKED>
__device__ __forceinline__ void skinny_chunk(const bf16_t* const (&wp)[SK_NF],
                                             const bf16_t* const (&xp)[SK_MAXMT], int kd,
                                             int rows, int64_t out_row0, int out_ld,
                                             int out_col, bf16_t* __restrict__ C, int lane,
                                             const int* slots) {
    f32x4_t acc[MT][SK_NF];
#pragma unroll
    for (int t = 0; t < MT; ++t)
#pragma unroll
        for (int f = 0; f < SK_NF; ++f) acc[t][f] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    stream_mma<MT, SK_MAXMT, 3, PACKED>(wp, xp, 0, kd / 64, acc);
    stream_store<MODE, MT>(acc, rows, out_row0, out_ld, out_col, C, lane, slots);
}

// The assignment slots s = t K + j (j < k_t) routed to expert e, in increasing order (so in
// increasing token order, as the dispatch orders an expert's rows), gathered by one wave into
// its LDS list; returns their number.  T K <= kSlotMax on this path.
constexpr int kSlotMax = 16 * ELB_MAX_EXPERTS;  // T K <= 16 N
__device__ __forceinline__ int gather_slots(const int* __restrict__ k,
                                            const int* __restrict__ ids, int T, int K, int e,
                                            int* list, int lane) {
    const uint64_t below = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
    int n = 0;
    // four 64-slot chunks per pass, their loads issued together (one memory round trip)
    for (int base = 0; base < T * K; base += 4 * kWave) {
        int id4[4], k4[4];
#pragma unroll
        for (int c = 0; c < 4; ++c) {
            const int slot = base + c * kWave + lane;
            id4[c] = (slot < T * K) ? ids[slot] : -1;
            k4[c] = (slot < T * K) ? k[slot / K] : 0;
        }
#pragma unroll
        for (int c = 0; c < 4; ++c) {
            const int slot = base + c * kWave + lane;
            const bool hit = id4[c] == e && slot - (slot / K) * K < k4[c];
            const uint64_t b = __ballot(hit);
            if (hit) list[n + __popcll(b & below)] = slot;
            n += __popcll(b);
        }
    }
    return n;
}

// MODE 0: A = x [T, d], W = W_gate_up [N, 2m, d], C = H [T K, m]
// MODE 1: A = H [T K, m], W = W_down [N, d, m], C = Y [T K, d]
// Rows are assignment slots t K + j, found by each wave from the routing itself (k, ids):
// no dispatch pass; every expert's waves write their slots' rows of H and Y, and the combine
// reads row t K + j.  counts (optional): assignments per expert, by each expert's first task.
// PACKED: W is the packed copy of those weights (elb_pack_expert_weights)
template <int MODE, bool PACKED>
// (2 waves per SIMD: the register ring of three stages fits in 256 registers)
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(2, 2))) void gemm_skinny(
    const bf16_t* __restrict__ A, const int* __restrict__ k, const int* __restrict__ ids,
    int T, int K, const bf16_t* __restrict__ W, int N, int d, int m, bf16_t* __restrict__ C,
    int* __restrict__ counts) {
    __shared__ int slots[4][kSlotMax];
    const int lane = threadIdx.x & 63;
    const int per_e = (MODE == 0) ? m / 32 : d / 64;  // tasks per expert
    const int nblk = (N * per_e + 3) / 4;
    const int per = (nblk + 7) >> 3;
    const int s = blockIdx.x >> 3;
    const int L = (blockIdx.x & 7) * per + s;
    if (s >= per || L >= nblk) return;
    const int task = L * 4 + (threadIdx.x >> 6);
    if (task >= N * per_e) return;  // wave-uniform; the kernel has no barriers
    const int e = task / per_e, c = task - e * per_e;
    int* list = slots[threadIdx.x >> 6];
    const int nrows = gather_slots(k, ids, T, K, e, list, lane);
    if (counts && c == 0 && lane == 0) counts[e] = nrows;
    if (nrows <= 0) return;

    const int kd = (MODE == 0) ? d : m;
    const int out_ld = (MODE == 0) ? m : d;
    const int out_col = (MODE == 0) ? 32 * c : 64 * c;
    for (int cb = 0; cb < nrows; cb += 16 * SK_MAXMT) {
        const int rows = nrows - cb < 16 * SK_MAXMT ? nrows - cb : 16 * SK_MAXMT;
        const bf16_t* wp[SK_NF];
        const bf16_t* xp[SK_MAXMT];
        stream_task<MODE, SK_MAXMT>(A, nullptr, W, e, c, cb, rows, d, m, lane, wp, xp, list, K);
        if (PACKED) stream_task_packed<MODE>(W, e, c, d, m, lane, wp);
        if (rows <= 16)
            skinny_chunk<MODE, 1, PACKED>(wp, xp, kd, rows, cb, out_ld, out_col, C, lane, list);
        else
            skinny_chunk<MODE, 2, PACKED>(wp, xp, kd, rows, cb, out_ld, out_col, C, lane, list);
    }
}

// Packing: one thread per 16-byte operand of the packed copy, in packed order, gathered from
// the row-major weights (gate/up then down; the packed copy has the same size).
__global__ __launch_bounds__(256) void pack_experts(const bf16_t* __restrict__ Wgu,
                                                    const bf16_t* __restrict__ Wd, int N, int d,
                                                    int m, bf16_t* __restrict__ P) {
    const int64_t n_gu = (int64_t)N * 2 * m * d / 8;  // 16-byte operands of W_gate_up
    const int64_t n_all = n_gu + (int64_t)N * d * m / 8;
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i >= n_all) return;
    const bool gu = i < n_gu;
    const int64_t j = gu ? i : i - n_gu;
    const int lane = (int)(j % 64);
    int64_t q = j / 64;
    const int f = (int)(q % 4);
    q /= 4;
    const int h = (int)(q % 2);
    q /= 2;
    const int ns = (gu ? d : m) / 64;
    const int s = (int)(q % ns);
    q /= ns;
    const int per_e = gu ? m / 32 : d / 64;
    const int c = (int)(q % per_e);
    const int e = (int)(q / per_e);
    const int l16 = lane & 15, kq = (lane >> 4) * 8;
    const int k = 64 * s + 32 * h + kq;
    int64_t src;
    if (gu) {
        const int wrow = (f < 2) ? 32 * c + 16 * f + l16 : m + 32 * c + 16 * (f - 2) + l16;
        src = ((int64_t)e * 2 * m + wrow) * d + k;
    } else {
        src = ((int64_t)e * d + 64 * c + 16 * f + l16) * m + k;
    }
    const u32x4_t v = *reinterpret_cast<const u32x4_t*>((gu ? Wgu : Wd) + src);
    *reinterpret_cast<u32x4_t*>(P + i * 8) = v;
}

unsigned blocks_for(int tasks) { return (unsigned)(((tasks + 3) / 4 + 7) / 8 * 8); }

}  // namespace

bool gemm_use_skinny(int dtype, int64_t T, int K, int N, int d, int m) {
    // at most 16 rows per expert on average: far below the bf16 ridge point (~300 rows), so
    // the weight stream bounds the GEMMs (T K <= 16 N <= kSlotMax, the waves' slot lists)
    return dtype == ELB_BF16 && T > 0 && T * K <= (int64_t)16 * N && m % 32 == 0 &&
           d % 64 == 0 && m % 64 == 0;
}

hipError_t launch_gemm_skinny(const void* x, const void* Wgu, const void* Wd, const void* packed,
                              const int* k, const int* ids, int64_t T, int K, int d, int N,
                              int m, void* H, void* Y, int* counts, hipStream_t s) {
    const bf16_t* pgu = (const bf16_t*)packed;
    const bf16_t* pd = pgu ? pgu + (int64_t)N * 2 * m * d : nullptr;
    const int t = (int)T;
    {
        ProfileScope prof("gemm_gate_up_skinny", s);
        if (pgu)
            ELB_LAUNCH((gemm_skinny<0, true>), dim3(blocks_for(N * (m / 32))), dim3(256),
                               0, s, (const bf16_t*)x, k, ids, t, K, pgu, N, d, m, (bf16_t*)H,
                               counts);
        else
            ELB_LAUNCH((gemm_skinny<0, false>), dim3(blocks_for(N * (m / 32))),
                               dim3(256), 0, s, (const bf16_t*)x, k, ids, t, K,
                               (const bf16_t*)Wgu, N, d, m, (bf16_t*)H, counts);
    }
    if (hipError_t e = hipGetLastError(); e != hipSuccess) return e;
    {
        ProfileScope prof("gemm_down_skinny", s);
        if (pd)
            ELB_LAUNCH((gemm_skinny<1, true>), dim3(blocks_for(N * (d / 64))), dim3(256),
                               0, s, (const bf16_t*)H, k, ids, t, K, pd, N, d, m, (bf16_t*)Y,
                               (int*)nullptr);
        else
            ELB_LAUNCH((gemm_skinny<1, false>), dim3(blocks_for(N * (d / 64))),
                               dim3(256), 0, s, (const bf16_t*)H, k, ids, t, K,
                               (const bf16_t*)Wd, N, d, m, (bf16_t*)Y, (int*)nullptr);
    }
    return hipGetLastError();
}

hipError_t launch_pack_experts(const void* Wgu, const void* Wd, int N, int d, int m,
                               void* packed, hipStream_t s) {
    const int64_t n_all = ((int64_t)N * 2 * m * d + (int64_t)N * d * m) / 8;
    if (n_all == 0) return hipSuccess;
    ProfileScope prof("pack_experts", s);
    ELB_LAUNCH(pack_experts, dim3((unsigned)((n_all + 255) / 256)), dim3(256), 0, s,
                       (const bf16_t*)Wgu, (const bf16_t*)Wd, N, d, m, (bf16_t*)packed);
    return hipGetLastError();
}

}  // namespace elb
