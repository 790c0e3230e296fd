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
template <int MODE, int MT>
__device__ __forceinline__ void skinny_chunk(const bf16_t* const (&wp)[SK_NF],
                                             const bf16_t* const (&xp)[SK_MAXMT], int kd,
                                             int rows, int64_t out_row0, int out_ld,
                                             int out_col, bf16_t* __restrict__ C, int lane) {
    f32x4_t acc[MT][SK_NF];
#pragma unroll
    for (int t = 0; t < MT; ++t)
#pragma unroll
        for (int f = 0; f < SK_NF; ++f) acc[t][f] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    stream_mma<MT, SK_MAXMT>(wp, xp, 0, kd / 64, acc);
    stream_store<MODE, MT>(acc, rows, out_row0, out_ld, out_col, C, lane);
}

// MODE 0: A = x [T, d] gathered through row_token, W = W_gate_up [N, 2m, d], C = H [rows, m]
// MODE 1: A = H [rows, m], W = W_down [N, d, m], C = Y [rows, d]
template <int MODE>
// (2 waves per SIMD: the register ring of three stages fits in 256 registers)
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(2, 2))) void gemm_skinny(
    const bf16_t* __restrict__ A, const int* __restrict__ row_token,
    const bf16_t* __restrict__ W, const int* __restrict__ offsets, int N, int d, int m,
    bf16_t* __restrict__ C) {
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
    const int row0 = offsets[e];
    const int nrows = offsets[e + 1] - row0;
    if (nrows <= 0) return;

    const int kd = (MODE == 0) ? d : m;
    const int out_ld = (MODE == 0) ? m : d;
    const int out_col = (MODE == 0) ? 32 * c : 64 * c;
    for (int cb = 0; cb < nrows; cb += 16 * SK_MAXMT) {
        const int rows = nrows - cb < 16 * SK_MAXMT ? nrows - cb : 16 * SK_MAXMT;
        const bf16_t* wp[SK_NF];
        const bf16_t* xp[SK_MAXMT];
        stream_task<MODE, SK_MAXMT>(A, row_token, W, e, c, row0 + cb, rows, d, m, lane, wp, xp);
        const int64_t orow = row0 + cb;
        if (rows <= 16) skinny_chunk<MODE, 1>(wp, xp, kd, rows, orow, out_ld, out_col, C, lane);
        else skinny_chunk<MODE, 2>(wp, xp, kd, rows, orow, out_ld, out_col, C, lane);
    }
}

unsigned blocks_for(int tasks) { return (unsigned)(((tasks + 3) / 4 + 7) / 8 * 8); }

}  // namespace

bool gemm_use_skinny(int dtype, int64_t T, int K, int N, int d, int m) {
    // at most 16 rows per expert on average: far below the bf16 ridge point (~300 rows), so
    // the weight stream bounds the GEMMs
    return dtype == ELB_BF16 && T > 0 && T * K <= (int64_t)16 * N && m % 32 == 0 &&
           d % 64 == 0 && m % 64 == 0;
}

hipError_t launch_gemm_skinny(const void* x, const void* Wgu, const void* Wd,
                              const int* row_token, const int* offsets, int d, int N, int m,
                              void* H, void* Y, hipStream_t s) {
    {
        ProfileScope prof("gemm_gate_up_skinny", s);
        hipLaunchKernelGGL(gemm_skinny<0>, dim3(blocks_for(N * (m / 32))), dim3(256), 0, s,
                           (const bf16_t*)x, row_token, (const bf16_t*)Wgu, offsets, N, d, m,
                           (bf16_t*)H);
    }
    if (hipError_t e = hipGetLastError(); e != hipSuccess) return e;
    {
        ProfileScope prof("gemm_down_skinny", s);
        hipLaunchKernelGGL(gemm_skinny<1>, dim3(blocks_for(N * (d / 64))), dim3(256), 0, s,
                           (const bf16_t*)H, (const int*)nullptr, (const bf16_t*)Wd, offsets,
                           N, d, m, (bf16_t*)Y);
    }
    return hipGetLastError();
}

}  // namespace elb
