// Grouped expert GEMMs for decode-sized batches: weight streaming.
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
#include "common.h"

namespace elb {

namespace {

typedef uint32_t u32x2_t __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2_vt __attribute__((ext_vector_type(2)));
typedef float f32x2_vt __attribute__((ext_vector_type(2)));

__device__ __forceinline__ uint32_t pack2(float lo, float hi) {
    const f32x2_vt v = {lo, hi};
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2_vt));
}

__device__ __forceinline__ float silu_f(float z) {
    return z * __builtin_amdgcn_rcpf(1.0f + __expf(-z));
}

constexpr int SK_NF = 4;     // 16-row weight fragments per task (64 weight rows)
constexpr int SK_MAXMT = 2;  // token tiles of 16 rows per chunk (32 rows)

// One chunk of up to 16 * MT token rows of a task.
//   wp[f]: lane's address in weight fragment f (row l16 of the fragment, k offset kq)
//   xp[t]: lane's address in token tile t (row l16, clamped to a valid row, k offset kq)
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

    // a stage: 64 of the contraction, two 32-deep halves h.  A ring of R register slots
    // keeps R - 1 stages in flight: stage j lives in slot j % R, and while stage j is
    // multiplied, stage j + R - 1 is loaded into the slot stage j - 1 has just freed.
    // Unrolled by R, so every slot index is a constant.  Loads past the last stage re-read
    // it (clamped) and are never used.
    constexpr int R = 3;
    bf16x8_t w[R][SK_NF][2], x[R][MT][2];
    const int ns = kd / 64;
    auto load = [&](int j, bf16x8_t (&ws)[SK_NF][2], bf16x8_t (&xs)[MT][2]) {
        const int k0 = (j < ns ? j : ns - 1) * 64;
#pragma unroll
        for (int h = 0; h < 2; ++h) {
#pragma unroll
            for (int f = 0; f < SK_NF; ++f)
                ws[f][h] = *reinterpret_cast<const bf16x8_t*>(wp[f] + k0 + 32 * h);
#pragma unroll
            for (int t = 0; t < MT; ++t)
                xs[t][h] = *reinterpret_cast<const bf16x8_t*>(xp[t] + k0 + 32 * h);
        }
    };
    auto mma = [&](const bf16x8_t (&ws)[SK_NF][2], const bf16x8_t (&xs)[MT][2]) {
#pragma unroll
        for (int h = 0; h < 2; ++h)
#pragma unroll
            for (int t = 0; t < MT; ++t)
#pragma unroll
                for (int f = 0; f < SK_NF; ++f)
                    acc[t][f] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ws[f][h], xs[t][h],
                                                                        acc[t][f], 0, 0, 0);
    };
#pragma unroll
    for (int p = 0; p < R - 1; ++p) load(p, w[p], x[p]);
    int j = 0;
    for (; j + R <= ns; j += R) {
#pragma unroll
        for (int p = 0; p < R; ++p) {
            const int q = (p + R - 1) % R;
            load(j + p + R - 1, w[q], x[q]);
            // keep this stage's loads ahead of its multiplies, and the multiplies of one
            // stage together, so the waits before them leave R - 1 stages in flight
            __builtin_amdgcn_sched_barrier(0);
            mma(w[p], x[p]);
            __builtin_amdgcn_sched_barrier(0);
        }
    }
#pragma unroll
    for (int p = 0; p < R; ++p) {  // the last stages (fewer than R)
        if (j + p < ns) {
            const int q = (p + R - 1) % R;
            load(j + p + R - 1, w[q], x[q]);
            mma(w[p], x[p]);
        }
    }

    // epilogue: lane holds token row (lane & 15) of each tile and, per fragment f, the 4
    // consecutive output columns 16 f' + (lane >> 4) * 4 + i of the task
    const int l16 = lane & 15;
    const int cq = (lane >> 4) * 4;
#pragma unroll
    for (int t = 0; t < MT; ++t) {
        const int r = 16 * t + l16;
        if (r >= rows) continue;
        bf16_t* dst = C + (out_row0 + r) * (int64_t)out_ld + out_col + cq;
        if (MODE == 0) {
#pragma unroll
            for (int f = 0; f < 2; ++f) {  // fragments 0, 1: gate; 2, 3: the matching up
                const f32x4_t g = acc[t][f], u = acc[t][f + 2];
                const u32x2_t pk = {pack2(silu_f(g[0]) * u[0], silu_f(g[1]) * u[1]),
                                    pack2(silu_f(g[2]) * u[2], silu_f(g[3]) * u[3])};
                *reinterpret_cast<u32x2_t*>(dst + 16 * f) = pk;
            }
        } else {
#pragma unroll
            for (int f = 0; f < SK_NF; ++f) {
                const f32x4_t v = acc[t][f];
                const u32x2_t pk = {pack2(v[0], v[1]), pack2(v[2], v[3])};
                *reinterpret_cast<u32x2_t*>(dst + 16 * f) = pk;
            }
        }
    }
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
    const int l16 = lane & 15, kq = (lane >> 4) * 8;
    const bf16_t* wp[SK_NF];
#pragma unroll
    for (int f = 0; f < SK_NF; ++f) {
        const int wrow = (MODE == 0) ? ((f < 2) ? 32 * c + 16 * f : m + 32 * c + 16 * (f - 2))
                                     : 64 * c + 16 * f;
        wp[f] = W + ((int64_t)e * ((MODE == 0) ? 2 * m : d) + wrow + l16) * kd + kq;
    }
    const int out_ld = (MODE == 0) ? m : d;
    const int out_col = (MODE == 0) ? 32 * c : 64 * c;
    for (int cb = 0; cb < nrows; cb += 16 * SK_MAXMT) {
        const int rows = nrows - cb < 16 * SK_MAXMT ? nrows - cb : 16 * SK_MAXMT;
        const bf16_t* xp[SK_MAXMT];
#pragma unroll
        for (int t = 0; t < SK_MAXMT; ++t) {
            int r = 16 * t + l16;
            r = r < rows ? r : rows - 1;  // rows past the chunk: a valid row, never stored
            const int64_t src = (MODE == 0) ? (int64_t)row_token[row0 + cb + r] * d
                                            : (int64_t)(row0 + cb + r) * m;
            xp[t] = A + src + kq;
        }
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
