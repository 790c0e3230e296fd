// Weight-streaming pieces of the grouped expert GEMMs, for few token rows per expert: one
// wave owns a task (expert e and 64 of its weight rows) and walks a range of 64-deep stages
// of the contraction, loading each weight row as whole 128-byte lines straight into MFMA
// operand registers (no LDS), with the WEIGHTS as the first operand of
// v_mfma_f32_16x16x32_bf16, so that a lane ends with 4 consecutive output columns of one
// token row.  The token rows (up to 16 * MT) are the second operand, read from L2.
//   gate/up (MODE 0): a task is 32 H columns: its 32 gate rows and the 32 matching up rows
//                     (SwiGLU in registers);  down (MODE 1): a task is 64 Y columns.
// Used by the decode-sized kernels and by the remainder blocks of the large-tile kernel.
#pragma once

#include "common.h"

namespace elb {

namespace {

typedef uint32_t u32x2s_t __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2s_t __attribute__((ext_vector_type(2)));
typedef float f32x2s_t __attribute__((ext_vector_type(2)));

__device__ __forceinline__ uint32_t stream_pack2(float lo, float hi) {
    const f32x2s_t v = {lo, hi};
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2s_t));
}

__device__ __forceinline__ float stream_silu(float z) {
    return z * __builtin_amdgcn_rcpf(1.0f + __expf(-z));
}

constexpr int SK_NF = 4;  // 16-row weight fragments per task (64 weight rows)

// Lane addresses of a task: wp[f] in weight fragment f (row l16, k offset kq) and xp[t] in
// token tile t (row l16 of rows [row0, row0 + rows), clamped to a valid row, k offset kq).
// slots (optional): the rows are assignment slots t K + j listed at slots[row0 + r] (gate/up
// reads token t's x row, down reads row slot of H) instead of the dispatch's row order.
template <int MODE, int MAXMT>
__device__ __forceinline__ void stream_task(const bf16_t* __restrict__ A,
                                            const int* __restrict__ row_token,
                                            const bf16_t* __restrict__ W, int e, int c,
                                            int row0, int rows, int d, int m, int lane,
                                            const bf16_t* (&wp)[SK_NF],
                                            const bf16_t* (&xp)[MAXMT],
                                            const int* slots = nullptr, int K = 1) {
    const int kd = (MODE == 0) ? d : m;
    const int l16 = lane & 15, kq = (lane >> 4) * 8;
#pragma unroll
    for (int f = 0; f < SK_NF; ++f) {
        const int wrow = (MODE == 0) ? ((f < 2) ? 32 * c + 16 * f : m + 32 * c + 16 * (f - 2))
                                     : 64 * c + 16 * f;
        wp[f] = W + ((int64_t)e * ((MODE == 0) ? 2 * m : d) + wrow + l16) * kd + kq;
    }
#pragma unroll
    for (int t = 0; t < MAXMT; ++t) {
        int r = 16 * t + l16;
        r = r < rows ? r : rows - 1;  // rows past the chunk: a valid row, never stored
        int64_t src;
        if (slots) {
            const int slot = slots[row0 + r];
            src = (MODE == 0) ? (int64_t)(slot / K) * d : (int64_t)slot * m;
        } else {
            src = (MODE == 0) ? (int64_t)row_token[row0 + r] * d : (int64_t)(row0 + r) * m;
        }
        xp[t] = A + src + kq;
    }
}

// Packed weights (elb_pack_expert_weights): a task's 64 weight rows are stored in the order
// they are loaded -- per stage s, half h and fragment f, the 64 lanes' 16-byte operands
// (weight row 16 f + lane % 16 of the task, k = 64 s + 32 h + 8 (lane / 16) .. + 8) -- so every
// load instruction reads 1 KB contiguous and a task is one contiguous stream.
constexpr int kPackUnit = 512;  // bf16 elements of one (stage, half, fragment) operand block

// Lane addresses in a packed task (stage 0, half 0): wp[f] = task base + f units + lane's 16 B
template <int MODE>
__device__ __forceinline__ void stream_task_packed(const bf16_t* __restrict__ P, int e, int c,
                                                   int d, int m, int lane,
                                                   const bf16_t* (&wp)[SK_NF]) {
    const int per_e = (MODE == 0) ? m / 32 : d / 64;
    const int ns = ((MODE == 0) ? d : m) / 64;
    const bf16_t* base = P + ((int64_t)e * per_e + c) * ns * (8 * kPackUnit);
#pragma unroll
    for (int f = 0; f < SK_NF; ++f) wp[f] = base + f * kPackUnit + lane * 8;
}

// acc[t][f] += the task's stages [s0, s1) (a stage is 64 of the contraction, two 32-deep
// halves).  A ring of R register slots keeps R - 1 stages in flight: stage j lives in slot
// j % R, and while stage j is multiplied, stage j + R - 1 is loaded into the slot stage j - 1
// has just freed.  Unrolled by R, so every slot index is a constant.  Loads past the last
// stage re-read it (clamped) and are never used.  PACKED: weights in the packed order, read
// with the non-temporal hint (a contiguous stream read once).
template <int MT, int MAXMT, int R = 3, bool PACKED = false>
__device__ __forceinline__ void stream_mma(const bf16_t* const (&wp)[SK_NF],
                                           const bf16_t* const (&xp)[MAXMT], int s0, int s1,
                                           f32x4_t (&acc)[MT][SK_NF]) {
    bf16x8_t w[R][SK_NF][2], x[R][MT][2];
    auto load = [&](int j, bf16x8_t (&ws)[SK_NF][2], bf16x8_t (&xs)[MT][2]) {
        const int s = s0 + j < s1 ? s0 + j : s1 - 1;
        const int k0 = s * 64;
#pragma unroll
        for (int h = 0; h < 2; ++h) {
#pragma unroll
            for (int f = 0; f < SK_NF; ++f) {
                if (PACKED)
                    ws[f][h] = __builtin_bit_cast(
                        bf16x8_t, __builtin_nontemporal_load(reinterpret_cast<const u32x4_t*>(
                                      wp[f] + (s * 8 + h * 4) * kPackUnit)));
                else
                    ws[f][h] = *reinterpret_cast<const bf16x8_t*>(wp[f] + k0 + 32 * h);
            }
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
    const int ns = s1 - s0;
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
}

// Store a task's outputs for token rows [0, rows): the lane holds token row (lane & 15) of
// each tile and, per fragment f, the 4 consecutive output columns 16 f + (lane >> 4) * 4 + i
// of the task (gate/up: SwiGLU of fragment f and f + 2, f < 2).  bf16 out, 8-byte stores.
// slots (optional): output row of r is slots[out_row0 + r] instead of out_row0 + r.
template <int MODE, int MT>
__device__ __forceinline__ void stream_store(const f32x4_t (&acc)[MT][SK_NF], int rows,
                                             int64_t out_row0, int out_ld, int out_col,
                                             bf16_t* __restrict__ C, int lane,
                                             const int* slots = nullptr) {
    const int l16 = lane & 15;
    const int cq = (lane >> 4) * 4;
#pragma unroll
    for (int t = 0; t < MT; ++t) {
        const int r = 16 * t + l16;
        if (r >= rows) continue;
        const int64_t orow = slots ? (int64_t)slots[out_row0 + r] : out_row0 + r;
        bf16_t* dst = C + orow * (int64_t)out_ld + out_col + cq;
        if (MODE == 0) {
#pragma unroll
            for (int f = 0; f < 2; ++f) {  // fragments 0, 1: gate; 2, 3: the matching up
                const f32x4_t g = acc[t][f], u = acc[t][f + 2];
                const u32x2s_t pk = {
                    stream_pack2(stream_silu(g[0]) * u[0], stream_silu(g[1]) * u[1]),
                    stream_pack2(stream_silu(g[2]) * u[2], stream_silu(g[3]) * u[3])};
                *reinterpret_cast<u32x2s_t*>(dst + 16 * f) = pk;
            }
        } else {
#pragma unroll
            for (int f = 0; f < SK_NF; ++f) {
                const f32x4_t v = acc[t][f];
                const u32x2s_t pk = {stream_pack2(v[0], v[1]), stream_pack2(v[2], v[3])};
                *reinterpret_cast<u32x2s_t*>(dst + 16 * f) = pk;
            }
        }
    }
}

}  // namespace

}  // namespace elb
