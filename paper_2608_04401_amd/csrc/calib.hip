// Calibration kernel for the roofline denominators (a measurement aid, not part of the layer):
// back-to-back bf16 matrix-core instructions with no memory traffic, so that the MFMA rate
// the chip sustains (clock and power included) can be reported beside the 2.5 PFLOP/s
// specification value.
//
// Each wave runs `iters` rounds of 8 independent v_mfma_f32_32x32x16_bf16 chains (8 x 16
// accumulator registers; independent chains keep the matrix pipeline full), on operands held
// in registers, and finally writes one sum per wave so the work cannot be removed.
#include "common.h"

namespace elb {

namespace {

typedef float f32x16c_t __attribute__((ext_vector_type(16)));

__global__ __launch_bounds__(256) void mfma_loop(int iters, float* __restrict__ out) {
    const int lane = threadIdx.x & 63;
    bf16x8_t a, b;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        a[i] = (__bf16)(0.001f * (float)((lane + i) & 7));
        b[i] = (__bf16)(0.001f * (float)((lane * 3 + i) & 7));
    }
    f32x16c_t acc[8];
#pragma unroll
    for (int c = 0; c < 8; ++c)
#pragma unroll
        for (int q = 0; q < 16; ++q) acc[c][q] = 0.f;
    for (int it = 0; it < iters; ++it) {
#pragma unroll
        for (int c = 0; c < 8; ++c)
            acc[c] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, acc[c], 0, 0, 0);
    }
    float s = 0.f;
#pragma unroll
    for (int c = 0; c < 8; ++c)
#pragma unroll
        for (int q = 0; q < 16; ++q) s += acc[c][q];
    if (lane == 0) out[blockIdx.x * 4 + (threadIdx.x >> 6)] = s;
}

}  // namespace

hipError_t launch_calibrate_mfma(int blocks, int iters, float* out, hipStream_t s) {
    ProfileScope prof("calibrate_mfma", s);
    ELB_LAUNCH(mfma_loop, dim3((unsigned)blocks), dim3(256), 0, s, iters, out);
    return hipGetLastError();
}

}  // namespace elb
