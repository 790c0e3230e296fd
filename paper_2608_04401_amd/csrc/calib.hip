// Calibration kernels for the roofline denominators (measurement aids, not part of the
// layer): back-to-back bf16 matrix-core instructions with no memory traffic, so that the MFMA
// rate the chip sustains (clock and power included) can be reported beside the 2.5 PFLOP/s
// specification value; and a read-only stream over a device buffer, the HBM read rate the
// read-dominated kernels (the decode weight streams, the combine) can be held against.
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

// Read-only stream: block b reads its own contiguous range of the buffer (per_block 16-byte
// chunks), 64 KB per step (sixteen coalesced 16-byte loads per lane, all in flight, with the
// non-temporal hint: a stream read once), and folds the words into one, which lane 0 of each
// wave writes out (one word per wave, so nothing can be removed).  n16: 16-byte chunks in the
// buffer.
constexpr int kReadUnroll = 16;

__global__ __launch_bounds__(256) void read_stream(const u32x4_t* __restrict__ buf,
                                                   int64_t n16, int64_t per_block,
                                                   uint32_t* __restrict__ out) {
    const int64_t lo = (int64_t)blockIdx.x * per_block;
    const int64_t hi = lo + per_block < n16 ? lo + per_block : n16;
    uint32_t acc = 0;
    int64_t i = lo + threadIdx.x;
    for (; i + 256 * (kReadUnroll - 1) < hi; i += 256 * kReadUnroll) {
        u32x4_t v[kReadUnroll];
#pragma unroll
        for (int u = 0; u < kReadUnroll; ++u) v[u] = __builtin_nontemporal_load(buf + i + 256 * u);
#pragma unroll
        for (int u = 0; u < kReadUnroll; ++u) acc ^= v[u][0] ^ v[u][1] ^ v[u][2] ^ v[u][3];
    }
    for (; i < hi; i += 256) {
        const u32x4_t a = __builtin_nontemporal_load(buf + i);
        acc ^= a[0] ^ a[1] ^ a[2] ^ a[3];
    }
    for (int m = 1; m < 64; m <<= 1) acc ^= __shfl_xor(acc, m);
    if ((threadIdx.x & 63) == 0) out[blockIdx.x * 4 + (threadIdx.x >> 6)] = acc;
}

}  // namespace

hipError_t launch_calibrate_read(const void* buf, int64_t bytes, int blocks, uint32_t* out,
                                 hipStream_t s) {
    ProfileScope prof("calibrate_read", s);
    const int64_t n16 = bytes / 16;
    ELB_LAUNCH(read_stream, dim3((unsigned)blocks), dim3(256), 0, s, (const u32x4_t*)buf, n16,
               (n16 + blocks - 1) / blocks, out);
    return hipGetLastError();
}

hipError_t launch_calibrate_mfma(int blocks, int iters, float* out, hipStream_t s) {
    ProfileScope prof("calibrate_mfma", s);
    ELB_LAUNCH(mfma_loop, dim3((unsigned)blocks), dim3(256), 0, s, iters, out);
    return hipGetLastError();
}

}  // namespace elb
