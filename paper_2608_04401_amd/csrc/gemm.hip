// Grouped expert GEMMs (the SwiGLU expert MLPs of the MoE layer, one GEMM pair per expert).
//
//   gate_up: for each expert e, the rows of x routed to e (gathered through row_token, never
//            materialised) times W_gate_up[e]^T, with SwiGLU fused in the epilogue:
//            H[r, c] = silu(g) * u, g = x_r . W_gate[e][c], u = x_r . W_up[e][c].
//   down:    Y[r, :] = H[r, :] W_down[e]^T for the rows r of expert e.
//
// Work list: expert e owns rows [offsets[e], offsets[e+1]) of the expert-major order and
// M-tiles [tile_off[e], tile_off[e+1]); both come from the dispatch scan, on the device, so
// the grid is launched with an upper bound of M-tiles and surplus blocks exit at once.
//
// bf16 path: CDNA4 MFMA v_mfma_f32_16x16x32_bf16, fp32 accumulation, block tile 128 x 128 x 64,
// 4 waves (2 x 2), 64 x 64 per wave, LDS double buffered with register prefetch, rows padded
// by 8 bf16 so that 16 lanes reading 16-byte fragments of 16 consecutive rows hit distinct
// banks.  In gate_up the 128 B-tile columns are 64 gate and the matching 64 up columns, and
// each wave owns matching gate/up 16-column pairs, so SwiGLU is applied in registers.
// fp32 path: plain VALU FMA tiles (64 x 64 x 16), for the fp32 configuration.
#include "common.h"

namespace elb {

namespace {

__device__ __forceinline__ void find_tile(const int* __restrict__ tile_off,
                                          const int* __restrict__ offsets, int N, int tile,
                                          int tile_rows, int& e, int& row0, int& rows) {
    int lo = 0, hi = N - 1;  // largest e with tile_off[e] <= tile
    while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (tile_off[mid] <= tile) lo = mid;
        else hi = mid - 1;
    }
    e = lo;
    row0 = offsets[e] + (tile - tile_off[e]) * tile_rows;
    const int end = offsets[e + 1];
    rows = end - row0 < tile_rows ? end - row0 : tile_rows;
}

__device__ __forceinline__ float silu(float z) { return z / (1.0f + __expf(-z)); }

// ------------------------------------------------------------------------------------------
// bf16 MFMA kernel
// ------------------------------------------------------------------------------------------
constexpr int BM = 128, BN = 128, BK = 64, LDK = BK + 8;

template <int MODE>  // 0 = gate_up (+SwiGLU -> H), 1 = down (-> Y)
__global__ __launch_bounds__(256) void gemm_bf16(const bf16_t* __restrict__ A,
                                                 const int* __restrict__ row_token,
                                                 const bf16_t* __restrict__ B,
                                                 const int* __restrict__ offsets,
                                                 const int* __restrict__ tile_off, int N, int d,
                                                 int m, bf16_t* __restrict__ C) {
    __shared__ __attribute__((aligned(16))) bf16_t As[2][BM][LDK];
    __shared__ __attribute__((aligned(16))) bf16_t Bs[2][BN][LDK];

    const int tile = blockIdx.x;
    if (tile >= tile_off[N]) return;  // block-uniform, before any barrier
    int e, row0, rows;
    find_tile(tile_off, offsets, N, tile, BM, e, row0, rows);

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wid = tid >> 6;
    const int wm = wid >> 1, wn = wid & 1;

    // K dimension of this GEMM and the row stride of A / B
    const int Kd = (MODE == 0) ? d : m;
    // per-thread global source rows for the 4 A chunks and 4 B chunks it loads
    const bf16_t* a_src[4];
    const bf16_t* b_src[4];
    int kc8[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int c = tid + 256 * i;
        const int r = c >> 3;
        kc8[i] = (c & 7) * 8;
        const int rr = r < rows ? r : rows - 1;  // rows past the expert's end: clamp, unused
        if (MODE == 0) {
            const int tok = row_token[row0 + rr];
            a_src[i] = A + (int64_t)tok * d;
            const int hc = blockIdx.y * 64;  // first H column of this tile
            const int brow = (r < 64) ? (hc + r) : (m + hc + (r - 64));
            b_src[i] = B + ((int64_t)e * 2 * m + brow) * d;
        } else {
            a_src[i] = A + (int64_t)(row0 + rr) * m;
            int brow = blockIdx.y * BN + r;
            brow = brow < d ? brow : d - 1;
            b_src[i] = B + ((int64_t)e * d + brow) * m;
        }
    }

    f32x4_t acc[4][4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};

    // B-tile row read by fragment ni of this wave (lane row l16 added by the caller)
    int brow_base[4];
#pragma unroll
    for (int ni = 0; ni < 4; ++ni)
        brow_base[ni] = (MODE == 0) ? ((ni < 2) ? (wn * 32 + ni * 16) : (64 + wn * 32 + (ni - 2) * 16))
                                    : (wn * 64 + ni * 16);

    u32x4_t ra[4], rb[4];
    const int nk = Kd / BK;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        ra[i] = *reinterpret_cast<const u32x4_t*>(a_src[i] + kc8[i]);
        rb[i] = *reinterpret_cast<const u32x4_t*>(b_src[i] + kc8[i]);
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int r = (tid + 256 * i) >> 3;
        *reinterpret_cast<u32x4_t*>(&As[0][r][kc8[i]]) = ra[i];
        *reinterpret_cast<u32x4_t*>(&Bs[0][r][kc8[i]]) = rb[i];
    }
    __syncthreads();
    const int l16 = lane & 15;
    const int kq = (lane >> 4) * 8;
    for (int kt = 0; kt < nk; ++kt) {
        const int buf = kt & 1;
        const bool more = kt + 1 < nk;
        if (more) {
            const int k0 = (kt + 1) * BK;
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                ra[i] = *reinterpret_cast<const u32x4_t*>(a_src[i] + k0 + kc8[i]);
                rb[i] = *reinterpret_cast<const u32x4_t*>(b_src[i] + k0 + kc8[i]);
            }
        }
#pragma unroll
        for (int ks = 0; ks < BK / 32; ++ks) {
            bf16x8_t af[4], bfr[4];
#pragma unroll
            for (int mi = 0; mi < 4; ++mi)
                af[mi] = *reinterpret_cast<const bf16x8_t*>(&As[buf][wm * 64 + mi * 16 + l16][ks * 32 + kq]);
#pragma unroll
            for (int ni = 0; ni < 4; ++ni)
                bfr[ni] = *reinterpret_cast<const bf16x8_t*>(&Bs[buf][brow_base[ni] + l16][ks * 32 + kq]);
#pragma unroll
            for (int mi = 0; mi < 4; ++mi)
#pragma unroll
                for (int ni = 0; ni < 4; ++ni)
                    acc[mi][ni] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[mi], bfr[ni], acc[mi][ni], 0, 0, 0);
        }
        if (more) {
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int r = (tid + 256 * i) >> 3;
                *reinterpret_cast<u32x4_t*>(&As[buf ^ 1][r][kc8[i]]) = ra[i];
                *reinterpret_cast<u32x4_t*>(&Bs[buf ^ 1][r][kc8[i]]) = rb[i];
            }
        }
        __syncthreads();
    }

    // epilogue: lane holds rows (lane>>4)*4 + r, column lane&15 of each 16x16 fragment
    const int rq = (lane >> 4) * 4;
    if (MODE == 0) {
#pragma unroll
        for (int mi = 0; mi < 4; ++mi)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int lr = wm * 64 + mi * 16 + rq + r;
                if (lr < rows) {
                    bf16_t* dst = C + (int64_t)(row0 + lr) * m + blockIdx.y * 64 + wn * 32 + l16;
#pragma unroll
                    for (int ni = 0; ni < 2; ++ni) {
                        const float g = acc[mi][ni][r];
                        const float u = acc[mi][ni + 2][r];
                        dst[ni * 16] = f32_to_bf16(silu(g) * u);
                    }
                }
            }
    } else {
#pragma unroll
        for (int mi = 0; mi < 4; ++mi)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int lr = wm * 64 + mi * 16 + rq + r;
                if (lr < rows) {
                    bf16_t* dst = C + (int64_t)(row0 + lr) * d;
#pragma unroll
                    for (int ni = 0; ni < 4; ++ni) {
                        const int col = blockIdx.y * BN + wn * 64 + ni * 16 + l16;
                        if (col < d) dst[col] = f32_to_bf16(acc[mi][ni][r]);
                    }
                }
            }
    }
}

// ------------------------------------------------------------------------------------------
// fp32 VALU kernel: tile 64 x 64, k-step 16, 256 threads each computing 4 x 4 outputs
// ------------------------------------------------------------------------------------------
constexpr int FBM = 64, FBN = 64, FBK = 16;

template <int MODE>
__global__ __launch_bounds__(256) void gemm_f32(const float* __restrict__ A,
                                                const int* __restrict__ row_token,
                                                const float* __restrict__ B,
                                                const int* __restrict__ offsets,
                                                const int* __restrict__ tile_off, int N, int d,
                                                int m, float* __restrict__ C) {
    __shared__ float As[FBK][FBM + 4];
    __shared__ float Bs[FBK][FBN + 4];
    const int tile = blockIdx.x;
    if (tile >= tile_off[N]) return;
    int e, row0, rows;
    find_tile(tile_off, offsets, N, tile, FBM, e, row0, rows);
    const int tid = threadIdx.x;
    const int tx = tid & 15, ty = tid >> 4;
    const int Kd = (MODE == 0) ? d : m;
    const int nout = (MODE == 0) ? m : d;  // output columns of this GEMM

    // loader: each thread loads one A element-quad and one B element-quad per k-step
    const int lr = tid >> 2;        // 0..63: tile row (A) / tile column (B)
    const int lk = (tid & 3) * 4;   // 0,4,8,12
    const int rr = lr < rows ? lr : rows - 1;
    const float* a_src;
    if (MODE == 0) a_src = A + (int64_t)row_token[row0 + rr] * d;
    else a_src = A + (int64_t)(row0 + rr) * m;
    const float* b_src;
    bool bvalid = true;
    if (MODE == 0) {
        const int hc = blockIdx.y * 32;
        const int col = (lr < 32) ? hc + lr : hc + (lr - 32);
        bvalid = col < m;
        const int brow = (lr < 32) ? (bvalid ? col : 0) : m + (bvalid ? col : 0);
        b_src = B + ((int64_t)e * 2 * m + brow) * d;
    } else {
        int brow = blockIdx.y * FBN + lr;
        bvalid = brow < d;
        b_src = B + ((int64_t)e * d + (bvalid ? brow : 0)) * m;
    }

    float acc[4][4] = {};
    for (int k0 = 0; k0 < Kd; k0 += FBK) {
        const float4 av = *reinterpret_cast<const float4*>(a_src + k0 + lk);
        const float4 bv = *reinterpret_cast<const float4*>(b_src + k0 + lk);
        As[lk + 0][lr] = av.x; As[lk + 1][lr] = av.y; As[lk + 2][lr] = av.z; As[lk + 3][lr] = av.w;
        Bs[lk + 0][lr] = bv.x; Bs[lk + 1][lr] = bv.y; Bs[lk + 2][lr] = bv.z; Bs[lk + 3][lr] = bv.w;
        __syncthreads();
#pragma unroll
        for (int kk = 0; kk < FBK; ++kk) {
            float a[4], b[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) a[i] = As[kk][ty * 4 + i];
            if (MODE == 0) {
                b[0] = Bs[kk][tx * 2];
                b[1] = Bs[kk][tx * 2 + 1];
                b[2] = Bs[kk][32 + tx * 2];
                b[3] = Bs[kk][32 + tx * 2 + 1];
            } else {
#pragma unroll
                for (int j = 0; j < 4; ++j) b[j] = Bs[kk][tx * 4 + j];
            }
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int j = 0; j < 4; ++j) acc[i][j] = fmaf(a[i], b[j], acc[i][j]);
        }
        __syncthreads();
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int r = ty * 4 + i;
        if (r >= rows) continue;
        float* dst = C + (int64_t)(row0 + r) * nout;
        if (MODE == 0) {
#pragma unroll
            for (int j = 0; j < 2; ++j) {
                const int col = blockIdx.y * 32 + tx * 2 + j;
                if (col < m) dst[col] = silu(acc[i][j]) * acc[i][j + 2];
            }
        } else {
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int col = blockIdx.y * FBN + tx * 4 + j;
                if (col < d) dst[col] = acc[i][j];
            }
        }
    }
}

}  // namespace

int gemm_tile_rows(int dtype) { return dtype == ELB_BF16 ? BM : FBM; }

hipError_t launch_gemm_gate_up(const void* x, const void* Wgu, const int* row_token,
                               const int* offsets, const int* tile_off, int64_t max_tiles,
                               int d, int N, int m, int dtype, void* H, hipStream_t s) {
    if (max_tiles <= 0) return hipSuccess;
    if (dtype == ELB_BF16) {
        ProfileScope prof("gemm_gate_up_bf16", s);
        hipLaunchKernelGGL(gemm_bf16<0>, dim3((unsigned)max_tiles, (unsigned)(m / 64)), dim3(256),
                           0, s, (const bf16_t*)x, row_token, (const bf16_t*)Wgu, offsets,
                           tile_off, N, d, m, (bf16_t*)H);
    } else {
        ProfileScope prof("gemm_gate_up_f32", s);
        hipLaunchKernelGGL(gemm_f32<0>, dim3((unsigned)max_tiles, (unsigned)((m + 31) / 32)),
                           dim3(256), 0, s, (const float*)x, row_token, (const float*)Wgu,
                           offsets, tile_off, N, d, m, (float*)H);
    }
    return hipGetLastError();
}

hipError_t launch_gemm_down(const void* H, const void* Wd, const int* offsets,
                            const int* tile_off, int64_t max_tiles, int d, int N, int m,
                            int dtype, void* Y, hipStream_t s) {
    if (max_tiles <= 0) return hipSuccess;
    if (dtype == ELB_BF16) {
        ProfileScope prof("gemm_down_bf16", s);
        hipLaunchKernelGGL(gemm_bf16<1>, dim3((unsigned)max_tiles, (unsigned)((d + BN - 1) / BN)),
                           dim3(256), 0, s, (const bf16_t*)H, (const int*)nullptr,
                           (const bf16_t*)Wd, offsets, tile_off, N, d, m, (bf16_t*)Y);
    } else {
        ProfileScope prof("gemm_down_f32", s);
        hipLaunchKernelGGL(gemm_f32<1>, dim3((unsigned)max_tiles, (unsigned)((d + FBN - 1) / FBN)),
                           dim3(256), 0, s, (const float*)H, (const int*)nullptr,
                           (const float*)Wd, offsets, tile_off, N, d, m, (float*)Y);
    }
    return hipGetLastError();
}

}  // namespace elb
