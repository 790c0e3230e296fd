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

// silu(z) = z / (1 + e^-z), with a hardware reciprocal (the result is rounded to bf16 or
// compared at 1e-4 in fp32, far above its error)
// Block -> tile mapping.  Blocks are dispatched round-robin over the 8 XCDs (block b runs on
// XCD b % 8), and each XCD has its own L2.  Tiles are numbered expert-major, M-tile, then
// N-tile innermost, and XCD x takes the contiguous range [x * per, (x + 1) * per) of that
// order, so the blocks resident on one XCD at a time share their experts' weight tiles and
// gathered token rows through that XCD's L2.  The grid is an upper bound (a multiple of 8);
// surplus blocks exit.
__device__ __forceinline__ bool xcd_tile(int b, int total, int nt_count, int& mt, int& nt) {
    const int per = (total + 7) >> 3;
    const int s = b >> 3;
    const int L = (b & 7) * per + s;
    if (s >= per || L >= total) return false;
    mt = L / nt_count;
    nt = L - mt * nt_count;
    return true;
}

__device__ __forceinline__ float silu(float z) {
    return z * __builtin_amdgcn_rcpf(1.0f + __expf(-z));
}

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

    const int nt_count = (MODE == 0) ? m / 64 : (d + BN - 1) / BN;
    int tile, ntile;
    if (!xcd_tile(blockIdx.x, tile_off[N] * nt_count, nt_count, tile, ntile)) return;
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
            const int hc = ntile * 64;  // first H column of this tile
            const int brow = (r < 64) ? (hc + r) : (m + hc + (r - 64));
            b_src[i] = B + ((int64_t)e * 2 * m + brow) * d;
        } else {
            a_src[i] = A + (int64_t)(row0 + rr) * m;
            int brow = ntile * BN + r;
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
                    bf16_t* dst = C + (int64_t)(row0 + lr) * m + ntile * 64 + wn * 32 + l16;
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
                        const int col = ntile * BN + wn * 64 + ni * 16 + l16;
                        if (col < d) dst[col] = f32_to_bf16(acc[mi][ni][r]);
                    }
                }
            }
    }
}

// ------------------------------------------------------------------------------------------
// bf16 MFMA kernel with LDS DMA and a 4-stage pipeline: 256 x 256 block tile, k-tiles of 32,
// 4 waves (2 x 2) of 128 x 128, v_mfma_f32_32x32x16_bf16.  Tiles are copied global -> LDS by
// global_load_lds_dwordx4 (no staging registers, no ds_write), three k-tiles ahead of the one
// being multiplied, so the copy latency is covered by three k-tiles of MFMA work.  LDS rows
// are unpadded (64 B) with their four 16-byte chunks XOR-swizzled per row so that the 16 lanes
// of one ds_read_b128 pass (16 consecutive rows, same logical chunk) hit distinct banks.
// ------------------------------------------------------------------------------------------
constexpr int LBM = 256, LBN = 256;

typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef __attribute__((address_space(3))) void lds_void_t;
typedef __attribute__((address_space(1))) void glb_void_t;

// physical 16-byte chunk of logical chunk c (0..3) in LDS row r
__device__ __forceinline__ int swz(int r, int c) {
    return c ^ (((r >> 2) & 1) | ((((r >> 1) ^ (r >> 3)) & 1) << 1));
}

// s_waitcnt vmcnt(n) (expcnt and lgkmcnt not waited on)
#define ELB_WAIT_VMCNT(n) __builtin_amdgcn_s_waitcnt(((n) & 15) | (((n) >> 4) << 14) | 0x0F70)

template <int MODE>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(1, 1))) void gemm_bf16_dma(const bf16_t* __restrict__ A,
                                                     const int* __restrict__ row_token,
                                                     const bf16_t* __restrict__ B,
                                                     const int* __restrict__ offsets,
                                                     const int* __restrict__ tile_off, int N,
                                                     int d, int m, bf16_t* __restrict__ C) {
    constexpr int TM = 256, TN = 256, TK = 32;
    // one array per pipeline stage, so that the compiler sees which stage each LDS access
    // and each copy touches
    __shared__ __attribute__((aligned(1024))) bf16_t As0[TM * TK], As1[TM * TK], As2[TM * TK], As3[TM * TK];
    __shared__ __attribute__((aligned(1024))) bf16_t Bs0[TN * TK], Bs1[TN * TK], Bs2[TN * TK], Bs3[TN * TK];

    const int nt_count = (MODE == 0) ? m / 128 : (d + TN - 1) / TN;
    int tile, ntile;
    if (!xcd_tile(blockIdx.x, tile_off[N] * nt_count, nt_count, tile, ntile)) return;
    int e, row0, rows;
    find_tile(tile_off, offsets, N, tile, TM, e, row0, rows);

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wid = tid >> 6;
    const int wm = wid >> 1, wn = wid & 1;
    const int Kd = (MODE == 0) ? d : m;

    // DMA sources: wave w copies rows [64w, 64w + 64) of each tile, 16 rows (1 KB) per
    // instruction; lane l fills physical chunk l & 3 of row 64w + 16i + (l >> 2), so it
    // fetches that row's logical chunk swz(row, l & 3) (the XOR is its own inverse).
    uint32_t a_off[4], b_off[4];  // element offsets of each row's chunk (k = 0)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int r = 64 * wid + 16 * i + (lane >> 2);
        const int c = swz(r, lane & 3);
        const int rr = r < rows ? r : rows - 1;  // rows past the expert's end: clamp, unused
        if (MODE == 0) {
            a_off[i] = (uint32_t)row_token[row0 + rr] * (uint32_t)d + c * 8;
            const int hc = ntile * 128;
            const int brow = (r < 128) ? (hc + r) : (m + hc + (r - 128));
            b_off[i] = ((uint32_t)e * 2u * (uint32_t)m + brow) * (uint32_t)d + c * 8;
        } else {
            a_off[i] = (uint32_t)(row0 + rr) * (uint32_t)m + c * 8;
            int brow = ntile * TN + r;
            brow = brow < d ? brow : d - 1;
            b_off[i] = ((uint32_t)e * (uint32_t)d + brow) * (uint32_t)m + c * 8;
        }
    }
    // The copies are issued with inline assembly: the compiler cannot tell which LDS stage a
    // copy writes, and would otherwise wait for every copy in flight before each LDS read.
    // Waits are explicit below (ELB_WAIT_VMCNT); M0 carries the wave's LDS destination and is
    // set in the same statement.
    auto issue = [&](bf16_t* as, bf16_t* bs, int k0) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const uint32_t la = __builtin_amdgcn_readfirstlane(
                (uint32_t)(uintptr_t)(lds_void_t*)(as + (64 * wid + 16 * i) * TK));
            const uint32_t lb = __builtin_amdgcn_readfirstlane(
                (uint32_t)(uintptr_t)(lds_void_t*)(bs + (64 * wid + 16 * i) * TK));
            const uint32_t va = (a_off[i] + k0) * 2u;  // byte offsets
            const uint32_t vb = (b_off[i] + k0) * 2u;
            asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dwordx4 %1, %2"
                         :: "s"(la), "v"(va), "s"(A) : "memory", "m0");
            asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dwordx4 %1, %2"
                         :: "s"(lb), "v"(vb), "s"(B) : "memory", "m0");
        }
    };

    // fragment addresses (element offsets inside a stage); the swizzle of a fragment row
    // depends on its row mod 16, which is l32 mod 16
    const int l32 = lane & 31;
    const int hi = lane >> 5;
    int a_frag[4], b_frag[4];
#pragma unroll
    for (int mi = 0; mi < 4; ++mi) a_frag[mi] = (wm * 128 + mi * 32 + l32) * TK;
#pragma unroll
    for (int ni = 0; ni < 4; ++ni) {
        const int br = (MODE == 0) ? ((ni < 2) ? (wn * 64 + ni * 32) : (128 + wn * 64 + (ni - 2) * 32))
                                   : (wn * 128 + ni * 32);
        b_frag[ni] = (br + l32) * TK;
    }
    const int c0 = swz(l32, hi) * 8, c1 = swz(l32, 2 + hi) * 8;

    f32x16_t acc[4][4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j)
#pragma unroll
            for (int q = 0; q < 16; ++q) acc[i][j][q] = 0.f;

    auto consume = [&](const bf16_t* as, const bf16_t* bs) {
        bf16x8_t a0[4], b0[4], a1[4], b1[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            a0[i] = *reinterpret_cast<const bf16x8_t*>(as + a_frag[i] + c0);
            b0[i] = *reinterpret_cast<const bf16x8_t*>(bs + b_frag[i] + c0);
        }
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            a1[i] = *reinterpret_cast<const bf16x8_t*>(as + a_frag[i] + c1);
            b1[i] = *reinterpret_cast<const bf16x8_t*>(bs + b_frag[i] + c1);
        }
#pragma unroll
        for (int mi = 0; mi < 4; ++mi)
#pragma unroll
            for (int ni = 0; ni < 4; ++ni)
                acc[mi][ni] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a0[mi], b0[ni], acc[mi][ni], 0, 0, 0);
#pragma unroll
        for (int mi = 0; mi < 4; ++mi)
#pragma unroll
            for (int ni = 0; ni < 4; ++ni)
                acc[mi][ni] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a1[mi], b1[ni], acc[mi][ni], 0, 0, 0);
    };

    // Stage j of k-tile kt is consumed after waiting for its copy: each issue() is 8 copy
    // instructions per wave and copies complete in order, so with s later stages already
    // issued the wave waits for vmcnt <= 8 s; the barrier then makes every wave's part
    // visible and guarantees that the stage about to be refilled is no longer being read.
    const int nk = Kd / TK;  // a multiple of 4 (Kd % 128 == 0 for this kernel)
    issue(As0, Bs0, 0);
    issue(As1, Bs1, TK);
    issue(As2, Bs2, 2 * TK);
    // A bare s_barrier, not __syncthreads(): the latter's workgroup fence would make the
    // compiler drain every copy in flight (vmcnt(0)) and collapse the pipeline.  Visibility
    // is explicit instead: each wave waits for its own copies of stage J, and every LDS read
    // of the stage being refilled has completed (its MFMAs consumed it) before the barrier.
#define ELB_STEP(J, AJ, BJ, AP, BP)                                   \
    {                                                                 \
        const int kj = kt + (J);                                      \
        if (kj + 2 < nk) ELB_WAIT_VMCNT(16);                          \
        else if (kj + 1 < nk) ELB_WAIT_VMCNT(8);                      \
        else ELB_WAIT_VMCNT(0);                                       \
        __builtin_amdgcn_s_barrier();                                 \
        if (kj + 3 < nk) issue(AP, BP, (kj + 3) * TK);                \
        consume(AJ, BJ);                                              \
    }
    for (int kt = 0; kt < nk; kt += 4) {
        ELB_STEP(0, As0, Bs0, As3, Bs3)
        ELB_STEP(1, As1, Bs1, As0, Bs0)
        ELB_STEP(2, As2, Bs2, As1, Bs1)
        ELB_STEP(3, As3, Bs3, As2, Bs2)
    }
#undef ELB_STEP

    const int rq = hi * 4;
#pragma unroll
    for (int mi = 0; mi < 4; ++mi)
#pragma unroll
        for (int q = 0; q < 16; ++q) {
            const int lr = wm * 128 + mi * 32 + (q >> 2) * 8 + rq + (q & 3);
            if (lr >= rows) continue;
            if (MODE == 0) {
                bf16_t* dst = C + (int64_t)(row0 + lr) * m + ntile * 128 + wn * 64 + l32;
#pragma unroll
                for (int ni = 0; ni < 2; ++ni)
                    dst[ni * 32] = f32_to_bf16(silu(acc[mi][ni][q]) * acc[mi][ni + 2][q]);
            } else {
                bf16_t* dst = C + (int64_t)(row0 + lr) * d;
#pragma unroll
                for (int ni = 0; ni < 4; ++ni) {
                    const int col = ntile * TN + wn * 128 + ni * 32 + l32;
                    if (col < d) dst[col] = f32_to_bf16(acc[mi][ni][q]);
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

unsigned grid8(int64_t blocks) { return (unsigned)((blocks + 7) / 8 * 8); }

}  // namespace

int gemm_tile_rows(int dtype, int64_t T, int K, int N, int m) {
    if (dtype != ELB_BF16) return FBM;
    const int64_t avg_rows = T * K / (N > 0 ? N : 1);
    return (m % 128 == 0 && T > 0 && avg_rows >= 192) ? LBM : BM;
}

hipError_t launch_gemm_gate_up(const void* x, const void* Wgu, const int* row_token,
                               const int* offsets, const int* tile_off, int64_t max_tiles,
                               int tile_rows, int d, int N, int m, int dtype, void* H,
                               hipStream_t s) {
    if (max_tiles <= 0) return hipSuccess;
    if (dtype == ELB_BF16 && tile_rows == LBM) {
        ProfileScope prof("gemm_gate_up_bf16", s);
        hipLaunchKernelGGL(gemm_bf16_dma<0>, dim3(grid8(max_tiles * (m / 128))),
                           dim3(256), 0, s, (const bf16_t*)x, row_token, (const bf16_t*)Wgu,
                           offsets, tile_off, N, d, m, (bf16_t*)H);
    } else if (dtype == ELB_BF16) {
        ProfileScope prof("gemm_gate_up_bf16_s", s);
        hipLaunchKernelGGL(gemm_bf16<0>, dim3(grid8(max_tiles * (m / 64))), dim3(256),
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
                            const int* tile_off, int64_t max_tiles, int tile_rows, int d, int N,
                            int m, int dtype, void* Y, hipStream_t s) {
    if (max_tiles <= 0) return hipSuccess;
    if (dtype == ELB_BF16 && tile_rows == LBM) {
        ProfileScope prof("gemm_down_bf16", s);
        hipLaunchKernelGGL(gemm_bf16_dma<1>, dim3(grid8(max_tiles * ((d + LBN - 1) / LBN))),
                           dim3(256), 0, s, (const bf16_t*)H, (const int*)nullptr,
                           (const bf16_t*)Wd, offsets, tile_off, N, d, m, (bf16_t*)Y);
    } else if (dtype == ELB_BF16) {
        ProfileScope prof("gemm_down_bf16_s", s);
        hipLaunchKernelGGL(gemm_bf16<1>, dim3(grid8(max_tiles * ((d + BN - 1) / BN))),
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
