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
// Kernels (all fp32 accumulation; the launchers at the end pick one per problem):
//  - gemm_bf16_dma: the prefill kernel (on average at least 96 rows per expert).  Block tile
//    256 x 256 x 64, 4 waves of 128 x 128 on v_mfma_f32_32x32x16_bf16, operands copied
//    global -> LDS by global_load_lds_dwordx4 into a 5-unit ring; remainder rows of a few
//    experts (TilePlan) go to extra blocks of the same launch (weight-streaming tasks of
//    gemm_stream.h).  Described in detail above the kernel.
//  - gemm_bf16: smaller problems.  v_mfma_f32_16x16x32_bf16, block tile 128 x 128 x 64,
//    4 waves (2 x 2) of 64 x 64, LDS double buffered with register prefetch, rows padded by
//    8 bf16 so that 16 lanes reading 16-byte fragments of 16 consecutive rows hit distinct
//    banks.  In gate_up the 128 B-tile columns are 64 gate and the matching 64 up columns,
//    and each wave owns matching gate/up 16-column pairs, so SwiGLU is applied in registers.
//  - decode-sized batches use gemm_skinny.hip instead (weight streaming).
// fp32 path: plain VALU FMA tiles (64 x 64 x 16), for the fp32 configuration.
#include "gemm_stream.h"

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
// bf16 MFMA kernel with LDS DMA: 256 x 256 block tile, k-tiles of 64, 4 waves (2 x 2) of
// 128 x 128, v_mfma_f32_32x32x16_bf16, one block per CU (the copy ring takes all 160 KB of LDS).
//
// Copies: global_load_lds_dwordx4 (no staging registers, no ds_write).  Each copy
// instruction moves 8 rows x 128 bytes, one whole cache line per row (full lines move more
// bytes per request than half lines).  With up to three M-tiles per expert the weight copies
// carry the non-temporal hint: each weight tile is read by the few M-tiles of its expert,
// close together in time, and streaming it keeps the caches for the token rows and for the
// other GEMM's operands (measured: down GEMM -8 %, gate/up unchanged); with more M-tiles the
// tiles are reused enough that the hint costs more than it saves, so the kernel takes it as an
// argument.  The A half (token rows) and the B half (weight rows) of a k-tile
// are separate 32 KB units of a 5-unit ring; the B half, which usually misses to HBM, is
// issued two k-tiles ahead of its use and the A half one k-tile ahead.  LDS rows are
// unpadded (128 B) with their eight 16-byte chunks XOR-swizzled per row so that the 16
// lanes of one ds_read_b128 pass (16 consecutive rows, same logical chunk) hit distinct banks.
//
// MFMA operands are swapped (weights as the first operand): each accumulator tile is then the
// transpose of the output tile, so a lane holds 4 consecutive output columns of one token row
// per group of 4 registers.  The epilogue writes them (bf16, 8 bytes per lane) into a padded
// row-major tile in LDS and the block then stores whole rows with 16-byte coalesced stores.
// ------------------------------------------------------------------------------------------
constexpr int LBM = 256, LBN = 256;

typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef uint32_t u32x2_t __attribute__((ext_vector_type(2)));

// physical 16-byte chunk of logical chunk c (0..7) in a 128-byte LDS row r
__device__ __forceinline__ int swz8(int r, int c) {
    return c ^ (((r >> 1) ^ ((r & 1) << 2)) & 7);
}


// two floats -> two bf16 (round to nearest even) in one v_cvt_pk_bf16_f32
typedef __bf16 bf16x2_vt __attribute__((ext_vector_type(2)));
typedef float f32x2_vt __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
    const f32x2_vt v = {lo, hi};
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2_vt));
}

// Remainder rows of the large-tile GEMM (TilePlan): for each expert e in tail_list, the
// 1..kTailRows rows past its last full M-tile, by extra blocks at the end of the grid, one per
// (listed expert, task) of gemm_stream.h.  The 4 waves split the contraction's 64-deep stages
// four ways; the partial tiles are summed in LDS in a fixed order and wave 0 stores them.
template <int MODE, int MT>
__device__ __forceinline__ void tail_task(const bf16_t* const (&wp)[SK_NF],
                                          const bf16_t* const (&xp)[2], int s0, int s1,
                                          int rows, int64_t out_row0, int out_ld, int out_col,
                                          bf16_t* __restrict__ C, char* lds) {
    const int lane = threadIdx.x & 63;
    const int w = threadIdx.x >> 6;
    f32x4_t acc[MT][SK_NF];
#pragma unroll
    for (int t = 0; t < MT; ++t)
#pragma unroll
        for (int f = 0; f < SK_NF; ++f) acc[t][f] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    if (s1 > s0) stream_mma<MT, 2>(wp, xp, s0, s1, acc);
    f32x4_t* r4 = reinterpret_cast<f32x4_t*>(lds);  // [wave][t][f][lane]
#pragma unroll
    for (int t = 0; t < MT; ++t)
#pragma unroll
        for (int f = 0; f < SK_NF; ++f) r4[((w * MT + t) * SK_NF + f) * 64 + lane] = acc[t][f];
    __syncthreads();
    if (w != 0) return;  // no barrier follows
#pragma unroll
    for (int t = 0; t < MT; ++t)
#pragma unroll
        for (int f = 0; f < SK_NF; ++f) {
            f32x4_t v = r4[(t * SK_NF + f) * 64 + lane];
#pragma unroll
            for (int ww = 1; ww < 4; ++ww) v += r4[((ww * MT + t) * SK_NF + f) * 64 + lane];
            acc[t][f] = v;
        }
    stream_store<MODE, MT>(acc, rows, out_row0, out_ld, out_col, C, lane);
}

template <int MODE>
__device__ __forceinline__ void tail_block(const bf16_t* __restrict__ A,
                                           const int* __restrict__ row_token,
                                           const bf16_t* __restrict__ B,
                                           const int* __restrict__ offsets,
                                           const int* __restrict__ tail_list, int task, int d,
                                           int m, int tile_rows, bf16_t* __restrict__ C,
                                           char* lds) {
    const int per_e = (MODE == 0) ? m / 32 : d / 64;
    const int i = task / per_e, c = task - i * per_e;
    if (i >= tail_list[0]) return;  // block-uniform, before any barrier
    const int e = tail_list[1 + i];
    const int ce = offsets[e + 1] - offsets[e];
    const int full = ce / tile_rows * tile_rows;
    const int rows = ce - full;  // 1..kTailRows (32) by the plan
    const int row0 = offsets[e] + full;
    const int lane = threadIdx.x & 63;
    const int w = threadIdx.x >> 6;
    const int ns = ((MODE == 0) ? d : m) / 64;
    const int s0 = ns * w / 4, s1 = ns * (w + 1) / 4;
    const bf16_t* wp[SK_NF];
    const bf16_t* xp[2];
    stream_task<MODE, 2>(A, row_token, B, e, c, row0, rows, d, m, lane, wp, xp);
    const int out_ld = (MODE == 0) ? m : d;
    const int out_col = (MODE == 0) ? 32 * c : 64 * c;
    if (rows <= 16) tail_task<MODE, 1>(wp, xp, s0, s1, rows, row0, out_ld, out_col, C, lds);
    else tail_task<MODE, 2>(wp, xp, s0, s1, rows, row0, out_ld, out_col, C, lds);
}

// NTW: the weight copies carry the non-temporal hint (the kernel below picks it by size)
template <int MODE, bool NTW>
__device__ __forceinline__ void gemm_dma_body(
    const bf16_t* __restrict__ A, const int* __restrict__ row_token,
    const bf16_t* __restrict__ B, const int* __restrict__ offsets,
    const int* __restrict__ tile_off, const int* __restrict__ tail_list, int big_blocks,
    int N, int d, int m, bf16_t* __restrict__ C, char* sm_bytes) {
    constexpr int TM = 256, TN = 256, TK = 64;
    constexpr int UNIT = TM * TK;  // elements of one ring unit: the A or the B half of a k-tile
    constexpr int NU = 5;          // units in the ring
    constexpr int OUTC = (MODE == 0) ? 128 : TN;  // output columns of the block
    constexpr int PITCH = OUTC * 2 + 16;          // bytes per row of the staged output tile
    static_assert(TM == TN && TM * PITCH <= NU * UNIT * 2, "staging tile exceeds LDS");
    bf16_t* const sm = reinterpret_cast<bf16_t*>(sm_bytes);
    if ((int)blockIdx.x >= big_blocks) {  // the remainder blocks after the tiles
        tail_block<MODE>(A, row_token, B, offsets, tail_list, (int)blockIdx.x - big_blocks, d,
                         m, TM, C, sm_bytes);
        return;
    }

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

    // Copy sources: wave w copies rows [64w, 64w + 64) of each tile, 8 rows (1 KB) per
    // instruction; lane l fills physical chunk l & 7 of row 64w + 8i + (l >> 3), so it
    // fetches that row's logical chunk swz8(row, l & 7) (the XOR is its own inverse).
    // The copy instruction adds a 32-bit per-lane byte offset to a 64-bit scalar base, so the
    // bases are per block: the expert's weight matrix, and in the down GEMM the tile's first
    // H row.  The offsets then stay below one expert's weights (2 m d or d m elements) or 256
    // H rows; only the gathered x rows of the gate/up GEMM are addressed from x itself, and
    // gemm_tile_rows sends a problem to this kernel only when T d elements take less than
    // 2^32 bytes.
    const bf16_t* const Ablk = (MODE == 0) ? A : A + (int64_t)row0 * m;
    const bf16_t* const Bblk = B + (int64_t)e * ((MODE == 0) ? 2 * m : d) * Kd;
    uint32_t a_off[8], b_off[8];  // element offsets of each row's chunk (k = 0)
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        const int r = 64 * wid + 8 * i + (lane >> 3);
        const int c = swz8(r, lane & 7);
        const int rr = r < rows ? r : rows - 1;  // rows past the expert's end: clamp, unused
        if (MODE == 0) {
            a_off[i] = (uint32_t)row_token[row0 + rr] * (uint32_t)d + c * 8;
            const int hc = ntile * 128;
            const int brow = (r < 128) ? (hc + r) : (m + hc + (r - 128));
            b_off[i] = (uint32_t)brow * (uint32_t)d + c * 8;
        } else {
            a_off[i] = (uint32_t)rr * (uint32_t)m + c * 8;
            int brow = ntile * TN + r;
            brow = brow < d ? brow : d - 1;
            b_off[i] = (uint32_t)brow * (uint32_t)m + c * 8;
        }
    }
    // LDS byte address of this wave's first 8-row group in unit 0
    const uint32_t lds0 = (uint32_t)(uintptr_t)(lds_void_t*)sm_bytes +
                          (uint32_t)__builtin_amdgcn_readfirstlane(wid * 64 * TK * 2);
    // The copies are inline assembly: the compiler cannot tell which unit a copy writes, and
    // would otherwise wait for every copy in flight before each LDS read.  Waits are explicit
    // (ELB_WAIT_VMCNT); M0 carries the LDS destination and is set in the same statement.
    // Each call is 8 copy instructions per wave.
    // copy instruction i (of 8) of a unit; nt: the non-temporal hint (the weight copies when
    // NTW)
    auto issue_one = [&](const bf16_t* src, const uint32_t (&off)[8], int unit, int k0, bool nt,
                         int i) {
        const uint32_t la = lds0 + (uint32_t)unit * (UNIT * 2) + i * 1024;
        const uint32_t va = (off[i] + k0) * 2u;
        if (nt)
            asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dwordx4 %1, %2 nt"
                         :: "s"(la), "v"(va), "s"(src) : "memory", "m0");
        else
            asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dwordx4 %1, %2"
                         :: "s"(la), "v"(va), "s"(src) : "memory", "m0");
    };
    auto issue = [&](const bf16_t* src, const uint32_t (&off)[8], int unit, int k0, bool nt) {
#pragma unroll
        for (int i = 0; i < 8; ++i) issue_one(src, off, unit, k0, nt, i);
    };

    // fragment rows (element offsets inside a stage)
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
    // element offset of the chunk this lane reads for k16-step kk (k = 16 kk .. 16 kk + 15);
    // fragment rows are l32 mod 16 modulo 16, so the swizzle depends on l32 only
    int cofs[4];
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) cofs[kk] = swz8(l32, 2 * kk + hi) * 8;

    f32x16_t acc[4][4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j)
#pragma unroll
            for (int q = 0; q < 16; ++q) acc[i][j][q] = 0.f;

    // Two fragment register sets: the 8 LDS reads of the next k16-step are issued between
    // the first 8 of the 16 MFMAs of the current one, which run on the other set.
    bf16x8_t fa0[4], fb0[4], fa1[4], fb1[4];
    auto load = [&](bf16x8_t (&fa)[4], bf16x8_t (&fb)[4], int ua, int ub, int kk) {
        const bf16_t* sa = sm + ua * UNIT + cofs[kk];
        const bf16_t* sb = sm + ub * UNIT + cofs[kk];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            fa[i] = *reinterpret_cast<const bf16x8_t*>(sa + a_frag[i]);
            fb[i] = *reinterpret_cast<const bf16x8_t*>(sb + b_frag[i]);
        }
    };
    auto mma = [&](const bf16x8_t (&fa)[4], const bf16x8_t (&fb)[4], bool reads) {
#pragma unroll
        for (int mi = 0; mi < 4; ++mi)
#pragma unroll
            for (int ni = 0; ni < 4; ++ni)
                acc[mi][ni] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fb[ni], fa[mi], acc[mi][ni], 0, 0, 0);
        if (reads) {
#pragma unroll
            for (int i = 0; i < 8; ++i) {
                __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);  // one LDS read
                __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // one MFMA
            }
            __builtin_amdgcn_sched_group_barrier(0x008, 8, 0);
        }
    };

    // Pipeline: the B half of k-tile t lives in unit 2t mod 5, its A half in unit 2t + 1
    // mod 5.  Once the fourth k16-step's fragments of tile t are read (after the second
    // step's MFMAs) each wave waits for its own copies of tile t + 1 and for its own LDS
    // reads; the barrier then makes tile t + 1 visible to every wave and frees tile t's two
    // units (every read of them has completed), which receive the A half of tile t + 2 and the
    // B half of tile t + 3 while the third and fourth steps' MFMAs run.  Copies complete in
    // order and each half is 8 instructions per wave; the only copies issued after tile
    // t + 1's are those of B(t + 2), so the wait is vmcnt <= 8 (0 near the end).
    // A bare s_barrier, not __syncthreads(): the latter's fence would make the compiler drain
    // every copy in flight.
    const int nk = Kd / TK;  // >= 1
    // as if barriers at t = -3, -2, -1 had issued B(0); A(0), B(1); A(1), B(2)
    issue(Bblk, b_off, 0, 0, NTW);
    issue(Ablk, a_off, 1, 0, false);
    if (nk > 1) {
        issue(Bblk, b_off, 2, TK, NTW);
        issue(Ablk, a_off, 3, TK, false);
        if (nk > 2) {
            issue(Bblk, b_off, 4, 2 * TK, NTW);
            ELB_WAIT_VMCNT(24);
        } else {
            ELB_WAIT_VMCNT(16);
        }
    } else {
        ELB_WAIT_VMCNT(0);
    }
    __builtin_amdgcn_s_barrier();
    int ub = 0, ua = 1;  // units of tile t
    load(fa0, fb0, ua, ub, 0);
    int t = 0;
    for (; t < nk - 1; ++t) {
        const int ub1 = ub + 2 >= NU ? ub + 2 - NU : ub + 2;  // units of tile t + 1
        const int ua1 = ua + 2 >= NU ? ua + 2 - NU : ua + 2;
        load(fa1, fb1, ua, ub, 1);
        mma(fa0, fb0, true);
        load(fa0, fb0, ua, ub, 2);
        mma(fa1, fb1, true);
        load(fa1, fb1, ua, ub, 3);
        __builtin_amdgcn_sched_barrier(0);
        if (t + 2 < nk) ELB_WAIT_VMCNT(8);
        else ELB_WAIT_VMCNT(0);
        asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
        // k16-steps 2 and 3 (32 MFMAs), with one of the 16 copy instructions of A(t + 2) and
        // B(t + 3) after every other MFMA: a copy that cannot issue at once then holds up one
        // MFMA slot, not a burst of them.  The next tile's step-0 reads go between the steps.
#pragma unroll
        for (int q = 0; q < 32; ++q) {
            const int mi = (q & 15) >> 2, ni = q & 3;
            if (q < 16)
                acc[mi][ni] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fb0[ni], fa0[mi],
                                                                      acc[mi][ni], 0, 0, 0);
            else
                acc[mi][ni] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fb1[ni], fa1[mi],
                                                                      acc[mi][ni], 0, 0, 0);
            __builtin_amdgcn_sched_barrier(0);
            if (q == 15) {
                load(fa0, fb0, ua1, ub1, 0);
                __builtin_amdgcn_sched_barrier(0);
            }
            if ((q & 1) == 1) {
                const int i = q >> 1;
                if (i < 8) {
                    if (t + 2 < nk) issue_one(Ablk, a_off, ub, (t + 2) * TK, false, i);  // -> unit 2t
                } else {
                    if (t + 3 < nk) issue_one(Bblk, b_off, ua, (t + 3) * TK, NTW, i - 8);
                }
                __builtin_amdgcn_sched_barrier(0);
            }
        }
        ub = ub1;
        ua = ua1;
    }
    {   // last k-tile
        load(fa1, fb1, ua, ub, 1);
        mma(fa0, fb0, true);
        load(fa0, fb0, ua, ub, 2);
        mma(fa1, fb1, true);
        load(fa1, fb1, ua, ub, 3);
        mma(fa0, fb0, true);
        mma(fa1, fb1, false);
    }

    // Epilogue through LDS: every wave is past its last LDS read of the stages.
    asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
    char* const stg = sm_bytes;
#pragma unroll
    for (int mi = 0; mi < 4; ++mi) {
        char* const rowp = stg + (wm * 128 + mi * 32 + l32) * PITCH + hi * 8;
#pragma unroll
        for (int ni = 0; ni < ((MODE == 0) ? 2 : 4); ++ni)
#pragma unroll
            for (int g = 0; g < 4; ++g) {
                float v[4];
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    const float a0 = acc[mi][ni][4 * g + r];
                    v[r] = (MODE == 0) ? silu(a0) * acc[mi][ni + 2][4 * g + r] : a0;
                }
                const int col = ((MODE == 0) ? wn * 64 : wn * 128) + ni * 32 + g * 8;
                u32x2_t pk = {pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3])};
                *reinterpret_cast<u32x2_t*>(rowp + col * 2) = pk;
            }
    }
    __syncthreads();
    // each thread stores one fixed 16-byte column chunk of every RPI-th row
    constexpr int CPR = OUTC * 2 / 16;  // 16-byte chunks per row
    constexpr int RPI = 256 / CPR;      // rows per pass of the block
    const int cc = tid % CPR, r0 = tid / CPR;
    const int ldc = (MODE == 0) ? m : d;
    const int col = ntile * OUTC + cc * 8;
    const bool col_ok = (MODE == 0) || col < d;
    const char* src = stg + r0 * PITCH + cc * 16;
    bf16_t* dst = C + (int64_t)(row0 + r0) * ldc + col;
#pragma unroll
    for (int b = 0; b < TM / RPI; b += 16) {
        u32x4_t v[16];
#pragma unroll
        for (int i = 0; i < 16; ++i)
            v[i] = *reinterpret_cast<const u32x4_t*>(src + (b + i) * RPI * PITCH);
#pragma unroll
        for (int i = 0; i < 16; ++i)
            if (col_ok && r0 + (b + i) * RPI < rows)
                *reinterpret_cast<u32x4_t*>(dst + (int64_t)(b + i) * RPI * ldc) = v[i];
    }
}

template <int MODE>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(1, 1))) void gemm_bf16_dma(
    const bf16_t* __restrict__ A, const int* __restrict__ row_token,
    const bf16_t* __restrict__ B, const int* __restrict__ offsets,
    const int* __restrict__ tile_off, const int* __restrict__ tail_list, int big_blocks,
    int N, int d, int m, bf16_t* __restrict__ C, int nt_weights) {
    // One array: its address is passed to the copy instructions (inline assembly), which tells
    // the compiler that all of it may be written there.
    __shared__ __attribute__((aligned(1024))) char sm_bytes[5 * 256 * 64 * 2];
    if (nt_weights)  // kernel-uniform
        gemm_dma_body<MODE, true>(A, row_token, B, offsets, tile_off, tail_list, big_blocks, N,
                                  d, m, C, sm_bytes);
    else
        gemm_dma_body<MODE, false>(A, row_token, B, offsets, tile_off, tail_list, big_blocks, N,
                                   d, m, C, sm_bytes);
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

int gemm_tile_rows(int dtype, int64_t T, int K, int N, int d, int m) {
    if (dtype != ELB_BF16) return FBM;
    const int64_t avg_rows = T * K / (N > 0 ? N : 1);
    // the large-tile kernel's 32-bit byte offsets: gathered x rows from x itself (T d
    // elements), weights from the expert's own matrix (2 m d elements); larger problems take
    // the 128-row kernel, which addresses with 64-bit pointers
    const bool offsets_fit = (uint64_t)T * (uint64_t)d * 2u < ((uint64_t)1 << 32) &&
                             (uint64_t)m * (uint64_t)d * 4u < ((uint64_t)1 << 32);
    // from about 96 rows per expert the 256-row tiles are faster (measured on the OLMoE-shaped
    // layer: at 120 rows per expert gate/up 161 -> 140 us; at 60 rows the two are even)
    return (m % 128 == 0 && d >= 128 && T > 0 && avg_rows >= 96 && offsets_fit) ? LBM : BM;
}

hipError_t launch_gemm_gate_up(const void* x, const void* Wgu, const int* row_token,
                               const int* offsets, const int* tile_off, const int* tail_list,
                               int64_t max_tiles, int tile_rows, int d, int N, int m,
                               int dtype, void* H, hipStream_t s, bool nt_weights) {
    if (max_tiles <= 0) return hipSuccess;
    if (dtype == ELB_BF16 && tile_rows == LBM) {
        ProfileScope prof("gemm_gate_up_bf16", s);
        const unsigned big = grid8(max_tiles * (m / 128));
        const unsigned tail = tail_list ? (unsigned)(kTailMax * (m / 32)) : 0u;
        ELB_LAUNCH(gemm_bf16_dma<0>, dim3(big + tail), dim3(256), 0, s,
                           (const bf16_t*)x, row_token, (const bf16_t*)Wgu, offsets, tile_off,
                           tail_list, (int)big, N, d, m, (bf16_t*)H, (int)nt_weights);
    } else if (dtype == ELB_BF16) {
        ProfileScope prof("gemm_gate_up_bf16_s", s);
        ELB_LAUNCH(gemm_bf16<0>, dim3(grid8(max_tiles * (m / 64))), dim3(256),
                           0, s, (const bf16_t*)x, row_token, (const bf16_t*)Wgu, offsets,
                           tile_off, N, d, m, (bf16_t*)H);
    } else {
        ProfileScope prof("gemm_gate_up_f32", s);
        ELB_LAUNCH(gemm_f32<0>, dim3((unsigned)max_tiles, (unsigned)((m + 31) / 32)),
                           dim3(256), 0, s, (const float*)x, row_token, (const float*)Wgu,
                           offsets, tile_off, N, d, m, (float*)H);
    }
    return hipGetLastError();
}

hipError_t launch_gemm_down(const void* H, const void* Wd, const int* offsets,
                            const int* tile_off, const int* tail_list, int64_t max_tiles,
                            int tile_rows, int d, int N, int m, int dtype, void* Y,
                            hipStream_t s, bool nt_weights) {
    if (max_tiles <= 0) return hipSuccess;
    if (dtype == ELB_BF16 && tile_rows == LBM) {
        ProfileScope prof("gemm_down_bf16", s);
        const unsigned big = grid8(max_tiles * ((d + LBN - 1) / LBN));
        const unsigned tail = tail_list ? (unsigned)(kTailMax * (d / 64)) : 0u;
        ELB_LAUNCH(gemm_bf16_dma<1>, dim3(big + tail), dim3(256), 0, s,
                           (const bf16_t*)H, (const int*)nullptr, (const bf16_t*)Wd, offsets,
                           tile_off, tail_list, (int)big, N, d, m, (bf16_t*)Y, (int)nt_weights);
    } else if (dtype == ELB_BF16) {
        ProfileScope prof("gemm_down_bf16_s", s);
        ELB_LAUNCH(gemm_bf16<1>, dim3(grid8(max_tiles * ((d + BN - 1) / BN))),
                           dim3(256), 0, s, (const bf16_t*)H, (const int*)nullptr,
                           (const bf16_t*)Wd, offsets, tile_off, N, d, m, (bf16_t*)Y);
    } else {
        ProfileScope prof("gemm_down_f32", s);
        ELB_LAUNCH(gemm_f32<1>, dim3((unsigned)max_tiles, (unsigned)((d + FBN - 1) / FBN)),
                           dim3(256), 0, s, (const float*)H, (const int*)nullptr,
                           (const float*)Wd, offsets, tile_off, N, d, m, (float*)Y);
    }
    return hipGetLastError();
}

}  // namespace elb
