// Internal declarations shared by the HIP sources of libelbow_moe (not part of the ABI).
#pragma once

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "elbow_moe.h"

namespace elb {

// bf16 is stored as uint16 (the upper half of an fp32 bit pattern).
typedef uint16_t bf16_t;
typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

__device__ __forceinline__ float bf16_to_f32(bf16_t v) {
    return __uint_as_float(((uint32_t)v) << 16);
}

// round to nearest even (finite inputs; NaN keeps a quiet NaN pattern)
__device__ __forceinline__ bf16_t f32_to_bf16(float f) {
    uint32_t u = __float_as_uint(f);
    if ((u & 0x7fffffffu) > 0x7f800000u) return (bf16_t)((u >> 16) | 0x40);
    u += 0x7fffu + ((u >> 16) & 1u);
    return (bf16_t)(u >> 16);
}

constexpr int kWave = 64;

// LDS pointers as 32-bit LDS addresses (for the M0 operand of global_load_lds_dwordx4)
typedef __attribute__((address_space(3))) void lds_void_t;

// s_waitcnt vmcnt(n) (expcnt and lgkmcnt not waited on); n a compile-time constant
#define ELB_WAIT_VMCNT(n) __builtin_amdgcn_s_waitcnt(((n) & 15) | (((n) >> 4) << 14) | 0x0F70)

// ---- kernel launchers (defined in the .hip files); each returns hipGetLastError() ----

// routing: logits [T, N] -> k [T], ids [T, K], w [T, K]
hipError_t launch_route(const float* logits, int64_t T, int N, const elb_route_params& p,
                        int* k, int* ids, float* w, hipStream_t s);

// routing variants (caps above kLaneMaxK, tail randomisation when `rand` is set, the elbow
// index `e` and angle `theta` when set); ids == nullptr: no selection (diagnostics only)
constexpr int kLaneMaxK = 16;  // largest cap of the lane-per-token routing kernel
// batches of at most this many tokens are latency-bound: the router GEMM splits the experts
// over blocks and the routing gives each token 16 lanes (N = 64)
constexpr int64_t kSmallBatch = 1024;
hipError_t launch_route_pair(const float* logits, const float* rand, int64_t T, int N,
                             const elb_route_params& p, int* k, int* ids, float* w, int* e,
                             float* theta, hipStream_t s);

// dispatch: number of 64-token groups; the histogram's row stride (groups rounded up to a
// multiple of 4, so that every expert's row is 16-byte aligned) and its size in ints
inline int64_t dispatch_groups(int64_t T) { return (T + kWave - 1) / kWave; }
inline int64_t dispatch_hist_ld(int64_t T) { return (dispatch_groups(T) + 3) & ~(int64_t)3; }
inline int64_t dispatch_hist_ints(int64_t T, int N) { return dispatch_hist_ld(T) * N; }
// up to this many groups the scatter sums the histogram itself (no scan launch); the
// histogram is then group-major ([hist_ld, N]: row g holds the N counts of group g), else
// expert-major ([N, hist_ld]) for the scan
constexpr int64_t kDirectGroups = 128;
// the split router's routing for T <= 64 kDirectGroups runs 16 tokens per block and writes
// one group-major histogram per quarter of each 64-token group: kHistSubs histograms of
// hist_ld x N ints, one after the other, which the scatter adds up
constexpr int kHistSubs = 4;
inline int split_hist_subs(int64_t T) {
    return dispatch_groups(T) <= kDirectGroups ? kHistSubs : 1;
}

// M-tiling of the grouped GEMMs, computed by the dispatch on the device from the counts.
// Each expert gets ceil(c / tile_rows) M-tiles, except that with tail_rows > 0 an expert with
// at least one full tile and a remainder of at most tail_rows rows may leave that remainder to
// the tail kernel (listed in tail_list: count, then expert ids) -- done only when it lowers
// the number of rounds of tiles_per_round M-tiles and at most tail_max experts are concerned.
struct TilePlan {
    int tile_rows;
    int tail_rows;
    int tiles_per_round;
    int tail_max;
};
constexpr int kTailMax = 16;   // most experts whose remainders go to the tail kernel
constexpr int kTailRows = 32;  // largest remainder the tail kernel takes

// hist: dispatch_hist_ints(T, N) int32 scratch (group-major up to kDirectGroups groups,
// else expert-major);
// tile_off [N + 1]; tail_list [kTailMax + 1]
// hist_ready: hist already holds the per-group counts (written by the split router), so the
// count launch is skipped; hist_subs: how many histograms it holds (split_hist_subs(T) from
// the split router, else 1)
hipError_t launch_dispatch(const int* k, const int* ids, int64_t T, int N, int K, int* counts,
                           int* offsets, int* row_token, int* inv, int* hist, int* tile_off,
                           int* tail_list, const TilePlan& plan, hipStream_t s,
                           bool hist_ready = false, int hist_subs = 1);

// router logits
hipError_t launch_router(const void* x, const void* Wr, int64_t T, int d, int N, int dtype,
                         float* logits, hipStream_t s);

// router GEMM fused with the routing (bf16, K <= kLaneMaxK); logits == nullptr: not written
bool router_route_fusable(int dtype, int K);
hipError_t launch_router_route(const void* x, const void* Wr, int64_t T, int d, int N,
                               const elb_route_params& p, float* logits, int* k, int* ids,
                               float* w, hipStream_t s);

// the layer's router and routing for large batches in two launches (N == 64, bf16, K <=
// kLaneMaxK, T > kSmallBatch, d % 256 == 0): partial logits per quarter of the contraction
// into part [4, T, 64] (workspace), then their sum and the routing; also writes the dispatch
// histogram: split_hist_subs(T) histograms [64, hist_ld] (column g = tokens [64 g, 64 g + 64),
// or its quarter j in histogram j).  Same bits as the other router paths.
// router + routing in one launch (N = 64, d % 256 == 0, at most kRouteDmaMaxT tokens,
// K <= kLaneMaxK): 16 tokens per block, the contraction's quarters in the block's four waves;
// the same bits as the split form; hist (optional) as launch_router_split_route writes it
// (kHistSubs histograms, group-major)
constexpr int64_t kRouteDmaMaxT = 4096;
static_assert(kRouteDmaMaxT <= 64 * kDirectGroups, "the one-launch form writes kHistSubs "
                                                   "histograms");
bool router_route_dma_usable(int dtype, int64_t T, int d, int N, int K);
hipError_t launch_router_route_dma(const void* x, const void* Wr, int64_t T, int d,
                                   const elb_route_params& p, float* logits, int* k, int* ids,
                                   float* w, int* hist, int64_t hist_ld, hipStream_t s);
bool router_split_usable(int dtype, int64_t T, int d, int N, int K);
hipError_t launch_router_split_route(const void* x, const void* Wr, int64_t T, int d,
                                     const elb_route_params& p, float* part, float* logits,
                                     int* k, int* ids, float* w, int* hist, int64_t hist_ld,
                                     hipStream_t s);

// the layer's router and routing for batches of at most kSmallBatch tokens with N == 64
// (bf16, K <= kLaneMaxK): one wave per (16 tokens, 16 experts, quarter of the contraction)
// into part [4, T, 64], then the 16-lane split routing (histograms as above, split_hist_subs(T)
// of them).  Same bits as the other router paths.
bool router_slices_usable(int dtype, int64_t T, int N, int K);
hipError_t launch_router_slices_route(const void* x, const void* Wr, int64_t T, int d,
                                      const elb_route_params& p, float* part, float* logits,
                                      int* k, int* ids, float* w, int* hist, int64_t hist_ld,
                                      hipStream_t s);

// grouped GEMMs
// rows per M-tile of the grouped GEMMs for this problem (the dispatch scan uses the same)
int gemm_tile_rows(int dtype, int64_t T, int K, int N, int d, int m);
// tail_list (large-tile kernels only, TilePlan): its experts' remainder rows are computed
// by extra blocks of the same launch.  nt_weights (large-tile kernels): the weight copies carry
// the non-temporal hint (gemm_stream_weights)
hipError_t launch_gemm_gate_up(const void* x, const void* Wgu, const int* row_token,
                               const int* offsets, const int* tile_off, const int* tail_list,
                               int64_t max_tiles, int tile_rows, int d, int N, int m,
                               int dtype, void* H, hipStream_t s, bool nt_weights);
hipError_t launch_gemm_down(const void* H, const void* Wd, const int* offsets,
                            const int* tile_off, const int* tail_list, int64_t max_tiles,
                            int tile_rows, int d, int N, int m, int dtype, void* Y,
                            hipStream_t s, bool nt_weights);
// whether the large-tile GEMMs stream the weights with the non-temporal hint: yes while an
// expert has at most about three M-tiles of rows (its weight tiles are read by few blocks),
// no above, where the tiles are read by many blocks and are better kept in the caches
inline bool gemm_stream_weights(int64_t T, int K, int N) {
    return T * K < (int64_t)768 * (N > 0 ? N : 1);
}

// decode-sized batches: weight-streaming gate/up (+SwiGLU) and down GEMMs, both launched
bool gemm_use_skinny(int dtype, int64_t T, int K, int N, int d, int m);
// rows are assignment slots t K + j found from the routing (k, ids) itself (no dispatch):
// H [T K, m], Y [T K, d]; counts (optional): assignments per expert.  packed: the weights'
// packed copy (launch_pack_experts) or nullptr for the row-major ones
hipError_t launch_gemm_skinny(const void* x, const void* Wgu, const void* Wd, const void* packed,
                              const int* k, const int* ids, int64_t T, int K, int d, int N,
                              int m, void* H, void* Y, int* counts, hipStream_t s);
// the packed copy of bf16 W_gate_up [N, 2m, d] and W_down [N, d, m] (same total size)
hipError_t launch_pack_experts(const void* Wgu, const void* Wd, int N, int d, int m,
                               void* packed, hipStream_t s);

// MI355X's last-level (Infinity) cache: data larger than this streams from HBM
constexpr size_t kLastLevelCacheBytes = (size_t)256 << 20;

// combine: y[t] = residual[t] + sum_j w[t, j] Y[inv[t, j]]  (inv == nullptr: row t K + j)
hipError_t launch_combine(const void* Y, const int* k, const int* inv, const float* w,
                          const void* residual, int64_t T, int d, int K, int dtype, void* y,
                          hipStream_t s);

// calibration: back-to-back bf16 MFMAs, blocks x 4 waves x iters x 8 of them; out [blocks * 4]
hipError_t launch_calibrate_mfma(int blocks, int iters, float* out, hipStream_t s);
hipError_t launch_calibrate_read(const void* buf, int64_t bytes, int blocks, uint32_t* out,
                                 hipStream_t s);

// ---- per-kernel timing hooks (api.hip) ----
// A ProfileScope names the launches made while it is alive (on the calling thread).  With the
// library's profiling on, every ELB_LAUNCH inside a scope carries a start and a stop event in
// its own dispatch (hipExtLaunchKernelGGL), so timing adds no packets, and no idle gaps,
// between kernels; with profiling off it is a plain launch.
struct ProfileScope {
    ProfileScope(const char* name, hipStream_t s);
    ~ProfileScope();
    const char* prev_name_;
    int prev_id_;
};
// events for the next launch of the current scope (false: profiling off or no scope)
bool profile_events(hipEvent_t* start, hipEvent_t* stop);

#define ELB_LAUNCH(kernel, grid, block, shmem, stream, ...)                                   \
    do {                                                                                      \
        hipEvent_t elb_e0_ = nullptr, elb_e1_ = nullptr;                                       \
        if (::elb::profile_events(&elb_e0_, &elb_e1_))                                         \
            hipExtLaunchKernelGGL(kernel, grid, block, shmem, stream, elb_e0_, elb_e1_, 0,     \
                                  __VA_ARGS__);                                               \
        else                                                                                  \
            hipLaunchKernelGGL(kernel, grid, block, shmem, stream, __VA_ARGS__);              \
    } while (0)

}  // namespace elb
