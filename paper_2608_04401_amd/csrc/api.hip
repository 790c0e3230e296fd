// C ABI of libelbow_moe: argument validation, workspace carving, launch order, timing hooks.
#include <algorithm>
#include <atomic>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <map>
#include <mutex>
#include <string>
#include <vector>

#include "common.h"

namespace elb {

namespace {

thread_local std::string g_err;

int fail(int code, const char* fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof(buf), fmt, ap);
    va_end(ap);
    g_err = buf;
    return code;
}

int hip_status(hipError_t e, const char* where) {
    if (e == hipSuccess) return ELB_OK;
    return fail(ELB_ERR_HIP, "%s: %s", where, hipGetErrorString(e));
}

constexpr size_t kAlign = 256;
inline size_t align_up(size_t v) { return (v + kAlign - 1) / kAlign * kAlign; }

// Sub-buffers carved from the caller's workspace, in this order.
struct Layout {
    size_t hist, tile_off, counts, offsets, row_token, inv, H, Y;  // expert part
    size_t logits, k, ids, w, part;                                // routing (forward only)
    size_t experts_end, total;
};

size_t esize(int dtype) { return dtype == ELB_BF16 ? 2 : 4; }

Layout layout(int64_t T, int d, int N, int m, int K, int dtype) {
    Layout L{};
    size_t o = 0;
    auto take = [&](size_t bytes) {
        const size_t at = o;
        o += align_up(bytes);
        return at;
    };
    const size_t rows = (size_t)T * K;
    // the split router's routing may write split_hist_subs(T) histograms
    L.hist = take((size_t)dispatch_hist_ints(T, N) * split_hist_subs(T) * 4);
    L.tile_off = take((size_t)(N + 1 + kTailMax + 1) * 4);  // tile_off, then tail_list
    L.counts = take((size_t)N * 4);
    L.offsets = take((size_t)(N + 1) * 4);
    L.row_token = take(rows * 4);
    L.inv = take(rows * 4);
    L.H = take(rows * m * esize(dtype));
    L.Y = take(rows * d * esize(dtype));
    L.experts_end = o;
    L.logits = take((size_t)T * N * 4);
    L.k = take((size_t)T * 4);
    L.ids = take(rows * 4);
    L.w = take(rows * 4);
    L.part = take((size_t)4 * T * N * 4);  // the split router's partial logits
    L.total = o;
    return L;
}

// compute units of the current device (cached; at least 1)
int cus_per_device() {
    static std::atomic<int> cache[64];
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
    int v = cache[dev].load();
    if (v == 0) {
        if (hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
            v < 1)
            v = 256;
        cache[dev].store(v);
    }
    return v;
}

int64_t max_tiles(int64_t T, int K, int N, int tile_rows) {
    // sum_e ceil(c_e / BM) <= (sum_e c_e + N (BM - 1)) / BM, sum_e c_e <= T K
    return (T * K + (int64_t)N * (tile_rows - 1)) / tile_rows;
}

int check_route_params(int N, const elb_route_params* p) {
    if (!p) return fail(ELB_ERR_INVALID_ARG, "params is NULL");
    if (N < 2) return fail(ELB_ERR_INVALID_ARG, "N = %d: need at least 2 experts", N);
    if (N > ELB_MAX_EXPERTS)
        return fail(ELB_ERR_UNSUPPORTED, "N = %d exceeds ELB_MAX_EXPERTS = %d", N,
                    ELB_MAX_EXPERTS);
    if (p->K < 1 || p->K > N)
        return fail(ELB_ERR_INVALID_ARG, "K = %d outside [1, N = %d]", p->K, N);
    if (!(p->eps >= 0.f) || !std::isfinite(p->eps))
        return fail(ELB_ERR_INVALID_ARG, "eps = %g must be finite and >= 0", (double)p->eps);
    if (p->mode != ELB_MODE_ELBOW && p->mode != ELB_MODE_TOPK)
        return fail(ELB_ERR_INVALID_ARG, "mode = %d is not an elb_mode", p->mode);
    if (p->renormalize != 0 && p->renormalize != 1)
        return fail(ELB_ERR_INVALID_ARG, "renormalize = %d must be 0 or 1", p->renormalize);
    return ELB_OK;
}

int check_dtype(int dtype) {
    if (dtype != ELB_F32 && dtype != ELB_BF16)
        return fail(ELB_ERR_INVALID_ARG, "dtype = %d is not an elb_dtype", dtype);
    return ELB_OK;
}

int check_expert_dims(int64_t T, int d, int N, int m, int K, int dtype) {
    if (int rc = check_dtype(dtype)) return rc;
    if (T < 0) return fail(ELB_ERR_INVALID_ARG, "T = %lld < 0", (long long)T);
    if (N < 2) return fail(ELB_ERR_INVALID_ARG, "N = %d: need at least 2 experts", N);
    if (N > ELB_MAX_EXPERTS)
        return fail(ELB_ERR_UNSUPPORTED, "N = %d exceeds ELB_MAX_EXPERTS = %d", N,
                    ELB_MAX_EXPERTS);
    if (K < 1 || K > N) return fail(ELB_ERR_INVALID_ARG, "K = %d outside [1, N = %d]", K, N);
    if (d < 1 || m < 1) return fail(ELB_ERR_INVALID_ARG, "d = %d, m = %d must be >= 1", d, m);
    const int g = dtype == ELB_BF16 ? 64 : 16;
    if (d % g || m % g)
        return fail(ELB_ERR_INVALID_ARG, "d = %d and m = %d must be multiples of %d for %s", d,
                    m, g, dtype == ELB_BF16 ? "bf16" : "f32");
    if (T * (int64_t)K >= (int64_t)1 << 31)
        return fail(ELB_ERR_UNSUPPORTED, "T * K = %lld assignments exceed 2^31",
                    (long long)(T * K));
    return ELB_OK;
}

// ---- the static scratch of the allocation-free entry point ----
// One array per GPU the library runs on (a __device__ variable lives in each device's copy of
// the code object).  In host code `scratch` is only a stand-in symbol: its device address is
// looked up with hipGetSymbolAddress, once per device with that device current, and only that
// address is passed to kernels.
constexpr size_t kScratchBytes = (size_t)ELB_NOALLOC_SCRATCH_BYTES;
static __device__ __attribute__((aligned(256))) char scratch[kScratchBytes];
std::mutex g_scratch_mu;
void* g_scratch_ptr[64] = {};

int scratch_address(void** out) {
    int dev = 0;
    if (hipError_t e = hipGetDevice(&dev)) return hip_status(e, "hipGetDevice");
    if (dev < 0 || dev >= 64) return fail(ELB_ERR_UNSUPPORTED, "device index %d >= 64", dev);
    std::lock_guard<std::mutex> lk(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void* p = nullptr;
        const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return hip_status(e, "hipGetSymbolAddress(scratch)");
        if (!p || (uintptr_t)p % kAlign)
            return fail(ELB_ERR_HIP, "scratch address %p is null or not %zu-byte aligned", p,
                        kAlign);
        g_scratch_ptr[dev] = p;
    }
    *out = g_scratch_ptr[dev];
    return ELB_OK;
}

// ---- per-kernel timing ----
struct Rec {
    const char* name;
    int scope;  // the ProfileScope instance (a scope may make several launches)
    hipEvent_t a, b;
};
std::atomic<int> g_prof_on{0};  // 0 off, 1 every launch, 2 the grouped expert GEMMs only
std::atomic<int> g_scope_seq{0};
std::mutex g_prof_mu;
std::vector<Rec> g_recs;
std::vector<hipEvent_t> g_pool;
thread_local const char* t_scope_name = nullptr;
thread_local int t_scope_id = 0;

hipEvent_t pool_get() {
    if (!g_pool.empty()) {
        hipEvent_t e = g_pool.back();
        g_pool.pop_back();
        return e;
    }
    // timing only: without the system-scope fence an event does not write back and
    // invalidate the caches
    hipEvent_t e = nullptr;
    if (hipEventCreateWithFlags(&e, hipEventDisableSystemFence) != hipSuccess) return nullptr;
    return e;
}

}  // namespace

ProfileScope::ProfileScope(const char* name, hipStream_t) : prev_name_(t_scope_name),
                                                            prev_id_(t_scope_id) {
    const int lvl = g_prof_on.load(std::memory_order_relaxed);
    if (lvl == 1 || (lvl == 2 && std::strncmp(name, "gemm_", 5) == 0)) {
        t_scope_name = name;
        t_scope_id = ++g_scope_seq;
    } else {
        t_scope_name = nullptr;
    }
}

ProfileScope::~ProfileScope() {
    t_scope_name = prev_name_;
    t_scope_id = prev_id_;
}

bool profile_events(hipEvent_t* start, hipEvent_t* stop) {
    if (!t_scope_name || !g_prof_on.load(std::memory_order_relaxed)) return false;
    std::lock_guard<std::mutex> lk(g_prof_mu);
    Rec r{t_scope_name, t_scope_id, pool_get(), pool_get()};
    if (!r.a || !r.b) {
        if (r.a) g_pool.push_back(r.a);
        if (r.b) g_pool.push_back(r.b);
        return false;
    }
    g_recs.push_back(r);
    *start = r.a;
    *stop = r.b;
    return true;
}

}  // namespace elb

using namespace elb;

extern "C" {

int elb_abi_version(void) { return ELB_ABI_VERSION; }

const char* elb_status_str(int status) {
    switch (status) {
        case ELB_OK: return "ELB_OK";
        case ELB_ERR_INVALID_ARG: return "ELB_ERR_INVALID_ARG";
        case ELB_ERR_UNSUPPORTED: return "ELB_ERR_UNSUPPORTED";
        case ELB_ERR_WORKSPACE: return "ELB_ERR_WORKSPACE";
        case ELB_ERR_HIP: return "ELB_ERR_HIP";
        default: return "ELB_ERR_UNKNOWN";
    }
}

const char* elb_last_error(void) { return g_err.c_str(); }

int elb_router_logits(const void* x, const void* W_router, int64_t T, int32_t d, int32_t N,
                      int32_t dtype, float* logits, void* stream) {
    g_err.clear();
    if (int rc = check_dtype(dtype)) return rc;
    if (T < 0) return fail(ELB_ERR_INVALID_ARG, "T = %lld < 0", (long long)T);
    if (N < 2) return fail(ELB_ERR_INVALID_ARG, "N = %d: need at least 2 experts", N);
    if (N > ELB_MAX_EXPERTS)
        return fail(ELB_ERR_UNSUPPORTED, "N = %d exceeds %d", N, ELB_MAX_EXPERTS);
    if (d < 1) return fail(ELB_ERR_INVALID_ARG, "d = %d < 1", d);
    if (dtype == ELB_BF16 && d % 32)
        return fail(ELB_ERR_INVALID_ARG, "bf16 router needs d %% 32 == 0 (d = %d)", d);
    if (T == 0) return ELB_OK;
    if (!x || !W_router || !logits) return fail(ELB_ERR_INVALID_ARG, "NULL tensor pointer");
    return hip_status(launch_router(x, W_router, T, d, N, dtype, logits, (hipStream_t)stream),
                      "router");
}

int elb_route(const float* logits, int64_t T, int32_t N, const elb_route_params* params,
              int32_t* k, int32_t* ids, float* w, void* stream) {
    g_err.clear();
    if (T < 0) return fail(ELB_ERR_INVALID_ARG, "T = %lld < 0", (long long)T);
    if (int rc = check_route_params(N, params)) return rc;
    if (T == 0) return ELB_OK;
    if (!logits || !k || !ids || !w) return fail(ELB_ERR_INVALID_ARG, "NULL tensor pointer");
    return hip_status(launch_route(logits, T, N, *params, k, ids, w, (hipStream_t)stream),
                      "route");
}

int elb_router_route(const void* x, const void* W_router, int64_t T, int32_t d, int32_t N,
                     int32_t dtype, const elb_route_params* params, float* logits_out,
                     int32_t* k, int32_t* ids, float* w, void* stream) {
    g_err.clear();
    if (int rc = check_dtype(dtype)) return rc;
    if (T < 0) return fail(ELB_ERR_INVALID_ARG, "T = %lld < 0", (long long)T);
    if (int rc = check_route_params(N, params)) return rc;
    if (d < 1) return fail(ELB_ERR_INVALID_ARG, "d = %d < 1", d);
    if (!router_route_fusable(dtype, params->K))
        return fail(ELB_ERR_UNSUPPORTED, "the fused router and routing needs bf16 and K <= %d",
                    kLaneMaxK);
    if (d % 32) return fail(ELB_ERR_INVALID_ARG, "bf16 router needs d %% 32 == 0 (d = %d)", d);
    if (T == 0) return ELB_OK;
    if (!x || !W_router || !k || !ids || !w)
        return fail(ELB_ERR_INVALID_ARG, "NULL tensor pointer");
    if (router_route_dma_usable(dtype, T, d, N, params->K))
        return hip_status(launch_router_route_dma(x, W_router, T, d, *params, logits_out, k,
                                                  ids, w, nullptr, 0, (hipStream_t)stream),
                          "router_route");
    return hip_status(launch_router_route(x, W_router, T, d, N, *params, logits_out, k, ids, w,
                                          (hipStream_t)stream),
                      "router_route");
}

int elb_route_tail_random(const float* logits, const float* rand, int64_t T, int32_t N,
                          const elb_route_params* params, int32_t* k_elbow, int32_t* ids,
                          float* w, void* stream) {
    g_err.clear();
    if (T < 0) return fail(ELB_ERR_INVALID_ARG, "T = %lld < 0", (long long)T);
    if (int rc = check_route_params(N, params)) return rc;
    if (T == 0) return ELB_OK;
    if (!logits || !rand || !k_elbow || !ids || !w)
        return fail(ELB_ERR_INVALID_ARG, "NULL tensor pointer");
    return hip_status(launch_route_pair(logits, rand, T, N, *params, k_elbow, ids, w, nullptr,
                                        nullptr, (hipStream_t)stream),
                      "route_tail_random");
}

int elb_elbow_angle(const float* logits, int64_t T, int32_t N, float eps, int32_t* e,
                    float* theta, void* stream) {
    g_err.clear();
    if (T < 0) return fail(ELB_ERR_INVALID_ARG, "T = %lld < 0", (long long)T);
    const elb_route_params p{N, eps, ELB_MODE_ELBOW, 0};
    if (int rc = check_route_params(N, &p)) return rc;
    if (T == 0) return ELB_OK;
    if (!logits) return fail(ELB_ERR_INVALID_ARG, "NULL tensor pointer");
    if (!e && !theta) return ELB_OK;  // nothing asked for
    return hip_status(launch_route_pair(logits, nullptr, T, N, p, nullptr, nullptr, nullptr, e,
                                        theta, (hipStream_t)stream),
                      "elbow_angle");
}

size_t elb_dispatch_workspace_bytes(int64_t T, int32_t N) {
    if (T < 0 || N < 1) return 0;
    return align_up((size_t)dispatch_hist_ints(T, N) * 4) +
           align_up((size_t)(N + 1 + kTailMax + 1) * 4);
}

int elb_dispatch(const int32_t* k, const int32_t* ids, int64_t T, int32_t N, int32_t K,
                 int32_t* counts, int32_t* offsets, int32_t* row_token, int32_t* inv,
                 void* workspace, size_t workspace_bytes, void* stream) {
    g_err.clear();
    if (T < 0) return fail(ELB_ERR_INVALID_ARG, "T = %lld < 0", (long long)T);
    if (N < 2) return fail(ELB_ERR_INVALID_ARG, "N = %d: need at least 2 experts", N);
    if (N > ELB_MAX_EXPERTS)
        return fail(ELB_ERR_UNSUPPORTED, "N = %d exceeds %d", N, ELB_MAX_EXPERTS);
    if (K < 1 || K > N) return fail(ELB_ERR_INVALID_ARG, "K = %d outside [1, N = %d]", K, N);
    if (T * (int64_t)K >= (int64_t)1 << 31)
        return fail(ELB_ERR_UNSUPPORTED, "T * K exceeds 2^31");
    if (!counts || !offsets) return fail(ELB_ERR_INVALID_ARG, "NULL tensor pointer");
    if (T > 0 && (!k || !ids || !row_token || !inv))
        return fail(ELB_ERR_INVALID_ARG, "NULL tensor pointer");
    const size_t need = elb_dispatch_workspace_bytes(T, N);
    if (!workspace || workspace_bytes < need)
        return fail(ELB_ERR_WORKSPACE, "workspace of %zu bytes, need %zu", workspace_bytes, need);
    if ((uintptr_t)workspace % kAlign)
        return fail(ELB_ERR_WORKSPACE, "workspace not %zu-byte aligned", kAlign);
    char* ws = (char*)workspace;
    int* hist = (int*)ws;
    int* tile_off = (int*)(ws + align_up((size_t)dispatch_hist_ints(T, N) * 4));
    const TilePlan plan{128, 0, 1, kTailMax};  // plain ceil(c / 128) tiles, no tail list use
    return hip_status(launch_dispatch(k, ids, T, N, K, counts, offsets, row_token, inv, hist,
                                      tile_off, tile_off + N + 1, plan, (hipStream_t)stream),
                      "dispatch");
}

size_t elb_moe_workspace_bytes(int64_t T, int32_t d, int32_t N, int32_t m, int32_t K,
                               int32_t dtype) {
    if (T < 0 || d < 1 || N < 1 || m < 1 || K < 1 || (dtype != ELB_F32 && dtype != ELB_BF16))
        return 0;
    return layout(T, d, N, m, K, dtype).total;
}

static int experts_impl(const void* x, const void* W_gate_up, const void* W_down,
                        const void* packed,
                        const int32_t* k, const int32_t* ids, const float* w,
                        const void* residual, int64_t T, int d, int N, int m, int K, int dtype,
                        void* y, char* ws, const Layout& L, int32_t* counts_out,
                        hipStream_t s, bool hist_ready = false, int hist_subs = 1) {
    int* hist = (int*)(ws + L.hist);
    int* tile_off = (int*)(ws + L.tile_off);
    int* counts = counts_out ? counts_out : (int*)(ws + L.counts);
    int* offsets = (int*)(ws + L.offsets);
    int* row_token = (int*)(ws + L.row_token);
    int* inv = (int*)(ws + L.inv);
    void* H = ws + L.H;
    void* Y = ws + L.Y;
    const int tr = gemm_tile_rows(dtype, T, K, N, d, m);
    const int64_t mt = max_tiles(T, K, N, tr);
    int* tail_list = tile_off + N + 1;
    // the large-tile kernel (256-row tiles, m / 128 tiles across per M-tile, one block per
    // CU) leaves short remainders to the tail kernel when that saves a round of blocks
    const bool big = (dtype == ELB_BF16 && tr == 256);
    const TilePlan plan{tr, big ? kTailRows : 0, big ? cus_per_device() / (m / 128) : 1,
                        kTailMax};
    if (gemm_use_skinny(dtype, T, K, N, d, m)) {
        // decode-sized: no dispatch; the expert waves find their slots from (k, ids) and
        // write rows t K + j of H and Y, which the combine reads directly
        if (int rc = hip_status(launch_gemm_skinny(x, W_gate_up, W_down, packed, k, ids, T, K,
                                                   d, N, m, H, Y, counts_out, s),
                                "gemm_skinny"))
            return rc;
        return hip_status(launch_combine(Y, k, nullptr, w, residual, T, d, K, dtype, y, s),
                          "combine");
    }
    if (int rc = hip_status(launch_dispatch(k, ids, T, N, K, counts, offsets, row_token, inv,
                                            hist, tile_off, tail_list, plan, s, hist_ready,
                                            hist_subs),
                            "dispatch"))
        return rc;
    {
        const bool ntw = gemm_stream_weights(T, K, N);
        if (int rc = hip_status(launch_gemm_gate_up(x, W_gate_up, row_token, offsets, tile_off,
                                                    big ? tail_list : nullptr, mt, tr, d, N, m,
                                                    dtype, H, s, ntw),
                                "gemm_gate_up"))
            return rc;
        if (int rc = hip_status(launch_gemm_down(H, W_down, offsets, tile_off,
                                                 big ? tail_list : nullptr, mt, tr, d, N, m,
                                                 dtype, Y, s, ntw),
                                "gemm_down"))
            return rc;
    }
    return hip_status(launch_combine(Y, k, inv, w, residual, T, d, K, dtype, y, s), "combine");
}

static int moe_experts_entry(const void* x, const void* W_gate_up, const void* W_down,
                             const void* packed, const int32_t* k, const int32_t* ids,
                             const float* w, const void* residual, int64_t T, int32_t d,
                             int32_t N, int32_t m, int32_t K, int32_t dtype, void* y,
                             void* workspace, size_t workspace_bytes, void* stream) {
    g_err.clear();
    if (int rc = check_expert_dims(T, d, N, m, K, dtype)) return rc;
    if (T == 0) return ELB_OK;
    if (!x || !W_gate_up || !W_down || !k || !ids || !w || !y)
        return fail(ELB_ERR_INVALID_ARG, "NULL tensor pointer");
    const Layout L = layout(T, d, N, m, K, dtype);
    if (!workspace || workspace_bytes < L.experts_end)
        return fail(ELB_ERR_WORKSPACE, "workspace of %zu bytes, need %zu", workspace_bytes,
                    L.experts_end);
    if ((uintptr_t)workspace % kAlign)
        return fail(ELB_ERR_WORKSPACE, "workspace not %zu-byte aligned", kAlign);
    return experts_impl(x, W_gate_up, W_down, packed, k, ids, w, residual, T, d, N, m, K,
                        dtype, y, (char*)workspace, L, nullptr, (hipStream_t)stream);
}

int elb_moe_experts(const void* x, const void* W_gate_up, const void* W_down,
                    const int32_t* k, const int32_t* ids, const float* w, const void* residual,
                    int64_t T, int32_t d, int32_t N, int32_t m, int32_t K, int32_t dtype,
                    void* y, void* workspace, size_t workspace_bytes, void* stream) {
    return moe_experts_entry(x, W_gate_up, W_down, nullptr, k, ids, w, residual, T, d, N, m, K,
                             dtype, y, workspace, workspace_bytes, stream);
}

int elb_moe_experts_packed(const void* x, const void* W_gate_up, const void* W_down,
                           const void* packed, const int32_t* k, const int32_t* ids,
                           const float* w, const void* residual, int64_t T, int32_t d,
                           int32_t N, int32_t m, int32_t K, int32_t dtype, void* y,
                           void* workspace, size_t workspace_bytes, void* stream) {
    return moe_experts_entry(x, W_gate_up, W_down, packed, k, ids, w, residual, T, d, N, m, K,
                             dtype, y, workspace, workspace_bytes, stream);
}

static int moe_forward_entry(const void* x, const void* W_router, const void* W_gate_up,
                             const void* W_down, const void* packed, const void* residual,
                             int64_t T, int32_t d, int32_t N, int32_t m, int32_t dtype,
                             const elb_route_params* params, void* y, void* workspace,
                             size_t workspace_bytes, float* logits_out, int32_t* k_out,
                             int32_t* ids_out, float* w_out, int32_t* counts_out,
                             void* stream) {
    g_err.clear();
    if (int rc = check_route_params(N, params)) return rc;
    if (int rc = check_expert_dims(T, d, N, m, params->K, dtype)) return rc;
    if (T == 0) return ELB_OK;
    if (!x || !W_router || !W_gate_up || !W_down || !y)
        return fail(ELB_ERR_INVALID_ARG, "NULL tensor pointer");
    const int K = params->K;
    const Layout L = layout(T, d, N, m, K, dtype);
    if (!workspace || workspace_bytes < L.total)
        return fail(ELB_ERR_WORKSPACE, "workspace of %zu bytes, need %zu", workspace_bytes,
                    L.total);
    if ((uintptr_t)workspace % kAlign)
        return fail(ELB_ERR_WORKSPACE, "workspace not %zu-byte aligned", kAlign);
    char* ws = (char*)workspace;
    hipStream_t s = (hipStream_t)stream;
    float* logits = logits_out ? logits_out : (float*)(ws + L.logits);
    int* k = k_out ? k_out : (int*)(ws + L.k);
    int* ids = ids_out ? ids_out : (int*)(ws + L.ids);
    float* w = w_out ? w_out : (float*)(ws + L.w);
    // Router and routing, by size (the same bits on every path): large batches with N = 64
    // and d % 256 == 0 split the contraction over four blocks per 64 tokens (two launches; the
    // second also writes the dispatch histogram); small batches with N = 64 take one wave per
    // (16 tokens, 16 experts, quarter of the contraction), then the same 16-lane split
    // routing; the rest the fused one-block kernel, or the router and routing kernels for
    // fp32 and caps above 16.
    const bool skinny = gemm_use_skinny(dtype, T, K, N, d, m);
    if (router_route_dma_usable(dtype, T, d, N, K)) {
        if (int rc = hip_status(
                launch_router_route_dma(x, W_router, T, d, *params, logits_out, k, ids, w,
                                        (int*)(ws + L.hist), dispatch_hist_ld(T), s),
                "router_route_dma"))
            return rc;
        return experts_impl(x, W_gate_up, W_down, packed, k, ids, w, residual, T, d, N, m, K,
                            dtype, y, ws, L, counts_out, s, true, split_hist_subs(T));
    }
    if (router_split_usable(dtype, T, d, N, K) && !skinny) {
        if (int rc = hip_status(
                launch_router_split_route(x, W_router, T, d, *params, (float*)(ws + L.part),
                                          logits_out, k, ids, w, (int*)(ws + L.hist),
                                          dispatch_hist_ld(T), s),
                "router_split_route"))
            return rc;
        return experts_impl(x, W_gate_up, W_down, packed, k, ids, w, residual, T, d, N, m, K,
                            dtype, y, ws, L, counts_out, s, true, split_hist_subs(T));
    }
    if (router_slices_usable(dtype, T, N, K)) {
        if (int rc = hip_status(
                launch_router_slices_route(x, W_router, T, d, *params, (float*)(ws + L.part),
                                           logits_out, k, ids, w, (int*)(ws + L.hist),
                                           dispatch_hist_ld(T), s),
                "router_slices_route"))
            return rc;
        return experts_impl(x, W_gate_up, W_down, packed, k, ids, w, residual, T, d, N, m, K,
                            dtype, y, ws, L, counts_out, s, true, split_hist_subs(T));
    }
    if (router_route_fusable(dtype, K) && !(N == 64 && T <= kSmallBatch)) {
        if (int rc = hip_status(launch_router_route(x, W_router, T, d, N, *params, logits_out,
                                                    k, ids, w, s), "router_route"))
            return rc;
    } else {
        if (int rc = hip_status(launch_router(x, W_router, T, d, N, dtype, logits, s),
                                "router"))
            return rc;
        if (int rc = hip_status(launch_route(logits, T, N, *params, k, ids, w, s), "route"))
            return rc;
    }
    return experts_impl(x, W_gate_up, W_down, packed, k, ids, w, residual, T, d, N, m, K,
                        dtype, y, ws, L, counts_out, s);
}

int elb_moe_forward(const void* x, const void* W_router, const void* W_gate_up,
                    const void* W_down, const void* residual, int64_t T, int32_t d, int32_t N,
                    int32_t m, int32_t dtype, const elb_route_params* params, void* y,
                    void* workspace, size_t workspace_bytes, float* logits_out,
                    int32_t* k_out, int32_t* ids_out, float* w_out, int32_t* counts_out,
                    void* stream) {
    return moe_forward_entry(x, W_router, W_gate_up, W_down, nullptr, residual, T, d, N, m,
                             dtype, params, y, workspace, workspace_bytes, logits_out, k_out,
                             ids_out, w_out, counts_out, stream);
}

int elb_moe_forward_packed(const void* x, const void* W_router, const void* W_gate_up,
                           const void* W_down, const void* packed, const void* residual,
                           int64_t T, int32_t d, int32_t N, int32_t m, int32_t dtype,
                           const elb_route_params* params, void* y, void* workspace,
                           size_t workspace_bytes, float* logits_out, int32_t* k_out,
                           int32_t* ids_out, float* w_out, int32_t* counts_out, void* stream) {
    return moe_forward_entry(x, W_router, W_gate_up, W_down, packed, residual, T, d, N, m,
                             dtype, params, y, workspace, workspace_bytes, logits_out, k_out,
                             ids_out, w_out, counts_out, stream);
}

int elb_moe_forward_noalloc(const void* x, const void* W_router, const void* W_gate_up,
                            const void* W_down, const void* residual, int64_t T, int32_t d,
                            int32_t N, int32_t m, int32_t dtype, const elb_route_params* params,
                            void* y, float* logits_out, int32_t* k_out, int32_t* ids_out,
                            float* w_out, int32_t* counts_out, void* stream) {
    g_err.clear();
    // every size check before any HIP call: an oversized problem is rejected on the host
    if (int rc = check_route_params(N, params)) return rc;
    if (int rc = check_expert_dims(T, d, N, m, params->K, dtype)) return rc;
    if (T == 0) return ELB_OK;
    if (!x || !W_router || !W_gate_up || !W_down || !y)
        return fail(ELB_ERR_INVALID_ARG, "NULL tensor pointer");
    const size_t need = layout(T, d, N, m, params->K, dtype).total;
    if (need > kScratchBytes)
        return fail(ELB_ERR_UNSUPPORTED,
                    "the layer needs %zu bytes of scratch; the allocation-free entry point has "
                    "%zu (use elb_moe_forward with a workspace)", need, kScratchBytes);
    void* ws = nullptr;
    if (int rc = scratch_address(&ws)) return rc;
    return moe_forward_entry(x, W_router, W_gate_up, W_down, nullptr, residual, T, d, N, m,
                             dtype, params, y, ws, kScratchBytes, logits_out, k_out, ids_out,
                             w_out, counts_out, stream);
}

size_t elb_packed_expert_bytes(int32_t N, int32_t d, int32_t m) {
    if (N < 1 || d < 1 || m < 1) return 0;
    return ((size_t)N * 2 * m * d + (size_t)N * d * m) * 2;
}

int elb_pack_expert_weights(const void* W_gate_up, const void* W_down, int32_t N, int32_t d,
                            int32_t m, int32_t dtype, void* packed, void* stream) {
    g_err.clear();
    if (dtype != ELB_BF16)
        return fail(ELB_ERR_UNSUPPORTED, "packed expert weights are bf16 only");
    if (N < 1 || N > ELB_MAX_EXPERTS)
        return fail(ELB_ERR_INVALID_ARG, "N = %d outside [1, %d]", N, ELB_MAX_EXPERTS);
    if (d < 64 || m < 64 || d % 64 || m % 64)
        return fail(ELB_ERR_INVALID_ARG, "d = %d and m = %d must be positive multiples of 64",
                    d, m);
    if (!W_gate_up || !W_down || !packed) return fail(ELB_ERR_INVALID_ARG, "NULL tensor pointer");
    return hip_status(launch_pack_experts(W_gate_up, W_down, N, d, m, packed,
                                          (hipStream_t)stream),
                      "pack_experts");
}

int64_t elb_calibrate_mfma_bf16(int32_t blocks, int32_t iters, float* out, void* stream) {
    g_err.clear();
    if (blocks < 1 || iters < 1)
        return -fail(ELB_ERR_INVALID_ARG, "blocks = %d and iters = %d must be >= 1", blocks, iters);
    if (!out) return -fail(ELB_ERR_INVALID_ARG, "NULL tensor pointer");
    if (int rc = hip_status(launch_calibrate_mfma(blocks, iters, out, (hipStream_t)stream),
                            "calibrate_mfma"))
        return -rc;
    return (int64_t)blocks * 4 * iters * 8;
}

int elb_calibrate_read_stream(const void* buf, int64_t bytes, int32_t blocks, uint32_t* out,
                              void* stream) {
    g_err.clear();
    if (!buf || !out) return fail(ELB_ERR_INVALID_ARG, "NULL tensor pointer");
    if (bytes < 16 || bytes % 16 || (uintptr_t)buf % 16)
        return fail(ELB_ERR_INVALID_ARG, "buffer of %lld bytes: need a positive multiple of 16, "
                    "16-byte aligned", (long long)bytes);
    if (blocks < 1) return fail(ELB_ERR_INVALID_ARG, "blocks = %d must be >= 1", blocks);
    return hip_status(launch_calibrate_read(buf, bytes, blocks, out, (hipStream_t)stream),
                      "calibrate_read");
}

int elb_profile_enable(int on) {
    if (on < 0 || on > 2) return fail(ELB_ERR_INVALID_ARG, "profiling level %d outside [0, 2]", on);
    g_prof_on.store(on);
    return ELB_OK;
}

int elb_profile_read(const char** names, double* total_ms, int64_t* launches, int cap) {
    std::lock_guard<std::mutex> lk(g_prof_mu);
    std::map<std::string, std::pair<double, int64_t>> acc;
    std::map<std::string, int> last_scope;
    std::vector<const char*> order;  // names in first-seen order (static strings)
    int rc = ELB_OK;
    for (Rec& r : g_recs) {
        float ms = 0.f;
        if (hipEventSynchronize(r.b) != hipSuccess ||
            hipEventElapsedTime(&ms, r.a, r.b) != hipSuccess)
            rc = ELB_ERR_HIP;
        auto it = acc.find(r.name);
        if (it == acc.end()) {
            acc[r.name] = {ms, 1};
            last_scope[r.name] = r.scope;
            order.push_back(r.name);
        } else {
            it->second.first += ms;
            if (last_scope[r.name] != r.scope) {  // a new scope instance: one more launch
                it->second.second += 1;
                last_scope[r.name] = r.scope;
            }
        }
        g_pool.push_back(r.a);
        g_pool.push_back(r.b);
    }
    g_recs.clear();
    if (rc != ELB_OK) return -fail(rc, "profile events failed");
    int n = 0;
    for (const char* nm : order) {
        if (n < cap) {
            if (names) names[n] = nm;
            if (total_ms) total_ms[n] = acc[nm].first;
            if (launches) launches[n] = acc[nm].second;
        }
        ++n;
    }
    return n;
}

}  // extern "C"
