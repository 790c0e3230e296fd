"""Python binding of libelbow_moe (ctypes): argument marshalling only.

Every function has the name of the C entry point it calls (include/elbow_moe.h) and takes
torch tensors that live on the GPU; torch provides device memory and the current stream,
every step of the computation runs in the library's HIP kernels.  There is no fallback:
if the library is missing or a call fails, an exception is raised.
"""
from __future__ import annotations

import ctypes as C
import os
from typing import Optional

import torch

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libelbow_moe.so")

ELB_F32, ELB_BF16 = 0, 1
MODE_ELBOW, MODE_TOPK = 0, 1
MAX_EXPERTS, MAX_K = 64, 64

_lib = None


class ElbError(RuntimeError):
    def __init__(self, fn: str, status: int, msg: str):
        super().__init__("%s failed: %s (%s)" % (fn, _status_str(status), msg))
        self.status = status


class RouteParams(C.Structure):
    _fields_ = [("K", C.c_int32), ("eps", C.c_float), ("mode", C.c_int32),
                ("renormalize", C.c_int32)]


def lib():
    """Load libelbow_moe.so (built by paper_2608_04401_amd.build); raise if it is missing."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError("libelbow_moe.so is not built (%s); run "
                           "`python -m paper_2608_04401_amd.build`" % LIB_PATH)
    L = C.CDLL(LIB_PATH)
    P, I32, I64, SZ = C.c_void_p, C.c_int32, C.c_int64, C.c_size_t
    sig = {
        "elb_abi_version": ([], C.c_int),
        "elb_status_str": ([C.c_int], C.c_char_p),
        "elb_last_error": ([], C.c_char_p),
        "elb_router_logits": ([P, P, I64, I32, I32, I32, P, P], C.c_int),
        "elb_route": ([P, I64, I32, C.POINTER(RouteParams), P, P, P, P], C.c_int),
        "elb_router_route": ([P, P, I64, I32, I32, I32, C.POINTER(RouteParams), P, P, P, P, P],
                             C.c_int),
        "elb_route_tail_random": ([P, P, I64, I32, C.POINTER(RouteParams), P, P, P, P],
                                  C.c_int),
        "elb_elbow_angle": ([P, I64, I32, C.c_float, P, P, P], C.c_int),
        "elb_dispatch_workspace_bytes": ([I64, I32], SZ),
        "elb_dispatch": ([P, P, I64, I32, I32, P, P, P, P, P, SZ, P], C.c_int),
        "elb_moe_workspace_bytes": ([I64, I32, I32, I32, I32, I32], SZ),
        "elb_moe_experts": ([P, P, P, P, P, P, P, I64, I32, I32, I32, I32, I32, P, P, SZ, P],
                            C.c_int),
        "elb_moe_forward": ([P, P, P, P, P, I64, I32, I32, I32, I32, C.POINTER(RouteParams), P,
                             P, SZ, P, P, P, P, P, P], C.c_int),
        "elb_packed_expert_bytes": ([I32, I32, I32], SZ),
        "elb_pack_expert_weights": ([P, P, I32, I32, I32, I32, P, P], C.c_int),
        "elb_moe_experts_packed": ([P, P, P, P, P, P, P, P, I64, I32, I32, I32, I32, I32, P, P,
                                    SZ, P], C.c_int),
        "elb_moe_forward_packed": ([P, P, P, P, P, P, I64, I32, I32, I32, I32,
                                    C.POINTER(RouteParams), P, P, SZ, P, P, P, P, P, P],
                                   C.c_int),
        "elb_moe_forward_noalloc": ([P, P, P, P, P, I64, I32, I32, I32, I32,
                                     C.POINTER(RouteParams), P, P, P, P, P, P, P], C.c_int),
        "elb_calibrate_mfma_bf16": ([I32, I32, P, P], C.c_int64),
        "elb_calibrate_read_stream": ([P, I64, I32, P, P], C.c_int),
        "elb_profile_enable": ([C.c_int], C.c_int),
        "elb_profile_read": ([C.POINTER(C.c_char_p), C.POINTER(C.c_double),
                              C.POINTER(C.c_int64), C.c_int], C.c_int),
    }
    for name, (args, res) in sig.items():
        f = getattr(L, name)
        f.argtypes = args
        f.restype = res
    _lib = L
    return L


def _status_str(s: int) -> str:
    return lib().elb_status_str(s).decode()


def _check(fn: str, status: int):
    if status != 0:
        raise ElbError(fn, status, lib().elb_last_error().decode())


def _ptr(t: Optional[torch.Tensor]):
    return None if t is None else C.c_void_p(t.data_ptr())


def _stream():
    return C.c_void_p(torch.cuda.current_stream().cuda_stream)


def _dtype_code(t: torch.Tensor) -> int:
    if t.dtype == torch.float32:
        return ELB_F32
    if t.dtype == torch.bfloat16:
        return ELB_BF16
    raise TypeError("unsupported dtype %s (float32 or bfloat16)" % t.dtype)


def _dev(*ts):
    for t in ts:
        if t is None:
            continue
        if not t.is_cuda:
            raise ValueError("tensors must be on the GPU")
        if not t.is_contiguous():
            raise ValueError("tensors must be contiguous")


_ws_cache: dict = {}


def workspace(nbytes: int, device) -> torch.Tensor:
    """A cached uint8 device buffer of at least nbytes (one per device)."""
    key = torch.device(device).index
    buf = _ws_cache.get(key)
    if buf is None or buf.numel() < nbytes:
        buf = torch.empty(max(int(nbytes), 1), dtype=torch.uint8, device=device)
        _ws_cache[key] = buf
    return buf


def elb_abi_version() -> int:
    return lib().elb_abi_version()


def elb_router_logits(x: torch.Tensor, W_router: torch.Tensor) -> torch.Tensor:
    _dev(x, W_router)
    T, d = x.shape
    N = W_router.shape[0]
    logits = torch.empty((T, N), dtype=torch.float32, device=x.device)
    _check("elb_router_logits", lib().elb_router_logits(
        _ptr(x), _ptr(W_router), T, d, N, _dtype_code(x), _ptr(logits), _stream()))
    return logits


def elb_route(logits: torch.Tensor, K: int, eps: float = 1e-8, mode: int = MODE_ELBOW,
              renormalize: bool = False):
    """-> (k [T] int32, ids [T, K] int32, w [T, K] float32)"""
    _dev(logits)
    if logits.dtype != torch.float32:
        raise TypeError("logits must be float32")
    T, N = logits.shape
    k = torch.empty(T, dtype=torch.int32, device=logits.device)
    ids = torch.empty((T, K), dtype=torch.int32, device=logits.device)
    w = torch.empty((T, K), dtype=torch.float32, device=logits.device)
    p = RouteParams(K, eps, mode, int(renormalize))
    _check("elb_route", lib().elb_route(_ptr(logits), T, N, C.byref(p), _ptr(k), _ptr(ids),
                                        _ptr(w), _stream()))
    return k, ids, w


def elb_router_route(x: torch.Tensor, W_router: torch.Tensor, K: int, eps: float = 1e-8,
                     mode: int = MODE_ELBOW, renormalize: bool = False,
                     with_logits: bool = False):
    """-> (k [T], ids [T, K], w [T, K], logits [T, N] or None)"""
    _dev(x, W_router)
    T, d = x.shape
    N = W_router.shape[0]
    dev = x.device
    k = torch.empty(T, dtype=torch.int32, device=dev)
    ids = torch.empty((T, K), dtype=torch.int32, device=dev)
    w = torch.empty((T, K), dtype=torch.float32, device=dev)
    logits = torch.empty((T, N), dtype=torch.float32, device=dev) if with_logits else None
    p = RouteParams(K, eps, mode, int(renormalize))
    _check("elb_router_route", lib().elb_router_route(
        _ptr(x), _ptr(W_router), T, d, N, _dtype_code(x), C.byref(p), _ptr(logits), _ptr(k),
        _ptr(ids), _ptr(w), _stream()))
    return k, ids, w, logits


def elb_route_tail_random(logits: torch.Tensor, rand: torch.Tensor, K: int, eps: float = 1e-8,
                          mode: int = MODE_ELBOW, renormalize: bool = False):
    """-> (k_elbow [T] int32, ids [T, K] int32, w [T, K] float32); rand [T, N] float32"""
    _dev(logits, rand)
    if logits.dtype != torch.float32 or rand.dtype != torch.float32:
        raise TypeError("logits and rand must be float32")
    if rand.shape != logits.shape:
        raise ValueError("rand must have the shape of logits")
    T, N = logits.shape
    k = torch.empty(T, dtype=torch.int32, device=logits.device)
    ids = torch.empty((T, K), dtype=torch.int32, device=logits.device)
    w = torch.empty((T, K), dtype=torch.float32, device=logits.device)
    p = RouteParams(K, eps, mode, int(renormalize))
    _check("elb_route_tail_random", lib().elb_route_tail_random(
        _ptr(logits), _ptr(rand), T, N, C.byref(p), _ptr(k), _ptr(ids), _ptr(w), _stream()))
    return k, ids, w


def elb_elbow_angle(logits: torch.Tensor, eps: float = 1e-8):
    """-> (e [T] int32, theta [T] float32 degrees)"""
    _dev(logits)
    if logits.dtype != torch.float32:
        raise TypeError("logits must be float32")
    T, N = logits.shape
    e = torch.empty(T, dtype=torch.int32, device=logits.device)
    theta = torch.empty(T, dtype=torch.float32, device=logits.device)
    _check("elb_elbow_angle", lib().elb_elbow_angle(_ptr(logits), T, N, eps, _ptr(e),
                                                    _ptr(theta), _stream()))
    return e, theta


def elb_dispatch(k: torch.Tensor, ids: torch.Tensor, N: int):
    """-> (counts [N], offsets [N+1], row_token [T*K], inv [T, K]) int32"""
    _dev(k, ids)
    T, K = ids.shape
    dev = ids.device
    counts = torch.empty(N, dtype=torch.int32, device=dev)
    offsets = torch.empty(N + 1, dtype=torch.int32, device=dev)
    row_token = torch.full((T * K,), -1, dtype=torch.int32, device=dev)
    inv = torch.empty((T, K), dtype=torch.int32, device=dev)
    nb = lib().elb_dispatch_workspace_bytes(T, N)
    ws = workspace(nb, dev)
    _check("elb_dispatch", lib().elb_dispatch(_ptr(k), _ptr(ids), T, N, K, _ptr(counts),
                                              _ptr(offsets), _ptr(row_token), _ptr(inv),
                                              _ptr(ws), ws.numel(), _stream()))
    return counts, offsets, row_token, inv


def elb_moe_workspace_bytes(T: int, d: int, N: int, m: int, K: int, dtype: int) -> int:
    return int(lib().elb_moe_workspace_bytes(T, d, N, m, K, dtype))


def elb_pack_expert_weights(W_gate_up: torch.Tensor, W_down: torch.Tensor) -> torch.Tensor:
    """The packed copy of bf16 expert weights for the decode-sized path (uint8 tensor)."""
    _dev(W_gate_up, W_down)
    N, m2, d = W_gate_up.shape
    m = m2 // 2
    packed = torch.empty(int(lib().elb_packed_expert_bytes(N, d, m)), dtype=torch.uint8,
                         device=W_gate_up.device)
    _check("elb_pack_expert_weights", lib().elb_pack_expert_weights(
        _ptr(W_gate_up), _ptr(W_down), N, d, m, _dtype_code(W_gate_up), _ptr(packed),
        _stream()))
    return packed


def elb_moe_experts(x, W_gate_up, W_down, k, ids, w, residual=None, out=None,
                    packed=None) -> torch.Tensor:
    """packed: optional packed weights (elb_pack_expert_weights) for the decode-sized path."""
    _dev(x, W_gate_up, W_down, k, ids, w, residual, out, packed)
    T, d = x.shape
    N, m2, _ = W_gate_up.shape
    m = m2 // 2
    K = ids.shape[1]
    dt = _dtype_code(x)
    y = torch.empty_like(x) if out is None else out
    nb = elb_moe_workspace_bytes(T, d, N, m, K, dt)
    ws = workspace(nb, x.device)
    if packed is None:
        _check("elb_moe_experts", lib().elb_moe_experts(
            _ptr(x), _ptr(W_gate_up), _ptr(W_down), _ptr(k), _ptr(ids), _ptr(w),
            _ptr(residual), T, d, N, m, K, dt, _ptr(y), _ptr(ws), ws.numel(), _stream()))
    else:
        _check("elb_moe_experts_packed", lib().elb_moe_experts_packed(
            _ptr(x), _ptr(W_gate_up), _ptr(W_down), _ptr(packed), _ptr(k), _ptr(ids), _ptr(w),
            _ptr(residual), T, d, N, m, K, dt, _ptr(y), _ptr(ws), ws.numel(), _stream()))
    return y


def elb_moe_forward(x, W_router, W_gate_up, W_down, K: int = 8, eps: float = 1e-8,
                    mode: int = MODE_ELBOW, renormalize: bool = False, residual=None,
                    out=None, debug: bool = False, packed=None):
    """The whole layer.  Returns y, or (y, dict of intermediates) when debug=True.
    packed: optional packed weights (elb_pack_expert_weights) for the decode-sized path."""
    _dev(x, W_router, W_gate_up, W_down, residual, out, packed)
    T, d = x.shape
    N = W_router.shape[0]
    m = W_down.shape[2]
    dt = _dtype_code(x)
    dev = x.device
    y = torch.empty_like(x) if out is None else out
    nb = elb_moe_workspace_bytes(T, d, N, m, K, dt)
    ws = workspace(nb, dev)
    dbg = {}
    if debug:
        dbg = {"logits": torch.empty((T, N), dtype=torch.float32, device=dev),
               "k": torch.empty(T, dtype=torch.int32, device=dev),
               "ids": torch.empty((T, K), dtype=torch.int32, device=dev),
               "w": torch.empty((T, K), dtype=torch.float32, device=dev),
               "counts": torch.empty(N, dtype=torch.int32, device=dev)}
    p = RouteParams(K, eps, mode, int(renormalize))
    tail = (_ptr(dbg.get("logits")), _ptr(dbg.get("k")), _ptr(dbg.get("ids")),
            _ptr(dbg.get("w")), _ptr(dbg.get("counts")), _stream())
    if packed is None:
        _check("elb_moe_forward", lib().elb_moe_forward(
            _ptr(x), _ptr(W_router), _ptr(W_gate_up), _ptr(W_down), _ptr(residual), T, d, N, m,
            dt, C.byref(p), _ptr(y), _ptr(ws), ws.numel(), *tail))
    else:
        _check("elb_moe_forward_packed", lib().elb_moe_forward_packed(
            _ptr(x), _ptr(W_router), _ptr(W_gate_up), _ptr(W_down), _ptr(packed),
            _ptr(residual), T, d, N, m, dt, C.byref(p), _ptr(y), _ptr(ws), ws.numel(), *tail))
    return (y, dbg) if debug else y


NOALLOC_SCRATCH_BYTES = 256 << 20


def elb_moe_forward_noalloc(x, W_router, W_gate_up, W_down, K: int = 8, eps: float = 1e-8,
                            mode: int = MODE_ELBOW, renormalize: bool = False, residual=None,
                            out=None, debug: bool = False):
    """The whole layer through the allocation-free entry point (the library's static scratch,
    no workspace).  Returns y, or (y, dict of intermediates) when debug=True."""
    _dev(x, W_router, W_gate_up, W_down, residual, out)
    T, d = x.shape
    N = W_router.shape[0]
    m = W_down.shape[2]
    dev = x.device
    y = torch.empty_like(x) if out is None else out
    dbg = {}
    if debug:
        dbg = {"logits": torch.empty((T, N), dtype=torch.float32, device=dev),
               "k": torch.empty(T, dtype=torch.int32, device=dev),
               "ids": torch.empty((T, K), dtype=torch.int32, device=dev),
               "w": torch.empty((T, K), dtype=torch.float32, device=dev),
               "counts": torch.empty(N, dtype=torch.int32, device=dev)}
    p = RouteParams(K, eps, mode, int(renormalize))
    _check("elb_moe_forward_noalloc", lib().elb_moe_forward_noalloc(
        _ptr(x), _ptr(W_router), _ptr(W_gate_up), _ptr(W_down), _ptr(residual), T, d, N, m,
        _dtype_code(x), C.byref(p), _ptr(y), _ptr(dbg.get("logits")), _ptr(dbg.get("k")),
        _ptr(dbg.get("ids")), _ptr(dbg.get("w")), _ptr(dbg.get("counts")), _stream()))
    return (y, dbg) if debug else y


def elb_moe_forward_prepared(x, W_router, W_gate_up, W_down, K: int = 8, eps: float = 1e-8,
                             mode: int = MODE_ELBOW, renormalize: bool = False, residual=None,
                             out=None, packed=None):
    """elb_moe_forward with its arguments marshalled once: returns (call, y), where call() enqueues
    the layer on the stream that was current here and raises on a failed status.  For timing
    loops, where the per-call argument checks would otherwise add host time."""
    _dev(x, W_router, W_gate_up, W_down, residual, out, packed)
    T, d = x.shape
    N = W_router.shape[0]
    m = W_down.shape[2]
    dt = _dtype_code(x)
    y = torch.empty_like(x) if out is None else out
    ws = workspace(elb_moe_workspace_bytes(T, d, N, m, K, dt), x.device)
    p = RouteParams(K, eps, mode, int(renormalize))
    L = lib()
    if packed is None:
        fn, name = L.elb_moe_forward, "elb_moe_forward"
        args = (_ptr(x), _ptr(W_router), _ptr(W_gate_up), _ptr(W_down), _ptr(residual), T, d, N,
                m, dt, C.byref(p), _ptr(y), _ptr(ws), ws.numel(), None, None, None, None, None,
                _stream())
    else:
        fn, name = L.elb_moe_forward_packed, "elb_moe_forward_packed"
        args = (_ptr(x), _ptr(W_router), _ptr(W_gate_up), _ptr(W_down), _ptr(packed),
                _ptr(residual), T, d, N, m, dt, C.byref(p), _ptr(y), _ptr(ws), ws.numel(), None,
                None, None, None, None, _stream())
    keep = (p, ws, y)  # referenced by the closure: the parameter block and buffers stay alive

    def call():
        rc = fn(*args)
        if rc != 0:
            _check(name, rc)
        return keep
    return call, y


def elb_calibrate_read_stream(buf: torch.Tensor, blocks: int, out: torch.Tensor) -> None:
    """Enqueue the read-only stream over the bytes of buf (out: blocks * 4 int32 words)."""
    _dev(buf, out)
    _check("elb_calibrate_read_stream", lib().elb_calibrate_read_stream(
        _ptr(buf), buf.numel() * buf.element_size(), blocks, _ptr(out), _stream()))


def elb_calibrate_mfma_bf16(blocks: int, iters: int) -> int:
    """Enqueue the back-to-back MFMA calibration kernel; returns the MFMA instruction count
    (each v_mfma_f32_32x32x16_bf16 is 32 * 32 * 16 * 2 FLOPs)."""
    out = torch.empty(blocks * 4, dtype=torch.float32, device="cuda")
    n = lib().elb_calibrate_mfma_bf16(blocks, iters, _ptr(out), _stream())
    if n < 0:
        _check("elb_calibrate_mfma_bf16", -n)
    return int(n)


def elb_profile_enable(on=True) -> None:
    """on: False/0 off, True/1 every launch, 2 the grouped expert GEMMs only."""
    _check("elb_profile_enable", lib().elb_profile_enable(int(on)))


def elb_profile_read() -> dict:
    """{kernel name: (total ms, launches)} since the last read; clears the records."""
    cap = 64
    names = (C.c_char_p * cap)()
    ms = (C.c_double * cap)()
    n_l = (C.c_int64 * cap)()
    n = lib().elb_profile_read(names, ms, n_l, cap)
    if n < 0:
        _check("elb_profile_read", -n)
    return {names[i].decode(): (ms[i], int(n_l[i])) for i in range(min(n, cap))}
