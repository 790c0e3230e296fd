"""ctypes wrapper of the fp64 CPU oracle (oracle.c).

TEST INFRASTRUCTURE ONLY: imported by the tests, the smoke check and the benchmark's
CPU-baseline leg, never by the GPU library or its binding.  Inputs are numpy arrays
(float32 for logits, activations and weights; bf16 values arrive as exactly-equal float32),
outputs are float64 / int32 numpy arrays.
"""
from __future__ import annotations

import ctypes as C
import os
import subprocess

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "oracle.c")
LIB = os.path.join(HERE, "liboracle.so")

MODE_ELBOW = 0
MODE_TOPK = 1
DEFAULT_EPS = 1e-8


def compile_source(src: str, out: str) -> str:
    """gcc -O2 -fopenmp (no fast-math) of one C file into a shared library."""
    tmp = out + ".tmp%d" % os.getpid()
    subprocess.check_call(["gcc", "-O2", "-fopenmp", "-std=c11", "-Wall", "-shared", "-fPIC",
                           src, "-o", tmp, "-lm"])
    os.replace(tmp, out)
    return out


def build(force: bool = False) -> str:
    """Compile oracle.c into liboracle.so (when missing or older than the source)."""
    if force or not os.path.exists(LIB) or os.path.getmtime(LIB) < os.path.getmtime(SRC):
        compile_source(SRC, LIB)
    return LIB


def _ptr(a):
    return None if a is None else a.ctypes.data_as(C.c_void_p)


def _f32(a):
    return np.ascontiguousarray(a, dtype=np.float32)


class Routing:
    """Per-token routing result: k [T], ids [T, K] (-1 pad), w [T, K] (0 pad),
    e [T] (0-based argmax, -1 in top-K mode), margin [T], competitor [T]."""

    def __init__(self, k, ids, w, e, margin, competitor):
        self.k, self.ids, self.w, self.e = k, ids, w, e
        self.margin, self.competitor = margin, competitor


class LayerResult:
    def __init__(self, y, logits, routing):
        self.y, self.logits, self.routing = y, logits, routing


class OracleLib:
    """The oracle's functions, bound to one compiled copy of oracle.c."""

    def __init__(self, path: str):
        lib = C.CDLL(path)
        P = C.c_void_p
        lib.orc_route.argtypes = [P, C.c_long, C.c_int, C.c_int, C.c_double, C.c_int, C.c_int,
                                  P, P, P, P, P, P]
        lib.orc_route_from_probs.argtypes = lib.orc_route.argtypes
        lib.orc_router_logits.argtypes = [P, P, C.c_long, C.c_int, C.c_int, P]
        lib.orc_router_logits.restype = None
        lib.orc_moe_experts.argtypes = [P, P, P, P, C.c_long, C.c_int, C.c_int, C.c_int,
                                        C.c_int, P, C.c_long, P, P, P, P]
        lib.orc_moe_forward.argtypes = [P, P, P, P, P, C.c_long, C.c_int, C.c_int, C.c_int,
                                        C.c_int, C.c_double, C.c_int, C.c_int, P, C.c_long,
                                        P, P, P, P, P, P]
        lib.orc_dispatch.argtypes = [P, P, C.c_long, C.c_int, C.c_int, P, P, P, P]
        lib.orc_elbow_angle.argtypes = [P, C.c_long, C.c_int, C.c_double, P, P]
        lib.orc_elbow_angle_from_probs.argtypes = lib.orc_elbow_angle.argtypes
        lib.orc_route_tail_random.argtypes = [P, P, C.c_long, C.c_int, C.c_int, C.c_double,
                                              C.c_int, P, P, P]
        self.lib = lib
        self.path = path

    def dispatch(self, k, ids, N: int):
        """Expert-major lists of a routing -> (counts [N], offsets [N+1], row_token [sum k],
        inv [T, K]) as int32."""
        kk = np.ascontiguousarray(k, np.int32)
        ii = np.ascontiguousarray(ids, np.int32)
        T, K = ii.shape
        counts = np.empty(N, np.int32)
        offsets = np.empty(N + 1, np.int32)
        row_token = np.empty(int(np.minimum(kk, K).clip(0).sum()), np.int32)
        inv = np.empty((T, K), np.int32)
        rc = self.lib.orc_dispatch(_ptr(kk), _ptr(ii), T, N, K, _ptr(counts), _ptr(offsets),
                                   _ptr(row_token), _ptr(inv))
        if rc != 0:
            raise ValueError("oracle dispatch: expert id out of range")
        return counts, offsets, row_token, inv

    def _route(self, fn, arr, N, K, eps, mode, renorm):
        T = arr.shape[0]
        k = np.empty(T, np.int32)
        ids = np.empty((T, K), np.int32)
        w = np.empty((T, K), np.float64)
        e = np.empty(T, np.int32)
        margin = np.empty(T, np.float64)
        comp = np.empty(T, np.int32)
        rc = fn(_ptr(arr), T, N, K, eps, mode, int(renorm), _ptr(k), _ptr(ids), _ptr(w),
                _ptr(e), _ptr(margin), _ptr(comp))
        if rc != 0:
            raise ValueError("oracle routing failed with code %d" % rc)
        return Routing(k, ids, w, e, margin, comp)

    def route(self, logits, K: int, eps: float = DEFAULT_EPS, mode: int = MODE_ELBOW,
              renorm: bool = False) -> Routing:
        """Route fp32 logits [T, N]: softmax, descending sort, elbow, cap at K."""
        lg = _f32(logits)
        return self._route(self.lib.orc_route, lg, lg.shape[1], K, eps, mode, renorm)

    def route_from_probs(self, p, K: int, eps: float = DEFAULT_EPS, mode: int = MODE_ELBOW,
                         renorm: bool = False) -> Routing:
        """The selection rule on given probability vectors [T, N] (float64, no softmax)."""
        pp = np.ascontiguousarray(p, dtype=np.float64)
        if pp.ndim == 1:
            pp = pp[None, :]
        return self._route(self.lib.orc_route_from_probs, pp, pp.shape[1], K, eps, mode,
                           renorm)

    def elbow_angle(self, logits, eps: float = DEFAULT_EPS):
        """Uncapped elbow index e [T] (int32) and elbow angle theta [T] (degrees, float64)
        of fp32 logits [T, N] (Section 2.3)."""
        lg = _f32(logits)
        return self._angle(self.lib.orc_elbow_angle, lg, eps)

    def elbow_angle_from_probs(self, p, eps: float = DEFAULT_EPS):
        """The same on given probability vectors [T, N] (float64)."""
        pp = np.ascontiguousarray(p, dtype=np.float64)
        if pp.ndim == 1:
            pp = pp[None, :]
        return self._angle(self.lib.orc_elbow_angle_from_probs, pp, eps)

    def _angle(self, fn, arr, eps):
        T, N = arr.shape
        e = np.empty(T, np.int32)
        th = np.empty(T, np.float64)
        rc = fn(_ptr(arr), T, N, eps, _ptr(e), _ptr(th))
        if rc != 0:
            raise ValueError("oracle elbow angle failed with code %d" % rc)
        return e, th

    def route_tail_random(self, logits, rand, K: int, eps: float = DEFAULT_EPS,
                          renorm: bool = False):
        """Tail randomisation: the elbow's k experts, then K - k experts outside them drawn
        by the smallest rand [T, N] values.  -> (k_elbow [T], ids [T, K], w [T, K])."""
        lg = _f32(logits)
        rd = _f32(rand)
        T, N = lg.shape
        if rd.shape != lg.shape:
            raise ValueError("rand must have the logits' shape")
        k = np.empty(T, np.int32)
        ids = np.empty((T, K), np.int32)
        w = np.empty((T, K), np.float64)
        rc = self.lib.orc_route_tail_random(_ptr(lg), _ptr(rd), T, N, K, eps, int(renorm),
                                            _ptr(k), _ptr(ids), _ptr(w))
        if rc != 0:
            raise ValueError("oracle tail randomisation failed with code %d" % rc)
        return k, ids, w

    def router_logits(self, x, W_router) -> np.ndarray:
        """fp64 logits [T, N] = x W_r^T."""
        x, Wr = _f32(x), _f32(W_router)
        T, d = x.shape
        N = Wr.shape[0]
        out = np.empty((T, N), np.float64)
        self.lib.orc_router_logits(_ptr(x), _ptr(Wr), T, d, N, _ptr(out))
        return out

    def moe_experts(self, x, W_gu, W_down, k, ids, w, tokens=None, residual=None):
        """Expert part of the layer for `tokens` (default: all) given their routing
        (k/ids/w rows aligned with `tokens`).  Returns fp64 y [len(tokens), d]."""
        x, Wgu, Wd = _f32(x), _f32(W_gu), _f32(W_down)
        T, d = x.shape
        N, m2, _ = Wgu.shape
        m = m2 // 2
        tok = (np.arange(T, dtype=np.int64) if tokens is None
               else np.ascontiguousarray(tokens, np.int64))
        K = ids.shape[1]
        kk = np.ascontiguousarray(k, np.int32)
        ii = np.ascontiguousarray(ids, np.int32)
        ww = np.ascontiguousarray(w, np.float64)
        res = None if residual is None else _f32(residual)
        y = np.empty((len(tok), d), np.float64)
        rc = self.lib.orc_moe_experts(_ptr(x), _ptr(Wgu), _ptr(Wd), _ptr(res), T, d, N, m, K,
                                      _ptr(tok), len(tok), _ptr(kk), _ptr(ii), _ptr(ww), _ptr(y))
        if rc != 0:
            raise ValueError("oracle expert pass failed with code %d" % rc)
        return y

    def moe_forward(self, x, W_router, W_gu, W_down, K: int, eps: float = DEFAULT_EPS,
                    mode: int = MODE_ELBOW, renorm: bool = False, tokens=None,
                    residual=None) -> LayerResult:
        """Whole layer (fp64 router, routing on the fp64 logits, experts) for `tokens`."""
        x, Wr, Wgu, Wd = _f32(x), _f32(W_router), _f32(W_gu), _f32(W_down)
        T, d = x.shape
        N = Wr.shape[0]
        m = Wd.shape[2]
        tok = (np.arange(T, dtype=np.int64) if tokens is None
               else np.ascontiguousarray(tokens, np.int64))
        n = len(tok)
        y = np.empty((n, d), np.float64)
        lg = np.empty((n, N), np.float64)
        k = np.empty(n, np.int32)
        ids = np.empty((n, K), np.int32)
        w = np.empty((n, K), np.float64)
        margin = np.empty(n, np.float64)
        res = None if residual is None else _f32(residual)
        rc = self.lib.orc_moe_forward(_ptr(x), _ptr(Wr), _ptr(Wgu), _ptr(Wd), _ptr(res), T, d,
                                      N, m, K, eps, mode, int(renorm), _ptr(tok), n, _ptr(y),
                                      _ptr(lg), _ptr(k), _ptr(ids), _ptr(w), _ptr(margin))
        if rc != 0:
            raise ValueError("oracle layer failed with code %d" % rc)
        return LayerResult(y, lg, Routing(k, ids, w, None, margin, None))


_default = None


def _lib() -> OracleLib:
    global _default
    if _default is None:
        _default = OracleLib(build())
    return _default


def route(*a, **kw) -> Routing:
    return _lib().route(*a, **kw)


def route_from_probs(*a, **kw) -> Routing:
    return _lib().route_from_probs(*a, **kw)


def router_logits(*a, **kw) -> np.ndarray:
    return _lib().router_logits(*a, **kw)


def moe_experts(*a, **kw) -> np.ndarray:
    return _lib().moe_experts(*a, **kw)


def dispatch(*a, **kw):
    return _lib().dispatch(*a, **kw)


def moe_forward(*a, **kw) -> LayerResult:
    return _lib().moe_forward(*a, **kw)


def elbow_angle(*a, **kw):
    return _lib().elbow_angle(*a, **kw)


def elbow_angle_from_probs(*a, **kw):
    return _lib().elbow_angle_from_probs(*a, **kw)


def route_tail_random(*a, **kw):
    return _lib().route_tail_random(*a, **kw)
