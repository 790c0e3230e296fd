"""The C-ABI library: it loads, exports every entry point declared in include/elbow_moe.h,
and rejects invalid arguments on the host before anything is launched (no GPU needed:
validation runs before any HIP call, and the dummy pointers below are never dereferenced).
"""
import ctypes as C
import os
import re

import pytest

from paper_2608_04401_amd import binding as B

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "elbow_moe.h")

OK, INVALID, UNSUPPORTED, WORKSPACE = 0, 1, 2, 3
DUMMY = C.c_void_p(0x1000)   # never dereferenced: every call below fails validation
DUMMY_MISALIGNED = C.c_void_p(0x1010)


def declared_functions():
    txt = open(HEADER).read()
    txt = re.sub(r"/\*.*?\*/", "", txt, flags=re.S)
    return sorted(set(re.findall(r"\b(elb_[a-z_]+)\s*\(", txt)))


def test_library_exports_every_declared_symbol():
    lib = B.lib()
    names = declared_functions()
    assert len(names) >= 12
    for n in names:
        assert hasattr(lib, n), n
    assert B.elb_abi_version() == 1


def test_status_strings():
    lib = B.lib()
    assert lib.elb_status_str(0) == b"ELB_OK"
    assert lib.elb_status_str(3) == b"ELB_ERR_WORKSPACE"
    assert lib.elb_status_str(99) == b"ELB_ERR_UNKNOWN"


def _route(T, N, K=8, eps=1e-8, mode=0, renorm=0, ptr=DUMMY, params=True):
    p = B.RouteParams(K, eps, mode, renorm)
    return B.lib().elb_route(ptr, T, N, C.byref(p) if params else None, ptr, ptr, ptr, None)


@pytest.mark.parametrize("T,N,K,eps,mode,renorm,want", [
    (-1, 64, 8, 1e-8, 0, 0, INVALID),        # negative T
    (10, 1, 1, 1e-8, 0, 0, INVALID),         # N < 2
    (10, 65, 8, 1e-8, 0, 0, UNSUPPORTED),    # N beyond the kernels
    (10, 64, 0, 1e-8, 0, 0, INVALID),        # K < 1
    (10, 8, 9, 1e-8, 0, 0, INVALID),         # K > N
    (10, 64, 65, 1e-8, 0, 0, INVALID),       # K > N at the largest N
    (10, 64, 8, -1.0, 0, 0, INVALID),        # eps < 0
    (10, 64, 8, float("nan"), 0, 0, INVALID),
    (10, 64, 8, 1e-8, 2, 0, INVALID),        # bad mode
    (10, 64, 8, 1e-8, 0, 2, INVALID),        # bad renormalize flag
])
def test_route_validation(T, N, K, eps, mode, renorm, want):
    assert _route(T, N, K, eps, mode, renorm) == want
    assert B.lib().elb_last_error() != b""


def test_route_null_and_empty():
    assert _route(10, 64, params=False) == INVALID
    assert _route(10, 64, ptr=None) == INVALID
    assert _route(0, 64, ptr=None) == OK          # T = 0: nothing to do, nothing launched


def test_experts_validation():
    lib = B.lib()
    f = lib.elb_moe_experts

    def call(T=16, d=128, N=8, m=128, K=4, dt=1, ws=DUMMY, wsb=1 << 40, y=DUMMY):
        return f(DUMMY, DUMMY, DUMMY, DUMMY, DUMMY, DUMMY, None, T, d, N, m, K, dt, y, ws, wsb,
                 None)
    assert call(d=96) == INVALID                  # bf16 needs d % 64 == 0
    assert call(m=100, dt=0) == INVALID           # f32 needs m % 16 == 0
    assert call(dt=7) == INVALID
    assert call(N=80) == UNSUPPORTED
    assert call(K=9) == INVALID
    assert call(ws=None) == WORKSPACE
    assert call(wsb=16) == WORKSPACE
    assert call(ws=DUMMY_MISALIGNED) == WORKSPACE       # not 256-byte aligned
    assert call(y=None) == INVALID
    assert call(T=0, ws=None, y=None) == OK


def test_workspace_sizes():
    lib = B.lib()
    small = lib.elb_moe_workspace_bytes(256, 128, 8, 256, 8, 0)
    big = lib.elb_moe_workspace_bytes(4096, 2048, 64, 1024, 8, 1)
    assert 0 < small < big
    # H and Y dominate: T K (m + d) bf16 elements
    assert big >= 4096 * 8 * (1024 + 2048) * 2
    assert lib.elb_moe_workspace_bytes(-1, 128, 8, 256, 8, 0) == 0
    assert lib.elb_dispatch_workspace_bytes(65536, 64) >= 1024 * 64 * 4


def test_dispatch_and_router_validation():
    lib = B.lib()
    assert lib.elb_dispatch(DUMMY, DUMMY, 100, 64, 8, DUMMY, DUMMY, DUMMY, DUMMY, DUMMY, 4,
                            None) == WORKSPACE
    assert lib.elb_dispatch(DUMMY, DUMMY, 100, 64, 65, DUMMY, DUMMY, DUMMY, DUMMY, DUMMY,
                            1 << 30, None) == INVALID
    assert lib.elb_dispatch(DUMMY, DUMMY, 100, 64, 8, DUMMY, DUMMY, DUMMY, DUMMY,
                            DUMMY_MISALIGNED, 1 << 30, None) == WORKSPACE  # not 256-byte aligned
    assert lib.elb_router_logits(DUMMY, DUMMY, 100, 100, 64, 1, DUMMY, None) == INVALID
    assert lib.elb_router_logits(DUMMY, DUMMY, 100, 128, 100, 1, DUMMY, None) == UNSUPPORTED


def test_profile_read_empty():
    assert B.elb_profile_read() == {}


def test_router_route_validation():
    lib = B.lib()
    p = B.RouteParams(8, 1e-8, 0, 0)
    call = lambda dt=1, d=128, p=p, T=10: lib.elb_router_route(
        DUMMY, DUMMY, T, d, 64, dt, C.byref(p), None, DUMMY, DUMMY, DUMMY, None)
    assert call(dt=0) == UNSUPPORTED                       # fp32: use the two calls
    assert call(p=B.RouteParams(17, 1e-8, 0, 0)) == UNSUPPORTED   # K above the lane kernel
    assert call(d=100) == INVALID                          # bf16 router needs d % 32 == 0
    assert call(p=B.RouteParams(8, -1.0, 0, 0)) == INVALID
    assert call(T=0) == OK


def test_variant_entry_points_validation():
    lib = B.lib()
    p = B.RouteParams(8, 1e-8, 0, 0)
    tr = lambda T=10, N=64, p=p, rand=DUMMY, ptr=DUMMY: lib.elb_route_tail_random(
        ptr, rand, T, N, C.byref(p) if p is not None else None, ptr, ptr, ptr, None)
    assert tr(T=-1) == INVALID
    assert tr(N=65) == UNSUPPORTED
    assert tr(p=B.RouteParams(65, 1e-8, 0, 0)) == INVALID      # K > N
    assert tr(p=None) == INVALID
    assert tr(rand=None) == INVALID                             # the draws are required
    assert tr(T=0, rand=None, ptr=None) == OK
    ang = lambda T=10, N=64, eps=1e-8, lg=DUMMY, e=DUMMY, th=DUMMY: lib.elb_elbow_angle(
        lg, T, N, eps, e, th, None)
    assert ang(N=1) == INVALID
    assert ang(N=65) == UNSUPPORTED
    assert ang(eps=-1.0) == INVALID
    assert ang(eps=float("inf")) == INVALID
    assert ang(lg=None) == INVALID
    assert ang(e=None, th=None) == OK                           # nothing asked for
    assert ang(T=0, lg=None) == OK
    # caps up to N are valid for the plain routing now (K = N: the uncapped elbow)
    assert _route(10, 64, K=64, ptr=None) == INVALID            # only the NULL pointers fail


def test_noalloc_rejects_oversized_problems_on_the_host():
    """The allocation-free entry point checks the layer's scratch need against its static
    array before any HIP call: the OLMoE-shaped layer at T = 8192 needs more than 256 MiB."""
    lib = B.lib()
    p = B.RouteParams(8, 1e-8, 0, 0)
    need = lib.elb_moe_workspace_bytes(8192, 2048, 64, 1024, 8, B.ELB_BF16)
    assert need > B.NOALLOC_SCRATCH_BYTES
    assert lib.elb_moe_workspace_bytes(4096, 2048, 64, 1024, 8, B.ELB_BF16) <= \
        B.NOALLOC_SCRATCH_BYTES
    rc = lib.elb_moe_forward_noalloc(DUMMY, DUMMY, DUMMY, DUMMY, None, 8192, 2048, 64, 1024,
                                     B.ELB_BF16, C.byref(p), DUMMY, None, None, None, None,
                                     None, None)
    assert rc == UNSUPPORTED
    assert b"scratch" in lib.elb_last_error()
    # the other argument checks come first, as in elb_moe_forward
    bad = B.RouteParams(0, 1e-8, 0, 0)
    assert lib.elb_moe_forward_noalloc(DUMMY, DUMMY, DUMMY, DUMMY, None, 64, 2048, 64, 1024,
                                       B.ELB_BF16, C.byref(bad), DUMMY, None, None, None,
                                       None, None, None) == INVALID
    assert lib.elb_moe_forward_noalloc(DUMMY, None, DUMMY, DUMMY, None, 64, 2048, 64, 1024,
                                       B.ELB_BF16, C.byref(p), DUMMY, None, None, None, None,
                                       None, None) == INVALID
    assert lib.elb_moe_forward_noalloc(None, None, None, None, None, 0, 2048, 64, 1024,
                                       B.ELB_BF16, C.byref(p), None, None, None, None, None,
                                       None, None) == OK


def test_read_stream_calibration_validates_on_the_host():
    """The read-stream calibration rejects a NULL buffer, sizes that are not a positive
    multiple of 16, a misaligned buffer and blocks < 1 before launching anything."""
    lib = B.lib()
    assert lib.elb_calibrate_read_stream(None, 1024, 4, DUMMY, None) == INVALID
    assert lib.elb_calibrate_read_stream(DUMMY, 1024, 4, None, None) == INVALID
    assert lib.elb_calibrate_read_stream(DUMMY, 0, 4, DUMMY, None) == INVALID
    assert lib.elb_calibrate_read_stream(DUMMY, 1000, 4, DUMMY, None) == INVALID
    assert lib.elb_calibrate_read_stream(C.c_void_p(DUMMY.value + 8), 1024, 4, DUMMY,
                                         None) == INVALID
    assert lib.elb_calibrate_read_stream(DUMMY, 1024, 0, DUMMY, None) == INVALID
