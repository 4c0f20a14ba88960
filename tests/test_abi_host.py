"""C ABI checks that need no GPU: the library loads, exports every entry point
the header declares, and rejects bad arguments on the host before any HIP
call (fake, never-dereferenced addresses stand in for device pointers)."""
import ctypes
import os
import re

import pytest

from paper_2604_21290_amd import api

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "graphleap.h")

import torch  # noqa: E402

pytestmark = pytest.mark.skipif(not os.path.exists(api.LIB_PATH),
                                reason="libgraphleap.so not built")
# Fake addresses must never reach a real device: the validation checks run
# only where no GPU is visible (device_count does not initialise the runtime).
host_only = pytest.mark.skipif(torch.cuda.device_count() > 0,
                               reason="host-only checks (fake pointers)")

A = 1 << 20          # fake 16-byte-aligned device addresses, far apart
P = lambda i: ctypes.c_void_p(A * (i + 1))  # noqa: E731


def header_functions():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"^\s*(?:gl_status|const char\*|int|size_t)\s+(gl_\w+)\(", text,
                                 re.M)))


def test_exports_every_declared_symbol():
    names = header_functions()
    assert len(names) >= 12
    L = api.lib()
    for n in names:
        assert hasattr(L, n), n
    assert set(names) == set(api.SIGNATURES), "binding and header disagree"


def test_header_constants_match_binding():
    text = open(HEADER).read()
    for name in ("GL_MAX_KD", "GL_MAX_M", "GL_MAX_K"):
        v = int(re.search(rf"#define {name} (\d+)", text).group(1))
        assert v == getattr(api, name)


def _knn(x=P(0), B=2, N=196, C=192, keys=None, M=196, k=9, d=1, dt=1, out=P(40)):
    st = api.lib().gl_knn_graph(x, B, N, C, keys, M, k, d, dt, out, None)
    return api.STATUS[st], api.lib().gl_last_error().decode()


@host_only
def test_knn_validation():
    assert _knn(x=None)[0] == "GL_ERR_NULL_PTR"
    assert _knn(out=None)[0] == "GL_ERR_NULL_PTR"
    assert _knn(dt=7)[0] == "GL_ERR_UNSUPPORTED"
    assert _knn(B=0)[0] == "GL_ERR_BAD_SHAPE"
    assert _knn(N=0, M=0)[0] == "GL_ERR_BAD_SHAPE"
    assert _knn(M=100)[0] == "GL_ERR_BAD_SHAPE"           # keys = x needs M == N
    assert _knn(keys=P(10), M=5000)[0] == "GL_ERR_BAD_SHAPE"
    assert _knn(C=12)[0] == "GL_ERR_UNSUPPORTED"           # bf16 needs C % 8 == 0
    assert _knn(C=10, dt=0)[0] == "GL_ERR_UNSUPPORTED"     # fp32 needs C % 4 == 0
    assert _knn(k=0)[0] == "GL_ERR_BAD_K"
    assert _knn(d=0)[0] == "GL_ERR_BAD_K"
    assert _knn(k=33, d=2)[0] == "GL_ERR_BAD_K"             # k*d > 64
    assert _knn(keys=P(10), M=10, k=6, d=2)[0] == "GL_ERR_BAD_K"   # k*d > M
    assert _knn(x=ctypes.c_void_p(A + 8))[0] == "GL_ERR_ALIGNMENT"
    assert _knn(out=ctypes.c_void_p(A * 41 + 2))[0] == "GL_ERR_ALIGNMENT"
    assert _knn(out=ctypes.c_void_p(A + 4096))[0] == "GL_ERR_ALIAS"  # idx inside x
    st, msg = _knn(k=65)
    assert st == "GL_ERR_BAD_K" and "k*dilation" in msg


def _mr(x=P(0), B=2, N=196, C=192, keys=None, M=196, idx=P(20), k=9, W=P(30), bias=None,
        Cout=192, dt=1, out=P(40), ws=None, wsb=0):
    st = api.lib().gl_mrconv(x, B, N, C, keys, M, idx, k, W, bias, Cout, dt, out, ws, wsb, None)
    return api.STATUS[st]


@host_only
def test_mrconv_validation():
    assert _mr(x=None) == "GL_ERR_NULL_PTR"
    assert _mr(idx=None) == "GL_ERR_NULL_PTR"
    assert _mr(W=None) == "GL_ERR_NULL_PTR"
    assert _mr(out=None) == "GL_ERR_NULL_PTR"
    assert _mr(dt=2) == "GL_ERR_UNSUPPORTED"
    assert _mr(Cout=0) == "GL_ERR_BAD_SHAPE"
    assert _mr(M=10) == "GL_ERR_BAD_SHAPE"
    assert _mr(k=0) == "GL_ERR_BAD_K"
    assert _mr(k=65) == "GL_ERR_BAD_K"
    assert _mr(C=20) == "GL_ERR_UNSUPPORTED"
    # one image's keys beyond 2^31 16-byte vectors (the kernels' row offsets)
    assert _mr(keys=P(10), M=1 << 24, C=1024) == "GL_ERR_BAD_SHAPE"
    # too wide for one LDS tile: the two-pass form takes it, with a workspace
    assert _mr(C=8192) == "GL_ERR_WORKSPACE"
    assert _mr(W=ctypes.c_void_p(A * 31 + 4)) == "GL_ERR_ALIGNMENT"
    assert _mr(bias=ctypes.c_void_p(A * 50 + 1)) == "GL_ERR_ALIGNMENT"
    assert _mr(out=ctypes.c_void_p(A + 64)) == "GL_ERR_ALIAS"    # out inside x
    assert _mr(out=ctypes.c_void_p(A * 31 + 64)) == "GL_ERR_ALIAS"  # out inside W


def _pool(x=P(0), B=2, H=56, W=56, C=80, r=4, dt=1, out=P(40)):
    return api.STATUS[api.lib().gl_pool_keys(x, B, H, W, C, r, dt, out, None)]


@host_only
def test_pool_validation():
    assert _pool(out=None) == "GL_ERR_NULL_PTR"
    assert _pool(r=3) == "GL_ERR_BAD_SHAPE"
    assert _pool(r=0) == "GL_ERR_BAD_SHAPE"
    assert _pool(C=12) == "GL_ERR_UNSUPPORTED"
    assert _pool(out=ctypes.c_void_p(A + 16)) == "GL_ERR_ALIAS"


def _max_pool(x=P(0), B=2, H=56, W=56, C=80, r=2, dt=1, out=P(40)):
    return api.STATUS[api.lib().gl_max_pool_nodes(x, B, H, W, C, r, dt, out, None)]


@host_only
def test_max_pool_validation():
    assert _max_pool(x=None) == "GL_ERR_NULL_PTR"
    assert _max_pool(out=None) == "GL_ERR_NULL_PTR"
    assert _max_pool(dt=2) == "GL_ERR_UNSUPPORTED"
    assert _max_pool(H=55) == "GL_ERR_BAD_SHAPE"            # 55 % 2 != 0
    assert _max_pool(r=0) == "GL_ERR_BAD_SHAPE"
    assert _max_pool(C=12) == "GL_ERR_UNSUPPORTED"            # bf16 needs C % 8 == 0
    assert _max_pool(C=10, dt=0) == "GL_ERR_UNSUPPORTED"      # fp32 needs C % 4 == 0
    assert _max_pool(out=ctypes.c_void_p(A * 40 + 8)) == "GL_ERR_ALIGNMENT"
    assert _max_pool(out=ctypes.c_void_p(A + 16)) == "GL_ERR_ALIAS"


@host_only
def test_mrconv_workspace():
    """The two-pass form (W beyond 8 KB per node of the fused tile) needs the
    caller's [B*N, 2C] workspace; the fused tile needs none."""
    L = api.lib()
    need = L.gl_mrconv_workspace_bytes(64, 196, 640, 9, 640, 1)
    assert need == 64 * 196 * 1280 * 2
    assert L.gl_mrconv_workspace_bytes(32, 196, 192, 9, 192, 1) == 0
    assert L.gl_mrconv_workspace_bytes(0, 196, 192, 9, 192, 1) == 0
    assert L.gl_mrconv_workspace_bytes(2, 196, 192, 9, 192, 5) == 0     # bad dtype
    assert L.gl_graphleap_workspace_bytes(64, 14, 14, 640, 1, 9, 1) == need
    assert L.gl_graphleap_workspace_bytes(32, 14, 14, 192, 1, 9, 1) == 0
    assert L.gl_graphleap_workspace_bytes(32, 14, 14, 192, 3, 9, 1) == 0  # 14 % 3 != 0
    big = dict(B=64, C=640, Cout=640)
    assert _mr(**big) == "GL_ERR_WORKSPACE"
    assert _mr(**big, ws=P(60), wsb=need - 1) == "GL_ERR_WORKSPACE"
    assert _mr(**big, ws=ctypes.c_void_p(A * 61 + 8), wsb=need) == "GL_ERR_WORKSPACE"
    assert _mr(**big, ws=P(0), wsb=need) == "GL_ERR_ALIAS"              # on top of x
    assert _mr(**big, ws=ctypes.c_void_p(A * 40), wsb=need) == "GL_ERR_ALIAS"  # ends in out
    # a workspace is accepted where none is needed
    assert _mr(ws=P(60), wsb=1) != "GL_ERR_WORKSPACE"
    # a good workspace passes every check; with no GPU the launch itself fails
    assert _mr(**big, ws=P(60), wsb=need) == "GL_ERR_HIP"
    L = api.lib()
    # channels too wide for the fused tile: Wh is expanded into a dense W in
    # the workspace, ahead of the two-pass rows
    assert L.gl_mrconv_heads_workspace_bytes(1, 196, 2560, 9, 16, 1) >= 2560 * 5120 * 2
    st = L.gl_mrconv_heads(P(0), 1, 196, 2560, None, 196, P(20), 9, P(30), None, 16, 1, P(40),
                           None, 0, None)
    assert api.STATUS[st] == "GL_ERR_WORKSPACE"
    # the fused tile reads Wh directly and needs none
    assert L.gl_mrconv_heads_workspace_bytes(64, 196, 640, 9, 8, 1) == 0
    assert L.gl_mrconv_heads_workspace_bytes(2, 196, 192, 9, 5, 1) == 0   # bad heads


@host_only
def test_mrconv_noalloc_validation():
    """gl_mrconv_noalloc checks like gl_mrconv and refuses layers whose
    two-pass rows exceed the library's scratch buffer before any HIP call."""
    L = api.lib()

    def na(B=2, N=196, C=192, Cout=192, x=P(0), out=P(40)):
        st = L.gl_mrconv_noalloc(x, B, N, C, None, N, P(20), 9, P(30), None, Cout, 1, out, None)
        return api.STATUS[st], L.gl_last_error().decode()

    assert na(x=None)[0] == "GL_ERR_NULL_PTR"
    assert na(out=ctypes.c_void_p(A + 64))[0] == "GL_ERR_ALIAS"
    st, msg = na(B=64, C=1024, Cout=1024, out=P(200))    # 51 MB of rows > 32 MiB
    assert st == "GL_ERR_WORKSPACE" and "scratch" in msg, msg
    text = open(HEADER).read()
    assert "#define GL_NOALLOC_SCRATCH_BYTES (32u << 20)" in text


@host_only
def test_handle_validation():
    L = api.lib()
    assert api.STATUS[L.gl_lookahead_destroy(None)] == "GL_ERR_BAD_HANDLE"
    assert api.STATUS[L.gl_lookahead_set_profiling(None, 4)] == "GL_ERR_BAD_HANDLE"
    assert api.STATUS[L.gl_graphleap_block(None, P(0), 1, 14, 14, 192, 1, None, P(1), 9, P(2),
                                           None, 1, P(3), None, 1, None, 0)] == "GL_ERR_BAD_HANDLE"
    assert api.STATUS[L.gl_lookahead_create(None, None, None)] == "GL_ERR_NULL_PTR"


def test_status_strings():
    L = api.lib()
    for code, name in api.STATUS.items():
        assert L.gl_status_string(code).decode() == name
    assert L.gl_status_string(99).decode() == "GL_ERR_UNKNOWN"


def _lin(x=P(0), R=64, K=64, W=P(10), b=None, Co=64, ai=0, ao=0, res=None, dt=1, out=P(20)):
    st = api.lib().gl_linear(x, R, K, W, b, Co, ai, ao, res, dt, out, None)
    return api.STATUS[st]


@host_only
def test_linear_validation():
    assert _lin(x=None) == "GL_ERR_NULL_PTR"
    assert _lin(W=None) == "GL_ERR_NULL_PTR"
    assert _lin(ai=2) == "GL_ERR_UNSUPPORTED"
    assert _lin(dt=3) == "GL_ERR_UNSUPPORTED"
    assert _lin(R=0) == "GL_ERR_BAD_SHAPE"
    assert _lin(K=12) == "GL_ERR_UNSUPPORTED"               # bf16 rows need K % 8 == 0
    assert _lin(x=ctypes.c_void_p(A + 8)) == "GL_ERR_ALIGNMENT"
    assert _lin(out=P(0)) == "GL_ERR_ALIAS"                  # out on top of x
    assert _lin(res=ctypes.c_void_p(A * 21 + 64)) == "GL_ERR_ALIAS"   # partial overlap with out


@host_only
def test_vig_validation():
    L = api.lib()
    n = L.gl_vig_workspace_bytes(2, 14, 14, 192, 1, 9, 1)
    assert n > 0
    assert L.gl_vig_workspace_bytes(2, 196, 1, 192, 1, 9, 1) == n     # same N, same carve-up
    assert L.gl_vig_workspace_bytes(2, 14, 14, 192, 2, 9, 1) == n     # keys fit its own region
    assert L.gl_vig_workspace_bytes(0, 14, 14, 192, 1, 9, 1) == 0
    assert L.gl_vig_workspace_bytes(2, 14, 14, 192, 3, 9, 1) == 0     # 3 does not divide 14
    assert L.gl_vig_workspace_bytes(2, 14, 14, 192, 0, 9, 1) == 0
    assert L.gl_vig_workspace_bytes(2, 14, 14, 192, 1, 0, 1) == 0
    pp = api.VigParams()
    st = L.gl_vig_stack(None, P(0), 2, 14, 14, 192, 1, 2, 9, (ctypes.c_int * 2)(1, 1),
                        ctypes.byref(pp), 1, 2, P(5), 1 << 30, P(9))
    assert api.STATUS[st] == "GL_ERR_BAD_HANDLE"
    st = L.gl_vig_block(None, P(0), 2, 14, 14, 192, 2, 9, P(10), ctypes.byref(pp), 1, P(5),
                        1 << 30, P(7), None, 1, P(9))
    assert api.STATUS[st] == "GL_ERR_BAD_HANDLE"


@host_only
def test_mrconv_heads_validation():
    L = api.lib()
    st = L.gl_mrconv_heads(P(0), 2, 196, 192, None, 196, P(10), 9, P(20), None, 5, 1, P(30), None,
                           0, None)
    assert api.STATUS[st] == "GL_ERR_BAD_SHAPE"          # 5 does not divide 192
    st = L.gl_mrconv_heads(P(0), 2, 196, 192, None, 196, P(10), 9, P(20), None, 0, 1, P(30), None,
                           0, None)
    assert api.STATUS[st] == "GL_ERR_BAD_SHAPE"
