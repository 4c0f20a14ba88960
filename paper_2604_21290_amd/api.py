"""Thin ctypes binding of libgraphleap.so (include/graphleap.h).

Argument marshalling only: tensors are passed as device pointers, streams as
hipStream_t; every step of the path runs in the library's HIP kernels.  The
binding allocates outputs and workspaces with torch when the caller does not
pass them (PyTorch supplies device memory and streams, nothing else).

The library must have been built (python -m paper_2604_21290_amd.build);
loading raises if it is missing -- there is no fallback path.
"""
from __future__ import annotations

import ctypes
import os

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libgraphleap.so")

GL_F32, GL_BF16 = 0, 1
GL_SCHED_LOOKAHEAD, GL_SCHED_STANDARD, GL_SCHED_LOOKAHEAD_FUSED = 0, 1, 2
GL_TIME_BUILD, GL_TIME_UPDATE, GL_TIME_FUSED, GL_TIME_LINEAR = 0, 1, 2, 3
GL_ACT_NONE, GL_ACT_GELU = 0, 1
GL_MAX_KD, GL_MAX_M, GL_MAX_K = 64, 4096, 64

STATUS = {0: "GL_OK", 1: "GL_ERR_NULL_PTR", 2: "GL_ERR_BAD_SHAPE", 3: "GL_ERR_BAD_K",
          4: "GL_ERR_UNSUPPORTED", 5: "GL_ERR_ALIGNMENT", 6: "GL_ERR_ALIAS", 7: "GL_ERR_HIP",
          8: "GL_ERR_BAD_HANDLE", 9: "GL_ERR_WORKSPACE"}

_vp, _i, _f, _sz = ctypes.c_void_p, ctypes.c_int, ctypes.c_float, ctypes.c_size_t

VIG_PARAMS = ("W_in", "b_in", "W_upd", "b_upd", "W_out", "b_out", "W_1", "b_1", "W_2", "b_2")


class VigParams(ctypes.Structure):
    """gl_vig_params: device pointers of one full block's weights (NULL biases allowed)."""
    _fields_ = [(n, ctypes.c_void_p) for n in VIG_PARAMS]

# name -> argtypes (every entry point returns gl_status as int unless noted)
SIGNATURES = {
    "gl_knn_graph": [_vp, _i, _i, _i, _vp, _i, _i, _i, _i, _vp, _vp],
    "gl_pool_keys": [_vp, _i, _i, _i, _i, _i, _i, _vp, _vp],
    "gl_max_pool_nodes": [_vp, _i, _i, _i, _i, _i, _i, _vp, _vp],
    "gl_mrconv_workspace_bytes": [_i, _i, _i, _i, _i, _i],
    "gl_mrconv": [_vp, _i, _i, _i, _vp, _i, _vp, _i, _vp, _vp, _i, _i, _vp, _vp, _sz, _vp],
    "gl_mrconv_noalloc": [_vp, _i, _i, _i, _vp, _i, _vp, _i, _vp, _vp, _i, _i, _vp, _vp],
    "gl_mrconv_heads": [_vp, _i, _i, _i, _vp, _i, _vp, _i, _vp, _vp, _i, _i, _vp, _vp, _sz, _vp],
    "gl_mrconv_heads_workspace_bytes": [_i, _i, _i, _i, _i, _i],
    "gl_lookahead_create": [_vp, _vp, ctypes.POINTER(_vp)],
    "gl_lookahead_destroy": [_vp],
    "gl_lookahead_set_profiling": [_vp, _i],
    "gl_lookahead_kernel_times": [_vp, _i, ctypes.POINTER(_f), _i, ctypes.POINTER(_i)],
    "gl_lookahead_bootstrap": [_vp, _vp, _i, _i, _i, _i, _i, _vp, _i, _i, _i, _vp],
    "gl_graphleap_workspace_bytes": [_i, _i, _i, _i, _i, _i, _i],
    "gl_graphleap_block": [_vp, _vp, _i, _i, _i, _i, _i, _vp, _vp, _i, _vp, _vp, _i, _vp, _vp, _i,
                           _vp, _sz],
    "gl_graphleap_stack": [_vp, _vp, _i, _i, _i, _i, _i, _i, _i, ctypes.POINTER(_i), _vp, _vp, _i,
                           _i, _vp, _vp, _vp, _vp, _vp, _sz],
    "gl_linear": [_vp, _i, _i, _vp, _vp, _i, _i, _i, _vp, _i, _vp, _vp],
    "gl_vig_workspace_bytes": [_i, _i, _i, _i, _i, _i, _i],
    "gl_vig_block": [_vp, _vp, _i, _i, _i, _i, _i, _i, _vp, ctypes.POINTER(VigParams), _i, _vp,
                     _sz, _vp, _vp, _i, _vp],
    "gl_vig_stack": [_vp, _vp, _i, _i, _i, _i, _i, _i, _i, ctypes.POINTER(_i),
                     ctypes.POINTER(VigParams), _i, _i, _vp, _sz, _vp],
    "gl_status_string": [_i],
    "gl_last_error": [],
    "gl_version": [],
}
RESTYPES = {"gl_status_string": ctypes.c_char_p, "gl_last_error": ctypes.c_char_p,
            "gl_vig_workspace_bytes": ctypes.c_size_t, "gl_mrconv_workspace_bytes": ctypes.c_size_t,
            "gl_mrconv_heads_workspace_bytes": ctypes.c_size_t,
            "gl_graphleap_workspace_bytes": ctypes.c_size_t}

_lib = None


class GraphLeapError(RuntimeError):
    def __init__(self, name: str, status: int, detail: str):
        super().__init__(f"{name}: {STATUS.get(status, status)}: {detail}")
        self.status = status


def lib() -> ctypes.CDLL:
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is not built; run `python -m paper_2604_21290_amd.build`")
        L = ctypes.CDLL(LIB_PATH)
        for name, args in SIGNATURES.items():
            fn = getattr(L, name)
            fn.argtypes = args
            fn.restype = RESTYPES.get(name, ctypes.c_int)
        _lib = L
    return _lib


def _check(name: str, status: int):
    if status != 0:
        raise GraphLeapError(name, status, lib().gl_last_error().decode())


def _call(name: str, *args):
    _check(name, getattr(lib(), name)(*args))


def _dt(t: torch.Tensor) -> int:
    if t.dtype == torch.float32:
        return GL_F32
    if t.dtype == torch.bfloat16:
        return GL_BF16
    raise TypeError(f"unsupported dtype {t.dtype}")


def _p(t):
    if t is None:
        return None
    if isinstance(t, Workspace):
        return ctypes.c_void_p(t.ptr)
    if not t.is_cuda or not t.is_contiguous():
        raise ValueError("tensors must be contiguous device tensors")
    return ctypes.c_void_p(t.data_ptr())


def _s(stream) -> ctypes.c_void_p:
    s = torch.cuda.current_stream() if stream is None else stream
    return ctypes.c_void_p(s.cuda_stream)


# ---------------------------------------------------------------------------
# single calls
# ---------------------------------------------------------------------------
def knn_graph(x: torch.Tensor, k: int, dilation: int = 1, keys: torch.Tensor | None = None,
              out: torch.Tensor | None = None, stream=None) -> torch.Tensor:
    """idx[B, N, k] int32: dilated kNN of each row of x among keys (or x)."""
    B, N, C = x.shape
    M = N if keys is None else keys.shape[1]
    if out is None:
        out = torch.empty((B, N, k), dtype=torch.int32, device=x.device)
    _call("gl_knn_graph", _p(x), B, N, C, _p(keys), M, k, dilation, _dt(x), _p(out), _s(stream))
    return out


def pool_keys(x: torch.Tensor, H: int, W: int, r: int, out: torch.Tensor | None = None,
              stream=None) -> torch.Tensor:
    B, N, C = x.shape
    if out is None:
        out = torch.empty((B, (H // r) * (W // r), C), dtype=x.dtype, device=x.device)
    _call("gl_pool_keys", _p(x), B, H, W, C, r, _dt(x), _p(out), _s(stream))
    return out


def max_pool_nodes(x: torch.Tensor, H: int, W: int, r: int = 2, out: torch.Tensor | None = None,
                   stream=None) -> torch.Tensor:
    """Node reduction between pyramid stages: r x r max pooling of the H x W grid."""
    B, N, C = x.shape
    if out is None:
        out = torch.empty((B, (H // r) * (W // r), C), dtype=x.dtype, device=x.device)
    _call("gl_max_pool_nodes", _p(x), B, H, W, C, r, _dt(x), _p(out), _s(stream))
    return out


class Workspace:
    """A caller-owned device workspace: a torch uint8 buffer (or none when the
    call needs 0 bytes), passed as pointer and size."""

    def __init__(self, nbytes: int, device):
        self.nbytes = int(nbytes)
        self.buf = torch.empty(self.nbytes, dtype=torch.uint8, device=device) if nbytes else None
        self.ptr = self.buf.data_ptr() if nbytes else None

    def record_stream(self, s):
        if self.buf is not None:
            self.buf.record_stream(s)


def mrconv_workspace(B: int, N: int, C: int, k: int, Cout: int, dtype, device) -> Workspace:
    """Workspace of gl_mrconv / gl_mrconv_heads for this layer (empty when the
    fused tile needs none)."""
    dt = GL_BF16 if dtype == torch.bfloat16 else GL_F32
    return Workspace(lib().gl_mrconv_workspace_bytes(B, N, C, k, Cout, dt), device)


def mrconv(x: torch.Tensor, idx: torch.Tensor, W: torch.Tensor, bias: torch.Tensor | None = None,
           keys: torch.Tensor | None = None, out: torch.Tensor | None = None,
           stream=None, ws: Workspace | None = None) -> torch.Tensor:
    """out[B, N, Cout] = [x_i, max_j (keys_j - x_i)] W^T + bias (gl_mrconv).
    ws: the call's workspace (allocated here when not given)."""
    B, N, C = x.shape
    M = N if keys is None else keys.shape[1]
    k = idx.shape[2]
    Cout = W.shape[0]
    if out is None:
        out = torch.empty((B, N, Cout), dtype=x.dtype, device=x.device)
    if ws is None:
        ws = mrconv_workspace(B, N, C, k, Cout, x.dtype, x.device)
    _call("gl_mrconv", _p(x), B, N, C, _p(keys), M, _p(idx), k, _p(W), _p(bias), Cout, _dt(x),
          _p(out), _p(ws), ws.nbytes, _s(stream))
    return out


def mrconv_heads_workspace(B: int, N: int, C: int, k: int, heads: int, dtype, device) -> Workspace:
    """Workspace of gl_mrconv_heads for this layer (empty for the grouped kernel)."""
    dt = GL_BF16 if dtype == torch.bfloat16 else GL_F32
    return Workspace(lib().gl_mrconv_heads_workspace_bytes(B, N, C, k, heads, dt), device)


def mrconv_heads(x: torch.Tensor, idx: torch.Tensor, Wh: torch.Tensor,
                 bias: torch.Tensor | None = None, keys: torch.Tensor | None = None,
                 out: torch.Tensor | None = None, stream=None,
                 ws: Workspace | None = None) -> torch.Tensor:
    """The multi-head update (gl_mrconv_heads): Wh [H, hd, 2hd] holds each head's
    [W_x,h | W_m,h]; out[B, N, C] with C = H * hd."""
    B, N, C = x.shape
    H, hd, two_hd = Wh.shape
    if H * hd != C or two_hd != 2 * hd:
        raise ValueError(f"mrconv_heads: Wh {tuple(Wh.shape)} does not match C={C}")
    M = N if keys is None else keys.shape[1]
    k = idx.shape[2]
    if out is None:
        out = torch.empty((B, N, C), dtype=x.dtype, device=x.device)
    if ws is None:
        ws = mrconv_heads_workspace(B, N, C, k, H, x.dtype, x.device)
    _call("gl_mrconv_heads", _p(x), B, N, C, _p(keys), M, _p(idx), k, _p(Wh), _p(bias), H,
          _dt(x), _p(out), _p(ws), ws.nbytes, _s(stream))
    return out


def mrconv_noalloc(x: torch.Tensor, idx: torch.Tensor, W: torch.Tensor,
                   bias: torch.Tensor | None = None, keys: torch.Tensor | None = None,
                   out: torch.Tensor | None = None, stream=None) -> torch.Tensor:
    """gl_mrconv_noalloc: the update with the library's own scratch buffer (no
    workspace; calls on one device must not overlap)."""
    B, N, C = x.shape
    M = N if keys is None else keys.shape[1]
    Cout = W.shape[0]
    if out is None:
        out = torch.empty((B, N, Cout), dtype=x.dtype, device=x.device)
    _call("gl_mrconv_noalloc", _p(x), B, N, C, _p(keys), M, _p(idx), idx.shape[2], _p(W), _p(bias),
          Cout, _dt(x), _p(out), _s(stream))
    return out


def linear(x: torch.Tensor, W: torch.Tensor, bias: torch.Tensor | None = None,
           act_in: int = GL_ACT_NONE, act_out: int = GL_ACT_NONE,
           residual: torch.Tensor | None = None, out: torch.Tensor | None = None,
           stream=None) -> torch.Tensor:
    """out[..., Cout] = act_out(act_in(x) W^T + bias) + residual over the last axis."""
    K = x.shape[-1]
    R = x.numel() // K
    Cout = W.shape[0]
    if out is None:
        out = torch.empty(x.shape[:-1] + (Cout,), dtype=x.dtype, device=x.device)
    _call("gl_linear", _p(x), R, K, _p(W), _p(bias), Cout, act_in, act_out, _p(residual), _dt(x),
          _p(out), _s(stream))
    return out


def vig_params(p: dict) -> VigParams:
    """gl_vig_params from a dict of device tensors keyed like VIG_PARAMS."""
    return VigParams(*[(p[n].data_ptr() if p.get(n) is not None else None) for n in VIG_PARAMS])


def _grid(N, H, W):
    """The node grid (H, W); a plain N-node set is the N x 1 grid."""
    if H is None:
        return N, 1
    if H * W != N:
        raise GraphLeapError("grid", 2, f"H*W={H * W} != N={N}")
    return H, W


def vig_workspace(x0: torch.Tensor, k: int, H=None, W=None, pool_r: int = 1) -> torch.Tensor:
    B, N, C = x0.shape
    H, W = _grid(N, H, W)
    n = lib().gl_vig_workspace_bytes(B, H, W, C, pool_r, k, _dt(x0))
    if not n:
        raise GraphLeapError("gl_vig_workspace_bytes", 2, "bad shape")
    return torch.empty(n, dtype=torch.uint8, device=x0.device)


# ---------------------------------------------------------------------------
# lookahead
# ---------------------------------------------------------------------------
class Lookahead:
    """Owns a gl_lookahead handle bound to an update stream and a build stream."""

    def __init__(self, s_update=None, s_build=None):
        self.s_update = s_update if s_update is not None else torch.cuda.current_stream()
        self.s_build = s_build if s_build is not None else torch.cuda.Stream()
        h = ctypes.c_void_p()
        _call("gl_lookahead_create", _s(self.s_update), _s(self.s_build), ctypes.byref(h))
        self._h = h

    def close(self):
        if self._h is not None and self._h.value:
            _call("gl_lookahead_destroy", self._h)
        self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def _keep(self, *ts):
        for t in ts:
            if t is not None:
                t.record_stream(self.s_build)

    def set_profiling(self, max_records: int):
        _call("gl_lookahead_set_profiling", self._h, max_records)

    def kernel_times_ms(self, which: int = GL_TIME_BUILD, cap: int = 1 << 16) -> list:
        """Durations (ms) of the profiled builds (GL_TIME_BUILD), updates
        (GL_TIME_UPDATE) or one-launch blocks (GL_TIME_FUSED)."""
        buf = (ctypes.c_float * cap)()
        n = ctypes.c_int()
        _call("gl_lookahead_kernel_times", self._h, which, buf, cap, ctypes.byref(n))
        return list(buf[: n.value])

    def bootstrap(self, x0, H, W, k, dilation0, pool_r=1, keys_ws=None, idx0=None):
        B, N, C = x0.shape
        if idx0 is None:
            idx0 = torch.empty((B, N, k), dtype=torch.int32, device=x0.device)
        self._keep(x0, keys_ws, idx0)
        _call("gl_lookahead_bootstrap", self._h, _p(x0), B, H, W, C, pool_r, _p(keys_ws), k,
              dilation0, _dt(x0), _p(idx0))
        return idx0

    def block(self, x_in, H, W, idx_use, Wt, bias=None, pool_r=1, keys_ws=None, x_out=None,
              idx_next=None, dilation_next=1, ws: Workspace | None = None):
        B, N, C = x_in.shape
        k = idx_use.shape[2]
        if x_out is None:
            x_out = torch.empty_like(x_in)
        if ws is None:
            ws = graphleap_workspace(x_in, H, W, k, pool_r)
        self._keep(x_in, keys_ws, idx_next)
        _call("gl_graphleap_block", self._h, _p(x_in), B, H, W, C, pool_r, _p(keys_ws),
              _p(idx_use), k, _p(Wt), _p(bias), _dt(x_in), _p(x_out), _p(idx_next),
              dilation_next, _p(ws), ws.nbytes)
        return x_out

    def vig_block(self, x_in, idx_use, params: dict, ws, u_out=None, x_out=None, idx_next=None,
                  dilation_next=1, H=None, W=None, pool_r=1):
        """One full ViG block; returns (x_out, u_out).  With pool_r > 1 the
        graphs index U's keys pooled pool_r x pool_r over the H x W grid."""
        B, N, C = x_in.shape
        H, W = _grid(N, H, W)
        k = idx_use.shape[2]
        x_out = torch.empty_like(x_in) if x_out is None else x_out
        u_out = torch.empty_like(x_in) if u_out is None else u_out
        self._keep(x_in, ws, u_out, idx_use, idx_next)
        pp = vig_params(params)
        _call("gl_vig_block", self._h, _p(x_in), B, H, W, C, pool_r, k, _p(idx_use),
              ctypes.byref(pp), _dt(x_in), _p(ws), ws.numel(), _p(u_out), _p(idx_next),
              dilation_next, _p(x_out))
        return x_out, u_out

    def vig_stack(self, x0, params: list, dilations, k, schedule=GL_SCHED_LOOKAHEAD_FUSED,
                  ws=None, x_out=None, H=None, W=None, pool_r=1):
        """len(dilations) full ViG blocks; params: list of dicts of device tensors.
        With pool_r > 1 keys are pooled pool_r x pool_r over the H x W grid."""
        B, N, C = x0.shape
        H, W = _grid(N, H, W)
        L = len(dilations)
        ws = vig_workspace(x0, k, H, W, pool_r) if ws is None else ws
        x_out = torch.empty_like(x0) if x_out is None else x_out
        dil = (ctypes.c_int * L)(*dilations)
        arr = (VigParams * L)(*[vig_params(p) for p in params])
        self._keep(x0, ws)
        _call("gl_vig_stack", self._h, _p(x0), B, H, W, C, pool_r, L, k, dil, arr, _dt(x0),
              schedule, _p(ws), ws.numel(), _p(x_out))
        return x_out

    def stack(self, x0, H, W, Ws, bs, dilations, k, pool_r=1, schedule=GL_SCHED_LOOKAHEAD,
              ws=None, x_out=None):
        """Run len(dilations) blocks; Ws [L, C, 2C], bs [L, C] or None."""
        B, N, C = x0.shape
        L = len(dilations)
        if ws is None:
            ws = make_stack_workspace(x0, H, W, k, pool_r)
        if x_out is None:
            x_out = torch.empty_like(x0)
        dil = (ctypes.c_int * L)(*dilations)
        self._keep(x0, ws["x"], ws["idx"], ws["keys"])
        ws["mr"].record_stream(self.s_build)
        _call("gl_graphleap_stack", self._h, _p(x0), B, H, W, C, pool_r, L, k, dil, _p(Ws),
              _p(bs), _dt(x0), schedule, _p(ws["x"]), _p(ws["idx"]), _p(ws["keys"]), _p(x_out),
              _p(ws["mr"]), ws["mr"].nbytes)
        return x_out


def graphleap_workspace(x0: torch.Tensor, H: int, W: int, k: int, pool_r: int = 1) -> Workspace:
    """The MRConv workspace of gl_graphleap_block / gl_graphleap_stack."""
    B, N, C = x0.shape
    return Workspace(lib().gl_graphleap_workspace_bytes(B, H, W, C, pool_r, k, _dt(x0)), x0.device)


def make_stack_workspace(x0: torch.Tensor, H: int, W: int, k: int, pool_r: int = 1) -> dict:
    B, N, C = x0.shape
    M = (H // pool_r) * (W // pool_r)
    return {
        "x": torch.empty((2, B, N, C), dtype=x0.dtype, device=x0.device),
        "idx": torch.empty((2, B, N, k), dtype=torch.int32, device=x0.device),
        "keys": torch.empty((B, M, C), dtype=x0.dtype, device=x0.device) if pool_r > 1 else None,
        "mr": graphleap_workspace(x0, H, W, k, pool_r),
    }


def version() -> int:
    return lib().gl_version()
