"""Python binding of libmhlmoe, the MI355X (gfx950) hot path of Multi-Head
LatentMoE: IO-aware routing and IO-aware expert computation.

The functions carry the C ABI's names (see include/mhlmoe.h) and only
marshal arguments: every step of the computation runs in the HIP kernels of
libmhlmoe.so.  PyTorch supplies device memory (outputs and workspaces the
caller did not pass) and the current HIP stream.  There is no CPU fallback:
if the library is not built, or a tensor is not on the GPU, the call raises.
"""
from __future__ import annotations

import ctypes
import os
import re
from typing import Optional

import torch

__all__ = [
    "MhlmoeError", "load_library", "library_path", "declared_functions",
    "MHLMOE_F32", "MHLMOE_BF16",
    "MHLMOE_OP_ROUTE", "MHLMOE_OP_BUCKET", "MHLMOE_OP_EXPERTS", "MHLMOE_OP_LAYER",
    "MHLMOE_OP_LAYER_BACKWARD",
    "mhlmoe_version", "mhlmoe_last_error", "mhlmoe_workspace_size",
    "mhlmoe_route", "mhlmoe_route_static", "mhlmoe_bucket", "mhlmoe_experts", "mhlmoe_layer",
    "mhlmoe_experts_gelu", "mhlmoe_layer_gelu",
    "mhlmoe_layer_backward", "workspace",
    "mhlmoe_timing_enable", "mhlmoe_timing_query", "mhlmoe_timing_reset",
]

_PKG = os.path.dirname(os.path.abspath(__file__))
_ROOT = os.path.dirname(_PKG)
HEADER = os.path.join(_ROOT, "include", "mhlmoe.h")

MHLMOE_OK, MHLMOE_EINVAL, MHLMOE_EUNSUPPORTED, MHLMOE_EWORKSPACE, MHLMOE_EHIP = range(5)
MHLMOE_F32, MHLMOE_BF16 = 0, 1
(MHLMOE_OP_ROUTE, MHLMOE_OP_BUCKET, MHLMOE_OP_EXPERTS, MHLMOE_OP_LAYER,
 MHLMOE_OP_LAYER_BACKWARD, MHLMOE_OP_LATENT_LAYER, MHLMOE_OP_LATENT_BACKWARD,
 MHLMOE_OP_ROUTE_BACKWARD) = range(8)
_STATUS = {0: "MHLMOE_OK", 1: "MHLMOE_EINVAL", 2: "MHLMOE_EUNSUPPORTED",
           3: "MHLMOE_EWORKSPACE", 4: "MHLMOE_EHIP"}

_P = ctypes.c_void_p
_I64 = ctypes.c_int64
_I = ctypes.c_int
_SZ = ctypes.c_size_t


class MhlmoeError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"{_STATUS.get(status, status)}: {message}")
        self.status = status


def library_path() -> str:
    return os.path.join(_PKG, "libmhlmoe.so")


_lib = None


def _declare(lib):
    lib.mhlmoe_version.restype = _I
    lib.mhlmoe_version.argtypes = []
    lib.mhlmoe_last_error.restype = ctypes.c_char_p
    lib.mhlmoe_last_error.argtypes = []
    lib.mhlmoe_workspace_size.argtypes = [_I, _I64, _I, _I, _I, _I, _I, _I, ctypes.POINTER(_SZ)]
    lib.mhlmoe_route.argtypes = [_P, _P, _P, _I64, _I, _I, _I, _I, _I, _P, _P, _P, _P, _SZ, _P]
    lib.mhlmoe_route_static.argtypes = [_P, _P, _P, _I64, _I, _I, _I, _I, _I, _P, _P, _P, _P]
    lib.mhlmoe_route_backward.argtypes = [_P] * 5 + [_I64, _I, _I, _I, _I, _I] + [_P] * 3 + [_SZ, _P]
    lib.mhlmoe_bucket.argtypes = [_P, _I64, _I, _I, _I, _P, _P, _P, _P, _SZ, _P]
    lib.mhlmoe_experts.argtypes = [_P, _P, _P, _P, _P, _P, _I64, _I, _I, _I, _I, _I, _I, _P, _P, _SZ, _P]
    lib.mhlmoe_layer.argtypes = ([_P] * 6 + [_I64, _I, _I, _I, _I, _I, _I] + [_P] * 5 + [_SZ, _P])
    lib.mhlmoe_layer_backward.argtypes = ([_P] * 8 + [_I64, _I, _I, _I, _I, _I, _I] + [_P] * 6 + [_SZ, _P])
    lib.mhlmoe_experts_gelu.argtypes = [_P] * 5 + [_I64, _I, _I, _I, _I, _I, _I, _P, _P, _SZ, _P]
    lib.mhlmoe_layer_gelu.argtypes = ([_P] * 5 + [_I64, _I, _I, _I, _I, _I, _I] + [_P] * 5 + [_SZ, _P])
    lib.mhlmoe_layer_gelu_backward.argtypes = ([_P] * 7 + [_I64, _I, _I, _I, _I, _I, _I]
                                               + [_P] * 5 + [_SZ, _P])
    lib.mhlmoe_layer_routed.argtypes = ([_P] * 7 + [_I64, _I, _I, _I, _I, _I, _I] + [_P] * 5
                                        + [_SZ, _P])
    lib.mhlmoe_layer_backward_routed.argtypes = ([_P] * 9 + [_I64, _I, _I, _I, _I, _I, _I]
                                                 + [_P] * 7 + [_SZ, _P])
    lib.mhlmoe_latent_layer.argtypes = [_P] * 8 + [_I64] + [_I] * 8 + [_P] * 8 + [_SZ, _P]
    lib.mhlmoe_latent_layer_backward.argtypes = ([_P] * 13 + [_I64] + [_I] * 8 + [_P] * 8
                                                 + [_SZ, _P])
    lib.mhlmoe_bias_update.argtypes = [_P, _P, _I, _I, ctypes.c_float, _P]
    lib.mhlmoe_timing_enable.argtypes = [_I]
    lib.mhlmoe_timing_query.argtypes = [ctypes.c_char_p, ctypes.POINTER(ctypes.c_double),
                                        ctypes.POINTER(_I64)]
    lib.mhlmoe_timing_reset.argtypes = []
    for name in ("mhlmoe_workspace_size", "mhlmoe_route", "mhlmoe_bucket", "mhlmoe_experts",
                 "mhlmoe_layer", "mhlmoe_layer_backward", "mhlmoe_experts_gelu",
                 "mhlmoe_layer_gelu", "mhlmoe_timing_enable",
                 "mhlmoe_timing_query", "mhlmoe_timing_reset"):
        getattr(lib, name).restype = _I
    return lib


def load_library():
    """Load the in-tree libmhlmoe.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        path = library_path()
        if not os.path.exists(path):
            raise RuntimeError(
                f"{path} is missing: build it with `python -m paper_2602_04870_amd.build` "
                "(there is no fallback implementation)")
        _lib = _declare(ctypes.CDLL(path))
    return _lib


def declared_functions(header: str = HEADER):
    """Names of the functions include/mhlmoe.h declares."""
    text = open(header).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(mhlmoe_[a-z_]+)\s*\(", text)))


def _check(status: int):
    if status != MHLMOE_OK:
        msg = load_library().mhlmoe_last_error().decode(errors="replace")
        raise MhlmoeError(status, msg)


def _dtype_code(t: torch.Tensor) -> int:
    if t.dtype == torch.float32:
        return MHLMOE_F32
    if t.dtype == torch.bfloat16:
        return MHLMOE_BF16
    raise TypeError(f"unsupported activation/weight dtype {t.dtype}")


def _dev(t: Optional[torch.Tensor], name: str, dtype=None, shape=None):
    """Device pointer of a contiguous GPU tensor (None -> NULL)."""
    if t is None:
        return None
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if t.device.type != "cuda":
        raise ValueError(f"{name} must be a GPU tensor (got {t.device}); libmhlmoe has no CPU path")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if dtype is not None and t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype} (got {t.dtype})")
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} must have shape {tuple(shape)} (got {tuple(t.shape)})")
    return ctypes.c_void_p(t.data_ptr())


def _stream(stream) -> ctypes.c_void_p:
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream))


def mhlmoe_version() -> int:
    return load_library().mhlmoe_version()


def mhlmoe_last_error() -> str:
    return load_library().mhlmoe_last_error().decode(errors="replace")


def mhlmoe_workspace_size(op: int, T: int, n_heads: int, d_head: int, n_experts: int,
                          top_k: int, d_ff: int = 0, dtype: int = MHLMOE_BF16) -> int:
    out = _SZ(0)
    _check(load_library().mhlmoe_workspace_size(op, T, n_heads, d_head, n_experts, top_k,
                                                d_ff, dtype, ctypes.byref(out)))
    return out.value


def workspace(op: int, T: int, n_heads: int, d_head: int, n_experts: int, top_k: int,
              d_ff: int = 0, dtype: int = MHLMOE_BF16, device="cuda") -> torch.Tensor:
    """Allocate a workspace tensor for entry point `op` (at least 1 byte)."""
    n = mhlmoe_workspace_size(op, T, n_heads, d_head, n_experts, top_k, d_ff, dtype)
    return torch.empty(max(n, 256), dtype=torch.uint8, device=device)


def _ws(ws, op, *shape):
    if ws is None:
        ws = workspace(op, *shape)
    return _dev(ws, "workspace", torch.uint8), ws.numel()


def mhlmoe_route(X, W_router, bias, top_k, *, idx=None, gate=None, counts=None,
                 workspace=None, stream=None):
    """Algorithm 1: returns (idx [T,Nh,k] int32, gate [T,Nh,k] f32,
    counts [Nh,Ne] int32)."""
    T, Nh, dh = X.shape
    Ne = W_router.shape[1]
    dt = _dtype_code(X)
    dev = X.device
    idx = idx if idx is not None else torch.empty((T, Nh, top_k), dtype=torch.int32, device=dev)
    gate = gate if gate is not None else torch.empty((T, Nh, top_k), dtype=torch.float32, device=dev)
    counts = counts if counts is not None else torch.empty((Nh, Ne), dtype=torch.int32, device=dev)
    wsp, wsn = _ws(workspace, MHLMOE_OP_ROUTE, T, Nh, dh, Ne, top_k, 0, dt)
    _check(load_library().mhlmoe_route(
        _dev(X, "X"), _dev(W_router, "W_router", torch.float32, (Nh, Ne, dh)),
        _dev(bias, "bias", torch.float32, (Nh, Ne)), T, Nh, dh, Ne, top_k, dt,
        _dev(idx, "idx", torch.int32, (T, Nh, top_k)),
        _dev(gate, "gate", torch.float32, (T, Nh, top_k)),
        _dev(counts, "counts", torch.int32, (Nh, Ne)), wsp, wsn, _stream(stream)))
    return idx, gate, counts


def mhlmoe_route_static(X, W_router, bias, top_k, *, idx, gate, counts, stream=None):
    """mhlmoe_route without a workspace (the library's static scratch):
    the caller passes the outputs idx [T,Nh,k] int32, gate [T,Nh,k] f32 and
    counts [Nh,Ne] int32, so the call allocates nothing."""
    T, Nh, dh = X.shape
    Ne = W_router.shape[1]
    _check(load_library().mhlmoe_route_static(
        _dev(X, "X"), _dev(W_router, "W_router", torch.float32, (Nh, Ne, dh)),
        _dev(bias, "bias", torch.float32, (Nh, Ne)), T, Nh, dh, Ne, top_k, _dtype_code(X),
        _dev(idx, "idx", torch.int32, (T, Nh, top_k)),
        _dev(gate, "gate", torch.float32, (T, Nh, top_k)),
        _dev(counts, "counts", torch.int32, (Nh, Ne)), _stream(stream)))
    return idx, gate, counts


def mhlmoe_route_backward(X, W_router, idx, gate, dgate, *, dX=None, dW_router=None,
                          workspace=None, stream=None):
    """Algorithm 2 from the gate gradient: returns (dX, dW_router)."""
    T, Nh, dh = X.shape
    Ne = W_router.shape[1]
    k = idx.shape[2]
    dt = _dtype_code(X)
    f32 = torch.float32
    dX = dX if dX is not None else torch.empty_like(X)
    dW_router = dW_router if dW_router is not None else torch.empty((Nh, Ne, dh), dtype=f32,
                                                                    device=X.device)
    wsp, wsn = _ws(workspace, MHLMOE_OP_ROUTE_BACKWARD, T, Nh, dh, Ne, k, 0, dt)
    _check(load_library().mhlmoe_route_backward(
        _dev(X, "X"), _dev(W_router, "W_router", f32, (Nh, Ne, dh)),
        _dev(idx, "idx", torch.int32, (T, Nh, k)), _dev(gate, "gate", f32, (T, Nh, k)),
        _dev(dgate, "dgate", f32, (T, Nh, k)), T, Nh, dh, Ne, k, dt,
        _dev(dX, "dX", X.dtype, (T, Nh, dh)), _dev(dW_router, "dW_router", f32, (Nh, Ne, dh)),
        wsp, wsn, _stream(stream)))
    return dX, dW_router


def mhlmoe_bucket(idx, n_experts, *, counts=None, offsets=None, perm=None, workspace=None,
                  stream=None):
    """Token clustering: returns (counts [Nh,Ne], offsets [Nh,Ne+1], perm [Nh,T*k])."""
    T, Nh, k = idx.shape
    Ne = n_experts
    dev = idx.device
    counts = counts if counts is not None else torch.empty((Nh, Ne), dtype=torch.int32, device=dev)
    offsets = offsets if offsets is not None else torch.empty((Nh, Ne + 1), dtype=torch.int32, device=dev)
    perm = perm if perm is not None else torch.empty((Nh, T * k), dtype=torch.int32, device=dev)
    wsp, wsn = _ws(workspace, MHLMOE_OP_BUCKET, T, Nh, 64, Ne, k, 0, MHLMOE_BF16)
    _check(load_library().mhlmoe_bucket(
        _dev(idx, "idx", torch.int32), T, Nh, Ne, k,
        _dev(counts, "counts", torch.int32, (Nh, Ne)),
        _dev(offsets, "offsets", torch.int32, (Nh, Ne + 1)),
        _dev(perm, "perm", torch.int32, (Nh, T * k)), wsp, wsn, _stream(stream)))
    return counts, offsets, perm


def mhlmoe_experts(X, idx, gate, W1, W3, W2, *, Y=None, workspace=None, stream=None):
    """Grouped SwiGLU experts + gate-weighted combine: returns Y [T,Nh,dh]."""
    T, Nh, dh = X.shape
    k = idx.shape[2]
    Ne, dff = W1.shape[1], W1.shape[2]
    dt = _dtype_code(X)
    Y = Y if Y is not None else torch.empty_like(X)
    wsp, wsn = _ws(workspace, MHLMOE_OP_EXPERTS, T, Nh, dh, Ne, k, dff, dt)
    _check(load_library().mhlmoe_experts(
        _dev(X, "X"), _dev(idx, "idx", torch.int32, (T, Nh, k)),
        _dev(gate, "gate", torch.float32, (T, Nh, k)),
        _dev(W1, "W1", X.dtype, (Nh, Ne, dff, dh)), _dev(W3, "W3", X.dtype, (Nh, Ne, dff, dh)),
        _dev(W2, "W2", X.dtype, (Nh, Ne, dh, dff)), T, Nh, dh, Ne, k, dff, dt,
        _dev(Y, "Y", X.dtype, (T, Nh, dh)), wsp, wsn, _stream(stream)))
    return Y


def mhlmoe_layer(X, W_router, bias, W1, W3, W2, top_k, *, Y=None, idx=None, gate=None,
                 counts=None, workspace=None, stream=None, return_routing=True):
    """Routing + experts.  Returns Y, or (Y, idx, gate, counts) when
    return_routing (routing outputs are then allocated if not passed)."""
    T, Nh, dh = X.shape
    Ne, dff = W1.shape[1], W1.shape[2]
    dt = _dtype_code(X)
    dev = X.device
    Y = Y if Y is not None else torch.empty_like(X)
    if return_routing:
        idx = idx if idx is not None else torch.empty((T, Nh, top_k), dtype=torch.int32, device=dev)
        gate = gate if gate is not None else torch.empty((T, Nh, top_k), dtype=torch.float32, device=dev)
        counts = counts if counts is not None else torch.empty((Nh, Ne), dtype=torch.int32, device=dev)
    wsp, wsn = _ws(workspace, MHLMOE_OP_LAYER, T, Nh, dh, Ne, top_k, dff, dt)
    _check(load_library().mhlmoe_layer(
        _dev(X, "X"), _dev(W_router, "W_router", torch.float32, (Nh, Ne, dh)),
        _dev(bias, "bias", torch.float32, (Nh, Ne)),
        _dev(W1, "W1", X.dtype, (Nh, Ne, dff, dh)), _dev(W3, "W3", X.dtype, (Nh, Ne, dff, dh)),
        _dev(W2, "W2", X.dtype, (Nh, Ne, dh, dff)), T, Nh, dh, Ne, top_k, dff, dt,
        _dev(Y, "Y", X.dtype, (T, Nh, dh)), _dev(idx, "idx", torch.int32, (T, Nh, top_k)),
        _dev(gate, "gate", torch.float32, (T, Nh, top_k)),
        _dev(counts, "counts", torch.int32, (Nh, Ne)), wsp, wsn, _stream(stream)))
    return (Y, idx, gate, counts) if return_routing else Y


def mhlmoe_experts_gelu(X, idx, gate, W_in, W_out, *, Y=None, workspace=None, stream=None):
    """Grouped two-matrix GELU experts (Sec. 3.4) + gate-weighted combine:
    returns Y [T,Nh,dh]."""
    T, Nh, dh = X.shape
    k = idx.shape[2]
    Ne, dff = W_in.shape[1], W_in.shape[2]
    dt = _dtype_code(X)
    Y = Y if Y is not None else torch.empty_like(X)
    wsp, wsn = _ws(workspace, MHLMOE_OP_EXPERTS, T, Nh, dh, Ne, k, dff, dt)
    _check(load_library().mhlmoe_experts_gelu(
        _dev(X, "X"), _dev(idx, "idx", torch.int32, (T, Nh, k)),
        _dev(gate, "gate", torch.float32, (T, Nh, k)),
        _dev(W_in, "W_in", X.dtype, (Nh, Ne, dff, dh)),
        _dev(W_out, "W_out", X.dtype, (Nh, Ne, dh, dff)), T, Nh, dh, Ne, k, dff, dt,
        _dev(Y, "Y", X.dtype, (T, Nh, dh)), wsp, wsn, _stream(stream)))
    return Y


def mhlmoe_layer_gelu(X, W_router, bias, W_in, W_out, top_k, *, Y=None, idx=None, gate=None,
                      counts=None, workspace=None, stream=None, return_routing=True):
    """Routing + the GELU experts.  Returns Y, or (Y, idx, gate, counts)."""
    T, Nh, dh = X.shape
    Ne, dff = W_in.shape[1], W_in.shape[2]
    dt = _dtype_code(X)
    dev = X.device
    Y = Y if Y is not None else torch.empty_like(X)
    if return_routing:
        idx = idx if idx is not None else torch.empty((T, Nh, top_k), dtype=torch.int32, device=dev)
        gate = gate if gate is not None else torch.empty((T, Nh, top_k), dtype=torch.float32, device=dev)
        counts = counts if counts is not None else torch.empty((Nh, Ne), dtype=torch.int32, device=dev)
    wsp, wsn = _ws(workspace, MHLMOE_OP_LAYER, T, Nh, dh, Ne, top_k, dff, dt)
    _check(load_library().mhlmoe_layer_gelu(
        _dev(X, "X"), _dev(W_router, "W_router", torch.float32, (Nh, Ne, dh)),
        _dev(bias, "bias", torch.float32, (Nh, Ne)),
        _dev(W_in, "W_in", X.dtype, (Nh, Ne, dff, dh)),
        _dev(W_out, "W_out", X.dtype, (Nh, Ne, dh, dff)), T, Nh, dh, Ne, top_k, dff, dt,
        _dev(Y, "Y", X.dtype, (T, Nh, dh)), _dev(idx, "idx", torch.int32, (T, Nh, top_k)),
        _dev(gate, "gate", torch.float32, (T, Nh, top_k)),
        _dev(counts, "counts", torch.int32, (Nh, Ne)), wsp, wsn, _stream(stream)))
    return (Y, idx, gate, counts) if return_routing else Y


def mhlmoe_layer_backward(X, W_router, W1, W3, W2, idx, gate, dY, *, dX=None, dW_router=None,
                          dW1=None, dW3=None, dW2=None, workspace=None, stream=None):
    """Backward of mhlmoe_layer: returns (dX, dW_router, dW1, dW3, dW2)."""
    T, Nh, dh = X.shape
    k = idx.shape[2]
    Ne, dff = W1.shape[1], W1.shape[2]
    dt = _dtype_code(X)
    dev = X.device
    f32 = torch.float32
    dX = dX if dX is not None else torch.empty_like(X)
    dW_router = dW_router if dW_router is not None else torch.empty((Nh, Ne, dh), dtype=f32, device=dev)
    dW1 = dW1 if dW1 is not None else torch.empty((Nh, Ne, dff, dh), dtype=f32, device=dev)
    dW3 = dW3 if dW3 is not None else torch.empty((Nh, Ne, dff, dh), dtype=f32, device=dev)
    dW2 = dW2 if dW2 is not None else torch.empty((Nh, Ne, dh, dff), dtype=f32, device=dev)
    wsp, wsn = _ws(workspace, MHLMOE_OP_LAYER_BACKWARD, T, Nh, dh, Ne, k, dff, dt)
    _check(load_library().mhlmoe_layer_backward(
        _dev(X, "X"), _dev(W_router, "W_router", f32, (Nh, Ne, dh)),
        _dev(W1, "W1", X.dtype, (Nh, Ne, dff, dh)), _dev(W3, "W3", X.dtype, (Nh, Ne, dff, dh)),
        _dev(W2, "W2", X.dtype, (Nh, Ne, dh, dff)), _dev(idx, "idx", torch.int32, (T, Nh, k)),
        _dev(gate, "gate", f32, (T, Nh, k)), _dev(dY, "dY", X.dtype, (T, Nh, dh)),
        T, Nh, dh, Ne, k, dff, dt, _dev(dX, "dX", X.dtype, (T, Nh, dh)),
        _dev(dW_router, "dW_router", f32, (Nh, Ne, dh)), _dev(dW1, "dW1", f32, (Nh, Ne, dff, dh)),
        _dev(dW3, "dW3", f32, (Nh, Ne, dff, dh)), _dev(dW2, "dW2", f32, (Nh, Ne, dh, dff)),
        wsp, wsn, _stream(stream)))
    return dX, dW_router, dW1, dW3, dW2


def mhlmoe_layer_routed(X, R, W_router, bias, W1, W3, W2, top_k, *, Y=None, idx=None,
                        gate=None, counts=None, workspace=None, stream=None,
                        return_routing=True):
    """Separate routing sub-tokens (Sec. 4.4): routes by R, computes the
    experts on X.  W3=None selects the two-matrix GELU expert (W1 = W_in,
    W2 = W_out).  Returns Y, or (Y, idx, gate, counts)."""
    T, Nh, dh = X.shape
    Ne, dff = W1.shape[1], W1.shape[2]
    dt = _dtype_code(X)
    dev = X.device
    Y = Y if Y is not None else torch.empty_like(X)
    if return_routing:
        idx = idx if idx is not None else torch.empty((T, Nh, top_k), dtype=torch.int32, device=dev)
        gate = gate if gate is not None else torch.empty((T, Nh, top_k), dtype=torch.float32, device=dev)
        counts = counts if counts is not None else torch.empty((Nh, Ne), dtype=torch.int32, device=dev)
    wsp, wsn = _ws(workspace, MHLMOE_OP_LAYER, T, Nh, dh, Ne, top_k, dff, dt)
    _check(load_library().mhlmoe_layer_routed(
        _dev(X, "X"), _dev(R, "R", X.dtype, (T, Nh, dh)),
        _dev(W_router, "W_router", torch.float32, (Nh, Ne, dh)),
        _dev(bias, "bias", torch.float32, (Nh, Ne)),
        _dev(W1, "W1", X.dtype, (Nh, Ne, dff, dh)), _dev(W3, "W3", X.dtype, (Nh, Ne, dff, dh)),
        _dev(W2, "W2", X.dtype, (Nh, Ne, dh, dff)), T, Nh, dh, Ne, top_k, dff, dt,
        _dev(Y, "Y", X.dtype, (T, Nh, dh)), _dev(idx, "idx", torch.int32, (T, Nh, top_k)),
        _dev(gate, "gate", torch.float32, (T, Nh, top_k)),
        _dev(counts, "counts", torch.int32, (Nh, Ne)), wsp, wsn, _stream(stream)))
    return (Y, idx, gate, counts) if return_routing else Y


def mhlmoe_layer_backward_routed(X, R, W_router, W1, W3, W2, idx, gate, dY, *, dX=None,
                                 dR=None, dW_router=None, dW1=None, dW3=None, dW2=None,
                                 workspace=None, stream=None):
    """Backward of mhlmoe_layer_routed: returns (dX, dR, dW_router, dW1, dW3, dW2).
    W3=None selects the GELU expert (W1 = W_in, W2 = W_out); dW3 is then None."""
    T, Nh, dh = X.shape
    k = idx.shape[2]
    Ne, dff = W1.shape[1], W1.shape[2]
    dt = _dtype_code(X)
    dev = X.device
    f32 = torch.float32
    dX = dX if dX is not None else torch.empty_like(X)
    dR = dR if dR is not None else torch.empty_like(X)
    dW_router = dW_router if dW_router is not None else torch.empty((Nh, Ne, dh), dtype=f32, device=dev)
    dW1 = dW1 if dW1 is not None else torch.empty((Nh, Ne, dff, dh), dtype=f32, device=dev)
    if W3 is None:
        dW3 = None
    elif dW3 is None:
        dW3 = torch.empty((Nh, Ne, dff, dh), dtype=f32, device=dev)
    dW2 = dW2 if dW2 is not None else torch.empty((Nh, Ne, dh, dff), dtype=f32, device=dev)
    wsp, wsn = _ws(workspace, MHLMOE_OP_LAYER_BACKWARD, T, Nh, dh, Ne, k, dff, dt)
    _check(load_library().mhlmoe_layer_backward_routed(
        _dev(X, "X"), _dev(R, "R", X.dtype, (T, Nh, dh)),
        _dev(W_router, "W_router", f32, (Nh, Ne, dh)),
        _dev(W1, "W1", X.dtype, (Nh, Ne, dff, dh)), _dev(W3, "W3", X.dtype, (Nh, Ne, dff, dh)),
        _dev(W2, "W2", X.dtype, (Nh, Ne, dh, dff)), _dev(idx, "idx", torch.int32, (T, Nh, k)),
        _dev(gate, "gate", f32, (T, Nh, k)), _dev(dY, "dY", X.dtype, (T, Nh, dh)),
        T, Nh, dh, Ne, k, dff, dt, _dev(dX, "dX", X.dtype, (T, Nh, dh)),
        _dev(dR, "dR", X.dtype, (T, Nh, dh)),
        _dev(dW_router, "dW_router", f32, (Nh, Ne, dh)), _dev(dW1, "dW1", f32, (Nh, Ne, dff, dh)),
        _dev(dW3, "dW3", f32, (Nh, Ne, dff, dh)), _dev(dW2, "dW2", f32, (Nh, Ne, dh, dff)),
        wsp, wsn, _stream(stream)))
    return dX, dR, dW_router, dW1, dW3, dW2


def mhlmoe_latent_layer(x, W_in, W_router, bias, W1, W3, W2, W_out, n_heads, top_k, *,
                        routing_tokens=False, out=None, X_lat=None, R_lat=None, Y_lat=None,
                        idx=None, gate=None, counts=None, workspace=None, stream=None):
    """The layer with its projections (Eq. (5)-(6); Eq. (9) with
    routing_tokens).  x [T, d_model]; W_in [(1 + routing_tokens) N, d_model];
    W_out [d_model, N].  Returns a dict with out, X_lat, R_lat (routing
    tokens only), Y_lat, idx, gate, counts."""
    T, d_model = x.shape
    Ne, dff, dh = W1.shape[1], W1.shape[2], W1.shape[3]
    Nh = n_heads
    N = Nh * dh
    rt = 1 if routing_tokens else 0
    dt = _dtype_code(x)
    dev = x.device

    def alloc(t, shape, dtype):
        return t if t is not None else torch.empty(shape, dtype=dtype, device=dev)

    out = alloc(out, (T, d_model), x.dtype)
    X_lat = alloc(X_lat, (T, Nh, dh), x.dtype)
    R_lat = alloc(R_lat, (T, Nh, dh), x.dtype) if rt else R_lat
    Y_lat = alloc(Y_lat, (T, Nh, dh), x.dtype)
    idx = alloc(idx, (T, Nh, top_k), torch.int32)
    gate = alloc(gate, (T, Nh, top_k), torch.float32)
    counts = alloc(counts, (Nh, Ne), torch.int32)
    wsp, wsn = _ws(workspace, MHLMOE_OP_LATENT_LAYER, T, Nh, dh, Ne, top_k, dff, dt)
    _check(load_library().mhlmoe_latent_layer(
        _dev(x, "x"), _dev(W_in, "W_in", x.dtype, ((1 + rt) * N, d_model)),
        _dev(W_router, "W_router", torch.float32, (Nh, Ne, dh)),
        _dev(bias, "bias", torch.float32, (Nh, Ne)),
        _dev(W1, "W1", x.dtype, (Nh, Ne, dff, dh)), _dev(W3, "W3", x.dtype, (Nh, Ne, dff, dh)),
        _dev(W2, "W2", x.dtype, (Nh, Ne, dh, dff)), _dev(W_out, "W_out", x.dtype, (d_model, N)),
        T, d_model, Nh, dh, Ne, top_k, dff, rt, dt, _dev(out, "out", x.dtype, (T, d_model)),
        _dev(X_lat, "X_lat", x.dtype, (T, Nh, dh)),
        _dev(R_lat, "R_lat", x.dtype, (T, Nh, dh)) if rt else None,
        _dev(Y_lat, "Y_lat", x.dtype, (T, Nh, dh)), _dev(idx, "idx", torch.int32, (T, Nh, top_k)),
        _dev(gate, "gate", torch.float32, (T, Nh, top_k)),
        _dev(counts, "counts", torch.int32, (Nh, Ne)), wsp, wsn, _stream(stream)))
    res = {"out": out, "X_lat": X_lat, "Y_lat": Y_lat, "idx": idx, "gate": gate, "counts": counts}
    if rt:
        res["R_lat"] = R_lat
    return res


def mhlmoe_latent_layer_backward(x, W_in, W_router, W1, W3, W2, W_out, X_lat, R_lat, Y_lat, idx,
                                 gate, dout, *, routing_tokens=False, workspace=None,
                                 stream=None):
    """Backward of mhlmoe_latent_layer: returns a dict with dx, dW_in,
    dW_router, dW1, dW3, dW2, dW_out (W3=None: the GELU expert, dW3 None)."""
    T, d_model = x.shape
    Nh, Ne, dff, dh = W1.shape
    k = idx.shape[2]
    N = Nh * dh
    rt = 1 if routing_tokens else 0
    dt = _dtype_code(x)
    dev = x.device
    f32 = torch.float32
    g = {"dx": torch.empty_like(x),
         "dW_in": torch.empty(((1 + rt) * N, d_model), dtype=f32, device=dev),
         "dW_router": torch.empty((Nh, Ne, dh), dtype=f32, device=dev),
         "dW1": torch.empty((Nh, Ne, dff, dh), dtype=f32, device=dev),
         "dW3": None if W3 is None else torch.empty((Nh, Ne, dff, dh), dtype=f32, device=dev),
         "dW2": torch.empty((Nh, Ne, dh, dff), dtype=f32, device=dev),
         "dW_out": torch.empty((d_model, N), dtype=f32, device=dev)}
    wsp, wsn = _ws(workspace, MHLMOE_OP_LATENT_BACKWARD, T, Nh, dh, Ne, k, dff, dt)
    _check(load_library().mhlmoe_latent_layer_backward(
        _dev(x, "x"), _dev(W_in, "W_in", x.dtype, ((1 + rt) * N, d_model)),
        _dev(W_router, "W_router", f32, (Nh, Ne, dh)),
        _dev(W1, "W1", x.dtype, (Nh, Ne, dff, dh)), _dev(W3, "W3", x.dtype, (Nh, Ne, dff, dh)),
        _dev(W2, "W2", x.dtype, (Nh, Ne, dh, dff)), _dev(W_out, "W_out", x.dtype, (d_model, N)),
        _dev(X_lat, "X_lat", x.dtype, (T, Nh, dh)),
        _dev(R_lat, "R_lat", x.dtype, (T, Nh, dh)) if rt else None,
        _dev(Y_lat, "Y_lat", x.dtype, (T, Nh, dh)), _dev(idx, "idx", torch.int32, (T, Nh, k)),
        _dev(gate, "gate", f32, (T, Nh, k)), _dev(dout, "dout", x.dtype, (T, d_model)),
        T, d_model, Nh, dh, Ne, k, dff, rt, dt,
        _dev(g["dx"], "dx"), _dev(g["dW_in"], "dW_in"), _dev(g["dW_router"], "dW_router"),
        _dev(g["dW1"], "dW1"), _dev(g["dW3"], "dW3"), _dev(g["dW2"], "dW2"),
        _dev(g["dW_out"], "dW_out"), wsp, wsn, _stream(stream)))
    return g


def mhlmoe_bias_update(counts, bias, rate: float, *, stream=None):
    """Aux-free load balancing (Sec. 2.2): bias += rate * sign(mean - count),
    per head, in place on the GPU.  Returns bias."""
    Nh, Ne = counts.shape
    _check(load_library().mhlmoe_bias_update(
        _dev(counts, "counts", torch.int32, (Nh, Ne)), _dev(bias, "bias", torch.float32, (Nh, Ne)),
        Nh, Ne, float(rate), _stream(stream)))
    return bias


def mhlmoe_layer_gelu_backward(X, W_router, W_in, W_out, idx, gate, dY, *, dX=None,
                               dW_router=None, dW_in=None, dW_out=None, workspace=None,
                               stream=None):
    """Backward of mhlmoe_layer_gelu: returns (dX, dW_router, dW_in, dW_out)."""
    T, Nh, dh = X.shape
    k = idx.shape[2]
    Ne, dff = W_in.shape[1], W_in.shape[2]
    dt = _dtype_code(X)
    dev = X.device
    f32 = torch.float32
    dX = dX if dX is not None else torch.empty_like(X)
    dW_router = dW_router if dW_router is not None else torch.empty((Nh, Ne, dh), dtype=f32, device=dev)
    dW_in = dW_in if dW_in is not None else torch.empty((Nh, Ne, dff, dh), dtype=f32, device=dev)
    dW_out = dW_out if dW_out is not None else torch.empty((Nh, Ne, dh, dff), dtype=f32, device=dev)
    wsp, wsn = _ws(workspace, MHLMOE_OP_LAYER_BACKWARD, T, Nh, dh, Ne, k, dff, dt)
    _check(load_library().mhlmoe_layer_gelu_backward(
        _dev(X, "X"), _dev(W_router, "W_router", f32, (Nh, Ne, dh)),
        _dev(W_in, "W_in", X.dtype, (Nh, Ne, dff, dh)),
        _dev(W_out, "W_out", X.dtype, (Nh, Ne, dh, dff)), _dev(idx, "idx", torch.int32, (T, Nh, k)),
        _dev(gate, "gate", f32, (T, Nh, k)), _dev(dY, "dY", X.dtype, (T, Nh, dh)),
        T, Nh, dh, Ne, k, dff, dt, _dev(dX, "dX", X.dtype, (T, Nh, dh)),
        _dev(dW_router, "dW_router", f32, (Nh, Ne, dh)),
        _dev(dW_in, "dW_in", f32, (Nh, Ne, dff, dh)), _dev(dW_out, "dW_out", f32, (Nh, Ne, dh, dff)),
        wsp, wsn, _stream(stream)))
    return dX, dW_router, dW_in, dW_out


def mhlmoe_timing_enable(on: bool = True) -> None:
    _check(load_library().mhlmoe_timing_enable(1 if on else 0))


def mhlmoe_timing_query(kernel: str):
    """(total_ms, launches) recorded for `kernel` since the last reset."""
    ms = ctypes.c_double(0.0)
    n = _I64(0)
    _check(load_library().mhlmoe_timing_query(kernel.encode(), ctypes.byref(ms), ctypes.byref(n)))
    return ms.value, n.value


def mhlmoe_timing_reset() -> None:
    _check(load_library().mhlmoe_timing_reset())
