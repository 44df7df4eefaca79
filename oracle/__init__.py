"""CPU oracle for the Multi-Head LatentMoE hot path — TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  The product library never loads it and
shares no code with it.

The arithmetic lives in ``mhlmoe_oracle.c`` (plain C, fp64, router logits
rounded to fp32 because the paper fixes the router at FP32 — Sec. 2.2 and
App. A).  This module compiles it with gcc and wraps it with ctypes, taking
and returning numpy arrays.  The dense projections around the heads
(Eq. (5)-(6), Eq. (9)) are plain fp64 numpy matmuls composed with it here.  Every wrapper validates shapes so that a wrong
call fails here rather than reading out of bounds in C.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
import threading

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
SOURCE = os.path.join(_HERE, "mhlmoe_oracle.c")
LIBRARY = os.path.join(_HERE, "liboracle.so")

_lock = threading.Lock()
_lib = None

_P = ctypes.c_void_p
_I64 = ctypes.c_int64
_I = ctypes.c_int


def compile_library(source: str = SOURCE, output: str = LIBRARY, flags=("-O2",)) -> str:
    """Compile the oracle C source into a shared library (gcc -O2 -fopenmp;
    ``flags`` replaces -O2, e.g. with sanitizer options)."""
    tmp = output + ".tmp%d" % os.getpid()
    cmd = ["gcc", *flags, "-std=c11", "-fPIC", "-shared", "-fopenmp",
           "-Wall", "-Wno-unknown-pragmas", source, "-o", tmp, "-lm"]
    subprocess.run(cmd, check=True, capture_output=True, text=True)
    os.replace(tmp, output)
    return output


def _declare(lib):
    lib.oracle_route.argtypes = [_I64, _I, _I, _I, _I, _P, _P, _P, _P, _P, _P, _P, _P]
    lib.oracle_bucket.argtypes = [_I64, _I, _I, _I, _P, _P, _P]
    lib.oracle_experts.argtypes = [_I64, _I, _I, _I, _I, _I, _P, _P, _P, _P, _P, _P, _P, _P]
    lib.oracle_layer.argtypes = [_I64, _I, _I, _I, _I, _I, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P]
    lib.oracle_layer_backward.argtypes = [_I64, _I, _I, _I, _I, _I] + [_P] * 14
    lib.oracle_experts_gelu.argtypes = [_I64, _I, _I, _I, _I, _I, _P, _P, _P, _P, _P, _P, _P]
    lib.oracle_layer_gelu.argtypes = [_I64, _I, _I, _I, _I, _I] + [_P] * 9
    lib.oracle_layer_backward_routed.argtypes = [_I64, _I, _I, _I, _I, _I] + [_P] * 16
    lib.oracle_layer_gelu_backward.argtypes = [_I64, _I, _I, _I, _I, _I] + [_P] * 12
    lib.oracle_route_backward.argtypes = [_I64, _I, _I, _I, _I] + [_P] * 8
    lib.oracle_bias_update.argtypes = [_I, _I, _P, ctypes.c_float, _P]
    lib.oracle_num_threads.argtypes = []
    for name in ("oracle_route", "oracle_bucket", "oracle_experts",
                 "oracle_layer", "oracle_layer_backward", "oracle_num_threads",
                 "oracle_experts_gelu", "oracle_layer_gelu", "oracle_bias_update",
                 "oracle_layer_backward_routed", "oracle_layer_gelu_backward",
                 "oracle_route_backward"):
        getattr(lib, name).restype = _I
    return lib


def load(path: str | None = None):
    """Load (compiling first if missing or stale) the oracle library."""
    global _lib
    if path is not None:
        return _declare(ctypes.CDLL(path))
    with _lock:
        if _lib is None:
            if (not os.path.exists(LIBRARY)
                    or os.path.getmtime(LIBRARY) < os.path.getmtime(SOURCE)):
                compile_library()
            _lib = _declare(ctypes.CDLL(LIBRARY))
    return _lib


class OracleError(RuntimeError):
    pass


def _f64(a, shape, name):
    a = np.ascontiguousarray(a, dtype=np.float64)
    if a.shape != tuple(shape):
        raise ValueError(f"{name}: expected shape {tuple(shape)}, got {a.shape}")
    return a


def _i32(a, shape, name):
    a = np.ascontiguousarray(a, dtype=np.int32)
    if a.shape != tuple(shape):
        raise ValueError(f"{name}: expected shape {tuple(shape)}, got {a.shape}")
    return a


def _ptr(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def round_bf16(a):
    """Round fp64 values to the nearest bfloat16 (8 significant bits, ties to
    even), returned as fp64.  v = m 2^e with 0.5 <= |m| < 1, so m 2^8 holds
    the 8 kept bits left of the point and rint (ties to even) rounds the rest;
    both steps are exact in fp64.  Finite normal inputs only."""
    m, e = np.frexp(np.asarray(a, dtype=np.float64))
    return np.ldexp(np.rint(m * 256.0) / 256.0, e)


def _check(status, what):
    if status != 0:
        raise OracleError(f"{what} failed with status {status}")


class Oracle:
    """Thin numpy front end over one loaded oracle library."""

    def __init__(self, lib=None):
        self.lib = lib if lib is not None else load()

    def num_threads(self) -> int:
        """Threads the oracle's OpenMP loops use."""
        return int(self.lib.oracle_num_threads())

    def route(self, X, W_router, bias=None, k=1):
        """Eq. (2)-(4) with Algorithm 1's bias.  Returns a dict with
        idx [T,Nh,k] int32, gate [T,Nh,k] f64, counts [Nh,Ne] int32,
        keys [T,Nh,min(k+1,Ne)] f32 (leading biased keys, selection order),
        s_top [T,Nh,k] f32 (unbiased fp32 scores of the selection)."""
        T, Nh, dh = X.shape
        Ne = W_router.shape[1]
        X = _f64(X, (T, Nh, dh), "X")
        W = _f64(W_router, (Nh, Ne, dh), "W_router")
        b = None if bias is None else _f64(bias, (Nh, Ne), "bias")
        if not 1 <= k <= Ne:
            raise ValueError("need 1 <= k <= Ne")
        nk = min(k + 1, Ne)
        idx = np.empty((T, Nh, k), np.int32)
        gate = np.empty((T, Nh, k), np.float64)
        counts = np.empty((Nh, Ne), np.int32)
        keys = np.empty((T, Nh, nk), np.float32)
        s_top = np.empty((T, Nh, k), np.float32)
        _check(self.lib.oracle_route(T, Nh, dh, Ne, k, _ptr(X), _ptr(W), _ptr(b),
                                     _ptr(idx), _ptr(gate), _ptr(counts),
                                     _ptr(keys), _ptr(s_top)), "oracle_route")
        return {"idx": idx, "gate": gate, "counts": counts, "keys": keys,
                "s_top": s_top}

    def route_backward(self, X, W_router, idx, gate, dgate, return_dS=False):
        """Algorithm 2: given the gate gradient dgate [T,Nh,k], returns a dict
        with dX [T,Nh,dh] and dW_router [Nh,Ne,dh] (f64), optionally dS."""
        T, Nh, dh = X.shape
        Ne = W_router.shape[1]
        k = idx.shape[2]
        X = _f64(X, (T, Nh, dh), "X")
        W = _f64(W_router, (Nh, Ne, dh), "W_router")
        idx = _i32(idx, (T, Nh, k), "idx")
        gate = _f64(gate, (T, Nh, k), "gate")
        dgate = _f64(dgate, (T, Nh, k), "dgate")
        out = {"dX": np.empty((T, Nh, dh)), "dW_router": np.empty((Nh, Ne, dh))}
        dS = np.empty((T, Nh, k)) if return_dS else None
        _check(self.lib.oracle_route_backward(T, Nh, dh, Ne, k, _ptr(X), _ptr(W), _ptr(idx),
                                              _ptr(gate), _ptr(dgate), _ptr(out["dX"]),
                                              _ptr(out["dW_router"]), _ptr(dS)),
               "oracle_route_backward")
        if return_dS:
            out["dS"] = dS
        return out

    def bucket(self, idx, Ne):
        """Token clustering (Sec. 3.4): offsets [Nh,Ne+1], perm [Nh,T*k]."""
        T, Nh, k = idx.shape
        idx = _i32(idx, (T, Nh, k), "idx")
        offsets = np.empty((Nh, Ne + 1), np.int32)
        perm = np.empty((Nh, T * k), np.int32)
        _check(self.lib.oracle_bucket(T, Nh, Ne, k, _ptr(idx), _ptr(offsets),
                                      _ptr(perm)), "oracle_bucket")
        return offsets, perm

    def experts(self, X, idx, gate, W1, W3, W2, return_slots=False):
        """Eq. (1) with SwiGLU experts.  Returns Y [T,Nh,dh] f64 (and the
        unscaled per-slot outputs [T,Nh,k,dh] when return_slots)."""
        T, Nh, dh = X.shape
        k = idx.shape[2]
        Ne, dff = W1.shape[1], W1.shape[2]
        X = _f64(X, (T, Nh, dh), "X")
        idx = _i32(idx, (T, Nh, k), "idx")
        gate = _f64(gate, (T, Nh, k), "gate")
        W1 = _f64(W1, (Nh, Ne, dff, dh), "W1")
        W3 = _f64(W3, (Nh, Ne, dff, dh), "W3")
        W2 = _f64(W2, (Nh, Ne, dh, dff), "W2")
        Y = np.empty((T, Nh, dh), np.float64)
        ys = np.empty((T, Nh, k, dh), np.float64) if return_slots else None
        _check(self.lib.oracle_experts(T, Nh, dh, Ne, k, dff, _ptr(X), _ptr(idx),
                                       _ptr(gate), _ptr(W1), _ptr(W3), _ptr(W2),
                                       _ptr(Y), _ptr(ys)), "oracle_experts")
        return (Y, ys) if return_slots else Y

    def experts_gelu(self, X, idx, gate, W_in, W_out, return_slots=False):
        """Eq. (1) with the two-matrix GELU expert of Sec. 3.4,
        y = W_out gelu(W_in x).  Returns Y [T,Nh,dh] f64 (and the unscaled
        per-slot outputs when return_slots)."""
        T, Nh, dh = X.shape
        k = idx.shape[2]
        Ne, dff = W_in.shape[1], W_in.shape[2]
        X = _f64(X, (T, Nh, dh), "X")
        idx = _i32(idx, (T, Nh, k), "idx")
        gate = _f64(gate, (T, Nh, k), "gate")
        Wi = _f64(W_in, (Nh, Ne, dff, dh), "W_in")
        Wo = _f64(W_out, (Nh, Ne, dh, dff), "W_out")
        Y = np.empty((T, Nh, dh), np.float64)
        ys = np.empty((T, Nh, k, dh), np.float64) if return_slots else None
        _check(self.lib.oracle_experts_gelu(T, Nh, dh, Ne, k, dff, _ptr(X), _ptr(idx),
                                            _ptr(gate), _ptr(Wi), _ptr(Wo), _ptr(Y),
                                            _ptr(ys)), "oracle_experts_gelu")
        return (Y, ys) if return_slots else Y

    def layer_gelu(self, X, W_router, bias, W_in, W_out, k):
        """Routing then the GELU experts; returns (Y, idx, gate, counts)."""
        T, Nh, dh = X.shape
        Ne, dff = W_in.shape[1], W_in.shape[2]
        X = _f64(X, (T, Nh, dh), "X")
        W = _f64(W_router, (Nh, Ne, dh), "W_router")
        b = None if bias is None else _f64(bias, (Nh, Ne), "bias")
        Wi = _f64(W_in, (Nh, Ne, dff, dh), "W_in")
        Wo = _f64(W_out, (Nh, Ne, dh, dff), "W_out")
        Y = np.empty((T, Nh, dh), np.float64)
        idx = np.empty((T, Nh, k), np.int32)
        gate = np.empty((T, Nh, k), np.float64)
        counts = np.empty((Nh, Ne), np.int32)
        _check(self.lib.oracle_layer_gelu(T, Nh, dh, Ne, k, dff, _ptr(X), _ptr(W), _ptr(b),
                                          _ptr(Wi), _ptr(Wo), _ptr(Y), _ptr(idx), _ptr(gate),
                                          _ptr(counts)), "oracle_layer_gelu")
        return Y, idx, gate, counts

    def bias_update(self, counts, bias, rate):
        """Aux-free load balancing (Sec. 2.2): returns the updated fp32 bias
        b + rate * sign(mean load - load), per head."""
        Nh, Ne = counts.shape
        c = _i32(counts, (Nh, Ne), "counts")
        b = np.array(bias, dtype=np.float32, copy=True).reshape(Nh, Ne)
        _check(self.lib.oracle_bias_update(Nh, Ne, _ptr(c), float(rate), _ptr(b)),
               "oracle_bias_update")
        return b

    def layer(self, X, W_router, bias, W1, W3, W2, k):
        """Routing then experts; returns (Y, idx, gate, counts)."""
        T, Nh, dh = X.shape
        Ne, dff = W1.shape[1], W1.shape[2]
        X = _f64(X, (T, Nh, dh), "X")
        W = _f64(W_router, (Nh, Ne, dh), "W_router")
        b = None if bias is None else _f64(bias, (Nh, Ne), "bias")
        W1 = _f64(W1, (Nh, Ne, dff, dh), "W1")
        W3 = _f64(W3, (Nh, Ne, dff, dh), "W3")
        W2 = _f64(W2, (Nh, Ne, dh, dff), "W2")
        Y = np.empty((T, Nh, dh), np.float64)
        idx = np.empty((T, Nh, k), np.int32)
        gate = np.empty((T, Nh, k), np.float64)
        counts = np.empty((Nh, Ne), np.int32)
        _check(self.lib.oracle_layer(T, Nh, dh, Ne, k, dff, _ptr(X), _ptr(W), _ptr(b),
                                     _ptr(W1), _ptr(W3), _ptr(W2), _ptr(Y),
                                     _ptr(idx), _ptr(gate), _ptr(counts)),
               "oracle_layer")
        return Y, idx, gate, counts

    def layer_routed(self, X, R, W_router, bias, W1, W3, W2, k):
        """Separate routing sub-tokens (Sec. 4.4, Eq. (9)): the router reads
        R [T,Nh,dh], the experts read X.  Returns (Y, idx, gate, counts)."""
        r = self.route(R, W_router, bias, k=k)
        Y = self.experts(X, r["idx"], r["gate"], W1, W3, W2)
        return Y, r["idx"], r["gate"], r["counts"]

    def latent_layer(self, x, W_in, W_router, bias, W1, W3, W2, W_out, n_heads, k,
                     routing_tokens=False, latent_round=None):
        """The layer with its projections (Eq. (5)-(6), Sec. 3.1):
        X_lat = split(W_in x) into n_heads sub-tokens of d_h, the per-head
        MoEs, out = W_out concat(Y_lat).  With routing_tokens W_in has 2N
        rows (Eq. (9), Sec. 4.4) and its last N produce the routing
        sub-tokens.  W3=None selects the two-matrix GELU expert.
        latent_round="bf16" rounds the sub-tokens to bfloat16 before the
        heads: the precision in which a bf16 implementation holds them, and
        so takes its routing decision.  Returns a dict with out, X_lat,
        R_lat, Y_lat (f64), idx, gate, counts."""
        x = np.asarray(x, dtype=np.float64)
        T = x.shape[0]
        dh = W_router.shape[2]
        N = n_heads * dh
        W_in = np.asarray(W_in, dtype=np.float64)
        W_out = np.asarray(W_out, dtype=np.float64)
        if W_in.shape != ((2 if routing_tokens else 1) * N, x.shape[1]):
            raise ValueError(f"W_in: unexpected shape {W_in.shape}")
        lat = x @ W_in.T
        if latent_round == "bf16":
            lat = round_bf16(lat)
        elif latent_round is not None:
            raise ValueError(f"unknown latent_round {latent_round!r}")
        X_lat = lat[:, :N].reshape(T, n_heads, dh)
        R_lat = lat[:, N:].reshape(T, n_heads, dh) if routing_tokens else X_lat
        r = self.route(R_lat, W_router, bias, k=k)
        if W3 is None:
            Y_lat = self.experts_gelu(X_lat, r["idx"], r["gate"], W1, W2)
        else:
            Y_lat = self.experts(X_lat, r["idx"], r["gate"], W1, W3, W2)
        out = Y_lat.reshape(T, N) @ W_out.T
        return {"out": out, "X_lat": X_lat, "R_lat": R_lat if routing_tokens else None,
                "Y_lat": Y_lat, "idx": r["idx"], "gate": r["gate"], "counts": r["counts"],
                "keys": r["keys"]}

    def latent_layer_backward(self, x, W_in, W_router, W1, W3, W2, W_out, X_lat, R_lat, Y_lat,
                              idx, gate, dout, routing_tokens=False):
        """Backward of latent_layer (SwiGLU experts) at the given saved
        activations: dY_lat = dout W_out, dW_out = dout^T Y_lat, the heads'
        backward (router gradients against R_lat with routing_tokens), then
        dW_in = [dX_lat; dR_lat]^T x and dx = dX_lat W_in_x (+ dR_lat W_in_r).
        Returns a dict with dx, dW_in, dW_router, dW1, dW3, dW2, dW_out."""
        x = np.asarray(x, dtype=np.float64)
        T = x.shape[0]
        Nh, _, _, dh = np.shape(W1)
        N = Nh * dh
        W_in = np.asarray(W_in, dtype=np.float64)
        W_out = np.asarray(W_out, dtype=np.float64)
        dout = np.asarray(dout, dtype=np.float64)
        Yl = np.asarray(Y_lat, dtype=np.float64).reshape(T, N)
        dY = (dout @ W_out).reshape(T, Nh, dh)
        g = self.layer_backward(X_lat, W_router, W1, W3, W2, idx, gate, dY,
                                R=R_lat if routing_tokens else None)
        dXl = g["dX"].reshape(T, N)
        dW_in = dXl.T @ x
        dx = dXl @ W_in[:N]
        if routing_tokens:
            dRl = g["dR"].reshape(T, N)
            dW_in = np.concatenate([dW_in, dRl.T @ x])
            dx = dx + dRl @ W_in[N:]
        return {"dx": dx, "dW_in": dW_in, "dW_router": g["dW_router"], "dW1": g["dW1"],
                "dW3": g.get("dW3"), "dW2": g["dW2"], "dW_out": dout.T @ Yl}

    def layer_backward(self, X, W_router, W1, W3, W2, idx, gate, dY,
                       return_dS=False, R=None):
        """Algorithm 2 plus the expert backward.  Returns a dict with
        dX, dW_router, dW1, dW3, dW2 (f64) and optionally dS.  With R (the
        routing sub-tokens of Sec. 4.4) the router input gradient is returned
        as dR, dW_router is taken against R, and dX holds the expert terms
        only.  W3=None selects the two-matrix GELU expert (W1 = W_in,
        W2 = W_out; no dW3 in the result)."""
        T, Nh, dh = X.shape
        k = idx.shape[2]
        Ne, dff = W1.shape[1], W1.shape[2]
        if W3 is None:
            if R is not None:
                raise ValueError("routing sub-tokens with the GELU expert are not wrapped")
            X = _f64(X, (T, Nh, dh), "X")
            W = _f64(W_router, (Nh, Ne, dh), "W_router")
            Wi = _f64(W1, (Nh, Ne, dff, dh), "W_in")
            Wo = _f64(W2, (Nh, Ne, dh, dff), "W_out")
            idx = _i32(idx, (T, Nh, k), "idx")
            gate = _f64(gate, (T, Nh, k), "gate")
            dY = _f64(dY, (T, Nh, dh), "dY")
            out = {"dX": np.empty((T, Nh, dh)), "dW_router": np.empty((Nh, Ne, dh)),
                   "dW1": np.empty((Nh, Ne, dff, dh)), "dW2": np.empty((Nh, Ne, dh, dff))}
            dS = np.empty((T, Nh, k), np.float64) if return_dS else None
            _check(self.lib.oracle_layer_gelu_backward(
                T, Nh, dh, Ne, k, dff, _ptr(X), _ptr(W), _ptr(Wi), _ptr(Wo), _ptr(idx),
                _ptr(gate), _ptr(dY), _ptr(out["dX"]), _ptr(out["dW_router"]),
                _ptr(out["dW1"]), _ptr(out["dW2"]), _ptr(dS)), "oracle_layer_gelu_backward")
            if return_dS:
                out["dS"] = dS
            return out
        X = _f64(X, (T, Nh, dh), "X")
        W = _f64(W_router, (Nh, Ne, dh), "W_router")
        W1 = _f64(W1, (Nh, Ne, dff, dh), "W1")
        W3 = _f64(W3, (Nh, Ne, dff, dh), "W3")
        W2 = _f64(W2, (Nh, Ne, dh, dff), "W2")
        idx = _i32(idx, (T, Nh, k), "idx")
        gate = _f64(gate, (T, Nh, k), "gate")
        dY = _f64(dY, (T, Nh, dh), "dY")
        out = {
            "dX": np.empty((T, Nh, dh), np.float64),
            "dW_router": np.empty((Nh, Ne, dh), np.float64),
            "dW1": np.empty((Nh, Ne, dff, dh), np.float64),
            "dW3": np.empty((Nh, Ne, dff, dh), np.float64),
            "dW2": np.empty((Nh, Ne, dh, dff), np.float64),
        }
        dS = np.empty((T, Nh, k), np.float64) if return_dS else None
        if R is not None:
            R = _f64(R, (T, Nh, dh), "R")
            out["dR"] = np.empty((T, Nh, dh), np.float64)
            _check(self.lib.oracle_layer_backward_routed(
                T, Nh, dh, Ne, k, dff, _ptr(X), _ptr(R), _ptr(W), _ptr(W1), _ptr(W3),
                _ptr(W2), _ptr(idx), _ptr(gate), _ptr(dY), _ptr(out["dX"]), _ptr(out["dR"]),
                _ptr(out["dW_router"]), _ptr(out["dW1"]), _ptr(out["dW3"]), _ptr(out["dW2"]),
                _ptr(dS)), "oracle_layer_backward_routed")
            if return_dS:
                out["dS"] = dS
            return out
        _check(self.lib.oracle_layer_backward(
            T, Nh, dh, Ne, k, dff, _ptr(X), _ptr(W), _ptr(W1), _ptr(W3), _ptr(W2),
            _ptr(idx), _ptr(gate), _ptr(dY), _ptr(out["dX"]), _ptr(out["dW_router"]),
            _ptr(out["dW1"]), _ptr(out["dW3"]), _ptr(out["dW2"]), _ptr(dS)),
            "oracle_layer_backward")
        if return_dS:
            out["dS"] = dS
        return out
