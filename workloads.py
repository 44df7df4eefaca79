"""Seeded synthetic workloads for the Multi-Head LatentMoE hot path.

This module only draws inputs.  It holds none of the method's arithmetic, so
both the CPU oracle (tests) and the HIP library (tests, benchmark) can be fed
from it without sharing any computation.

Recipe (the same for every configuration):
  * numpy ``default_rng(seed)``, draws in the fixed order
    X, W_router, [per-head expert rank permutations], W1, [W3], W2, [dY]
    (W3 only for the SwiGLU expert; the two-matrix GELU expert of Sec. 3.4
    uses W1 as W_in and W2 as W_out);
  * X ~ N(0, 1); W_router, W1, W3 ~ N(0, 1/d_h); W2 ~ N(0, 1/d_ff)
    (variance 1/fan_in); dY ~ N(0, 1);
  * bf16 configurations round X, W1, W3, W2 and dY from fp32 to bf16 with
    round-to-nearest-even; W_router and the bias stay fp32 (the paper's router
    runs in FP32);
  * the skewed configuration adds a per-head Zipf load-balancing bias
    b[h, e] = -s * ln(1 + rank_h(e)) with s = 1.1 and rank_h a seeded
    permutation of the experts.  Used as the bias that only steers selection,
    it weights expert of rank r (1-based) by r^-s, the Zipf law the paper uses
    for its skew experiment (Fig. 3 caption: skew 1 and 2 put 80.8% and 99.8%
    of the load on the first of four expert shards when 768 experts are
    split contiguously).

The paper trains on FineWebEdu with learned routers; those inputs are not
available, and these Gaussian inputs plus the Zipf bias stand in for them.
"""
from __future__ import annotations

import dataclasses
from typing import Optional

import numpy as np


@dataclasses.dataclass(frozen=True)
class Shape:
    T: int
    n_heads: int
    d_head: int
    n_experts: int
    top_k: int
    d_ff: int
    dtype: str = "bf16"          # "f32" or "bf16": X, W1, W3, W2, Y, dY
    bias: str = "none"           # "none" or "zipf"
    zipf_s: float = 1.1
    backward: bool = False
    expert: str = "swiglu"       # "swiglu" (W1, W3, W2) or "gelu" (W_in = W1, W_out = W2)

    @property
    def slots(self) -> int:
        return self.T * self.n_heads * self.top_k

    def with_T(self, T: int) -> "Shape":
        return dataclasses.replace(self, T=T)


# The five workloads of the hot-path contract (seed 0 for all).
CONFIGS = {
    "tiny_f32_t256": Shape(256, 4, 64, 16, 2, 128, "f32"),
    "bf16_t4096_e64": Shape(4096, 8, 128, 64, 8, 256, "bf16"),
    "headline_bf16_t16384_e128": Shape(16384, 16, 128, 128, 8, 256, "bf16"),
    "granular_bf16_t16384_e256": Shape(16384, 16, 128, 256, 16, 128, "bf16"),
    "skewed_bf16_t65536_e1024": Shape(65536, 8, 128, 1024, 32, 128, "bf16",
                              bias="zipf", zipf_s=1.1, backward=True),
}
CONFIG_ORDER = list(CONFIGS)

# The paper's own expert form (Sec. 3.4, two-matrix GELU) at its MH LatentMoE
# layer shapes (N_h 8, d_h 128; 384 experts, k 4, expert hidden 256 for the
# 0.2B-2.2B model, and its finer-grained 768-expert, k 8, hidden 128 variant),
# four 2048-token sequences per batch.
GELU_CONFIGS = {
    "gelu_bf16_t8192_e384": Shape(8192, 8, 128, 384, 4, 256, "bf16", expert="gelu"),
    "gelu_bf16_t8192_e768": Shape(8192, 8, 128, 768, 8, 128, "bf16", expert="gelu"),
}
ALL_CONFIGS = {**CONFIGS, **GELU_CONFIGS}


# ---------------------------------------------------------------------------
# bf16 storage helpers (input preparation only)
# ---------------------------------------------------------------------------

def f32_to_bf16_bits(a: np.ndarray) -> np.ndarray:
    """Round fp32 to bf16 (round to nearest, ties to even); returns uint16."""
    u = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32)
    lsb = (u >> np.uint32(16)) & np.uint32(1)
    r = (u + np.uint32(0x7FFF) + lsb) >> np.uint32(16)
    return r.astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (np.ascontiguousarray(b, dtype=np.uint16).astype(np.uint32)
            << np.uint32(16)).view(np.float32)


def bf16_bits_to_f64(b: np.ndarray) -> np.ndarray:
    return bf16_bits_to_f32(b).astype(np.float64)


@dataclasses.dataclass
class Workload:
    """Host copies of one workload's inputs.

    ``X``, ``W1``, ``W3``, ``W2`` and ``dY`` are stored in the configuration's
    dtype: float32 arrays for "f32", uint16 bf16 bit patterns for "bf16".
    ``W_router`` and ``bias`` are float32.  ``exact(name)`` returns the exact
    float64 value of any of them (bf16 and fp32 values are exact in fp64).
    """
    shape: Shape
    seed: int
    X: np.ndarray
    W_router: np.ndarray
    bias: Optional[np.ndarray]
    W1: np.ndarray
    W3: Optional[np.ndarray]
    W2: np.ndarray
    dY: Optional[np.ndarray] = None

    def exact(self, name: str, index=None) -> np.ndarray:
        a = getattr(self, name)
        if a is None:
            return None
        if index is not None:
            a = a[index]
        if a.dtype == np.uint16:
            return bf16_bits_to_f64(a)
        return np.asarray(a, dtype=np.float64)


def _normal(rng, shape, std, dtype_name):
    a = rng.standard_normal(size=shape, dtype=np.float32)
    if std != 1.0:
        a *= np.float32(std)
    if dtype_name == "bf16":
        return f32_to_bf16_bits(a)
    return a


def zipf_bias(rng, n_heads: int, n_experts: int, s: float) -> np.ndarray:
    """b[h, e] = -s * ln(1 + rank_h(e)) with a seeded rank permutation."""
    b = np.empty((n_heads, n_experts), np.float32)
    for h in range(n_heads):
        rank = rng.permutation(n_experts)
        b[h] = (-s * np.log1p(rank.astype(np.float64))).astype(np.float32)
    return b


def generate(shape: Shape, seed: int = 0) -> Workload:
    """Draw one workload in the fixed order described in the module doc."""
    rng = np.random.default_rng(seed)
    T, Nh, dh, Ne, dff = shape.T, shape.n_heads, shape.d_head, shape.n_experts, shape.d_ff
    X = _normal(rng, (T, Nh, dh), 1.0, shape.dtype)
    W_router = rng.standard_normal(size=(Nh, Ne, dh), dtype=np.float32)
    W_router *= np.float32(1.0 / np.sqrt(dh))
    bias = None
    if shape.bias == "zipf":
        bias = zipf_bias(rng, Nh, Ne, shape.zipf_s)
    elif shape.bias != "none":
        raise ValueError(f"unknown bias kind {shape.bias!r}")
    if shape.expert not in ("swiglu", "gelu"):
        raise ValueError(f"unknown expert kind {shape.expert!r}")
    W1 = _normal(rng, (Nh, Ne, dff, dh), 1.0 / np.sqrt(dh), shape.dtype)
    W3 = (_normal(rng, (Nh, Ne, dff, dh), 1.0 / np.sqrt(dh), shape.dtype)
          if shape.expert == "swiglu" else None)
    W2 = _normal(rng, (Nh, Ne, dh, dff), 1.0 / np.sqrt(dff), shape.dtype)
    dY = _normal(rng, (T, Nh, dh), 1.0, shape.dtype) if shape.backward else None
    return Workload(shape, seed, X, W_router, bias, W1, W3, W2, dY)


def routing_subtokens(shape: Shape, seed: int = 0) -> np.ndarray:
    """Separate routing sub-tokens r_{t,i} (Sec. 4.4, Eq. (9)) for the
    workload drawn with ``generate(shape, seed)``: [T, N_h, d_h], drawn like X
    (N(0, 1), the configuration's dtype) from a stream of their own, so the
    workload's other inputs are unchanged."""
    rng = np.random.default_rng([seed, 94])
    return _normal(rng, (shape.T, shape.n_heads, shape.d_head), 1.0, shape.dtype)


def latent_inputs(shape: Shape, d_model: int, routing_tokens: bool = False, seed: int = 0):
    """Inputs of the layer with its projections (Eq. (5)-(6), Eq. (9)) around
    the per-head weights of ``generate(shape, seed)``, from a stream of their
    own: x [T, d_model] ~ N(0, 1); W_in [(1 + routing_tokens) N, d_model] ~
    N(0, 1/d_model); W_out [d_model, N] ~ N(0, 1/N) (N = N_h d_h), in the
    configuration's dtype.  With ``shape.backward`` also dout [T, d_model] ~
    N(0, 1) and stand-ins for the saved activations X_lat, R_lat, Y_lat
    [T, N_h, d_h] ~ N(0, 1) (so the backward can be checked on its own)."""
    rng = np.random.default_rng([seed, 95])
    T, N = shape.T, shape.n_heads * shape.d_head
    lat = (shape.T, shape.n_heads, shape.d_head)
    rows = (2 if routing_tokens else 1) * N
    out = {"x": _normal(rng, (T, d_model), 1.0, shape.dtype),
           "W_in": _normal(rng, (rows, d_model), 1.0 / np.sqrt(d_model), shape.dtype),
           "W_out": _normal(rng, (d_model, N), 1.0 / np.sqrt(N), shape.dtype)}
    if shape.backward:
        out["dout"] = _normal(rng, (T, d_model), 1.0, shape.dtype)
        out["X_lat"] = _normal(rng, lat, 1.0, shape.dtype)
        out["R_lat"] = _normal(rng, lat, 1.0, shape.dtype) if routing_tokens else None
        out["Y_lat"] = _normal(rng, lat, 1.0, shape.dtype)
    return out


def random_counts(n_heads: int, n_experts: int, seed: int, total: int = 4096) -> np.ndarray:
    """Per-head expert loads [n_heads, n_experts] int32 covering the cases the
    bias update distinguishes: head 0 perfectly balanced (when n_experts
    divides total), head 1 all on one expert, head 2 all zero, the rest
    multinomial draws of ``total`` slots with a random per-head skew."""
    rng = np.random.default_rng(seed)
    c = np.empty((n_heads, n_experts), np.int64)
    for h in range(n_heads):
        if h == 0 and total % n_experts == 0:
            c[h] = total // n_experts
        elif h == 1:
            c[h] = 0
            c[h, rng.integers(n_experts)] = total
        elif h == 2:
            c[h] = 0
        else:
            w = rng.random(n_experts) ** rng.uniform(0.0, 4.0)
            c[h] = rng.multinomial(total, w / w.sum())
    return c.astype(np.int32)


def sample_rows(T: int, n: int, seed: int = 1234) -> np.ndarray:
    """A sorted, seeded sample of token rows that always includes the first
    and last token (the ragged tail of any tiling)."""
    if n >= T:
        return np.arange(T)
    rng = np.random.default_rng(seed)
    rows = rng.choice(T, size=n, replace=False)
    rows[0], rows[-1] = 0, T - 1
    return np.unique(rows)


def random_routing(T: int, n_heads: int, n_experts: int, top_k: int, seed: int = 7,
                   skew: float = 0.0):
    """Arbitrary valid routing input for the expert step alone: k distinct
    experts per (token, head), drawn with probability proportional to
    rank^-skew over a seeded per-head expert ranking, and positive gates that
    sum to one.  Returns (idx int32 [T,Nh,k], gate float32 [T,Nh,k])."""
    rng = np.random.default_rng(seed)
    idx = np.empty((T, n_heads, top_k), np.int32)
    for h in range(n_heads):
        order = rng.permutation(n_experts)
        w = np.arange(1, n_experts + 1, dtype=np.float64) ** -skew
        # Gumbel top-k: k distinct draws without replacement, weights w
        g = rng.gumbel(size=(T, n_experts)) + np.log(w)[None, :]
        pick = np.argpartition(-g, top_k - 1, axis=1)[:, :top_k]
        idx[:, h, :] = order[pick]
    gate = rng.random((T, n_heads, top_k)).astype(np.float64) + 0.05
    gate /= gate.sum(-1, keepdims=True)
    return idx, gate.astype(np.float32)


def to_device(a: np.ndarray, device="cuda"):
    """Upload one host array to the GPU as a torch tensor (uint16 bf16 bit
    patterns become torch.bfloat16)."""
    import torch
    if a is None:
        return None
    if a.dtype == np.uint16:
        t = torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16)
    else:
        t = torch.from_numpy(np.ascontiguousarray(a))
    return t.to(device)
