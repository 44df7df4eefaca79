"""GPU parity of separate routing sub-tokens (Sec. 4.4, Eq. (9)): the router
reads r_{t,i}, the experts read x_{t,i}.  Through the C ABI against the CPU
oracle (whose routed backward is pinned by finite differences in X, R and
W_router in tests/oracle_pins.py), plus the identities that hold exactly:
with R = X the forward equals mhlmoe_layer bit for bit, and the expert
weight gradients never depend on R.

Tolerances as elsewhere: indices bit-exact except near ties, gates within
1e-3, outputs and gradients within 2e-2 relative L2 (bf16), 1e-4 (fp32).
"""
import dataclasses

import numpy as np
import pytest
import torch

import paper_2602_04870_amd as mh
import workloads
from tests.gpu_util import (REL_L2, DeviceWorkload, announce, check_expert_blocks, check_routing,
                            check_rows, needs_gpu, rel_l2, to_device, to_host_f64)

pytestmark = [pytest.mark.gpu, needs_gpu]


def _bits(t):
    return t.view(torch.int16) if t.dtype == torch.bfloat16 else t.view(torch.int32)


FWD = [
    # T, Nh, dh, Ne, k, dff, dtype, bias, expert
    (256, 4, 64, 16, 2, 128, "f32", "none", "swiglu"),
    (4096, 8, 128, 64, 4, 128, "bf16", "none", "swiglu"),
    (37, 3, 64, 40, 5, 96, "bf16", "zipf", "swiglu"),      # ragged T, odd k
    (300, 2, 128, 200, 8, 64, "bf16", "zipf", "swiglu"),   # Ne not a multiple of 32
    (129, 2, 128, 33, 3, 256, "bf16", "none", "gelu"),     # the paper's GELU expert
]


@pytest.mark.parametrize("case", FWD, ids=lambda c: "T%d_h%d_d%d_e%d_k%d_f%d_%s_%s_%s" % c)
def test_routed_forward_parity(case, oracle_instance):
    T, Nh, dh, Ne, k, dff, dt, bias, expert = case
    s = workloads.Shape(T, Nh, dh, Ne, k, dff, dt, bias=bias, expert=expert)
    w = workloads.generate(s, 11)
    R = workloads.routing_subtokens(s, 11)
    announce(f"routed forward {case}")
    d = DeviceWorkload(w)
    Rd = to_device(R)
    Y, idx, gate, counts = mh.mhlmoe_layer_routed(d.X, Rd, d.W_router, d.bias, d.W1, d.W3,
                                                  d.W2, k)
    torch.cuda.synchronize()
    assert torch.all(counts.sum(dim=1) == T * k)
    rows = workloads.sample_rows(T, 384)
    Rr = workloads.bf16_bits_to_f64(R[rows]) if R.dtype == np.uint16 else R[rows].astype(np.float64)
    r = oracle_instance.route(Rr, w.exact("W_router"), w.exact("bias"), k=k)
    ok = check_routing(idx.cpu().numpy()[rows], gate.cpu().numpy()[rows].astype(np.float64),
                       r["idx"], r["gate"], r["keys"], k, str(case))
    Xr = w.exact("X", rows)
    if expert == "gelu":
        Yo = oracle_instance.experts_gelu(Xr, r["idx"], r["gate"], w.exact("W1"), w.exact("W2"))
    else:
        Yo = oracle_instance.experts(Xr, r["idx"], r["gate"], w.exact("W1"), w.exact("W3"),
                                     w.exact("W2"))
    rows_ok = np.all(ok, axis=1)
    check_rows(to_host_f64(Y)[rows][rows_ok], Yo[rows_ok], dt, f"routed {case}")


@pytest.mark.parametrize("case", [FWD[0], FWD[1], FWD[4]], ids=lambda c: "%s_%s" % (c[6], c[8]))
def test_routed_with_r_equal_x_is_the_layer(case):
    T, Nh, dh, Ne, k, dff, dt, bias, expert = case
    s = workloads.Shape(T, Nh, dh, Ne, k, dff, dt, bias=bias, expert=expert)
    w = workloads.generate(s, 12)
    announce(f"routed R = X {case}")
    d = DeviceWorkload(w)
    a = mh.mhlmoe_layer_routed(d.X, d.X, d.W_router, d.bias, d.W1, d.W3, d.W2, k)
    if expert == "gelu":
        b = mh.mhlmoe_layer_gelu(d.X, d.W_router, d.bias, d.W1, d.W2, k)
    else:
        b = mh.mhlmoe_layer(d.X, d.W_router, d.bias, d.W1, d.W3, d.W2, k)
    torch.cuda.synchronize()
    for name, x, y in zip(("Y", "idx", "gate", "counts"), a, b):
        assert torch.equal(_bits(x), _bits(y)), name


# ---------------------------------------------------------------------------
# backward
# ---------------------------------------------------------------------------

GRADS = ("dX", "dR", "dW_router", "dW1", "dW3", "dW2")
BWD = [
    # T, Nh, dh, Ne, k, dff, skew
    (256, 4, 128, 16, 2, 128, 0.0),
    (37, 3, 64, 40, 5, 96, 0.0),         # ragged T, odd k
    (513, 2, 64, 1024, 8, 64, 1.1),      # most experts get no slot
    (2048, 8, 128, 1024, 32, 128, 1.1),  # the skewed workload's shape at 2048 tokens
]


def _bwd_inputs(case, seed):
    T, Nh, dh, Ne, k, dff, skew = case
    s = workloads.Shape(T, Nh, dh, Ne, k, dff, "bf16", backward=True)
    w = workloads.generate(s, seed)
    R = workloads.routing_subtokens(s, seed)
    idx, gate = workloads.random_routing(T, Nh, Ne, k, seed=seed + 100, skew=skew)
    return w, R, idx, gate


@pytest.mark.parametrize("case", BWD, ids=lambda c: "T%d_h%d_d%d_e%d_k%d_f%d_s%g" % c)
def test_routed_backward_parity(case, oracle_instance):
    w, R, idx, gate = _bwd_inputs(case, 21)
    announce(f"routed backward {case}")
    d = DeviceWorkload(w)
    Rd, idxd, gated = to_device(R), to_device(idx), to_device(gate)
    got = dict(zip(GRADS, mh.mhlmoe_layer_backward_routed(
        d.X, Rd, d.W_router, d.W1, d.W3, d.W2, idxd, gated, d.dY)))
    shared = mh.mhlmoe_layer_backward(d.X, d.W_router, d.W1, d.W3, d.W2, idxd, gated, d.dY)
    torch.cuda.synchronize()
    # the expert weight gradients do not depend on the router's input
    for name, ref in zip(("dW1", "dW3", "dW2"), shared[2:]):
        assert torch.equal(got[name], ref), name
    want = oracle_instance.layer_backward(w.exact("X"), w.exact("W_router"), w.exact("W1"),
                                          w.exact("W3"), w.exact("W2"), idx, gate, w.exact("dY"),
                                          R=workloads.bf16_bits_to_f64(R))
    T, Nh, dh, Ne, k, dff, skew = case
    counts = np.stack([np.bincount(idx[:, h].ravel(), minlength=Ne) for h in range(Nh)])
    for n in GRADS:
        if n in ("dX", "dR"):
            check_rows(to_host_f64(got[n]), want[n], "bf16", f"routed backward {case} {n}")
        else:
            check_expert_blocks(to_host_f64(got[n]), want[n], counts,
                                f"routed backward {case} {n}")
    empty = torch.from_numpy(counts == 0).cuda()
    assert not torch.any(got["dW_router"][empty] != 0)


def test_routed_backward_with_r_equal_x():
    """R = X: the two input gradients add up to mhlmoe_layer_backward's dX
    (each is rounded to bf16 once, so within bf16 rounding), and every weight
    gradient is bit for bit the same (both paths take dW_router from the
    router's input rows with the same kernels)."""
    case = (1000, 4, 128, 64, 8, 256, 0.5)
    w, _, idx, gate = _bwd_inputs(case, 22)
    announce("routed backward R = X")
    d = DeviceWorkload(w)
    idxd, gated = to_device(idx), to_device(gate)
    dX, dR, dWr, dW1, dW3, dW2 = mh.mhlmoe_layer_backward_routed(
        d.X, d.X, d.W_router, d.W1, d.W3, d.W2, idxd, gated, d.dY)
    rX, rWr, rW1, rW3, rW2 = mh.mhlmoe_layer_backward(d.X, d.W_router, d.W1, d.W3, d.W2, idxd,
                                                      gated, d.dY)
    torch.cuda.synchronize()
    total = dX.double() + dR.double()
    err = float(torch.linalg.vector_norm(total - rX.double()) / torch.linalg.vector_norm(rX.double()))
    assert err <= 1e-2, err
    for a, b in ((dWr, rWr), (dW1, rW1), (dW3, rW3), (dW2, rW2)):
        assert torch.equal(a, b)


def test_routed_backward_is_deterministic_and_checks_aliasing():
    case = (700, 2, 64, 32, 4, 64, 1.1)
    w, R, idx, gate = _bwd_inputs(case, 23)
    s = w.shape
    announce("routed backward determinism")
    d = DeviceWorkload(w)
    Rd, idxd, gated = to_device(R), to_device(idx), to_device(gate)
    ws = mh.workspace(mh.MHLMOE_OP_LAYER_BACKWARD, s.T, s.n_heads, s.d_head, s.n_experts,
                      s.top_k, s.d_ff, mh.MHLMOE_BF16)
    a = mh.mhlmoe_layer_backward_routed(d.X, Rd, d.W_router, d.W1, d.W3, d.W2, idxd, gated,
                                        d.dY, workspace=ws)
    ws.fill_(0x5A)
    b = mh.mhlmoe_layer_backward_routed(d.X, Rd, d.W_router, d.W1, d.W3, d.W2, idxd, gated,
                                        d.dY, workspace=ws)
    torch.cuda.synchronize()
    for x, y in zip(a, b):
        assert torch.equal(_bits(x), _bits(y))
    same = torch.empty_like(d.X)
    with pytest.raises(mh.MhlmoeError) as e:
        mh.mhlmoe_layer_backward_routed(d.X, Rd, d.W_router, d.W1, d.W3, d.W2, idxd, gated,
                                        d.dY, dX=same, dR=same)
    assert e.value.status == mh.MHLMOE_EINVAL


def test_routed_backward_empty_batch():
    announce("routed backward T = 0")
    Nh, dh, Ne, k, dff = 2, 64, 8, 2, 64
    X = torch.empty((0, Nh, dh), dtype=torch.bfloat16, device="cuda")
    Wr = torch.randn(Nh, Ne, dh, device="cuda")
    W1 = torch.randn(Nh, Ne, dff, dh, device="cuda").bfloat16()
    W2 = torch.randn(Nh, Ne, dh, dff, device="cuda").bfloat16()
    idx = torch.empty((0, Nh, k), dtype=torch.int32, device="cuda")
    gate = torch.empty((0, Nh, k), dtype=torch.float32, device="cuda")
    nan = float("nan")
    outs = dict(dW_router=torch.full((Nh, Ne, dh), nan, device="cuda"),
                dW1=torch.full((Nh, Ne, dff, dh), nan, device="cuda"),
                dW3=torch.full((Nh, Ne, dff, dh), nan, device="cuda"),
                dW2=torch.full((Nh, Ne, dh, dff), nan, device="cuda"))
    dX, dR, *grads = mh.mhlmoe_layer_backward_routed(X, X, Wr, W1, W1, W2, idx, gate, X, **outs)
    torch.cuda.synchronize()
    assert dX.shape == dR.shape == (0, Nh, dh)
    for g in grads:
        assert torch.all(g == 0)
