"""Empty batches (T = 0) through every entry point the other GPU tests do not
already take there: outputs with no token rows stay empty, per-expert counts
come back zero and weight gradients come back zero (an empty sum), all
written over sentinel values so that a skipped write shows.
"""
import math

import pytest
import torch

import paper_2602_04870_amd as mh
from tests.gpu_util import announce, needs_gpu

pytestmark = [pytest.mark.gpu, needs_gpu]

NH, DH, NE, K, DFF = 2, 128, 8, 2, 128
BF = torch.bfloat16
F32 = torch.float32


def _rows(*shape, dtype=BF):
    return torch.empty((0, *shape), dtype=dtype, device="cuda")


def _w(*shape, dtype=BF):
    g = torch.Generator(device="cpu").manual_seed(17)
    return (0.05 * torch.randn(*shape, generator=g)).to(dtype).cuda()


def _nan(*shape):
    return torch.full(shape, math.nan, dtype=F32, device="cuda")


def _weights():
    return dict(W_router=_w(NH, NE, DH, dtype=F32), bias=torch.zeros(NH, NE, device="cuda"),
                W1=_w(NH, NE, DFF, DH), W3=_w(NH, NE, DFF, DH), W2=_w(NH, NE, DH, DFF))


def test_route_and_route_backward_empty():
    announce("route / route_backward T = 0")
    w = _weights()
    counts = torch.full((NH, NE), -1, dtype=torch.int32, device="cuda")
    idx, gate, counts = mh.mhlmoe_route(_rows(NH, DH), w["W_router"], w["bias"], K, counts=counts)
    dWr = _nan(NH, NE, DH)
    dX, dWr = mh.mhlmoe_route_backward(_rows(NH, DH), w["W_router"], idx, gate,
                                       _rows(NH, K, dtype=F32), dW_router=dWr)
    torch.cuda.synchronize()
    assert idx.shape == (0, NH, K) and gate.shape == (0, NH, K)
    assert torch.all(counts == 0)
    assert dX.shape == (0, NH, DH) and torch.all(dWr == 0)


@pytest.mark.parametrize("gelu", [False, True], ids=["swiglu", "gelu"])
def test_routed_layer_and_backward_empty(gelu):
    announce(f"layer_routed / backward_routed T = 0 gelu={gelu}")
    w = _weights()
    W3 = None if gelu else w["W3"]
    X, R = _rows(NH, DH), _rows(NH, DH)
    counts = torch.full((NH, NE), -1, dtype=torch.int32, device="cuda")
    Y, idx, gate, counts = mh.mhlmoe_layer_routed(X, R, w["W_router"], w["bias"], w["W1"], W3,
                                                  w["W2"], K, counts=counts)
    grads = dict(dW_router=_nan(NH, NE, DH), dW1=_nan(NH, NE, DFF, DH),
                 dW2=_nan(NH, NE, DH, DFF))
    if not gelu:
        grads["dW3"] = _nan(NH, NE, DFF, DH)
    dX, dR, dWr, dW1, dW3, dW2 = mh.mhlmoe_layer_backward_routed(
        X, R, w["W_router"], w["W1"], W3, w["W2"], idx, gate, _rows(NH, DH), **grads)
    torch.cuda.synchronize()
    assert Y.shape == (0, NH, DH) and torch.all(counts == 0)
    assert dX.shape == (0, NH, DH) and dR.shape == (0, NH, DH)
    for t in (dWr, dW1, dW2) + (() if gelu else (dW3,)):
        assert torch.all(t == 0)
    assert (dW3 is None) == gelu


def test_experts_and_gelu_layer_empty():
    announce("experts / experts_gelu / layer_gelu T = 0")
    w = _weights()
    idx = _rows(NH, K, dtype=torch.int32)
    gate = _rows(NH, K, dtype=F32)
    Y = mh.mhlmoe_experts(_rows(NH, DH), idx, gate, w["W1"], w["W3"], w["W2"])
    Yg = mh.mhlmoe_experts_gelu(_rows(NH, DH), idx, gate, w["W1"], w["W2"])
    counts = torch.full((NH, NE), -1, dtype=torch.int32, device="cuda")
    Yl, _, _, counts = mh.mhlmoe_layer_gelu(_rows(NH, DH), w["W_router"], w["bias"], w["W1"],
                                            w["W2"], K, counts=counts)
    torch.cuda.synchronize()
    assert Y.shape == Yg.shape == Yl.shape == (0, NH, DH)
    assert torch.all(counts == 0)


@pytest.mark.parametrize("routing_tokens", [False, True], ids=["shared", "routing_tokens"])
def test_latent_layer_forward_empty(routing_tokens):
    announce(f"latent_layer T = 0 routing_tokens={routing_tokens}")
    d_model = 96
    w = _weights()
    N = NH * DH
    W_in = _w((2 if routing_tokens else 1) * N, d_model)
    W_out = _w(d_model, N)
    counts = torch.full((NH, NE), -1, dtype=torch.int32, device="cuda")
    res = mh.mhlmoe_latent_layer(_rows(d_model), W_in, w["W_router"], w["bias"], w["W1"],
                                 w["W3"], w["W2"], W_out, NH, K,
                                 routing_tokens=routing_tokens, counts=counts)
    torch.cuda.synchronize()
    assert res["out"].shape == (0, d_model)
    assert res["X_lat"].shape == res["Y_lat"].shape == (0, NH, DH)
    assert torch.all(res["counts"] == 0)
