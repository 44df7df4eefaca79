"""GPU parity of the paper's own expert form (Sec. 3.4): the two-matrix GELU
MLP y = W_out gelu(W_in x), through mhlmoe_experts_gelu / mhlmoe_layer_gelu,
against the CPU oracle (whose GELU expert is pinned by Sec. 3.4's
block-sparse-attention construction in tests/oracle_pins.py).

The GPU runs every workload whole; the oracle checks a seeded sample of token
rows (tokens are independent).  Tolerances as for the SwiGLU path: indices
bit-exact except near ties, gates within 1e-3, outputs within 2e-2 relative
L2 (bf16).
"""
import numpy as np
import pytest
import torch

import paper_2602_04870_amd as mh
import workloads
from tests.gpu_util import (REL_L2, DeviceWorkload, announce, check_routing, needs_gpu,
                            rel_l2, to_device, to_host_f64)

pytestmark = [pytest.mark.gpu, needs_gpu]

GELU = list(workloads.GELU_CONFIGS)


def _workload(name):
    return workloads.generate(workloads.GELU_CONFIGS[name], 0)


@pytest.mark.parametrize("name", GELU)
def test_gelu_layer_parity(name, oracle_instance):
    w = _workload(name)
    s = w.shape
    announce(f"gelu layer {name}")
    d = DeviceWorkload(w)
    Y, idx, gate, counts = mh.mhlmoe_layer_gelu(d.X, d.W_router, d.bias, d.W1, d.W2, s.top_k)
    torch.cuda.synchronize()
    assert torch.all(counts.sum(dim=1) == s.T * s.top_k)
    rows = workloads.sample_rows(s.T, 256)
    Xr = w.exact("X", rows)
    r = oracle_instance.route(Xr, w.exact("W_router"), w.exact("bias"), k=s.top_k)
    ok = check_routing(idx.cpu().numpy()[rows], gate.cpu().numpy()[rows].astype(np.float64),
                       r["idx"], r["gate"], r["keys"], s.top_k, name)
    Yo = oracle_instance.experts_gelu(Xr, r["idx"], r["gate"], w.exact("W1"), w.exact("W2"))
    rows_ok = np.all(ok, axis=1)
    err = rel_l2(to_host_f64(Y)[rows][rows_ok], Yo[rows_ok])
    print(f"[gelu layer] {name} rel-L2 = {err:.3e} over {rows_ok.sum()} rows", flush=True)
    assert err <= REL_L2["bf16"]


@pytest.mark.parametrize("name", GELU)
def test_gelu_experts_parity(name, oracle_instance):
    w = _workload(name)
    s = w.shape
    idx, gate = workloads.random_routing(s.T, s.n_heads, s.n_experts, s.top_k, seed=5)
    announce(f"gelu experts {name}")
    d = DeviceWorkload(w)
    Y = mh.mhlmoe_experts_gelu(d.X, to_device(idx), to_device(gate), d.W1, d.W2)
    torch.cuda.synchronize()
    rows = workloads.sample_rows(s.T, 512)
    Yo = oracle_instance.experts_gelu(w.exact("X", rows), idx[rows],
                                      gate[rows].astype(np.float64), w.exact("W1"),
                                      w.exact("W2"))
    err = rel_l2(to_host_f64(Y)[rows], Yo)
    print(f"[gelu experts] {name} rel-L2 = {err:.3e}", flush=True)
    assert err <= REL_L2["bf16"]


EDGE = [
    # T, Nh, Ne, k, dff, bias  (d_head 128, bf16: the supported GELU shapes)
    (37, 2, 40, 5, 128, "none"),     # ragged T, N_e % 32 != 0, odd k
    (300, 3, 64, 1, 384, "none"),    # k = 1, d_ff = 384 (12 chunks of 32)
    (129, 2, 33, 3, 512, "zipf"),    # just past a token block, d_ff = 512
    (255, 2, 16, 16, 256, "none"),   # k = N_e: dense softmax mixture of GELU MLPs
]


@pytest.mark.parametrize("case", EDGE, ids=lambda c: "T%d_h%d_e%d_k%d_f%d_%s" % c)
def test_gelu_edge_layer(case, oracle_instance):
    T, Nh, Ne, k, dff, bias = case
    shape = workloads.Shape(T, Nh, 128, Ne, k, dff, "bf16", bias=bias, expert="gelu")
    w = workloads.generate(shape, seed=3)
    announce(f"gelu edge {case}")
    d = DeviceWorkload(w)
    Y, idx, gate, _ = mh.mhlmoe_layer_gelu(d.X, d.W_router, d.bias, d.W1, d.W2, k)
    Y2 = mh.mhlmoe_layer_gelu(d.X, d.W_router, d.bias, d.W1, d.W2, k, return_routing=False)
    torch.cuda.synchronize()
    assert torch.equal(Y, Y2), "GELU layer not bitwise reproducible"
    Yo, oi, og, _ = oracle_instance.layer_gelu(w.exact("X"), w.exact("W_router"),
                                               w.exact("bias"), w.exact("W1"), w.exact("W2"), k)
    r = oracle_instance.route(w.exact("X"), w.exact("W_router"), w.exact("bias"), k=k)
    ok = check_routing(idx.cpu().numpy(), gate.cpu().numpy().astype(np.float64), oi, og,
                       r["keys"], k, str(case))
    rows_ok = np.all(ok, axis=1)
    err = rel_l2(to_host_f64(Y)[rows_ok], Yo[rows_ok])
    print(f"[gelu edge] {case} rel-L2 = {err:.3e}", flush=True)
    assert err <= REL_L2["bf16"]


def test_gelu_unsupported_shapes_are_rejected():
    """fp32, d_head 64 and d_ff not a multiple of 128 return EUNSUPPORTED
    before anything is launched."""
    dev = torch.device("cuda", 0)
    for dt, dh, dff in ((torch.float32, 128, 128), (torch.bfloat16, 64, 128),
                        (torch.bfloat16, 128, 96)):
        T, Nh, Ne, k = 8, 2, 4, 2
        X = torch.zeros((T, Nh, dh), dtype=dt, device=dev)
        Wr = torch.zeros((Nh, Ne, dh), dtype=torch.float32, device=dev)
        Wi = torch.zeros((Nh, Ne, dff, dh), dtype=dt, device=dev)
        Wo = torch.zeros((Nh, Ne, dh, dff), dtype=dt, device=dev)
        with pytest.raises(mh.MhlmoeError) as e:
            mh.mhlmoe_layer_gelu(X, Wr, None, Wi, Wo, k)
        assert e.value.status == mh.MHLMOE_EUNSUPPORTED, str(e.value)
