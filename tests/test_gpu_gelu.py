"""GPU parity of the paper's own expert form (Sec. 3.4): the two-matrix GELU
MLP y = W_out gelu(W_in x), through mhlmoe_experts_gelu / mhlmoe_layer_gelu,
against the CPU oracle (whose GELU expert is pinned by Sec. 3.4's
block-sparse-attention construction in tests/oracle_pins.py).

The GPU runs every workload whole; the oracle checks a seeded sample of token
rows (tokens are independent).  Tolerances as for the SwiGLU path: indices
bit-exact except near ties, gates within 1e-3, outputs within 2e-2 relative
L2 (bf16), pooled, and every (token, head) row within 5e-2 of its own norm
(every (head, expert) block of a weight gradient likewise).
"""
import numpy as np
import pytest
import torch

import paper_2602_04870_amd as mh
import workloads
from tests.gpu_util import (REL_L2, DeviceWorkload, announce, check_expert_blocks, check_routing,
                            check_rows, needs_gpu, rel_l2, to_device, to_host_f64)

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
    check_rows(to_host_f64(Y)[rows][rows_ok], Yo[rows_ok], "bf16", f"gelu layer {name}")


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
    check_rows(to_host_f64(Y)[rows], Yo, "bf16", f"gelu experts {name}")


@pytest.mark.parametrize("dff", [128, 256, 384, 512])
def test_gelu_experts_many_tiles_per_workgroup(dff, oracle_instance):
    """4096 tokens x 8 heads x k 8 over 64 experts: 512 slots per (head,
    expert), 2048 tiles of 128 slots for the kernel's 512 workgroups, so every
    workgroup walks four tiles and its weight ring wraps across tile
    boundaries (d_ff 128-512: 4-16 chunks of 32 per tile)."""
    shape = workloads.Shape(4096, 8, 128, 64, 8, dff, "bf16", expert="gelu")
    w = workloads.generate(shape, seed=11)
    idx, gate = workloads.random_routing(shape.T, shape.n_heads, shape.n_experts, shape.top_k,
                                         seed=13)
    announce(f"gelu experts many tiles d_ff {dff}")
    d = DeviceWorkload(w)
    Y = mh.mhlmoe_experts_gelu(d.X, to_device(idx), to_device(gate), d.W1, d.W2)
    Y2 = mh.mhlmoe_experts_gelu(d.X, to_device(idx), to_device(gate), d.W1, d.W2)
    torch.cuda.synchronize()
    assert torch.equal(Y, Y2), "GELU experts not bitwise reproducible"
    rows = workloads.sample_rows(shape.T, 192)
    Yo = oracle_instance.experts_gelu(w.exact("X", rows), idx[rows],
                                      gate[rows].astype(np.float64), w.exact("W1"),
                                      w.exact("W2"))
    check_rows(to_host_f64(Y)[rows], Yo, "bf16", f"gelu experts many tiles d_ff {dff}")


EDGE = [
    # T, Nh, Ne, k, dff, bias  (bf16 at d_head 128 and 64: the pipelined kernels)
    (37, 2, 40, 5, 128, "none"),     # ragged T, N_e % 32 != 0, odd k
    (300, 3, 64, 1, 384, "none"),    # k = 1, d_ff = 384 (12 chunks of 32)
    (129, 2, 33, 3, 512, "zipf"),    # just past a token block, d_ff = 512
    (255, 2, 16, 16, 256, "none"),   # k = N_e: dense softmax mixture of GELU MLPs
    (1200, 2, 4, 3, 256, "zipf"),    # >= 768 slots per expert: 256-row tiles at d_head 128
    (1000, 1, 2, 2, 128, "none"),    # the same with 4 chunks per tile
]


@pytest.mark.parametrize("dh", [128, 64])
@pytest.mark.parametrize("case", EDGE, ids=lambda c: "T%d_h%d_e%d_k%d_f%d_%s" % c)
def test_gelu_edge_layer(case, dh, oracle_instance):
    T, Nh, Ne, k, dff, bias = case
    shape = workloads.Shape(T, Nh, dh, Ne, k, dff, "bf16", bias=bias, expert="gelu")
    w = workloads.generate(shape, seed=3)
    announce(f"gelu edge {case} d_head {dh}")
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
    err, _ = check_rows(to_host_f64(Y)[rows_ok], Yo[rows_ok], "bf16", f"gelu edge {case} d_head {dh}")
    assert err <= REL_L2["bf16"]


# fp32, and d_ff values that are not multiples of 128: the generic FFN kernel
# (gate-scaled per-slot outputs over half tiles) in its GELU form.
GENERIC = [
    # T, Nh, Ne, k, dff, bias, dtype
    (300, 2, 16, 2, 128, "none", "f32"),
    (129, 3, 40, 5, 96, "zipf", "f32"),    # ragged T, odd k, d_ff 96
    (257, 2, 24, 3, 96, "zipf", "bf16"),   # d_ff 96 (3 chunks)
    (200, 2, 12, 4, 160, "none", "bf16"),  # d_ff 160 (5 chunks)
    (1500, 1, 2, 2, 32, "none", "bf16"),   # one chunk; experts with several tiles
]


@pytest.mark.parametrize("dh", [128, 64])
@pytest.mark.parametrize("case", GENERIC, ids=lambda c: "T%d_h%d_e%d_k%d_f%d_%s_%s" % c)
def test_gelu_generic_kernel_layer(case, dh, oracle_instance):
    T, Nh, Ne, k, dff, bias, dt = case
    shape = workloads.Shape(T, Nh, dh, Ne, k, dff, dt, bias=bias, expert="gelu")
    w = workloads.generate(shape, seed=7)
    announce(f"gelu generic {case} d_head {dh}")
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
    err, _ = check_rows(to_host_f64(Y)[rows_ok], Yo[rows_ok], dt, f"gelu generic {case} d_head {dh}")
    assert err <= REL_L2[dt]


def test_gelu_experts_f32(oracle_instance):
    """mhlmoe_experts_gelu in fp32 from a given routing (every slot's gate
    applied by the generic kernel)."""
    shape = workloads.Shape(600, 2, 128, 8, 4, 256, "f32", expert="gelu")
    w = workloads.generate(shape, seed=9)
    idx, gate = workloads.random_routing(shape.T, shape.n_heads, shape.n_experts, shape.top_k,
                                         seed=9)
    announce("gelu experts f32")
    d = DeviceWorkload(w)
    Y = mh.mhlmoe_experts_gelu(d.X, to_device(idx), to_device(gate), d.W1, d.W2)
    torch.cuda.synchronize()
    Yo = oracle_instance.experts_gelu(w.exact("X"), idx, gate.astype(np.float64), w.exact("W1"),
                                      w.exact("W2"))
    err, _ = check_rows(to_host_f64(Y), Yo, "f32", "gelu experts f32")
    assert err <= REL_L2["f32"]


def test_gelu_unsupported_shapes_are_rejected():
    """d_head outside {64, 128}, d_ff not a multiple of 32 or above 512, and
    an fp32 backward return EUNSUPPORTED before anything is launched."""
    dev = torch.device("cuda", 0)
    for dt, dh, dff in ((torch.float32, 96, 128), (torch.bfloat16, 64, 80),
                        (torch.bfloat16, 128, 544)):
        T, Nh, Ne, k = 8, 2, 4, 2
        X = torch.zeros((T, Nh, dh), dtype=dt, device=dev)
        Wr = torch.zeros((Nh, Ne, dh), dtype=torch.float32, device=dev)
        Wi = torch.zeros((Nh, Ne, dff, dh), dtype=dt, device=dev)
        Wo = torch.zeros((Nh, Ne, dh, dff), dtype=dt, device=dev)
        with pytest.raises(mh.MhlmoeError) as e:
            mh.mhlmoe_layer_gelu(X, Wr, None, Wi, Wo, k)
        assert e.value.status == mh.MHLMOE_EUNSUPPORTED, str(e.value)
    T, Nh, dh, Ne, k, dff = 8, 2, 128, 4, 2, 128
    X = torch.zeros((T, Nh, dh), dtype=torch.float32, device=dev)
    with pytest.raises(mh.MhlmoeError) as e:
        mh.mhlmoe_layer_gelu_backward(
            X, torch.zeros((Nh, Ne, dh), device=dev), torch.zeros((Nh, Ne, dff, dh), device=dev),
            torch.zeros((Nh, Ne, dh, dff), device=dev),
            torch.zeros((T, Nh, k), dtype=torch.int32, device=dev),
            torch.zeros((T, Nh, k), device=dev), X)
    assert e.value.status == mh.MHLMOE_EUNSUPPORTED, str(e.value)


# ---------------------------------------------------------------------------
# backward of the GELU expert
# ---------------------------------------------------------------------------

GELU_GRADS = ("dX", "dW_router", "dW1", "dW2")
GELU_BWD = [
    # T, Nh, dh, Ne, k, dff, skew
    (256, 4, 128, 16, 2, 128, 0.0),
    (37, 3, 64, 40, 5, 96, 0.0),          # ragged T, odd k; d_h 64 and d_ff 96 (backward only)
    (513, 2, 128, 384, 4, 256, 1.1),      # the paper's 384-expert shape, skewed, few tokens
    (2048, 8, 128, 768, 8, 128, 0.0),     # the finer-grained paper shape at 2048 tokens
    (150, 2, 128, 24, 3, 96, 0.5),        # odd chunk count at d_head 128: one chunk per dW workgroup
    (2500, 2, 128, 3, 2, 128, 0.0),       # ~1700 slots per expert: several full tiles each
]


def _gelu_bwd_inputs(case, seed):
    T, Nh, dh, Ne, k, dff, skew = case
    s = workloads.Shape(T, Nh, dh, Ne, k, dff, "bf16", backward=True, expert="gelu")
    w = workloads.generate(s, seed)
    idx, gate = workloads.random_routing(T, Nh, Ne, k, seed=seed + 100, skew=skew)
    return w, idx, gate


def _gpu_gelu_backward(w, idx, gate, workspace=None):
    d = DeviceWorkload(w)
    out = mh.mhlmoe_layer_gelu_backward(d.X, d.W_router, d.W1, d.W2, to_device(idx),
                                        to_device(gate), d.dY, workspace=workspace)
    torch.cuda.synchronize()
    return dict(zip(GELU_GRADS, out))


@pytest.mark.parametrize("case", GELU_BWD, ids=lambda c: "T%d_h%d_d%d_e%d_k%d_f%d_s%g" % c)
def test_gelu_backward_parity(case, oracle_instance):
    w, idx, gate = _gelu_bwd_inputs(case, 41)
    announce(f"gelu backward {case}")
    got = _gpu_gelu_backward(w, idx, gate)
    want = oracle_instance.layer_backward(w.exact("X"), w.exact("W_router"), w.exact("W1"), None,
                                          w.exact("W2"), idx, gate, w.exact("dY"))
    T, Nh, dh, Ne, k, dff, skew = case
    counts = np.stack([np.bincount(idx[:, h].ravel(), minlength=Ne) for h in range(Nh)])
    for n in GELU_GRADS:
        if n == "dX":
            check_rows(to_host_f64(got[n]), want[n], "bf16", f"gelu backward {case} dX")
        else:
            check_expert_blocks(to_host_f64(got[n]), want[n], counts, f"gelu backward {case} {n}")
    empty = torch.from_numpy(counts == 0).cuda()
    for n in ("dW_router", "dW1", "dW2"):
        assert not torch.any(got[n][empty] != 0), n


def test_gelu_backward_deterministic_and_empty():
    case = (700, 2, 128, 32, 4, 256, 1.1)
    w, idx, gate = _gelu_bwd_inputs(case, 42)
    s = w.shape
    announce("gelu backward determinism, T = 0")
    ws = mh.workspace(mh.MHLMOE_OP_LAYER_BACKWARD, s.T, s.n_heads, s.d_head, s.n_experts,
                      s.top_k, s.d_ff, mh.MHLMOE_BF16)
    a = _gpu_gelu_backward(w, idx, gate, ws)
    ws.fill_(0x5A)
    b = _gpu_gelu_backward(w, idx, gate, ws)
    for n in GELU_GRADS:
        x, y = a[n], b[n]
        if x.dtype == torch.bfloat16:
            x, y = x.view(torch.int16), y.view(torch.int16)
        assert torch.equal(x, y), n
    Nh, dh, Ne, k, dff = 2, 128, 8, 2, 128
    X = torch.empty((0, Nh, dh), dtype=torch.bfloat16, device="cuda")
    nan = float("nan")
    outs = dict(dW_router=torch.full((Nh, Ne, dh), nan, device="cuda"),
                dW_in=torch.full((Nh, Ne, dff, dh), nan, device="cuda"),
                dW_out=torch.full((Nh, Ne, dh, dff), nan, device="cuda"))
    dX, *grads = mh.mhlmoe_layer_gelu_backward(
        X, torch.randn(Nh, Ne, dh, device="cuda"),
        torch.randn(Nh, Ne, dff, dh, device="cuda").bfloat16(),
        torch.randn(Nh, Ne, dh, dff, device="cuda").bfloat16(),
        torch.empty((0, Nh, k), dtype=torch.int32, device="cuda"),
        torch.empty((0, Nh, k), dtype=torch.float32, device="cuda"), X, **outs)
    torch.cuda.synchronize()
    for g in grads:
        assert torch.all(g == 0)


def test_gelu_routed_and_latent_backward(oracle_instance):
    """The GELU expert through the routed backward (R = X: weight gradients
    bit for bit those of mhlmoe_layer_gelu_backward, dX + dR its dX within
    bf16 rounding) and through the latent-layer backward (against the
    oracle)."""
    case = (600, 4, 128, 64, 4, 256, 0.5)
    w, idx, gate = _gelu_bwd_inputs(case, 43)
    announce("gelu routed / latent backward")
    d = DeviceWorkload(w)
    idxd, gated = to_device(idx), to_device(gate)
    ref = mh.mhlmoe_layer_gelu_backward(d.X, d.W_router, d.W1, d.W2, idxd, gated, d.dY)
    dX, dR, dWr, dWi, _, dWo = mh.mhlmoe_layer_backward_routed(
        d.X, d.X, d.W_router, d.W1, None, d.W2, idxd, gated, d.dY)
    torch.cuda.synchronize()
    for a, b in ((dWr, ref[1]), (dWi, ref[2]), (dWo, ref[3])):
        assert torch.equal(a, b)
    tot = dX.double() + dR.double()
    assert float(torch.linalg.vector_norm(tot - ref[0].double()) /
                 torch.linalg.vector_norm(ref[0].double())) <= 1e-2
    s = w.shape
    li = workloads.latent_inputs(s, 1024, False, 43)
    dl = {n: to_device(v) for n, v in li.items()}
    g = mh.mhlmoe_latent_layer_backward(dl["x"], dl["W_in"], d.W_router, d.W1, None, d.W2,
                                        dl["W_out"], dl["X_lat"], None, dl["Y_lat"], idxd, gated,
                                        dl["dout"])
    torch.cuda.synchronize()
    ex = workloads.bf16_bits_to_f64
    want = oracle_instance.latent_layer_backward(
        ex(li["x"]), ex(li["W_in"]), w.exact("W_router"), w.exact("W1"), None, w.exact("W2"),
        ex(li["W_out"]), ex(li["X_lat"]), None, ex(li["Y_lat"]), idx, gate, ex(li["dout"]))
    counts = np.stack([np.bincount(idx[:, h].ravel(), minlength=s.n_experts)
                       for h in range(s.n_heads)])
    for n in ("dx", "dW_in", "dW_out"):
        check_rows(to_host_f64(g[n]), want[n], "bf16", f"gelu latent backward {n}")
    for n in ("dW_router", "dW1", "dW2"):
        check_expert_blocks(to_host_f64(g[n]), want[n], counts, f"gelu latent backward {n}")



def test_gelu_layer_16_heads_of_64(oracle_instance):
    """The paper's 16 x 64 head configuration (Table 2: the same latent width
    as 8 x 128) at the 0.2B-2.2B layer's expert shape (384 experts per head,
    k = 4, d_ff 256) over four 2048-token sequences, through the d_h-64 GELU
    kernel; sampled rows against the oracle."""
    shape = workloads.Shape(8192, 16, 64, 384, 4, 256, "bf16", expert="gelu")
    w = workloads.generate(shape, seed=7)
    announce("gelu layer 16 x 64 heads")
    d = DeviceWorkload(w)
    Y, idx, gate, counts = mh.mhlmoe_layer_gelu(d.X, d.W_router, d.bias, d.W1, d.W2, shape.top_k)
    torch.cuda.synchronize()
    assert torch.all(counts.sum(dim=1) == shape.T * shape.top_k)
    rows = workloads.sample_rows(shape.T, 256)
    Xr = w.exact("X", rows)
    r = oracle_instance.route(Xr, w.exact("W_router"), w.exact("bias"), k=shape.top_k)
    ok = check_routing(idx.cpu().numpy()[rows], gate.cpu().numpy()[rows].astype(np.float64),
                       r["idx"], r["gate"], r["keys"], shape.top_k, "gelu 16x64")
    Yo = oracle_instance.experts_gelu(Xr, r["idx"], r["gate"], w.exact("W1"), w.exact("W2"))
    rows_ok = np.all(ok, axis=1)
    check_rows(to_host_f64(Y)[rows][rows_ok], Yo[rows_ok], "bf16", "gelu layer 16 x 64")
