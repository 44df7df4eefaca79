"""GPU parity of the layer with its projections (Eq. (5)-(6), Sec. 3.1; with
separate routing sub-tokens, Eq. (9), Sec. 4.4) through the C ABI, against
the CPU oracle (fp64 matmuls around the pinned heads; see
tests/oracle_pins.py).

The sub-tokens X_lat = W_in x are held in the dtype of the path, so the
router decides on rounded values; the oracle rounds its fp64 sub-tokens to
bf16 the same way (``latent_round="bf16"``) before routing.  The GPU's
sub-tokens (fp32 accumulation, rounded once) may still differ from the
oracle's correctly rounded ones by one bf16 unit in rare elements, which the
index rule's tie window absorbs.  Tolerances otherwise as elsewhere.
"""
import numpy as np
import pytest
import torch

import paper_2602_04870_amd as mh
import workloads
from tests.gpu_util import (REL_L2, announce, check_expert_blocks, check_routing, check_rows,
                            needs_gpu, rel_l2, to_device,
                            to_host_f64)

pytestmark = [pytest.mark.gpu, needs_gpu]


def _exact(a):
    return workloads.bf16_bits_to_f64(a) if a.dtype == np.uint16 else np.asarray(a, np.float64)


FWD = [
    # T, Nh, dh, Ne, k, dff, dtype, bias, expert, d_model, routing_tokens
    (4096, 8, 128, 64, 4, 128, "bf16", "none", "swiglu", 1024, False),
    # the configuration the steps-either-side sweep times (bf16_t4096_e64, d_model 1024)
    (4096, 8, 128, 64, 8, 256, "bf16", "none", "swiglu", 1024, False),
    (4096, 8, 128, 64, 8, 256, "bf16", "none", "swiglu", 1024, True),
    (1000, 8, 128, 64, 4, 128, "bf16", "zipf", "swiglu", 1536, True),
    (777, 8, 128, 384, 4, 256, "bf16", "none", "gelu", 1024, False),
    (256, 4, 64, 16, 2, 128, "f32", "none", "swiglu", 200, True),
]


@pytest.mark.parametrize("case", FWD, ids=lambda c: "T%d_h%d_d%d_e%d_k%d_f%d_%s_%s_%s_dm%d_rt%d" % c)
def test_latent_forward_parity(case, oracle_instance):
    T, Nh, dh, Ne, k, dff, dt, bias, expert, dm, rt = case
    s = workloads.Shape(T, Nh, dh, Ne, k, dff, dt, bias=bias, expert=expert)
    w = workloads.generate(s, 31)
    li = workloads.latent_inputs(s, dm, rt, 31)
    announce(f"latent forward {case}")
    dev = {n: to_device(v) for n, v in li.items()}
    r = mh.mhlmoe_latent_layer(dev["x"], dev["W_in"], to_device(w.W_router), to_device(w.bias),
                               to_device(w.W1), to_device(w.W3), to_device(w.W2), dev["W_out"],
                               Nh, k, routing_tokens=rt)
    torch.cuda.synchronize()
    assert torch.all(r["counts"].sum(dim=1) == T * k)
    rows = workloads.sample_rows(T, 256)
    want = oracle_instance.latent_layer(
        _exact(li["x"])[rows], _exact(li["W_in"]), w.exact("W_router"), w.exact("bias"),
        w.exact("W1"), w.exact("W3"), w.exact("W2"), _exact(li["W_out"]), Nh, k,
        routing_tokens=rt, latent_round="bf16" if dt == "bf16" else None)
    # the sub-tokens: rarely different, and then by at most one bf16 unit
    # plus the fp32 accumulation bound d_model 2^-24 sum_i |x_i| |w_i|
    # (which dominates where the dot product cancels)
    xa = np.abs(_exact(li["x"])[rows])
    wa = np.abs(_exact(li["W_in"]))
    N = Nh * dh
    for name, w_rows in (("X_lat", wa[:N]), ("R_lat", wa[N:]))[:2 if rt else 1]:
        got = to_host_f64(r[name])[rows]
        ref = want[name]
        err = rel_l2(got, ref)
        print(f"[latent] {case} {name} rel-L2 = {err:.3e}", flush=True)
        if dt == "bf16":
            frac = np.mean(got != ref)
            assert frac < 1e-2, f"{name}: {frac:.2%} of elements differ"
            acc = (dm * 2.0 ** -24 * (xa @ w_rows.T)).reshape(ref.shape)
            assert np.all(np.abs(got - ref) <= 2.0 ** -7 * np.abs(ref) + acc)
        else:
            assert err <= 1e-6
    ok = check_routing(r["idx"].cpu().numpy()[rows], r["gate"].cpu().numpy()[rows].astype(np.float64),
                       want["idx"], want["gate"], want["keys"], k, str(case))
    rows_ok = np.all(ok, axis=1)
    for name in ("Y_lat", "out"):
        got = to_host_f64(r[name])[rows][rows_ok]
        check_rows(got, want[name][rows_ok], dt, f"latent {case} {name}")


def _bits(t):
    return t.view(torch.int16) if t.dtype == torch.bfloat16 else t.view(torch.int32)


def test_latent_identity_projections_equal_the_layer():
    """W_in = W_out = I (d_model = N): every projection product is one term
    plus zeros, exact in any order, so the latent layer reproduces
    mhlmoe_layer on x bit for bit."""
    s = workloads.Shape(2048, 8, 128, 64, 4, 128, "bf16")
    w = workloads.generate(s, 32)
    announce("latent identity projections")
    N = s.n_heads * s.d_head
    X = to_device(w.X)
    eye = torch.eye(N, device="cuda").bfloat16()
    Wr, b = to_device(w.W_router), to_device(w.bias)
    W1, W3, W2 = to_device(w.W1), to_device(w.W3), to_device(w.W2)
    r = mh.mhlmoe_latent_layer(X.reshape(s.T, N), eye, Wr, b, W1, W3, W2, eye, s.n_heads,
                               s.top_k)
    Y, idx, gate, counts = mh.mhlmoe_layer(X, Wr, b, W1, W3, W2, s.top_k)
    torch.cuda.synchronize()
    assert torch.equal(_bits(r["X_lat"]), _bits(X))
    assert torch.equal(r["idx"], idx) and torch.equal(_bits(r["gate"]), _bits(gate))
    assert torch.equal(_bits(r["out"].reshape(Y.shape)), _bits(Y))


BWD = [
    # T, Nh, dh, Ne, k, dff, skew, d_model, routing_tokens
    (512, 4, 64, 16, 2, 128, 0.0, 256, False),
    (4096, 8, 128, 64, 8, 256, 0.0, 1024, False),  # as timed by the steps-either-side sweep
    (1000, 8, 128, 64, 4, 128, 1.1, 1024, True),
    (300, 2, 128, 40, 5, 96, 0.0, 384, True),
]


@pytest.mark.parametrize("case", BWD, ids=lambda c: "T%d_h%d_d%d_e%d_k%d_f%d_s%g_dm%d_rt%d" % c)
def test_latent_backward_parity(case, oracle_instance):
    T, Nh, dh, Ne, k, dff, skew, dm, rt = case
    s = workloads.Shape(T, Nh, dh, Ne, k, dff, "bf16", backward=True)
    w = workloads.generate(s, 33)
    li = workloads.latent_inputs(s, dm, rt, 33)
    idx, gate = workloads.random_routing(T, Nh, Ne, k, seed=133, skew=skew)
    announce(f"latent backward {case}")
    dev = {n: to_device(v) for n, v in li.items()}
    g = mh.mhlmoe_latent_layer_backward(
        dev["x"], dev["W_in"], to_device(w.W_router), to_device(w.W1), to_device(w.W3),
        to_device(w.W2), dev["W_out"], dev["X_lat"], dev["R_lat"], dev["Y_lat"], to_device(idx),
        to_device(gate), dev["dout"], routing_tokens=rt)
    torch.cuda.synchronize()
    want = oracle_instance.latent_layer_backward(
        _exact(li["x"]), _exact(li["W_in"]), w.exact("W_router"), w.exact("W1"), w.exact("W3"),
        w.exact("W2"), _exact(li["W_out"]), _exact(li["X_lat"]),
        _exact(li["R_lat"]) if rt else None, _exact(li["Y_lat"]), idx, gate, _exact(li["dout"]),
        routing_tokens=rt)
    counts = np.stack([np.bincount(idx[:, h].ravel(), minlength=Ne) for h in range(Nh)])
    for n in ("dx", "dW_in", "dW_out"):
        check_rows(to_host_f64(g[n]), want[n], "bf16", f"latent backward {case} {n}")
    for n in ("dW_router", "dW1", "dW3", "dW2"):
        check_expert_blocks(to_host_f64(g[n]), want[n], counts, f"latent backward {case} {n}")


def test_latent_backward_empty_batch():
    announce("latent backward T = 0")
    s = workloads.Shape(0, 2, 64, 8, 2, 64, "bf16", backward=True)
    w = workloads.generate(s, 34)
    li = workloads.latent_inputs(s, 96, True, 34)
    dev = {n: to_device(v) for n, v in li.items()}
    idx = torch.empty((0, 2, 2), dtype=torch.int32, device="cuda")
    gate = torch.empty((0, 2, 2), dtype=torch.float32, device="cuda")
    g = mh.mhlmoe_latent_layer_backward(
        dev["x"], dev["W_in"], to_device(w.W_router), to_device(w.W1), to_device(w.W3),
        to_device(w.W2), dev["W_out"], dev["X_lat"], dev["R_lat"], dev["Y_lat"], idx, gate,
        dev["dout"], routing_tokens=True)
    torch.cuda.synchronize()
    assert g["dx"].shape == (0, 96)
    for n in ("dW_in", "dW_out", "dW_router", "dW1", "dW3", "dW2"):
        assert torch.all(g[n] == 0), n


def test_latent_plan_cache_turnover():
    """Calls at 140 different token counts need 280 projection plans, more
    than the library keeps, so its plan cache is emptied on the way; every
    call still reproduces mhlmoe_layer bit for bit (identity projections)."""
    announce("latent plan cache turnover")
    Nh, dh, Ne, k, dff = 2, 64, 8, 2, 64
    N = Nh * dh
    s = workloads.Shape(140, Nh, dh, Ne, k, dff, "bf16")
    w = workloads.generate(s, 35)
    X = to_device(w.X)
    eye = torch.eye(N, device="cuda").bfloat16()
    Wr, W1, W3, W2 = (to_device(w.W_router), to_device(w.W1), to_device(w.W3), to_device(w.W2))
    for T in range(1, 141):
        Xt = X[:T].contiguous()
        r = mh.mhlmoe_latent_layer(Xt.reshape(T, N), eye, Wr, None, W1, W3, W2, eye, Nh, k)
        Y = mh.mhlmoe_layer(Xt, Wr, None, W1, W3, W2, k, return_routing=False)
        torch.cuda.synchronize()
        assert torch.equal(_bits(r["out"].reshape(Y.shape)), _bits(Y)), T
