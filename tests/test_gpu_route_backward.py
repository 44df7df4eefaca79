"""GPU parity of the IO-aware routing backward on its own (Algorithm 2,
Sec. 3.3) through mhlmoe_route_backward, against the CPU oracle (pinned by
finite differences of the gates and by the chain rule into the layer
backward in tests/oracle_pins.py).

Routing inputs (idx, gate) and the gate gradient come from the seeded
generator.  Tolerances: 2e-2 relative L2 for bf16 dX (fp32 accumulation,
one rounding), 1e-4 for fp32; dW_router is fp32 either way; experts without
slots get exact zeros.
"""
import numpy as np
import pytest
import torch

import paper_2602_04870_amd as mh
import workloads
from tests.gpu_util import (REL_L2, announce, check_expert_blocks, check_rows, needs_gpu, rel_l2,
                            to_device, to_host_f64)

pytestmark = [pytest.mark.gpu, needs_gpu]

CASES = [
    # T, Nh, dh, Ne, k, dtype, skew
    (256, 4, 64, 16, 2, "f32", 0.0),
    (4096, 8, 128, 64, 8, "bf16", 0.0),
    (37, 3, 64, 40, 5, "bf16", 0.0),        # ragged T, odd k
    (513, 2, 128, 1024, 8, "f32", 1.1),     # most experts get no slot
    (2048, 8, 128, 1024, 32, "bf16", 1.1),  # the skewed workload's shape at 2048 tokens
]


def _inputs(case, seed):
    T, Nh, dh, Ne, k, dt, skew = case
    w = workloads.generate(workloads.Shape(T, Nh, dh, Ne, k, 32, dt), seed)
    idx, gate = workloads.random_routing(T, Nh, Ne, k, seed=seed + 100, skew=skew)
    dgate = np.random.default_rng(seed + 200).standard_normal((T, Nh, k)).astype(np.float32)
    return w, idx, gate, dgate


@pytest.mark.parametrize("case", CASES, ids=lambda c: "T%d_h%d_d%d_e%d_k%d_%s_s%g" % c)
def test_route_backward_parity(case, oracle_instance):
    T, Nh, dh, Ne, k, dt, skew = case
    w, idx, gate, dgate = _inputs(case, 51)
    announce(f"route backward {case}")
    dX, dWr = mh.mhlmoe_route_backward(to_device(w.X), to_device(w.W_router), to_device(idx),
                                       to_device(gate), to_device(dgate))
    torch.cuda.synchronize()
    want = oracle_instance.route_backward(w.exact("X"), w.exact("W_router"), idx, gate, dgate)
    counts = np.stack([np.bincount(idx[:, h].ravel(), minlength=Ne) for h in range(Nh)])
    check_rows(to_host_f64(dX), want["dX"], dt, f"route backward {case} dX")
    check_expert_blocks(to_host_f64(dWr), want["dW_router"], counts,
                        f"route backward {case} dW_router", dt)
    assert not torch.any(dWr[torch.from_numpy(counts == 0).cuda()] != 0)


def test_route_backward_deterministic_and_empty():
    case = (3000, 4, 128, 256, 16, "bf16", 1.1)
    w, idx, gate, dgate = _inputs(case, 52)
    T, Nh, dh, Ne, k = 3000, 4, 128, 256, 16
    announce("route backward determinism, T = 0")
    ws = mh.workspace(mh.MHLMOE_OP_ROUTE_BACKWARD, T, Nh, dh, Ne, k, 0, mh.MHLMOE_BF16)
    args = (to_device(w.X), to_device(w.W_router), to_device(idx), to_device(gate),
            to_device(dgate))
    a = mh.mhlmoe_route_backward(*args, workspace=ws)
    ws.fill_(0x5A)
    b = mh.mhlmoe_route_backward(*args, workspace=ws)
    torch.cuda.synchronize()
    assert torch.equal(a[0].view(torch.int16), b[0].view(torch.int16))
    assert torch.equal(a[1], b[1])
    X0 = torch.empty((0, Nh, dh), dtype=torch.bfloat16, device="cuda")
    e0 = torch.empty((0, Nh, k), dtype=torch.float32, device="cuda")
    dWr = torch.full((Nh, Ne, dh), float("nan"), device="cuda")
    dX0, dWr = mh.mhlmoe_route_backward(X0, args[1], torch.empty((0, Nh, k), dtype=torch.int32,
                                                                 device="cuda"), e0, e0,
                                        dW_router=dWr)
    torch.cuda.synchronize()
    assert dX0.shape == (0, Nh, dh) and torch.all(dWr == 0)
