"""GPU parity of the auxiliary-loss-free bias update (Sec. 2.2) through the C
ABI: bias[h, e] += rate * sign(mean load - load), one fp32 addition per
entry, so the GPU result must equal the oracle's bit for bit.

Loads come from the seeded generator (balanced, one-hot, empty and skewed
heads); the oracle's update rule is pinned in tests/oracle_pins.py.
"""
import numpy as np
import pytest
import torch

import paper_2602_04870_amd as mh
import workloads
from tests.gpu_util import announce, needs_gpu

pytestmark = [pytest.mark.gpu, needs_gpu]

CASES = [
    # n_heads, n_experts, total slots per head, rate
    (4, 16, 4096, 1e-3),
    (8, 64, 65536, 0.125),
    (3, 1, 100, 0.5),            # one expert: always equal to the mean
    (5, 1000, 999, 1e-3),        # mean below 1, Ne not a multiple of 256
    (1024, 1024, 1 << 20, 1e-3),  # largest supported shape
    (8, 384, 8192 * 4, 1e-8),    # below half an ulp of most biases
    (6, 257, 3000, 0.0),         # zero rate: unchanged
]


@pytest.mark.parametrize("case", CASES, ids=lambda c: "h%d_e%d_n%d_r%g" % c)
def test_bias_update_bitwise(case, oracle_instance):
    Nh, Ne, total, rate = case
    counts = workloads.random_counts(Nh, Ne, seed=Nh * 1000 + Ne, total=total)
    rng = np.random.default_rng(Ne)
    bias = (rng.standard_normal((Nh, Ne)) * rng.choice([1e-3, 1.0, 100.0], (Nh, 1))).astype(np.float32)
    bias[0, 0] = 0.0
    announce(f"bias update {case}")
    b = torch.from_numpy(bias).cuda()
    mh.mhlmoe_bias_update(torch.from_numpy(counts).cuda(), b, rate)
    torch.cuda.synchronize()
    want = oracle_instance.bias_update(counts, bias, np.float32(rate))
    got = b.cpu().numpy()
    bad = np.flatnonzero(got.view(np.uint32) != want.view(np.uint32))
    assert bad.size == 0, f"{bad.size} entries differ, first at {np.unravel_index(bad[0], got.shape)}"


def test_bias_update_balances_routing():
    """Alternating routing (Algorithm 1 with the bias) and the update on the
    GPU shrinks the spread of per-expert loads of a router that favours a few
    experts, as the method intends."""
    s = workloads.Shape(4096, 4, 128, 64, 4, 128, "bf16", bias="zipf", zipf_s=1.5)
    w = workloads.generate(s, 0)
    announce("bias update closed loop")
    X = workloads.to_device(w.X)
    Wr = workloads.to_device(w.W_router)
    b = workloads.to_device(w.bias).clone()
    spreads = []
    for _ in range(200):
        _, _, counts = mh.mhlmoe_route(X, Wr, b, s.top_k)
        spreads.append((counts.max(dim=1).values - counts.min(dim=1).values).cpu().numpy())
        mh.mhlmoe_bias_update(counts, b, 0.02)
    torch.cuda.synchronize()
    first, last = spreads[0].astype(float), np.mean(spreads[-20:], axis=0)
    print(f"[bias update] load spread per head: {first} -> {last}", flush=True)
    assert np.all(last < 0.25 * first)


def test_bias_update_rejects_bad_arguments():
    c = torch.zeros((2, 8), dtype=torch.int32, device="cuda")
    b = torch.zeros((2, 8), dtype=torch.float32, device="cuda")
    for rate in (-1e-3, float("nan"), float("inf")):
        with pytest.raises(mh.MhlmoeError) as e:
            mh.mhlmoe_bias_update(c, b, rate)
        assert e.value.status == mh.MHLMOE_EINVAL
    c2 = torch.zeros((1, 1025), dtype=torch.int32, device="cuda")
    b2 = torch.zeros((1, 1025), dtype=torch.float32, device="cuda")
    with pytest.raises(mh.MhlmoeError) as e:
        mh.mhlmoe_bias_update(c2, b2, 1e-3)
    assert e.value.status == mh.MHLMOE_EINVAL
    torch.cuda.synchronize()
    assert torch.all(b == 0)
