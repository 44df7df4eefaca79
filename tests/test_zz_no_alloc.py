"""mhlmoe_route_static, the routing entry point that allocates nothing (its
scratch is the library's static device array), against mhlmoe_route on the
same inputs: idx, gate and counts must be bitwise equal.  Two calls in a row
share the array, the second on a smaller input; the first workload needs
16 MiB of the 32 MiB scratch."""
import pytest
import torch

import paper_2602_04870_amd as mh
from tests.gpu_util import announce, needs_gpu

pytestmark = [pytest.mark.gpu, needs_gpu]

# T, N_h, d_h, N_e, k, dtype, bias: the skewed workload's routing shape, then
# a smaller one with a bias, ragged T, 64-bit keys and odd k
CASES = [(65536, 8, 128, 1024, 32, torch.bfloat16, False),
         (1000, 4, 64, 200, 7, torch.float32, True)]


def _inputs(T, Nh, dh, Ne, dt, bias, seed):
    g = torch.Generator(device="cuda").manual_seed(seed)
    X = torch.randn((T, Nh, dh), generator=g, device="cuda").to(dt)
    Wr = torch.randn((Nh, Ne, dh), generator=g, device="cuda") / dh ** 0.5
    b = torch.randn((Nh, Ne), generator=g, device="cuda") if bias else None
    return X, Wr, b


def test_route_static_matches_route_on_two_calls_in_a_row():
    for i, (T, Nh, dh, Ne, k, dt, bias) in enumerate(CASES):
        announce(f"route_static call {i}: T={T} Nh={Nh} dh={dh} Ne={Ne} k={k} {dt}")
        X, Wr, b = _inputs(T, Nh, dh, Ne, dt, bias, seed=70 + i)
        idx, gate, counts = mh.mhlmoe_route(X, Wr, b, k)
        out = dict(idx=torch.full((T, Nh, k), -7, dtype=torch.int32, device="cuda"),
                   gate=torch.full((T, Nh, k), float("nan"), device="cuda"),
                   counts=torch.full((Nh, Ne), -7, dtype=torch.int32, device="cuda"))
        torch.cuda.synchronize()
        mh.mhlmoe_route_static(X, Wr, b, k, **out)
        torch.cuda.synchronize()
        assert torch.equal(out["idx"], idx)
        assert torch.equal(out["gate"].view(torch.int32), gate.view(torch.int32))
        assert torch.equal(out["counts"], counts)
        assert torch.all(counts.sum(dim=1) == T * k)
