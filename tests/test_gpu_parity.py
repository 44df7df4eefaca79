"""GPU parity: libmhlmoe (through its C ABI) against the CPU oracle on the same
seeded inputs.

Every GPU call runs the full workload in the configuration the benchmark
times; where the oracle would take too long for the whole workload, it is run
on a seeded sample of token rows (tokens are independent in routing and in
the expert computation, so a row's oracle result does not depend on the other
rows).  Tolerances follow the contract: indices bit-exact except near ties
(oracle keys closer than 1e-3), gates within 1e-3, outputs within 2e-2
relative L2 (bf16) or 1e-4 (fp32), pooled over the compared rows, and every
single (token, head) row within 5e-2 (bf16) or 1e-3 (fp32) of its own norm
(see tests/gpu_util.py: check_rows); clustering is bit-exact.
"""
import numpy as np
import pytest
import torch

import paper_2602_04870_amd as mh
import workloads
from tests.gpu_util import (REL_L2, DeviceWorkload, announce, check_routing, check_rows,
                            needs_gpu, rel_l2, to_device, to_host_f64, workload)

pytestmark = [pytest.mark.gpu, needs_gpu]

CONFIGS = workloads.CONFIG_ORDER
# rows of the oracle sample per config (None = all rows)
ROUTE_ROWS = {"tiny_f32_t256": None, "bf16_t4096_e64": None, "headline_bf16_t16384_e128": 4096,
              "granular_bf16_t16384_e256": 4096, "skewed_bf16_t65536_e1024": 1024}
FFN_ROWS = {"tiny_f32_t256": None, "bf16_t4096_e64": 512, "headline_bf16_t16384_e128": 256,
            "granular_bf16_t16384_e256": 256, "skewed_bf16_t65536_e1024": 128}


def _rows(name, table):
    T = workloads.CONFIGS[name].T
    n = table[name]
    return workloads.sample_rows(T, n) if n else np.arange(T)


@pytest.mark.parametrize("name", CONFIGS)
def test_route_parity(name, oracle_instance):
    w = workload(name)
    s = w.shape
    announce(f"route {name}")
    d = DeviceWorkload(w)
    idx, gate, counts = mh.mhlmoe_route(d.X, d.W_router, d.bias, s.top_k)
    torch.cuda.synchronize()
    g_idx = idx.cpu().numpy()
    g_gate = gate.cpu().numpy().astype(np.float64)
    g_counts = counts.cpu().numpy()
    # counts are exactly the histogram of the GPU's own selection
    for h in range(s.n_heads):
        assert np.array_equal(g_counts[h], np.bincount(g_idx[:, h].ravel(), minlength=s.n_experts))
    assert np.all(g_counts.sum(-1) == s.T * s.top_k)
    rows = _rows(name, ROUTE_ROWS)
    r = oracle_instance.route(w.exact("X", rows), w.exact("W_router"), w.exact("bias"), k=s.top_k)
    ok = check_routing(g_idx[rows], g_gate[rows], r["idx"], r["gate"], r["keys"], s.top_k, name)
    if len(rows) == s.T:
        # oracle counts differ from the GPU's only through excused rows
        bad = ~ok
        for h in range(s.n_heads):
            d_or = np.bincount(r["idx"][:, h][bad[:, h]].ravel(), minlength=s.n_experts)
            d_gp = np.bincount(g_idx[:, h][bad[:, h]].ravel(), minlength=s.n_experts)
            assert np.array_equal(r["counts"][h] - d_or, g_counts[h] - d_gp)


@pytest.mark.parametrize("name", CONFIGS)
def test_bucket_parity(name, oracle_instance):
    s = workloads.CONFIGS[name]
    idx, _ = workloads.random_routing(s.T, s.n_heads, s.n_experts, s.top_k, seed=11,
                                      skew=1.1 if s.bias == "zipf" else 0.0)
    announce(f"bucket {name}")
    counts, offsets, perm = mh.mhlmoe_bucket(to_device(idx), s.n_experts)
    torch.cuda.synchronize()
    o_off, o_perm = oracle_instance.bucket(idx, s.n_experts)
    assert np.array_equal(offsets.cpu().numpy(), o_off)
    assert np.array_equal(counts.cpu().numpy(), np.diff(o_off, axis=-1))
    assert np.array_equal(perm.cpu().numpy(), o_perm)


@pytest.mark.parametrize("name", CONFIGS)
def test_experts_parity(name, oracle_instance):
    w = workload(name)
    s = w.shape
    idx, gate = workloads.random_routing(s.T, s.n_heads, s.n_experts, s.top_k, seed=5,
                                         skew=1.1 if s.bias == "zipf" else 0.0)
    announce(f"experts {name}")
    d = DeviceWorkload(w)
    Y = mh.mhlmoe_experts(d.X, to_device(idx), to_device(gate), d.W1, d.W3, d.W2)
    torch.cuda.synchronize()
    rows = _rows(name, FFN_ROWS)
    Yo = oracle_instance.experts(w.exact("X", rows), idx[rows], gate[rows].astype(np.float64),
                                 w.exact("W1"), w.exact("W3"), w.exact("W2"))
    check_rows(to_host_f64(Y)[rows], Yo, s.dtype, f"experts {name}")


@pytest.mark.parametrize("name", CONFIGS)
def test_layer_parity(name, oracle_instance):
    w = workload(name)
    s = w.shape
    announce(f"layer {name}")
    d = DeviceWorkload(w)
    Y, idx, gate, counts = mh.mhlmoe_layer(d.X, d.W_router, d.bias, d.W1, d.W3, d.W2, s.top_k)
    torch.cuda.synchronize()
    rows = _rows(name, FFN_ROWS)
    Xr = w.exact("X", rows)
    r = oracle_instance.route(Xr, w.exact("W_router"), w.exact("bias"), k=s.top_k)
    ok = check_routing(idx.cpu().numpy()[rows], gate.cpu().numpy()[rows].astype(np.float64),
                       r["idx"], r["gate"], r["keys"], s.top_k, name)
    Yo = oracle_instance.experts(Xr, r["idx"], r["gate"], w.exact("W1"), w.exact("W3"),
                                 w.exact("W2"))
    rows_ok = np.all(ok, axis=1)
    check_rows(to_host_f64(Y)[rows][rows_ok], Yo[rows_ok], s.dtype, f"layer {name}")


@pytest.mark.parametrize("name", [n for n in CONFIGS if n != "tiny_f32_t256"])
def test_layer_is_deterministic(name):
    w = workload(name)
    s = w.shape
    announce(f"determinism {name}")
    d = DeviceWorkload(w)
    ws = mh.workspace(mh.MHLMOE_OP_LAYER, s.T, s.n_heads, s.d_head, s.n_experts, s.top_k, s.d_ff,
                      mh.MHLMOE_BF16)
    a = mh.mhlmoe_layer(d.X, d.W_router, d.bias, d.W1, d.W3, d.W2, s.top_k, workspace=ws)
    ws.fill_(0x5A)  # workspace contents must not matter
    b = mh.mhlmoe_layer(d.X, d.W_router, d.bias, d.W1, d.W3, d.W2, s.top_k, workspace=ws)
    torch.cuda.synchronize()
    for x, y in zip(a, b):
        assert torch.equal(x.view(torch.int16) if x.dtype == torch.bfloat16 else x,
                           y.view(torch.int16) if y.dtype == torch.bfloat16 else y)


def test_head_split_equals_full_layer():
    """Head Parallel shards heads across GPUs; running two halves of the heads
    as separate calls must reproduce the full call bit for bit."""
    w = workload("bf16_t4096_e64")
    s = w.shape
    announce("head split bf16 T4096")
    d = DeviceWorkload(w)
    Y, idx, gate, counts = mh.mhlmoe_layer(d.X, d.W_router, d.bias, d.W1, d.W3, d.W2, s.top_k)
    half = s.n_heads // 2
    for lo, hi in ((0, half), (half, s.n_heads)):
        Yh, ih, gh, ch = mh.mhlmoe_layer(d.X[:, lo:hi].contiguous(), d.W_router[lo:hi].contiguous(),
                                         None, d.W1[lo:hi].contiguous(), d.W3[lo:hi].contiguous(),
                                         d.W2[lo:hi].contiguous(), s.top_k)
        torch.cuda.synchronize()
        assert torch.equal(Yh.view(torch.int16), Y[:, lo:hi].contiguous().view(torch.int16))
        assert torch.equal(ih, idx[:, lo:hi]) and torch.equal(gh, gate[:, lo:hi])
        assert torch.equal(ch, counts[lo:hi])


# ---------------------------------------------------------------------------
# edge cases, checked in full against the oracle
# ---------------------------------------------------------------------------

EDGE = [
    # T, Nh, dh, Ne, k, dff, dtype, bias
    (1, 2, 64, 8, 2, 64, "bf16", "none"),
    (37, 3, 128, 40, 5, 96, "bf16", "none"),       # ragged T, Ne % 32 != 0, odd k
    (129, 2, 128, 33, 3, 128, "bf16", "zipf"),     # T just past a token block
    (255, 2, 64, 16, 16, 64, "bf16", "none"),      # k = Ne: dense softmax mixture
    (300, 2, 128, 64, 1, 32, "bf16", "none"),      # k = 1
    (200, 2, 128, 100, 32, 128, "bf16", "zipf"),   # largest k
    (130, 2, 128, 24, 4, 256, "f32", "none"),      # fp32 at d_head 128
    (77, 1, 64, 1, 1, 64, "f32", "none"),          # N_e = k = 1: dense SwiGLU MLP
    (513, 2, 128, 1024, 8, 64, "bf16", "zipf"),    # largest N_e
    (150, 2, 128, 200, 6, 64, "bf16", "zipf"),     # 32-bit keys with 8 index bits, k % 4 != 0
    (90, 2, 64, 160, 4, 64, "bf16", "none"),       # N_e > 128 at d_head 64: 64-bit keys
    (140, 2, 128, 256, 16, 128, "f32", "none"),    # fp32 X with 8 index bits
    (70, 2, 128, 48, 4, 512, "bf16", "none"),      # largest d_ff (16 chunks) at d_head 128
    (70, 2, 64, 48, 4, 512, "bf16", "zipf"),       # largest d_ff at d_head 64
    (45, 2, 128, 20, 3, 480, "bf16", "none"),      # d_ff of 15 chunks (no q32 instantiation)
    (16, 1024, 64, 4, 2, 32, "bf16", "none"),      # the most heads, smallest d_ff
    (97, 2, 64, 1000, 7, 64, "bf16", "zipf"),      # 64-bit keys, N_e % 32 != 0, odd k
    (60, 2, 64, 300, 3, 32, "f32", "none"),        # fp32 X with 64-bit keys at d_head 64
    # 64-bit keys with the longer lists (two wavefronts per SIMD)
    (600, 2, 128, 1024, 16, 64, "bf16", "zipf"),   # lists of 16
    (300, 2, 64, 777, 32, 64, "bf16", "none"),     # lists of 32, N_e % 32 != 0, no bias
    (200, 2, 128, 300, 20, 64, "f32", "none"),     # fp32 X, k = 20 (lists of 32)
    (150, 2, 128, 400, 5, 64, "f32", "zipf"),      # fp32 X, k = 5 (lists of 8)
    # >= 768 slots per expert on average: the bf16 d_h-128 FFN's 256-row tiles
    (1000, 2, 128, 8, 8, 256, "bf16", "none"),     # 4 tiles per expert, the last ragged
    (800, 2, 128, 6, 6, 128, "bf16", "zipf"),      # k = N_e, skewed gates, 4 chunks per tile
    (800, 2, 128, 3, 3, 384, "bf16", "none"),      # 12 chunks per tile
    (900, 1, 128, 2, 2, 512, "bf16", "none"),      # 16 chunks per tile
    (768, 2, 128, 4, 4, 128, "bf16", "none"),      # exactly 768 slots per expert
]


@pytest.mark.parametrize("case", EDGE, ids=lambda c: "T%d_h%d_d%d_e%d_k%d_f%d_%s_%s" % c)
def test_edge_layer(case, oracle_instance):
    T, Nh, dh, Ne, k, dff, dt, bias = case
    w = workloads.generate(workloads.Shape(T, Nh, dh, Ne, k, dff, dt, bias=bias), seed=3)
    announce(f"edge layer {case}")
    d = DeviceWorkload(w)
    Y, idx, gate, counts = mh.mhlmoe_layer(d.X, d.W_router, d.bias, d.W1, d.W3, d.W2, k)
    torch.cuda.synchronize()
    Yo, oi, og, oc = oracle_instance.layer(w.exact("X"), w.exact("W_router"), w.exact("bias"),
                                           w.exact("W1"), w.exact("W3"), w.exact("W2"), k)
    r = oracle_instance.route(w.exact("X"), w.exact("W_router"), w.exact("bias"), k=k)
    ok = check_routing(idx.cpu().numpy(), gate.cpu().numpy().astype(np.float64), oi, og, r["keys"],
                       k, str(case))
    rows_ok = np.all(ok, axis=1)
    check_rows(to_host_f64(Y)[rows_ok], Yo[rows_ok], dt, f"edge {case}")
    # clustering of the GPU's own selection is the stable sort of it
    c2, off, perm = mh.mhlmoe_bucket(idx, Ne)
    o_off, o_perm = oracle_instance.bucket(idx.cpu().numpy(), Ne)
    assert np.array_equal(perm.cpu().numpy(), o_perm)
    assert torch.equal(c2, counts)


def test_forced_single_expert_is_dropless(oracle_instance):
    """A huge bias sends every token of a head to one expert (k = 1): all T
    slots must be computed (no capacity limit) and the gate is exactly 1."""
    T, Nh, dh, Ne, k, dff = 1000, 2, 128, 64, 1, 128
    w = workloads.generate(workloads.Shape(T, Nh, dh, Ne, k, dff, "bf16"), seed=4)
    w.bias = np.zeros((Nh, Ne), np.float32)
    w.bias[0, 17] = 1e4
    w.bias[1, 63] = 1e4
    announce("forced single expert")
    d = DeviceWorkload(w)
    Y, idx, gate, counts = mh.mhlmoe_layer(d.X, d.W_router, d.bias, d.W1, d.W3, d.W2, k)
    torch.cuda.synchronize()
    assert np.all(idx.cpu().numpy()[:, 0] == 17) and np.all(idx.cpu().numpy()[:, 1] == 63)
    assert torch.all(gate == 1.0)
    assert counts[0, 17].item() == T and counts[1, 63].item() == T
    Yo, *_ = oracle_instance.layer(w.exact("X"), w.exact("W_router"), w.exact("bias"),
                                   w.exact("W1"), w.exact("W3"), w.exact("W2"), k)
    check_rows(to_host_f64(Y), Yo, "bf16", "forced single expert")


def test_empty_batch_is_a_noop():
    announce("T = 0")
    X = torch.empty((0, 2, 64), dtype=torch.bfloat16, device="cuda")
    W = torch.randn(2, 8, 64, device="cuda")
    W1 = torch.randn(2, 8, 64, 64, device="cuda").bfloat16()
    W2 = torch.randn(2, 8, 64, 64, device="cuda").bfloat16()
    Y, idx, gate, counts = mh.mhlmoe_layer(X, W, None, W1, W1, W2, 2)
    torch.cuda.synchronize()
    assert Y.shape == (0, 2, 64) and torch.all(counts == 0)
    idx2, gate2, counts2 = mh.mhlmoe_route(X, W, None, 2)
    torch.cuda.synchronize()
    assert torch.all(counts2 == 0)


# ---------------------------------------------------------------------------
# the 32-bit selection keys at large router logits
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("Ne,k,scale", [(100, 8, 60.0), (200, 6, 60.0), (256, 16, 60.0)])
def test_route_32bit_keys_at_large_logits(Ne, k, scale, oracle_instance):
    """For N_e <= 256 the kernel's selection keys keep the fp32 key's order-
    preserving image above its low b = ceil(log2 N_e) bits, so two keys whose
    relative difference is below 2^(b-23) compare by expert index.  With the
    router weights scaled by 60 (logits of a few hundred), that window
    exceeds the 1e-3 near-tie rule; every row must still select the oracle's
    experts except where the oracle's keys at the boundary (or at a swapped
    pair) lie within max(1e-3, 2^(b-23) |key|) of each other, and the gates of
    rows with the oracle's set are exact to 1e-3."""
    T, Nh, dh = 2048, 2, 128
    w = workloads.generate(workloads.Shape(T, Nh, dh, Ne, k, 32, "bf16", bias="zipf"), seed=8)
    w.W_router = (w.W_router * np.float32(scale)).astype(np.float32)
    announce(f"route large logits Ne={Ne} k={k} scale={scale}")
    d = DeviceWorkload(w)
    idx, gate, counts = mh.mhlmoe_route(d.X, d.W_router, d.bias, k)
    torch.cuda.synchronize()
    r = oracle_instance.route(w.exact("X"), w.exact("W_router"), w.exact("bias"), k=k)
    g_idx = idx.cpu().numpy()
    keys = r["keys"].astype(np.float64)
    b = int(np.ceil(np.log2(Ne)))
    print(f"[large logits] max |key| {np.abs(keys).max():.1f}, window 2^{b - 23} relative", flush=True)
    win = lambda x, y: np.maximum(1e-3, 2.0 ** (b - 23) * np.maximum(np.abs(x), np.abs(y)))
    same_set = np.all(np.sort(g_idx, -1) == np.sort(r["idx"], -1), axis=-1)
    exact = np.all(g_idx == r["idx"], axis=-1)
    bad = 0
    for t, h in zip(*np.nonzero(~exact)):
        if not same_set[t, h]:
            ok = keys.shape[-1] > k and keys[t, h, k - 1] - keys[t, h, k] < win(keys[t, h, k - 1],
                                                                                 keys[t, h, k])
        else:
            # positions that differ sit inside runs of keys within the window
            diff = np.flatnonzero(g_idx[t, h] != r["idx"][t, h])
            kk = keys[t, h, :k]
            near = lambda p, q: kk[p] - kk[q] < win(kk[p], kk[q])
            ok = all((p > 0 and near(p - 1, p)) or (p + 1 < k and near(p, p + 1)) for p in diff)
        bad += not ok
    print(f"[large logits] rows {g_idx.shape[0] * Nh}, inexact {int((~exact).sum())}, "
          f"outside the window {bad}", flush=True)
    assert bad == 0
    gi = np.take_along_axis(gate.cpu().numpy().astype(np.float64), np.argsort(g_idx, -1), -1)
    go = np.take_along_axis(r["gate"], np.argsort(r["idx"], -1), -1)
    assert np.abs(gi - go)[same_set].max() <= 1e-3
