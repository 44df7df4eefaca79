"""The seeded input recipe: bf16 rounding and the Zipf skew convention."""
import json
import os

import numpy as np
import pytest
import torch

import workloads

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "zipf_skew.json")


def test_bf16_rounding_matches_torch():
    rng = np.random.default_rng(0)
    a = np.concatenate([rng.standard_normal(100000).astype(np.float32) * 10.0 ** rng.integers(-6, 6, 100000),
                        np.array([0.0, -0.0, 1.0, -1.0, 3.0e38, 1.0 + 2.0 ** -8, 1.0 + 3 * 2.0 ** -8], np.float32)])
    a = a.astype(np.float32)
    ours = workloads.f32_to_bf16_bits(a)
    ref = torch.from_numpy(a).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(ours, ref)
    assert np.array_equal(workloads.bf16_bits_to_f32(ours),
                          torch.from_numpy(ours.view(np.int16)).view(torch.bfloat16).float().numpy())


def test_zipf_convention_reproduces_paper_figure():
    g = json.load(open(GOLDEN))
    n, shards = g["n_experts"], g["n_shards"]
    r = np.arange(1, n + 1, dtype=np.float64)
    for skew, want in g["share_of_first_shard"].items():
        p = r ** -float(skew)
        share = p[: n // shards].sum() / p.sum()
        assert round(share, g["printed_decimals"]) == want


def test_zipf_bias_is_log_rank_weight():
    """exp(b) normalised is the Zipf pmf over each head's seeded rank order."""
    rng = np.random.default_rng(0)
    b = workloads.zipf_bias(rng, 3, 50, 1.1)
    for h in range(3):
        w = np.exp(b[h].astype(np.float64))
        order = np.argsort(-w)
        ranks = np.arange(1, 51, dtype=np.float64)
        np.testing.assert_allclose(w[order] / w.sum(), ranks ** -1.1 / np.sum(ranks ** -1.1), rtol=1e-6)
        assert b[h].max() == 0.0


def test_generate_is_seeded_and_shaped():
    s = workloads.CONFIGS["tiny_f32_t256"]
    a, b = workloads.generate(s, 0), workloads.generate(s, 0)
    assert np.array_equal(a.X, b.X) and np.array_equal(a.W2, b.W2)
    assert a.X.shape == (256, 4, 64) and a.X.dtype == np.float32
    assert a.W1.shape == (4, 16, 128, 64) and a.W2.shape == (4, 16, 64, 128)
    s2 = workloads.Shape(33, 2, 64, 8, 2, 128, "bf16", bias="zipf", backward=True)
    w = workloads.generate(s2, 3)
    assert w.X.dtype == np.uint16 and w.W_router.dtype == np.float32
    assert w.bias.shape == (2, 8) and w.dY.shape == (33, 2, 64)
    np.testing.assert_allclose(np.std(w.exact("X")), 1.0, rtol=0.1)


def test_sample_rows_covers_both_ends():
    rows = workloads.sample_rows(1000, 50)
    assert rows[0] == 0 and rows[-1] == 999 and len(rows) == 50
    assert np.all(np.diff(rows) > 0)
