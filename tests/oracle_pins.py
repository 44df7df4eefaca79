"""Pins that tie the CPU oracle to the paper and to mathematics, not to itself.

Each ``pin_*`` function takes an ``oracle.Oracle`` and raises AssertionError
when the oracle disagrees with something fixed independently of it:

  * brute force on tiny inputs (heap selection over numpy logits, numpy's
    stable argsort for the counting sort);
  * the literal dense form of Eq. (1)-(4): every expert evaluated, a softmax
    over all N_e masked scores (scipy), zero weight off the selection;
  * special cases that reduce to textbook routines (N_e = k = 1 is a dense
    SwiGLU MLP; k = N_e is a dense softmax mixture);
  * for the paper's two-matrix GELU expert, Sec. 3.4's own construction:
    block-sparse attention with score_mod(s) = log(gelu(s) + 1), whose output
    times its softmax denominator minus the summed values is the expert;
  * invariants (gates sum to 1, counts sum to T*k, bias invariance,
    head independence, token-permutation equivariance);
  * central finite differences of the forward for the backward.

The same functions run against mutant builds of the oracle (see
test_oracle_mutants.py): every planted mistake must fail at least one pin.
Only numpy and scipy are used here, never the HIP library.
"""
from __future__ import annotations

import heapq

import numpy as np
from scipy.special import expit, softmax
from scipy.stats import norm


# ---------------------------------------------------------------------------
# tiny seeded inputs
# ---------------------------------------------------------------------------

def tiny(seed, T, Nh, dh, Ne, dff, dyadic=False, bias=None):
    """Tiny inputs.  ``dyadic`` draws small multiples of powers of two so that
    every router dot product is exact in fp32 and fp64 whatever the summation
    order (and exact ties appear, exercising the tie-break)."""
    rng = np.random.default_rng(seed)
    if dyadic:
        X = rng.integers(-32, 33, size=(T, Nh, dh)) / 16.0
        W = rng.integers(-64, 65, size=(Nh, Ne, dh)) / 64.0
    else:
        X = rng.standard_normal((T, Nh, dh))
        W = rng.standard_normal((Nh, Ne, dh)) / np.sqrt(dh)
    W = W.astype(np.float32).astype(np.float64)
    W1 = rng.standard_normal((Nh, Ne, dff, dh)) / np.sqrt(dh)
    W3 = rng.standard_normal((Nh, Ne, dff, dh)) / np.sqrt(dh)
    W2 = rng.standard_normal((Nh, Ne, dh, dff)) / np.sqrt(dff)
    b = None
    if bias == "random":
        b = rng.standard_normal((Nh, Ne)).astype(np.float32).astype(np.float64)
    elif bias == "dyadic":
        b = (rng.integers(-16, 17, size=(Nh, Ne)) / 8.0)
    return X, W, b, W1, W3, W2


def np_logits32(X, W):
    """fp32 router scores from numpy (fp64 product, rounded once)."""
    return np.einsum("thd,hed->the", X, W).astype(np.float32)


def np_keys32(X, W, b):
    s = np_logits32(X, W)
    if b is None:
        return s
    return (s + b.astype(np.float32)[None, :, :]).astype(np.float32)


def heap_topk(keys, k):
    """Brute-force arg-top-k per row with heapq: largest key, then lowest
    expert index.  keys: [T, Nh, Ne] -> idx [T, Nh, k]."""
    T, Nh, Ne = keys.shape
    out = np.empty((T, Nh, k), np.int32)
    for t in range(T):
        for h in range(Nh):
            best = heapq.nsmallest(k, ((-float(keys[t, h, e]), e) for e in range(Ne)))
            out[t, h] = [e for _, e in best]
    return out


def all_expert_outputs(X, W1, W3, W2):
    """E_e(x) for every token, head and expert: [T, Nh, Ne, dh] (numpy)."""
    a = np.einsum("thd,hefd->thef", X, W1)
    b = np.einsum("thd,hefd->thef", X, W3)
    u = a * expit(a) * b
    return np.einsum("thef,hedf->thed", u, W2)


def dense_gates(s32, idx):
    """Eq. (2)-(3) literally: g' = s on the selection, -inf elsewhere,
    softmax over all N_e (scipy)."""
    T, Nh, Ne = s32.shape
    gp = np.full((T, Nh, Ne), -np.inf)
    tt, hh = np.meshgrid(np.arange(T), np.arange(Nh), indexing="ij")
    for j in range(idx.shape[2]):
        gp[tt, hh, idx[:, :, j]] = s32[tt, hh, idx[:, :, j]].astype(np.float64)
    return softmax(gp, axis=-1)


def _assert_close(a, b, rtol, what):
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    err = np.max(np.abs(a - b)) / max(np.max(np.abs(b)), 1e-300)
    assert err <= rtol, f"{what}: max rel err {err:.3e} > {rtol:.1e}"


# ---------------------------------------------------------------------------
# pins
# ---------------------------------------------------------------------------

def pin_topk_brute_force_dyadic(o):
    """Selection (Eq. 3 with Algorithm 1's biased key) equals a heap select on
    exact scores; exact ties resolve to the lower expert index."""
    for seed, bias in ((1, None), (2, "dyadic")):
        X, W, b, *_ = tiny(seed, 23, 3, 8, 13, 4, dyadic=True, bias=bias)
        for k in (1, 3, 13):
            r = o.route(X, W, b, k=k)
            want = heap_topk(np_keys32(X, W, b), k)
            assert np.array_equal(r["idx"], want), f"idx mismatch (k={k}, bias={bias})"
    # exact ties are present in this data, so the tie-break was exercised
    keys = np_keys32(*tiny(1, 23, 3, 8, 13, 4, dyadic=True)[:2], None)
    assert any(len(np.unique(row)) < row.size for row in keys.reshape(-1, 13))


def pin_topk_brute_force_gaussian(o):
    """Same as above on Gaussian inputs with a random bias; rows whose fp32
    keys come within 1e-6 of a tie at the selection boundary are skipped
    (fp64 summation order could differ there)."""
    X, W, b, *_ = tiny(3, 41, 2, 16, 17, 4, bias="random")
    k = 5
    r = o.route(X, W, b, k=k)
    keys = np_keys32(X, W, b)
    want = heap_topk(keys, k)
    srt = -np.sort(-keys, axis=-1)
    safe = np.min(np.abs(np.diff(srt[..., : k + 1], axis=-1)), axis=-1) > 1e-6
    assert safe.mean() > 0.9
    assert np.array_equal(r["idx"][safe], want[safe])
    # keys output is the sorted leading keys
    assert np.array_equal(r["keys"][safe], srt[..., : k + 1][safe])


def pin_gates_dense_softmax(o):
    """Gates equal the N_e-wide softmax of Eq. (2) with -inf off the
    selection, taken on the unbiased scores (bias removed, Algorithm 1)."""
    X, W, b, *_ = tiny(4, 19, 3, 8, 9, 4, bias="random")
    k = 4
    r = o.route(X, W, b, k=k)
    sel = heap_topk(np_keys32(X, W, b), k)
    ok = np.all(np.sort(sel, -1) == np.sort(r["idx"], -1), axis=-1)
    assert ok.mean() > 0.9
    g = dense_gates(np_logits32(X, W), r["idx"])
    tt, hh, jj = np.meshgrid(np.arange(19), np.arange(3), np.arange(k), indexing="ij")
    got = np.zeros_like(g)
    got[tt, hh, r["idx"]] = r["gate"]
    _assert_close(got, g, 1e-12, "gates vs dense softmax")


def pin_gates_ignore_bias_values(o):
    """A large non-uniform bias on a chosen set forces that set, and the gates
    are then the softmax of the UNBIASED scores over it."""
    X, W, _, *_ = tiny(5, 11, 2, 8, 10, 4)
    k = 3
    forced = np.array([[7, 2, 5], [0, 9, 4]])
    b = np.zeros((2, 10))
    rng = np.random.default_rng(6)
    for h in range(2):
        b[h, forced[h]] = 100.0 + rng.random(k)
    b = b.astype(np.float32).astype(np.float64)
    r = o.route(X, W, b, k=k)
    for h in range(2):
        assert np.all(np.sort(r["idx"][:, h], -1) == np.sort(forced[h]))
    s = np_logits32(X, W).astype(np.float64)
    for t in range(11):
        for h in range(2):
            want = softmax(s[t, h, r["idx"][t, h]])
            _assert_close(r["gate"][t, h], want, 1e-12, "forced-set gates")


def pin_invariants(o):
    """Gates are positive and sum to 1; counts are the bincount of idx and
    sum to T*k per head; without bias gates come out descending."""
    X, W, b, *_ = tiny(7, 50, 4, 8, 12, 4)
    for k in (1, 4, 12):
        r = o.route(X, W, None, k=k)
        assert np.all(r["gate"] > 0)
        assert np.max(np.abs(r["gate"].sum(-1) - 1.0)) <= 1e-12
        assert np.all(r["counts"].sum(-1) == 50 * k)
        for h in range(4):
            assert np.array_equal(r["counts"][h], np.bincount(r["idx"][:, h].ravel(), minlength=12))
        assert np.all(np.diff(r["gate"], axis=-1) <= 0)
        # each row selects k distinct experts
        assert all(len(set(row)) == k for row in r["idx"].reshape(-1, k))


def pin_bias_constant_shift(o):
    """Adding the same constant to every bias of a head changes neither the
    selection (away from fp32 near-ties) nor the gates."""
    X, W, b, *_ = tiny(8, 30, 2, 8, 11, 4, bias="random")
    k = 4
    r0 = o.route(X, W, b, k=k)
    r1 = o.route(X, W, b + np.array([[0.5], [-0.25]]), k=k)
    gap = np.min(np.abs(np.diff(r0["keys"].astype(np.float64), axis=-1)), axis=-1)
    safe = gap > 1e-5
    assert safe.mean() > 0.9
    assert np.array_equal(r0["idx"][safe], r1["idx"][safe])
    _assert_close(r0["gate"][safe], r1["gate"][safe], 1e-12, "bias shift gates")


def pin_bucket_stable_argsort(o):
    """Token clustering equals numpy's stable argsort of each head's flattened
    (t, j) expert list; offsets are the exclusive scan of the bincount."""
    rng = np.random.default_rng(9)
    T, Nh, k, Ne = 37, 3, 4, 9
    idx = rng.integers(0, Ne, size=(T, Nh, k)).astype(np.int32)
    idx[:, 2, :] = 4                       # one head: every slot to one expert
    offsets, perm = o.bucket(idx, Ne)
    for h in range(Nh):
        flat = idx[:, h, :].ravel()
        assert np.array_equal(perm[h], np.argsort(flat, kind="stable"))
        cnt = np.bincount(flat, minlength=Ne)
        assert np.array_equal(offsets[h], np.concatenate([[0], np.cumsum(cnt)]))


def pin_experts_dense_mixture(o):
    """Sparse Y equals the dense Eq. (1): every expert evaluated (numpy) and
    mixed with the N_e-wide gate vector that is zero off the selection."""
    X, W, b, W1, W3, W2 = tiny(10, 13, 3, 8, 7, 6, bias="random")
    k = 3
    r = o.route(X, W, b, k=k)
    Y = o.experts(X, r["idx"], r["gate"], W1, W3, W2)
    g = dense_gates(np_logits32(X, W), r["idx"])
    Yd = np.einsum("the,thed->thd", g, all_expert_outputs(X, W1, W3, W2))
    _assert_close(Y, Yd, 1e-12, "sparse vs dense mixture")
    Y2, _, _, _ = o.layer(X, W, b, W1, W3, W2, k)
    _assert_close(Y2, Y, 0.0, "layer == route then experts")


def pin_single_expert_is_dense_swiglu(o):
    """N_e = k = 1: gate 1 and Y is the dense SwiGLU MLP W2(silu(W1 x)*(W3 x))."""
    X, W, _, W1, W3, W2 = tiny(11, 9, 2, 8, 1, 5)
    Y, idx, gate, counts = o.layer(X, W, None, W1, W3, W2, 1)
    assert np.all(idx == 0) and np.all(gate == 1.0) and np.all(counts == 9)
    for h in range(2):
        x = X[:, h, :]
        a = x @ W1[h, 0].T
        u = a * expit(a) * (x @ W3[h, 0].T)
        _assert_close(Y[:, h, :], u @ W2[h, 0].T, 1e-12, "dense SwiGLU")


def pin_k_equals_ne_dense_softmax_mixture(o):
    """k = N_e: every expert selected, gates are the plain softmax of all
    scores (scipy) and Y is the dense softmax-gated mixture."""
    X, W, _, W1, W3, W2 = tiny(12, 7, 2, 8, 5, 4)
    Y, idx, gate, _ = o.layer(X, W, None, W1, W3, W2, 5)
    s = np_logits32(X, W).astype(np.float64)
    p = softmax(s, axis=-1)
    tt, hh, _ = np.meshgrid(np.arange(7), np.arange(2), np.arange(5), indexing="ij")
    _assert_close(gate, p[tt, hh, idx], 1e-12, "k=Ne gates")
    Yd = np.einsum("the,thed->thd", p, all_expert_outputs(X, W1, W3, W2))
    _assert_close(Y, Yd, 1e-12, "k=Ne mixture")


def pin_head_independence_and_token_equivariance(o):
    """Heads share nothing (Eq. 6): perturbing head 1's parameters leaves
    head 0 bit-identical.  Tokens are independent: permuting them permutes
    every per-token output bit-identically."""
    X, W, b, W1, W3, W2 = tiny(13, 17, 2, 8, 6, 5, bias="random")
    k = 2
    Y, idx, gate, _ = o.layer(X, W, b, W1, W3, W2, k)
    W_, b_, W1_, W3_, W2_ = (a.copy() for a in (W, b, W1, W3, W2))
    for a in (W_, b_, W1_, W3_, W2_):
        a[1] = a[1] * -1.5 + 0.25
    Yp, idxp, gatep, _ = o.layer(X, W_, b_, W1_, W3_, W2_, k)
    assert np.array_equal(idx[:, 0], idxp[:, 0])
    assert np.array_equal(gate[:, 0], gatep[:, 0])
    assert np.array_equal(Y[:, 0], Yp[:, 0])
    assert not np.array_equal(Y[:, 1], Yp[:, 1])
    p = np.random.default_rng(14).permutation(17)
    Yq, idxq, gateq, _ = o.layer(X[p], W, b, W1, W3, W2, k)
    assert np.array_equal(idxq, idx[p]) and np.array_equal(gateq, gate[p])
    assert np.array_equal(Yq, Y[p])


# ---------------------------------------------------------------------------
# the paper's two-matrix GELU expert (Sec. 3.4)
# ---------------------------------------------------------------------------

def gelu_ref(z):
    """gelu(z) = z * Phi(z), the Gaussian CDF taken from scipy.stats.norm."""
    return z * norm.cdf(z)


def pin_gelu_flexattention_identity(o):
    """Sec. 3.4 writes an expert as block-sparse attention: Q = x, K = the
    expert's W_in rows, V = its W_out columns, score_mod(s) = log(gelu(s) + 1).
    The softmax output O' times the denominator l (the sum of gelu(s_j) + 1),
    minus sum_j V_j, is the expert output.  Built here from numpy, scipy's
    softmax and the normal CDF, and compared with the oracle's GELU experts,
    per slot and gate-weighted."""
    X, W, b, W1, _, W2 = tiny(21, 11, 2, 8, 5, 6, bias="random")
    k = 3
    r = o.route(X, W, b, k=k)
    Y, ys = o.experts_gelu(X, r["idx"], r["gate"], W1, W2, return_slots=True)
    T, Nh, dh = X.shape
    for t in range(T):
        for h in range(Nh):
            acc = np.zeros(dh)
            for j in range(k):
                e = r["idx"][t, h, j]
                K = W1[h, e]                    # [dff][dh]
                V = W2[h, e].T                  # [dff][dh]: neuron f's value row
                m = np.log(gelu_ref(K @ X[t, h]) + 1.0)
                ell = np.sum(np.exp(m))
                y = (softmax(m) @ V) * ell - V.sum(axis=0)
                _assert_close(ys[t, h, j], y, 1e-12, "expert = O' l - 1V")
                acc += r["gate"][t, h, j] * y
            _assert_close(Y[t, h], acc, 1e-12, "gate-weighted GELU combine")
    Y2, idx2, _, _ = o.layer_gelu(X, W, b, W1, W2, k)
    assert np.array_equal(idx2, r["idx"])
    _assert_close(Y2, Y, 0.0, "layer_gelu == route then experts_gelu")


def pin_gelu_unit_expert_values(o):
    """One neuron that reads input coordinate 2 and writes it back
    (W_in = W_out = e_2): y_2 = gelu(x_2), against z Phi(z) from scipy at
    points across the curve; gelu(0) = 0 exactly."""
    z = np.array([-6.0, -3.0, -1.0, -0.5, 0.0, 0.25, 1.0, 2.5, 8.0])
    T = len(z)
    X = np.zeros((T, 1, 4))
    X[:, 0, 2] = z
    Wi = np.zeros((1, 1, 1, 4))
    Wi[0, 0, 0, 2] = 1.0
    Wo = np.zeros((1, 1, 4, 1))
    Wo[0, 0, 2, 0] = 1.0
    idx = np.zeros((T, 1, 1), np.int32)
    gate = np.ones((T, 1, 1))
    Y = o.experts_gelu(X, idx, gate, Wi, Wo)
    _assert_close(Y[:, 0, 2], gelu_ref(z), 1e-14, "gelu values")
    assert Y[4, 0, 2] == 0.0 and np.all(Y[:, 0, [0, 1, 3]] == 0.0)


# ---------------------------------------------------------------------------
# auxiliary-loss-free load balancing (Sec. 2.2)
# ---------------------------------------------------------------------------

def pin_bias_update_rule(o):
    """A head whose loads are all equal keeps its bias exactly; with loads
    3, 2, 1, 1 (mean 7/4, not an integer) the two loaded experts lose the rate
    and the two light ones gain it; each bias moves by one fp32 addition
    (numpy float32 arithmetic), so a step below half an ulp leaves it as is."""
    counts = np.array([[5, 5, 5, 5], [3, 2, 1, 1]], np.int32)
    b0 = np.array([[0.25, -1.0, 3.0, 0.0], [1.0, 1.0, -2.0, 0.5]], np.float32)
    r = np.float32(0.125)
    b = o.bias_update(counts, b0, r)
    assert np.array_equal(b[0], b0[0])
    want = np.array([b0[1, 0] - r, b0[1, 1] - r, b0[1, 2] + r, b0[1, 3] + r], np.float32)
    assert np.array_equal(b[1], want), (b[1], want)
    tiny_rate = np.float32(1e-8)            # < half an ulp of 1.0 in fp32
    b2 = o.bias_update(counts, np.ones((2, 4), np.float32), tiny_rate)
    assert np.array_equal(b2, np.ones((2, 4), np.float32) + tiny_rate)
    assert np.all(b2 == 1.0)


def pin_bias_update_balances_load(o):
    """The method's purpose: starting from a router that favours a few
    experts, alternating routing (with the bias, Algorithm 1) and the update
    shrinks the spread of per-expert loads."""
    rng = np.random.default_rng(31)
    T, Nh, dh, Ne, k = 256, 2, 8, 8, 2
    X = rng.standard_normal((T, Nh, dh))
    W = (rng.standard_normal((Nh, Ne, dh)) / np.sqrt(dh)).astype(np.float32).astype(np.float64)
    W[:, :2, :] += 0.6 * np.sign(X.mean(axis=0))[:, None, :]   # experts 0 and 1 preferred
    b = np.zeros((Nh, Ne), np.float32)
    spread0 = None
    for _ in range(60):
        r = o.route(X, W, b.astype(np.float64), k=k)
        counts = r["counts"]
        spread = (counts.max(axis=1) - counts.min(axis=1)).astype(np.float64)
        spread0 = spread if spread0 is None else spread0
        b = o.bias_update(counts, b, 0.05)
    assert np.all(spread < 0.5 * spread0), (spread0, spread)


def _fd_inputs():
    """Dyadic inputs whose fp32 router scores are exact (so finite differences
    see no fp32 rounding) and whose selection margins all exceed 1e-2."""
    T, Nh, dh, Ne, k, dff = 4, 2, 6, 5, 2, 3
    for seed in range(100, 400):
        X, W, _, W1, W3, W2 = tiny(seed, T, Nh, dh, Ne, dff, dyadic=True)
        srt = -np.sort(-np_logits32(X, W), axis=-1)
        if np.min(np.diff(-srt, axis=-1)) >= 2e-2:
            return (T, Nh, dh, Ne, k, dff), X, W, W1, W3, W2
    raise RuntimeError("no well-separated seed found")


def pin_backward_finite_differences(o):
    """The analytic backward equals central finite differences of
    L = <dY, Y(X, W_router, W1, W3, W2)> computed with the forward oracle
    (selection held by margins > 1e-2; step 2^-10 keeps router scores exact
    in fp32)."""
    (T, Nh, dh, Ne, k, dff), X, W, W1, W3, W2 = _fd_inputs()
    dY = np.random.default_rng(15).standard_normal((T, Nh, dh))
    Y, idx, gate, _ = o.layer(X, W, None, W1, W3, W2, k)
    g = o.layer_backward(X, W, W1, W3, W2, idx, gate, dY)
    step = 2.0 ** -10
    params = {"X": X, "W_router": W, "W1": W1, "W3": W3, "W2": W2}

    def loss(p):
        Yp, idxp, _, _ = o.layer(p["X"], p["W_router"], None, p["W1"], p["W3"], p["W2"], k)
        assert np.array_equal(idxp, idx), "selection moved under the FD step"
        return float(np.sum(dY * Yp))

    for name, grad_name in (("X", "dX"), ("W_router", "dW_router"),
                            ("W1", "dW1"), ("W3", "dW3"), ("W2", "dW2")):
        base = params[name]
        fd = np.empty_like(base)
        for i in range(base.size):
            plus = dict(params)
            minus = dict(params)
            bp = base.copy().ravel()
            bm = base.copy().ravel()
            bp[i] += step
            bm[i] -= step
            plus[name] = bp.reshape(base.shape)
            minus[name] = bm.reshape(base.shape)
            fd.ravel()[i] = (loss(plus) - loss(minus)) / (2 * step)
        err = np.max(np.abs(fd - g[grad_name])) / max(np.max(np.abs(fd)), 1e-12)
        assert err < 2e-5, f"{grad_name}: FD rel err {err:.2e}"
    # experts that received no slot have exactly zero gradient
    used = np.zeros((Nh, Ne), bool)
    for h in range(Nh):
        used[h, np.unique(idx[:, h])] = True
    for name in ("dW_router", "dW1", "dW3", "dW2"):
        assert np.all(g[name][~used] == 0.0)


def pin_route_backward_finite_differences(o):
    """Algorithm 2 on its own: for L = sum c * gate(X, W_router) with the
    selection held, dX and dW_router equal central finite differences
    through the forward oracle (dyadic inputs keep the fp32 scores exact);
    and its dS is the layer backward's dS when the gate gradient is
    <dY, y_j> (the chain rule through Eq. (1))."""
    (T, Nh, dh, Ne, k, dff), X, W, W1, W3, W2 = _fd_inputs()
    c = np.random.default_rng(19).standard_normal((T, Nh, k))
    r = o.route(X, W, None, k=k)
    g = o.route_backward(X, W, r["idx"], r["gate"], c, return_dS=True)
    step = 2.0 ** -10

    def loss(Xp, Wp):
        rp = o.route(Xp, Wp, None, k=k)
        assert np.array_equal(rp["idx"], r["idx"]), "selection moved under the FD step"
        return float(np.sum(c * rp["gate"]))

    for name, grad in (("X", "dX"), ("W_router", "dW_router")):
        base = X if name == "X" else W
        fd = np.empty_like(base)
        for i in range(base.size):
            bp = base.copy().ravel()
            bm = base.copy().ravel()
            bp[i] += step
            bm[i] -= step
            args_p = (bp.reshape(base.shape), W) if name == "X" else (X, bp.reshape(base.shape))
            args_m = (bm.reshape(base.shape), W) if name == "X" else (X, bm.reshape(base.shape))
            fd.ravel()[i] = (loss(*args_p) - loss(*args_m)) / (2 * step)
        err = np.max(np.abs(fd - g[grad])) / max(np.max(np.abs(fd)), 1e-12)
        assert err < 2e-5, f"route {grad}: FD rel err {err:.2e}"
    dY = np.random.default_rng(20).standard_normal((T, Nh, dh))
    _, ys = o.experts(X, r["idx"], r["gate"], W1, W3, W2, return_slots=True)
    dgate = np.einsum("thd,thjd->thj", dY, ys)
    lb = o.layer_backward(X, W, W1, W3, W2, r["idx"], r["gate"], dY, return_dS=True)
    rb = o.route_backward(X, W, r["idx"], r["gate"], dgate, return_dS=True)
    assert np.allclose(rb["dS"], lb["dS"], rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(rb["dW_router"], lb["dW_router"], rtol=1e-11, atol=1e-13)


def pin_gelu_backward_finite_differences(o):
    """The GELU expert's backward (Sec. 3.4's two-matrix expert) equals
    central finite differences of L = <dY, Y(X, W_router, W_in, W_out)>
    through the forward oracle; its dW_in / dW_out of experts without slots
    are exactly zero."""
    (T, Nh, dh, Ne, k, dff), X, W, Wi, _, Wo = _fd_inputs()
    dY = np.random.default_rng(18).standard_normal((T, Nh, dh))
    Y, idx, gate, _ = o.layer_gelu(X, W, None, Wi, Wo, k)
    g = o.layer_backward(X, W, Wi, None, Wo, idx, gate, dY)
    assert "dW3" not in g
    step = 2.0 ** -10
    params = {"X": X, "W_router": W, "W_in": Wi, "W_out": Wo}

    def loss(p):
        Yp, idxp, _, _ = o.layer_gelu(p["X"], p["W_router"], None, p["W_in"], p["W_out"], k)
        assert np.array_equal(idxp, idx), "selection moved under the FD step"
        return float(np.sum(dY * Yp))

    for name, grad in (("X", "dX"), ("W_router", "dW_router"), ("W_in", "dW1"),
                       ("W_out", "dW2")):
        base = params[name]
        fd = np.empty_like(base)
        for i in range(base.size):
            bp = base.copy().ravel()
            bm = base.copy().ravel()
            bp[i] += step
            bm[i] -= step
            fd.ravel()[i] = (loss({**params, name: bp.reshape(base.shape)}) -
                             loss({**params, name: bm.reshape(base.shape)})) / (2 * step)
        err = np.max(np.abs(fd - g[grad])) / max(np.max(np.abs(fd)), 1e-12)
        assert err < 2e-5, f"GELU {grad}: FD rel err {err:.2e}"
    used = np.zeros((Nh, Ne), bool)
    for h in range(Nh):
        used[h, np.unique(idx[:, h])] = True
    for name in ("dW_router", "dW1", "dW2"):
        assert np.all(g[name][~used] == 0.0)


def pin_routed_backward_finite_differences(o):
    """Separate routing sub-tokens (Sec. 4.4): with L = <dY, Y(X, R)> where
    the router reads R and the experts read X, the returned dX and dR equal
    central finite differences taken in X and in R separately, dW_router that
    taken in W_router, and the expert weight gradients match those of the
    shared-input backward at the same selection."""
    (T, Nh, dh, Ne, k, dff), X, W, W1, W3, W2 = _fd_inputs()
    # R: a second dyadic input with the same well-separated routing margins
    R = None
    for seed in range(400, 700):
        Rc = tiny(seed, T, Nh, dh, Ne, dff, dyadic=True)[0]
        srt = -np.sort(-np_logits32(Rc, W), axis=-1)
        if np.min(np.diff(-srt, axis=-1)) >= 2e-2:
            R = Rc
            break
    assert R is not None
    dY = np.random.default_rng(16).standard_normal((T, Nh, dh))
    Y, idx, gate, _ = o.layer_routed(X, R, W, None, W1, W3, W2, k)
    g = o.layer_backward(X, W, W1, W3, W2, idx, gate, dY, R=R)
    step = 2.0 ** -10
    params = {"X": X, "R": R, "W_router": W}

    def loss(p):
        Yp, idxp, _, _ = o.layer_routed(p["X"], p["R"], p["W_router"], None, W1, W3, W2, k)
        assert np.array_equal(idxp, idx), "selection moved under the FD step"
        return float(np.sum(dY * Yp))

    for name, grad_name in (("X", "dX"), ("R", "dR"), ("W_router", "dW_router")):
        base = params[name]
        fd = np.empty_like(base)
        for i in range(base.size):
            bp = base.copy().ravel()
            bm = base.copy().ravel()
            bp[i] += step
            bm[i] -= step
            fd.ravel()[i] = (loss({**params, name: bp.reshape(base.shape)}) -
                             loss({**params, name: bm.reshape(base.shape)})) / (2 * step)
        err = np.max(np.abs(fd - g[grad_name])) / max(np.max(np.abs(fd)), 1e-12)
        assert err < 2e-5, f"{grad_name}: FD rel err {err:.2e}"
    shared = o.layer_backward(X, W, W1, W3, W2, idx, gate, dY)
    for name in ("dW1", "dW3", "dW2"):
        assert np.array_equal(g[name], shared[name]), name


# ---------------------------------------------------------------------------
# the projections around the heads (Eq. (5)-(6), Eq. (9))
# ---------------------------------------------------------------------------

def pin_round_bf16(o):
    """bfloat16 keeps 8 significant bits with ties to even: 1 + 2^-8 (half
    way, even neighbour 1) -> 1; 1 + 3 2^-8 -> 1 + 2^-6; just above half way
    rounds up; and on fp32 values it equals torch's float32 -> bfloat16
    conversion (a library routine of its own)."""
    from oracle import round_bf16
    assert round_bf16(1.0 + 2.0 ** -8) == 1.0
    assert round_bf16(1.0 + 3 * 2.0 ** -8) == 1.0 + 2.0 ** -6
    assert round_bf16(1.0 + 2.0 ** -8 + 2.0 ** -30) == 1.0 + 2.0 ** -7
    assert round_bf16(-(1.0 + 2.0 ** -8 + 2.0 ** -30)) == -(1.0 + 2.0 ** -7)
    assert round_bf16(3.0 * 2.0 ** -100) == 3.0 * 2.0 ** -100
    import torch
    rng = np.random.default_rng(3)
    v = (rng.standard_normal(50000) * np.exp(rng.uniform(-30, 30, 50000))).astype(np.float32)
    want = torch.from_numpy(v).bfloat16().double().numpy()
    assert np.array_equal(round_bf16(v.astype(np.float64)), want)


def pin_latent_identity_projections(o):
    """With W_in = I and W_out = I (d_model = N) the latent layer is the
    per-head layer on x read as [T, N_h, d_h] (Eq. (5)'s split is that view),
    exactly; with W_in = [I; P] for a permutation P of the latent coordinates
    the router reads the permuted sub-tokens (Eq. (9)) and the result is
    layer_routed on them."""
    T, Nh, dh, Ne, k, dff = 16, 2, 8, 6, 2, 16
    N = Nh * dh
    X, W, b, W1, W3, W2 = tiny(41, T, Nh, dh, Ne, dff, bias="random")
    x = X.reshape(T, N)
    eye = np.eye(N)
    r = o.latent_layer(x, eye, W, b, W1, W3, W2, eye, Nh, k)
    Y, idx, gate, counts = o.layer(X, W, b, W1, W3, W2, k)
    assert np.array_equal(r["X_lat"], X)
    assert np.array_equal(r["idx"], idx) and np.array_equal(r["gate"], gate)
    assert np.array_equal(r["out"], Y.reshape(T, N))
    p = np.random.default_rng(42).permutation(N)
    Pm = eye[p]                               # (Pm x)[i] = x[p[i]]
    rr = o.latent_layer(x, np.concatenate([eye, Pm]), W, b, W1, W3, W2, eye, Nh, k,
                        routing_tokens=True)
    Rt = x[:, p].reshape(T, Nh, dh)
    Yr, idr, gr, _ = o.layer_routed(X, Rt, W, b, W1, W3, W2, k)
    assert np.array_equal(rr["R_lat"], Rt)
    assert np.array_equal(rr["idx"], idr) and np.array_equal(rr["out"], Yr.reshape(T, N))
    assert not np.array_equal(idr, idx), "the permutation should change some routes"


def _latent_fd_inputs(routing_tokens):
    """Dyadic x, W_in and W_router whose router scores stay exact in fp32
    under the finite-difference steps (multiples of 2^-20 below 16 in
    magnitude), with margins > 2e-2 among the k + 1 best scores (so the
    selection and its order hold)."""
    T, d, Nh, dh, Ne, k, dff = 3, 5, 2, 4, 5, 2, 3
    N = Nh * dh
    rows = (2 if routing_tokens else 1) * N
    for seed in range(500, 900):
        rng = np.random.default_rng(seed)
        x = rng.integers(-8, 9, size=(T, d)) / 8.0
        W_in = rng.integers(-8, 9, size=(rows, d)) / 16.0
        Wr = rng.integers(-64, 65, size=(Nh, Ne, dh)) / 64.0
        W1 = rng.standard_normal((Nh, Ne, dff, dh)) / 2.0
        W3 = rng.standard_normal((Nh, Ne, dff, dh)) / 2.0
        W2 = rng.standard_normal((Nh, Ne, dh, dff)) / np.sqrt(dff)
        W_out = rng.standard_normal((d, N)) / np.sqrt(N)
        lat = x @ W_in.T
        R = (lat[:, N:] if routing_tokens else lat[:, :N]).reshape(T, Nh, dh)
        srt = -np.sort(-np_logits32(R, Wr), axis=-1)[..., :k + 1]
        if np.min(np.diff(-srt, axis=-1)) >= 2e-2:
            return (Nh, k), x, W_in, Wr, W1, W3, W2, W_out
    raise RuntimeError("no well-separated seed found")


def pin_latent_backward_finite_differences(o):
    """The latent backward's dx, dW_in and dW_out (with and without routing
    sub-tokens) equal central finite differences of L = <dout, out(x, W_in,
    W_out)> through the forward oracle (selection held by the margins)."""
    for rt in (False, True):
        (Nh, k), x, W_in, Wr, W1, W3, W2, W_out = _latent_fd_inputs(rt)
        dout = np.random.default_rng(17).standard_normal((x.shape[0], W_out.shape[0]))
        f = o.latent_layer(x, W_in, Wr, None, W1, W3, W2, W_out, Nh, k, routing_tokens=rt)
        g = o.latent_layer_backward(x, W_in, Wr, W1, W3, W2, W_out, f["X_lat"], f["R_lat"],
                                    f["Y_lat"], f["idx"], f["gate"], dout, routing_tokens=rt)
        params = {"x": x, "W_in": W_in, "W_out": W_out}
        step = 2.0 ** -10

        def loss(p):
            r = o.latent_layer(p["x"], p["W_in"], Wr, None, W1, W3, W2, p["W_out"], Nh, k,
                               routing_tokens=rt)
            assert np.array_equal(r["idx"], f["idx"]), "selection moved under the FD step"
            return float(np.sum(dout * r["out"]))

        for name, grad in (("x", "dx"), ("W_in", "dW_in"), ("W_out", "dW_out")):
            base = params[name]
            fd = np.empty_like(base)
            for i in range(base.size):
                bp = base.copy().ravel()
                bm = base.copy().ravel()
                bp[i] += step
                bm[i] -= step
                fd.ravel()[i] = (loss({**params, name: bp.reshape(base.shape)}) -
                                 loss({**params, name: bm.reshape(base.shape)})) / (2 * step)
            err = np.max(np.abs(fd - g[grad])) / max(np.max(np.abs(fd)), 1e-12)
            assert err < 2e-5, f"routing_tokens={rt} {grad}: FD rel err {err:.2e}"


ALL_PINS = [
    pin_topk_brute_force_dyadic,
    pin_topk_brute_force_gaussian,
    pin_gates_dense_softmax,
    pin_gates_ignore_bias_values,
    pin_invariants,
    pin_bias_constant_shift,
    pin_bucket_stable_argsort,
    pin_experts_dense_mixture,
    pin_single_expert_is_dense_swiglu,
    pin_k_equals_ne_dense_softmax_mixture,
    pin_head_independence_and_token_equivariance,
    pin_backward_finite_differences,
    pin_routed_backward_finite_differences,
    pin_gelu_backward_finite_differences,
    pin_route_backward_finite_differences,
    pin_gelu_flexattention_identity,
    pin_gelu_unit_expert_values,
    pin_bias_update_rule,
    pin_bias_update_balances_load,
    pin_round_bf16,
    pin_latent_identity_projections,
    pin_latent_backward_finite_differences,
]
