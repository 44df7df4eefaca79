"""Helpers for the GPU parity tests: device upload/download of workloads and
the comparison rules (spec tolerances)."""
from __future__ import annotations

import functools
import sys

import numpy as np
import pytest
import torch

import workloads

GATE_ATOL = 1e-3          # gates: absolute
TIE_GAP = 1e-3            # idx may differ only where the oracle's keys are this close
REL_L2 = {"bf16": 2e-2, "f32": 1e-4}

needs_gpu = pytest.mark.skipif(not torch.cuda.is_available(), reason="needs a GPU")


def announce(msg: str):
    """Name the case before a GPU step (so a crash still says what ran)."""
    print(f"[case] {msg}", flush=True)
    sys.stdout.flush()


to_device = workloads.to_device


def to_host_f64(t: torch.Tensor) -> np.ndarray:
    if t.dtype == torch.bfloat16:
        return t.float().cpu().numpy().astype(np.float64)
    return t.cpu().numpy().astype(np.float64)


@functools.lru_cache(maxsize=2)
def workload(name: str, seed: int = 0) -> workloads.Workload:
    return workloads.generate(workloads.CONFIGS[name], seed)


class DeviceWorkload:
    def __init__(self, w: workloads.Workload):
        self.w = w
        self.X = to_device(w.X)
        self.W_router = to_device(w.W_router)
        self.bias = to_device(w.bias)
        self.W1 = to_device(w.W1)
        self.W3 = to_device(w.W3)
        self.W2 = to_device(w.W2)
        self.dY = to_device(w.dY) if w.dY is not None else None


def rel_l2(got: np.ndarray, want: np.ndarray) -> float:
    return float(np.linalg.norm((got - want).ravel()) / max(np.linalg.norm(want.ravel()), 1e-300))


def classify_routing(g_idx, o_idx, o_keys, k):
    """Per (row, head): 'exact', 'order' (same set, order differs only among
    oracle keys closer than TIE_GAP), 'tie' (set differs and the oracle's
    k-th and (k+1)-th keys differ by less than TIE_GAP) or 'bad'."""
    exact = np.all(g_idx == o_idx, axis=-1)
    same_set = np.all(np.sort(g_idx, -1) == np.sort(o_idx, -1), axis=-1)
    keys = o_keys.astype(np.float64)
    nk = keys.shape[-1]
    if nk > k:
        boundary_tie = (keys[..., k - 1] - keys[..., k]) < TIE_GAP
    else:
        boundary_tie = np.zeros(exact.shape, bool)
    inner_gaps = keys[..., : k - 1] - keys[..., 1:k] if k > 1 else np.zeros(exact.shape + (0,))
    # positions where the order differs must sit inside a run of near-equal keys
    diff_pos = g_idx != o_idx
    near_next = np.concatenate([inner_gaps < TIE_GAP, np.zeros(exact.shape + (1,), bool)], -1)
    near_prev = np.concatenate([np.zeros(exact.shape + (1,), bool), inner_gaps < TIE_GAP], -1)
    order_ok = np.all(~diff_pos | near_next | near_prev, axis=-1)
    cls = np.full(exact.shape, "bad", dtype=object)
    cls[~exact & ~same_set & boundary_tie] = "tie"
    cls[~exact & same_set & order_ok] = "order"
    cls[exact] = "exact"
    return cls


def check_routing(g_idx, g_gate, o_idx, o_gate, o_keys, k, what=""):
    """Assert the spec rule; return the boolean mask of rows whose
    selection matches as a set (usable for output comparison)."""
    cls = classify_routing(g_idx, o_idx, o_keys, k)
    n_bad = int(np.sum(cls == "bad"))
    counts = {c: int(np.sum(cls == c)) for c in ("exact", "order", "tie", "bad")}
    print(f"[routing] {what} rows={cls.size} {counts}", flush=True)
    assert n_bad == 0, f"{what}: {n_bad} (token, head) rows select different experts without a near tie"
    assert counts["tie"] + counts["order"] <= max(8, 0.05 * cls.size), f"{what}: too many excused rows {counts}"
    ok = (cls == "exact") | (cls == "order")
    # gates compared per expert (sorted by index) where the sets agree
    gi = np.argsort(g_idx, -1)
    oi = np.argsort(o_idx, -1)
    gg = np.take_along_axis(g_gate, gi, -1)
    og = np.take_along_axis(o_gate, oi, -1)
    err = np.abs(gg - og)[ok]
    gmax = float(err.max()) if err.size else 0.0
    print(f"[routing] {what} max |gate err| = {gmax:.3e}", flush=True)
    assert gmax <= GATE_ATOL, f"{what}: gate error {gmax} > {GATE_ATOL}"
    return ok


# ---------------------------------------------------------------------------
# Localised checks beside the pooled relative L2 (a pooled figure over many
# rows can hide one wrong row or one wrong expert).
# ---------------------------------------------------------------------------

# Largest relative error of a single output row (token, head) or of one
# (head, expert) gradient block.  bf16: the path rounds three times on the way
# to an output (the intermediate h, the per-slot output, the final sum), each
# with a relative error of at most 2^-9 per element; over a d_h-wide row the
# errors average towards ~4e-3 RMS, so a row at 5e-2 is more than ten such
# roundings off and a wholly wrong row (relative error ~1) fails by far.
ROW_REL = {"bf16": 5e-2, "f32": 1e-3}
# Rows (blocks) are measured against max(own norm, FLOOR x a reference scale),
# so that a row whose true value nearly cancels is held to the absolute error
# its rounded terms allow rather than to a relative one.
FLOOR = 0.1


def check_rows(got, want, dtype, what, tol=None):
    """Pooled rel-L2 <= REL_L2[dtype] and every row (last axis) within
    ROW_REL[dtype] of max(||want_row||, FLOOR x RMS row norm).  Returns
    (pooled, worst row)."""
    g = np.asarray(got, np.float64).reshape(-1, np.shape(got)[-1])
    w = np.asarray(want, np.float64).reshape(-1, np.shape(want)[-1])
    pooled = rel_l2(g, w)
    if g.shape[0] == 0:
        return pooled, 0.0
    rn = np.linalg.norm(w, axis=1)
    en = np.linalg.norm(g - w, axis=1)
    scale = max(float(np.sqrt(np.mean(rn * rn))), 1e-300)
    rel = en / np.maximum(rn, FLOOR * scale)
    worst = float(rel.max())
    over = int(np.sum(rel > REL_L2[dtype]))
    print(f"[rows] {what}: pooled {pooled:.3e}, worst row {worst:.3e} (row {int(rel.argmax())}), "
          f"{over} of {len(rel)} rows above {REL_L2[dtype]}", flush=True)
    assert pooled <= (tol or REL_L2[dtype]), f"{what}: pooled rel-L2 {pooled:.3e}"
    assert worst <= ROW_REL[dtype], f"{what}: row {int(rel.argmax())} rel {worst:.3e} > {ROW_REL[dtype]}"
    return pooled, worst


def check_expert_blocks(got, want, counts, what, dtype="bf16"):
    """Per (head, expert) check of a weight gradient [Nh][Ne][...] given the
    slot counts [Nh][Ne]: experts without slots must be exactly zero; every
    other block within ROW_REL[dtype] of max(||want_he||, FLOOR x
    sqrt(c_he / S_h) x ||want_h||) (S_h the head's slots: the norm a block
    of c_he independent slot contributions would have), so a cold expert is
    held to its own size rather than drowned by the hot ones.  Pooled rel-L2
    over the tensor <= REL_L2[dtype]."""
    g = np.asarray(got, np.float64)
    w = np.asarray(want, np.float64)
    Nh, Ne = counts.shape
    g = g.reshape(Nh, Ne, -1)
    w = w.reshape(Nh, Ne, -1)
    pooled = rel_l2(g, w)
    empty = counts == 0
    assert not np.any(g[empty] != 0), f"{what}: an expert without slots has a non-zero gradient"
    bn = np.linalg.norm(w, axis=2)
    en = np.linalg.norm(g - w, axis=2)
    hn = np.linalg.norm(w.reshape(Nh, -1), axis=1)[:, None]
    S = np.maximum(counts.sum(axis=1, keepdims=True), 1)
    ref = np.maximum(bn, FLOOR * np.sqrt(counts / S) * hn)
    rel = np.where(empty, 0.0, en / np.maximum(ref, 1e-300))
    h, e = np.unravel_index(int(rel.argmax()), rel.shape)
    worst = float(rel.max())
    print(f"[experts] {what}: pooled {pooled:.3e}, worst (head {h}, expert {e}, {counts[h, e]} slots) "
          f"{worst:.3e} over {int((~empty).sum())} experts with slots", flush=True)
    assert pooled <= REL_L2[dtype], f"{what}: pooled rel-L2 {pooled:.3e}"
    assert worst <= ROW_REL[dtype], f"{what}: head {h} expert {e} rel {worst:.3e} > {ROW_REL[dtype]}"
    return pooled, worst
