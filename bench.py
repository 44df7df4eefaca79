#!/usr/bin/env python3
"""Benchmark of the Multi-Head LatentMoE per-GPU hot path (libmhlmoe).

One step = one `mhlmoe_layer` forward (routing, clustering, grouped SwiGLU
experts, combine) over the whole workload (`mhlmoe_layer_gelu`, the paper's
two-matrix GELU expert, for the gelu_* workloads), followed, for the workload that
trains (skewed_bf16_t65536_e1024), by one `mhlmoe_layer_backward` on a fixed dY;
the metric is routed tokens per second per MoE layer on one GPU.  Inputs are synthetic, seeded, and resident
in device memory before the timed region.  To keep the 256 MB Infinity Cache
from serving a step with the previous step's data, the steps cycle through
several copies of the inputs (weights and activations) totalling > 512 MB.

Prints ONE JSON line with, beside the throughput:
  roofline      the dominant kernel (the grouped expert FFN) against the
                roof that bounds it: bf16 MFMA peak (algorithmic flops per
                launch / the kernel's mean duration) or, for workloads below
                the ridge point (few slots per expert), HBM peak (algorithmic
                bytes per launch / duration); durations measured with HIP
                events recorded by the library on the stream the kernel runs
                on, over the timed steps;
  cpu_baseline  the CPU oracle on this host, on the same workload;
  kernels       every kernel's mean duration; route_roofline the routing
                kernel against HBM bandwidth.

    python bench.py [--steps K] [--warmup W] [--workload bf16_t4096_e64]
"""
from __future__ import annotations

import argparse
import dataclasses
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

# Published MI355X peaks (dense).
PEAK_HBM_GBS = 8000.0
PEAK_TFLOPS = {"bf16": 2516.6, "f32": 157.3}
MALL_BYTES = 256 << 20

KERNELS = ("route_fwd", "hist", "count_scan", "scatter", "ffn", "combine", "bwd_dx",
           "bwd_combine", "bwd_dw", "router_dw")
# MFMA flops per slot, in units of d_h * d_ff, that each kernel must do at the
# least: the forward FFN's two GEMMs (W1, W3: 4; W2: 2); in the backward the
# recomputed W1/W3 products, v = W2^T dy and dX = W1^T da + W3^T db are
# charged to bwd_dx (4 + 2 + 4) and only the weight gradients (dW1, dW3: 4;
# dW2: 2) to bwd_dw, whose own recomputation is overhead.
ALGO_FLOPS = {"ffn": 6.0, "bwd_dx": 10.0, "bwd_dw": 6.0}
EXEC_FLOPS = {"ffn": 6.0, "bwd_dx": 10.0, "bwd_dw": 12.0}


def parse_args(argv=None):
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--workload", default="bf16_t4096_e64")
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--sets", type=int, default=0,
                    help="input copies cycled through (0 = enough to exceed 2x the MALL)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=10.0,
                    help="minimum CPU-oracle time for the baseline")
    ap.add_argument("--copy-calibration-mib", type=int, default=0,
                    help="also run one device-to-device copy of this many MiB "
                         "(reference kernel for rocprofv3 FETCH_SIZE/WRITE_SIZE scaling)")
    ap.add_argument("--backward", action="store_true",
                    help="add one mhlmoe_layer_backward to every step of a forward-only "
                         "workload (to profile the backward kernels at its shape)")
    ap.add_argument("--traffic", default=os.path.join(ROOT, "profiles", "ffn_traffic.json"),
                    help="measured HBM traffic summary to attach (if it matches the kernel source)")
    return ap.parse_args(argv)


def algorithmic(shape):
    """Algorithmic bytes / flops per launch of the route and FFN kernels."""
    e = 4 if shape.dtype == "f32" else 2
    T, Nh, dh, Ne, k, dff = (shape.T, shape.n_heads, shape.d_head, shape.n_experts,
                            shape.top_k, shape.d_ff)
    slots = T * Nh * k
    route_bytes = (T * Nh * dh * e + Nh * Ne * dh * 4 + (Nh * Ne * 4 if shape.bias != "none" else 0)
                   + slots * 4 * 2 + Nh * Ne * 4)
    nmat = ffn_matrices(shape)
    ffn_flops = 2 * nmat * slots * dh * dff
    ffn_bytes = nmat * Nh * Ne * dh * dff * e + T * Nh * dh * e * 2 + slots * (4 + 4)
    return route_bytes, ffn_flops, ffn_bytes


def ffn_bound(mfma, nbytes, peak_tflops):
    """Which roof bounds the FFN: its algorithmic flops at the MFMA peak, or
    its algorithmic bytes (each expert's weights read once, X read and Y
    written once) at the HBM peak, whichever takes longer.  Below the ridge
    point (peak flops / peak bandwidth, ~315 flop/B for bf16) the kernel is
    HBM-bound: few slots per expert leave every weight byte with little work.
    Returns the fields that replace the MFMA-only roofline when HBM bounds,
    and both fractions either way."""
    us = mfma["mean_us"]
    gbs = nbytes / (us * 1e-6) / 1e9
    intensity = mfma["flops_per_launch"] / nbytes
    ridge = peak_tflops * 1e12 / (PEAK_HBM_GBS * 1e9)
    out = {"flop_per_byte": round(intensity, 1), "ridge_flop_per_byte": round(ridge, 1),
           "frac_mfma": mfma["frac"], "frac_hbm": round(gbs / PEAK_HBM_GBS, 4)}
    if intensity < ridge:
        out.update({"bound": "hbm", "achieved": round(gbs, 1), "peak": PEAK_HBM_GBS,
                    "unit": "GB/s", "frac": out["frac_hbm"]})
    return out


def ffn_matrices(shape):
    """Weight matrices per expert: 3 (SwiGLU) or 2 (the GELU expert)."""
    return 2 if shape.expert == "gelu" else 3


def kernel_source_digest():
    import hashlib
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2602_04870_amd", "csrc")
    for name in ("experts.hip", "ffn_common.hpp", "device_common.hpp", "launch.hpp"):
        with open(os.path.join(csrc, name), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def load_traffic(path, workload, launches_bytes):
    """HBM bytes per FFN launch from a committed rocprofv3 counter summary,
    or None when absent or taken on a different kernel source."""
    try:
        with open(path) as f:
            t = json.load(f)
    except (OSError, ValueError):
        return None
    entry = t.get(workload)
    if not entry or entry.get("kernel_source") != kernel_source_digest():
        return None
    return entry.get("bytes_per_launch")


def cpu_baseline(w, min_seconds, backward):
    """Time the CPU oracle on the workload (the whole layer forward, plus its
    backward when the workload trains).  Tokens are independent in every
    per-token step, so a seeded sample of rows is timed: the sample grows
    from 64 rows until one pass takes >= min_seconds / 4 or covers the whole
    workload, then passes are repeated until min_seconds have elapsed (at
    most 8 passes)."""
    import oracle
    import workloads
    o = oracle.Oracle()
    s = w.shape
    Wr, b = w.exact("W_router"), w.exact("bias")
    W1, W3, W2 = w.exact("W1"), w.exact("W3"), w.exact("W2")

    def one_pass(rows):
        X = w.exact("X", rows)
        t0 = time.perf_counter()
        if s.expert == "gelu":
            _, idx, gate, _ = o.layer_gelu(X, Wr, b, W1, W2, s.top_k)
        else:
            _, idx, gate, _ = o.layer(X, Wr, b, W1, W3, W2, s.top_k)
        if backward:
            o.layer_backward(X, Wr, W1, W3, W2, idx, gate, w.exact("dY", rows))
        return time.perf_counter() - t0

    n = min(64, s.T)
    while True:
        rows = workloads.sample_rows(s.T, n, seed=99)
        dt = one_pass(rows)
        if dt >= min_seconds / 4 or len(rows) == s.T:
            break
        n = min(s.T, max(2 * n, int(n * (min_seconds / 4) / max(dt, 1e-3))))
    passes, elapsed = 1, dt
    while passes < 8 and elapsed < min_seconds:
        elapsed += one_pass(rows)
        passes += 1
    what = "forward + backward" if backward else "forward"
    sample = (f"the whole {s.T}-token workload" if len(rows) == s.T
              else f"{len(rows)} of {s.T} tokens (seeded sample)")
    return {"value": len(rows) * passes / elapsed, "unit": "tokens/s", "cores": o.num_threads(),
            "kind": "oracle",
            "sample": f"layer {what} on {sample}, all {s.n_heads} heads, {passes} pass(es), "
                      f"{elapsed:.1f} s"}


def cpu_model():
    """The host CPU's model name (from /proc/cpuinfo) and its logical CPUs."""
    name = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    name = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return name, os.cpu_count()


def cpu_baseline_one_thread(workload, seed, min_seconds, backward):
    """The same oracle timing in a child process with OMP_NUM_THREADS=1."""
    import subprocess
    env = dict(os.environ, OMP_NUM_THREADS="1")
    res = subprocess.run([sys.executable, os.path.abspath(__file__), "--cpu-baseline-only",
                          workload, str(seed), str(min_seconds), "1" if backward else "0"],
                         capture_output=True, text=True, env=env, timeout=600)
    if res.returncode != 0:
        return {"error": res.stderr[-300:]}
    return json.loads(res.stdout.strip().splitlines()[-1])


def _kernel_label(name):
    """Short label of a demangled kernel name ("ffn_kernel<128, false>")."""
    import re
    m = re.search(r"([A-Za-z_][A-Za-z0-9_]*(?:<[^()]*>)?)\(", name)
    return m.group(1) if m else name[:60]


def summarize_kernel_trace(db):
    """Markdown table of a rocprofv3 --kernel-trace --stats database."""
    import sqlite3
    c = sqlite3.connect(db)
    rows = c.execute("select name, total_calls, average, percentage from top_kernels").fetchall()
    out = ["| kernel | calls | mean duration (us) | share of GPU time |", "|---|---:|---:|---:|"]
    for n, calls, avg, pct in rows:
        out.append(f"| `{_kernel_label(n)}` | {calls} | {avg:.2f} | {pct:.1f}% |")
    return "\n".join(out)


SIMDS_PER_CU = 4
XCDS = 8


def summarize_counters(db, num_cu=256):
    """Markdown table of the SQ/GRBM counters of a rocprofv3 --pmc database,
    averaged per dispatch for each kernel, with the derived figures:
    MFMA busy = SQ_VALU_MFMA_BUSY_CYCLES / (GRBM_GUI_ACTIVE / XCDs x SIMDs) (the share of
    the kernel's active cycles in which each SIMD's matrix core was busy),
    VALU instructions per MFMA instruction, transcendental share of VALU."""
    import sqlite3
    import statistics as st
    c = sqlite3.connect(db)
    d = {}
    for n, cn, v in c.execute("select kernel_name, counter_name, value from counters_collection"):
        d.setdefault(_kernel_label(n), {}).setdefault(cn, []).append(v)
    names = sorted({cn for v in d.values() for cn in v})
    head = ["kernel", "dispatches"] + names + ["MFMA busy", "VALU/MFMA"]
    out = ["| " + " | ".join(head) + " |", "|" + "---|" * len(head)]
    res = {}
    for lab in sorted(d, key=lambda k: -st.mean(d[k].get("GRBM_GUI_ACTIVE", [0]))):
        m = {cn: st.mean(v) for cn, v in d[lab].items()}
        nd = max(len(v) for v in d[lab].values())
        # GRBM_GUI_ACTIVE comes summed over the 8 XCDs' instances
        busy = (m["SQ_VALU_MFMA_BUSY_CYCLES"] / (m["GRBM_GUI_ACTIVE"] / XCDS * num_cu * SIMDS_PER_CU)
                if m.get("GRBM_GUI_ACTIVE") and "SQ_VALU_MFMA_BUSY_CYCLES" in m else None)
        ratio = (m["SQ_INSTS_VALU"] / m["SQ_INSTS_MFMA"]
                 if m.get("SQ_INSTS_MFMA") and "SQ_INSTS_VALU" in m else None)
        res[lab] = dict(m, mfma_busy=busy, valu_per_mfma=ratio)
        cells = [f"`{lab}`", str(nd)] + [f"{m[cn]:,.0f}" if cn in m else "" for cn in names]
        cells += [f"{100 * busy:.1f}%" if busy is not None else "",
                  f"{ratio:.2f}" if ratio is not None else ""]
        out.append("| " + " | ".join(cells) + " |")
    return res, "\n".join(out)


def summarize_traffic(fetch_db, write_db, workload, copy_mib):
    """Per-dispatch HBM traffic of the FFN kernel from two rocprofv3 --pmc runs
    (FETCH_SIZE, WRITE_SIZE; KiB per dispatch), each scaled by what the same
    counter reads for the calibration copy of copy_mib MiB."""
    import sqlite3
    import statistics as st

    def per_kernel(db, counter):
        c = sqlite3.connect(db)
        d = {}
        for n, g, v in c.execute("select kernel_name, grid_size, value from counters_collection "
                                 "where counter_name = ?", (counter,)):
            d.setdefault((_kernel_label(n), g), []).append(v)
        return d

    copy_kib = copy_mib * 1024.0
    res = {"workload": workload, "copy_calibration_mib": copy_mib,
           "kernel_source": kernel_source_digest()}
    lines = []
    for counter, db in (("FETCH_SIZE", fetch_db), ("WRITE_SIZE", write_db)):
        d = per_kernel(db, counter)
        # the calibration copy is the largest plain copy in the run
        copy = max((max(v), k) for k, v in d.items() if "copy" in k[0].lower())
        factor = copy_kib / copy[0]
        ffn = [v for k, v in d.items() if k[0].startswith("ffn_")]
        if not ffn:
            raise SystemExit("no FFN kernel dispatches in " + db)
        kib = st.mean(ffn[0])
        res[counter] = {"ffn_kib_per_dispatch": kib, "copy_kib_measured": copy[0],
                        "scale": factor, "ffn_bytes_scaled": kib * 1024.0 * factor}
        lines.append(f"| {counter} | {kib:,.0f} KiB | {copy[0]:,.0f} KiB for {copy_kib:,.0f} KiB "
                     f"| x{factor:.3f} | {kib * 1024 * factor / 1e6:,.1f} MB |")
        for (lab, g), v in sorted(d.items()):
            if "copy" not in lab.lower():
                res[counter].setdefault("kernels", {})[lab] = st.mean(v) * 1024.0 * factor
    res["bytes_per_launch"] = res["FETCH_SIZE"]["ffn_bytes_scaled"] + res["WRITE_SIZE"]["ffn_bytes_scaled"]
    table = ["| counter | FFN per dispatch (raw) | calibration copy (raw vs actual) | scale | FFN scaled |",
             "|---|---:|---:|---:|---:|"] + lines
    return res, "\n".join(table)


# ---------------------------------------------------------------------------
# Per-component sweeps at the paper's shapes against in-house naive baselines
# (python bench.py --sweep routing|experts|steps): one JSON line per point.
# ---------------------------------------------------------------------------

def _time_ms(fn, reps, torch):
    fn()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(reps):
        fn()
    torch.cuda.synchronize()
    return (time.perf_counter() - t0) * 1e3 / reps


def _peak_extra_bytes(fn, torch):
    """Device memory a call allocates beyond what exists before it (peak)."""
    torch.cuda.synchronize()
    torch.cuda.reset_peak_memory_stats()
    base = torch.cuda.memory_allocated()
    fn()
    torch.cuda.synchronize()
    return torch.cuda.max_memory_allocated() - base


def sweep_routing(reps=5):
    """IO-aware routing (mhlmoe_route, and mhlmoe_route_backward from a gate
    gradient: Algorithm 2) against routing with materialised logits: fp32
    X W_r^T [T, N_h, N_e] by torch.bmm, torch.topk, softmax over the k
    selected scores, and its autograd backward (dense dlogits).  The paper's
    shape: B 40 x T 2048 tokens, N_h 8, d_h 128 (Fig. 4); k 8."""
    import numpy as np
    import torch
    import paper_2602_04870_amd as mh
    import workloads
    dev = torch.device("cuda", 0)
    T, Nh, dh, k = 40 * 2048, 8, 128, 8
    for Ne in (64, 128, 256, 512, 1024):
        w = workloads.generate(workloads.Shape(T, Nh, dh, Ne, k, 32, "bf16"), 0)
        X = workloads.to_device(w.X)
        Wr = workloads.to_device(w.W_router)
        idx = torch.empty((T, Nh, k), dtype=torch.int32, device=dev)
        gate = torch.empty((T, Nh, k), dtype=torch.float32, device=dev)
        counts = torch.empty((Nh, Ne), dtype=torch.int32, device=dev)
        ws = mh.workspace(mh.MHLMOE_OP_ROUTE, T, Nh, dh, Ne, k, 0, mh.MHLMOE_BF16, device=dev)
        ours = lambda: mh.mhlmoe_route(X, Wr, None, k, idx=idx, gate=gate, counts=counts,
                                       workspace=ws)
        ours_ms = _time_ms(ours, reps, torch)
        ours_bytes = ws.numel() + idx.numel() * 4 + gate.numel() * 4 + counts.numel() * 4
        G = torch.randn((T, Nh, k), dtype=torch.float32, device=dev)
        wsb = mh.workspace(mh.MHLMOE_OP_ROUTE_BACKWARD, T, Nh, dh, Ne, k, 0, mh.MHLMOE_BF16,
                           device=dev)
        dXo = torch.empty_like(X)
        dWo = torch.empty((Nh, Ne, dh), dtype=torch.float32, device=dev)
        ours_b = lambda: mh.mhlmoe_route_backward(X, Wr, idx, gate, G, dX=dXo,  # noqa: E731
                                                  dW_router=dWo, workspace=wsb)
        ours()
        ours_bwd_ms = _time_ms(ours_b, reps, torch)

        def ours_fb():
            ours()
            ours_b()

        ours_fb_ms = _time_ms(ours_fb, reps, torch)
        ours_fb_bytes = ours_bytes + wsb.numel() + dXo.numel() * 2 + dWo.numel() * 4
        Xh = X.float().permute(1, 0, 2).contiguous()      # [Nh, T, dh]
        Wt = Wr.transpose(1, 2).contiguous()               # [Nh, dh, Ne]

        def naive_fwd(Wt_=Wt, Xh_=Xh):
            logits = torch.bmm(Xh_, Wt_)                   # [Nh, T, Ne], materialised
            sel = logits.topk(k, dim=-1).indices
            return sel, torch.softmax(logits.gather(-1, sel), dim=-1)

        def naive_fwd_bwd():
            Wg = Wt.clone().requires_grad_(True)
            Xg = Xh.clone().requires_grad_(True)
            _, g = naive_fwd(Wg, Xg)
            (g * G.permute(1, 0, 2)).sum().backward()

        naive_ms = _time_ms(naive_fwd, reps, torch)
        naive_fb_ms = _time_ms(naive_fwd_bwd, reps, torch)
        naive_bytes = _peak_extra_bytes(naive_fwd_bwd, torch)
        torch.cuda.synchronize()
        sel, g = naive_fwd()
        same = float((sel.permute(1, 0, 2).to(torch.int32) == idx).all(dim=-1).float().mean())
        print(json.dumps({"sweep": "routing", "T": T, "n_heads": Nh, "d_head": dh, "top_k": k,
                          "n_experts": Ne, "ours_fwd_ms": round(ours_ms, 4),
                          "ours_device_bytes": int(ours_bytes),
                          "ours_bwd_ms": round(ours_bwd_ms, 4),
                          "ours_fwd_bwd_ms": round(ours_fb_ms, 4),
                          "ours_fwd_bwd_device_bytes": int(ours_fb_bytes),
                          "naive_fwd_ms": round(naive_ms, 4),
                          "naive_fwd_bwd_ms": round(naive_fb_ms, 4),
                          "naive_fwd_bwd_peak_bytes": int(naive_bytes),
                          "rows_same_selection": round(same, 5)}), flush=True)
        del w, X, Wr, Xh, Wt, ws, wsb, dXo, dWo
        torch.cuda.empty_cache()


def sweep_experts(reps=5):
    """IO-aware GELU experts (mhlmoe_experts_gelu: clustering, FFN with the
    intermediate on chip, combine) against a naive grouped GEMM: slots sorted
    by (head, expert), padded to the largest group, torch.bmm into a
    materialised [groups, cap, d_e] intermediate, gelu, torch.bmm, gather
    back, gate-weighted sum.  Backward (Fig. 5, right): ours is
    mhlmoe_layer_gelu_backward (with a zero router, so only the expert and
    gate terms carry weight); the naive one is the same padded bmm chain's
    backward written out (the products autograd would issue, with every
    transposed operand made contiguous first).  The paper's shape: B 4 x T
    512 tokens, N_h 8, d_h 128, k 4 (Fig. 5), d_e in {128, 256}; uniform
    random routing."""
    import numpy as np
    import torch
    import paper_2602_04870_amd as mh
    import workloads
    dev = torch.device("cuda", 0)
    T, Nh, dh, k = 4 * 512, 8, 128, 4
    for dff in (128, 256):
        for Ne in (64, 128, 256, 512, 1024):
            w = workloads.generate(workloads.Shape(T, Nh, dh, Ne, k, dff, "bf16", expert="gelu"), 0)
            X = workloads.to_device(w.X)
            Wi = workloads.to_device(w.W1)
            Wo = workloads.to_device(w.W2)
            idx_h, gate_h = workloads.random_routing(T, Nh, Ne, k, seed=5)
            idx = workloads.to_device(idx_h)
            gate = workloads.to_device(gate_h)
            Y = torch.empty_like(X)
            ws = mh.workspace(mh.MHLMOE_OP_EXPERTS, T, Nh, dh, Ne, k, dff, mh.MHLMOE_BF16,
                              device=dev)
            ours = lambda: mh.mhlmoe_experts_gelu(X, idx, gate, Wi, Wo, Y=Y, workspace=ws)
            ours_ms = _time_ms(ours, reps, torch)
            ours_bytes = ws.numel()
            E = Nh * Ne
            # the naive baseline's weights pre-arranged for torch.bmm (outside the timing)
            WiT = Wi.reshape(E, dff, dh).transpose(1, 2).contiguous()   # [E, dh, dff]
            WoT = Wo.reshape(E, dh, dff).transpose(1, 2).contiguous()   # [E, dff, dh]
            head = torch.arange(Nh, device=dev).view(1, Nh, 1)

            def naive():
                grp = (head * Ne + idx.long()).reshape(-1)               # slot -> group
                order = torch.argsort(grp, stable=True)
                cnt = torch.bincount(grp, minlength=E)
                cap = int(cnt.max())
                start = torch.cumsum(cnt, 0) - cnt
                sg = grp[order]
                pos = torch.arange(order.numel(), device=dev) - start[sg]
                rows = (order // k)                                      # token * Nh + head
                xs = X.reshape(T * Nh, dh)[rows]
                buf = torch.zeros((E, cap, dh), dtype=X.dtype, device=dev)
                buf[sg, pos] = xs
                h = torch.bmm(buf, WiT)                                  # [E, cap, dff]
                h = torch.nn.functional.gelu(h.float()).to(X.dtype)
                yb = torch.bmm(h, WoT)                                   # [E, cap, dh]
                ys = torch.empty((order.numel(), dh), dtype=torch.float32, device=dev)
                ys[order] = yb[sg, pos].float()
                y = (ys.view(T, Nh, k, dh) * gate.unsqueeze(-1)).sum(dim=2)
                return y.to(X.dtype)

            naive_ms = _time_ms(naive, reps, torch)
            naive_bytes = _peak_extra_bytes(naive, torch)
            torch.cuda.synchronize()
            ours()
            yn = naive()
            torch.cuda.synchronize()
            rel = float((Y.float() - yn.float()).norm() / yn.float().norm())

            # backward
            dY = torch.randn_like(X, dtype=torch.float32).to(X.dtype)
            Wr0 = torch.zeros((Nh, Ne, dh), dtype=torch.float32, device=dev)
            wsb = mh.workspace(mh.MHLMOE_OP_LAYER_BACKWARD, T, Nh, dh, Ne, k, dff,
                               mh.MHLMOE_BF16, device=dev)
            ours_b = lambda: mh.mhlmoe_layer_gelu_backward(X, Wr0, Wi, Wo, idx, gate, dY,  # noqa: E731
                                                           workspace=wsb)
            ours_bwd_ms = _time_ms(ours_b, reps, torch)

            def naive_bwd():
                grp = (head * Ne + idx.long()).reshape(-1)
                order = torch.argsort(grp, stable=True)
                cnt = torch.bincount(grp, minlength=E)
                cap = int(cnt.max())
                start = torch.cumsum(cnt, 0) - cnt
                sg = grp[order]
                pos = torch.arange(order.numel(), device=dev) - start[sg]
                rows = (order // k)
                g_sl = gate.reshape(-1)[order]                               # gates of the sorted slots
                buf = torch.zeros((E, cap, dh), dtype=X.dtype, device=dev)
                buf[sg, pos] = X.reshape(T * Nh, dh)[rows]
                hpre = torch.bmm(buf, WiT)                                   # recomputed
                hg = torch.nn.functional.gelu(hpre.float()).to(X.dtype)
                dyb = torch.zeros((E, cap, dh), dtype=X.dtype, device=dev)
                dyb[sg, pos] = (dY.reshape(T * Nh, dh)[rows].float() * g_sl[:, None]).to(X.dtype)
                dWoT = torch.bmm(hg.transpose(1, 2).contiguous(), dyb)      # [E, dff, dh]
                dhg = torch.bmm(dyb, WoT.transpose(1, 2).contiguous())      # [E, cap, dff]
                z = hpre.float()
                cdf = 0.5 * (1.0 + torch.erf(z * 0.7071067811865476))
                dh_ = (dhg.float() * (cdf + z * torch.exp(-0.5 * z * z) * 0.3989422804014327)
                       ).to(X.dtype)
                dWiT = torch.bmm(buf.transpose(1, 2).contiguous(), dh_)     # [E, dh, dff]
                dbuf = torch.bmm(dh_, WiT.transpose(1, 2).contiguous())     # [E, cap, dh]
                dX = torch.zeros((T * Nh, dh), dtype=torch.float32, device=dev)
                dX.index_add_(0, rows, dbuf[sg, pos].float())
                yb = torch.bmm(hg, WoT)
                dgate = (yb[sg, pos].float() * dY.reshape(T * Nh, dh)[rows].float()).sum(-1)
                return dX.to(X.dtype).reshape(T, Nh, dh), dWiT, dWoT, dgate

            naive_bwd_ms = _time_ms(naive_bwd, reps, torch)
            naive_bwd_bytes = _peak_extra_bytes(naive_bwd, torch)
            torch.cuda.synchronize()
            ob = ours_b()
            nb_ = naive_bwd()
            torch.cuda.synchronize()
            rel_dx = float((ob[0].float() - nb_[0].float()).norm() / nb_[0].float().norm())
            print(json.dumps({"sweep": "experts", "T": T, "n_heads": Nh, "d_head": dh,
                              "top_k": k, "d_ff": dff, "n_experts": Ne,
                              "ours_fwd_ms": round(ours_ms, 4),
                              "ours_workspace_bytes": int(ours_bytes),
                              "naive_fwd_ms": round(naive_ms, 4),
                              "naive_fwd_peak_bytes": int(naive_bytes),
                              "rel_l2_ours_vs_naive": round(rel, 6),
                              "ours_bwd_ms": round(ours_bwd_ms, 4),
                              "ours_bwd_workspace_bytes": int(wsb.numel()),
                              "naive_bwd_ms": round(naive_bwd_ms, 4),
                              "naive_bwd_peak_bytes": int(naive_bwd_bytes),
                              "rel_l2_dx_ours_vs_naive": round(rel_dx, 6)}), flush=True)
            del w, X, Wi, Wo, WiT, WoT, ws, wsb
            torch.cuda.empty_cache()


def sweep_steps(reps=20):
    """The steps either side of the hot path at the 4096-token, 8 x 128,
    64-expert, k = 8, d_ff 256 bf16 workload (d_model = 8 x 128 = 1024): the layer
    alone, with separate routing sub-tokens (Sec. 4.4), and with its W_in /
    W_out projections (Eq. (5)-(6)), forward and backward; the projection
    GEMMs' rate against the bf16 MFMA peak; the aux-free bias update; and
    the separate-input router-weight gradient at the skewed 65536-token,
    1024-expert workload.  Per-kernel times are HIP events around each
    launch on its stream (mhlmoe_timing_*)."""
    import torch
    import paper_2602_04870_amd as mh
    import workloads
    dev = torch.device("cuda", 0)
    s = workloads.CONFIGS["bf16_t4096_e64"]
    T, Nh, dh, Ne, k, dff = s.T, s.n_heads, s.d_head, s.n_experts, s.top_k, s.d_ff
    dm, N = Nh * dh, Nh * dh
    sb = workloads.Shape(T, Nh, dh, Ne, k, dff, "bf16", backward=True)
    w = workloads.generate(sb, 0)
    d = {n: workloads.to_device(getattr(w, n)) for n in ("X", "W_router", "W1", "W3", "W2", "dY")}
    R = workloads.to_device(workloads.routing_subtokens(sb, 0))
    li = {n: workloads.to_device(v) for n, v in workloads.latent_inputs(sb, dm, False, 0).items()}
    li2 = {n: workloads.to_device(v) for n, v in workloads.latent_inputs(sb, dm, True, 0).items()}
    idx_h, gate_h = workloads.random_routing(T, Nh, Ne, k, seed=3)
    idx, gate = workloads.to_device(idx_h), workloads.to_device(gate_h)
    peak = 2516.6  # bf16 dense MFMA TFLOP/s

    def ws(op):
        return mh.workspace(op, T, Nh, dh, Ne, k, dff, mh.MHLMOE_BF16, device=dev)

    wl, wb = ws(mh.MHLMOE_OP_LAYER), ws(mh.MHLMOE_OP_LAYER_BACKWARD)
    wlat, wlatb = ws(mh.MHLMOE_OP_LATENT_LAYER), ws(mh.MHLMOE_OP_LATENT_BACKWARD)
    cases = [
        ("layer", lambda: mh.mhlmoe_layer(d["X"], d["W_router"], None, d["W1"], d["W3"], d["W2"],
                                          k, workspace=wl), {}),
        ("layer_routed", lambda: mh.mhlmoe_layer_routed(d["X"], R, d["W_router"], None, d["W1"],
                                                        d["W3"], d["W2"], k, workspace=wl), {}),
        ("latent_layer", lambda: mh.mhlmoe_latent_layer(
            li["x"], li["W_in"], d["W_router"], None, d["W1"], d["W3"], d["W2"], li["W_out"], Nh,
            k, workspace=wlat), {"proj_in": 2 * T * dm * N, "proj_out": 2 * T * N * dm}),
        ("latent_layer_routing_tokens", lambda: mh.mhlmoe_latent_layer(
            li2["x"], li2["W_in"], d["W_router"], None, d["W1"], d["W3"], d["W2"], li2["W_out"],
            Nh, k, routing_tokens=True, workspace=wlat),
         {"proj_in": 2 * 2 * T * dm * N, "proj_out": 2 * T * N * dm}),
        ("layer_backward", lambda: mh.mhlmoe_layer_backward(
            d["X"], d["W_router"], d["W1"], d["W3"], d["W2"], idx, gate, d["dY"], workspace=wb),
         {}),
        ("layer_backward_routed", lambda: mh.mhlmoe_layer_backward_routed(
            d["X"], R, d["W_router"], d["W1"], d["W3"], d["W2"], idx, gate, d["dY"],
            workspace=wb), {}),
        ("latent_backward", lambda: mh.mhlmoe_latent_layer_backward(
            li["x"], li["W_in"], d["W_router"], d["W1"], d["W3"], d["W2"], li["W_out"],
            li["X_lat"], None, li["Y_lat"], idx, gate, li["dout"], workspace=wlatb),
         {"proj_bwd": 4 * 2 * T * dm * N}),
        ("latent_backward_routing_tokens", lambda: mh.mhlmoe_latent_layer_backward(
            li2["x"], li2["W_in"], d["W_router"], d["W1"], d["W3"], d["W2"], li2["W_out"],
            li2["X_lat"], li2["R_lat"], li2["Y_lat"], idx, gate, li2["dout"],
            routing_tokens=True, workspace=wlatb), {"proj_bwd": 6 * 2 * T * dm * N}),
    ]
    counts = torch.from_numpy(workloads.random_counts(Nh, Ne, 1, T * k)).to(dev)
    bias = torch.zeros((Nh, Ne), dtype=torch.float32, device=dev)
    cases.append(("bias_update", lambda: mh.mhlmoe_bias_update(counts, bias, 1e-3), {}))
    for name, fn, flops in cases:
        ms = _time_ms(fn, reps, torch)
        mh.mhlmoe_timing_enable(True)
        mh.mhlmoe_timing_reset()
        for _ in range(reps):
            fn()
        torch.cuda.synchronize()
        kern = {}
        for kn in ("route_fwd", "ffn", "combine", "bwd_dx", "bwd_combine", "bwd_dw", "router_dw",
                   "proj_in", "proj_out", "proj_bwd", "bias_update"):
            tot, n = mh.mhlmoe_timing_query(kn)
            if n:
                kern[kn] = {"us_per_call": round(tot * 1e3 / reps, 2)}
                if kn in flops:
                    tf = flops[kn] / (tot * 1e-3 / reps) / 1e12
                    kern[kn].update({"tflops": round(tf, 1), "frac_bf16_peak": round(tf / peak, 3)})
        mh.mhlmoe_timing_enable(False)
        mh.mhlmoe_timing_reset()
        print(json.dumps({"sweep": "steps", "workload": "bf16_t4096_e64", "d_model": dm,
                          "entry": name, "ms_per_call": round(ms, 4), "kernels": kern}),
              flush=True)
    del wl, wb, wlat, wlatb
    torch.cuda.empty_cache()
    # the separate-input router-weight gradient where experts are hottest
    sk = dataclasses.replace(workloads.CONFIGS["skewed_bf16_t65536_e1024"], backward=True)
    w = workloads.generate(sk, 0)
    d = {n: workloads.to_device(getattr(w, n)) for n in ("X", "W_router", "W1", "W3", "W2", "dY")}
    R = workloads.to_device(workloads.routing_subtokens(sk, 0))
    idx_h, gate_h = workloads.random_routing(sk.T, sk.n_heads, sk.n_experts, sk.top_k, seed=0,
                                             skew=sk.zipf_s)
    idx, gate = workloads.to_device(idx_h), workloads.to_device(gate_h)
    wb = mh.workspace(mh.MHLMOE_OP_LAYER_BACKWARD, sk.T, sk.n_heads, sk.d_head, sk.n_experts,
                      sk.top_k, sk.d_ff, mh.MHLMOE_BF16, device=dev)
    for name, fn in (
            ("layer_backward", lambda: mh.mhlmoe_layer_backward(
                d["X"], d["W_router"], d["W1"], d["W3"], d["W2"], idx, gate, d["dY"],
                workspace=wb)),
            ("layer_backward_routed", lambda: mh.mhlmoe_layer_backward_routed(
                d["X"], R, d["W_router"], d["W1"], d["W3"], d["W2"], idx, gate, d["dY"],
                workspace=wb))):
        ms = _time_ms(fn, 3, torch)
        mh.mhlmoe_timing_enable(True)
        mh.mhlmoe_timing_reset()
        fn()
        torch.cuda.synchronize()
        kern = {}
        for kn in ("bwd_dx", "bwd_combine", "bwd_dw", "router_dw"):
            tot, n = mh.mhlmoe_timing_query(kn)
            if n:
                kern[kn] = {"us_per_call": round(tot * 1e3, 1)}
        mh.mhlmoe_timing_enable(False)
        mh.mhlmoe_timing_reset()
        print(json.dumps({"sweep": "steps", "workload": "skewed_bf16_t65536_e1024",
                          "entry": name, "ms_per_call": round(ms, 3), "kernels": kern}),
              flush=True)


def main(argv=None):
    if argv is None:
        argv = sys.argv[1:]
    if argv and argv[0] == "--sweep":
        import torch
        if not torch.cuda.is_available():
            print("bench.py needs a GPU", file=sys.stderr)
            return 1
        {"routing": sweep_routing, "experts": sweep_experts, "steps": sweep_steps}[argv[1]]()
        return 0
    if argv and argv[0] == "--summarize-kernel-trace":
        print(summarize_kernel_trace(argv[1]))
        return 0
    if argv and argv[0] == "--cpu-baseline-only":
        # --cpu-baseline-only WORKLOAD SEED SECONDS BACKWARD (the oracle on the host, no GPU)
        import workloads
        shape = workloads.ALL_CONFIGS[argv[1]]
        if argv[4] == "1":
            shape = dataclasses.replace(shape, backward=True)
        w = workloads.generate(shape, int(argv[2]))
        print(json.dumps(cpu_baseline(w, float(argv[3]), argv[4] == "1")))
        return 0
    if argv and argv[0] == "--summarize-counters":
        # --summarize-counters PMC.db
        print(summarize_counters(argv[1])[1])
        return 0
    if argv and argv[0] == "--summarize-traffic":
        # --summarize-traffic FETCH.db WRITE.db WORKLOAD COPY_MIB [OUT.json]
        res, table = summarize_traffic(argv[1], argv[2], argv[3], int(argv[4]))
        if len(argv) > 5:
            try:
                with open(argv[5]) as f:
                    allr = json.load(f)
            except (OSError, ValueError):
                allr = {}
            allr[argv[3]] = res
            with open(argv[5], "w") as f:
                json.dump(allr, f, indent=1, sort_keys=True)
        print(table)
        return 0
    args = parse_args(argv)
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py measures the single-GPU hot path only (Head Parallel's inter-GPU "
              "exchange is not part of this build); run it with --gpus 1.", file=sys.stderr)
        return 2

    import numpy as np
    import torch

    import paper_2602_04870_amd as mh
    import workloads

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        return 1
    shape = workloads.ALL_CONFIGS[args.workload]
    if args.backward and shape.expert == "swiglu":
        shape = dataclasses.replace(shape, backward=True)
    w = workloads.generate(shape, args.seed)
    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)
    print(f"[bench] {args.workload} T={shape.T} Nh={shape.n_heads} dh={shape.d_head} "
          f"Ne={shape.n_experts} k={shape.top_k} dff={shape.d_ff} {shape.dtype}", file=sys.stderr,
          flush=True)

    names = ("X", "W_router", "bias", "W1", "W2") + (("W3",) if shape.expert == "swiglu" else ()) + \
        (("dY",) if shape.backward else ())
    base = {n: workloads.to_device(getattr(w, n)) for n in names}
    set_bytes = sum(t.numel() * t.element_size() for t in base.values() if t is not None)
    set_bytes += 2 * base["X"].numel() * base["X"].element_size()  # Y + routing outputs, roughly
    nsets = args.sets or max(1, math.ceil(2 * MALL_BYTES / set_bytes))
    sets = [base] + [{n: (t.clone() if t is not None else None) for n, t in base.items()}
                     for _ in range(nsets - 1)]
    T, Nh, dh, Ne, k, dff = (shape.T, shape.n_heads, shape.d_head, shape.n_experts, shape.top_k,
                            shape.d_ff)
    dt = mh.MHLMOE_BF16 if shape.dtype == "bf16" else mh.MHLMOE_F32
    outs = []
    for _ in range(nsets):
        outs.append(dict(Y=torch.empty_like(base["X"]),
                         idx=torch.empty((T, Nh, k), dtype=torch.int32, device=dev),
                         gate=torch.empty((T, Nh, k), dtype=torch.float32, device=dev),
                         counts=torch.empty((Nh, Ne), dtype=torch.int32, device=dev)))
    ws = mh.workspace(mh.MHLMOE_OP_LAYER, T, Nh, dh, Ne, k, dff, dt, device=dev)
    stream = torch.cuda.current_stream()
    if shape.backward:
        f32 = torch.float32
        grads = dict(dW_router=torch.empty((Nh, Ne, dh), dtype=f32, device=dev),
                     dW1=torch.empty((Nh, Ne, dff, dh), dtype=f32, device=dev),
                     dW3=torch.empty((Nh, Ne, dff, dh), dtype=f32, device=dev),
                     dW2=torch.empty((Nh, Ne, dh, dff), dtype=f32, device=dev))
        for o in outs:
            o["dX"] = torch.empty_like(base["X"])
        ws_b = mh.workspace(mh.MHLMOE_OP_LAYER_BACKWARD, T, Nh, dh, Ne, k, dff, dt, device=dev)

    def step(i):
        s, o = sets[i % nsets], outs[i % nsets]
        if shape.expert == "gelu":
            mh.mhlmoe_layer_gelu(s["X"], s["W_router"], s["bias"], s["W1"], s["W2"], k,
                                 Y=o["Y"], idx=o["idx"], gate=o["gate"], counts=o["counts"],
                                 workspace=ws, stream=stream)
        else:
            mh.mhlmoe_layer(s["X"], s["W_router"], s["bias"], s["W1"], s["W3"], s["W2"], k,
                            Y=o["Y"], idx=o["idx"], gate=o["gate"], counts=o["counts"],
                            workspace=ws, stream=stream)
        if shape.backward:
            mh.mhlmoe_layer_backward(s["X"], s["W_router"], s["W1"], s["W3"], s["W2"], o["idx"],
                                     o["gate"], s["dY"], dX=o["dX"], workspace=ws_b, stream=stream,
                                     **grads)

    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()

    # Timed region: K steps, nothing but the layer calls between two
    # synchronisations (the throughput reported as `value`).
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        step(i)
    torch.cuda.synchronize()
    ms_per_step = (time.perf_counter() - t0) * 1e3 / args.steps

    # Warm Infinity Cache: the same K steps on one input set (every step after
    # the first finds its inputs in the 256 MB MALL where they fit); reported
    # beside the cold figure above, never as `value`.
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        step(0)
    torch.cuda.synchronize()
    warm_ms = (time.perf_counter() - t0) * 1e3 / args.steps

    # The same K steps again with the library recording two HIP events around
    # every kernel on the stream it runs on: per-kernel mean durations for the
    # roofline.  (The events add a few microseconds per kernel, so this pass
    # is not the one whose wall time is reported.)
    mh.mhlmoe_timing_reset()
    mh.mhlmoe_timing_enable(True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        step(i)
    torch.cuda.synchronize()
    inst_ms = (time.perf_counter() - t0) * 1e3 / args.steps
    mh.mhlmoe_timing_enable(False)
    kern = {}
    for name in KERNELS:
        total, n = mh.mhlmoe_timing_query(name)
        if n:
            kern[name] = {"mean_us": total * 1e3 / n, "launches": n}
    mh.mhlmoe_timing_reset()

    if args.copy_calibration_mib:
        n = args.copy_calibration_mib << 20
        src = torch.empty(n, dtype=torch.uint8, device=dev)
        src.fill_(1)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        print(f"[bench] copy calibration: {args.copy_calibration_mib} MiB read + written",
              file=sys.stderr, flush=True)

    route_bytes, ffn_flops, ffn_bytes = algorithmic(shape)
    peak = PEAK_TFLOPS[shape.dtype]
    slots_dd = T * Nh * k * dh * dff

    def mfma_roofline(name):
        us = kern[name]["mean_us"]
        flops = (2 * ffn_matrices(shape) if name == "ffn" else ALGO_FLOPS[name]) * slots_dd
        achieved = flops / (us * 1e-6) / 1e12
        return {"bound": "mfma", "achieved": round(achieved, 2), "peak": peak, "unit": "TFLOP/s",
                "frac": round(achieved / peak, 4), "kernel": name, "flops_per_launch": flops,
                "executed_flops_per_launch": (2 * ffn_matrices(shape) if name == "ffn"
                                              else EXEC_FLOPS[name]) * slots_dd,
                "mean_us": round(us, 3)}

    # the dominant kernel: the MFMA kernel with the largest mean duration
    dominant = max((n for n in ALGO_FLOPS if n in kern), key=lambda n: kern[n]["mean_us"])
    roofline = mfma_roofline(dominant)
    roofline["traffic"] = (load_traffic(args.traffic, args.workload, None)
                           if dominant == "ffn" else None)
    if dominant == "ffn":
        roofline["algorithmic_bytes_per_launch"] = ffn_bytes
        roofline.update(ffn_bound(roofline, ffn_bytes, peak))
    others = {n: mfma_roofline(n) for n in ALGO_FLOPS if n in kern and n != dominant}
    r_us = kern["route_fwd"]["mean_us"]
    route_gbs = route_bytes / (r_us * 1e-6) / 1e9
    # the router's scores: 2 T N_h d_h N_e flops of fp32 dot products, done as
    # two bf16 MFMA passes (hi and lo parts of W_router) for bf16 X
    route_flops = 2 * T * Nh * dh * Ne
    route_exec = route_flops * (2 if shape.dtype == "bf16" else 1)
    route_roofline = {"bound": "hbm", "achieved": round(route_gbs, 1), "peak": PEAK_HBM_GBS,
                      "unit": "GB/s", "frac": round(route_gbs / PEAK_HBM_GBS, 4),
                      "kernel": "route_fwd", "bytes_per_launch": route_bytes,
                      "flops_per_launch": route_flops, "executed_mfma_flops": route_exec,
                      "frac_mfma_executed": round(route_exec / (r_us * 1e-6) / (peak * 1e12), 4),
                      "flop_per_byte": round(route_flops / route_bytes, 1)}
    # The whole experts call (clustering + FFN + combine), as the %MFMA of the
    # expert computation is defined over it, and the clustering's own %HBM
    # (it reads idx and writes perm: 8 bytes per slot, plus the per-block
    # histograms it reads and the offsets it writes).
    slots = T * Nh * k
    bucket = [n for n in ("hist", "count_scan", "scatter") if n in kern]
    b_us = sum(kern[n]["mean_us"] for n in bucket)
    nblk = -(-T // 128)
    bucket_bytes = 8 * slots + 4 * Nh * nblk * Ne * 3 + 4 * Nh * (2 * Ne + 1)
    e_us = b_us + kern["ffn"]["mean_us"] + kern["combine"]["mean_us"]
    experts_roofline = {
        "kernels": bucket + ["ffn", "combine"], "mean_us": round(e_us, 3),
        "flops_per_launch": ffn_flops,
        "frac_mfma": round(ffn_flops / (e_us * 1e-6) / (peak * 1e12), 4),
        "bucket_us": round(b_us, 3), "bucket_bytes": bucket_bytes,
        "bucket_frac_hbm": round(bucket_bytes / (b_us * 1e-6) / (PEAK_HBM_GBS * 1e9), 4)}

    cpu = None
    if not args.no_cpu_baseline and int(os.environ.get("RANK", "0")) == 0:
        print("[bench] timing the CPU oracle", file=sys.stderr, flush=True)
        cpu = cpu_baseline(w, args.cpu_seconds, shape.backward)
        model, ncpu = cpu_model()
        cpu["cpu_model"] = model
        cpu["logical_cpus"] = ncpu
        print("[bench] timing the CPU oracle on one thread", file=sys.stderr, flush=True)
        one = cpu_baseline_one_thread(args.workload, args.seed, args.cpu_seconds / 2,
                                      shape.backward)
        cpu["one_thread"] = ({k: one[k] for k in ("value", "unit", "cores", "sample")}
                             if "value" in one else one)

    value = T / (ms_per_step * 1e-3)
    out = {
        "metric": "routed tokens/sec per MoE layer (1 GPU)"
                  + (", forward + backward" if shape.backward else ""),
        "value": round(value, 1),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": shape.dtype,
        "data": "synthetic",
        "config": {"workload": args.workload, "T": T, "n_heads": Nh, "d_head": dh,
                   "n_experts": Ne, "top_k": k, "d_ff": dff, "bias": shape.bias,
                   "expert": shape.expert,
                   "pass": "forward+backward" if shape.backward else "forward",
                   "input_sets_cycled": nsets},
        "roofline": roofline,
        "cpu_baseline": cpu,
        "route_roofline": route_roofline,
        "mfma_rooflines": others,
        "experts_roofline": experts_roofline,
        "warm_mall_ms_per_step": round(warm_ms, 5),
        "kernels": {n: round(v["mean_us"], 3) for n, v in kern.items()},
        "kernel_unit": "us (mean per launch over K event-instrumented steps)",
        "ms_per_step_instrumented": round(inst_ms, 5),
    }
    print(json.dumps(out), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
