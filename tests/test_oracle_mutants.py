"""Planted mistakes in the oracle must each fail at least one pin.

Each mutant is a one-place textual change to oracle/mhlmoe_oracle.c (a
dropped term, a wrong sign, index or operand), built with gcc into a temporary
library and run against every pin in a child process.  This shows that the
pins constrain each step of the oracle, not just its overall shape.  All
mutants stay in bounds; nothing here touches a GPU.
"""
import os
import subprocess
import sys

import pytest

import oracle

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

MUTANTS = [
    ("router_operand_transposed",
     "acc += x[i] * w[(int64_t)e * dh + i];", "acc += x[i] * w[(int64_t)i * Ne + e];"),
    ("router_every_head_uses_head0",
     "const double *w = W_router + (int64_t)h * Ne * dh;", "const double *w = W_router;"),
    ("router_drops_last_term",
     "for (int i = 0; i < dh; ++i)\n            acc += x[i]", "for (int i = 0; i + 1 < dh; ++i)\n            acc += x[i]"),
    ("bias_sign_flipped",
     "key = s[e] + (float)bias[", "key = s[e] - (float)bias["),
    ("tie_break_toward_higher_index",
     "return (a->e > b->e) - (a->e < b->e);", "return (a->e < b->e) - (a->e > b->e);"),
    ("selection_ascending",
     "if (a->key > b->key) return -1;\n    if (a->key < b->key) return 1;",
     "if (a->key < b->key) return -1;\n    if (a->key > b->key) return 1;"),
    ("gate_uses_biased_key",
     "gate[th * k + j] = exp((double)s[id[j]] - m) / z;", "gate[th * k + j] = exp((double)ent[j].key - m) / z;"),
    ("gate_not_normalised",
     "gate[th * k + j] = exp((double)s[id[j]] - m) / z;", "gate[th * k + j] = exp((double)s[id[j]] - m);"),
    ("counts_double_counted",
     "counts[(int64_t)h * Ne + idx[(t * Nh + h) * k + j]] += 1;",
     "counts[(int64_t)h * Ne + idx[(t * Nh + h) * k + j]] += 2;"),
    ("bucket_wrong_slot_id",
     "= (int32_t)(t * k + j);", "= (int32_t)(t + j * T);"),
    ("bucket_offsets_inclusive",
     "offsets[(int64_t)h * (Ne + 1) + e] = (int32_t)cursor[e];",
     "offsets[(int64_t)h * (Ne + 1) + e] = (int32_t)(e < Ne ? cursor[e + 1] : cursor[e]);"),
    ("swiglu_silu_on_up_projection",
     "u[f] = silu(sa) * sb;", "u[f] = sa * silu(sb);"),
    ("swiglu_w1_w3_swapped",
     "sa += w1[(int64_t)f * dh + i] * x[i];\n            sb += w3[(int64_t)f * dh + i] * x[i];",
     "sa += w3[(int64_t)f * dh + i] * x[i];\n            sb += w1[(int64_t)f * dh + i] * x[i];"),
    ("down_projection_transposed",
     "for (int f = 0; f < dff; ++f) acc += w2[(int64_t)i * dff + f] * u[f];",
     "for (int f = 0; f < dff; ++f) acc += w2[(int64_t)f * dh + i] * u[f];"),
    ("combine_drops_gate",
     "for (int i = 0; i < dh; ++i) out[i] += g * y[i];", "for (int i = 0; i < dh; ++i) out[i] += y[i];"),
    ("bwd_softmax_sign",
     "const int64_t he = (int64_t)h * Ne + id[j];\n                const double ds = g[j] * (dg[j] - gdg);",
     "const int64_t he = (int64_t)h * Ne + id[j];\n                const double ds = g[j] * (dg[j] + gdg);"),
    ("bwd_router_dx_dropped",
     "dr[i] += ds * wr[i];", "dr[i] += 0.0 * wr[i];"),
    ("bwd_router_dw_uses_weight",
     "dwr[i] += ds * r[i];", "dwr[i] += ds * wr[i];"),
    ("bwd_dsilu_wrong",
     "const double dsilu = sig * (1.0 + aj[f] * (1.0 - sig));", "const double dsilu = sig * (1.0 - sig);"),
    ("bwd_dw2_drops_gate",
     "dw2[(int64_t)i * dff + f] += g[j] * dy[i] * uj[f];", "dw2[(int64_t)i * dff + f] += dy[i] * uj[f];"),
    ("bwd_du_transposed",
     "acc += w2[(int64_t)i * dff + f] * dy[i];", "acc += w2[(int64_t)f * dh + i] * dy[i];"),
    ("bwd_db_uses_b",
     "const double db = du[f] * aj[f] * sig;", "const double db = du[f] * bj[f] * sig;"),
    ("gelu_tanh_approximation",
     "static double gelu(double z) { return 0.5 * z * (1.0 + erf(z / sqrt(2.0))); }",
     "static double gelu(double z) { return 0.5 * z * (1.0 + tanh(0.7978845608028654 * (z + 0.044715 * z * z * z))); }"),
    ("gelu_drops_half",
     "return 0.5 * z * (1.0 + erf(z / sqrt(2.0)));", "return z * (1.0 + erf(z / sqrt(2.0)));"),
    ("gelu_w_in_transposed",
     "for (int i = 0; i < dh; ++i) s += w_in[(int64_t)f * dh + i] * x[i];",
     "for (int i = 0; i < dh; ++i) s += w_in[(int64_t)i * dff + f] * x[i];"),
    ("gelu_w_out_transposed",
     "for (int f = 0; f < dff; ++f) acc += w_out[(int64_t)i * dff + f] * u[f];",
     "for (int f = 0; f < dff; ++f) acc += w_out[(int64_t)f * dh + i] * u[f];"),
    ("bias_update_sign_flipped",
     "if (d > 0) *b = *b + rate;", "if (d > 0) *b = *b - rate;"),
    ("bias_update_integer_mean",
     "const int64_t d = S - c * Ne;  /* sign of mean - c */",
     "const int64_t d = S / Ne - c;  /* sign of mean - c */"),
    ("bias_update_tie_moves",
     "else if (d < 0) *b = *b - rate;", "else *b = *b - rate;"),
    ("route_bwd_softmax_mean_dropped",
     "const double ds = g[j] * (dg[j] - gdg);\n                if (dS) dS[th * k + j] = ds;\n                const int64_t he",
     "const double ds = g[j] * dg[j];\n                if (dS) dS[th * k + j] = ds;\n                const int64_t he"),
    ("route_bwd_dw_uses_weight",
     "dwr[i] += ds * x[i];", "dwr[i] += ds * wr[i];"),
    ("gelu_bwd_grad_drops_density",
     "return 0.5 * (1.0 + erf(z / sqrt(2.0))) + z * exp(-0.5 * z * z) / sqrt(2.0 * pi);",
     "return 0.5 * (1.0 + erf(z / sqrt(2.0)));"),
    ("gelu_bwd_dx_dropped",
     "dx[i] += da * w1[(int64_t)f * dh + i];", "dx[i] += 0.0 * w1[(int64_t)f * dh + i];"),
    ("routed_bwd_router_reads_x",
     "dwr[i] += ds * r[i];", "dwr[i] += ds * x[i];"),
    ("routed_bwd_router_grad_to_dx",
     "dr[i] += ds * wr[i];", "dx[i] += ds * wr[i];"),
    ("bwd_dx_w3_term_dropped",
     "dx[i] += da * w1[(int64_t)f * dh + i] +\n                                 db * w3[(int64_t)f * dh + i];",
     "dx[i] += da * w1[(int64_t)f * dh + i];"),
]

CHILD = r"""
import sys
sys.path.insert(0, {root!r})
import oracle
from tests import oracle_pins
o = oracle.Oracle(oracle.load({lib!r}))
failed = []
for pin in oracle_pins.ALL_PINS:
    try:
        pin(o)
    except Exception as e:  # AssertionError or an oracle error status
        failed.append(pin.__name__)
print("FAILED_PINS", failed)
sys.exit(0 if failed else 3)
"""


# Mistakes planted in the Python composition of the projections
# (oracle/__init__.py), re-executed in the oracle module's namespace.
PY_MUTANTS = [
    ("bf16_round_half_up",
     "np.rint(m * 256.0) / 256.0", "np.floor(m * 256.0 + 0.5) / 256.0"),
    ("latent_input_not_transposed",
     "lat = x @ W_in.T", "lat = x @ W_in.reshape(W_in.shape[1], W_in.shape[0])"),
    ("routing_tokens_ignored",
     "R_lat = lat[:, N:].reshape(T, n_heads, dh) if routing_tokens else X_lat",
     "R_lat = X_lat"),
    ("latent_out_projection_transposed",
     "out = Y_lat.reshape(T, N) @ W_out.T", "out = Y_lat.reshape(T, N) @ W_out.reshape(N, -1)"),
    ("latent_bwd_dx_drops_routing_term",
     "dx = dx + dRl @ W_in[N:]", "dx = dx + 0.0 * (dRl @ W_in[N:])"),
    ("latent_bwd_dw_in_wrong_operand",
     "dW_in = dXl.T @ x", "dW_in = dXl.T @ (x * 0.5)"),
    ("latent_bwd_dw_out_swapped",
     '"dW_out": dout.T @ Yl', '"dW_out": (Yl.T @ dout).reshape(dout.shape[1], -1)'),
]

PY_CHILD = r"""
import sys
sys.path.insert(0, {root!r})
import oracle
src = open(oracle.__file__).read().replace({old!r}, {new!r})
exec(compile(src, oracle.__file__, "exec"), oracle.__dict__)
from tests import oracle_pins
o = oracle.Oracle()
failed = []
for pin in oracle_pins.ALL_PINS:
    try:
        pin(o)
    except Exception as e:
        failed.append(pin.__name__)
print("FAILED_PINS", failed)
sys.exit(0 if failed else 3)
"""


@pytest.mark.parametrize("name,old,new", PY_MUTANTS, ids=[m[0] for m in PY_MUTANTS])
def test_python_mutant_is_caught(name, old, new):
    src = open(oracle.__file__).read()
    assert src.count(old) == 1, f"mutation site for {name} not unique/found"
    res = subprocess.run([sys.executable, "-c", PY_CHILD.format(root=ROOT, old=old, new=new)],
                         capture_output=True, text=True, timeout=300,
                         env=dict(os.environ, OMP_NUM_THREADS="2"))
    assert res.returncode != 3, f"mutant {name} survived every pin\n{res.stdout}{res.stderr}"
    assert res.returncode == 0, f"mutant {name} crashed: {res.returncode}\n{res.stderr[-2000:]}"


@pytest.mark.parametrize("name,old,new", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_mutant_is_caught(name, old, new, tmp_path):
    src = open(oracle.SOURCE).read()
    assert src.count(old) == 1, f"mutation site for {name} not unique/found"
    mutant_src = tmp_path / "mutant.c"
    mutant_src.write_text(src.replace(old, new))
    lib = str(tmp_path / "libmutant.so")
    oracle.compile_library(str(mutant_src), lib)
    res = subprocess.run([sys.executable, "-c", CHILD.format(root=ROOT, lib=lib)],
                         capture_output=True, text=True, timeout=300,
                         env=dict(os.environ, OMP_NUM_THREADS="2"))
    assert res.returncode != 3, f"mutant {name} survived every pin\n{res.stdout}{res.stderr}"
    # a crash also counts as caught, but every mutant here should fail cleanly
    assert res.returncode == 0, f"mutant {name} crashed: {res.returncode}\n{res.stderr[-2000:]}"
