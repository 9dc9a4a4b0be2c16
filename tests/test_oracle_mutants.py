"""Plant plausible mistakes into a copy of the oracle (CPU only) and check that
at least one pin catches each of them."""
import functools
import os
import subprocess

import pytest

import oracle
from oracle import oracle as orc_mod
from oracle_pins import ALL_PINS

SRC = os.path.join(os.path.dirname(orc_mod.__file__), "bi_oracle.c")

# (name, text in bi_oracle.c, replacement, count)
MUTANTS = [
    ("b_axis_swapped", "const double b = Bf[((size_t)i * P + flat) * U + u];",
     "const double b = Bf[((size_t)(flat % md->n[f]) * P + (i + flat / md->n[f]) % P) * U + u];", 1),
    ("b_fixed_state_weighted", "if (j != skip) w *= q[qoff[dl[j]] + idx[j]];", "w *= q[qoff[dl[j]] + idx[j]];", 1),
    ("vmp_linear_b", "acc += (logB ? LN(b) : b) * w;", "acc += b * w;", 1),
    ("fwd_from_same_step", "fwd = b_contract(md, Bf, f, s, uprev, qprev, qoff, -1, 0, 1);",
     "fwd = b_contract(md, Bf, f, s, uprev, qcur, qoff, -1, 0, 1);", 1),
    ("mmp_bwd_from_same_step", "m += qnext[qoff[j] + sn] *", "m += qcur[qoff[j] + sn] *", 1),
    ("only_self_children", "if (pos < 0) continue;", "if (pos < 0 || j != f) continue;", 1),
    ("mmp_mean_of_two", "(fwd + bwd) / (double)(1 + children)", "0.5 * (fwd + bwd)", 1),
    ("fpi_prior_expected_log", "LN(b_contract(md, Bf, f, i, u, qp, qoff, -1, 0, 0))",
     "b_contract(md, Bf, f, i, u, qp, qoff, -1, 0, 1)", 1),
    ("mmp_no_half", "(fwd + bwd) / (double)(1 + children)", "(fwd + bwd)", 1),
    ("mmp_last_half", "v[s] = lam[(size_t)t * ntot + qoff[f] + s] + fwd;",
     "v[s] = lam[(size_t)t * ntot + qoff[f] + s] + 0.5 * fwd;", 1),
    ("lik_keeps_own_factor", "if (j != i) w *= q[qoff[d[j]] + idx[j]];", "w *= q[qoff[d[j]] + idx[j]];", 1),
    ("lik_axis_order", "for (int i = k - 1; i >= 0; --i) {\n                if (++idx[i]",
     "for (int i = 0; i < k; ++i) {\n                if (++idx[i]", 1),
    ("vmp_drops_prior", "fwd = LN(p0[s]);", "fwd = 0.0;", 1),
    ("caller_prior_ignored", "if (prior) return prior + (size_t)a * ntot + qoff[f];", "", 1),
    ("predict_transposed", "p += Bf[((size_t)i * nf + j) * U[f] + u] * q[(size_t)a * ntot + off + j];",
     "p += Bf[((size_t)j * nf + i) * U[f] + u] * q[(size_t)a * ntot + off + j];", 1),
    ("predict_general_agent_stride", "b_contract(&md, Bf, f, i, u, q + (size_t)a * ntot, qoff, -1, 0, 0)",
     "b_contract(&md, Bf, f, i, u, q, qoff, -1, 0, 0)", 1),
    ("predict_general_action", "b_contract(&md, Bf, f, i, u, q + (size_t)a * ntot, qoff, -1, 0, 0)",
     "b_contract(&md, Bf, f, i, 0, q + (size_t)a * ntot, qoff, -1, 0, 0)", 1),
    ("predict_general_log_b", "b_contract(&md, Bf, f, i, u, q + (size_t)a * ntot, qoff, -1, 0, 0)",
     "b_contract(&md, Bf, f, i, u, q + (size_t)a * ntot, qoff, -1, 0, 1)", 1),
    ("predict_general_out_offset", "out[(size_t)a * ntot + qoff[f] + i] = b_contract(",
     "out[(size_t)a * ntot + i] = b_contract(", 1),
    ("damping_swapped", "(1.0 - tau) * q[s] + tau * q_new[s]", "tau * q[s] + (1.0 - tau) * q_new[s]", 1),
    ("damping_ignored", "q[s] = tau == 1.0 ? q_new[s] :", "q[s] = 1 ? q_new[s] :", 1),
    ("soft_weight_dropped", "v += om[o] * LN(Am[(size_t)o * P + e]);", "v += LN(Am[(size_t)o * P + e]);", 1),
    ("soft_block_offset", "ob->soft + (size_t)t * ob->ksum + ob->koff[m];", "ob->soft + (size_t)t * ob->ksum;", 1),
    ("soft_outcome_axis", "v += om[o] * LN(Am[(size_t)o * P + e]);", "v += om[o] * LN(Am[(size_t)o + e * md->K[m]]);",
     1),
    ("softmax_sign", "v[i] = exp(v[i] - mx);", "v[i] = exp(mx - v[i]);", 1),
    ("no_log_clamp", "return log(x > ORC_EPS ? x : ORC_EPS);", "return log(x > 0 ? x : 1e-300);", 1),
]


@functools.lru_cache(maxsize=None)
def _mutant_lib(tmpdir, name):
    src = open(SRC).read()
    for mname, old, new, count in MUTANTS:
        if mname == name:
            assert old in src, f"mutation anchor of {name} not found"
            src = src.replace(old, new, count)
    path = os.path.join(tmpdir, f"mut_{name}.c")
    with open(path, "w") as fh:
        fh.write(src)
    so = path[:-2] + ".so"
    subprocess.run(["gcc", "-O2", "-std=c11", "-fopenmp", "-fPIC", "-shared", "-o", so, path, "-lm"], check=True)
    return orc_mod.load_library(so)


@pytest.mark.parametrize("name", [m[0] for m in MUTANTS if m[3] > 0])
def test_mutant_is_caught(name, tmp_path_factory):
    lib = _mutant_lib(str(tmp_path_factory.getbasetemp()), name)
    infer = functools.partial(oracle.infer, lib=lib)
    failed = []
    for pin, (fn, tol) in ALL_PINS.items():
        try:
            err = fn(infer)
        except (ValueError, FloatingPointError):
            err = float("inf")
        if not err <= tol:
            failed.append(pin)
    assert failed, f"planted mistake {name} passed every pin"
