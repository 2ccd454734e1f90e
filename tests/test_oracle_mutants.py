"""Mutation check of the oracle pins (CPU only).

Each case plants one plausible mistake in a copy of the oracle source (a
dropped term, a flipped sign, a swapped constant, a transposed operand),
builds it, and runs the pin suite against that build in a subprocess.  The
pins must fail for every mutant; a mutant that survives would mean a mistake
of that kind in the oracle could go unnoticed.
"""
import os
import subprocess
import sys
import tempfile

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "eprop_oracle.cpp")

# (name, original text, replacement, expected number of occurrences replaced)
MUTANTS = [
    ("trace_sign", "const double e = pj * (s.zbar[i] - bj * ea);",
     "const double e = pj * (s.zbar[i] + bj * ea);", 1),
    ("no_readout_filter_on_trace", "dW[l][ji] += Lj * s.ebar[ji];", "dW[l][ji] += Lj * e;", 1),
    ("epsa_decay_without_psi", "s.epsa[ji] = pj * s.zbar[i] + (c.rho - bj * pj) * ea;",
     "s.epsa[ji] = pj * s.zbar[i] + (c.rho) * ea;", 1),
    ("epsa_decay_kappa", "s.epsa[ji] = pj * s.zbar[i] + (c.rho - bj * pj) * ea;",
     "s.epsa[ji] = pj * s.zbar[i] + (c.kappa - bj * pj) * ea;", 1),
    ("presyn_filter_kappa", "s.zbar[i] = c.alpha * s.zbar[i] + s.p[i];",
     "s.zbar[i] = c.kappa * s.zbar[i] + s.p[i];", 1),
    ("delta_sign", "- (k == label ? 1.0 : 0.0);", "+ (k == label ? 1.0 : 0.0);", 1),
    ("learning_signal_transposed", "Lj += (double)Fo[(size_t)k * N + j] * s.delta[k];",
     "Lj += (double)Fo[(size_t)j * K + k] * s.delta[k];", 1),
    ("feedback_ignored", "const float* Fo = (Fb && Fb[l]) ? Fb[l] : Wo;", "const float* Fo = Wo;", 1),
    ("feedback_in_readout", "if (s.z[j] != 0.0) Y += (double)Wo[(size_t)k * N + j] * s.z[j];",
     "if (s.z[j] != 0.0) Y += (double)Fo[(size_t)k * N + j] * s.z[j];", 1),
    ("surrogate_unclamped", "(u > 0.0 ? u : 0.0)", "u", 1),
    ("adaptation_path_dropped", "a = a + zp;", "a = a + R(0) * zp;", 1),
    ("reset_dropped", "v = v - reset * zp;", "v = v - R(0) * zp;", 1),
    ("readout_trace_alpha", "s.ztil[j] = c.kappa * s.ztil[j] + s.z[j];",
     "s.ztil[j] = c.alpha * s.ztil[j] + s.z[j];", 1),
    ("drive_transposed", "(R)Wl[(size_t)j * s.n_pre + i]", "(R)Wl[(size_t)i * N + j]", 1),
    ("readout_grad_unfiltered", "dWout[l][(size_t)k * N + j] += s.delta[k] * s.ztil[j];",
     "dWout[l][(size_t)k * N + j] += s.delta[k] * s.z[j];", 1),
    ("diagonal_kept", "for (int j = 0; j < N; ++j) dW[l][(size_t)j * n_pre + n_in_l + j] = 0.0;",
     "", 1),
    ("threshold_adaptation_sign", "A = thr + A;", "A = thr - A;", 1),
    ("reset_through_membrane_decay", "ev = (c.alpha - c.reset * pj) * V + c.reset * bj * pj * ea;",
     "ev = c.alpha * V + c.reset * bj * pj * ea;", 1),
    ("reset_through_coupling_dropped", "ev = (c.alpha - c.reset * pj) * V + c.reset * bj * pj * ea;",
     "ev = (c.alpha - c.reset * pj) * V;", 1),
    ("online_update_from_current_weights", "Wcur[l][ji] = on_grid((double)W0[l][ji] - lr * dW[l][ji]);",
     "Wcur[l][ji] = on_grid((double)Wcur[l][ji] - lr * dW[l][ji]);", 1),
    ("two_compartment_feedback_dropped", "h21 = c.bap * pp", "h21 = 0.0 * pp", 1),
    ("two_compartment_coupling_transposed", "const double ed_new = h21 * es + h22 * ed + s.p[i];",
     "const double ed_new = h12 * es + h22 * ed + s.p[i];", 1),
    ("two_compartment_current_psi_in_jacobian", "const double pp = s.psi_prev[j];",
     "const double pp = s.psi[j];", 1),
    ("two_compartment_soma_reads_new_dendrite", "sm = sm + (R)c.coupling * s.a[j];",
     "sm = sm + (R)c.coupling * d;", 1),
    ("online_feedback_ignored", "steps(c, Wcur, Woutcur, Fb, x,", "steps(c, Wcur, Woutcur, nullptr, x,", 1),
    ("online_readout_not_updated", "Woutcur[l][kj] = on_grid((double)Wout0[l][kj] - lr * dWout[l][kj]);",
     "Woutcur[l][kj] = Wout0[l][kj];", 1),
]


@pytest.mark.parametrize("name,old,new,count", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_pins_catch_planted_mistake(name, old, new, count, tmp_path):
    from oracle import build as obuild
    src = open(SRC).read()
    assert src.count(old) >= count, f"pattern for {name} not found"
    mutant_src = tmp_path / "mutant.cpp"
    mutant_src.write_text(src.replace(old, new, count))
    lib = str(tmp_path / "libmutant.so")
    obuild.build(str(mutant_src), lib)
    env = dict(os.environ, EPROP_ORACLE_LIB=lib)
    res = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider",
                          os.path.join(ROOT, "tests", "test_oracle_pins.py")],
                         env=env, cwd=ROOT, capture_output=True, text=True, timeout=600)
    assert res.returncode != 0, f"mutant {name} survived the pins:\n{res.stdout[-2000:]}"
