"""The pins are sensitive: plant plausible mistakes in a copy of the oracle.

Each mutant is a textual edit of a temporary copy of the oracle's C source,
compiled on the CPU; the committed oracle is untouched.  Every mutant must
make at least one pin of test_oracle_pins fail.
"""
import os
import subprocess

import pytest

import oracle
from tests import test_oracle_pins as pins

MUTANTS = {
    "rx_sign": ("mat2 u = {{{c, -I * s}, {-I * s, c}}};", "mat2 u = {{{c, I * s}, {I * s, c}}};"),
    "ry_transposed": ("mat2 u = {{{c, -s}, {s, c}}};", "mat2 u = {{{c, s}, {-s, c}}};"),
    "rz_direction": ("mat2 u = {{{cexp(-I * t / 2), 0}, {0, cexp(I * t / 2)}}};",
                     "mat2 u = {{{cexp(I * t / 2), 0}, {0, cexp(-I * t / 2)}}};"),
    "rot_order": ("return mul2(a, mul2(b, c));", "return mul2(c, mul2(b, a));"),
    "full_angle": ("static mat2 m_ry(double t) {\n    double c = cos(t / 2), s = sin(t / 2);",
                   "static mat2 m_ry(double t) {\n    double c = cos(t), s = sin(t);"),
    "cnot_direction": ("bc = (size_t)1 << c, bt = (size_t)1 << t;",
                       "bc = (size_t)1 << t, bt = (size_t)1 << c;"),
    "cz_or": ("if ((x & ba) && (x & bb)) psi[x] = -psi[x];",
              "if ((x & ba) || (x & bb)) psi[x] = -psi[x];"),
    "z_sign": ("acc += ((x >> j) & 1) ? -p : p;", "acc += ((x >> j) & 1) ? p : -p;"),
    "vjp_factor": ("acc *= 2.0;", "acc *= 1.0;"),
    "vjp_no_dagger": ("apply_op(lam, n, op, ang, 1);", "apply_op(lam, n, op, ang, 0);"),
    "vjp_wrong_state": ("const cplx *prev = st + (size_t)k * N;",
                        "const cplx *prev = st + (size_t)(k + 1) * N;"),
    "dry_sign": ("mat2 u = {{{-0.5 * s, -0.5 * c}, {0.5 * c, -0.5 * s}}};",
                 "mat2 u = {{{-0.5 * s, 0.5 * c}, {-0.5 * c, -0.5 * s}}};"),
    "h_sign": ("h += ((x >> j) & 1) ? -g[j] : g[j];", "h += ((x >> j) & 1) ? g[j] : -g[j];"),
    "slot_overwrite": ("dparams[(size_t)b * P + op->idx[s]] += acc;",
                       "dparams[(size_t)b * P + op->idx[s]] = acc;"),
    "input_slot_dropped": ("else dinputs[(size_t)b * F + op->idx[s]] += acc;", "else (void)0;"),
}

PIN_CALLS = [
    ("single_gate", lambda o: pins.test_single_gate_closed_forms(o)),
    ("bloch_formula", lambda o: pins.test_rx_rz_ry_bloch_formula(o)),
    ("product_bloch", lambda o: pins.test_random_product_circuits_vs_bloch(o, 3)),
    ("dense", lambda o: pins.test_random_circuits_vs_dense(o, 4, 3)),
    ("classical", lambda o: pins.test_classical_cnot_networks(o, 5)),
    ("one_layer", lambda o: pins.test_one_layer_closed_forms(o, 1, 4)),
    ("one_layer_cz", lambda o: pins.test_one_layer_closed_forms(o, 4, 9)),
    ("param_shift", lambda o: pins.test_vjp_vs_parameter_shift(o, 3, 12)),
    ("grad_closed", lambda o: pins.test_single_qubit_gradient_closed_form(o)),
]


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutant_fails_some_pin(tmp_path, monkeypatch, name):
    old, new = MUTANTS[name]
    src = open(oracle._SRC).read()
    assert src.count(old) == 1, f"mutation anchor for {name} not unique"
    path = tmp_path / "mutant.c"
    path.write_text(src.replace(old, new))
    so = tmp_path / f"liboracle_{name}.so"
    subprocess.check_call(["gcc", "-std=c99", "-O2", "-fopenmp", "-fPIC", "-shared",
                           "-o", str(so), str(path), "-lm"])
    monkeypatch.setattr(oracle, "_lib", oracle.open_library(str(so)))
    failed = []
    for pin, call in PIN_CALLS:
        try:
            call(oracle)
        except (AssertionError, ValueError):
            failed.append(pin)
    assert failed, f"mutant {name} passed every pin"
