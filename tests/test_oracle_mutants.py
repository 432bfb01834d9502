"""The pins are sensitive: plant plausible mistakes in a copy of the oracle.

Each mutant is a textual edit of a temporary copy of the oracle's C source,
compiled on the CPU; the committed oracle is untouched.  Every mutant must
make at least one pin of test_oracle_pins fail.
"""
import os
import subprocess

import pytest

import oracle
from tests import test_oracle_gates as gates
from tests import test_oracle_pins as pins

MUTANTS = {
    "rx_sign": ("return mk2(c, -I * s, -I * s, c); }", "return mk2(c, I * s, I * s, c); }"),
    "ry_transposed": ("return mk2(c, -s, s, c); }", "return mk2(c, s, -s, c); }"),
    "rz_direction": ("return mk2(cexp(-I * t / 2), 0, 0, cexp(I * t / 2)); }",
                     "return mk2(cexp(I * t / 2), 0, 0, cexp(-I * t / 2)); }"),
    "rot_order": ("return mul2(x, mul2(y, z));", "return mul2(z, mul2(y, x));"),
    "full_angle": ("static mat2 m_ry(double t) { double c = cos(t / 2), s = sin(t / 2);",
                   "static mat2 m_ry(double t) { double c = cos(t), s = sin(t);"),
    "control_on_wire1": ("M[(1 + 2 * i) * 4 + (1 + 2 * j)] = u.m[i][j];",
                         "M[(2 + i) * 4 + (2 + j)] = u.m[i][j];"),
    "cz_as_cx": ("case ORC_CZ: return one_qubit(ORC_Z, a, -1);",
                 "case ORC_CZ: return one_qubit(ORC_X, a, -1);"),
    "z_sign": ("acc += ((x >> j) & 1) ? -p : p;", "acc += ((x >> j) & 1) ? p : -p;"),
    "vjp_factor": ("acc *= 2.0 * op->mul[s];", "acc *= 1.0 * op->mul[s];"),
    "vjp_no_mul": ("acc *= 2.0 * op->mul[s];", "acc *= 2.0;"),
    "affine_add_dropped": ("ang[s] = op->mul[s] * inputs[(size_t)b * F + op->idx[s]] + op->add[s];",
                           "ang[s] = op->mul[s] * inputs[(size_t)b * F + op->idx[s]];"),
    "vjp_no_dagger": ("apply_op(lam, n, op, ang, 1);", "apply_op(lam, n, op, ang, 0);"),
    "vjp_wrong_state": ("const cplx *prev = st + (size_t)k * N;",
                        "const cplx *prev = st + (size_t)(k + 1) * N;"),
    "dry_sign": ("return mk2(-0.5 * s, -0.5 * c, 0.5 * c, -0.5 * s);",
                 "return mk2(-0.5 * s, 0.5 * c, -0.5 * c, -0.5 * s);"),
    "h_sign": ("h += ((x >> j) & 1) ? -g[j] : g[j];", "h += ((x >> j) & 1) ? g[j] : -g[j];"),
    "slot_overwrite": ("dparams[(size_t)b * P + op->idx[s]] += acc;",
                       "dparams[(size_t)b * P + op->idx[s]] = acc;"),
    "input_slot_dropped": ("else dinputs[(size_t)b * F + op->idx[s]] += acc;", "else (void)0;"),
    "hadamard_as_ry": ("case ORC_H: return mk2(r2, r2, r2, -r2);",
                       "case ORC_H: return mk2(r2, -r2, r2, r2);"),
    "s_conjugated": ("case ORC_S: return mk2(1, 0, 0, I);", "case ORC_S: return mk2(1, 0, 0, -I);"),
    "t_eighth": ("case ORC_T: return mk2(1, 0, 0, cexp(I * ORC_PI / 4));",
                 "case ORC_T: return mk2(1, 0, 0, cexp(I * ORC_PI / 8));"),
    "sx_as_sxdg": ("case ORC_SX: return mk2(0.5 * (1 + I), 0.5 * (1 - I), 0.5 * (1 - I), 0.5 * (1 + I));",
                   "case ORC_SX: return mk2(0.5 * (1 - I), 0.5 * (1 + I), 0.5 * (1 + I), 0.5 * (1 - I));"),
    "u3_phi_lambda_swapped": ("default: return mk2(c, -el * s, ep * s, epl * c);",
                              "default: return mk2(c, -ep * s, el * s, epl * c);"),
    "u3_dphi_wrong": ("case 1: return mk2(0, 0, I * ep * s, I * epl * c);",
                      "case 1: return mk2(0, 0, I * ep * s, 0);"),
    "u2_slot_shift": ("case ORC_U2: return m_u3(ORC_PI / 2, a[0], a[1], d < 0 ? -1 : d + 1);",
                      "case ORC_U2: return m_u3(ORC_PI / 2, a[0], a[1], d < 0 ? -1 : d);"),
    "yy_sign": ("else M[(l ^ 3) * 4 + l] += cg * (par ? 1.0 : -1.0);",
                "else M[(l ^ 3) * 4 + l] += cg * (par ? -1.0 : 1.0);"),
    "zz_parity": ("if (kind == ORC_RZZ) M[l * 4 + l] += cg * (par ? -1.0 : 1.0);",
                  "if (kind == ORC_RZZ) M[l * 4 + l] += cg * ((l & 1) ? -1.0 : 1.0);"),
    "ccx_target": ("M[((l & 3) == 3 ? l ^ 4 : l) * 8 + l] = 1;",
                   "M[((l & 5) == 5 ? l ^ 2 : l) * 8 + l] = 1;"),
    "cswap_swaps_control": ("if (l & 1) r = (l & 1) | (((l >> 2) & 1) << 1) | (((l >> 1) & 1) << 2);",
                            "if (l & 4) r = (l & 4) | ((l & 1) << 1) | ((l >> 1) & 1);"),
    "swap_identity": ("for (int l = 0; l < 4; ++l) M[(((l & 1) << 1) | (l >> 1)) * 4 + l] = 1;",
                      "for (int l = 0; l < 4; ++l) M[l * 4 + l] = 1;"),
    "controlled_no_identity": ("if (d < 0) { M[0 * 4 + 0] = 1; M[2 * 4 + 2] = 1; }",
                               "if (d < 0) { M[0 * 4 + 0] = 1; }"),
    "controlled_derivative_identity": ("if (d < 0) { M[0 * 4 + 0] = 1; M[2 * 4 + 2] = 1; }",
                                       "{ M[0 * 4 + 0] = 1; M[2 * 4 + 2] = 1; }"),
    "wire_order_reversed": ("if ((l >> i) & 1) off[l] |= (size_t)1 << w[i];",
                            "if ((l >> i) & 1) off[l] |= (size_t)1 << w[k - 1 - i];"),
    "cp_phase_on_target_only": ("default: return one_qubit(ORC_P, a, d); /* ORC_CP */",
                                "default: return one_qubit(ORC_RZ, a, d); /* ORC_CP */"),
    "psi0_ignored": ("if (psi0) memcpy(psi, psi0 + (size_t)b * N * 2, N * sizeof(cplx));\n        else psi[0] = 1.0;",
                     "psi[0] = 1.0;"),
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
    ("psi0_bloch", lambda o: pins.test_psi0_product_states_vs_bloch(o, 2)),
    ("gates_dense", lambda o: gates.test_general_circuits_vs_dense(o, 4, 3)),
    ("gates_truth", lambda o: gates.test_classical_gates_truth_tables(o)),
    ("gates_control", lambda o: [gates.test_controlled_gates_by_control_value(o, k, s)
                                 for k, s in (("CRX", "RX"), ("CP", "P"), ("CNOT", "X"))]),
    ("gates_u3_bloch", lambda o: gates.test_u3_and_h_bloch(o)),
    ("gates_identities", lambda o: [gates.test_gate_identities(o, *i) for i in gates.IDENTITIES]),
    ("gates_shift", lambda o: gates.test_general_vjp_vs_parameter_shift(o, 3, 1)),
    ("gates_fd", lambda o: gates.test_controlled_rotation_vjp_vs_differences(o, 2, 0)),
    ("gates_affine", lambda o: gates.test_affine_angles_equal_substituted_constants(o)),
    ("gates_chain", lambda o: gates.test_affine_chain_rule(o)),
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
            break
    assert failed, f"mutant {name} passed every pin"
