"""The rotation rewrite behind the generated kernels, checked on the CPU.

The generated kernels apply R_P(theta) = cos(phi') (I - i tan(phi') P) P^m
(phi' = theta/2 - m pi/2 in [-pi/4, pi/4]), keep the Paulis P^m aside as a
frame that only flips signs, and apply the cos(phi') factors in blocks.  This
test replays that bookkeeping gate by gate on a dense state (numpy, complex128)
for random circuits and compares <Z_q> with the oracle: it pins the
decomposition, the frame updates through CNOT / CZ and the <Z> sign rule that
the kernels rely on.  No GPU is involved.
"""
import numpy as np
import pytest

import oracle
from paper_2607_11985_amd import workloads as W

X = np.array([[0, 1], [1, 0]], complex)
Y = np.array([[0, -1j], [1j, 0]])
Z = np.diag([1.0, -1.0]).astype(complex)
I2 = np.eye(2)
PAULI = {"RX": X, "RY": Y, "RZ": Z}


def apply1(psi, m, q, n):
    psi = psi.reshape([2] * n)
    ax = n - 1 - q  # qubit q is bit q of the basis index
    psi = np.moveaxis(np.tensordot(m, psi, axes=([1], [ax])), 0, ax)
    return psi.reshape(-1)


def lowered(ops, params, inputs, b):
    def ang(a):
        src, v = a
        return v if src == "const" else (params[b, v] if src == "param" else inputs[b, v])
    out = []
    for o in ops:
        if o.kind == "ROT":
            ph, th, om = (ang(a) for a in o.angles)
            out += [("RZ", o.wires[0], ph), ("RY", o.wires[0], th), ("RZ", o.wires[0], om)]
        elif o.kind in ("CNOT", "CZ"):
            out.append((o.kind, o.wires[0], o.wires[1]))
        else:
            out.append((o.kind, o.wires[0], ang(o.angles[0])))
    return out


def tangent_expvals(ops, n, params, inputs, block=24):
    idx = np.arange(2 ** n)
    E = np.zeros((params.shape[0], n))
    for b in range(params.shape[0]):
        psi = np.zeros(2 ** n, complex)
        psi[0] = 1.0
        fx = fz = 0  # frame: x bits, z bits
        scale, since = 1.0, 0
        for g in lowered(ops, params, inputs, b):
            if g[0] == "CNOT":
                c, t = g[1], g[2]
                m = ((idx >> c) & 1) == 1
                psi = np.where(m, psi[idx ^ (1 << t)], psi)
                fx ^= ((fx >> c) & 1) << t
                fz ^= ((fz >> t) & 1) << c
                continue
            if g[0] == "CZ":
                a, bb = g[1], g[2]
                psi = psi * np.where(((idx >> a) & 1) & ((idx >> bb) & 1), -1, 1)
                fz ^= (((fx >> a) & 1) << bb) | (((fx >> bb) & 1) << a)
                continue
            kind, q, th = g
            c, s = np.cos(th / 2), np.sin(th / 2)
            odd = abs(s) > abs(c)
            t = -c / s if odd else s / c
            assert abs(t) <= 1 + 1e-12
            anti = {"RX": fz >> q, "RY": (fx ^ fz) >> q, "RZ": fx >> q}[kind] & 1
            psi = apply1(psi, I2 - 1j * (-t if anti else t) * PAULI[kind], q, n)
            scale *= abs(s) if odd else abs(c)
            since += 1
            if since == block:
                psi, scale, since = psi * scale, 1.0, 0
            if odd:
                fx ^= (1 << q) if kind in ("RX", "RY") else 0
                fz ^= (1 << q) if kind in ("RY", "RZ") else 0
        psi = psi * scale
        assert abs(np.vdot(psi, psi) - 1) < 1e-9
        for q in range(n):
            e = np.sum(np.where((idx >> q) & 1, -1.0, 1.0) * np.abs(psi) ** 2)
            E[b, q] = -e if (fx >> q) & 1 else e
    return E


@pytest.mark.parametrize("n,seed", [(3, 1), (5, 2), (7, 3), (8, 4)])
def test_tangent_form_matches_oracle(n, seed):
    ops, P, F = W.random_circuit(n, 30 + 8 * n, seed=900 + seed,
                                 kinds=("RX", "RY", "RZ", "ROT", "CNOT", "CZ"))
    params, inputs = W.random_inputs(3, P, F, seed=910 + seed)
    E = tangent_expvals(ops, n, params.astype(np.float64), inputs.astype(np.float64))
    Er = oracle.forward(ops, n, params, inputs)
    assert np.max(np.abs(E - Er)) < 1e-10
