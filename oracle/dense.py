"""Dense-unitary forward pass -- TEST INFRASTRUCTURE ONLY (a second oracle).

Independent of the C oracle: every gate is a full 2^n x 2^n matrix built a
different way.  Rotations are matrix exponentials exp(-i t G / 2) of Pauli
strings (scipy.linalg.expm), phase-type gates are e^{i a} times such an
exponential (S, T, SX, P, U3 as e^{i(p+l)/2} RZ(p) RY(t) RZ(l)), controlled
gates are sums of projector products |0><0|_c (x) I + |1><1|_c (x) U, SWAP is
(I + XX + YY + ZZ)/2, and the three-qubit gates are projector sums too.  One-
qubit factors are lifted to n qubits with Kronecker products (qubit j = bit j
of the basis index, so qubit 0 is the right-most factor).  The whole circuit
is the ordered matrix product applied to |0...0> (or a given initial state),
and <Z_j> is read off the probabilities (Algorithm 1, return statement).
Meant for n <= 8.
"""
from __future__ import annotations

import numpy as np
from scipy.linalg import expm

_X = np.array([[0, 1], [1, 0]], dtype=np.complex128)
_Y = np.array([[0, -1j], [1j, 0]], dtype=np.complex128)
_Z = np.array([[1, 0], [0, -1]], dtype=np.complex128)
_PAULI = {"RX": _X, "RY": _Y, "RZ": _Z}


_I2 = np.eye(2, dtype=np.complex128)
_P0 = np.diag([1.0, 0.0]).astype(np.complex128)
_P1 = np.diag([0.0, 1.0]).astype(np.complex128)


def rotation(kind: str, t: float) -> np.ndarray:
    return expm(-0.5j * t * _PAULI[kind])


def rot(phi: float, theta: float, omega: float) -> np.ndarray:
    """ROT(phi, theta, omega) = RZ(omega) RY(theta) RZ(phi)."""
    return rotation("RZ", omega) @ rotation("RY", theta) @ rotation("RZ", phi)


def u3(theta: float, phi: float, lam: float) -> np.ndarray:
    return np.exp(0.5j * (phi + lam)) * rot(lam, theta, phi)


def lift_1q(u: np.ndarray, q: int, n: int) -> np.ndarray:
    return np.kron(np.kron(np.eye(1 << (n - q - 1)), u), np.eye(1 << q))


def op_on(n: int, factors: dict) -> np.ndarray:
    """Kronecker product with factors[q] on qubit q and identity elsewhere."""
    m = np.eye(1, dtype=np.complex128)
    for q in range(n - 1, -1, -1):
        m = np.kron(m, factors.get(q, _I2))
    return m


def controlled(u: np.ndarray, c: int, t: int, n: int) -> np.ndarray:
    return op_on(n, {c: _P0}) + op_on(n, {c: _P1, t: u})


def cnot_matrix(c: int, t: int, n: int) -> np.ndarray:
    N = 1 << n
    m = np.zeros((N, N), dtype=np.complex128)
    for x in range(N):
        y = x ^ (((x >> c) & 1) << t)
        m[y, x] = 1.0
    return m


def cz_matrix(a: int, b: int, n: int) -> np.ndarray:
    N = 1 << n
    d = np.array([-1.0 if ((x >> a) & 1) and ((x >> b) & 1) else 1.0 for x in range(N)])
    return np.diag(d).astype(np.complex128)


def swap_matrix(a: int, b: int, n: int, extra=None) -> np.ndarray:
    extra = extra or {}
    terms = [op_on(n, dict(extra))]
    for P in (_X, _Y, _Z):
        f = dict(extra)
        f[a], f[b] = P, P
        terms.append(op_on(n, f))
    return 0.5 * sum(terms)


_FIXED_1Q = {
    "ID": lambda: _I2, "X": lambda: _X, "Y": lambda: _Y, "Z": lambda: _Z,
    "H": lambda: (_X + _Z) / np.sqrt(2.0),
    "S": lambda: np.exp(0.25j * np.pi) * rotation("RZ", np.pi / 2),
    "SDG": lambda: np.exp(-0.25j * np.pi) * rotation("RZ", -np.pi / 2),
    "T": lambda: np.exp(0.125j * np.pi) * rotation("RZ", np.pi / 4),
    "TDG": lambda: np.exp(-0.125j * np.pi) * rotation("RZ", -np.pi / 4),
    "SX": lambda: np.exp(0.25j * np.pi) * rotation("RX", np.pi / 2),
    "SXDG": lambda: np.exp(-0.25j * np.pi) * rotation("RX", -np.pi / 2),
}


def _angle(spec, params_row, inputs_row):
    src, v = spec[0], spec[1]
    if src == "const":
        return float(v)
    x = float(params_row[int(v)]) if src == "param" else float(inputs_row[int(v)])
    mul = float(spec[2]) if len(spec) > 2 else 1.0
    add = float(spec[3]) if len(spec) > 3 else 0.0
    return mul * x + add


def gate_unitary(op, n: int, a) -> np.ndarray:
    k, w = op.kind, op.wires
    if k in ("CNOT", "CX"):
        return cnot_matrix(w[0], w[1], n)
    if k == "CZ":
        return cz_matrix(w[0], w[1], n)
    if k in _FIXED_1Q:
        return lift_1q(_FIXED_1Q[k](), w[0], n)
    if k in ("RX", "RY", "RZ"):
        return lift_1q(rotation(k, a[0]), w[0], n)
    if k == "ROT":
        return lift_1q(rot(*a), w[0], n)
    if k in ("P", "U1"):
        return lift_1q(np.exp(0.5j * a[0]) * rotation("RZ", a[0]), w[0], n)
    if k == "U2":
        return lift_1q(u3(np.pi / 2, a[0], a[1]), w[0], n)
    if k in ("U3", "U"):
        return lift_1q(u3(*a), w[0], n)
    if k == "CY":
        return controlled(_Y, w[0], w[1], n)
    if k == "CH":
        return controlled(_FIXED_1Q["H"](), w[0], w[1], n)
    if k in ("CRX", "CRY", "CRZ"):
        return controlled(rotation(k[1:], a[0]), w[0], w[1], n)
    if k == "CP":
        return controlled(np.exp(0.5j * a[0]) * rotation("RZ", a[0]), w[0], w[1], n)
    if k in ("RXX", "RYY", "RZZ"):
        P = _PAULI["R" + k[1]]
        return expm(-0.5j * a[0] * op_on(n, {w[0]: P, w[1]: P}))
    if k == "SWAP":
        return swap_matrix(w[0], w[1], n)
    if k == "CCX":
        c0, c1, t = w
        return np.eye(1 << n) - op_on(n, {c0: _P1, c1: _P1}) + op_on(n, {c0: _P1, c1: _P1, t: _X})
    if k == "CSWAP":
        c, a0, b0 = w
        return op_on(n, {c: _P0}) + swap_matrix(a0, b0, n, {c: _P1})
    raise ValueError(k)


def circuit_unitary(ops, n: int, params_row, inputs_row) -> np.ndarray:
    U = np.eye(1 << n, dtype=np.complex128)
    for op in ops:
        a = [_angle(s, params_row, inputs_row) for s in op.angles]
        U = gate_unitary(op, n, a) @ U
    return U


def forward(ops, n: int, params, inputs, want_state: bool = False, psi0=None):
    params = np.asarray(params, dtype=np.float64)
    inputs = np.asarray(inputs, dtype=np.float64)
    B = params.shape[0]
    N = 1 << n
    E = np.zeros((B, n))
    states = np.zeros((B, N), dtype=np.complex128)
    signs = np.array([[1.0 - 2.0 * ((x >> j) & 1) for j in range(n)] for x in range(N)])
    for b in range(B):
        U = circuit_unitary(ops, n, params[b], inputs[b])
        psi = U[:, 0] if psi0 is None else U @ np.asarray(psi0[b], dtype=np.complex128)
        states[b] = psi
        E[b] = (np.abs(psi) ** 2) @ signs
    return (E, states) if want_state else E
