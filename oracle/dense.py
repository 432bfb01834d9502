"""Dense-unitary forward pass -- TEST INFRASTRUCTURE ONLY (a second oracle).

Independent of the C oracle: every gate is a full 2^n x 2^n matrix.  One-qubit
rotations are built as matrix exponentials exp(-i t P / 2) of the Pauli
matrices (scipy.linalg.expm), lifted to n qubits with Kronecker products
(qubit j = bit j of the basis index, so qubit 0 is the right-most factor);
CNOT and CZ are written as permutation / diagonal matrices from their action
on basis states.  The whole circuit is the ordered matrix product applied to
|0...0> (or a given initial state), and <Z_j> is read off the probabilities (Algorithm 1, return
statement).  Meant for n <= 8.
"""
from __future__ import annotations

import numpy as np
from scipy.linalg import expm

_X = np.array([[0, 1], [1, 0]], dtype=np.complex128)
_Y = np.array([[0, -1j], [1j, 0]], dtype=np.complex128)
_Z = np.array([[1, 0], [0, -1]], dtype=np.complex128)
_PAULI = {"RX": _X, "RY": _Y, "RZ": _Z}


def rotation(kind: str, t: float) -> np.ndarray:
    return expm(-0.5j * t * _PAULI[kind])


def rot(phi: float, theta: float, omega: float) -> np.ndarray:
    """ROT(phi, theta, omega) = RZ(omega) RY(theta) RZ(phi)."""
    return rotation("RZ", omega) @ rotation("RY", theta) @ rotation("RZ", phi)


def lift_1q(u: np.ndarray, q: int, n: int) -> np.ndarray:
    return np.kron(np.kron(np.eye(1 << (n - q - 1)), u), np.eye(1 << q))


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


def _angle(spec, params_row, inputs_row):
    src, v = spec
    if src == "param":
        return float(params_row[int(v)])
    if src == "input":
        return float(inputs_row[int(v)])
    return float(v)


def circuit_unitary(ops, n: int, params_row, inputs_row) -> np.ndarray:
    U = np.eye(1 << n, dtype=np.complex128)
    for op in ops:
        if op.kind == "CNOT":
            G = cnot_matrix(op.wires[0], op.wires[1], n)
        elif op.kind == "CZ":
            G = cz_matrix(op.wires[0], op.wires[1], n)
        elif op.kind == "ROT":
            a = [_angle(s, params_row, inputs_row) for s in op.angles]
            G = lift_1q(rot(*a), op.wires[0], n)
        else:
            G = lift_1q(rotation(op.kind, _angle(op.angles[0], params_row, inputs_row)),
                        op.wires[0], n)
        U = G @ U
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
