"""Pins of the oracle's general static gate set (the OpenQASM standard gates
the compile phase lowers, Sec. 3 and Algorithm 1) and of affine angles.

Independent facts used:
  * a dense construction that builds every gate another way (matrix
    exponentials of Pauli strings with explicit global phases, projector sums
    for controlled, swap and three-qubit gates): oracle.dense;
  * algebraic identities between gates (H^2 = I, S^2 = Z, T^2 = S, SX^2 = X,
    H Z H = X, U3 special cases, CP(pi) = CZ, SWAP = three CNOTs, R_ZZ as a
    CNOT-conjugated RZ, ...), compared as exact states from random Psi_0;
  * truth tables of the classical gates (SWAP, CCX, CSWAP) on basis states;
  * Bloch-vector closed forms for U3 and H;
  * controlled gates with the control in |0> (identity) and |1> (the target
    gate);
  * gradients: the two-term shift rule where it is exact, central differences
    for the controlled rotations, and the chain rule through mul * value + add.
"""
import math

import numpy as np
import pytest

from paper_2607_11985_amd import workloads as W

TOL = 1e-13
Op = W.Op


def _states(rng, B, n):
    s = rng.normal(size=(B, 1 << n)) + 1j * rng.normal(size=(B, 1 << n))
    return s / np.linalg.norm(s, axis=1, keepdims=True)


def _run(oracle_mod, ops, n, psi0, params=None, inputs=None):
    B = psi0.shape[0]
    p = np.zeros((B, 1)) if params is None else params
    x = np.zeros((B, 1)) if inputs is None else inputs
    _, st = oracle_mod.forward(ops, n, p, x, want_state=True, psi0=psi0)
    return st


def _same(a, b, tol=TOL):
    assert np.max(np.abs(a - b)) < tol, float(np.max(np.abs(a - b)))


def _same_up_to_phase(a, b, tol=1e-12):
    for u, v in zip(a, b):
        k = int(np.argmax(np.abs(v)))
        ph = u[k] / v[k]
        assert abs(abs(ph) - 1) < tol
        assert np.max(np.abs(u - ph * v)) < tol


def C(v):
    return ("const", float(v))


# ------------------------------------------------------------- vs dense

@pytest.mark.parametrize("n,seed", [(1, 0), (2, 1), (3, 2), (4, 3), (5, 4)])
def test_general_circuits_vs_dense(oracle_mod, n, seed):
    from oracle import dense
    ops, P, F = W.random_circuit(n, 40, seed=500 + seed, kinds=W.GENERAL_KINDS,
                                 p_affine=0.4)
    p, x = W.random_inputs(3, P, F, seed=510 + seed)
    psi0 = _states(np.random.default_rng(520 + seed), 3, n)
    E, st = oracle_mod.forward(ops, n, p, x, want_state=True, psi0=psi0)
    Ed, sd = dense.forward(ops, n, p, x, want_state=True, psi0=psi0)
    assert np.max(np.abs(E - Ed)) < 1e-12
    # both constructions are exact matrices: states agree without a phase
    assert np.max(np.abs(st - sd)) < 1e-12


@pytest.mark.parametrize("kind", [k for k in W.GENERAL_KINDS])
def test_each_gate_vs_dense(oracle_mod, kind):
    from oracle import dense
    nw, na = W.GATE_SHAPES[kind]
    n = 4
    rng = np.random.default_rng(sum(map(ord, kind)))
    wires = tuple(int(v) for v in rng.choice(n, size=nw, replace=False))
    ang = tuple(C(rng.uniform(-4, 4)) for _ in range(na))
    ops = [Op(kind, wires, ang)]
    psi0 = _states(rng, 2, n)
    st = _run(oracle_mod, ops, n, psi0)
    _, sd = dense.forward(ops, n, np.zeros((2, 1)), np.zeros((2, 1)), want_state=True, psi0=psi0)
    _same(st, sd, 1e-12)


# ------------------------------------------------------------ identities

IDENTITIES = [
    ("HH=I", [Op("H", (1,)), Op("H", (1,))], [Op("ID", (1,))]),
    ("SS=Z", [Op("S", (0,)), Op("S", (0,))], [Op("Z", (0,))]),
    ("TT=S", [Op("T", (2,)), Op("T", (2,))], [Op("S", (2,))]),
    ("SXSX=X", [Op("SX", (1,)), Op("SX", (1,))], [Op("X", (1,))]),
    ("SSDG=I", [Op("S", (1,)), Op("SDG", (1,))], []),
    ("TTDG=I", [Op("TDG", (0,)), Op("T", (0,))], []),
    ("SXSXDG=I", [Op("SXDG", (2,)), Op("SX", (2,))], []),
    ("HZH=X", [Op("H", (0,)), Op("Z", (0,)), Op("H", (0,))], [Op("X", (0,))]),
    ("HXH=Z", [Op("H", (2,)), Op("X", (2,)), Op("H", (2,))], [Op("Z", (2,))]),
    ("XY=iZ", [Op("Y", (1,)), Op("X", (1,))], [Op("Z", (1,))], 1j),
    ("RX(pi)=-iX", [Op("RX", (0,), (C(math.pi),))], [Op("X", (0,))], -1j),
    ("RXX(pi)=-iXX", [Op("RXX", (0, 2), (C(math.pi),))], [Op("X", (0,)), Op("X", (2,))], -1j),
    ("SX=e^{i pi/4}RX(pi/2)", [Op("SX", (2,))], [Op("RX", (2,), (C(math.pi / 2),))],
     np.exp(0.25j * math.pi)),
    ("U3(t,0,0)=RY", [Op("U3", (1,), (C(0.7), C(0), C(0)))], [Op("RY", (1,), (C(0.7),))]),
    ("U3(t,-pi/2,pi/2)=RX", [Op("U3", (0,), (C(1.3), C(-math.pi / 2), C(math.pi / 2)))],
     [Op("RX", (0,), (C(1.3),))]),
    ("U3(0,0,l)=P", [Op("U3", (2,), (C(0), C(0), C(0.9)))], [Op("P", (2,), (C(0.9),))]),
    ("U2=U3(pi/2)", [Op("U2", (1,), (C(0.4), C(-1.1)))],
     [Op("U3", (1,), (C(math.pi / 2), C(0.4), C(-1.1)))]),
    ("P(pi/2)=S", [Op("P", (0,), (C(math.pi / 2),))], [Op("S", (0,))]),
    ("P(pi/4)=T", [Op("P", (0,), (C(math.pi / 4),))], [Op("T", (0,))]),
    ("CP(pi)=CZ", [Op("CP", (0, 2), (C(math.pi),))], [Op("CZ", (0, 2))]),
    ("CP symmetric", [Op("CP", (0, 2), (C(0.8),))], [Op("CP", (2, 0), (C(0.8),))]),
    ("CZ symmetric", [Op("CZ", (1, 2))], [Op("CZ", (2, 1))]),
    ("SWAP=3CNOT", [Op("SWAP", (0, 2))],
     [Op("CNOT", (0, 2)), Op("CNOT", (2, 0)), Op("CNOT", (0, 2))]),
    ("SWAP symmetric", [Op("SWAP", (1, 2))], [Op("SWAP", (2, 1))]),
    ("CY=S CX SDG", [Op("CY", (1, 0))], [Op("SDG", (0,)), Op("CNOT", (1, 0)), Op("S", (0,))]),
    ("CZ=H CX H", [Op("CZ", (2, 1))], [Op("H", (1,)), Op("CNOT", (2, 1)), Op("H", (1,))]),
    ("RZZ=CX RZ CX", [Op("RZZ", (0, 2), (C(1.1),))],
     [Op("CNOT", (0, 2)), Op("RZ", (2,), (C(1.1),)), Op("CNOT", (0, 2))]),
    ("RXX=HH RZZ HH", [Op("RXX", (1, 2), (C(-0.6),))],
     [Op("H", (1,)), Op("H", (2,)), Op("RZZ", (1, 2), (C(-0.6),)), Op("H", (1,)), Op("H", (2,))]),
    ("RYY=RX RZZ RX", [Op("RYY", (0, 1), (C(2.2),))],
     [Op("RX", (0,), (C(math.pi / 2),)), Op("RX", (1,), (C(math.pi / 2),)),
      Op("RZZ", (0, 1), (C(2.2),)),
      Op("RX", (0,), (C(-math.pi / 2),)), Op("RX", (1,), (C(-math.pi / 2),))]),
    ("CRZ=RZ CX RZ CX", [Op("CRZ", (1, 2), (C(0.9),))],
     [Op("RZ", (2,), (C(0.45),)), Op("CNOT", (1, 2)), Op("RZ", (2,), (C(-0.45),)),
      Op("CNOT", (1, 2))]),
    ("CRY=RY CX RY CX", [Op("CRY", (0, 1), (C(-1.7),))],
     [Op("RY", (1,), (C(-0.85),)), Op("CNOT", (0, 1)), Op("RY", (1,), (C(0.85),)),
      Op("CNOT", (0, 1))]),
    ("CRX=H CRZ H", [Op("CRX", (2, 0), (C(2.5),))],
     [Op("H", (0,)), Op("CRZ", (2, 0), (C(2.5),)), Op("H", (0,))]),
    ("CH=RY CZ RY", [Op("CH", (0, 2))],
     [Op("RY", (2,), (C(-math.pi / 4),)), Op("CZ", (0, 2)), Op("RY", (2,), (C(math.pi / 4),))]),
    ("CCX controls symmetric", [Op("CCX", (0, 1, 2))], [Op("CCX", (1, 0, 2))]),
    ("CSWAP targets symmetric", [Op("CSWAP", (2, 0, 1))], [Op("CSWAP", (2, 1, 0))]),
    ("CCX^2=I", [Op("CCX", (2, 0, 1)), Op("CCX", (2, 0, 1))], []),
]


IDENTITIES = [i if len(i) == 4 else i + (1.0,) for i in IDENTITIES]


@pytest.mark.parametrize("name,lhs,rhs,phase", IDENTITIES, ids=[i[0] for i in IDENTITIES])
def test_gate_identities(oracle_mod, name, lhs, rhs, phase):
    """lhs = phase * rhs as operators, checked on random states (all exact)."""
    n = 3
    psi0 = _states(np.random.default_rng(600), 3, n)
    a = _run(oracle_mod, lhs, n, psi0)
    b = _run(oracle_mod, rhs, n, psi0) if rhs else psi0
    _same(a, phase * b)


# ------------------------------------------------------- truth tables

def _basis(n, k):
    s = np.zeros((1, 1 << n), dtype=complex)
    s[0, k] = 1.0
    return s


def test_classical_gates_truth_tables(oracle_mod):
    n = 4
    for k in range(1 << n):
        bit = lambda q: (k >> q) & 1
        # SWAP(0, 3)
        y = k & ~0b1001 | (bit(0) << 3) | (bit(3) << 0)
        _same(_run(oracle_mod, [Op("SWAP", (0, 3))], n, _basis(n, k)), _basis(n, y))
        # CCX(2, 0 -> 1)
        y = k ^ ((bit(2) & bit(0)) << 1)
        _same(_run(oracle_mod, [Op("CCX", (2, 0, 1))], n, _basis(n, k)), _basis(n, y))
        # CSWAP(3; 1, 2)
        y = k
        if bit(3):
            y = k & ~0b0110 | (bit(1) << 2) | (bit(2) << 1)
        _same(_run(oracle_mod, [Op("CSWAP", (3, 1, 2))], n, _basis(n, k)), _basis(n, y))
        # X flips, Z / S / T only phase
        _same(_run(oracle_mod, [Op("X", (2,))], n, _basis(n, k)), _basis(n, k ^ 4))
        ph = {0: 1, 1: 1j}[bit(1)]
        _same(_run(oracle_mod, [Op("S", (1,))], n, _basis(n, k)), ph * _basis(n, k))
        ph = np.exp(0.25j * math.pi) if bit(2) else 1
        _same(_run(oracle_mod, [Op("T", (2,))], n, _basis(n, k)), ph * _basis(n, k))
        # RZZ(t) on a basis state: phase e^{-i t/2 (-1)^{x_a + x_b}}
        t = 0.77
        ph = np.exp(-0.5j * t * (1 - 2 * (bit(0) ^ bit(2))))
        _same(_run(oracle_mod, [Op("RZZ", (0, 2), (C(t),))], n, _basis(n, k)),
              ph * _basis(n, k))


@pytest.mark.parametrize("kind,single", [("CRX", "RX"), ("CRY", "RY"), ("CRZ", "RZ"),
                                         ("CP", "P"), ("CY", "Y"), ("CH", "H"), ("CNOT", "X"),
                                         ("CZ", "Z")])
def test_controlled_gates_by_control_value(oracle_mod, kind, single):
    """Control |0>: nothing happens; control |1>: the single-qubit gate on the target."""
    n = 3
    c, t = 2, 0
    rng = np.random.default_rng(610)
    na = W.GATE_SHAPES[kind][1]
    ang = tuple(C(rng.uniform(-3, 3)) for _ in range(na))
    for cv in (0, 1):
        other = _states(rng, 2, 2)  # qubits 0, 1
        psi0 = np.zeros((2, 8), dtype=complex)
        for k in range(4):
            psi0[:, k | (cv << 2)] = other[:, k]
        got = _run(oracle_mod, [Op(kind, (c, t), ang)], n, psi0)
        ref = psi0 if cv == 0 else _run(oracle_mod, [Op(single, (t,), ang)], n, psi0)
        _same(got, ref)


# ------------------------------------------------------ Bloch closed forms

def test_u3_and_h_bloch(oracle_mod):
    """U3(t, p, l)|0> has Bloch vector (sin t cos p, sin t sin p, cos t); a
    following H swaps the x and z components."""
    rng = np.random.default_rng(620)
    P = rng.uniform(-4, 4, size=(30, 3))
    ops = [Op("U3", (0,), (("param", 0), ("param", 1), ("param", 2)))]
    E = oracle_mod.forward(ops, 1, P, np.zeros((30, 1)))
    assert np.max(np.abs(E[:, 0] - np.cos(P[:, 0]))) < TOL
    E = oracle_mod.forward(ops + [Op("H", (0,))], 1, P, np.zeros((30, 1)))
    assert np.max(np.abs(E[:, 0] - np.sin(P[:, 0]) * np.cos(P[:, 1]))) < TOL
    # S before H maps y to x: <Z> = -sin t sin p
    E = oracle_mod.forward(ops + [Op("SDG", (0,)), Op("H", (0,))], 1, P, np.zeros((30, 1)))
    assert np.max(np.abs(E[:, 0] - np.sin(P[:, 0]) * np.sin(P[:, 1]))) < TOL
    # SX = RX(pi/2) up to phase: <Z> of SX U3|0> = cos t cos(pi/2) - ... = y-component
    E = oracle_mod.forward(ops + [Op("SX", (0,))], 1, P, np.zeros((30, 1)))
    assert np.max(np.abs(E[:, 0] - np.sin(P[:, 0]) * np.sin(P[:, 1]))) < TOL


# --------------------------------------------------------- affine angles

def test_affine_angles_equal_substituted_constants(oracle_mod):
    rng = np.random.default_rng(630)
    ops, P, F = W.random_circuit(4, 30, seed=631, kinds=W.GENERAL_KINDS, p_affine=1.0,
                                 p_const=0.0)
    p, x = W.random_inputs(2, P, F, seed=632)
    E = oracle_mod.forward(ops, 4, p, x)
    for b in range(2):
        const_ops = []
        for op in ops:
            ang = []
            for spec in op.angles:
                v = float(p[b, spec[1]] if spec[0] == "param" else x[b, spec[1]])
                mul = spec[2] if len(spec) > 2 else 1.0
                add = spec[3] if len(spec) > 3 else 0.0
                ang.append(C(mul * v + add))
            const_ops.append(Op(op.kind, op.wires, tuple(ang)))
        Eb = oracle_mod.forward(const_ops, 4, np.zeros((1, 1)), np.zeros((1, 1)))
        assert np.max(np.abs(E[b] - Eb[0])) < TOL


# -------------------------------------------------------------- gradients

_SHIFT_EXACT = tuple(k for k in W.GENERAL_KINDS if k not in ("CRX", "CRY", "CRZ"))


@pytest.mark.parametrize("n,seed", [(2, 0), (3, 1), (4, 2)])
def test_general_vjp_vs_parameter_shift(oracle_mod, n, seed):
    ops, P, F = W.random_circuit(n, 25, seed=640 + seed, kinds=_SHIFT_EXACT, p_affine=0.5)
    p, x = W.random_inputs(3, P, F, seed=650 + seed)
    g = W.random_cotangent(3, n, seed=660 + seed).astype(np.float64)
    dp, dx, _ = oracle_mod.vjp(ops, n, p, x, g)
    sp, sx = oracle_mod.param_shift_grad(ops, n, p, x, g)
    assert np.max(np.abs(dp - sp)) < 1e-12 and np.max(np.abs(dx - sx)) < 1e-12


@pytest.mark.parametrize("n,seed", [(2, 0), (4, 1)])
def test_controlled_rotation_vjp_vs_differences(oracle_mod, n, seed):
    ops, P, F = W.random_circuit(n, 20, seed=670 + seed,
                                 kinds=("CRX", "CRY", "CRZ", "RY", "H", "CNOT"), p_affine=0.5)
    p, x = W.random_inputs(3, P, F, seed=680 + seed)
    g = W.random_cotangent(3, n, seed=690 + seed).astype(np.float64)
    dp, dx, _ = oracle_mod.vjp(ops, n, p, x, g)
    fp, fx = oracle_mod.fd_grad(ops, n, p, x, g, h=1e-5)
    assert np.max(np.abs(dp - fp)) < 1e-8 and np.max(np.abs(dx - fx)) < 1e-8


def test_controlled_rotation_shift_rule_is_not_exact(oracle_mod):
    """The two-term rule fails for CRX (three generator eigenvalues): a check
    that the difference test above is the one that decides."""
    ops = [Op("H", (0,)), Op("CRX", (0, 1), (("param", 0),)), Op("H", (0,))]
    p = np.array([[0.9]])
    g = np.array([[1.0, 0.0]])
    dp, _, _ = oracle_mod.vjp(ops, 2, p, np.zeros((1, 1)), g)
    sp, _ = oracle_mod.param_shift_grad(ops, 2, p, np.zeros((1, 1)), g)
    # closed form: <Z_0> = Re <0| RX(t) |0> = cos(t/2)  ->  d/dt = -sin(t/2) / 2
    ref = -0.5 * math.sin(0.45)
    assert abs(dp[0, 0] - ref) < 1e-13
    assert abs(sp[0, 0] - ref) > 1e-3


def test_affine_chain_rule(oracle_mod):
    """d/dx of f(mul x + add) = mul f'(mul x + add): a scaled, offset copy of RY."""
    rng = np.random.default_rng(700)
    xs = rng.uniform(-3, 3, size=(20, 1))
    ops = [Op("RY", (0,), (("input", 0, -1.5, 0.25),))]
    E = oracle_mod.forward(ops, 1, np.zeros((20, 1)), xs)
    assert np.max(np.abs(E[:, 0] - np.cos(-1.5 * xs[:, 0] + 0.25))) < TOL
    _, dx, _ = oracle_mod.vjp(ops, 1, np.zeros((20, 1)), xs, np.ones((20, 1)))
    assert np.max(np.abs(dx[:, 0] - 1.5 * np.sin(-1.5 * xs[:, 0] + 0.25))) < TOL
