"""GPU parity of circuits that end in entanglers: CNOTs and CZs with no rotation
after them on their qubits are not run but folded into the measurement (<Z_j>
becomes the expectation of a Z-string before them, the adjoint starts from that
string's lambda, the probabilities are read through the CNOTs' basis
permutation).  Against the oracle, which applies every gate: E, both gradient
arrays, probabilities, from |0...0> and from a Haar-random Psi_0, resident and
streaming, both engines, and a circuit made of entanglers only.  Bars as in
test_gpu_parity and test_gpu_psi0_probs.
"""
import numpy as np
import pytest

import oracle
from paper_2607_11985_amd import workloads as W
from tests.parity_util import check_E, check_grads, check_step, note
from tests.test_gpu_parity import torch_mod  # noqa: F401

pytestmark = pytest.mark.gpu
P_TOL = 1e-5


def tail_circuit(n, seed, n_rot=None):
    """Random rotations (and some entanglers) followed by a dense entangler
    network whose CNOTs chain through every qubit."""
    rng = np.random.default_rng(seed)
    body, P, F = W.random_circuit(n, n_rot if n_rot is not None else 10 * n, seed=seed)
    tail = []
    for _ in range(3 * n):
        a, b = (int(v) for v in rng.choice(n, size=2, replace=False))
        tail.append(W.Op("CNOT" if rng.random() < 0.7 else "CZ", (a, b)))
    for i in range(n - 1):
        tail.append(W.Op("CNOT", (i, i + 1)))
    return body + tail, P, F


@pytest.mark.parametrize("n,path,engine", [(2, "auto", "jit"), (5, "auto", "jit"),
                                           (9, "auto", "jit"), (13, "auto", "jit"),
                                           (15, "auto", "jit"), (7, "auto", "interp"),
                                           (15, "auto", "interp")])
def test_trailing_entanglers(torch_mod, n, path, engine):
    torch = torch_mod
    from paper_2607_11985_amd.api import Circuit
    ops, P, F = tail_circuit(n, 19000 + n)
    B = 3
    params, inputs = W.random_inputs(B, P, F, seed=19100 + n)
    cot = W.random_cotangent(B, n, seed=19200 + n)
    psi0 = W.random_states(B, n, seed=19300 + n)
    note(f"trailing entanglers n={n} path={path} engine={engine}")
    c = Circuit(ops, n, P, F, path=path, engine=engine)
    tp, tx = torch.from_numpy(params).cuda(), torch.from_numpy(inputs).cuda()
    for s0 in (None, psi0):
        ts = torch.from_numpy(s0).cuda() if s0 is not None else None
        E, pr, ws = c.forward_ex(tp, tx, ts, probs=True, training=True)
        dp, dx = c.backward(tp, tx, torch.from_numpy(cot).cuda(), ws)
        torch.cuda.synchronize()
        dpr, dxr, Er = oracle.vjp(ops, n, params, inputs, cot, psi0=s0)
        check_E(E.cpu().numpy(), Er)
        check_grads({"dp": dp.cpu().numpy(), "dx": dx.cpu().numpy()}, dpr, dxr, cot)
        _, st = oracle.forward(ops, n, params, inputs, want_state=True, psi0=s0)
        err = float(np.max(np.abs(pr.cpu().numpy() - np.abs(st) ** 2)))
        assert err <= P_TOL, f"probabilities max abs err {err:.3e}"


@pytest.mark.parametrize("n", [4, 14])
def test_entanglers_only(torch_mod, n):
    """Nothing but entanglers: no gate runs at all; E and the probabilities come
    from Psi_0 through the folded network."""
    torch = torch_mod
    from paper_2607_11985_amd.api import Circuit
    ops, P, F = tail_circuit(n, 19500 + n, n_rot=0)
    ops = [o for o in ops if o.kind in ("CNOT", "CZ")]
    B = 2
    psi0 = W.random_states(B, n, seed=19600 + n)
    note(f"entanglers only n={n}")
    c = Circuit(ops, n, 0, 0)
    E, pr = c.forward_ex(None, torch.zeros((B, 0), device="cuda"),
                         torch.from_numpy(psi0).cuda(), probs=True)
    torch.cuda.synchronize()
    Er, st = oracle.forward(ops, n, np.zeros((B, 1)), np.zeros((B, 1)), want_state=True,
                            psi0=psi0)
    check_E(E.cpu().numpy(), Er)
    assert float(np.max(np.abs(pr.cpu().numpy() - np.abs(st) ** 2))) <= P_TOL


def diagonal_tail_circuit(n, seed):
    """Random rotations, then a stretch rich in diagonal gates (RZ, CZ) mixed
    with CNOTs and a few RX / RY: the diagonal gates that commute with every
    later gate are dropped, the others stay."""
    rng = np.random.default_rng(seed)
    body, P, F = W.random_circuit(n, 8 * n, seed=seed, n_params=12 * n, n_inputs=n)
    tail = []
    for _ in range(6 * n):
        u = rng.random()
        q = int(rng.integers(n))
        if u < 0.4:
            src = "param" if rng.random() < 0.7 else "input"
            idx = int(rng.integers(P if src == "param" else F))
            tail.append(W.Op("RZ", (q,), ((src, idx),)))
        elif u < 0.65 and n > 1:
            a, b = (int(v) for v in rng.choice(n, size=2, replace=False))
            tail.append(W.Op("CZ", (a, b)))
        elif u < 0.9 and n > 1:
            a, b = (int(v) for v in rng.choice(n, size=2, replace=False))
            tail.append(W.Op("CNOT", (a, b)))
        else:
            tail.append(W.Op("RX" if rng.random() < 0.5 else "RY", (q,),
                             (("param", int(rng.integers(P))),)))
    return body + tail, P, F


@pytest.mark.parametrize("n,path,engine", [(3, "auto", "jit"), (9, "auto", "jit"),
                                           (13, "auto", "jit"), (15, "auto", "jit"),
                                           (6, "auto", "interp"), (14, "auto", "interp")])
def test_trailing_diagonal_gates(torch_mod, n, path, engine):
    """E, both gradient arrays (the dropped gates' slots included: zero up to
    the other occurrences of their parameters) and probabilities against the
    oracle, from |0...0> and from a Haar-random Psi_0, and the training step."""
    torch = torch_mod
    from paper_2607_11985_amd.api import Circuit
    ops, P, F = diagonal_tail_circuit(n, 19700 + n)
    B = 3
    params, inputs = W.random_inputs(B, P, F, seed=19800 + n)
    cot = W.random_cotangent(B, n, seed=19900 + n)
    psi0 = W.random_states(B, n, seed=20000 + n)
    note(f"trailing diagonal gates n={n} path={path} engine={engine}")
    c = Circuit(ops, n, P, F, path=path, engine=engine)
    tp, tx = torch.from_numpy(params).cuda(), torch.from_numpy(inputs).cuda()
    for s0 in (None, psi0):
        ts = torch.from_numpy(s0).cuda() if s0 is not None else None
        E, pr, ws = c.forward_ex(tp, tx, ts, probs=True, training=True)
        dp, dx = c.backward(tp, tx, torch.from_numpy(cot).cuda(), ws)
        torch.cuda.synchronize()
        dpr, dxr, Er = oracle.vjp(ops, n, params, inputs, cot, psi0=s0)
        check_E(E.cpu().numpy(), Er)
        check_grads({"dp": dp.cpu().numpy(), "dx": dx.cpu().numpy()}, dpr, dxr, cot)
        _, st = oracle.forward(ops, n, params, inputs, want_state=True, psi0=s0)
        err = float(np.max(np.abs(pr.cpu().numpy() - np.abs(st) ** 2)))
        assert err <= P_TOL, f"probabilities max abs err {err:.3e}"
    y = np.random.default_rng(20100 + n).uniform(-1, 1, size=B).astype(np.float32)
    E, dp, dx, g = c.train_step(tp, tx, "mse_meanz", torch.from_numpy(y).cuda(), want_cot=True)
    torch.cuda.synchronize()
    check_step(E.cpu().numpy(), g.cpu().numpy(), dp.cpu().numpy(), dx.cpu().numpy(), ops, n,
               params, inputs, y.astype(np.float64), "mse_meanz", B)
