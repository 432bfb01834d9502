"""Runs of RZs applied as one diagonal (generated kernels): the forward
multiplies each amplitude by the run's product once, the adjoint takes every
gradient of the run from Im(conj(lambda) psi) and multiplies psi and lambda
by the inverse product once.  Circuits built to reach every form of a run:
RZs on register and on thread / tile bits, two RZs of one qubit in a row (a
product factor per bit), RZs on bits under a swap frame (CNOTs with a high
control and a low target before the layer), one parameter read by several
RZs of a run (its partials summed in one pending slot), affine angles, and
constant RZs between them (which stay gate by gate).  Against the oracle:
forward, adjoint and training step, on every kernel geometry (4 amplitudes
per thread with lane gates, 16 resident, 16 streaming with product heads).
Bars as in test_gpu_parity."""
import numpy as np
import pytest

import oracle
from paper_2607_11985_amd import workloads as W
from tests.parity_util import check_E, check_grads, check_step, note
from tests.test_gpu_parity import torch_mod  # noqa: F401

pytestmark = pytest.mark.gpu


def diag_run_circuit(n, seed, layers=4):
    """RY encoding, then per layer: CNOTs from the upper half onto the lower
    half, a layer of RZs (some qubits take two in a row, a few a constant),
    a layer of RY / RX, another layer of RZs (two in a row on the last four
    qubits), CZs on every other layer and a CNOT ring.  Angles: own parameters, affine ones, inputs, and four shared
    parameters that many RZs read."""
    rng = np.random.default_rng(seed)
    P, F = 4 + 5 * n * layers, n
    ops = [W.Op("RY", (q,), (("input", q),)) for q in range(n)]
    nxt = [4]

    def angle():
        u = rng.random()
        if u < 0.15:
            return ("param", int(rng.integers(4)))
        if u < 0.22:
            return ("input", int(rng.integers(F)))
        p = nxt[0]
        nxt[0] += 1
        if u < 0.4:
            mul = float(np.float32(rng.choice([-1.0, 1.0]) * rng.uniform(0.5, 2.0)))
            return ("param", p, mul, float(np.float32(rng.uniform(-2.0, 2.0))))
        return ("param", p)

    for layer in range(layers):
        for q in range(n // 2):
            ops.append(W.Op("CNOT", (n - 1 - q, q)))
        for q in range(n):
            ops.append(W.Op("RZ", (q,), (angle(),)))
            if rng.random() < 0.3:
                ops.append(W.Op("RZ", (q,), (angle(),)))
            if rng.random() < 0.1:
                ops.append(W.Op("RZ", (q,), (("const", float(np.float32(rng.uniform(-3, 3)))),)))
        for q in range(n):
            ops.append(W.Op("RX" if (q + layer) % 3 == 0 else "RY", (q,), (angle(),)))
        for q in range(n):
            ops.append(W.Op("RZ", (q,), (angle(),)))
            if q >= n - 4:  # the qubits the RX / RY layer left on register bits: two RZs
                ops.append(W.Op("RZ", (q,), (angle(),)))
        if layer % 2:
            ops += [W.Op("CZ", (q, q + 1)) for q in range(0, n - 1, 2)]
        ops += [W.Op("CNOT", (q, (q + 1) % n)) for q in range(n)]
    assert nxt[0] <= P
    return ops, P, F


@pytest.mark.parametrize("n,path", [(6, "auto"), (8, "auto"), (11, "auto"), (12, "auto"),
                                    (14, "stream"), (16, "auto")])
def test_diagonal_runs(torch_mod, n, path):
    torch = torch_mod
    from paper_2607_11985_amd.api import Circuit
    ops, P, F = diag_run_circuit(n, 29000 + n)
    B = 3
    params, inputs = W.random_inputs(B, P, F, seed=29100 + n)
    cot = W.random_cotangent(B, n, seed=29200 + n)
    c = Circuit(ops, n, P, F, path=path)
    note(f"diagonal runs n={n} path={c.info()['path']} ops={len(ops)}")
    tp, tx = torch.from_numpy(params).cuda(), torch.from_numpy(inputs).cuda()
    E, ws = c.forward(tp, tx, training=True)
    dp, dx = c.backward(tp, tx, torch.from_numpy(cot).cuda(), ws)
    torch.cuda.synchronize()
    dpr, dxr, Er = oracle.vjp(ops, n, params, inputs, cot)
    check_E(E.cpu().numpy(), Er)
    check_grads({"dp": dp.cpu().numpy(), "dx": dx.cpu().numpy()}, dpr, dxr, cot)
    y = np.random.default_rng(29300 + n).uniform(-1, 1, size=B).astype(np.float32)
    E, dp, dx, g = c.train_step(tp, tx, "mse_meanz", torch.from_numpy(y).cuda(), want_cot=True)
    torch.cuda.synchronize()
    check_step(E.cpu().numpy(), g.cpu().numpy(), dp.cpu().numpy(), dx.cpu().numpy(), ops, n,
               params, inputs, y.astype(np.float64), "mse_meanz", B)
