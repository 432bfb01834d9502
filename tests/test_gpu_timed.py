"""GPU parity of the kernels the benchmark times, against the double-precision oracle.

bench.py times one vqc_train_step per step (forward, loss head and adjoint; a
single generated kernel on the resident path, the streaming passes otherwise)
on the five workloads at their full batch.  These tests run exactly those calls
and compare every row (configs 1, 2) or sampled rows (configs 3-5) with the
oracle.  The resident path at 14 qubits (generated kernels), which the automatic
path choice does not take, is checked the same way.

The oracle never sees a GPU value: it evaluates the loss head on its own E, and
the gradient bar allows for the cotangent difference that follows from E's own
bar (tests/parity_util.py, check_step).
"""
import numpy as np
import pytest

import oracle
from paper_2607_11985_amd import workloads as W
from tests.parity_util import check_E, check_rows, check_step, note, oracle_cotangent
from tests.test_gpu_parity import torch_mod  # noqa: F401

pytestmark = pytest.mark.gpu


def run_step(torch, circ, w):
    p = torch.from_numpy(w.params).cuda()
    x = torch.from_numpy(w.inputs).cuda()
    y = torch.from_numpy(w.y).cuda() if w.y is not None else None
    E, dp, dx, g = circ.train_step(p, x, w.loss, y, want_cot=True)
    torch.cuda.synchronize()
    return tuple(t.cpu().numpy() for t in (E, g, dp, dx))


def y_of(w, rows):
    return None if w.y is None else w.y[rows].astype(np.float64)


@pytest.mark.parametrize("idx", [1, 2])
def test_train_step_config_full(torch_mod, idx):
    """The timed step of configs 1 and 2 (one generated kernel) on every row."""
    from paper_2607_11985_amd.api import Circuit
    w = W.make_config(idx)
    note(f"train step {w.name} full batch {w.batch}, every row")
    c = Circuit(w.ops, w.n_qubits, w.n_params, w.n_inputs)
    assert c.info()["path"] == 1
    E, g, dp, dx = run_step(torch_mod, c, w)
    rows = np.arange(w.batch)
    check_step(E, g, dp, dx, w.ops, w.n_qubits, w.params, w.inputs, y_of(w, rows), w.loss,
               w.batch)


@pytest.mark.parametrize("idx,rows", [(3, [0, 1, 2047, 4094, 4095]), (4, [0, 4097, 8191]),
                                      (5, [0, 131, 255])])
def test_train_step_config_sampled(torch_mod, idx, rows):
    """The timed step of configs 3-5 at full batch; the oracle checks sampled rows
    (rows are independent; the MSE heads average over the full batch)."""
    from paper_2607_11985_amd.api import Circuit
    w = W.make_config(idx)
    note(f"train step {w.name} full batch {w.batch}, oracle rows {rows}")
    c = Circuit(w.ops, w.n_qubits, w.n_params, w.n_inputs)
    E, g, dp, dx = run_step(torch_mod, c, w)
    assert np.all(np.isfinite(E)) and np.all(np.abs(E) <= 1 + 1e-5)
    assert np.all(np.isfinite(dp)) and np.all(np.isfinite(dx))
    check_step(E[rows], g[rows], dp[rows], dx[rows], w.ops, w.n_qubits, w.params[rows],
               w.inputs[rows], y_of(w, rows), w.loss, w.batch)


@pytest.mark.parametrize("loss", ["mean", "mse_meanz"])
def test_resident_jit_n14_random(torch_mod, loss):
    """The generated resident kernels at 14 qubits (the whole state on one
    workgroup): forward, adjoint and the one-launch step on a random circuit."""
    torch = torch_mod
    from paper_2607_11985_amd.api import Circuit
    n, B = 14, 3
    ops, P, F = W.random_circuit(n, 110, seed=17014)
    params, inputs = W.random_inputs(B, P, F, seed=17114)
    y = np.random.default_rng(17214).uniform(-1, 1, size=B).astype(np.float32)
    note(f"resident jit n=14 random circuit loss={loss}")
    c = Circuit(ops, n, P, F, path="resident", engine="jit")
    assert c.info()["path"] == 1 and c.info()["engine"] == 0
    p = torch.from_numpy(params).cuda()
    x = torch.from_numpy(inputs).cuda()
    Er = oracle.forward(ops, n, params, inputs)
    cot = oracle_cotangent(loss, Er, y.astype(np.float64), B)
    # forward + adjoint with the oracle's cotangent
    E, ws = c.forward(p, x, training=True)
    dp, dx = c.backward(p, x, torch.from_numpy(cot.astype(np.float32)).cuda(), ws)
    torch.cuda.synchronize()
    check_E(E.cpu().numpy(), Er)
    dpr, dxr, _ = oracle.vjp(ops, n, params, inputs, cot.astype(np.float32).astype(np.float64))
    check_rows(np.concatenate([dp.cpu().numpy(), dx.cpu().numpy()], axis=1),
               np.concatenate([dpr, dxr], axis=1), cot, "gradient (fwd + bwd)")
    # the one-launch step
    Es, dps, dxs, gs = c.train_step(p, x, loss, torch.from_numpy(y).cuda(), want_cot=True)
    torch.cuda.synchronize()
    check_step(Es.cpu().numpy(), gs.cpu().numpy(), dps.cpu().numpy(), dxs.cpu().numpy(), ops,
               n, params, inputs, y.astype(np.float64), loss, B)


def test_config4_resident_jit_sampled(torch_mod):
    """Config 4 (14 qubits, B = 8192) on the resident path with the generated
    kernels: the one-launch step, and forward + adjoint, on sampled rows."""
    torch = torch_mod
    from paper_2607_11985_amd.api import Circuit
    w = W.make_config(4)
    rows = [0, 5000, 8191]
    note(f"{w.name} resident jit, oracle rows {rows}")
    c = Circuit(w.ops, w.n_qubits, w.n_params, w.n_inputs, path="resident", engine="jit")
    assert c.info()["path"] == 1
    E, g, dp, dx = run_step(torch, c, w)
    check_step(E[rows], g[rows], dp[rows], dx[rows], w.ops, w.n_qubits, w.params[rows],
               w.inputs[rows], y_of(w, rows), w.loss, w.batch)
    # forward + adjoint with a seeded cotangent
    cot = W.random_cotangent(w.batch, w.n_qubits, seed=17400)
    p = torch.from_numpy(w.params).cuda()
    x = torch.from_numpy(w.inputs).cuda()
    E2, ws = c.forward(p, x, training=True)
    dp2, dx2 = c.backward(p, x, torch.from_numpy(cot).cuda(), ws)
    torch.cuda.synchronize()
    Er = oracle.forward(w.ops, w.n_qubits, w.params[rows], w.inputs[rows])
    check_E(E2.cpu().numpy()[rows], Er)
    dpr, dxr, _ = oracle.vjp(w.ops, w.n_qubits, w.params[rows], w.inputs[rows], cot[rows])
    c64 = cot[rows].astype(np.float64)
    check_rows(dp2.cpu().numpy()[rows], dpr, c64, "dparams")
    check_rows(dx2.cpu().numpy()[rows], dxr, c64, "dinputs")
