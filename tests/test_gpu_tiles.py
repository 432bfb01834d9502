"""GPU parity of the streaming path with 13- and 12-qubit tiles (two and four
workgroups per CU) against the oracle: forward, adjoint, the training step,
Psi_0 and probabilities.  Bars as in test_gpu_parity / test_gpu_psi0_probs."""
import numpy as np
import pytest

import oracle
from paper_2607_11985_amd import workloads as W
from tests.parity_util import check_step
from tests.test_gpu_parity import check_E, check_grads, note, torch_mod  # noqa: F401

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("n,B,kinds,tile", [(14, 3, W.KINDS, 13), (15, 2, W.GENERAL_KINDS, 13),
                                             (16, 2, W.KINDS, 13), (17, 1, W.KINDS, 13),
                                             (16, 2, W.GENERAL_KINDS, 14), (14, 3, W.KINDS, 12),
                                             (16, 2, W.GENERAL_KINDS, 12)])
def test_tile13_parity(torch_mod, n, B, kinds, tile):
    torch = torch_mod
    from paper_2607_11985_amd.api import Circuit
    ops, P, F = W.random_circuit(n, 100, seed=15000 + n, kinds=kinds, p_affine=0.3)
    params, x = W.random_inputs(B, P, F, seed=15100 + n)
    cot = W.random_cotangent(B, n, seed=15200 + n)
    note(f"{tile}-qubit tiles n={n} B={B}")
    c = Circuit(ops, n, P, F, path="stream", tile_qubits=tile)
    info = c.info()
    assert info["tile_qubits"] == tile and info["threads"] == 1 << (tile - 4)
    tp, tx = torch.from_numpy(params).cuda(), torch.from_numpy(x).cuda()
    s0 = W.random_states(B, n, seed=15300 + n)
    E, pr, ws = c.forward_ex(tp, tx, torch.from_numpy(s0).cuda(), probs=True, training=True)
    dp, dx = c.backward(tp, tx, torch.from_numpy(cot).cuda(), ws)
    torch.cuda.synchronize()
    dpr, dxr, Er = oracle.vjp(ops, n, params, x, cot, psi0=s0)
    check_E(E.cpu().numpy(), Er)
    check_grads({"dp": dp.cpu().numpy(), "dx": dx.cpu().numpy()}, dpr, dxr, cot)
    _, st = oracle.forward(ops, n, params, x, want_state=True, psi0=s0)
    assert np.max(np.abs(pr.cpu().numpy() - np.abs(st) ** 2)) <= 1e-5


def test_tile13_train_step_config5_sampled(torch_mod):
    """The 16-qubit workload at full batch with 13-qubit tiles; sampled rows."""
    torch = torch_mod
    from paper_2607_11985_amd.api import Circuit
    w = W.make_config(5)
    rows = [0, w.batch // 2, w.batch - 1]
    note(f"config {w.name} with 13-qubit tiles, rows {rows}")
    c = Circuit(w.ops, w.n_qubits, w.n_params, w.n_inputs, tile_qubits=13)
    E, dp, dx, g = c.train_step(torch.from_numpy(w.params).cuda(),
                                torch.from_numpy(w.inputs).cuda(), w.loss, None, want_cot=True)
    torch.cuda.synchronize()
    E, dp, dx, g = (t.cpu().numpy() for t in (E, dp, dx, g))
    check_step(E[rows], g[rows], dp[rows], dx[rows], w.ops, w.n_qubits, w.params[rows],
               w.inputs[rows], None, w.loss, w.batch)


@pytest.mark.parametrize("n,tile,loss", [(14, 12, "mse_meanz"), (16, 12, "mean"),
                                         (15, 13, "mse_z0")])
def test_32_amplitude_streaming_kernels(torch_mod, n, tile, loss):
    """reg_bits = 5: the streaming passes hold 32 amplitudes per thread (one DPP
    gradient sum per rotation instead of the batched flush): forward with
    Psi_0 and probabilities, adjoint, and the training step (its own plan with
    a product head)."""
    torch = torch_mod
    from paper_2607_11985_amd.api import Circuit
    ops, P, F = W.random_circuit(n, 12 * n, seed=15600 + n, kinds=W.GENERAL_KINDS, p_affine=0.3)
    B = 3
    params, x = W.random_inputs(B, P, F, seed=15700 + n)
    cot = W.random_cotangent(B, n, seed=15800 + n)
    note(f"32-amplitude streaming kernels n={n} tiles={tile}")
    c = Circuit(ops, n, P, F, path="stream", tile_qubits=tile, reg_bits=5)
    info = c.info()
    assert info["tile_qubits"] == tile and info["threads"] == 1 << (tile - 5)
    tp, tx = torch.from_numpy(params).cuda(), torch.from_numpy(x).cuda()
    s0 = W.random_states(B, n, seed=15900 + n)
    E, pr, ws = c.forward_ex(tp, tx, torch.from_numpy(s0).cuda(), probs=True, training=True)
    dp, dx = c.backward(tp, tx, torch.from_numpy(cot).cuda(), ws)
    torch.cuda.synchronize()
    dpr, dxr, Er = oracle.vjp(ops, n, params, x, cot, psi0=s0)
    check_E(E.cpu().numpy(), Er)
    check_grads({"dp": dp.cpu().numpy(), "dx": dx.cpu().numpy()}, dpr, dxr, cot)
    _, st = oracle.forward(ops, n, params, x, want_state=True, psi0=s0)
    assert np.max(np.abs(pr.cpu().numpy() - np.abs(st) ** 2)) <= 1e-5
    y = np.random.default_rng(16000 + n).uniform(-1, 1, size=B).astype(np.float32)
    E, dp, dx, g = c.train_step(tp, tx, loss, torch.from_numpy(y).cuda(), want_cot=True)
    torch.cuda.synchronize()
    check_step(E.cpu().numpy(), g.cpu().numpy(), dp.cpu().numpy(), dx.cpu().numpy(), ops, n,
               params, x, y.astype(np.float64), loss, B)
