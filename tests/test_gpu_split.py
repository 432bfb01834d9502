"""The streaming training step runs the two halves of its batch on two streams
(the caller's and the library's side stream).  Checked here: equal bit for bit
to the separate forward, loss and backward calls (one stream, the whole batch)
for odd and even batches and every loss head (the MSE heads average over the
whole batch, not over a half), with shared parameters, and within the oracle's
bars on sampled rows; and ordered on the caller's stream, so that work queued
there after the call sees the whole step."""
import numpy as np
import pytest

from paper_2607_11985_amd import workloads as W
from tests.parity_util import check_step, note
from tests.test_gpu_parity import torch_mod  # noqa: F401

pytestmark = pytest.mark.gpu


def separate(torch, c, p, x, loss, yt):
    from paper_2607_11985_amd.api import loss_grad
    E, ws = c.forward(p, x, training=True)
    g = loss_grad(loss, E, yt)
    dp, dx = c.backward(p, x, g, ws)
    torch.cuda.synchronize()
    return [t.cpu().numpy() for t in (E, g, dp, dx)]


@pytest.mark.parametrize("n,B,loss,shared", [(14, 2, "mse_z0", False), (14, 3, "mse_meanz", False),
                                             (15, 5, "mean", True), (16, 4, "mse_meanz", False),
                                             (16, 7, "sum", False)])
def test_split_step_equals_separate_calls(torch_mod, n, B, loss, shared):
    torch = torch_mod
    from paper_2607_11985_amd.api import Circuit
    ops, P, F = W.random_circuit(n, 12 * n, seed=21000 + n + B)
    # every qubit starts with an entangler: no head, so that the step runs the
    # same passes as the separate calls (test_gpu_stream_head covers heads)
    ops = [W.Op("CZ", (q, (q + 1) % n)) for q in range(0, n, 2)] + ops
    params, inputs = W.random_inputs(B, P, F, seed=21100 + n + B)
    y = np.random.default_rng(21200 + B).uniform(-1, 1, size=B).astype(np.float32)
    c = Circuit(ops, n, P, F, path="stream", shared_params=shared)
    assert c.info()["step_head_rotations"] == 0
    note(f"split step n={n} B={B} loss={loss} shared={shared} tiles={c.info()['tile_qubits']}")
    p = torch.from_numpy(np.ascontiguousarray(params[0] if shared else params)).cuda()
    x = torch.from_numpy(inputs).cuda()
    yt = torch.from_numpy(y).cuda()
    E, dp, dx, g = c.train_step(p, x, loss, yt, want_cot=True)
    torch.cuda.synchronize()
    got = [t.cpu().numpy() for t in (E, g, dp, dx)]
    ref = separate(torch, c, p, x, loss, yt)
    for name, a, b in zip(("E", "g", "dparams", "dinputs"), got, ref):
        assert np.array_equal(a, b), f"{name} differs from the separate calls"
    if not shared:
        rows = [0, B - 1]  # one row from each half
        check_step(got[0][rows], got[1][rows], got[2][rows], got[3][rows], ops, n,
                   params[rows], inputs[rows], y[rows].astype(np.float64), loss, B)


def test_split_step_ordered_on_caller_stream(torch_mod):
    """On a non-default stream: a copy queued there right after the call (no
    synchronization in between) reads the finished gradients of both halves."""
    torch = torch_mod
    from paper_2607_11985_amd import _lib
    from paper_2607_11985_amd.api import Circuit
    w = W.make_config(5, batch=16)
    B, n = w.batch, w.n_qubits
    c = Circuit(w.ops, n, w.n_params, w.n_inputs)
    dev = torch.device("cuda", 0)
    note(f"{w.name} B={B}: step on a side stream of the caller, then a copy on it")
    p = torch.from_numpy(w.params).to(dev)
    x = torch.from_numpy(w.inputs).to(dev)
    E = torch.full((B, n), float("nan"), device=dev)
    dp = torch.full((B, w.n_params), float("nan"), device=dev)
    dx = torch.full((B, w.n_inputs), float("nan"), device=dev)
    nb = c.workspace_bytes(B, 2)
    ws = torch.empty(nb, dtype=torch.uint8, device=dev)
    s = torch.cuda.Stream(dev)
    s.wait_stream(torch.cuda.current_stream(dev))
    with torch.cuda.stream(s):
        _lib.vqc_train_step(c.handle, B, p.data_ptr(), x.data_ptr(), _lib.LOSS["sum"], None,
                            E.data_ptr(), None, dp.data_ptr(), dx.data_ptr(), ws.data_ptr(), nb,
                            s.cuda_stream)
        copies = [t.clone() for t in (E, dp, dx)]
    torch.cuda.synchronize()
    for a, b in zip(copies, (E, dp, dx)):
        a, b = a.cpu().numpy(), b.cpu().numpy()
        assert np.all(np.isfinite(a)), "a copy ran before the step finished"
        assert np.array_equal(a, b)


@pytest.mark.parametrize("n,B", [(14, 2), (15, 5), (16, 3)])
def test_split_forward_backward(torch_mod, n, B):
    """vqc_forward (inference and training workspaces), vqc_forward_ex with
    Psi_0 and probabilities, and vqc_backward, each on two streams, against the
    oracle on every row (B rows span both halves)."""
    torch = torch_mod
    import oracle
    from paper_2607_11985_amd.api import Circuit
    from tests.parity_util import check_E, check_grads
    ops, P, F = W.random_circuit(n, 10 * n, seed=21500 + n + B)
    params, inputs = W.random_inputs(B, P, F, seed=21600 + n + B)
    cot = W.random_cotangent(B, n, seed=21700 + n + B)
    psi0 = W.random_states(B, n, seed=21800 + n + B)
    c = Circuit(ops, n, P, F, path="stream")
    note(f"split forward/backward n={n} B={B}")
    p = torch.from_numpy(params).cuda()
    x = torch.from_numpy(inputs).cuda()
    Ei = c.forward(p, x, training=False)
    Et, ws = c.forward(p, x, training=True)
    dp, dx = c.backward(p, x, torch.from_numpy(cot).cuda(), ws)
    E0, pr, ws0 = c.forward_ex(p, x, torch.from_numpy(psi0).cuda(), probs=True, training=True)
    dp0, dx0 = c.backward(p, x, torch.from_numpy(cot).cuda(), ws0)
    torch.cuda.synchronize()
    assert np.array_equal(Ei.cpu().numpy(), Et.cpu().numpy())
    dpr, dxr, Er = oracle.vjp(ops, n, params, inputs, cot)
    check_E(Et.cpu().numpy(), Er)
    check_grads({"dp": dp.cpu().numpy(), "dx": dx.cpu().numpy()}, dpr, dxr, cot)
    dpr0, dxr0, Er0 = oracle.vjp(ops, n, params, inputs, cot, psi0=psi0)
    check_E(E0.cpu().numpy(), Er0)
    check_grads({"dp": dp0.cpu().numpy(), "dx": dx0.cpu().numpy()}, dpr0, dxr0, cot)
    _, st = oracle.forward(ops, n, params, inputs, want_state=True, psi0=psi0)
    assert float(np.max(np.abs(pr.cpu().numpy() - np.abs(st) ** 2))) <= 1e-5


def test_split_calls_ordered_on_caller_stream(torch_mod):
    """vqc_forward then vqc_backward on a non-default stream, and a copy queued
    right after them: the copy reads the finished gradients of both halves."""
    torch = torch_mod
    from paper_2607_11985_amd import _lib
    from paper_2607_11985_amd.api import Circuit
    w = W.make_config(5, batch=16)
    B, n = w.batch, w.n_qubits
    c = Circuit(w.ops, n, w.n_params, w.n_inputs)
    dev = torch.device("cuda", 0)
    note(f"{w.name} B={B}: forward and backward on a side stream of the caller, then a copy")
    p = torch.from_numpy(w.params).to(dev)
    x = torch.from_numpy(w.inputs).to(dev)
    g = torch.full((B, n), 0.25, device=dev)
    E = torch.full((B, n), float("nan"), device=dev)
    dp = torch.full((B, w.n_params), float("nan"), device=dev)
    dx = torch.full((B, w.n_inputs), float("nan"), device=dev)
    nb = c.workspace_bytes(B, 1)
    ws = torch.empty(nb, dtype=torch.uint8, device=dev)
    s = torch.cuda.Stream(dev)
    s.wait_stream(torch.cuda.current_stream(dev))
    with torch.cuda.stream(s):
        _lib.vqc_forward(c.handle, B, p.data_ptr(), x.data_ptr(), E.data_ptr(), ws.data_ptr(), nb,
                         s.cuda_stream)
        _lib.vqc_backward(c.handle, B, p.data_ptr(), x.data_ptr(), g.data_ptr(), ws.data_ptr(), nb,
                          dp.data_ptr(), dx.data_ptr(), s.cuda_stream)
        copies = [t.clone() for t in (E, dp, dx)]
    torch.cuda.synchronize()
    for a, b in zip(copies, (E, dp, dx)):
        a, b = a.cpu().numpy(), b.cpu().numpy()
        assert np.all(np.isfinite(a)), "a copy ran before the calls finished"
        assert np.array_equal(a, b)
