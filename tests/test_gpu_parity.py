"""GPU parity: the HIP path (through the C ABI) against the double-precision oracle.

Bars (tests/parity_util.py): E within 1e-5 absolute; gradients per sample row
within 1e-4 of the row's max-norm (+ a floor of 1e-6 sum |cot|), over the whole
row and, with at least four parameters and four inputs, over each array.
Every input and cotangent is seeded and synthetic and reaches both sides as the
same float32 values; nothing the oracle sees comes from the GPU.
"""
import numpy as np
import pytest

import oracle
from paper_2607_11985_amd import workloads as W
from tests.parity_util import (E_TOL, G_FLOOR, G_REL, check_E, check_grad,  # noqa: F401
                               check_grads, check_rows, check_step, fd_bound, gpu_run, note,
                               oracle_central_differences)

pytestmark = pytest.mark.gpu

@pytest.fixture(scope="module")
def torch_mod():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    from paper_2607_11985_amd import _lib
    _lib.load()  # fails loudly if the HIP library is not built
    return torch


def samples_per_wg(n):
    """Samples per workgroup of the resident kernels at the default width."""
    nq = max(n, 4)
    R = 2 if nq <= 8 else 3 if nq <= 10 else 4
    T = 1 << (nq - R)
    return max(1, 64 // T)


@pytest.mark.parametrize("n", list(range(1, 15)))
def test_random_circuit_parity(torch_mod, n):
    S = samples_per_wg(n)
    B = 2 * S + 1 if S > 1 else 3
    n_ops = 40 + 6 * n
    ops, P, F = W.random_circuit(n, n_ops, seed=1000 + n)
    params, inputs = W.random_inputs(B, P, F, seed=2000 + n)
    cot = W.random_cotangent(B, n, seed=3000 + n)
    note(f"random circuit n={n} B={B} ops={n_ops}")
    r = gpu_run(torch_mod, ops, n, P, F, params, inputs, cot)
    dpr, dxr, Er = oracle.vjp(ops, n, params, inputs, cot)
    check_E(r["E"], Er)
    check_grads(r, dpr, dxr, cot)


@pytest.mark.parametrize("n", [5, 9, 13])
def test_entangler_heavy_parity(torch_mod, n):
    """Dense CNOT/CZ networks between rotations: exercises every exchange layout."""
    ops, P, F = W.random_circuit(n, 150, seed=77 + n, kinds=("RY", "CNOT", "CZ", "RX", "CNOT"))
    B = 5
    params, inputs = W.random_inputs(B, P, F, seed=88 + n)
    cot = W.random_cotangent(B, n, seed=99 + n)
    note(f"entangler-heavy n={n}")
    r = gpu_run(torch_mod, ops, n, P, F, params, inputs, cot)
    dpr, dxr, Er = oracle.vjp(ops, n, params, inputs, cot)
    check_E(r["E"], Er)
    check_grads(r, dpr, dxr, cot)


@pytest.mark.parametrize("n,path,B", [(14, "stream", 3), (15, "auto", 3), (16, "auto", 2),
                                      (17, "auto", 1)])
def test_streaming_parity(torch_mod, n, path, B):
    """HBM-streamed tiles of 14 qubits (n = 14 forced onto the streaming path is a
    cross-path check of the same circuit family the resident path runs)."""
    ops, P, F = W.random_circuit(n, 120, seed=4000 + n)
    params, inputs = W.random_inputs(B, P, F, seed=5000 + n)
    cot = W.random_cotangent(B, n, seed=6000 + n)
    note(f"streaming n={n} path={path} B={B}")
    r = gpu_run(torch_mod, ops, n, P, F, params, inputs, cot, path=path)
    info = r["circ"].info()
    assert info["path"] == 2 and (n == 14 or info["fwd_passes"] > 1)
    dpr, dxr, Er = oracle.vjp(ops, n, params, inputs, cot)
    check_E(r["E"], Er)
    check_grads(r, dpr, dxr, cot)


@pytest.mark.parametrize("n,path,reg_bits", [(3, "auto", 0), (8, "auto", 2), (9, "auto", 3),
                                             (13, "auto", 0), (15, "auto", 0)])
def test_interpreter_engine_parity(torch_mod, n, path, reg_bits):
    """The precompiled schedule interpreter against the oracle, and bit-level
    agreement of E with the generated kernels is not required (different
    instruction order), only both within the bar."""
    ops, P, F = W.random_circuit(n, 40 + 6 * n, seed=7000 + n)
    B = 5
    params, inputs = W.random_inputs(B, P, F, seed=7100 + n)
    cot = W.random_cotangent(B, n, seed=7200 + n)
    note(f"interpreter n={n} path={path} reg_bits={reg_bits}")
    dpr, dxr, Er = oracle.vjp(ops, n, params, inputs, cot)
    for engine in ("interp", "jit"):
        r = gpu_run(torch_mod, ops, n, P, F, params, inputs, cot, path=path, engine=engine,
                    reg_bits=reg_bits)
        assert r["circ"].info()["engine"] == (1 if engine == "interp" else 0)
        check_E(r["E"], Er)
        check_grads(r, dpr, dxr, cot)


@pytest.mark.parametrize("idx", [1, 2])
def test_config_full_batch(torch_mod, idx):
    w = W.make_config(idx)
    note(f"config {w.name} full batch {w.batch}")
    Er = oracle.forward(w.ops, w.n_qubits, w.params, w.inputs)
    cot = oracle.loss_cotangent(w.loss, Er, w.y).astype(np.float32)
    r = gpu_run(torch_mod, w.ops, w.n_qubits, w.n_params, w.n_inputs, w.params, w.inputs, cot)
    dpr, dxr, _ = oracle.vjp(w.ops, w.n_qubits, w.params, w.inputs, cot)
    check_E(r["E"], Er)
    check_grads(r, dpr, dxr, cot)


@pytest.mark.parametrize("idx,rows", [(3, [0, 1, 2047, 4095]), (4, [0, 4097, 8191]),
                                      (5, [0, 255])])
def test_config_full_batch_sampled(torch_mod, idx, rows):
    """Full batch on the GPU in the benchmark's launch configuration; the oracle
    checks sampled rows (rows are independent).  The MSE cotangent of a sampled
    row comes from the oracle's own E; other rows get a seeded random cotangent."""
    w = W.make_config(idx)
    note(f"config {w.name} full batch {w.batch}, oracle rows {rows}")
    Er = oracle.forward(w.ops, w.n_qubits, w.params[rows], w.inputs[rows])
    cot = W.random_cotangent(w.batch, w.n_qubits, seed=5 + idx)
    g_rows = np.zeros((len(rows), w.n_qubits))
    for i, b in enumerate(rows):
        if w.loss == "mse_z0":
            g_rows[i, 0] = 2.0 * (Er[i, 0] - w.y[b]) / w.batch
        elif w.loss == "mse_meanz":
            g_rows[i, :] = 2.0 * (Er[i].mean() - w.y[b]) / (w.n_qubits * w.batch)
        else:
            g_rows[i] = oracle.loss_cotangent(w.loss, Er[i:i + 1])[0]
    cot[rows] = g_rows.astype(np.float32)
    r = gpu_run(torch_mod, w.ops, w.n_qubits, w.n_params, w.n_inputs, w.params, w.inputs, cot)
    assert np.all(np.isfinite(r["E"])) and np.all(np.abs(r["E"]) <= 1 + 1e-5)
    dpr, dxr, _ = oracle.vjp(w.ops, w.n_qubits, w.params[rows], w.inputs[rows], cot[rows])
    check_E(r["E"][rows], Er)
    check_grads({"dp": r["dp"][rows], "dx": r["dx"][rows]}, dpr, dxr, cot[rows])


@pytest.mark.parametrize("n,loss,path,engine", [
    (1, "sum", "auto", "jit"), (3, "mean", "auto", "jit"), (6, "mse_z0", "auto", "jit"),
    (8, "mse_meanz", "auto", "jit"), (9, "mse_meanz", "auto", "jit"), (12, "mse_z0", "auto", "jit"),
    (13, "mse_meanz", "auto", "jit"), (14, "mean", "stream", "jit"),
    (15, "mse_meanz", "auto", "jit"), (7, "mse_meanz", "auto", "interp"),
    (14, "mse_z0", "resident", "interp")])
def test_train_step_parity(torch_mod, n, loss, path, engine):
    """vqc_train_step (forward, loss head and adjoint in one call; one launch on
    the resident path) against the oracle, and against the three separate calls."""
    torch = torch_mod
    from paper_2607_11985_amd.api import Circuit, loss_grad
    S = samples_per_wg(n)
    B = 2 * S + 1 if S > 1 else 5
    ops, P, F = W.random_circuit(n, 40 + 5 * n, seed=8000 + n)
    params, inputs = W.random_inputs(B, P, F, seed=8100 + n)
    y = np.random.default_rng(8200 + n).uniform(-1, 1, size=B).astype(np.float32)
    note(f"train step n={n} loss={loss} path={path} engine={engine} B={B}")
    c = Circuit(ops, n, P, F, path=path, engine=engine)
    p = torch.from_numpy(params).cuda()
    x = torch.from_numpy(inputs).cuda()
    yt = torch.from_numpy(y).cuda()
    E, dp, dx, g = c.train_step(p, x, loss, yt, want_cot=True)
    torch.cuda.synchronize()
    E, dp, dx, g = (t.cpu().numpy() for t in (E, dp, dx, g))
    check_step(E, g, dp, dx, ops, n, params, inputs, y.astype(np.float64), loss, B)
    # the separate calls give the same results up to rounding (the step builds
    # the state after the heads as a product instead of running their gates)
    E2, ws = c.forward(p, x, training=True)
    g2 = loss_grad(loss, E2, yt)
    dp2, dx2 = c.backward(p, x, g2, ws)
    torch.cuda.synchronize()
    assert np.max(np.abs(E2.cpu().numpy() - E)) <= 2e-6
    assert np.max(np.abs(g2.cpu().numpy() - g)) <= 2e-6
    check_grads({"dp": dp2.cpu().numpy(), "dx": dx2.cpu().numpy()}, dp, dx, g)


@pytest.mark.parametrize("n,path,engine", [(6, "auto", "jit"), (9, "auto", "jit"),
                                           (12, "auto", "jit"), (15, "auto", "jit"),
                                           (9, "auto", "interp"), (15, "auto", "interp")])
def test_shared_params_parity(torch_mod, n, path, engine):
    """One parameter vector for the whole batch (Algorithm 1's shared theta):
    dparams is the sum of the samples' gradients; the inputs stay per sample."""
    torch = torch_mod
    from paper_2607_11985_amd.api import Circuit
    ops, P, F = W.random_circuit(n, 40 + 5 * n, seed=9000 + n)
    B = 2 * samples_per_wg(n) + 3
    theta, inputs = W.random_inputs(B, P, F, seed=9100 + n)
    theta = theta[0]
    params = np.repeat(theta[None, :], B, axis=0)  # the oracle sees the shared row per sample
    cot = W.random_cotangent(B, n, seed=9200 + n)
    note(f"shared params n={n} path={path} engine={engine} B={B}")
    c = Circuit(ops, n, P, F, path=path, engine=engine, shared_params=True)
    assert c.info()["shared_params"] == 1
    p = torch.from_numpy(np.ascontiguousarray(theta)).cuda()
    x = torch.from_numpy(inputs).cuda()
    g = torch.from_numpy(cot.astype(np.float32)).cuda()
    E, ws = c.forward(p, x, training=True)
    dp, dx = c.backward(p, x, g, ws)
    Es, dps, dxs = c.train_step(p, x, "sum")
    torch.cuda.synchronize()
    dpr, dxr, Er = oracle.vjp(ops, n, params, inputs, cot)
    check_E(E.cpu().numpy(), Er)
    check_grad(dx.cpu().numpy(), dxr, cot, "dinputs")
    dp_sum = dpr.sum(axis=0)
    err = np.max(np.abs(dp.cpu().numpy() - dp_sum))
    assert err <= G_REL * np.max(np.abs(dp_sum)) + G_FLOOR * np.sum(np.abs(cot)), err
    # the training step with the summed objective: the cotangent is all ones
    ones = np.ones((B, n))
    dpr1, dxr1, _ = oracle.vjp(ops, n, params, inputs, ones)
    check_E(Es.cpu().numpy(), Er)
    check_grad(dxs.cpu().numpy(), dxr1, ones, "dinputs (step)")
    ref1 = dpr1.sum(axis=0)
    err = np.max(np.abs(dps.cpu().numpy() - ref1))
    assert err <= G_REL * np.max(np.abs(ref1)) + G_FLOOR * np.sum(np.abs(ones)), err


@pytest.mark.parametrize("n,engine,shared", [(4, "jit", False), (9, "jit", False),
                                             (12, "jit", False), (7, "interp", False),
                                             (10, "jit", True), (15, "jit", False),
                                             (14, "interp", True)])
def test_fd_backward(torch_mod, n, engine, shared):
    """Central differences through the shifted-batch forward, against the same
    differences at the same h on the oracle side (every slot moved in the
    params / inputs arrays).  The truncation error is common to both, so the
    bound is the float32 rounding of E over h (fd_bound)."""
    torch = torch_mod
    from paper_2607_11985_amd.api import Circuit
    ops, P, F = W.random_circuit(n, 30 + 4 * n, seed=9300 + n)
    B = 3
    params, inputs = W.random_inputs(B, P, F, seed=9400 + n)
    if shared:
        params = np.repeat(params[:1], B, axis=0)
    cot = W.random_cotangent(B, n, seed=9500 + n)
    note(f"fd backward n={n} engine={engine} shared={shared}")
    c = Circuit(ops, n, P, F, engine=engine, shared_params=shared)
    h = 0.25
    p = torch.from_numpy(np.ascontiguousarray(params[0] if shared else params)).cuda()
    dp, dx = c.fd_backward(p, torch.from_numpy(inputs).cuda(),
                           torch.from_numpy(cot.astype(np.float32)).cuda(), h=h)
    torch.cuda.synchronize()
    dpr, dxr = oracle_central_differences(ops, n, params, inputs, cot, h)
    bound = fd_bound(ops, params, inputs, cot, h)
    if shared:
        dpr = dpr.sum(axis=0, keepdims=True)
        bp = bound.sum(keepdims=True)
    else:
        bp = bound
    assert np.all(np.abs(dp.cpu().numpy().reshape(dpr.shape) - dpr) <= bp)
    assert np.all(np.abs(dx.cpu().numpy() - dxr) <= bound)


def test_fd_backward_streaming_chunks(torch_mod):
    """The 16-qubit workload's structure at B = 64: the shifted copies of all
    400 slots (51 GiB of states in two buffers) run in chunks of slots; sampled rows against
    the oracle's differences at the same h."""
    torch = torch_mod
    from paper_2607_11985_amd.api import Circuit
    w = W.make_config(5, batch=64)
    rows = [0, 63]
    note(f"fd backward streaming chunks {w.name} B={w.batch}")
    c = Circuit(w.ops, w.n_qubits, w.n_params, w.n_inputs)
    cot = W.random_cotangent(w.batch, w.n_qubits, seed=9600)
    h = 0.25
    dp, dx = c.fd_backward(torch.from_numpy(w.params).cuda(), torch.from_numpy(w.inputs).cuda(),
                           torch.from_numpy(cot).cuda(), h=h)
    torch.cuda.synchronize()
    dpr, dxr = oracle_central_differences(w.ops, w.n_qubits, w.params[rows], w.inputs[rows],
                                          cot[rows], h)
    bound = fd_bound(w.ops, w.params[rows], w.inputs[rows], cot[rows], h)
    assert np.all(np.abs(dp.cpu().numpy()[rows] - dpr) <= bound)
    assert np.all(np.abs(dx.cpu().numpy()[rows] - dxr) <= bound)


def test_loss_grad_kernel(torch_mod):
    from paper_2607_11985_amd.api import loss_grad
    rng = np.random.default_rng(4)
    for B, n in ((1, 3), (300, 14), (8192, 14), (37, 1)):
        E = rng.uniform(-1, 1, size=(B, n)).astype(np.float32)
        y = rng.uniform(-1, 1, size=B).astype(np.float32)
        for kind in ("sum", "mean", "mse_z0", "mse_meanz"):
            g = loss_grad(kind, torch_mod.from_numpy(E).cuda(), torch_mod.from_numpy(y).cuda())
            ref = oracle.loss_cotangent(kind, E.astype(np.float64), y.astype(np.float64))
            err = np.max(np.abs(g.cpu().numpy() - ref))
            assert err <= 1e-6 * max(1.0, np.max(np.abs(ref))), (kind, B, n, err)


def test_edge_cases(torch_mod):
    torch = torch_mod
    from paper_2607_11985_amd.api import Circuit
    # empty circuit: E = 1, gradients are zero
    c = Circuit([], 5, 2, 3)
    p = torch.zeros((4, 2), device="cuda")
    x = torch.zeros((4, 3), device="cuda")
    E, ws = c.forward(p, x, training=True)
    dp, dx = c.backward(p, x, torch.ones((4, 5), device="cuda"), ws)
    assert torch.all(E == 1) and torch.all(dp == 0) and torch.all(dx == 0)
    # batch 0 is a no-op
    E0 = c.forward(torch.zeros((0, 2), device="cuda"), torch.zeros((0, 3), device="cuda"))
    assert E0.shape == (0, 5)
    # constants only (P = F = 0)
    ops = [W.Op("RY", (0,), (("const", 0.7),)), W.Op("CNOT", (0, 2))]
    c = Circuit(ops, 3, 0, 0)
    E = c.forward(None, torch.zeros((2, 0), device="cuda"))
    Er = oracle.forward(ops, 3, np.zeros((2, 1)), np.zeros((2, 1)))
    check_E(E.cpu().numpy(), Er)


def test_backward_twice_and_determinism(torch_mod):
    torch = torch_mod
    w = W.make_config(2)
    cot = W.random_cotangent(w.batch, w.n_qubits, seed=12)
    a = gpu_run(torch, w.ops, w.n_qubits, w.n_params, w.n_inputs, w.params, w.inputs, cot)
    b = gpu_run(torch, w.ops, w.n_qubits, w.n_params, w.n_inputs, w.params, w.inputs, cot)
    assert np.array_equal(a["E"], b["E"])
    assert np.array_equal(a["dp"], b["dp"]) and np.array_equal(a["dx"], b["dx"])
    from paper_2607_11985_amd.api import Circuit
    c = Circuit(w.ops, w.n_qubits, w.n_params, w.n_inputs)
    p = torch.from_numpy(w.params).cuda()
    x = torch.from_numpy(w.inputs).cuda()
    g = torch.from_numpy(cot).cuda()
    E, ws = c.forward(p, x, training=True)
    d1 = c.backward(p, x, g, ws)
    d2 = c.backward(p, x, g, ws)
    assert torch.equal(d1[0], d2[0]) and torch.equal(d1[1], d2[1])


def test_autograd_function(torch_mod):
    torch = torch_mod
    from paper_2607_11985_amd.api import Circuit, VQCFunction
    w = W.make_config(1)
    c = Circuit(w.ops, w.n_qubits, w.n_params, w.n_inputs)
    p = torch.from_numpy(w.params).cuda().requires_grad_(True)
    x = torch.from_numpy(w.inputs).cuda().requires_grad_(True)
    E = VQCFunction.apply(c, p, x)
    E.sum().backward()
    dpr, dxr, Er = oracle.vjp(w.ops, 4, w.params, w.inputs, np.ones((w.batch, 4)))
    check_E(E.detach().cpu().numpy(), Er)
    check_grads({"dp": p.grad.cpu().numpy(), "dx": x.grad.cpu().numpy()}, dpr, dxr,
                np.ones((w.batch, 4)))


@pytest.mark.parametrize("n,reg_bits,loss", [(9, 2, "mse_meanz"), (11, 2, "mean"), (8, 3, "mse_z0")])
def test_four_amplitude_kernels_spanning_waves(torch_mod, n, reg_bits, loss):
    """Four amplitudes per thread with a sample over several waves (lane-bit
    gates, lane swaps, exchanges across waves, the tangent form's factor
    tables), and eight per thread at n = 8: forward, adjoint and the one-launch
    training step against the oracle."""
    torch = torch_mod
    from paper_2607_11985_amd.api import Circuit
    ops, P, F = W.random_circuit(n, 12 * n, seed=16000 + n)
    B = 5
    params, inputs = W.random_inputs(B, P, F, seed=16100 + n)
    cot = W.random_cotangent(B, n, seed=16200 + n)
    note(f"4-amplitude kernels n={n} reg_bits={reg_bits}")
    r = gpu_run(torch, ops, n, P, F, params, inputs, cot, reg_bits=reg_bits)
    dpr, dxr, Er = oracle.vjp(ops, n, params, inputs, cot)
    check_E(r["E"], Er)
    check_grads(r, dpr, dxr, cot)
    y = np.random.default_rng(16300 + n).uniform(-1, 1, size=B).astype(np.float32)
    c = Circuit(ops, n, P, F, reg_bits=reg_bits)
    E, dp, dx, g = c.train_step(torch.from_numpy(params).cuda(), torch.from_numpy(inputs).cuda(),
                                loss, torch.from_numpy(y).cuda(), want_cot=True)
    torch.cuda.synchronize()
    E, dp, dx, g = (t.cpu().numpy() for t in (E, dp, dx, g))
    check_step(E, g, dp, dx, ops, n, params, inputs, y.astype(np.float64), loss, B)
