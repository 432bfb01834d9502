"""The streaming training step with a product head: its circuit is planned
without the heads' rotations, its first forward pass starts from the product
state after the heads, its last adjoint pass contracts lambda against the
heads' states per tile, and a last kernel sums those partials over the tiles
and walks each head back for its rotations' gradients.  Checked against the
oracle, which runs every gate, and against the separate forward / backward
calls (which run the heads as gates; both sides against the oracle, and
within half its E bar of each other): heads of every kind and length, heads
that end after other qubits' entanglers, constant and affine angles,
parameters shared between heads and later gates, shared parameters over the
batch, circuits that are heads only, general gates, odd batches (two halves on
two streams) and a batch of one, configs 4 and 5 on sampled rows.  Bars as in
test_gpu_parity."""
import numpy as np
import pytest

import oracle
from paper_2607_11985_amd import workloads as W
from tests.parity_util import G_FLOOR, G_REL, check_E, check_grad, check_grads, check_step, note
from tests.test_gpu_head import head_circuit
from tests.test_gpu_parity import torch_mod  # noqa: F401

pytestmark = pytest.mark.gpu


def run_and_check(torch, ops, n, P, F, B, loss, seed, shared=False, rows=None):
    from paper_2607_11985_amd.api import Circuit, loss_grad
    params, inputs = W.random_inputs(B, P, F, seed=seed)
    y = np.random.default_rng(seed + 7).uniform(-1, 1, size=B).astype(np.float32)
    c = Circuit(ops, n, P, F, path="stream", shared_params=shared)
    info = c.info()
    assert info["path"] == 2 and info["step_head_rotations"] > 0, info
    p = torch.from_numpy(np.ascontiguousarray(params[0] if shared else params)).cuda()
    x = torch.from_numpy(inputs).cuda()
    yt = torch.from_numpy(y).cuda()
    E, dp, dx, g = c.train_step(p, x, loss, yt, want_cot=True)
    torch.cuda.synchronize()
    E, dp, dx, g = (t.cpu().numpy() for t in (E, dp, dx, g))
    if not shared:
        r = list(range(B)) if rows is None else rows
        check_step(E[r], g[r], dp[r], dx[r], ops, n, params[r], inputs[r],
                   y[r].astype(np.float64), loss, B)
    # the separate calls run the head rotations as gates
    E2, ws = c.forward(p, x, training=True)
    g2 = loss_grad(loss, E2, yt)
    dp2, dx2 = c.backward(p, x, g2, ws)
    torch.cuda.synchronize()
    if not shared:
        r = list(range(B)) if rows is None else rows
        Er = oracle.forward(ops, n, params[r], inputs[r])
        note(f"E errors against the oracle: step {np.max(np.abs(E[r] - Er)):.2e}, separate calls "
             f"{np.max(np.abs(E2.cpu().numpy()[r] - Er)):.2e}")
        check_E(E2.cpu().numpy()[r], Er)
    # two plans rounded independently (the step's has no head rotations, and
    # its runs of RZs form differently): each is held to the oracle's bar
    # above, and they agree within half of it
    assert np.max(np.abs(E2.cpu().numpy() - E)) <= 5e-6
    assert np.max(np.abs(g2.cpu().numpy() - g)) <= 5e-6
    if shared:
        # one parameter vector: against the oracle's gradient summed over the batch
        rows_p = np.repeat(params[:1], B, axis=0)
        dpr, dxr, Er = oracle.vjp(ops, n, rows_p, inputs, g.astype(np.float64))
        check_E(E, Er)
        check_grad(dx, dxr, g, "dinputs")
        ref = dpr.sum(axis=0)
        for got in (dp, dp2.cpu().numpy()):
            err = float(np.max(np.abs(got - ref)))
            assert err <= G_REL * np.max(np.abs(ref)) + G_FLOOR * np.sum(np.abs(g)), err
    else:
        check_grads({"dp": dp2.cpu().numpy(), "dx": dx2.cpu().numpy()}, dp, dx, g)


@pytest.mark.parametrize("n,loss,B", [(14, "sum", 3), (14, "mse_meanz", 1), (15, "mean", 4),
                                      (15, "mse_z0", 5), (16, "mse_meanz", 2), (16, "sum", 3)])
def test_stream_heads_random(torch_mod, n, loss, B):
    ops, P, F = head_circuit(n, 25000 + n)
    note(f"streaming heads n={n} loss={loss} B={B} ops={len(ops)}")
    run_and_check(torch_mod, ops, n, P, F, B, loss, 25100 + n + B)


@pytest.mark.parametrize("n,trailing", [(14, False), (14, True), (16, True)])
def test_stream_heads_only(torch_mod, n, trailing):
    """Every rotation is in a head: the step's passes run no rotation at all."""
    ops, P, F = head_circuit(n, 25500 + n, body=False, late=False, trailing=trailing)
    note(f"streaming heads only n={n} trailing={trailing} ops={len(ops)}")
    run_and_check(torch_mod, ops, n, P, F, 3, "mse_meanz", 25600 + n)


@pytest.mark.parametrize("n", [14, 16])
def test_stream_heads_general_gates(torch_mod, n):
    """General gates lowered to rotations: the heads are the lowered rotations
    before a qubit's first entangler, whatever gate they came from."""
    ops, P, F = W.random_circuit(n, 10 * n, seed=25800 + n, kinds=W.GENERAL_KINDS,
                                 p_affine=0.3)
    note(f"streaming heads general gates n={n} ops={len(ops)}")
    run_and_check(torch_mod, ops, n, P, F, 3, "mse_z0", 25900 + n)


def test_stream_heads_shared_params(torch_mod):
    """One parameter vector for the batch: the heads' gradients join the
    per-sample rows before the fixed-order sum."""
    ops, P, F = head_circuit(15, 26000)
    note("streaming heads, shared parameters, n=15")
    run_and_check(torch_mod, ops, 15, P, F, 5, "mean", 26100, shared=True)


@pytest.mark.parametrize("idx", [4, 5])
def test_stream_heads_configs(torch_mod, idx):
    """Configs 4 and 5 (their encoding and first layer are heads) on a small
    batch, sampled rows against the oracle."""
    w = W.make_config(idx, batch=6)
    note(f"{w.name} streaming heads B=6")
    run_and_check(torch_mod, w.ops, w.n_qubits, w.n_params, w.n_inputs, 6, w.loss, 26200 + idx,
                  rows=[0, 5])


def test_stream_no_step_plan_without_heads(torch_mod):
    """A circuit whose every qubit starts with an entangler has no head: the
    step runs the circuit's own passes (bit for bit the separate calls)."""
    torch = torch_mod
    from paper_2607_11985_amd.api import Circuit, loss_grad
    n = 14
    ops, P, F = W.random_circuit(n, 8 * n, seed=26300)
    ops = [W.Op("CZ", (q, q + 1)) for q in range(0, n - 1, 2)] + ops
    c = Circuit(ops, n, P, F, path="stream")
    assert c.info()["step_head_rotations"] == 0
    params, inputs = W.random_inputs(3, P, F, seed=26301)
    p, x = torch.from_numpy(params).cuda(), torch.from_numpy(inputs).cuda()
    E, dp, dx = c.train_step(p, x, "sum")
    E2, ws = c.forward(p, x, training=True)
    dp2, dx2 = c.backward(p, x, loss_grad("sum", E2, None), ws)
    torch.cuda.synchronize()
    for a, b in ((E, E2), (dp, dp2), (dx, dx2)):
        assert np.array_equal(a.cpu().numpy(), b.cpu().numpy())
