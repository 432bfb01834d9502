"""The generated resident training step builds the state after every qubit's
head (its rotations before the first entangler on it) as a product state, and
takes those rotations' gradients from lambda contracted against the other
qubits' states.  Checked against the oracle, which runs every gate, and against
the separate forward / backward calls (which run the heads as gates): heads of
every kind and length (none on some qubits), constant and affine angles,
parameters shared between heads and later gates, heads that end after other
qubits' entanglers, circuits that are heads only (with and without trailing
entanglers), and general gates whose lowering starts with rotations.  Bars as
in test_gpu_parity."""
import numpy as np
import pytest

from paper_2607_11985_amd import workloads as W
from tests.parity_util import check_grads, check_step, note
from tests.test_gpu_parity import torch_mod  # noqa: F401

pytestmark = pytest.mark.gpu
LOSSES = ["sum", "mean", "mse_z0", "mse_meanz"]


def head_ops(n, rng, P, F, first):
    """Random heads for the qubits in `first`: 0 to 4 rotations each, angles
    from parameters (shared pool), affine inputs and constants."""
    heads = {q: [] for q in first}
    for q in first:
        for _ in range(int(rng.integers(0, 5))):
            kind = ("RX", "RY", "RZ")[int(rng.integers(3))]
            u = rng.random()
            if u < 0.15:
                ang = ("const", float(rng.uniform(-3.2, 3.2)))
            elif u < 0.45:
                mul = float(np.float32(rng.choice([-1, 1]) * rng.uniform(0.25, 2.0)))
                ang = ("input", int(rng.integers(F)), mul, float(np.float32(rng.uniform(-1, 1))))
            else:
                ang = ("param", int(rng.integers(P)))
            heads[q].append(W.Op(kind, (q,), (ang,)))
    # interleave the qubits' heads, each in its own order
    ops = []
    left = {q: list(v) for q, v in heads.items() if v}
    while left:
        q = list(left)[int(rng.integers(len(left)))]
        ops.append(left[q].pop(0))
        if not left[q]:
            del left[q]
    return ops


def head_circuit(n, seed, body=True, late=True, trailing=False):
    rng = np.random.default_rng(seed)
    P, F = 3 * n, n
    early = list(range(n)) if not late else [q for q in range(n) if q % 3]
    ops = head_ops(n, rng, P, F, early)
    if late:
        # entanglers among the early qubits, then the other qubits' heads
        for i in range(len(early) - 1):
            ops.append(W.Op("CNOT", (early[i], early[i + 1])))
        ops += head_ops(n, rng, P, F, [q for q in range(n) if q not in early])
    if body:
        b, _, _ = W.random_circuit(n, 8 * n, seed=seed + 1, n_params=P, n_inputs=F,
                                   p_affine=0.3)
        ops += b
    if trailing:
        for q in range(n - 1):
            ops.append(W.Op("CNOT", (q, q + 1)))
        ops.append(W.Op("CZ", (0, n - 1)))
    return ops, P, F


def run_and_check(torch, ops, n, P, F, B, loss, seed):
    from paper_2607_11985_amd.api import Circuit, loss_grad
    params, inputs = W.random_inputs(B, P, F, seed=seed)
    y = np.random.default_rng(seed + 7).uniform(-1, 1, size=B).astype(np.float32)
    c = Circuit(ops, n, P, F, path="resident", engine="jit")
    assert c.info()["path"] == 1
    p = torch.from_numpy(params).cuda()
    x = torch.from_numpy(inputs).cuda()
    yt = torch.from_numpy(y).cuda()
    E, dp, dx, g = c.train_step(p, x, loss, yt, want_cot=True)
    torch.cuda.synchronize()
    E, dp, dx, g = (t.cpu().numpy() for t in (E, dp, dx, g))
    check_step(E, g, dp, dx, ops, n, params, inputs, y.astype(np.float64), loss, B)
    # the separate calls run the head rotations as gates
    E2, ws = c.forward(p, x, training=True)
    g2 = loss_grad(loss, E2, yt)
    dp2, dx2 = c.backward(p, x, g2, ws)
    torch.cuda.synchronize()
    assert np.max(np.abs(E2.cpu().numpy() - E)) <= 2e-6
    check_grads({"dp": dp2.cpu().numpy(), "dx": dx2.cpu().numpy()}, dp, dx, g)


@pytest.mark.parametrize("n,loss", [(8, "sum"), (8, "mse_meanz"), (9, "mean"), (10, "mse_z0"),
                                    (11, "mse_meanz"), (12, "sum"), (13, "mean"),
                                    (14, "mse_z0")])
def test_heads_random(torch_mod, n, loss):
    ops, P, F = head_circuit(n, 23000 + n)
    note(f"heads n={n} loss={loss} ops={len(ops)}")
    run_and_check(torch_mod, ops, n, P, F, 3, loss, 23100 + n)


@pytest.mark.parametrize("n,trailing", [(8, False), (8, True), (12, False), (12, True)])
def test_heads_only(torch_mod, n, trailing):
    """Every rotation is in a head: the sweeps run no rotation at all."""
    ops, P, F = head_circuit(n, 23500 + n, body=False, late=False, trailing=trailing)
    note(f"heads only n={n} trailing={trailing} ops={len(ops)}")
    run_and_check(torch_mod, ops, n, P, F, 4, "mse_meanz", 23600 + n)


@pytest.mark.parametrize("n", [8, 10, 12])
def test_heads_general_gates(torch_mod, n):
    """General gates (U3, Rot, phase, controlled rotations ...) lowered to
    rotations: the heads are the lowered rotations before a qubit's first
    entangler, whatever gate they came from."""
    ops, P, F = W.random_circuit(n, 10 * n, seed=23800 + n, kinds=W.GENERAL_KINDS,
                                 p_affine=0.3)
    note(f"heads general gates n={n} ops={len(ops)}")
    run_and_check(torch_mod, ops, n, P, F, 3, "mse_z0", 23900 + n)


@pytest.mark.parametrize("idx", [2, 3])
def test_heads_configs_all_losses(torch_mod, idx):
    """Configs 2 and 3 (their embedding and first layer are heads) with every
    loss head, sampled rows of a small batch."""
    w = W.make_config(idx, batch=5)
    for loss in LOSSES:
        note(f"{w.name} heads loss={loss}")
        run_and_check(torch_mod, w.ops, w.n_qubits, w.n_params, w.n_inputs, 5, loss,
                      24000 + idx)
