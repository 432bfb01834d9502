"""The swap frame of the generated kernels: CNOTs whose control sits on a
thread / tile bit and whose target sits on a register bit only record, per
thread, that the target bit's registers are swapped; later RY / RZ on that bit
run with the angle (and the adjoint's gradient) negated, register CNOTs spread
the frame, and LDS exchanges and pass stores fold it into their addresses,
CZs and the epilogues resolve it.  Circuits dense in CNOTs (every control /
target placement), interleaved with rotations of every kind and CZs, against
the oracle: forward, adjoint, training step (resident and streaming, both
with product heads), Psi_0 and probabilities.  Bars as in test_gpu_parity."""
import numpy as np
import pytest

import oracle
from paper_2607_11985_amd import workloads as W
from tests.parity_util import check_E, check_grads, check_step, note
from tests.test_gpu_parity import torch_mod  # noqa: F401

pytestmark = pytest.mark.gpu
P_TOL = 1e-5


def cnot_dense_circuit(n, seed, n_gates):
    """Runs of CNOTs (random control / target pairs, chains, fans out of one
    control) between single rotations of every kind and a few CZs."""
    rng = np.random.default_rng(seed)
    P, F = 3 * n, n
    ops = [W.Op("RY", (q,), (("input", q),)) for q in range(n)]
    while len(ops) < n_gates:
        u = rng.random()
        if u < 0.45:
            run = int(rng.integers(1, 6))
            if rng.random() < 0.3:  # a fan: one control, several targets
                c = int(rng.integers(n))
                for tq in rng.choice([q for q in range(n) if q != c], size=min(run, n - 1),
                                     replace=False):
                    ops.append(W.Op("CNOT", (c, int(tq))))
            else:
                for _ in range(run):
                    a, b = (int(v) for v in rng.choice(n, size=2, replace=False))
                    ops.append(W.Op("CNOT", (a, b)))
        elif u < 0.9:
            kind = ("RX", "RY", "RZ")[int(rng.integers(3))]
            ops.append(W.Op(kind, (int(rng.integers(n)),), (("param", int(rng.integers(P))),)))
        else:
            a, b = (int(v) for v in rng.choice(n, size=2, replace=False))
            ops.append(W.Op("CZ", (a, b)))
    return ops, P, F


@pytest.mark.parametrize("n,path", [(6, "auto"), (9, "auto"), (11, "auto"), (12, "auto"),
                                    (13, "auto"), (14, "stream"), (15, "auto"), (16, "auto")])
def test_cnot_dense_circuits(torch_mod, n, path):
    torch = torch_mod
    from paper_2607_11985_amd.api import Circuit
    ops, P, F = cnot_dense_circuit(n, 28000 + n, 16 * n)
    B = 3
    params, inputs = W.random_inputs(B, P, F, seed=28100 + n)
    cot = W.random_cotangent(B, n, seed=28200 + n)
    psi0 = W.random_states(B, n, seed=28300 + n)
    c = Circuit(ops, n, P, F, path=path)
    note(f"CNOT-dense n={n} path={path} ops={len(ops)} info={c.info()['path']}")
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
    y = np.random.default_rng(28400 + n).uniform(-1, 1, size=B).astype(np.float32)
    E, dp, dx, g = c.train_step(tp, tx, "mse_z0", torch.from_numpy(y).cuda(), want_cot=True)
    torch.cuda.synchronize()
    check_step(E.cpu().numpy(), g.cpu().numpy(), dp.cpu().numpy(), dx.cpu().numpy(), ops, n,
               params, inputs, y.astype(np.float64), "mse_z0", B)
