"""GPU parity of the general static gate set (the OpenQASM standard gates the
compile phase lowers, Sec. 3 and Algorithm 1) and of affine angles
(mul * value + add), against the double-precision oracle, which applies every
gate as its own matrix (no lowering).  Bars as in test_gpu_parity.
"""
import numpy as np
import pytest

import oracle
from paper_2607_11985_amd import workloads as W
from tests.parity_util import check_step, fd_bound, oracle_central_differences
from tests.test_gpu_parity import (check_E, check_grad, check_grads, gpu_run, note,  # noqa: F401
                                   samples_per_wg, torch_mod)

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("n", [1, 2, 3, 4, 6, 8, 9, 11, 13])
def test_general_gates_resident(torch_mod, n):
    S = samples_per_wg(n)
    B = 2 * S + 1 if S > 1 else 3
    ops, P, F = W.random_circuit(n, 30 + 5 * n, seed=11000 + n, kinds=W.GENERAL_KINDS,
                                 p_affine=0.4)
    params, inputs = W.random_inputs(B, P, F, seed=11100 + n)
    cot = W.random_cotangent(B, n, seed=11200 + n)
    note(f"general gates n={n} B={B} ops={len(ops)}")
    r = gpu_run(torch_mod, ops, n, P, F, params, inputs, cot)
    dpr, dxr, Er = oracle.vjp(ops, n, params, inputs, cot)
    check_E(r["E"], Er)
    check_grads(r, dpr, dxr, cot)


@pytest.mark.parametrize("n,path", [(14, "stream"), (15, "auto"), (16, "auto")])
def test_general_gates_streaming(torch_mod, n, path):
    B = 2
    ops, P, F = W.random_circuit(n, 70, seed=11300 + n, kinds=W.GENERAL_KINDS, p_affine=0.4)
    params, inputs = W.random_inputs(B, P, F, seed=11400 + n)
    cot = W.random_cotangent(B, n, seed=11500 + n)
    note(f"general gates streaming n={n} path={path}")
    r = gpu_run(torch_mod, ops, n, P, F, params, inputs, cot, path=path)
    assert r["circ"].info()["path"] == 2
    dpr, dxr, Er = oracle.vjp(ops, n, params, inputs, cot)
    check_E(r["E"], Er)
    check_grads(r, dpr, dxr, cot)


@pytest.mark.parametrize("kind", list(W.GENERAL_KINDS))
def test_each_gate_between_rotations(torch_mod, kind):
    """One gate of each kind, on random wires, between layers of parametrized
    rotations (so that its action on a generic state is visible), with its own
    angles read from params (scaled and offset) or inputs."""
    n = 5
    rng = np.random.default_rng(sum(map(ord, kind)))
    nw, na = W.GATE_SHAPES[kind]
    wires = tuple(int(v) for v in rng.choice(n, size=nw, replace=False))
    layer = lambda base: [W.Op("RY", (q,), (("param", base + q),)) for q in range(n)] + \
        [W.Op("RZ", (q,), (("param", base + n + q),)) for q in range(n)]
    ang = tuple(("param", 4 * n + s, float(np.float32(1.5 - s)), float(np.float32(0.25 * s)))
                if s % 2 == 0 else ("input", s) for s in range(na))
    ops = layer(0) + [W.Op(kind, wires, ang)] + layer(2 * n)
    P, F = 4 * n + 3, 3
    B = 6
    params, inputs = W.random_inputs(B, P, F, seed=11600)
    cot = W.random_cotangent(B, n, seed=11700)
    note(f"gate {kind} on wires {wires}")
    dpr, dxr, Er = oracle.vjp(ops, n, params, inputs, cot)
    for engine in ("jit", "interp"):
        r = gpu_run(torch_mod, ops, n, P, F, params, inputs, cot, engine=engine)
        check_E(r["E"], Er)
        check_grads(r, dpr, dxr, cot)


@pytest.mark.parametrize("n,path", [(5, "auto"), (12, "auto"), (14, "stream")])
def test_general_gates_interpreter(torch_mod, n, path):
    ops, P, F = W.random_circuit(n, 60, seed=11800 + n, kinds=W.GENERAL_KINDS, p_affine=0.5)
    B = 3
    params, inputs = W.random_inputs(B, P, F, seed=11900 + n)
    cot = W.random_cotangent(B, n, seed=12000 + n)
    note(f"general gates interpreter n={n} path={path}")
    r = gpu_run(torch_mod, ops, n, P, F, params, inputs, cot, path=path, engine="interp")
    dpr, dxr, Er = oracle.vjp(ops, n, params, inputs, cot)
    check_E(r["E"], Er)
    check_grads(r, dpr, dxr, cot)


@pytest.mark.parametrize("n,loss,path", [(6, "mse_z0", "auto"), (10, "mean", "auto"),
                                         (15, "mse_meanz", "auto")])
def test_general_gates_train_step(torch_mod, n, loss, path):
    torch = torch_mod
    from paper_2607_11985_amd.api import Circuit
    ops, P, F = W.random_circuit(n, 50, seed=12100 + n, kinds=W.GENERAL_KINDS, p_affine=0.4)
    B = 5
    params, inputs = W.random_inputs(B, P, F, seed=12200 + n)
    y = np.random.default_rng(12300 + n).uniform(-1, 1, size=B).astype(np.float32)
    note(f"general gates train step n={n} loss={loss}")
    c = Circuit(ops, n, P, F, path=path)
    E, dp, dx, g = c.train_step(torch.from_numpy(params).cuda(), torch.from_numpy(inputs).cuda(),
                                loss, torch.from_numpy(y).cuda(), want_cot=True)
    torch.cuda.synchronize()
    E, dp, dx, g = (t.cpu().numpy() for t in (E, dp, dx, g))
    check_step(E, g, dp, dx, ops, n, params, inputs, y.astype(np.float64), loss, B)


def test_general_gates_shared_params(torch_mod):
    torch = torch_mod
    from paper_2607_11985_amd.api import Circuit
    n, B = 7, 9
    ops, P, F = W.random_circuit(n, 50, seed=12400, kinds=W.GENERAL_KINDS, p_affine=0.5)
    theta, inputs = W.random_inputs(B, P, F, seed=12500)
    theta = theta[0]
    params = np.repeat(theta[None, :], B, axis=0)
    cot = W.random_cotangent(B, n, seed=12600)
    note("general gates shared params")
    c = Circuit(ops, n, P, F, shared_params=True)
    p = torch.from_numpy(np.ascontiguousarray(theta)).cuda()
    x = torch.from_numpy(inputs).cuda()
    E, ws = c.forward(p, x, training=True)
    dp, dx = c.backward(p, x, torch.from_numpy(cot).cuda(), ws)
    torch.cuda.synchronize()
    dpr, dxr, Er = oracle.vjp(ops, n, params, inputs, cot)
    check_E(E.cpu().numpy(), Er)
    check_grad(dx.cpu().numpy(), dxr, cot, "dinputs")
    ref = dpr.sum(axis=0)
    err = np.max(np.abs(dp.cpu().numpy() - ref))
    assert err <= 1e-4 * np.max(np.abs(ref)) + 1e-6 * np.sum(np.abs(cot)), err


def test_affine_fd_backward(torch_mod):
    """Central differences move the source value (then mul * value + add): the
    same differences at the same h on the oracle side, bound by fd_bound."""
    torch = torch_mod
    from paper_2607_11985_amd.api import Circuit
    n, B = 6, 3
    ops, P, F = W.random_circuit(n, 40, seed=12700, kinds=W.GENERAL_KINDS, p_affine=1.0,
                                 p_const=0.0)
    params, inputs = W.random_inputs(B, P, F, seed=12800)
    cot = W.random_cotangent(B, n, seed=12900)
    note("affine fd backward")
    c = Circuit(ops, n, P, F)
    h = 0.25
    dp, dx = c.fd_backward(torch.from_numpy(params).cuda(), torch.from_numpy(inputs).cuda(),
                           torch.from_numpy(cot).cuda(), h=h)
    torch.cuda.synchronize()
    dpr, dxr = oracle_central_differences(ops, n, params, inputs, cot, h)
    bound = fd_bound(ops, params, inputs, cot, h)
    assert np.all(np.abs(dp.cpu().numpy() - dpr) <= bound)
    assert np.all(np.abs(dx.cpu().numpy() - dxr) <= bound)


@pytest.mark.parametrize("n", [5, 8, 10])
def test_layers_sharing_one_angle(torch_mod, n):
    """Layers whose rotations all read one parameter (scaled and offset), next
    to layers reading one parameter or input per qubit: the generated kernels
    encode such occurrence runs as compares instead of a table."""
    layers = []
    for l in range(3):
        mul, add = float(np.float32(1.5 - l)), float(np.float32(0.25 * l))
        layers += [W.Op("RX", (q,), (("param", l, mul, add),)) for q in range(n)]
        layers += [W.Op("RY", (q,), (("param", 3 + l * n + q),)) for q in range(n)]
        layers += [W.Op("CNOT", (q, (q + 1) % n)) for q in range(n)]
        layers += [W.Op("RZ", (q,), (("input", q, -2.0, 0.0),)) for q in range(n)]
    P, F = 3 + 3 * n, n
    B = 7
    params, inputs = W.random_inputs(B, P, F, seed=12900 + n)
    cot = W.random_cotangent(B, n, seed=13000 + n)
    note(f"shared-angle layers n={n}")
    r = gpu_run(torch_mod, layers, n, P, F, params, inputs, cot)
    dpr, dxr, Er = oracle.vjp(layers, n, params, inputs, cot)
    check_E(r["E"], Er)
    check_grads(r, dpr, dxr, cot)


@pytest.mark.parametrize("n", [6, 8, 9])
def test_cnot_on_every_qubit_pair(torch_mod, n):
    """CNOTs between every ordered pair of qubits, between rotation layers, so
    that controls and targets meet on register bits, lane bits (DPP moves, the
    masked moves of controls on lane bits 2-5) and wave bits."""
    ops = []
    k = 0
    for c in range(n):
        ops += [W.Op("RY", (q,), (("param", k + q),)) for q in range(n)]
        k += n
        for t in range(n):
            if t != c:
                ops.append(W.Op("CNOT", (c, t)))
        ops += [W.Op("RX", (q,), (("input", q),)) for q in range(n)]
    P, F = k, n
    B = 3
    params, inputs = W.random_inputs(B, P, F, seed=13100 + n)
    cot = W.random_cotangent(B, n, seed=13200 + n)
    note(f"cnot pairs n={n}")
    dpr, dxr, Er = oracle.vjp(ops, n, params, inputs, cot)
    for reg_bits in (0, 2):
        r = gpu_run(torch_mod, ops, n, P, F, params, inputs, cot, reg_bits=reg_bits)
        check_E(r["E"], Er)
        check_grads(r, dpr, dxr, cot)


@pytest.mark.parametrize("n,path", [(8, "auto"), (14, "stream")])
def test_many_constant_gates_keep_the_norm(torch_mod, n, path):
    """Hundreds of fixed gates (H, S, T, SX, Toffolis), each followed by its
    inverse, on a basis state: every <Z_q> is exactly +-1, and the GPU's is
    +-(the state's norm squared).  The float (cos, sin) pairs of the gates'
    angles are picked so that their norm errors cancel over the circuit; the
    nearest floats of these angles all shrink the norm, by about 5e-8 per
    rotation, which would put <Z> 1e-5 off after a few hundred."""
    torch = torch_mod
    rng = np.random.default_rng(27000 + n)
    ops = [W.Op("RY", (q,), (("param", q),)) for q in range(n)]
    inverse = {"H": "H", "S": "SDG", "SDG": "S", "T": "TDG", "TDG": "T", "SX": "SXDG",
               "SXDG": "SX"}
    kinds = sorted(inverse)
    for _ in range(30 * n):
        if rng.random() < 0.1:
            a, b, c = (int(v) for v in rng.choice(n, size=3, replace=False))
            ops += [W.Op("CCX", (a, b, c)), W.Op("CCX", (a, b, c))]
        else:
            k, q = kinds[int(rng.integers(len(kinds)))], int(rng.integers(n))
            ops += [W.Op(k, (q,)), W.Op(inverse[k], (q,))]
    P, F, B = n, 1, 2
    params = np.zeros((B, P), dtype=np.float32)  # |0...0> and |1...1>
    params[1] = np.float32(np.pi)
    inputs = np.zeros((B, F), dtype=np.float32)
    note(f"constant gates n={n} path={path} ops={len(ops)}")
    r = gpu_run(torch, ops, n, P, F, params, inputs, None, path=path)
    Er = oracle.forward(ops, n, params, inputs)
    assert np.allclose(np.abs(Er), 1.0, atol=1e-9)
    check_E(r["E"], Er)
