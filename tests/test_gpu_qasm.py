"""GPU parity of circuits given as OpenQASM text (vqc_compile_qasm): the text
goes to the library's front end, the equivalent gate list straight to the
oracle.  Bars as in test_gpu_parity; probabilities as in test_gpu_psi0_probs."""
import math

import numpy as np
import pytest

import oracle
from paper_2607_11985_amd import workloads as W
from tests.qasm_writer import to_qasm
from tests.test_gpu_parity import check_E, check_grads, note, torch_mod  # noqa: F401

pytestmark = pytest.mark.gpu
Op = W.Op


def run_qasm(torch, src, inputs, params, x, cot, path="auto", psi0=None, probs=False):
    from paper_2607_11985_amd.api import Circuit
    c = Circuit.from_qasm(src, inputs=inputs, path=path)
    p = torch.from_numpy(np.ascontiguousarray(params)).cuda()
    xt = torch.from_numpy(np.ascontiguousarray(x)).cuda()
    s0 = torch.from_numpy(np.ascontiguousarray(psi0)).cuda() if psi0 is not None else None
    E, pr, ws = c.forward_ex(p, xt, s0, probs=probs, training=True)
    dp, dx = c.backward(p, xt, torch.from_numpy(cot).cuda(), ws)
    torch.cuda.synchronize()
    return {"circ": c, "E": E.cpu().numpy(), "probs": pr.cpu().numpy() if probs else None,
            "dp": dp.cpu().numpy(), "dx": dx.cpu().numpy()}


@pytest.mark.parametrize("n,version,path", [(4, 2, "auto"), (10, 3, "auto"), (15, 3, "auto")])
def test_written_programs(torch_mod, n, version, path):
    ops, P, F = W.random_circuit(n, 60, seed=14000 + n, kinds=W.GENERAL_KINDS, p_affine=0.5)
    B = 4
    params, x = W.random_inputs(B, P, F, seed=14100 + n)
    cot = W.random_cotangent(B, n, seed=14200 + n)
    note(f"qasm program n={n} version={version}")
    r = run_qasm(torch_mod, to_qasm(ops, n, P, F, version=version), ("x",), params, x, cot, path)
    assert (r["circ"].n, r["circ"].P, r["circ"].F) == (n, P, F)
    dpr, dxr, Er = oracle.vjp(ops, n, params, x, cot)
    check_E(r["E"], Er)
    check_grads(r, dpr, dxr, cot)


QAOA = """OPENQASM 3.0;
include "stdgates.inc";
// MaxCut QAOA on a ring of {n} vertices, {p} layers
qubit[{n}] q;
bit[{n}] c;
input array[float[32], {p}] gamma;
input array[float[32], {p}] beta;
gate cost(g) a, b {{ rzz(-g) a, b; }}
h q;
{layers}
c = measure q;
"""


def qaoa_program(n, p):
    layers = []
    for l in range(p):
        for i in range(n):
            layers.append(f"cost(gamma[{l}]) q[{i}], q[{(i + 1) % n}];")
        layers.append(f"rx(2 * beta[{l}]) q;")
    return QAOA.format(n=n, p=p, layers="\n".join(layers))


def qaoa_ops(n, p):
    """The same circuit as a gate list: params [gamma_0..gamma_{p-1}, beta_0..]."""
    ops = [Op("H", (q,)) for q in range(n)]
    for l in range(p):
        for i in range(n):
            ops.append(Op("RZZ", (i, (i + 1) % n), (("param", l, -1.0, 0.0),)))
        ops += [Op("RX", (q,), (("param", p + l, 2.0, 0.0),)) for q in range(n)]
    return ops


@pytest.mark.parametrize("n,p", [(6, 2), (12, 3), (16, 2)])
def test_qaoa_program(torch_mod, n, p):
    """The paper's workloads include QAOA; here a MaxCut ansatz on a ring with a
    user gate, broadcasting and terminal measurement, read as probabilities."""
    B = 3
    rng = np.random.default_rng(14300 + n)
    params = rng.uniform(0, math.pi, size=(B, 2 * p)).astype(np.float32)
    x = np.zeros((B, 0), dtype=np.float32)
    cot = W.random_cotangent(B, n, seed=14400 + n)
    note(f"qaoa n={n} p={p}")
    r = run_qasm(torch_mod, qaoa_program(n, p), (), params, x, cot, probs=True)
    ops = qaoa_ops(n, p)
    dpr, dxr, Er = oracle.vjp(ops, n, params, np.zeros((B, 1)), cot)
    check_E(r["E"], Er)
    check_grads({"dp": r["dp"], "dx": np.zeros((B, 0))}, dpr, np.zeros((B, 0)), cot)
    pr = oracle.probabilities(ops, n, params, np.zeros((B, 1)))
    assert np.max(np.abs(r["probs"] - pr)) <= 1e-5
    # MaxCut expectation from the probabilities: a property at any size
    cut = np.array([sum(((k >> i) & 1) != ((k >> ((i + 1) % n)) & 1) for i in range(n))
                    for k in range(1 << n)])
    assert np.max(np.abs(r["probs"] @ cut - pr @ cut)) <= 1e-3


QFT = """OPENQASM 2.0;
include "qelib1.inc";
qreg q[{n}];
creg c[{n}];
{body}
measure q -> c;
"""


def qft_ops(n):
    ops = []
    for j in range(n - 1, -1, -1):
        ops.append(Op("H", (j,)))
        for k in range(j - 1, -1, -1):
            ops.append(Op("CP", (k, j), (("const", math.pi / 2 ** (j - k)),)))
    for i in range(n // 2):
        ops.append(Op("SWAP", (i, n - 1 - i)))
    return ops


def test_qft_program_on_basis_and_random_states(torch_mod):
    """A constant circuit (every gate cached at compile time) from Psi_0: the
    QFT of a basis state |k> has uniform probabilities 2^-n."""
    n = 7
    body = []
    for j in range(n - 1, -1, -1):
        body.append(f"h q[{j}];")
        for k in range(j - 1, -1, -1):
            body.append(f"cu1(pi/{2 ** (j - k)}) q[{k}], q[{j}];")
    for i in range(n // 2):
        body.append(f"swap q[{i}], q[{n - 1 - i}];")
    src = QFT.format(n=n, body="\n".join(body))
    B = 4
    s0 = W.random_states(B, n, seed=14500, kind="basis")
    s1 = W.random_states(B, n, seed=14501)
    note("qft program")
    for psi0 in (s0, s1):
        r = run_qasm(torch_mod, src, (), np.zeros((B, 0), np.float32), np.zeros((B, 0), np.float32),
                     np.zeros((B, n), np.float32), psi0=psi0, probs=True)
        Er, st = oracle.forward(qft_ops(n), n, np.zeros((B, 1)), np.zeros((B, 1)),
                                want_state=True, psi0=psi0)
        check_E(r["E"], Er)
        assert np.max(np.abs(r["probs"] - np.abs(st) ** 2)) <= 1e-5
    assert np.max(np.abs(r["probs"] - 1.0 / (1 << n))) > 1e-3  # random states: not uniform
    r = run_qasm(torch_mod, src, (), np.zeros((B, 0), np.float32), np.zeros((B, 0), np.float32),
                 np.zeros((B, n), np.float32), psi0=s0, probs=True)
    assert np.max(np.abs(r["probs"] - 1.0 / (1 << n))) <= 1e-6
