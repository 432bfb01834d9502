"""Host side of the runs of RZs applied as one diagonal: the generated
kernels (read back from the compile check, no GPU) hold fused runs in the
forward and the adjoint on every kernel geometry, and the circuits of
test_gpu_diag_runs reach the forms of a run that its GPU parity tests are
there for: a product factor for two RZs of one bit, a frame-negated angle,
and one parameter's partials summed in one pending slot.  Also the planner's
list schedule: runs of many RZs, with the exchange counts of circuit order."""
import os
import re

import pytest

from paper_2607_11985_amd import _lib
from paper_2607_11985_amd import workloads as W
from tests.test_gpu_diag_runs import diag_run_circuit


def generated(tmp_path, ops, n, P, F, path=0):
    os.environ["VQC_JIT_DUMP"] = str(tmp_path)
    try:
        rc, h = _lib.vqc_compile_raw(_lib.encode_ops(ops), len(ops), n, P, F,
                                     _lib.vqc_compile_opts(device=-1, path=path))
        assert rc == 0, _lib.vqc_last_error()
        info = _lib.vqc_circuit_info(h)
        _lib.vqc_jit_check(h)
        _lib.vqc_destroy(h)
    finally:
        del os.environ["VQC_JIT_DUMP"]
    return info, {p.stem: p.read_text() for p in tmp_path.glob("*.hip")}


def runs(text):
    return [int(m) for m in re.findall(r"// (\d+) RZs as one diagonal", text)]


@pytest.mark.parametrize("n,path,fwd,bwd", [(8, 0, "vqc_rf", "vqc_rb"), (12, 0, "vqc_rf", "vqc_rb"),
                                            (14, 2, "vqc_sf", "vqc_sb")])
def test_runs_generated(tmp_path, n, path, fwd, bwd):
    ops, P, F = diag_run_circuit(n, 29000 + n)
    info, src = generated(tmp_path, ops, n, P, F, path)
    f = "".join(t for k, t in src.items() if k.startswith(fwd))
    b = "".join(t for k, t in src.items() if k.startswith(bwd))
    assert runs(f) and runs(b), sorted(src)
    assert max(runs(b)) >= 4
    every = "".join(src.values())
    # two RZs of one register bit in a run: a product factor for that bit
    assert re.search(r"double F\d+r = 1\.0, F\d+i = ", every)
    # an RZ on a bit under the swap frame, inside a run (16 amplitudes per
    # thread; the kernels with lane gates keep no frame)
    if n > 8:
        assert re.search(r"const float t\d+ = flip_sign\(tc\d+\.x, fs\d\);", every)
    # one parameter read by two RZs of a run: the second partial adds to the pending slot
    blocks = re.findall(r"RZs as one diagonal\n(.*?)gate_boundary", b, re.S)
    assert any(re.search(r"pd(\d+) = g;.*pd\1 \+= g;", blk, re.S) for blk in blocks)


def run_members(text):
    """The angle occurrences of every run of a generated kernel that reads its
    tables ahead (LDS tables): a run's first member is the entry the previous
    gate read ahead, the others are read in the run."""
    members, ahead = [], None
    for line in text.splitlines():
        if "RZs as one diagonal" in line:
            members.append([ahead])
        m = re.search(r"const float2 tc\d+ = w\.tab\[(\d+)\];", line)
        if m and members and len(members[-1]) and "tc0" not in line:
            members[-1].append(int(m.group(1)))
        m = re.search(r"tcn = w\.tab\[(\d+)\];", line)
        if m:
            ahead = int(m.group(1))
    return members


def test_constant_rz_stay_gate_by_gate(tmp_path):
    """RZs with constant angles (T gates) beside variable ones: never in a
    run (an RX layer at the end keeps the RZs from being dropped as diagonal
    gates before the measurement).  Occurrences: RY 0..n-1, then per qubit q
    the constant RZ at n + 2q and the variable one at n + 2q + 1."""
    n = 12
    ops = [W.Op("RY", (q,), (("param", q),)) for q in range(n)]
    for q in range(n):
        ops += [W.Op("RZ", (q,), (("const", 0.785398),)), W.Op("RZ", (q,), (("param", n + q),))]
    ops += [W.Op("CNOT", (q, (q + 1) % n)) for q in range(n)]
    ops += [W.Op("RX", (q,), (("param", 2 * n + q),)) for q in range(n)]
    _, src = generated(tmp_path, ops, n, 3 * n, 1)
    for name in ("vqc_rf", "vqc_rb"):
        members = run_members(src[name])
        assert members, f"{name}: the variable RZs form runs"
        occ = [o for run in members for o in run]
        assert len(occ) == len(set(occ)) and len(occ) >= n // 2, (name, members)
        assert all(o >= n and (o - n) % 2 == 1 for o in occ), (name, members)


def test_hold_back_keeps_exchange_counts():
    """The list schedule (RZs held back) does not add exchanges on the five
    workloads: their counts are those planned in circuit order."""
    want = {1: (0, 0), 2: (14, 14), 3: (33, 33), 4: (34, 33), 5: (62, 62)}
    for idx, ex in want.items():
        w = W.make_config(idx, batch=2)
        rc, h = _lib.vqc_compile_raw(_lib.encode_ops(w.ops), len(w.ops), w.n_qubits, w.n_params,
                                     w.n_inputs, _lib.vqc_compile_opts(device=-1))
        assert rc == 0
        info = _lib.vqc_circuit_info(h)
        _lib.vqc_destroy(h)
        assert (info["fwd_exchanges"], info["bwd_exchanges"]) == ex, (idx, info)
