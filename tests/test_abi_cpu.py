"""C ABI checks that need no GPU: exports, validation and host-only plans.

vqc_compile with device = -1 plans on the host only and makes no HIP call,
so every validation path of the compile phase is exercised here.
"""
import ctypes
import math
import re

import pytest

from paper_2607_11985_amd import _lib
from paper_2607_11985_amd import workloads as W


@pytest.fixture(scope="module")
def lib():
    return _lib.load()


def host_compile(ops, n, P, F, path=0, reserved=None, raw=None, reg_bits=0, engine=0):
    arr = raw if raw is not None else _lib.encode_ops(ops)
    opts = _lib.vqc_compile_opts(device=-1, path=path, reg_bits=reg_bits, engine=engine)
    if reserved is not None:
        opts.reserved[0] = reserved
    return _lib.vqc_compile_raw(arr, len(ops) if raw is None else raw._n, n, P, F, opts)


def test_exports_every_declared_function(lib):
    names = _lib.header_functions()
    assert {"vqc_compile", "vqc_forward", "vqc_backward", "vqc_destroy",
            "vqc_workspace_bytes", "vqc_loss_grad", "vqc_last_error",
            "vqc_circuit_info", "vqc_jit_check", "vqc_forward_ex", "vqc_train_step",
            "vqc_fd_backward", "vqc_parse_qasm", "vqc_compile_qasm"} <= set(names)
    for name in names:
        assert hasattr(lib, name), name


def test_header_constants_match_binding():
    text = open(_lib.HEADER).read()
    defs = dict(re.findall(r"#define\s+(VQC_\w+)\s+(-?\d+)", text))
    for name in ("VQC_OK", "VQC_ERR_INVALID_ARG", "VQC_ERR_UNSUPPORTED", "VQC_ERR_TOO_LARGE",
                 "VQC_ERR_WORKSPACE", "VQC_ERR_HIP", "VQC_ERR_OOM"):
        assert int(defs[name]) == getattr(_lib, name)
    for k, v in _lib.KIND.items():
        assert int(defs["VQC_" + k]) == v
    assert int(defs["VQC_SRC_PARAM"]) == 0 and int(defs["VQC_SRC_CONST"]) == 2
    assert int(defs["VQC_LOSS_MSE_MEANZ"]) == _lib.LOSS["mse_meanz"]
    assert int(defs["VQC_ENGINE_JIT"]) == _lib.VQC_ENGINE_JIT
    assert int(defs["VQC_ENGINE_INTERP"]) == _lib.VQC_ENGINE_INTERP
    assert ctypes.sizeof(_lib.vqc_compile_opts) == 32 and ctypes.sizeof(_lib.vqc_info) == 96
    assert ctypes.sizeof(_lib.vqc_op) == 64


@pytest.mark.parametrize("idx", [1, 2, 3, 4, 5])
def test_configs_plan_on_host(idx):
    w = W.make_config(idx, batch=2)
    rc, h = host_compile(w.ops, w.n_qubits, w.n_params, w.n_inputs)
    assert rc == 0, _lib.vqc_last_error()
    info = _lib.vqc_circuit_info(h)
    rot, ent, nops = W.count_ops(w.ops)
    assert info["n_rotations"] == rot and info["n_ops"] == nops
    stream = w.n_qubits >= 14
    assert info["path"] == (_lib.VQC_PATH_STREAM if stream else _lib.VQC_PATH_RESIDENT)
    # the streaming path uses 12-qubit tiles (four workgroups per CU) where they
    # take at most a quarter more passes than 13 (configs 4 and 5)
    tile = 12 if stream else max(4, w.n_qubits)
    assert info["tile_qubits"] == tile
    if w.n_qubits >= 14:
        assert info["fwd_passes"] > 1 and info["bwd_passes"] > 1
    assert info["lds_bytes_bwd"] <= 160 * 1024
    # forward and backward sweep each hold one instruction per primitive plus
    # exchanges, except the trailing entanglers (no rotation after them on their
    # qubits), which the measurement absorbs: here the last layer's CNOT ring / CZ
    # chain; and except the diagonal gates that commute with every gate after
    # them: here every qubit's last RZ (each layer ends in RZ before its
    # entanglers)
    blocked, trailing = set(), 0
    for o in reversed(w.ops):
        if o.kind in ("CNOT", "CZ") and not blocked & set(o.wires):
            trailing += 1
        else:
            blocked |= set(o.wires)
    assert trailing == (w.n_qubits - 1 if idx == 4 else w.n_qubits)
    last = {}
    for o in w.ops:
        if o.kind not in ("CNOT", "CZ"):
            last[o.wires[0]] = o.kind
    assert all(k in ("RZ", "ROT") for k in last.values())
    n_prims = sum(3 if o.kind == "ROT" else 1 for o in w.ops) - trailing - w.n_qubits
    assert info["fwd_instructions"] == n_prims + info["fwd_exchanges"]
    assert info["bwd_instructions"] == n_prims + info["bwd_exchanges"]
    assert _lib.vqc_workspace_bytes(h, 0, 1) == 0
    assert _lib.vqc_workspace_bytes(h, 10, 4) == ctypes.c_size_t(-1).value
    step = _lib.vqc_workspace_bytes(h, 10, 2)
    if stream:  # training workspace plus the cotangent rows
        assert step >= _lib.vqc_workspace_bytes(h, 10, 1) + 10 * w.n_qubits * 4
    else:       # the resident step keeps every state on chip
        assert step == 0
    assert _lib.vqc_workspace_bytes(h, 10, 0) == (0 if not stream else
                                                  _lib.vqc_workspace_bytes(h, 10, 0))
    assert _lib.vqc_workspace_bytes(h, 10, 1) >= 10 * (1 << w.n_qubits) * 8 * (3 if stream else 1)
    _lib.vqc_destroy(h)


def test_host_only_handle_cannot_run(lib):
    w = W.make_config(1, batch=2)
    rc, h = host_compile(w.ops, 4, w.n_params, w.n_inputs)
    assert rc == 0
    rc = lib.vqc_forward(h, 2, 1, 1, 1, None, 0, None)
    assert rc == _lib.VQC_ERR_INVALID_ARG and "host-only" in _lib.vqc_last_error()
    rc = lib.vqc_backward(h, 2, 1, 1, 1, 1, 1 << 20, 1, 1, None)
    assert rc == _lib.VQC_ERR_INVALID_ARG
    rc = lib.vqc_train_step(h, 2, 1, 1, 0, None, 1, None, 1, 1, None, 0, None)
    assert rc == _lib.VQC_ERR_INVALID_ARG and "host-only" in _lib.vqc_last_error()
    _lib.vqc_destroy(h)


def test_null_handle_and_out(lib):
    assert lib.vqc_forward(None, 1, None, None, None, None, 0, None) == _lib.VQC_ERR_INVALID_ARG
    assert lib.vqc_backward(None, 1, None, None, None, None, 0, None, None, None) == \
        _lib.VQC_ERR_INVALID_ARG
    assert lib.vqc_circuit_info(None, None) == _lib.VQC_ERR_INVALID_ARG
    assert lib.vqc_train_step(None, 1, None, None, 0, None, None, None, None, None, None, 0,
                              None) == _lib.VQC_ERR_INVALID_ARG
    assert lib.vqc_workspace_bytes(None, 1, 1) == ctypes.c_size_t(-1).value
    lib.vqc_destroy(None)
    arr = _lib.encode_ops([])
    opts = _lib.vqc_compile_opts(device=-1)
    assert lib.vqc_compile(arr, 0, 2, 0, 0, ctypes.byref(opts), None) == _lib.VQC_ERR_INVALID_ARG


def _one(kind, wires, angles=()):
    return [W.Op(kind, wires, angles)]


BAD = [
    ("wire_high", _one("RY", (3,), (("param", 0),)), 3, 1, 0, _lib.VQC_ERR_INVALID_ARG, "wire"),
    ("wire_negative", _one("RX", (-1,), (("param", 0),)), 3, 1, 0, _lib.VQC_ERR_INVALID_ARG, "wire"),
    ("cnot_same", _one("CNOT", (1, 1)), 3, 0, 0, _lib.VQC_ERR_INVALID_ARG, "twice"),
    ("ccx_same", _one("CCX", (0, 2, 0)), 3, 0, 0, _lib.VQC_ERR_INVALID_ARG, "twice"),
    ("cswap_high", _one("CSWAP", (0, 1, 3)), 3, 0, 0, _lib.VQC_ERR_INVALID_ARG, "wire"),
    ("zero_mul", _one("RY", (0,), (("param", 0, 0.0, 0.1),)), 2, 1, 0, _lib.VQC_ERR_INVALID_ARG,
     "mul"),
    ("inf_mul", _one("CRX", (0, 1), (("input", 0, math.inf, 0.0),)), 2, 0, 1,
     _lib.VQC_ERR_INVALID_ARG, "mul"),
    ("nan_offset", _one("U3", (0,), (("param", 0, 1.0, math.nan), ("const", 0.0),
                                     ("const", 0.0))), 2, 1, 0, _lib.VQC_ERR_INVALID_ARG,
     "finite"),
    ("cz_high", _one("CZ", (0, 5)), 3, 0, 0, _lib.VQC_ERR_INVALID_ARG, "wire"),
    ("param_range", _one("RZ", (0,), (("param", 4),)), 2, 4, 0, _lib.VQC_ERR_INVALID_ARG, "param"),
    ("input_range", _one("RZ", (0,), (("input", 1),)), 2, 0, 1, _lib.VQC_ERR_INVALID_ARG, "input"),
    ("input_negative", _one("RZ", (0,), (("input", -1),)), 2, 0, 1, _lib.VQC_ERR_INVALID_ARG, "input"),
    ("nan_const", _one("RX", (0,), (("const", math.nan),)), 2, 0, 0, _lib.VQC_ERR_INVALID_ARG, "finite"),
    ("zero_qubits", [], 0, 0, 0, _lib.VQC_ERR_INVALID_ARG, "n_qubits"),
    ("too_many_qubits", [], 21, 0, 0, _lib.VQC_ERR_TOO_LARGE, "n_qubits"),
    ("negative_params", [], 2, -1, 0, _lib.VQC_ERR_INVALID_ARG, "n_params"),
]


@pytest.mark.parametrize("case", BAD, ids=[b[0] for b in BAD])
def test_compile_rejects(case):
    _, ops, n, P, F, code, text = case
    rc, h = host_compile(ops, n, P, F)
    assert rc == code
    assert text in _lib.vqc_last_error()
    assert not h.value


def test_compile_rejects_unknown_kind_and_source():
    arr = _lib.encode_ops(_one("RX", (0,), (("param", 0),)))
    arr[0].kind = 32
    rc, _ = _lib.vqc_compile_raw(arr, 1, 2, 1, 0, _lib.vqc_compile_opts(device=-1))
    assert rc == _lib.VQC_ERR_INVALID_ARG and "kind" in _lib.vqc_last_error()
    arr = _lib.encode_ops(_one("RX", (0,), (("param", 0),)))
    arr[0].src[0] = 7
    rc, _ = _lib.vqc_compile_raw(arr, 1, 2, 1, 0, _lib.vqc_compile_opts(device=-1))
    assert rc == _lib.VQC_ERR_INVALID_ARG and "source" in _lib.vqc_last_error()


def test_compile_rejects_options():
    rc, _ = host_compile([], 2, 0, 0, reserved=1)
    assert rc == _lib.VQC_ERR_INVALID_ARG and "reserved" in _lib.vqc_last_error()
    rc, _ = host_compile([], 2, 0, 0, path=7)
    assert rc == _lib.VQC_ERR_INVALID_ARG
    rc, _ = host_compile([], 2, 0, 0, engine=2)
    assert rc == _lib.VQC_ERR_INVALID_ARG and "engine" in _lib.vqc_last_error()
    arr = _lib.encode_ops([])
    rc, _ = _lib.vqc_compile_raw(arr, 0, 2, 0, 0, _lib.vqc_compile_opts(device=-1, shared_params=2))
    assert rc == _lib.VQC_ERR_INVALID_ARG and "shared_params" in _lib.vqc_last_error()
    for n, bad in ((6, 1), (6, 5), (6, -1), (6, 6), (15, 3), (15, 6)):
        rc, _ = host_compile([], n, 0, 0, reg_bits=bad)
        assert rc == _lib.VQC_ERR_INVALID_ARG and "reg_bits" in _lib.vqc_last_error()
    rc, _ = host_compile([], 15, 0, 0, path=_lib.VQC_PATH_RESIDENT)
    assert rc == _lib.VQC_ERR_UNSUPPORTED
    arr = _lib.encode_ops([])
    rc, _ = _lib.vqc_compile_raw(arr, -1, 2, 0, 0, _lib.vqc_compile_opts(device=-1))
    assert rc == _lib.VQC_ERR_INVALID_ARG
    rc = _lib.load().vqc_compile(None, 3, 2, 0, 0, ctypes.byref(_lib.vqc_compile_opts(device=-1)),
                                 ctypes.byref(ctypes.c_void_p()))
    assert rc == _lib.VQC_ERR_INVALID_ARG


def test_loss_grad_validation(lib):
    assert lib.vqc_loss_grad(9, 4, 2, 1, 1, 1, None) == _lib.VQC_ERR_INVALID_ARG
    assert lib.vqc_loss_grad(0, -1, 2, 1, 1, 1, None) == _lib.VQC_ERR_INVALID_ARG
    assert lib.vqc_loss_grad(2, 4, 2, 1, None, 1, None) == _lib.VQC_ERR_INVALID_ARG
    assert lib.vqc_loss_grad(0, 4, 2, None, None, 1, None) == _lib.VQC_ERR_INVALID_ARG
    assert lib.vqc_loss_grad(0, 0, 2, None, None, None, None) == _lib.VQC_OK


@pytest.mark.parametrize("n", [1, 2, 4, 5, 8, 11, 14])
def test_random_circuits_plan(n):
    ops, P, F = W.random_circuit(n, 60, seed=n)
    rc, h = host_compile(ops, n, P, F)
    assert rc == 0, _lib.vqc_last_error()
    info = _lib.vqc_circuit_info(h)
    nq = max(n, 4)
    R = 2 if nq <= 8 else 3 if nq <= 10 else 4
    k = 13 if nq >= 14 else nq  # streamed from 14 qubits, in 13-qubit tiles
    assert info["threads"] == max(64, 1 << (k - R))
    _lib.vqc_destroy(h)


def test_empty_circuit_plans():
    rc, h = host_compile([], 3, 0, 0)
    assert rc == 0
    info = _lib.vqc_circuit_info(h)
    assert info["fwd_instructions"] == 0 and info["n_rotations"] == 0
    _lib.vqc_destroy(h)


@pytest.mark.parametrize("engine", [0, 1])
def test_info_reports_engine(engine):
    rc, h = host_compile([], 3, 0, 0, engine=engine)
    assert rc == 0
    assert _lib.vqc_circuit_info(h)["engine"] == engine
    _lib.vqc_destroy(h)


@pytest.mark.parametrize("reg_bits", [2, 3, 4])
def test_register_width_option(reg_bits):
    ops, P, F = W.random_circuit(9, 50, seed=9)
    rc, h = host_compile(ops, 9, P, F, reg_bits=reg_bits)
    assert rc == 0, _lib.vqc_last_error()
    info = _lib.vqc_circuit_info(h)
    assert info["threads"] == max(64, 1 << (9 - reg_bits))
    _lib.vqc_destroy(h)


# Run-time code generation: every kind of instruction the generator emits
# (register / thread / tile positions of rotations, CNOT and CZ, exchanges,
# gradient slots) must compile for gfx950.  No GPU is needed for this.
JIT_CASES = [
    ("n1", 1, 0, 0), ("n5_r2", 5, 0, 2), ("n7_r3", 7, 0, 3), ("n11", 11, 0, 0),
    ("n13", 13, 0, 0), ("n15_stream", 15, 0, 0),
]


@pytest.mark.parametrize("case", JIT_CASES, ids=[c[0] for c in JIT_CASES])
def test_generated_kernels_compile(case):
    _, n, path, reg_bits = case
    ops, P, F = W.random_circuit(n, 30 + 3 * n, seed=31 + n,
                                 kinds=("RX", "RY", "RZ", "ROT", "CNOT", "CZ"))
    rc, h = host_compile(ops, n, P, F, path=path, reg_bits=reg_bits)
    assert rc == 0, _lib.vqc_last_error()
    _lib.vqc_jit_check(h)
    _lib.vqc_destroy(h)


def test_generated_kernels_compile_config2():
    w = W.make_config(2, batch=2)
    rc, h = host_compile(w.ops, w.n_qubits, w.n_params, w.n_inputs)
    assert rc == 0
    _lib.vqc_jit_check(h)
    _lib.vqc_destroy(h)


def test_forward_ex_validation(lib):
    assert lib.vqc_forward_ex(None, 1, None, None, None, None, None, None, 0,
                              None) == _lib.VQC_ERR_INVALID_ARG
    ops, P, F = W.random_circuit(3, 10, seed=3)
    rc, h = host_compile(ops, 3, P, F)
    assert rc == 0
    # a host-only handle cannot run
    assert lib.vqc_forward_ex(h, 1, None, None, None, None, None, None, 0,
                              None) == _lib.VQC_ERR_INVALID_ARG
    assert "host-only" in _lib.vqc_last_error()
    _lib.vqc_destroy(h)


def test_fd_backward_validation(lib):
    assert lib.vqc_fd_backward(None, 1, None, None, None, 1e-2, None, 0, None, None,
                               None) == _lib.VQC_ERR_INVALID_ARG
    w = W.make_config(5, batch=2)
    rc, h = host_compile(w.ops, w.n_qubits, w.n_params, w.n_inputs)
    assert rc == 0
    # streaming: one chunk of slots at a time, its shifted copies' states (two
    # buffers, passes alternate between them) within 2 GiB: 4 samples x 2
    # shifts x 2 buffers x 512 KiB = 8 MiB per slot, 256 of the 400 slots per
    # chunk (2 GiB of states) plus their E rows
    nb = _lib.vqc_workspace_bytes(h, 4, 3)
    state = (1 << 16) * 8
    assert 4 * 2 * 2 * 256 * state <= nb < 4 * 2 * 2 * 256 * state * 1.2
    # a large batch takes smaller chunks: the workspace stays near the budget
    nb = _lib.vqc_workspace_bytes(h, 256, 3)
    assert (2 << 30) * 0.9 <= nb <= (2 << 30) * 1.2
    _lib.vqc_destroy(h)
    w = W.make_config(2, batch=2)
    rc, h = host_compile(w.ops, w.n_qubits, w.n_params, w.n_inputs)
    assert _lib.vqc_workspace_bytes(h, 4, 3) >= 4 * 2 * (w.n_params + w.n_inputs) * 8 * 4
    _lib.vqc_destroy(h)


def test_jit_check_null(lib):
    assert lib.vqc_jit_check(None) == _lib.VQC_ERR_INVALID_ARG


@pytest.mark.parametrize("idx", [2, 5])
def test_shared_params_workspace(idx):
    """Shared parameters add the per-sample gradient rows [B, P] to the
    training workspaces and change nothing else."""
    w = W.make_config(idx, batch=2)
    arr = _lib.encode_ops(w.ops)
    sizes = {}
    for shared in (0, 1):
        rc, h = _lib.vqc_compile_raw(arr, len(w.ops), w.n_qubits, w.n_params, w.n_inputs,
                                     _lib.vqc_compile_opts(device=-1, shared_params=shared))
        assert rc == 0, _lib.vqc_last_error()
        assert _lib.vqc_circuit_info(h)["shared_params"] == shared
        sizes[shared] = [_lib.vqc_workspace_bytes(h, 10, m) for m in (0, 1, 2)]
        _lib.vqc_destroy(h)
    assert sizes[1][0] == sizes[0][0]
    for m in (1, 2):
        assert sizes[1][m] >= sizes[0][m] + 10 * w.n_params * 4


def test_tile_qubits_option():
    ops, P, F = W.random_circuit(15, 20, seed=5)
    arr = _lib.encode_ops(ops)
    for tq, code in ((11, _lib.VQC_ERR_INVALID_ARG), (15, _lib.VQC_ERR_INVALID_ARG)):
        rc, _ = _lib.vqc_compile_raw(arr, len(ops), 15, P, F,
                                     _lib.vqc_compile_opts(device=-1, tile_qubits=tq))
        assert rc == code and "tile_qubits" in _lib.vqc_last_error()
    for tq in (12, 13):
        rc, _ = _lib.vqc_compile_raw(arr, len(ops), 15, P, F,
                                     _lib.vqc_compile_opts(device=-1, tile_qubits=tq, engine=1))
        assert rc == _lib.VQC_ERR_UNSUPPORTED
        rc, h = _lib.vqc_compile_raw(arr, len(ops), 15, P, F,
                                     _lib.vqc_compile_opts(device=-1, tile_qubits=tq))
        assert rc == 0
        info = _lib.vqc_circuit_info(h)
        assert info["tile_qubits"] == tq and info["threads"] == 1 << (tq - 4)
        assert info["path"] == 2
        _lib.vqc_jit_check(h)
        _lib.vqc_destroy(h)


@pytest.mark.parametrize("idx,heads", [(4, 42), (5, 64)])
def test_streaming_step_plan(idx, heads):
    """The streaming training step's own plan: it leaves out every qubit's head
    (RY encoding and the first layer's rotations here), so that its passes run
    the other rotations only; the inference forward keeps the whole circuit."""
    w = W.make_config(idx, batch=2)
    rc, h = host_compile(w.ops, w.n_qubits, w.n_params, w.n_inputs)
    assert rc == 0, _lib.vqc_last_error()
    info = _lib.vqc_circuit_info(h)
    assert info["path"] == 2
    assert info["step_head_rotations"] == heads
    assert 1 <= info["step_fwd_passes"] <= info["fwd_passes"]
    assert info["step_bwd_passes"] == info["step_fwd_passes"]
    _lib.vqc_jit_check(h)
    _lib.vqc_destroy(h)


def test_no_step_plan_without_heads_or_generated_kernels():
    n = 14
    ops, P, F = W.random_circuit(n, 5 * n, seed=77)
    lead = [W.Op("CZ", (q, q + 1)) for q in range(0, n - 1, 2)]
    for o, engine, want in ((ops, 0, True), (lead + ops, 0, False), (ops, 1, False)):
        rc, h = host_compile(o, n, P, F, engine=engine)
        assert rc == 0, _lib.vqc_last_error()
        assert (_lib.vqc_circuit_info(h)["step_head_rotations"] > 0) == want
        _lib.vqc_destroy(h)
    w = W.make_config(2, batch=2)  # resident: the step kernel builds its heads itself
    rc, h = host_compile(w.ops, w.n_qubits, w.n_params, w.n_inputs)
    assert _lib.vqc_circuit_info(h)["step_head_rotations"] == 0
    _lib.vqc_destroy(h)
