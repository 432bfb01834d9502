"""ctypes binding of libvqc.so: the C ABI of include/vqc.h under the same names.

Argument marshalling only -- every step of the computation runs in the HIP
library.  Loading fails loudly when the library has not been built; there is
no fallback implementation.
"""
from __future__ import annotations

import ctypes
import os
import re

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "_build", "libvqc.so")
HEADER = os.path.join(os.path.dirname(_PKG), "include", "vqc.h")

# constants of include/vqc.h
VQC_OK = 0
VQC_ERR_INVALID_ARG = -1
VQC_ERR_UNSUPPORTED = -2
VQC_ERR_TOO_LARGE = -3
VQC_ERR_WORKSPACE = -4
VQC_ERR_HIP = -5
VQC_ERR_OOM = -6
VQC_NOALLOC_SCRATCH_BYTES = 64 << 20
VQC_PATH_AUTO, VQC_PATH_RESIDENT, VQC_PATH_STREAM = 0, 1, 2
VQC_ENGINE_JIT, VQC_ENGINE_INTERP = 0, 1
KIND = {name: code for code, name in enumerate((
    "RX", "RY", "RZ", "ROT", "CNOT", "CZ", "ID", "X", "Y", "Z", "H", "S", "SDG", "T", "TDG",
    "SX", "SXDG", "P", "U2", "U3", "CY", "CH", "SWAP", "CRX", "CRY", "CRZ", "CP", "RXX", "RYY",
    "RZZ", "CCX", "CSWAP"))}
KIND_ALIASES = {"CX": "CNOT", "U1": "P", "U": "U3"}
SRC = {"param": 0, "input": 1, "const": 2}
LOSS = {"sum": 0, "mean": 1, "mse_z0": 2, "mse_meanz": 3}


class vqc_op(ctypes.Structure):
    _fields_ = [("kind", ctypes.c_int32), ("wires", ctypes.c_int32 * 3),
                ("src", ctypes.c_int32 * 3), ("idx", ctypes.c_int32 * 3),
                ("val", ctypes.c_float * 3), ("mul", ctypes.c_float * 3)]


class vqc_compile_opts(ctypes.Structure):
    _fields_ = [("device", ctypes.c_int32), ("path", ctypes.c_int32),
                ("reg_bits", ctypes.c_int32), ("engine", ctypes.c_int32),
                ("shared_params", ctypes.c_int32), ("tile_qubits", ctypes.c_int32),
                ("reserved", ctypes.c_int32 * 2)]


class vqc_info(ctypes.Structure):
    _fields_ = [(name, ctypes.c_int32) for name in (
        "n_qubits", "n_params", "n_inputs", "n_ops", "n_rotations", "path",
        "tile_qubits", "threads", "fwd_passes", "bwd_passes", "fwd_exchanges",
        "bwd_exchanges", "fwd_instructions", "bwd_instructions", "lds_bytes_fwd",
        "lds_bytes_bwd", "engine", "shared_params", "step_head_rotations",
        "step_fwd_passes", "step_bwd_passes")] + [("reserved", ctypes.c_int32 * 3)]


class VQCError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"[{code}] {msg}")
        self.code = code


_lib = None
_vp = ctypes.c_void_p


def load():
    """Load the built library (raises if it is missing)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"HIP library not built: {LIB_PATH} is missing "
                           "(run `python -m paper_2607_11985_amd.build`)")
    lib = ctypes.CDLL(LIB_PATH)
    lib.vqc_compile.argtypes = [ctypes.POINTER(vqc_op), ctypes.c_int32, ctypes.c_int32,
                                ctypes.c_int32, ctypes.c_int32,
                                ctypes.POINTER(vqc_compile_opts), ctypes.POINTER(_vp)]
    lib.vqc_compile.restype = ctypes.c_int
    lib.vqc_parse_qasm.argtypes = [ctypes.c_char_p, ctypes.c_char_p, ctypes.POINTER(vqc_op),
                                   ctypes.c_int32] + [ctypes.POINTER(ctypes.c_int32)] * 4
    lib.vqc_parse_qasm.restype = ctypes.c_int
    lib.vqc_compile_qasm.argtypes = [ctypes.c_char_p, ctypes.c_char_p,
                                     ctypes.POINTER(vqc_compile_opts), ctypes.POINTER(_vp)]
    lib.vqc_compile_qasm.restype = ctypes.c_int
    lib.vqc_destroy.argtypes = [_vp]
    lib.vqc_destroy.restype = None
    lib.vqc_workspace_bytes.argtypes = [_vp, ctypes.c_int64, ctypes.c_int32]
    lib.vqc_workspace_bytes.restype = ctypes.c_size_t
    lib.vqc_forward.argtypes = [_vp, ctypes.c_int64, _vp, _vp, _vp, _vp, ctypes.c_size_t, _vp]
    lib.vqc_forward.restype = ctypes.c_int
    lib.vqc_forward_ex.argtypes = [_vp, ctypes.c_int64, _vp, _vp, _vp, _vp, _vp, _vp,
                                   ctypes.c_size_t, _vp]
    lib.vqc_forward_ex.restype = ctypes.c_int
    lib.vqc_backward.argtypes = [_vp, ctypes.c_int64, _vp, _vp, _vp, _vp, ctypes.c_size_t,
                                 _vp, _vp, _vp]
    lib.vqc_backward.restype = ctypes.c_int
    lib.vqc_loss_grad.argtypes = [ctypes.c_int32, ctypes.c_int64, ctypes.c_int32, _vp, _vp,
                                  _vp, _vp]
    lib.vqc_loss_grad.restype = ctypes.c_int
    lib.vqc_train_step.argtypes = [_vp, ctypes.c_int64, _vp, _vp, ctypes.c_int32, _vp, _vp, _vp,
                                   _vp, _vp, _vp, ctypes.c_size_t, _vp]
    lib.vqc_train_step.restype = ctypes.c_int
    lib.vqc_train_step_noalloc.argtypes = [_vp, ctypes.c_int64, _vp, _vp, ctypes.c_int32, _vp,
                                           _vp, _vp, _vp, _vp, _vp]
    lib.vqc_train_step_noalloc.restype = ctypes.c_int
    lib.vqc_fd_backward.argtypes = [_vp, ctypes.c_int64, _vp, _vp, _vp, ctypes.c_float, _vp,
                                    ctypes.c_size_t, _vp, _vp, _vp]
    lib.vqc_fd_backward.restype = ctypes.c_int
    lib.vqc_jit_check.argtypes = [_vp]
    lib.vqc_jit_check.restype = ctypes.c_int
    lib.vqc_circuit_info.argtypes = [_vp, ctypes.POINTER(vqc_info)]
    lib.vqc_circuit_info.restype = ctypes.c_int
    lib.vqc_last_error.argtypes = []
    lib.vqc_last_error.restype = ctypes.c_char_p
    _lib = lib
    return lib


def header_functions() -> list:
    """Names of the functions include/vqc.h declares."""
    text = open(HEADER).read()
    return sorted(set(re.findall(r"^\s*(?:const\s+)?[a-z_]+\s*\*?\s*(vqc_[a-z_]+)\s*\(",
                                 text, flags=re.M)))


def _check(rc: int):
    if rc != VQC_OK:
        raise VQCError(rc, load().vqc_last_error().decode())


def encode_ops(ops) -> ctypes.Array:
    """Gate list (kind, wires, angles) -> vqc_op array.  An angle is
    ("const", value), (src, index) or (src, index, mul, add)."""
    arr = (vqc_op * max(1, len(ops)))()
    for k, op in enumerate(ops):
        r = arr[k]
        r.kind = KIND[KIND_ALIASES.get(op.kind, op.kind)]
        w = list(op.wires) + [-1, -1, -1]
        r.wires[0], r.wires[1], r.wires[2] = w[0], w[1], w[2]
        for s, spec in enumerate(op.angles):
            src, v = spec[0], spec[1]
            r.src[s] = SRC[src]
            r.mul[s] = 1.0
            if src == "const":
                r.val[s] = float(v)
            else:
                r.idx[s] = int(v)
                if len(spec) > 2:
                    r.mul[s] = float(spec[2])
                if len(spec) > 3:
                    r.val[s] = float(spec[3])
    return arr


def vqc_compile(ops, n_qubits: int, n_params: int, n_inputs: int, device: int = 0,
                path: int = VQC_PATH_AUTO, reg_bits: int = 0, engine: int = VQC_ENGINE_JIT,
                shared_params: int = 0, tile_qubits: int = 0):
    lib = load()
    arr = encode_ops(ops)
    opts = vqc_compile_opts(device=device, path=path, reg_bits=reg_bits, engine=engine,
                            shared_params=shared_params, tile_qubits=tile_qubits)
    h = _vp()
    _check(lib.vqc_compile(arr, len(ops), n_qubits, n_params, n_inputs, ctypes.byref(opts),
                           ctypes.byref(h)))
    return h


def vqc_compile_raw(arr, n_ops, n_qubits, n_params, n_inputs, opts):
    """Unchecked call (returns (status, handle)) for validation tests."""
    lib = load()
    h = _vp()
    rc = lib.vqc_compile(arr, n_ops, n_qubits, n_params, n_inputs,
                         ctypes.byref(opts) if opts is not None else None, ctypes.byref(h))
    return rc, h


def vqc_parse_qasm(source: str, input_names: str | None = None):
    """(vqc_op array, n_ops, n_qubits, n_params, n_inputs) of an OpenQASM program."""
    lib = load()
    counts = [ctypes.c_int32() for _ in range(4)]
    src = source.encode()
    names = input_names.encode() if input_names else None
    _check(lib.vqc_parse_qasm(src, names, None, 0, *[ctypes.byref(c) for c in counts]))
    n = counts[0].value
    arr = (vqc_op * max(1, n))()
    _check(lib.vqc_parse_qasm(src, names, arr, n, *[ctypes.byref(c) for c in counts]))
    return arr, n, counts[1].value, counts[2].value, counts[3].value


def vqc_compile_qasm(source: str, input_names: str | None = None, device: int = 0,
                     path: int = VQC_PATH_AUTO, reg_bits: int = 0, engine: int = VQC_ENGINE_JIT,
                     shared_params: int = 0, tile_qubits: int = 0):
    lib = load()
    opts = vqc_compile_opts(device=device, path=path, reg_bits=reg_bits, engine=engine,
                            shared_params=shared_params, tile_qubits=tile_qubits)
    h = _vp()
    _check(lib.vqc_compile_qasm(source.encode(), input_names.encode() if input_names else None,
                                ctypes.byref(opts), ctypes.byref(h)))
    return h


def vqc_destroy(h):
    load().vqc_destroy(h)


def vqc_workspace_bytes(h, batch: int, training: int) -> int:
    return int(load().vqc_workspace_bytes(h, batch, training))


def vqc_forward(h, batch, params_ptr, inputs_ptr, expvals_ptr, ws_ptr, ws_bytes, stream):
    _check(load().vqc_forward(h, batch, params_ptr, inputs_ptr, expvals_ptr, ws_ptr, ws_bytes,
                              stream))


def vqc_forward_ex(h, batch, params_ptr, inputs_ptr, psi0_ptr, expvals_ptr, probs_ptr, ws_ptr,
                   ws_bytes, stream):
    _check(load().vqc_forward_ex(h, batch, params_ptr, inputs_ptr, psi0_ptr, expvals_ptr,
                                 probs_ptr, ws_ptr, ws_bytes, stream))


def vqc_backward(h, batch, params_ptr, inputs_ptr, grad_ptr, ws_ptr, ws_bytes, dparams_ptr,
                 dinputs_ptr, stream):
    _check(load().vqc_backward(h, batch, params_ptr, inputs_ptr, grad_ptr, ws_ptr, ws_bytes,
                               dparams_ptr, dinputs_ptr, stream))


def vqc_train_step(h, batch, params_ptr, inputs_ptr, loss_kind, y_ptr, expvals_ptr, grad_ptr,
                   dparams_ptr, dinputs_ptr, ws_ptr, ws_bytes, stream):
    _check(load().vqc_train_step(h, batch, params_ptr, inputs_ptr, loss_kind, y_ptr, expvals_ptr,
                                 grad_ptr, dparams_ptr, dinputs_ptr, ws_ptr, ws_bytes, stream))


def vqc_train_step_noalloc(h, batch, params_ptr, inputs_ptr, loss_kind, y_ptr, expvals_ptr,
                           grad_ptr, dparams_ptr, dinputs_ptr, stream):
    _check(load().vqc_train_step_noalloc(h, batch, params_ptr, inputs_ptr, loss_kind, y_ptr,
                                         expvals_ptr, grad_ptr, dparams_ptr, dinputs_ptr, stream))


def vqc_loss_grad(kind: int, batch: int, n: int, e_ptr, y_ptr, g_ptr, stream):
    _check(load().vqc_loss_grad(kind, batch, n, e_ptr, y_ptr, g_ptr, stream))


def vqc_fd_backward(h, batch, params_ptr, inputs_ptr, grad_ptr, step, ws_ptr, ws_bytes,
                    dparams_ptr, dinputs_ptr, stream):
    _check(load().vqc_fd_backward(h, batch, params_ptr, inputs_ptr, grad_ptr, step, ws_ptr,
                                  ws_bytes, dparams_ptr, dinputs_ptr, stream))


def vqc_jit_check(h):
    _check(load().vqc_jit_check(h))


def vqc_circuit_info(h) -> dict:
    info = vqc_info()
    _check(load().vqc_circuit_info(h, ctypes.byref(info)))
    return {name: getattr(info, name) for name, _ in vqc_info._fields_ if name != "reserved"}


def vqc_last_error() -> str:
    return load().vqc_last_error().decode()
