"""Double-precision CPU oracle -- TEST INFRASTRUCTURE ONLY.

Only `tests/`, `__graft_entry__.smoke()` and the CPU-baseline leg of
`bench.py` may import this package.  The product path (the HIP library and its
Python binding) never imports it, and it imports nothing from the product.

Contents
  forward(...)          plain complex128 statevector forward pass (C, OpenMP
                        over samples): Sec. 3 and Algorithm 1.
  vjp(...)              exact vector-Jacobian product by stored states and
                        explicit derivative matrices (Sec. 3 "Gate Application
                        and Differentiation").
  param_shift_grad(...) gradients from forward passes only (two-term shift rule,
                        exact for R_P(t) = exp(-i t P/2)); independent of vjp.
  fd_grad(...)          central finite differences (the paper's FD policy,
                        Sec. 4.2.3), independent of vjp.
  probabilities(...)    basis-state probabilities |Psi_k|^2 of the final state.
  loss_cotangent(...)   d loss / d E for the scalar objectives of the
                        workloads (mean of <Z>, sum, MSE heads; Sec. 4.2.3).
  dense                 a second, independent forward by dense 2^n x 2^n
                        matrices built with matrix exponentials (n <= 8).

Ops are any objects with `.kind`, `.wires`, `.angles` in the backend-neutral
gate-list format of the workload generator.  Kinds: RX RY RZ ROT CNOT(CX) CZ,
ID X Y Z H S SDG T TDG SX SXDG, P(U1) U2 U3(U), CY CH SWAP CRX CRY CRZ CP RXX
RYY RZZ, CCX CSWAP (wire 0 is the control of controlled gates).
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from typing import Sequence

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "vqc_oracle.c")
_BUILD = os.path.join(_HERE, "_build")
_LIB_PATH = os.path.join(_BUILD, "liboracle.so")

_GATES = ("RX", "RY", "RZ", "ROT", "CNOT", "CZ",
          "ID", "X", "Y", "Z", "H", "S", "SDG", "T", "TDG", "SX", "SXDG",
          "P", "U2", "U3",
          "CY", "CH", "SWAP", "CRX", "CRY", "CRZ", "CP", "RXX", "RYY", "RZZ",
          "CCX", "CSWAP")
_KIND = {g: i for i, g in enumerate(_GATES)}
_KIND.update({"CX": _KIND["CNOT"], "U1": _KIND["P"], "U": _KIND["U3"]})
_SRC_CODE = {"param": 0, "input": 1, "const": 2}

OP_DTYPE = np.dtype([("kind", np.int32), ("w", np.int32, 3), ("src", np.int32, 3),
                     ("idx", np.int32, 3), ("mul", np.float64, 3), ("add", np.float64, 3)],
                    align=True)

_lib = None


def build(force: bool = True) -> str:
    """Compile the oracle with gcc (plain C99, OpenMP, no fast-math)."""
    os.makedirs(_BUILD, exist_ok=True)
    if force or not os.path.exists(_LIB_PATH):
        tmp = _LIB_PATH + ".tmp"
        cmd = ["gcc", "-std=c99", "-O2", "-fopenmp", "-fPIC", "-shared",
               "-o", tmp, _SRC, "-lm"]
        subprocess.check_call(cmd)
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


def open_library(path: str):
    """Load an oracle build at `path` and declare its entry points."""
    lib = ctypes.CDLL(path)
    dp = ctypes.POINTER(ctypes.c_double)
    lib.oracle_forward.argtypes = [ctypes.c_void_p, ctypes.c_int, ctypes.c_int,
                                   ctypes.c_int, dp, ctypes.c_int, dp,
                                   ctypes.c_int, dp, dp, ctypes.c_int,
                                   ctypes.c_int, ctypes.c_double, ctypes.c_int, dp]
    lib.oracle_forward.restype = ctypes.c_int
    lib.oracle_vjp.argtypes = [ctypes.c_void_p, ctypes.c_int, ctypes.c_int,
                               ctypes.c_int, dp, ctypes.c_int, dp, ctypes.c_int,
                               dp, dp, dp, dp, ctypes.c_int, dp]
    lib.oracle_vjp.restype = ctypes.c_int
    lib.oracle_op_size.restype = ctypes.c_int
    assert lib.oracle_op_size() == OP_DTYPE.itemsize, "oracle_op layout mismatch"
    return lib


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            build(force=False)
        _lib = open_library(_LIB_PATH)
    return _lib


def encode_ops(ops: Sequence) -> np.ndarray:
    """Gate records.  An angle is ("const", value), or (src, index) or
    (src, index, mul, add) for src in {"param", "input"}: mul * value + add."""
    rec = np.zeros(max(1, len(ops)), dtype=OP_DTYPE)
    for k, op in enumerate(ops):
        rec[k]["kind"] = _KIND[op.kind]
        w = list(op.wires) + [-1] * (3 - len(op.wires))
        rec[k]["w"] = w[:3]
        for s, spec in enumerate(op.angles):
            src, v = spec[0], spec[1]
            rec[k]["src"][s] = _SRC_CODE[src]
            if src == "const":
                rec[k]["add"][s] = float(v)
            else:
                rec[k]["idx"][s] = int(v)
                rec[k]["mul"][s] = float(spec[2]) if len(spec) > 2 else 1.0
                rec[k]["add"][s] = float(spec[3]) if len(spec) > 3 else 0.0
    return rec


def _dptr(a: np.ndarray):
    return a.ctypes.data_as(ctypes.POINTER(ctypes.c_double))


def _as2d(a, B, width):
    a = np.ascontiguousarray(np.asarray(a, dtype=np.float64).reshape(B, width))
    if a.size == 0:
        a = np.zeros((B, max(width, 1)), dtype=np.float64)
    return a


def _psi0(psi0, B, n):
    if psi0 is None:
        return None
    a = np.ascontiguousarray(np.asarray(psi0, dtype=np.complex128).reshape(B, 1 << n))
    return a


def forward(ops, n, params, inputs, want_state=False, shift=None, nthreads=0, psi0=None):
    """E [B, n] (float64); with want_state also the final states [B, 2^n] c128.

    params [B, P] and inputs [B, F] are taken as given (float32 values are
    upcast exactly).  shift = (op_index, angle_slot, delta) offsets one angle
    of one gate in every sample.  psi0 [B, 2^n]: initial states (default
    |0...0>), Algorithm 1's optional input.
    """
    lib = _load()
    params = np.asarray(params)
    inputs = np.asarray(inputs)
    B = params.shape[0]
    P = params.shape[1] if params.ndim == 2 else 0
    F = inputs.shape[1] if inputs.ndim == 2 else 0
    p = _as2d(params, B, P)
    x = _as2d(inputs, B, F)
    rec = encode_ops(ops)
    E = np.zeros((B, n), dtype=np.float64)
    st = np.zeros((B, 1 << n), dtype=np.complex128) if want_state else None
    so, ss, sd = shift if shift is not None else (-1, 0, 0.0)
    s0 = _psi0(psi0, B, n)
    rc = lib.oracle_forward(rec.ctypes.data, len(ops), n, B, _dptr(p), max(P, 1),
                            _dptr(x), max(F, 1), _dptr(E),
                            st.ctypes.data_as(ctypes.POINTER(ctypes.c_double))
                            if st is not None else None,
                            so, ss, sd, nthreads,
                            s0.ctypes.data_as(ctypes.POINTER(ctypes.c_double))
                            if s0 is not None else None)
    if rc != 0:
        raise ValueError(f"oracle_forward failed ({rc})")
    return (E, st) if want_state else E


def vjp(ops, n, params, inputs, grad_out, nthreads=0, psi0=None):
    """(dparams [B,P], dinputs [B,F], E [B,n]) in float64 for cotangent grad_out
    (psi0: initial states as in forward)."""
    lib = _load()
    params = np.asarray(params)
    inputs = np.asarray(inputs)
    B = params.shape[0]
    P = params.shape[1]
    F = inputs.shape[1]
    p = _as2d(params, B, P)
    x = _as2d(inputs, B, F)
    g = np.ascontiguousarray(np.asarray(grad_out, dtype=np.float64).reshape(B, n))
    dp = np.zeros((B, max(P, 1)), dtype=np.float64)
    dx = np.zeros((B, max(F, 1)), dtype=np.float64)
    E = np.zeros((B, n), dtype=np.float64)
    rec = encode_ops(ops)
    s0 = _psi0(psi0, B, n)
    rc = lib.oracle_vjp(rec.ctypes.data, len(ops), n, B, _dptr(p), max(P, 1), _dptr(x),
                        max(F, 1), _dptr(g), _dptr(dp), _dptr(dx), _dptr(E), nthreads,
                        s0.ctypes.data_as(ctypes.POINTER(ctypes.c_double))
                        if s0 is not None else None)
    if rc != 0:
        raise ValueError(f"oracle_vjp failed ({rc})")
    return dp[:, :P], dx[:, :F], E


def _occurrences(ops):
    """(gate, slot, source, index, mul) of every non-constant angle."""
    for k, op in enumerate(ops):
        for s, spec in enumerate(op.angles):
            if spec[0] != "const":
                yield k, s, spec[0], int(spec[1]), float(spec[2]) if len(spec) > 2 else 1.0


def probabilities(ops, n, params, inputs, psi0=None, nthreads=0):
    """Basis-state probabilities |Psi_k|^2 [B, 2^n] of the final state: the
    other output the execute phase offers besides <Z> (Sec. 3)."""
    _, st = forward(ops, n, params, inputs, want_state=True, nthreads=nthreads, psi0=psi0)
    return np.abs(st) ** 2


def _shift_grad(ops, n, params, inputs, grad_out, delta, coef, psi0=None):
    params = np.asarray(params)
    inputs = np.asarray(inputs)
    B = params.shape[0]
    g = np.asarray(grad_out, dtype=np.float64).reshape(B, n)
    dp = np.zeros((B, params.shape[1]))
    dx = np.zeros((B, inputs.shape[1]))
    for k, s, src, idx, mul in _occurrences(ops):
        ep = forward(ops, n, params, inputs, shift=(k, s, +delta), psi0=psi0)
        em = forward(ops, n, params, inputs, shift=(k, s, -delta), psi0=psi0)
        d = mul * coef * np.sum(g * (ep - em), axis=1)  # chain rule through the affine angle
        (dp if src == "param" else dx)[:, idx] += d
    return dp, dx


def param_shift_grad(ops, n, params, inputs, grad_out, psi0=None):
    """Two-term parameter-shift rule per angle occurrence, summed per slot:
    d f / d t = [f(t + pi/2) - f(t - pi/2)] / 2, exact when the angle enters as
    exp(-i t G) with G of two eigenvalues 1/2 apart up to a shared offset (the
    Pauli rotations, R_PP, P, CP, and the Euler angles of U3 / U2 / ROT) -- not
    for the controlled rotations, whose generator has three eigenvalues."""
    return _shift_grad(ops, n, params, inputs, grad_out, np.pi / 2, 0.5, psi0)


def fd_grad(ops, n, params, inputs, grad_out, h=1e-5, psi0=None):
    """Central finite differences per angle occurrence, summed per slot."""
    return _shift_grad(ops, n, params, inputs, grad_out, h, 0.5 / h, psi0)


def loss_cotangent(kind: str, E: np.ndarray, y=None) -> np.ndarray:
    """d loss / d E for the workload objectives (float64).

    sum       : L = sum_b sum_i E[b,i]                   -> g = 1
    mean      : L = sum_b mean_i E[b,i]                  -> g = 1/n
                (the paper's shared objective, the mean of single-qubit <Z>,
                 taken per sample)
    mse_z0    : L = mean_b (E[b,0] - y_b)^2              -> g[b,0] = 2 (E[b,0]-y_b)/B
    mse_meanz : L = mean_b (mean_i E[b,i] - y_b)^2       -> g[b,i] = 2 (s_b-y_b)/(n B)
    """
    E = np.asarray(E, dtype=np.float64)
    B, n = E.shape
    g = np.zeros_like(E)
    if kind == "sum":
        g[:] = 1.0
    elif kind == "mean":
        g[:] = 1.0 / n
    elif kind == "mse_z0":
        g[:, 0] = 2.0 * (E[:, 0] - np.asarray(y, dtype=np.float64)) / B
    elif kind == "mse_meanz":
        s = E.mean(axis=1)
        g[:] = (2.0 * (s - np.asarray(y, dtype=np.float64)) / (n * B))[:, None]
    else:
        raise ValueError(kind)
    return g
