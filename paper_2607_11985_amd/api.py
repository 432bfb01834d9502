"""Torch-facing wrapper of the C ABI: device memory and streams come from torch,
every computation runs in libvqc.so.

    circ = Circuit(ops, n_qubits, n_params, n_inputs)
    E = VQCFunction.apply(circ, params, inputs)      # params/inputs: cuda fp32
    E.sum().backward()                                # adjoint-method gradients
"""
from __future__ import annotations

import torch

from . import _lib

_PATHS = {"auto": _lib.VQC_PATH_AUTO, "resident": _lib.VQC_PATH_RESIDENT,
          "stream": _lib.VQC_PATH_STREAM}
_ENGINES = {"jit": _lib.VQC_ENGINE_JIT, "interp": _lib.VQC_ENGINE_INTERP}


def _ptr(t):
    return None if t is None else t.data_ptr()


def _stream(device):
    return torch.cuda.current_stream(device).cuda_stream


def _as_rows(x, batch, width, device, name):
    if width == 0:
        return None
    if x is None:
        raise ValueError(f"{name} is required (width {width})")
    if x.dtype != torch.float32 or x.device != device or not x.is_contiguous():
        raise ValueError(f"{name} must be a contiguous float32 tensor on {device}")
    if tuple(x.shape) != (batch, width):
        raise ValueError(f"{name} must have shape {(batch, width)}, got {tuple(x.shape)}")
    return x


class Circuit:
    """A compiled static circuit (compile once, execute many: Sec. 3)."""

    def __init__(self, ops, n_qubits: int, n_params: int, n_inputs: int, device: int = 0,
                 path: str = "auto", reg_bits: int = 0, engine: str = "jit",
                 shared_params: bool = False, tile_qubits: int = 0):
        self.ops = list(ops)
        self.n = int(n_qubits)
        self.P = int(n_params)
        self.F = int(n_inputs)
        self.shared = bool(shared_params)
        self.device = torch.device("cuda", device)
        self.handle = _lib.vqc_compile(self.ops, self.n, self.P, self.F, device=device,
                                       path=_PATHS[path], reg_bits=reg_bits,
                                       engine=_ENGINES[engine], shared_params=int(self.shared),
                                       tile_qubits=tile_qubits)

    @classmethod
    def from_qasm(cls, source: str, inputs=(), device: int = 0, path: str = "auto",
                  reg_bits: int = 0, engine: str = "jit", shared_params: bool = False):
        """Compile an OpenQASM program (vqc_compile_qasm).  `inputs`: names of the
        declared inputs that are data features; the other declared inputs are
        trainable parameters, in declaration order."""
        self = cls.__new__(cls)
        names = ",".join(inputs) if inputs else None
        self.handle = _lib.vqc_compile_qasm(source, names, device=device, path=_PATHS[path],
                                            reg_bits=reg_bits, engine=_ENGINES[engine],
                                            shared_params=int(bool(shared_params)))
        info = _lib.vqc_circuit_info(self.handle)
        self.ops = None
        self.n = info["n_qubits"]
        self.P = info["n_params"]
        self.F = info["n_inputs"]
        self.shared = bool(shared_params)
        self.device = torch.device("cuda", device)
        return self

    def _params(self, params, B):
        """Per-sample rows [B, P], or the shared vector [P]."""
        if not self.shared:
            return _as_rows(params, B, self.P, self.device, "params")
        if self.P == 0:
            return None
        return _as_rows(params.reshape(1, -1), 1, self.P, self.device, "params").reshape(-1)

    def _batch(self, params, inputs):
        if inputs is not None and (self.shared or params is None):
            return int(inputs.shape[0])
        return int(params.shape[0])

    def __del__(self):
        h = getattr(self, "handle", None)
        if h is not None and _lib._lib is not None:
            _lib.vqc_destroy(h)
            self.handle = None

    def info(self) -> dict:
        return _lib.vqc_circuit_info(self.handle)

    def workspace_bytes(self, batch: int, training: bool = True) -> int:
        return _lib.vqc_workspace_bytes(self.handle, batch, int(training))

    def new_workspace(self, batch: int, training: bool = True):
        nb = self.workspace_bytes(batch, training)
        return torch.empty(max(nb, 1), dtype=torch.uint8, device=self.device), nb

    def forward(self, params, inputs, training: bool = False, workspace=None, out=None):
        """E [B, n]; with training=True also the workspace for backward()."""
        B = self._batch(params, inputs)
        params = self._params(params, B)
        inputs = _as_rows(inputs, B, self.F, self.device, "inputs")
        E = out if out is not None else torch.empty((B, self.n), dtype=torch.float32,
                                                   device=self.device)
        ws, nb = None, 0
        if training or self.workspace_bytes(B, False) > 0:
            if workspace is None:
                workspace, nb = self.new_workspace(B, training)
            else:
                nb = workspace.numel()
            ws = workspace
        _lib.vqc_forward(self.handle, B, _ptr(params), _ptr(inputs), E.data_ptr(), _ptr(ws),
                         nb, _stream(self.device))
        return (E, ws) if training else E

    def forward_ex(self, params, inputs, psi0=None, expvals: bool = True, probs: bool = False,
                   training: bool = False, workspace=None):
        """(E or None, probabilities or None[, workspace]) from the initial states
        psi0 [B, 2^n] complex64 (default |0...0>)."""
        B = self._batch(params, inputs) if (params is not None or inputs is not None) \
            else int(psi0.shape[0])
        params = self._params(params, B)
        inputs = _as_rows(inputs, B, self.F, self.device, "inputs")
        if psi0 is not None:
            if psi0.dtype != torch.complex64 or psi0.device != self.device or \
                    not psi0.is_contiguous() or tuple(psi0.shape) != (B, 1 << self.n):
                raise ValueError(f"psi0 must be a contiguous complex64 tensor of shape "
                                 f"{(B, 1 << self.n)} on {self.device}")
        E = torch.empty((B, self.n), dtype=torch.float32, device=self.device) if expvals else None
        pr = torch.empty((B, 1 << self.n), dtype=torch.float32, device=self.device) \
            if probs else None
        ws, nb = None, 0
        if training or self.workspace_bytes(B, False) > 0:
            if workspace is None:
                workspace, nb = self.new_workspace(B, training)
            else:
                nb = workspace.numel()
            ws = workspace
        _lib.vqc_forward_ex(self.handle, B, _ptr(params), _ptr(inputs), _ptr(psi0), _ptr(E),
                            _ptr(pr), _ptr(ws), nb, _stream(self.device))
        return (E, pr, ws) if training else (E, pr)

    def backward(self, params, inputs, grad_out, workspace, dparams=None, dinputs=None):
        """Per-sample gradients (dparams [B,P], dinputs [B,F]) of sum(grad_out * E)."""
        B = int(grad_out.shape[0])
        params = self._params(params, B)
        inputs = _as_rows(inputs, B, self.F, self.device, "inputs")
        grad_out = _as_rows(grad_out, B, self.n, self.device, "grad_out")
        if dparams is None:
            shape = (self.P,) if self.shared else (B, self.P)
            dparams = torch.empty(shape, dtype=torch.float32, device=self.device)
        if dinputs is None:
            dinputs = torch.empty((B, self.F), dtype=torch.float32, device=self.device)
        _lib.vqc_backward(self.handle, B, _ptr(params), _ptr(inputs), grad_out.data_ptr(),
                          workspace.data_ptr(), workspace.numel(),
                          dparams.data_ptr() if self.P else None,
                          dinputs.data_ptr() if self.F else None, _stream(self.device))
        return dparams, dinputs


    def train_step(self, params, inputs, loss: str, y=None, workspace=None, want_cot=False):
        """Forward, loss cotangent and adjoint gradients in one call.

        Returns (E, dparams, dinputs), plus the cotangent g when want_cot."""
        B = self._batch(params, inputs)
        params = self._params(params, B)
        inputs = _as_rows(inputs, B, self.F, self.device, "inputs")
        if y is not None:
            y = _as_rows(y.reshape(B, 1), B, 1, self.device, "y")
        E = torch.empty((B, self.n), dtype=torch.float32, device=self.device)
        g = torch.empty_like(E) if want_cot else None
        dparams = torch.empty((self.P,) if self.shared else (B, self.P), dtype=torch.float32,
                              device=self.device)
        dinputs = torch.empty((B, self.F), dtype=torch.float32, device=self.device)
        nb = _lib.vqc_workspace_bytes(self.handle, B, 2)
        if workspace is None and nb > 0:
            workspace = torch.empty(nb, dtype=torch.uint8, device=self.device)
        _lib.vqc_train_step(self.handle, B, _ptr(params), _ptr(inputs), _lib.LOSS[loss], _ptr(y),
                            E.data_ptr(), _ptr(g), dparams.data_ptr() if self.P else None,
                            dinputs.data_ptr() if self.F else None, _ptr(workspace),
                            workspace.numel() if workspace is not None else 0,
                            _stream(self.device))
        return (E, dparams, dinputs, g) if want_cot else (E, dparams, dinputs)


    def fd_backward(self, params, inputs, grad_out, h: float = 1e-2):
        """Central-difference gradients (the paper's FD mode)."""
        B = int(grad_out.shape[0])
        params = self._params(params, B)
        inputs = _as_rows(inputs, B, self.F, self.device, "inputs")
        grad_out = _as_rows(grad_out, B, self.n, self.device, "grad_out")
        dparams = torch.empty((self.P,) if self.shared else (B, self.P), dtype=torch.float32,
                              device=self.device)
        dinputs = torch.empty((B, self.F), dtype=torch.float32, device=self.device)
        nb = _lib.vqc_workspace_bytes(self.handle, B, 3)
        ws = torch.empty(max(nb, 1), dtype=torch.uint8, device=self.device)
        _lib.vqc_fd_backward(self.handle, B, _ptr(params), _ptr(inputs), grad_out.data_ptr(),
                             float(h), ws.data_ptr(), nb, dparams.data_ptr() if self.P else None,
                             dinputs.data_ptr() if self.F else None, _stream(self.device))
        return dparams, dinputs


def loss_grad(kind: str, E, y=None, out=None):
    """Cotangent dL/dE of a scalar objective, computed on the GPU."""
    B, n = E.shape
    g = out if out is not None else torch.empty_like(E)
    _lib.vqc_loss_grad(_lib.LOSS[kind], B, n, E.data_ptr(), _ptr(y), g.data_ptr(),
                       _stream(E.device))
    return g


class VQCFunction(torch.autograd.Function):
    """E = circuit(params, inputs) with adjoint-method backward."""

    @staticmethod
    def forward(ctx, circuit: Circuit, params, inputs):
        E, ws = circuit.forward(params, inputs, training=True)
        ctx.circuit = circuit
        ctx.ws = ws
        ctx.save_for_backward(params, inputs)
        return E

    @staticmethod
    def backward(ctx, gE):
        params, inputs = ctx.saved_tensors
        dp, dx = ctx.circuit.backward(params, inputs, gE.contiguous(), ctx.ws)
        return None, dp, dx
