"""Seeded synthetic workloads: circuit structures and input draws.

This module describes *what* is simulated -- the gate lists of the five
synthetic circuit families and the seeded float32 draws that feed them -- and
holds none of the simulation arithmetic.  It is the only code shared by the
HIP path and the double-precision oracle: both receive the same gate list and
the same float32 arrays from here.

Gate-list format (a plain, backend-neutral description of a static circuit,
Sec. 3 "Static Circuit Scope": gate identity and wiring are fixed, only the
angles vary at run time):

    Op(kind, wires, angles)
      kind   : "RX" | "RY" | "RZ" | "ROT" | "CNOT" | "CZ"
      wires  : (q,) for one-qubit kinds; (control, target) for CNOT;
               (a, b) for CZ
      angles : one entry per angle slot (1 for RX/RY/RZ, 3 for ROT as
               (phi, theta, omega), none for CNOT/CZ); each entry is
               ("param", p) | ("input", f) | ("const", value)

Readings of the paper used here (the paper does not fix them):
  * qubit j is bit j of the basis index (little-endian);
  * ROT(phi, theta, omega) is RZ(omega) RY(theta) RZ(phi), phi applied first;
  * inside a layer all one-qubit gates come first (qubit 0..n-1, each qubit's
    gates in the listed order), then the entanglers;
  * CNOT rings are CNOT(i, (i+r) mod n) for i = 0..n-1 in ascending order;
  * parameter layout: two-angle layers p = (l*n + i)*2 + s, three-angle
    (ROT) layers p = (l*n + i)*3 + s; encoded input f = qubit index.
"""
from __future__ import annotations

import math
from dataclasses import dataclass
from typing import List, Sequence, Tuple

import numpy as np

SEED_BASE = 260711985

KINDS = ("RX", "RY", "RZ", "ROT", "CNOT", "CZ")
# the general static gate set: kind -> (wires, angles).  Structure only (the
# generators draw circuits over it); what each gate computes is not here.
GATE_SHAPES = {
    "RX": (1, 1), "RY": (1, 1), "RZ": (1, 1), "ROT": (1, 3), "CNOT": (2, 0), "CZ": (2, 0),
    "ID": (1, 0), "X": (1, 0), "Y": (1, 0), "Z": (1, 0), "H": (1, 0), "S": (1, 0),
    "SDG": (1, 0), "T": (1, 0), "TDG": (1, 0), "SX": (1, 0), "SXDG": (1, 0),
    "P": (1, 1), "U2": (1, 2), "U3": (1, 3),
    "CY": (2, 0), "CH": (2, 0), "SWAP": (2, 0), "CRX": (2, 1), "CRY": (2, 1), "CRZ": (2, 1),
    "CP": (2, 1), "RXX": (2, 1), "RYY": (2, 1), "RZZ": (2, 1),
    "CCX": (3, 0), "CSWAP": (3, 0),
}
GENERAL_KINDS = tuple(GATE_SHAPES)
N_ANGLES = {k: v[1] for k, v in GATE_SHAPES.items()}


@dataclass(frozen=True)
class Op:
    """One gate: kind, wires (controls first), angle specs.  An angle spec is
    ("const", value), or (src, index) / (src, index, mul, add) with src in
    {"param", "input"}, meaning mul * value + add."""
    kind: str
    wires: Tuple[int, ...]
    angles: Tuple[tuple, ...] = ()


@dataclass
class Workload:
    """One seeded problem instance: circuit plus float32 inputs."""
    name: str
    n_qubits: int
    ops: List[Op]
    n_params: int
    n_inputs: int
    params: np.ndarray      # float32 [B, P]
    inputs: np.ndarray      # float32 [B, F]
    y: np.ndarray | None    # float32 [B] regression target, or None
    loss: str               # "sum" | "mean" | "mse_z0" | "mse_meanz"
    description: str

    @property
    def batch(self) -> int:
        return int(self.params.shape[0])


# ---------------------------------------------------------------- structures

def _encoding(n: int, kind: str = "RY") -> List[Op]:
    return [Op(kind, (i,), (("input", i),)) for i in range(n)]


def _ring(n: int, r: int = 1) -> List[Op]:
    return [Op("CNOT", (i, (i + r) % n)) for i in range(n)]


def hea_circuit(n: int, layers: int) -> Tuple[List[Op], int, int]:
    """RY(x_i) encoding, then `layers` x [RY(a), RZ(b) per qubit; CNOT ring]."""
    ops = _encoding(n)
    for l in range(layers):
        for i in range(n):
            base = (l * n + i) * 2
            ops.append(Op("RY", (i,), (("param", base + 0),)))
            ops.append(Op("RZ", (i,), (("param", base + 1),)))
        ops += _ring(n, 1)
    return ops, 2 * layers * n, n


def strongly_entangling_circuit(n: int, layers: int) -> Tuple[List[Op], int, int]:
    """RY(x_i) encoding, then `layers` x [ROT per qubit; CNOT(i,(i+r)%n)],
    with range r = (l mod (n-1)) + 1 for 0-based layer l."""
    ops = _encoding(n)
    for l in range(layers):
        for i in range(n):
            base = (l * n + i) * 3
            ops.append(Op("ROT", (i,), (("param", base), ("param", base + 1),
                                         ("param", base + 2))))
        r = (l % (n - 1)) + 1 if n > 1 else 0
        if n > 1:
            ops += _ring(n, r)
    return ops, 3 * layers * n, n


def reupload_circuit(n: int, layers: int) -> Tuple[List[Op], int, int]:
    """Data re-uploading: `layers` x [RX(x_i), RY(a), RZ(b) per qubit; CZ(i,i+1)
    for i = 0..n-2 (no wrap)].  x_i is re-used in every layer."""
    ops: List[Op] = []
    for l in range(layers):
        for i in range(n):
            base = (l * n + i) * 2
            ops.append(Op("RX", (i,), (("input", i),)))
            ops.append(Op("RY", (i,), (("param", base + 0),)))
            ops.append(Op("RZ", (i,), (("param", base + 1),)))
        ops += [Op("CZ", (i, i + 1)) for i in range(n - 1)]
    return ops, 2 * layers * n, n


def rot_ring_circuit(n: int, layers: int) -> Tuple[List[Op], int, int]:
    """RY(x_i) encoding, then `layers` x [ROT per qubit; CNOT ring r=1]."""
    ops = _encoding(n)
    for l in range(layers):
        for i in range(n):
            base = (l * n + i) * 3
            ops.append(Op("ROT", (i,), (("param", base), ("param", base + 1),
                                         ("param", base + 2))))
        ops += _ring(n, 1)
    return ops, 3 * layers * n, n


# ----------------------------------------------------------------- configs

CONFIGS = {
    1: dict(name="c1_hea_n4", n=4, B=64, builder=hea_circuit, layers=2,
            x=("uniform", -math.pi, math.pi), p=("uniform", 0.0, 2 * math.pi),
            y=None, loss="sum",
            description="n=4, B=64: RY encoding; 2 layers RY,RZ + CNOT ring; "
                        "gradient of sum <Z_i>"),
    2: dict(name="c2_hea_n8", n=8, B=1024, builder=hea_circuit, layers=4,
            x=("uniform", -math.pi, math.pi), p=("uniform", 0.0, 2 * math.pi),
            y=None, loss="mean",
            description="n=8, B=1024: RY encoding; 4 layers RY,RZ + CNOT ring; "
                        "gradient of mean <Z_i>"),
    3: dict(name="c3_strongly_entangling_n12", n=12, B=4096,
            builder=strongly_entangling_circuit, layers=6,
            x=("uniform", -math.pi, math.pi), p=("uniform", 0.0, 2 * math.pi),
            y=("uniform", -1.0, 1.0), loss="mse_z0",
            description="n=12, B=4096: RY encoding; 6 strongly-entangling "
                        "layers (ROT + CNOT range r); MSE(<Z_0>, y)"),
    4: dict(name="c4_reupload_n14", n=14, B=8192, builder=reupload_circuit,
            layers=10, x=("uniform", -math.pi, math.pi),
            p=("normal", 0.0, 0.1), y=("uniform", -1.0, 1.0),
            loss="mse_meanz",
            description="n=14, B=8192: 10 re-uploading layers RX(x),RY,RZ + CZ "
                        "chain; MSE(sum<Z_i>/14, y)"),
    5: dict(name="c5_rot_ring_n16", n=16, B=256, builder=rot_ring_circuit,
            layers=8, x=("uniform", -math.pi, math.pi),
            p=("uniform", 0.0, 2 * math.pi), y=None, loss="mean",
            description="n=16, B=256: RY encoding; 8 layers ROT + CNOT ring; "
                        "gradient of mean <Z_i>"),
}


def _draw(rng: np.random.Generator, spec, shape) -> np.ndarray:
    kind, a, b = spec
    if kind == "uniform":
        v = rng.uniform(a, b, size=shape)
    elif kind == "normal":
        v = rng.normal(a, b, size=shape)
    else:
        raise ValueError(kind)
    return v.astype(np.float64).astype(np.float32)


def make_config(idx: int, batch: int | None = None) -> Workload:
    """Build configuration `idx` (1..5) with its seeded float32 inputs.

    Draw order: inputs [B,F], then params [B,P] (row-major, i.e. in the
    parameter-layout order within each row), then y [B] when the loss needs
    it.  All draws are float64 rounded to float32.  `batch` overrides B; a
    smaller batch gives the leading rows of a *different* stream, so sampled
    checks of the full configuration should slice the full arrays instead.
    """
    c = CONFIGS[idx]
    B = c["B"] if batch is None else int(batch)
    ops, P, F = c["builder"](c["n"], c["layers"])
    rng = np.random.default_rng(SEED_BASE + idx)
    x = _draw(rng, c["x"], (B, F))
    p = _draw(rng, c["p"], (B, P))
    y = _draw(rng, c["y"], (B,)) if c["y"] is not None else None
    return Workload(name=c["name"], n_qubits=c["n"], ops=ops, n_params=P,
                    n_inputs=F, params=p, inputs=x, y=y, loss=c["loss"],
                    description=c["description"])


def random_cotangent(batch: int, n: int, seed: int) -> np.ndarray:
    """Seeded cotangent g ~ U(-1, 1) of shape [B, n] (float32)."""
    rng = np.random.default_rng(seed)
    return rng.uniform(-1.0, 1.0, size=(batch, n)).astype(np.float32)


def random_circuit(n: int, n_ops: int, seed: int, n_params: int = 0,
                   n_inputs: int = 0, kinds: Sequence[str] = KINDS,
                   p_const: float = 0.1, p_affine: float = 0.0) -> Tuple[List[Op], int, int]:
    """A seeded random static circuit over `kinds` (structure only).

    Angle sources are drawn among params, inputs and constants; parameters
    and inputs may be re-used by several gates.  With p_affine > 0 that share
    of the non-constant angles gets a random (mul, add) (float32 values, mul
    in +-[0.25, 2]).  Returns (ops, P, F) with P, F at least 1 so that every
    array is non-empty.
    """
    rng = np.random.default_rng(seed)
    P = max(1, n_params or n_ops)
    F = max(1, n_inputs or n)
    ops: List[Op] = []
    kinds = [k for k in kinds if GATE_SHAPES[k][0] <= n]
    for _ in range(n_ops):
        k = kinds[int(rng.integers(len(kinds)))]
        nw, na = GATE_SHAPES[k]
        if nw == 1:
            wires = (int(rng.integers(n)),)
        else:
            wires = tuple(int(v) for v in rng.choice(n, size=nw, replace=False))
        ang = []
        for _s in range(na):
            u = rng.random()
            if u < p_const:
                ang.append(("const", float(np.float32(rng.uniform(-4, 4)))))
                continue
            src = "input" if u < 0.5 else "param"
            idx = int(rng.integers(F if src == "input" else P))
            if p_affine > 0 and rng.random() < p_affine:
                mul = float(np.float32(rng.choice([-1.0, 1.0]) * rng.uniform(0.25, 2.0)))
                add = float(np.float32(rng.uniform(-3.0, 3.0)))
                ang.append((src, idx, mul, add))
            else:
                ang.append((src, idx))
        ops.append(Op(k, wires, tuple(ang)))
    return ops, P, F


def random_inputs(batch: int, n_params: int, n_inputs: int, seed: int):
    """Seeded float32 params ~ U(0, 2pi) [B,P] and inputs ~ U(-pi, pi) [B,F]."""
    rng = np.random.default_rng(seed)
    x = _draw(rng, ("uniform", -math.pi, math.pi), (batch, n_inputs))
    p = _draw(rng, ("uniform", 0.0, 2 * math.pi), (batch, n_params))
    return p, x


def random_states(batch: int, n: int, seed: int, kind: str = "haar") -> np.ndarray:
    """Seeded initial states [B, 2^n] complex64 (the optional Psi_0).

    haar   : complex Gaussian amplitudes scaled to unit norm (Haar-random pure
             states), norm taken in float64 before rounding to complex64
    basis  : |k_b> with k_b uniform in [0, 2^n)
    sparse : a unit-norm state on 4 random basis states (peaked probabilities)
    """
    rng = np.random.default_rng(seed)
    N = 1 << n
    if kind == "basis":
        s = np.zeros((batch, N), dtype=np.complex128)
        s[np.arange(batch), rng.integers(0, N, size=batch)] = 1.0
    elif kind == "sparse":
        s = np.zeros((batch, N), dtype=np.complex128)
        for b in range(batch):
            idx = rng.choice(N, size=min(4, N), replace=False)
            s[b, idx] = rng.normal(size=len(idx)) + 1j * rng.normal(size=len(idx))
        s /= np.linalg.norm(s, axis=1, keepdims=True)
    else:
        s = rng.normal(size=(batch, N)) + 1j * rng.normal(size=(batch, N))
        s /= np.linalg.norm(s, axis=1, keepdims=True)
    return s.astype(np.complex64)


def count_ops(ops: Sequence[Op]):
    """(rotation primitives, entanglers, ops) -- ROT counts as 3 primitives."""
    rot = sum(N_ANGLES[o.kind] for o in ops)
    ent = sum(1 for o in ops if GATE_SHAPES[o.kind][0] > 1)
    return rot, ent, len(ops)
