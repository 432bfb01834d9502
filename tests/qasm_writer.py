"""Test-side OpenQASM writer and gate-record decoder (host logic only).

to_qasm() renders a gate list of the workload format as an OpenQASM 3 program:
the parameters as `input array[float[32], P] theta`, the data features as
`input array[float[32], F] x`, affine angles as `mul * name[i] + add`.  The
tests feed the text to the library's front end and the gate list itself to
the oracle, so the two never share a parse.
"""
import numpy as np

QASM_NAME = {
    "RX": "rx", "RY": "ry", "RZ": "rz", "CNOT": "cx", "CZ": "cz", "ID": "id", "X": "x", "Y": "y",
    "Z": "z", "H": "h", "S": "s", "SDG": "sdg", "T": "t", "TDG": "tdg", "SX": "sx", "SXDG": "sxdg",
    "P": "p", "U2": "u2", "U3": "u3", "CY": "cy", "CH": "ch", "SWAP": "swap", "CRX": "crx",
    "CRY": "cry", "CRZ": "crz", "CP": "cp", "RXX": "rxx", "RYY": "ryy", "RZZ": "rzz",
    "CCX": "ccx", "CSWAP": "cswap", "ROT": "rot",
}
KIND_OF_CODE = ("RX", "RY", "RZ", "ROT", "CNOT", "CZ", "ID", "X", "Y", "Z", "H", "S", "SDG", "T",
                "TDG", "SX", "SXDG", "P", "U2", "U3", "CY", "CH", "SWAP", "CRX", "CRY", "CRZ",
                "CP", "RXX", "RYY", "RZZ", "CCX", "CSWAP")
ARITY = {"CNOT": 2, "CZ": 2, "CY": 2, "CH": 2, "SWAP": 2, "CRX": 2, "CRY": 2, "CRZ": 2, "CP": 2,
         "RXX": 2, "RYY": 2, "RZZ": 2, "CCX": 3, "CSWAP": 3}
N_ANG = {"RX": 1, "RY": 1, "RZ": 1, "P": 1, "CRX": 1, "CRY": 1, "CRZ": 1, "CP": 1, "RXX": 1,
         "RYY": 1, "RZZ": 1, "U2": 2, "ROT": 3, "U3": 3}


def _num(v):
    return repr(float(np.float32(v)))


def _angle(spec):
    if spec[0] == "const":
        return _num(spec[1])
    name = "theta" if spec[0] == "param" else "x"
    mul = spec[2] if len(spec) > 2 else 1.0
    add = spec[3] if len(spec) > 3 else 0.0
    text = f"{name}[{int(spec[1])}]"
    if mul != 1.0:
        text = f"{_num(mul)} * {text}"
    if add != 0.0:
        text = f"{text} + {_num(add)}" if add > 0 else f"{text} - {_num(-add)}"
    return text


def to_qasm(ops, n, P, F, version=3):
    lines = ["OPENQASM 3.0;" if version == 3 else "OPENQASM 2.0;",
             'include "stdgates.inc";' if version == 3 else 'include "qelib1.inc";']
    lines.append(f"qubit[{n}] q;" if version == 3 else f"qreg q[{n}];")
    lines.append(f"input array[float[32], {max(P, 1)}] theta;")
    lines.append(f"input array[float[32], {max(F, 1)}] x;")
    if any(o.kind == "ROT" for o in ops):
        lines.append("gate rot(a, b, c) w { rz(a) w; ry(b) w; rz(c) w; }")
    for o in ops:
        args = ", ".join(_angle(s) for s in o.angles)
        wires = ", ".join(f"q[{w}]" for w in o.wires)
        name = QASM_NAME[o.kind]
        lines.append(f"{name}({args}) {wires};" if o.angles else f"{name} {wires};")
    return "\n".join(lines) + "\n"


def decode(arr, n_ops):
    """vqc_op records -> [(kind, wires, angles)] with angles as in the workload
    format (("const", v) or (src, idx, mul, add))."""
    out = []
    for k in range(n_ops):
        r = arr[k]
        kind = KIND_OF_CODE[r.kind]
        wires = tuple(int(r.wires[i]) for i in range(ARITY.get(kind, 1)))
        ang = []
        for s in range(N_ANG.get(kind, 0)):
            if r.src[s] == 2:
                ang.append(("const", float(r.val[s])))
            else:
                ang.append(("param" if r.src[s] == 0 else "input", int(r.idx[s]), float(r.mul[s]),
                            float(r.val[s])))
        out.append((kind, wires, tuple(ang)))
    return out


def normalize(ops):
    """Workload ops in the decoded form (float32-rounded values)."""
    out = []
    for o in ops:
        ang = []
        for s in o.angles:
            if s[0] == "const":
                ang.append(("const", float(np.float32(s[1]))))
            else:
                mul = s[2] if len(s) > 2 else 1.0
                add = s[3] if len(s) > 3 else 0.0
                ang.append((s[0], int(s[1]), float(np.float32(mul)), float(np.float32(add))))
        out.append((o.kind, tuple(o.wires), tuple(ang)))
    return out
