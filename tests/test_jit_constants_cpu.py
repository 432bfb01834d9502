"""Host logic of the generated kernels' compiled-in constants: the angle
occurrence records (source, index, mul, add; or cos, sin of a constant angle)
that the kernel generator writes as runs of compares, or as a table when the
circuit has many runs.  The generated source is read back (the compile check
writes it on the host, no GPU) and its records are checked against the gate
list."""
import math
import os
import re

import numpy as np
import pytest

from paper_2607_11985_amd import _lib
from paper_2607_11985_amd import workloads as W

SRC = {"param": 0, "input": 1, "const": 2}


def generated_source(tmp_path, ops, n, P, F):
    os.environ["VQC_JIT_DUMP"] = str(tmp_path)
    try:
        rc, h = _lib.vqc_compile_raw(_lib.encode_ops(ops), len(ops), n, P, F,
                                     _lib.vqc_compile_opts(device=-1))
        assert rc == 0, _lib.vqc_last_error()
        _lib.vqc_jit_check(h)
        _lib.vqc_destroy(h)
    finally:
        del os.environ["VQC_JIT_DUMP"]
    return (tmp_path / "vqc_rf.hip").read_text()


def occ_records(text, nocc):
    body = text[text.index("static OccRec occ("):]
    body = body[:body.index("\n}\n")]
    if "static constexpr OccRec t[]" in body:
        items = re.findall(r"\{(-?\d+), (-?\d+), ([-0-9a-fx.p+]+)f, ([-0-9a-fx.p+]+)f\}", body)
        return "table", [(int(s), int(i), float.fromhex(a), float.fromhex(b))
                         for s, i, a, b in items[:nocc]]
    runs = re.findall(r"(?:if \(o < (\d+)\) )?r = OccRec\{(-?\d+), ([^,]+), "
                      r"([-0-9a-fx.p+]+)f, ([-0-9a-fx.p+]+)f\};", body)
    recs = []
    for o in range(nocc):
        for end, s, idx, a, b in runs:
            if end == "" or o < int(end):
                m = re.fullmatch(r"o \+ (-?\d+)", idx)
                recs.append((int(s), o + int(m.group(1)) if m else int(idx),
                             float.fromhex(a), float.fromhex(b)))
                break
    return "runs", recs


def test_runs_of_layers(tmp_path):
    """Shared-angle layers (one affine parameter per layer), per-qubit
    parameters and scaled inputs: nine runs, encoded as compares."""
    n = 8
    ops, want = [], []
    for l in range(3):
        mul, add = float(np.float32(1.5 - l)), float(np.float32(0.25 * l))
        ops += [W.Op("RX", (q,), (("param", l, mul, add),)) for q in range(n)]
        want += [(0, l, mul, add)] * n
        ops += [W.Op("RY", (q,), (("param", 3 + l * n + q),)) for q in range(n)]
        want += [(0, 3 + l * n + q, 1.0, 0.0) for q in range(n)]
        ops += [W.Op("CNOT", (q, (q + 1) % n)) for q in range(n)]
        ops += [W.Op("RZ", (q,), (("input", q, -2.0, 0.0),)) for q in range(n)]
        want += [(1, q, -2.0, 0.0) for q in range(n)]
    form, recs = occ_records(generated_source(tmp_path, ops, n, 3 + 3 * n, n), len(want))
    assert form == "runs"
    assert recs == want


def test_many_runs_use_a_table(tmp_path):
    """Constant angles interleaved with parameters and inputs: each constant
    is a run of its own, so the records go to a table; constants carry their
    cos and sin of the half angle."""
    n, ops, want = 3, [], []
    rng = np.random.default_rng(5)
    for k in range(30):
        q = k % n
        kind = ("RX", "RY", "RZ")[k % 3]
        if k % 3 == 0:
            ops.append(W.Op(kind, (q,), (("param", k),)))
            want.append((0, k, None))
        elif k % 3 == 1:
            v = float(np.float32(rng.uniform(-3, 3)))
            ops.append(W.Op(kind, (q,), (("const", v),)))
            want.append((2, None, v))
        else:
            ops.append(W.Op(kind, (q,), (("input", k % 4),)))
            want.append((1, k % 4, None))
    form, recs = occ_records(generated_source(tmp_path, ops, n, 30, 4), len(want))
    assert form == "table" and len(recs) == len(want)
    for (s, i, a, b), (ws, wi, v) in zip(recs, want):
        assert s == ws
        if ws == 2:
            assert abs(a - math.cos(v / 2)) < 1e-6 and abs(b - math.sin(v / 2)) < 1e-6
        else:
            assert i == wi and (a, b) == (1.0, 0.0)
