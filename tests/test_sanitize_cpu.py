"""Host code under AddressSanitizer and UndefinedBehaviorSanitizer (no GPU).

1. The library's host-only code -- compile-phase validation and lowering, the
   stream and register-tile planners, the kernel source generator, the
   OpenQASM front end and the C ABI's argument checks -- built with g++
   -fsanitize=address,undefined into tests/sanitize/host_harness.cpp, which
   drives it with seeded random gate lists (valid and malformed, device = -1)
   and seeded mutations of generated OpenQASM programs.
2. The oracle's C code built the same way and called through its Python
   binding on random circuits over every gate kind, with and without Psi_0.
Any sanitizer report fails the test (halt_on_error, leaks included for the
harness).  No HIP call is made: the device launchers are stubs that abort.
"""
import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2607_11985_amd", "csrc")
SAN = ["-fsanitize=address,undefined", "-fno-omit-frame-pointer", "-fno-sanitize-recover=all",
       "-g", "-O1"]
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")


def _run(cmd, env=None, timeout=600):
    p = subprocess.run(cmd, capture_output=True, text=True, env=env, timeout=timeout)
    assert p.returncode == 0, f"{' '.join(cmd[:3])}... rc {p.returncode}\n{p.stdout[-3000:]}\n{p.stderr[-6000:]}"
    return p


def _env(extra):
    env = dict(os.environ)
    env.update(extra)
    return env


@pytest.fixture(scope="module")
def harness(tmp_path_factory):
    from paper_2607_11985_amd.build import BUILD, write_embedded_headers
    # a directory of this test process's own (pytest's temporary directories,
    # outside the repository): parallel test workers must not overwrite an
    # executable another one runs
    out = str(tmp_path_factory.mktemp("sanitize"))
    os.makedirs(BUILD, exist_ok=True)
    srcs = [os.path.join(ROOT, "tests", "sanitize", "host_harness.cpp"),
            write_embedded_headers()] + \
        [os.path.join(CSRC, f) for f in ("api.cpp", "planner.cpp", "qasm.cpp", "jit.cpp",
                                         "jit_compile.cpp")]
    flags = ["g++", "-std=c++17", "-D__HIP_PLATFORM_AMD__", "-I", os.path.join(ROCM, "include"),
             "-I", os.path.join(ROOT, "include"), "-I", CSRC] + SAN

    def obj(src):
        o = os.path.join(out, os.path.basename(src) + ".o")
        _run(flags + ["-c", src, "-o", o])
        return o

    with ThreadPoolExecutor(max_workers=min(6, os.cpu_count() or 1)) as ex:
        objs = list(ex.map(obj, srcs))
    exe = os.path.join(out, "host_harness")
    _run(["g++"] + SAN + objs + ["-L", os.path.join(ROCM, "lib"),
                                 "-Wl,-rpath," + os.path.join(ROCM, "lib"), "-lamdhip64",
                                 "-lhiprtc", "-o", exe])
    return exe


@pytest.mark.parametrize("seed", [1, 2])
def test_host_library_under_sanitizers(harness, seed):
    p = _run([harness, str(seed), "250", "1500"],
             env=_env({"ASAN_OPTIONS": "detect_leaks=1:abort_on_error=1",
                       "UBSAN_OPTIONS": "halt_on_error=1:print_stacktrace=1"}))
    assert "0 failures" in p.stdout, p.stdout


ORACLE_SCRIPT = r"""
import sys
import numpy as np
sys.path.insert(0, sys.argv[1])
import oracle
from paper_2607_11985_amd import workloads as W
oracle._lib = oracle.open_library(sys.argv[2])
for n in (1, 3, 5, 7):
    ops, P, F = W.random_circuit(n, 40, seed=900 + n, kinds=W.GENERAL_KINDS, p_affine=0.3)
    p, x = W.random_inputs(3, P, F, seed=901 + n)
    g = W.random_cotangent(3, n, seed=902 + n)
    E, st = oracle.forward(ops, n, p, x, want_state=True)
    dp, dx, E2 = oracle.vjp(ops, n, p, x, g)
    s0 = W.random_states(3, n, seed=903 + n)
    E3 = oracle.forward(ops, n, p, x, psi0=s0)
    dp3, dx3, _ = oracle.vjp(ops, n, p, x, g, psi0=s0)
    Es = oracle.forward(ops, n, p, x, shift=(0, 0, 0.25))
    assert all(np.all(np.isfinite(a)) for a in (E, st, dp, dx, E2, E3, dp3, dx3, Es))
    assert np.allclose(E, E2)
print("oracle ok")
"""


def test_oracle_under_sanitizers(tmp_path):
    lib = str(tmp_path / "liboracle_san.so")
    _run(["gcc", "-std=c99", "-fopenmp", "-fPIC", "-shared"] + SAN +
         ["-o", lib, os.path.join(ROOT, "oracle", "vqc_oracle.c"), "-lm"])
    asan = subprocess.run(["gcc", "-print-file-name=libasan.so"], capture_output=True,
                          text=True).stdout.strip()
    p = _run([sys.executable, "-c", ORACLE_SCRIPT, ROOT, lib],
             env=_env({"LD_PRELOAD": asan, "ASAN_OPTIONS": "detect_leaks=0:abort_on_error=1",
                       "UBSAN_OPTIONS": "halt_on_error=1:print_stacktrace=1",
                       "OMP_NUM_THREADS": "2"}))
    assert "oracle ok" in p.stdout
