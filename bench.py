"""Throughput of the batched VQC hot path on one MI355X.

One step = one pass of the whole hot path over one batch of synthetic input:
forward (every gate, <Z>), the workload's loss-head cotangent, and the adjoint
sweep (gradients for every parameter and input), on one HIP stream with the
inputs resident in HBM.  By default a step is one vqc_train_step call (a single
launch on the resident path: the state never leaves the chip); --separate
times vqc_forward + vqc_loss_grad + vqc_backward instead, and those calls'
timings are reported beside the step either way.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--config 1..5]

Prints one JSON line.  value = circuit evaluations (forward E + full
gradient) per second = B * K / timed seconds, the K steps bracketed by events.
The dominant kernel is timed again as K back-to-back launches for the
roofline.  Every timed step's outputs are checked bit for bit against the
first one, and the fused step against the separate calls.
"""
from __future__ import annotations

import argparse
import json
import os
import platform
import subprocess
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "circuit evals/sec (fwd+adjoint grad) at n=4..16; % of LDS/HBM BW peak"
CSRC = os.path.join(ROOT, "paper_2607_11985_amd", "csrc")
PROFILES = os.path.join(ROOT, "profiles")
PEAK_FP32_TFLOPS = 157.3     # MI355X fp32 vector peak (packed FMA, 256 CU x 2.4 GHz)
PEAK_HBM_GBS = 8000.0        # MI355X HBM3E
DEFAULT_CONFIG = 2


def algorithmic_flops(w):
    """Per-sample flops of the method (gate by gate), forward and backward.

    forward : every rotation updates each amplitude with a 2x2 whose entries are
              c, s or c +- i s: 6 flops per amplitude; <Z_j> needs |a|^2 (3) and
              one signed add per qubit (n) per amplitude.
    backward: lambda = H psi costs n + 2 per amplitude; every rotation costs
              4 per amplitude for Im<lambda|P|psi> plus 6 on each of psi and
              lambda to un-apply it (16).  CNOT and CZ are data movement (0).
    """
    from paper_2607_11985_amd import workloads as W
    R, _, _ = W.count_ops(w.ops)
    N = float(1 << w.n_qubits)
    n = w.n_qubits
    return N * (6 * R + 3 + n), N * (16 * R + n + 2)


def cpu_baseline(w, budget_s=12.0):
    """The oracle as it stands (forward, loss cotangent, VJP) on host cores,
    on a bounded sample of the same workload."""
    import oracle
    rows_total = w.batch
    chunk = max(1, min(rows_total, 64 if w.n_qubits <= 10 else 8 if w.n_qubits <= 12 else 2))
    done, t0, start = 0, time.perf_counter(), 0
    while time.perf_counter() - t0 < budget_s:
        sel = slice(start, start + chunk)
        E = oracle.forward(w.ops, w.n_qubits, w.params[sel], w.inputs[sel])
        ycut = w.y[sel] if w.y is not None else None
        g = oracle.loss_cotangent(w.loss, E, ycut)
        if w.loss in ("mse_z0", "mse_meanz"):
            g *= E.shape[0] / w.batch  # the objective averages over the whole batch
        oracle.vjp(w.ops, w.n_qubits, w.params[sel], w.inputs[sel], g)
        done += E.shape[0]
        start = (start + chunk) % rows_total
    dt = time.perf_counter() - t0
    cores = int(os.environ.get("OMP_NUM_THREADS", os.cpu_count() or 1))
    return {"value": done / dt, "unit": "circuit evals/s", "cores": cores, "kind": "oracle",
            "sample": f"{done} samples of {w.name} (rows taken cyclically in chunks of {chunk}), "
                      f"{dt:.1f} s, forward + loss cotangent + VJP in complex128"}


def kernel_source_hash():
    """Hash of the HIP/C++ sources; traffic counters taken on other sources are stale."""
    import hashlib
    h = hashlib.sha256()
    for name in sorted(os.listdir(CSRC)):
        if name.endswith((".hip", ".cpp", ".h")):
            with open(os.path.join(CSRC, name), "rb") as f:
                h.update(name.encode() + f.read())
    return h.hexdigest()[:16]


def measured_traffic(workload, kernel):
    """HBM bytes per launch from the committed counter record, or None when the
    record is missing or was taken on different kernel sources."""
    path = os.path.join(PROFILES, f"traffic_{workload}.json")
    try:
        with open(path) as f:
            rec = json.load(f)
    except (OSError, ValueError):
        return None
    if rec.get("source_hash") != kernel_source_hash():
        return None
    k = rec.get("kernels", {}).get(kernel)
    return None if k is None else k.get("bytes_per_launch")


def copy_calibration(size_mib=1024, reps=10):
    """A plain device-to-device copy of known size, for scaling the HBM counters."""
    import torch
    n = size_mib << 20
    src = torch.empty(n, dtype=torch.uint8, device="cuda")
    dst = torch.empty_like(src)
    src.fill_(1)
    torch.cuda.synchronize()
    for _ in range(reps):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_bytes_read": n, "copy_bytes_written": n, "reps": reps}), flush=True)


def cpu_model():
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return platform.processor()


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--config", type=int, default=DEFAULT_CONFIG, choices=[1, 2, 3, 4, 5])
    ap.add_argument("--engine", default="jit", choices=["jit", "interp"],
                    help="kernels generated for the circuit (jit) or the precompiled "
                         "schedule interpreter (interp)")
    ap.add_argument("--reg-bits", type=int, default=0,
                    help="amplitudes per thread = 2^reg_bits (0: the library's default)")
    ap.add_argument("--tile-qubits", type=int, default=0,
                    help="streaming tile size, 12, 13 or 14 (0: the library's default)")
    ap.add_argument("--graph", action="store_true",
                    help="time HIP graph replays of the step instead of its launches")
    ap.add_argument("--separate", action="store_true",
                    help="time vqc_forward + vqc_loss_grad + vqc_backward instead of "
                         "vqc_train_step")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-budget", type=float, default=12.0)
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run a 1 GiB device copy (counter calibration) and exit")
    args = ap.parse_args()
    if args.copy_calibration:
        copy_calibration()
        return
    if args.gpus != 1:
        print(json.dumps({"error": "this engine runs on one GPU: samples are independent, so a "
                          "multi-GPU run would shard the batch with no communication; "
                          "run with --gpus 1"}))
        sys.exit(2)

    import torch
    from paper_2607_11985_amd import _lib, workloads as W
    from paper_2607_11985_amd.api import Circuit

    if not os.path.exists(_lib.LIB_PATH):
        from paper_2607_11985_amd.build import build_library
        build_library()
    assert torch.cuda.is_available(), "bench.py needs a GPU"
    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)
    w = W.make_config(args.config)
    B, n = w.batch, w.n_qubits
    t0 = time.time()
    circ = Circuit(w.ops, n, w.n_params, w.n_inputs, device=0, engine=args.engine,
                   reg_bits=args.reg_bits, tile_qubits=args.tile_qubits)
    compile_s = time.time() - t0
    info = circ.info()
    p = torch.from_numpy(w.params).to(dev)
    x = torch.from_numpy(w.inputs).to(dev)
    y = torch.from_numpy(w.y).to(dev) if w.y is not None else None
    E = torch.empty((B, n), dtype=torch.float32, device=dev)
    g = torch.empty_like(E)
    dp = torch.empty((B, w.n_params), dtype=torch.float32, device=dev)
    dx = torch.empty((B, w.n_inputs), dtype=torch.float32, device=dev)
    ws, nb = circ.new_workspace(B, training=True)
    nb_step = circ.workspace_bytes(B, 2)
    ws_step = torch.empty(max(nb_step, 1), dtype=torch.uint8, device=dev)
    stream = torch.cuda.current_stream(dev)
    s = stream.cuda_stream
    h = circ.handle
    loss_kind = _lib.LOSS[w.loss]
    pp, xp, yp = p.data_ptr(), x.data_ptr(), (y.data_ptr() if y is not None else None)
    dpp = dp.data_ptr() if w.n_params else None
    dxp = dx.data_ptr() if w.n_inputs else None

    def fwd(st):
        _lib.vqc_forward(h, B, pp, xp, E.data_ptr(), ws.data_ptr(), nb, st)

    def loss(st):
        _lib.vqc_loss_grad(loss_kind, B, n, E.data_ptr(), yp, g.data_ptr(), st)

    def bwd(st):
        _lib.vqc_backward(h, B, pp, xp, g.data_ptr(), ws.data_ptr(), nb, dpp, dxp, st)

    def separate(st):
        fwd(st); loss(st); bwd(st)

    def fused(st):
        _lib.vqc_train_step(h, B, pp, xp, loss_kind, yp, E.data_ptr(), g.data_ptr(), dpp, dxp,
                            ws_step.data_ptr() if nb_step else None, nb_step, st)

    step = separate if args.separate else fused

    def ev():
        return torch.cuda.Event(enable_timing=True)

    def back_to_back(call, K):
        """Average duration of K launches of `call` issued back to back."""
        e0, e1 = ev(), ev()
        e0.record(stream)
        for _ in range(K):
            call(s)
        e1.record(stream)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / K

    K = args.steps
    for _ in range(args.warmup):
        separate(s)
    torch.cuda.synchronize()
    ref = [t.clone() for t in (E, g, dp, dx)]
    for _ in range(args.warmup):
        fused(s)
    torch.cuda.synchronize()
    # the fused step reproduces the separate calls (up to the compiler's rounding)
    dev_max = max(float((t - r).abs().max()) if t.numel() else 0.0
                  for t, r in zip((E, g, dp, dx), ref))
    if dev_max > 1e-4:
        raise SystemExit(f"training step differs from the separate calls by {dev_max}")

    # separate calls, each bracketed by events (includes host launch gaps)
    evs = [[ev() for _ in range(4)] for _ in range(K)]
    torch.cuda.synchronize()
    for k in range(K):
        e = evs[k]
        e[0].record(stream); fwd(s)
        e[1].record(stream); loss(s)
        e[2].record(stream); bwd(s)
        e[3].record(stream)
    torch.cuda.synchronize()
    fwd_ms = float(np.mean([e[0].elapsed_time(e[1]) for e in evs]))
    loss_ms = float(np.mean([e[1].elapsed_time(e[2]) for e in evs]))
    bwd_ms = float(np.mean([e[2].elapsed_time(e[3]) for e in evs]))
    separate_ms = back_to_back(separate, K)

    # the timed region: K steps
    use_graph = args.graph
    if use_graph:
        graph = torch.cuda.CUDAGraph()
        cap = torch.cuda.Stream(device=dev)  # default priority
        cap.wait_stream(stream)
        with torch.cuda.graph(graph, stream=cap):
            step(cap.cuda_stream)
        stream.wait_stream(cap)
        torch.cuda.synchronize()
    step(s)
    torch.cuda.synchronize()
    ref = [t.clone() for t in (E, g, dp, dx)]
    t_start, t_end = ev(), ev()
    torch.cuda.synchronize()
    t_start.record(stream)
    for _ in range(K):
        if use_graph:
            graph.replay()
        else:
            step(s)
    t_end.record(stream)
    torch.cuda.synchronize()
    total_ms = t_start.elapsed_time(t_end)
    ms_per_step = total_ms / K
    value = B * K / (total_ms / 1e3)
    for t, r in zip((E, g, dp, dx), ref):
        if not torch.equal(t, r):
            raise SystemExit("a timed step differs from the first one")

    # the dominant kernel: the one-launch training step on the resident path,
    # else the adjoint (all of its passes), timed as K back-to-back launches
    f_fwd, f_bwd = algorithmic_flops(w)
    resident = info["path"] == 1
    if resident and not args.separate:
        dominant, dom_ms, flops_sample = "train_step", back_to_back(fused, K), f_fwd + f_bwd
    elif bwd_ms >= fwd_ms:
        dominant, dom_ms, flops_sample = "backward", back_to_back(bwd, K), f_bwd
    else:
        dominant, dom_ms, flops_sample = "forward", back_to_back(fwd, K), f_fwd

    # forward-only rate (inference, no state saved), outside the timed region
    inf_ms = back_to_back(lambda st: circ.forward(p, x, out=E), K)

    flops = flops_sample * B
    achieved = flops / (dom_ms / 1e3) / 1e12
    if args.engine == "jit":
        kname = {(1, "train_step"): "vqc_rs", (1, "forward"): "vqc_rf", (1, "backward"): "vqc_rb",
                 (2, "forward"): "vqc_sf*", (2, "backward"): "vqc_sb*"}[(info["path"], dominant)]
    else:
        kname = ("stream_kernel" if info["path"] == 2 else
                 "resident_step_kernel" if dominant == "train_step" else "resident_kernel")
    kname += f" ({dominant}, all passes)" if info["path"] == 2 else f" ({dominant})"
    roofline = {"bound": "alu", "kernel": kname, "achieved": achieved,
                "peak": PEAK_FP32_TFLOPS, "unit": "TFLOP/s", "frac": achieved / PEAK_FP32_TFLOPS,
                "traffic": measured_traffic(w.name, dominant),
                "flops_per_launch": flops, "avg_launch_ms": dom_ms,
                "source_hash": kernel_source_hash()}

    out = {
        "metric": METRIC, "value": value, "unit": "circuit evals/s", "n_gpus": 1,
        "steps": K, "warmup": args.warmup, "ms_per_step": ms_per_step,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "c64",
        "data": "synthetic (seeded draws of the configuration; no dataset)",
        "config": {"workload": w.name, "description": w.description, "n_qubits": n, "batch": B,
                   "n_params": w.n_params, "n_inputs": w.n_inputs, "ops": len(w.ops),
                   "loss": w.loss, "path": "resident" if info["path"] == 1 else "stream",
                   "threads_per_workgroup": info["threads"], "engine": args.engine,
                   "reg_bits": args.reg_bits or "default",
                   "tile_qubits": circ.info()["tile_qubits"] if circ.info()["path"] == 2 else None,
                   "compile_s": round(compile_s, 2),
                   "exchanges_fwd_bwd": [info["fwd_exchanges"], info["bwd_exchanges"]]},
        "step": ("vqc_forward + vqc_loss_grad + vqc_backward" if args.separate else
                 "vqc_train_step"),
        "timing": "hip graph replays of the step" if use_graph else "launches on one stream",
        "separate_calls_ms_per_step": separate_ms,
        "kernel_ms": {"forward_train": fwd_ms, "loss_grad": loss_ms, "backward": bwd_ms,
                      "forward_inference": inf_ms, f"{dominant}_back_to_back": dom_ms},
        "forward_only_evals_per_s": B / (inf_ms / 1e3),
        "roofline": roofline,
        "env": {"torch": torch.__version__, "hip": getattr(torch.version, "hip", None),
                "gpu": torch.cuda.get_device_name(dev), "host_cpu": cpu_model(),
                "host_cores": os.cpu_count()},
    }
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(w, args.cpu_budget)
        out["gpu_over_cpu"] = value / out["cpu_baseline"]["value"]
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
