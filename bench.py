"""Throughput of the batched VQC hot path on one MI355X.

One step = one pass of the whole hot path over one batch of synthetic input:
forward (the circuit's gates, the state after every qubit's leading rotations
built as a product, gates that change no output left out; <Z>), the
workload's loss-head cotangent, and the adjoint sweep (gradients for every
parameter and input), on one HIP stream with the inputs resident in HBM.  A step is one vqc_train_step call (a single launch on
the resident path: the state never leaves the chip; the streaming passes
otherwise); --separate times vqc_forward + vqc_loss_grad + vqc_backward.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--config 0..5]

--config 0 (the default) measures all five workloads in one run and prints ONE
JSON line whose headline is the 16-qubit workload (the largest n of the metric,
the HBM-streaming path); every workload's own record sits under "configs".
--config k measures only workload k.

Per workload: W untimed warmup steps, then exactly K steps bracketed by
synchronisations and HIP events (value = B K / seconds); then at least five
more brackets of K' >= K steps (each >= 0.2 s) for mean, std and median; the
step is also timed as back-to-back launches for the roofline; every timed step
is compared bit for bit with the first one.  Outside the timed regions the
oracle runs on the host's cores on a bounded sample of rows (cpu_baseline),
and those rows of the timed step's outputs are compared with it.
"""
from __future__ import annotations

import argparse
import json
import math
import os
import platform
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
HEADLINE = 5                 # the 16-qubit streaming workload
E_TOL, G_REL, G_FLOOR = 1e-5, 1e-4, 1e-6   # the parity bars of the tests


# ----------------------------------------------------------- algorithmic work

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


def io_bytes(w):
    """Per-sample HBM bytes every step moves besides states: params, inputs and
    the target read; E, the cotangent and both gradients written (fp32)."""
    P, F, n = w.n_params, w.n_inputs, w.n_qubits
    return 4 * (P + F + (1 if w.y is not None else 0) + 2 * n + P + F)


def state_rw_per_sample(info):
    """State reads + writes (in units of one 2^n complex64 state) of one streaming
    training step.  Forward: the first pass only writes (it starts from
    |0...0>), every later pass reads and writes psi (each pass's output is
    kept).  Adjoint (one pass per forward pass, in reverse): the first reads
    psi_G and writes lambda, the middle ones read the state their forward pass
    saved and lambda and write lambda, the last reads both and stores nothing;
    a single pass only reads psi_G.  The training step runs the passes of its own
    plan when the circuit has heads (first pass: the product state)."""
    nf, nb = info["fwd_passes"], info["bwd_passes"]
    if info.get("step_fwd_passes"):
        nf, nb = info["step_fwd_passes"], info["step_bwd_passes"]
    fwd = 1 + 2 * (nf - 1)
    adj = 1 if nb == 1 else 2 + 3 * (nb - 2) + 2
    return fwd + adj


def algorithmic_bytes(w, info, B):
    """HBM bytes of one training step (the unit of the roofline)."""
    per = io_bytes(w)
    if info["path"] == 2:
        per += state_rw_per_sample(info) * (1 << w.n_qubits) * 8
    return per * B


# ----------------------------------------------------------- counter records

def kernel_source_hash():
    """Hash of the HIP/C++ sources; counters taken on other sources are stale."""
    import hashlib
    h = hashlib.sha256()
    for name in sorted(os.listdir(CSRC)):
        if name.endswith((".hip", ".cpp", ".h")) and name != "probes.hip":
            with open(os.path.join(CSRC, name), "rb") as f:
                h.update(name.encode() + f.read())
    return h.hexdigest()[:16]


def measured_traffic(workload, B):
    """HBM bytes per step from the committed counter record (FETCH_SIZE and
    WRITE_SIZE, scaled by the copy calibration), or None when the record is
    missing, was taken at another batch or on different kernel sources."""
    path = os.path.join(PROFILES, f"traffic_{workload}.json")
    try:
        with open(path) as f:
            rec = json.load(f)
    except (OSError, ValueError):
        return None
    if rec.get("source_hash") != kernel_source_hash() or rec.get("batch") != B:
        return None
    return rec.get("step_bytes")


# ----------------------------------------------------------- calibration, probes

def copy_calibration(size_mib=1024, reps=10):
    """A plain device-to-device copy of known size, for scaling the HBM counters."""
    import torch
    n = size_mib << 20
    src = torch.empty(n, dtype=torch.uint8, device="cuda")
    dst = torch.empty_like(src)
    src.fill_(1)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        dst.copy_(src)
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / reps
    print(json.dumps({"copy_bytes_read": n, "copy_bytes_written": n, "reps": reps,
                      "ms_per_copy": ms, "copy_GBps": 2 * n / ms / 1e6}), flush=True)


def run_probe(kind, reps=10):
    """Peak microbenchmarks (csrc/probes.hip, built into libvqc_probes.so): the
    FMA issue ceiling of this build (packed FP32 off) and the LDS read bandwidth
    with 16- and 4-byte loads, timed with HIP events on torch's stream."""
    import ctypes
    import torch
    from paper_2607_11985_amd.build import PROBES
    lib = ctypes.CDLL(PROBES)
    lib.vqc_probe_fma.argtypes = [ctypes.c_void_p, ctypes.c_int, ctypes.c_int, ctypes.c_void_p]
    lib.vqc_probe_lds.argtypes = [ctypes.c_void_p, ctypes.c_int, ctypes.c_int, ctypes.c_int,
                                  ctypes.c_void_p]
    lib.vqc_probe_work.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_int]
    lib.vqc_probe_work.restype = ctypes.c_double
    blocks = 256 * 8  # eight 256-thread workgroups per CU
    out = torch.empty(blocks * 256, dtype=torch.float32, device="cuda")
    stream = torch.cuda.current_stream()
    s = stream.cuda_stream
    res = {"probe": kind, "blocks": blocks, "threads": 256}
    cases = [("fma", 0, 4096, 0)] if kind == "fma" else [("lds128", 1, 8192, 16),
                                                        ("lds32", 1, 16384, 4)]
    for name, k, iters, width in cases:
        def launch():
            rc = (lib.vqc_probe_fma(out.data_ptr(), blocks, iters, s) if k == 0 else
                  lib.vqc_probe_lds(out.data_ptr(), blocks, iters, width, s))
            if rc:
                raise RuntimeError(f"probe launch failed: {rc}")
        launch()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(reps):
            launch()
        e1.record(stream)
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / reps
        work = lib.vqc_probe_work(k, blocks, iters, width)
        if k == 0:
            res[name] = {"ms": ms, "TFLOPs": work / ms / 1e9,
                         "frac_of_157.3": work / ms / 1e9 / PEAK_FP32_TFLOPS}
        else:
            res[name] = {"ms": ms, "TBps": work / ms / 1e9,
                         "bytes_per_clk_per_CU_at_2.4GHz": work / (ms / 1e3) / 256 / 2.4e9}
    print(json.dumps(res), flush=True)


# ----------------------------------------------------------- the oracle leg

def cpu_baseline(w, gpu_out, budget_s):
    """The oracle as it stands (forward, loss cotangent, VJP) on the host's cores,
    on a bounded sample of rows of the same workload (rows taken cyclically in
    chunks, one OpenMP thread per row); the rows it computes are compared with
    the timed step's outputs (E, cotangent, dparams, dinputs) at the tests' bars."""
    import oracle
    rows_total = w.batch
    cores = int(os.environ.get("OMP_NUM_THREADS", os.cpu_count() or 1))
    chunk = max(1, min(rows_total, 64 if w.n_qubits <= 10 else cores))
    done, start = 0, 0
    seen = {}
    t0 = time.perf_counter()
    while True:
        sel = np.arange(start, min(start + chunk, rows_total))
        E = oracle.forward(w.ops, w.n_qubits, w.params[sel], w.inputs[sel])
        ycut = w.y[sel] if w.y is not None else None
        g = oracle.loss_cotangent(w.loss, E, ycut)
        if w.loss in ("mse_z0", "mse_meanz"):
            g *= E.shape[0] / w.batch  # the objective averages over the whole batch
        dp, dx, _ = oracle.vjp(w.ops, w.n_qubits, w.params[sel], w.inputs[sel], g)
        done += len(sel)
        for i, b in enumerate(sel):
            if int(b) not in seen:
                seen[int(b)] = (E[i], g[i], dp[i], dx[i])
        start = 0 if sel[-1] + 1 >= rows_total else int(sel[-1]) + 1
        if time.perf_counter() - t0 >= budget_s:
            break
    dt = time.perf_counter() - t0
    rec = {"value": done / dt, "unit": "circuit evals/s", "cores": cores, "kind": "oracle",
           "sample": f"{done} samples of {w.name} (rows cyclically in chunks of {chunk}), "
                     f"{dt:.1f} s, forward + loss cotangent + VJP in complex128"}
    rec["parity"] = parity_of(w, gpu_out, seen)
    return rec


def parity_of(w, gpu_out, seen):
    """Errors of the timed step's rows against the oracle rows (the bars of the
    tests: E within 1e-5; gradient rows within 1e-4 of their max-norm plus the
    floor, plus, for an MSE head, the effect of the cotangent's own error)."""
    rows = sorted(seen)
    E, g, dp, dx = (t[rows].astype(np.float64) for t in gpu_out)
    Er = np.stack([seen[b][0] for b in rows])
    gr = np.stack([seen[b][1] for b in rows])
    dpr = np.stack([seen[b][2] for b in rows])
    dxr = np.stack([seen[b][3] for b in rows])
    kmax = 0.0
    tot = {}
    for o in w.ops:
        for a in o.angles:
            if a[0] != "const":
                tot[(a[0], a[1])] = tot.get((a[0], a[1]), 0.0) + (abs(a[2]) if len(a) > 2 else 1)
    kmax = max(tot.values()) if tot else 0.0
    allow = 0.0 if w.loss in ("sum", "mean") else kmax * 2 * E_TOL / w.batch

    def row_rel(a, ref):
        if a.size == 0:
            return 0.0, True
        err = np.max(np.abs(a - ref), axis=1)
        scale = np.max(np.abs(ref), axis=1)
        bar = G_REL * scale + G_FLOOR * np.sum(np.abs(gr), axis=1) + allow
        return float(np.max(err / np.maximum(scale, 1e-30))), bool(np.all(err <= bar))

    e_err = float(np.max(np.abs(E - Er)))
    g_err = float(np.max(np.abs(g - gr)))
    both, ok_b = row_rel(np.concatenate([dp, dx], 1), np.concatenate([dpr, dxr], 1))
    rp, ok_p = row_rel(dp, dpr)
    rx, ok_x = row_rel(dx, dxr)
    ok = e_err <= E_TOL and ok_b and ok_p and ok_x
    return {"rows": len(rows), "E_abs_max": e_err, "cot_abs_max": g_err,
            "grad_row_rel_max": both, "dparams_row_rel_max": rp, "dinputs_row_rel_max": rx,
            "within_bars": ok}


# ----------------------------------------------------------- one workload

def measure(idx, args, torch, dev, want_cpu, cpu_budget):
    from paper_2607_11985_amd import _lib, workloads as W
    from paper_2607_11985_amd.api import Circuit

    w = W.make_config(idx, batch=args.batch or None)
    B, n = w.batch, w.n_qubits
    t0 = time.time()
    circ = Circuit(w.ops, n, w.n_params, w.n_inputs, device=dev.index, engine=args.engine,
                   reg_bits=args.reg_bits, tile_qubits=args.tile_qubits,
                   path=args.path)
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

    def timed(call, K):
        """Milliseconds of K calls issued back to back, bracketed by events."""
        torch.cuda.synchronize()
        e0, e1 = ev(), ev()
        e0.record(stream)
        for _ in range(K):
            call(s)
        e1.record(stream)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1)

    K, Wm = args.steps, args.warmup
    for _ in range(max(Wm, 1)):
        separate(s)
    torch.cuda.synchronize()
    ref = [t.clone() for t in (E, g, dp, dx)]
    for _ in range(max(Wm, 1)):
        fused(s)
    torch.cuda.synchronize()
    # the fused step reproduces the separate calls up to rounding (it builds the
    # heads' state as a product where the separate calls run their gates)
    dev_max = max(float((t - r).abs().max()) if t.numel() else 0.0
                  for t, r in zip((E, g, dp, dx), ref))
    if dev_max > 1e-5:
        raise SystemExit(f"{w.name}: training step differs from the separate calls by {dev_max}")
    for _ in range(Wm):
        step(s)
    torch.cuda.synchronize()
    graph = None
    if args.graph:
        # one step captured into a HIP graph, then timed as replays
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            step(torch.cuda.current_stream(dev).cuda_stream)
        torch.cuda.synchronize()
        step = lambda st: graph.replay()  # noqa: E731
        for _ in range(max(Wm, 1)):
            step(s)
        torch.cuda.synchronize()
    first = [t.clone() for t in (E, g, dp, dx)]

    # ---- the timed region: exactly K steps
    total_ms = timed(step, K)
    ms_per_step = total_ms / K
    value = B * K / (total_ms / 1e3)
    for t, r in zip((E, g, dp, dx), first):
        if not torch.equal(t, r):
            raise SystemExit(f"{w.name}: a timed step differs from the first one")
    gpu_out = [t.cpu().numpy() for t in (E, g, dp, dx)]

    # ---- repeats: >= 5 brackets of K' >= K steps, each >= 0.2 s (--repeats 0:
    # none, for profiler runs)
    Kr = max(K, int(math.ceil(0.2 / max(ms_per_step / 1e3, 1e-9)))) if args.repeats else K
    rates = []
    for _ in range(max(args.repeats, 5) if args.repeats else 0):
        ms = timed(step, Kr)
        rates.append(B * Kr / (ms / 1e3))
    for t, r in zip((E, g, dp, dx), first):
        if not torch.equal(t, r):
            raise SystemExit(f"{w.name}: a repeated step differs from the first one")
    rates = np.array(rates) if rates else np.array([value, value])

    # ---- per-call times of the separate calls (events around each call)
    Kc = max(3, min(K, 50))
    evs = [[ev() for _ in range(4)] for _ in range(Kc)]
    torch.cuda.synchronize()
    for k in range(Kc):
        e = evs[k]
        e[0].record(stream); fwd(s)
        e[1].record(stream); loss(s)
        e[2].record(stream); bwd(s)
        e[3].record(stream)
    torch.cuda.synchronize()
    fwd_ms = float(np.mean([e[0].elapsed_time(e[1]) for e in evs]))
    loss_ms = float(np.mean([e[1].elapsed_time(e[2]) for e in evs]))
    bwd_ms = float(np.mean([e[2].elapsed_time(e[3]) for e in evs]))
    inf_ms = timed(lambda st: circ.forward(p, x, out=E), Kc) / Kc

    # ---- roofline of the step: back-to-back steps on the bench's stream
    Kb = max(K, Kr)
    step_ms = timed(step, Kb) / Kb
    f_fwd, f_bwd = algorithmic_flops(w)
    flops = (f_fwd + f_bwd) * B
    abytes = algorithmic_bytes(w, info, B)
    alu = flops / (step_ms / 1e3) / 1e12
    hbm = abytes / (step_ms / 1e3) / 1e9
    alu_frac, hbm_frac = alu / PEAK_FP32_TFLOPS, hbm / PEAK_HBM_GBS
    resident = info["path"] == 1
    if args.engine == "jit":
        head = info["step_head_rotations"] > 0  # the step's own plan (product head)
        kname = "vqc_rs (one launch)" if resident else (
            ("vqc_ht, vqc_hf*, reduce_e_loss, vqc_hb*, vqc_hg" if head else
             "vqc_st, vqc_sf*, reduce_e_loss, vqc_sb*, reduce_grad")
            + " (one step: each batch half on its own stream)")
    else:
        kname = "resident_step_kernel" if resident else \
            "stream_kernel passes (one step: each batch half on its own stream)"
    if args.separate:
        kname = "vqc_forward + vqc_loss_grad + vqc_backward (one step)"
    if hbm_frac >= alu_frac:
        roof = {"bound": "hbm", "achieved": hbm, "peak": PEAK_HBM_GBS, "unit": "GB/s",
                "frac": hbm_frac}
    else:
        roof = {"bound": "alu", "achieved": alu, "peak": PEAK_FP32_TFLOPS, "unit": "TFLOP/s",
                "frac": alu_frac}
    roof.update({"traffic": measured_traffic(w.name, B), "kernel": kname,
                 "avg_launch_ms": step_ms, "bytes_per_launch": abytes,
                 "flops_per_launch": flops,
                 "hbm": {"achieved_GBps": hbm, "peak_GBps": PEAK_HBM_GBS, "frac": hbm_frac},
                 "alu": {"achieved_TFLOPs": alu, "peak_TFLOPs": PEAK_FP32_TFLOPS,
                         "frac": alu_frac},
                 "source_hash": kernel_source_hash()})

    rec = {
        "workload": w.name, "description": w.description, "n_qubits": n, "batch": B,
        "n_params": w.n_params, "n_inputs": w.n_inputs, "ops": len(w.ops), "loss": w.loss,
        "path": "resident" if resident else "stream",
        "threads_per_workgroup": info["threads"], "engine": args.engine,
        "tile_qubits": info["tile_qubits"] if not resident else None,
        "passes_fwd_bwd": [info["fwd_passes"], info["bwd_passes"]],
        "step_head_rotations": info["step_head_rotations"],
        "exchanges_fwd_bwd": [info["fwd_exchanges"], info["bwd_exchanges"]],
        "compile_s": round(compile_s, 2),
        "value": value, "ms_per_step": ms_per_step, "steps": K,
        "repeats": {"brackets": len(rates), "steps_per_bracket": Kr,
                    "mean": float(rates.mean()), "std": float(rates.std(ddof=1)),
                    "median": float(np.median(rates))},
        "kernel_ms": {"forward_train": fwd_ms, "loss_grad": loss_ms, "backward": bwd_ms,
                      "forward_inference": inf_ms, "step_back_to_back": step_ms},
        "forward_only_evals_per_s": B / (inf_ms / 1e3),
        "roofline": roof,
    }
    del ws, ws_step
    if want_cpu:
        rec["cpu_baseline"] = cpu_baseline(w, gpu_out, cpu_budget)
        rec["gpu_over_cpu"] = value / rec["cpu_baseline"]["value"]
    return rec


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
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--config", type=int, default=0, choices=[0, 1, 2, 3, 4, 5],
                    help="0: all five workloads, headline the 16-qubit one")
    ap.add_argument("--batch", type=int, default=0,
                    help="override the workload's batch (e.g. 1024 for the 16-qubit "
                         "workload to overflow the 256 MB Infinity Cache)")
    ap.add_argument("--repeats", type=int, default=5,
                    help="repeat brackets for mean/std/median (at least 5; 0 = none)")
    ap.add_argument("--engine", default="jit", choices=["jit", "interp"])
    ap.add_argument("--path", default="auto", choices=["auto", "resident", "stream"])
    ap.add_argument("--reg-bits", type=int, default=0)
    ap.add_argument("--tile-qubits", type=int, default=0)
    ap.add_argument("--separate", action="store_true",
                    help="time vqc_forward + vqc_loss_grad + vqc_backward")
    ap.add_argument("--graph", action="store_true",
                    help="time replays of one step captured into a HIP graph")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-budget", type=float, default=5.0,
                    help="seconds of oracle work per workload (twice that for the headline)")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run a 1 GiB device copy (counter calibration) and exit")
    ap.add_argument("--probe", choices=["fma", "lds"],
                    help="only run a peak microbenchmark and exit")
    args = ap.parse_args()
    if args.gpus != 1:
        print(json.dumps({"error": "this engine runs on one GPU: samples are independent, so a "
                          "multi-GPU run would shard the batch with no communication; "
                          "run with --gpus 1"}))
        sys.exit(2)
    if args.copy_calibration:
        copy_calibration()
        return
    if args.probe:
        run_probe(args.probe)
        return

    import torch
    from paper_2607_11985_amd import _lib

    _lib.load()  # fails loudly when the HIP library is not built
    assert torch.cuda.is_available(), "bench.py needs a GPU"
    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)
    order = [1, 2, 3, 4, 5] if args.config == 0 else [args.config]
    head = HEADLINE if args.config == 0 else args.config
    recs = {}
    for idx in order:
        budget = args.cpu_budget * (2 if idx == head else 1)
        recs[idx] = measure(idx, args, torch, dev, not args.no_cpu_baseline, budget)
        print(f"# {recs[idx]['workload']}: {recs[idx]['value']:.4g} evals/s", file=sys.stderr,
              flush=True)
    r = recs[head]
    out = {
        "metric": METRIC, "value": r["value"], "unit": "circuit evals/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": r["ms_per_step"],
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "c64",
        "data": "synthetic (seeded draws of the configuration; no dataset)",
        "config": {k: r[k] for k in ("workload", "description", "n_qubits", "batch", "n_params",
                                     "n_inputs", "ops", "loss", "path", "tile_qubits",
                                     "passes_fwd_bwd", "step_head_rotations", "engine",
                                     "compile_s")},
        "step": ("vqc_forward + vqc_loss_grad + vqc_backward" if args.separate else
                 "vqc_train_step"),
        "timing": ("replays of a HIP graph of one step, HIP events" if args.graph else
                   "launches on the caller's stream (the streaming path forks each batch "
                   "half to its own stream and joins), HIP events"),
        "repeats": r["repeats"],
        "kernel_ms": r["kernel_ms"],
        "forward_only_evals_per_s": r["forward_only_evals_per_s"],
        "roofline": r["roofline"],
    }
    if "cpu_baseline" in r:
        out["cpu_baseline"] = r["cpu_baseline"]
        out["gpu_over_cpu"] = r["gpu_over_cpu"]
    out["configs"] = {recs[i]["workload"]: recs[i] for i in order}
    out["env"] = {"torch": torch.__version__, "hip": getattr(torch.version, "hip", None),
                  "gpu": torch.cuda.get_device_name(dev), "host_cpu": cpu_model(),
                  "host_cores": os.cpu_count()}
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
