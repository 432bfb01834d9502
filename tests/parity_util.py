"""Bars and checks shared by the GPU parity tests (HIP path against the oracle).

Bars (complex64 on the GPU, complex128 in the oracle):
  E      : max |E - E_ref| <= E_TOL = 1e-5 (absolute)
  grads  : per sample row, max |g - g_ref| <= G_REL max |g_ref| + G_FLOOR sum_j |cot_j|
           over the row's whole gradient vector (parameters and inputs together),
           and, where a row has at least four parameters and four inputs, over each
           of the two arrays on its own as well.
Every input and cotangent reaches both sides as the same float32 values; the
oracle never receives a value the GPU computed.  Where the GPU forms a cotangent
itself (the training step's loss head), the oracle forms its own from its own E
and the bar gains the first-order effect of the difference (check_step).
"""
import sys

import numpy as np

import oracle

E_TOL = 1e-5
G_REL = 1e-4
G_FLOOR = 1e-6


def note(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def gpu_run(torch, ops, n, P, F, params, inputs, cot=None, path="auto", engine="jit",
            reg_bits=0):
    """Forward (training) and, given a cotangent, backward through the C ABI."""
    from paper_2607_11985_amd.api import Circuit
    circ = Circuit(ops, n, P, F, path=path, engine=engine, reg_bits=reg_bits)
    p = torch.from_numpy(np.ascontiguousarray(params)).cuda()
    x = torch.from_numpy(np.ascontiguousarray(inputs)).cuda()
    E, ws = circ.forward(p, x, training=True)
    out = {"E": None, "dp": None, "dx": None, "circ": circ}
    if cot is not None:
        g = torch.from_numpy(np.ascontiguousarray(cot, dtype=np.float32)).cuda()
        dp, dx = circ.backward(p, x, g, ws)
        torch.cuda.synchronize()
        out["dp"], out["dx"] = dp.cpu().numpy(), dx.cpu().numpy()
    torch.cuda.synchronize()
    out["E"] = E.cpu().numpy()
    return out


def check_E(E, Eref):
    err = float(np.max(np.abs(E.astype(np.float64) - Eref))) if E.size else 0.0
    assert err <= E_TOL, f"E max abs err {err:.3e}"
    return err


def check_rows(g, gref, cot, what, allow=0.0):
    """Row max-norm bar: max|g - g_ref| <= G_REL max|g_ref| + G_FLOOR sum|cot| + allow."""
    if g.size == 0:
        return 0.0
    g = g.astype(np.float64)
    err = np.max(np.abs(g - gref), axis=1)
    scale = np.max(np.abs(gref), axis=1)
    bar = (G_REL * scale + G_FLOOR * np.sum(np.abs(np.asarray(cot, dtype=np.float64)), axis=1)
           + allow)
    bad = err > bar
    assert not np.any(bad), (f"{what}: rows {np.nonzero(bad)[0][:8]} err {err[bad][:4]} "
                             f"scale {scale[bad][:4]} bar {bar[bad][:4]}")
    return float(np.max(err / np.maximum(scale, 1e-30)))


def check_grad(g, gref, cot, what):
    return check_rows(g, gref, cot, what)


def check_grads(r, dpr, dxr, cot, allow=0.0):
    """The concatenated [dparams | dinputs] rows, and each array on its own when
    both have at least four columns (there a row's own max is well conditioned)."""
    err = check_rows(np.concatenate([r["dp"], r["dx"]], axis=1),
                     np.concatenate([dpr, dxr], axis=1), cot, "gradient", allow)
    if r["dp"].shape[1] >= 4 and r["dx"].shape[1] >= 4:
        check_rows(r["dp"], dpr, cot, "dparams", allow)
        check_rows(r["dx"], dxr, cot, "dinputs", allow)
    return err


def k_max(ops):
    """Largest sum of |mul| over the occurrences of one parameter or input: a bound
    on |dE_j / d slot| (every rotation moves <Z_j> by at most its angle's rate)."""
    tot = {}
    for o in ops:
        for a in o.angles:
            if a[0] == "const":
                continue
            mul = abs(a[2]) if len(a) > 2 else 1.0
            tot[(a[0], a[1])] = tot.get((a[0], a[1]), 0.0) + mul
    return max(tot.values()) if tot else 0.0


def oracle_cotangent(loss, Er, y_rows, batch):
    """The loss head's cotangent evaluated on the oracle's own E rows (batch: the
    batch size the MSE mean runs over)."""
    n = Er.shape[1]
    if loss == "sum":
        return np.ones_like(Er)
    if loss == "mean":
        return np.full_like(Er, 1.0 / n)
    if loss == "mse_z0":
        g = np.zeros_like(Er)
        g[:, 0] = 2.0 * (Er[:, 0] - y_rows) / batch
        return g
    return np.repeat((2.0 * (Er.mean(axis=1) - y_rows) / (n * batch))[:, None], n, axis=1)


def check_step(E, g, dp, dx, ops, n, params, inputs, y_rows, loss, batch, psi0=None):
    """Outputs of a training step (rows of the batch) against the oracle.

    The oracle evaluates the loss head on its own E.  With an MSE head the GPU's
    cotangent then differs from it by at most 2 E_TOL / batch summed over the
    qubits (E is within E_TOL), and a slot with |dE_j / d slot| <= k_max moves by
    at most k_max * 2 E_TOL / batch: the gradient bar adds that term (zero for
    the sum and mean heads, whose cotangent is a constant)."""
    Er = oracle.forward(ops, n, params, inputs, psi0=psi0)
    check_E(E, Er)
    gref = oracle_cotangent(loss, Er, y_rows, batch)
    if g is not None:
        gerr = float(np.max(np.abs(g.astype(np.float64) - gref)))
        assert gerr <= 2 * E_TOL / batch + 1e-6 * max(1.0, float(np.max(np.abs(gref)))), gerr
    dpr, dxr, _ = oracle.vjp(ops, n, params, inputs, gref, psi0=psi0)
    allow = 0.0 if loss in ("sum", "mean") else k_max(ops) * 2 * E_TOL / batch
    return check_grads({"dp": dp, "dx": dx}, dpr, dxr, gref, allow)


def oracle_central_differences(ops, n, params, inputs, cot, h):
    """The FD mode's definition on the oracle side: for every sample b and slot s
    (parameters, then inputs), sum_j cot[b, j] (E_j(s + h) - E_j(s - h)) / (2 h),
    with the slot's value moved in the params / inputs arrays, so that every gate
    reading the slot sees the shift (as the library's FD mode does).  Returns
    (dparams [B, P], dinputs [B, F])."""
    params = np.asarray(params, dtype=np.float64)
    inputs = np.asarray(inputs, dtype=np.float64)
    B, P = params.shape
    F = inputs.shape[1]
    NS = P + F
    ps = np.repeat(np.repeat(params[:, None, None, :], NS, axis=1), 2, axis=2)
    xs = np.repeat(np.repeat(inputs[:, None, None, :], NS, axis=1), 2, axis=2)
    for s in range(NS):
        arr, col = (ps, s) if s < P else (xs, s - P)
        arr[:, s, 0, col] += h
        arr[:, s, 1, col] -= h
    E = oracle.forward(ops, n, ps.reshape(B * NS * 2, P), xs.reshape(B * NS * 2, F))
    E = E.reshape(B, NS, 2, n)
    d = np.einsum("bsj,bj->bs", E[:, :, 0, :] - E[:, :, 1, :], np.asarray(cot, np.float64))
    d /= 2.0 * h
    return d[:, :P], d[:, P:]


def fd_bound(ops, params, inputs, cot, h):
    """Bound on |FD_gpu - FD_oracle| at the same h, per sample row: each of the
    two GPU evaluations has E within E_TOL, giving sum|cot| E_TOL / h, and the GPU
    forms value +- h in float32, a rounding of at most 2^-24 (max|value| + h)
    per side that moves L by at most k_max sum|cot| times it."""
    vmax = max(float(np.max(np.abs(params))) if np.size(params) else 0.0,
               float(np.max(np.abs(inputs))) if np.size(inputs) else 0.0)
    gs = np.sum(np.abs(np.asarray(cot, np.float64)), axis=1, keepdims=True)
    shift = 2.0 ** -24 * (vmax + h)
    return gs * (E_TOL + k_max(ops) * shift) / h
