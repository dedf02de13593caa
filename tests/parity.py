"""Parity metrics and gates of the GPU tests (not collected by pytest).

Pure NumPy, so the gates themselves are tested on the CPU: a faithful bf16
result (the oracle with bf16 storage, reading r4) passes them, and results
with a planted mistake (a wrong column, a wrong row, a wrong optimizer step)
fail them (tests/test_parity_gates_cpu.py).

Metrics, per tensor x against the oracle's x_ref:
  rel   ||x - x_ref|| / ||x_ref||;
  row   the worst row of x - x_ref as a fraction of a typical row of x_ref,
        max_i ||x_i - r_i|| / sqrt(mean_i ||r_i||^2);
  col   the same over columns.
Tensors are viewed as [rows, last dim] ([tokens, features] for h_out and
dL/dh_out, [out, in] for weight gradients); a vector is one column, so its
row metric is the worst element against the tensor's RMS.  One wrong feature
column of an 8B-wide h_out moves rel by only 1/sqrt(4096), but its col
metric by about 1.

Gates.  fp32: rel <= 1e-4 on everything, row and col <= RC_F32.  bf16: the
loss and the updated parameters at 2e-2; h_out, dL/dh_out and every gradient
at max(2e-2, FLOOR_MULT x its bf16 storage floor) for rel and
max(RC_MIN, FLOOR_MULT x floor) for row and col, the floors being those of
the same inputs in tests/golden/bf16_floor.json (written by
tests/golden/make_bf16_floor.py from the oracle alone).
"""
import hashlib
import json
import os

import numpy as np

TOL = {"f32": 1e-4, "bf16": 2e-2}
RC_F32 = 1e-3       # fp32 row/column gate
RC_MIN = 0.1        # bf16 row/column gate never below this
FLOOR_MULT = 1.5    # bf16 gates sit at this multiple of the storage floor
ADAM_RESOLVED = 0.5  # bf16 AdamW deltas are gated where |g_ref| >= this x rms(g_ref)

FLOOR_FILE = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "bf16_floor.json")


def rel_err(a, b):
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    return float(np.linalg.norm(a - b) / max(np.linalg.norm(b), 1e-30))


def _as2d(x):
    x = np.asarray(x, np.float64)
    if x.ndim == 0:
        return x.reshape(1, 1)
    if x.ndim == 1:
        return x.reshape(-1, 1)
    return x.reshape(-1, x.shape[-1])


def rowcol_err(x, ref):
    """(row, col): the worst row and column of x - ref, each against the RMS
    row (column) norm of ref."""
    d, r = _as2d(x) - _as2d(ref), _as2d(ref)
    rn = np.sqrt(np.mean(np.sum(r * r, axis=1)))
    cn = np.sqrt(np.mean(np.sum(r * r, axis=0)))
    row = float(np.max(np.linalg.norm(d, axis=1)) / max(rn, 1e-30))
    col = float(np.max(np.linalg.norm(d, axis=0)) / max(cn, 1e-30))
    return row, col


def tensor_metrics(x, ref):
    x = np.asarray(x, np.float64).reshape(np.shape(ref))
    row, col = rowcol_err(x, ref)
    return dict(rel=rel_err(x, ref), row=row, col=col)


def fingerprint(params, batch):
    """A digest of the inputs a floor was measured on: every array's key,
    shape and every 1009th value."""
    h = hashlib.sha256()
    items = sorted(params.items()) + sorted((k, v) for k, v in batch.items()
                                            if k in ("h_in", "labels", "seq_lens", "pos_ids",
                                                     "head_w", "head_norm_w", "head_norm_b")
                                            and v is not None)
    for k, v in items:
        a = np.ascontiguousarray(np.asarray(v))
        h.update(k.encode())
        h.update(str(a.shape).encode())
        h.update(np.ascontiguousarray(a.reshape(-1)[::1009]).astype(np.float64).tobytes())
    return h.hexdigest()


def load_floor(case, params, batch, per_step=False):
    """The stored bf16 storage floor of a case, checked to belong to these
    inputs.  per_step: the list of floors of each step of a several-step
    case (each from the same state of the exact trajectory)."""
    floors = json.load(open(FLOOR_FILE))
    if case not in floors:
        raise KeyError(f"no bf16 floor stored for case {case!r}: run tests/golden/make_bf16_floor.py")
    f = floors[case]
    if f["fingerprint"] != fingerprint(params, batch):
        raise ValueError(f"the inputs of case {case!r} changed since its bf16 floor was stored: "
                         "run tests/golden/make_bf16_floor.py")
    if per_step:
        return f.get("steps", [f["tensors"]])
    return f["tensors"]


def results_metrics(dev, ref):
    """Metrics of every compared quantity of one run (dicts as built by
    the parity tests: losses, h_out, dh_out, grads[s], masters[s])."""
    out = {}
    for s, (a, b) in enumerate(zip(dev["losses"], ref["losses"])):
        out[f"loss{s}"] = dict(rel=abs(a - b) / max(abs(b), 1e-30))
    for k in ("h_out", "dh_out"):
        if k in dev and k in ref:
            out[k] = tensor_metrics(dev[k], ref[k])
    for s in range(len(dev["grads"])):
        for k in ref["grads"][s]:
            out[f"g{s}:{k}"] = tensor_metrics(dev["grads"][s][k], ref["grads"][s][k])
    for s in range(1, len(dev.get("masters", []))):
        for k in dev["masters"][s]:
            out[f"p{s}:{k}"] = dict(rel=rel_err(dev["masters"][s][k], ref["masters"][s][k]))
    return out


def _delta_metrics(dev, ref, optimizer, dtype, grad_tol):
    """Update deltas theta_new - theta_old.  SGD: -lr g, gated like the
    gradient.  AdamW: in fp32 on every element whose first-step gradient is
    resolvable (above 1e-4 of its RMS); in bf16 on the elements whose
    first-step gradient is at least ADAM_RESOLVED x its RMS, far above the
    storage noise, so that Adam's step (about -lr sign(g) at first) cannot
    flip on noise there.  The device keeps the master in fp32, so a delta is
    resolved only to one ulp of the new value: ||dd - rd|| < tol ||rd|| +
    ||ulp(theta_new)||."""
    out = {}
    for s in range(1, len(dev["masters"])):
        for k in dev["masters"][s]:
            dd = dev["masters"][s][k] - dev["masters"][s - 1][k]
            rd = ref["masters"][s][k] - ref["masters"][s - 1][k]
            ulp = np.spacing(np.abs(ref["masters"][s][k]).astype(np.float32)).astype(np.float64)
            tol = grad_tol(f"g0:{k}") if optimizer == "sgd" else TOL[dtype]
            if optimizer == "sgd":
                keep = np.ones(np.shape(rd), bool)
            else:
                g0 = np.abs(ref["grads"][0][k])
                rms = np.sqrt(np.mean(g0 ** 2))
                thr = 1e-4 * rms + 1e-12 if dtype == "f32" else ADAM_RESOLVED * rms
                keep = g0 >= thr
                if dtype == "bf16" and rms == 0.0:
                    keep = np.zeros(np.shape(rd), bool)
            if not np.any(keep):
                continue
            err = np.linalg.norm((dd - rd)[keep])
            val = err / (np.linalg.norm(rd[keep]) + np.linalg.norm(ulp[keep]) / tol)
            out[f"d{s}:{k}"] = (val, tol)
    return out


def gate(dev, ref, dtype, optimizer, floor=None, gate_adam_delta=True):
    """Every metric against its bound; raises AssertionError listing the
    worst ratios when any exceeds 1.  Returns {name: (value, bound)}."""
    tol = TOL[dtype]
    floor = floor or {}

    def fl(name, metric):
        return floor.get(name, {}).get(metric, 0.0)

    def grad_tol(name):
        return tol if dtype == "f32" else max(tol, FLOOR_MULT * fl(name, "rel"))

    def rc_tol(name, metric):
        return RC_F32 if dtype == "f32" else max(RC_MIN, FLOOR_MULT * fl(name, metric))

    checks = {}
    for name, m in results_metrics(dev, ref).items():
        if name.startswith("loss") or name.startswith("p"):
            checks[name] = (m["rel"], tol)
            continue
        checks[name] = (m["rel"], grad_tol(name))
        checks[name + "#row"] = (m["row"], rc_tol(name, "row"))
        checks[name + "#col"] = (m["col"], rc_tol(name, "col"))
    if gate_adam_delta or optimizer == "sgd":
        checks.update(_delta_metrics(dev, ref, optimizer, dtype, grad_tol))
    ratio = {k: v / b for k, (v, b) in checks.items()}
    worst = sorted(ratio, key=ratio.get, reverse=True)
    if ratio[worst[0]] >= 1.0:
        raise AssertionError("parity gate failed: " + ", ".join(
            f"{k} = {checks[k][0]:.3g} (bound {checks[k][1]:.3g})" for k in worst[:6]))
    return checks
