"""Shared pieces of the GPU tests: moving synthetic tensors to the device,
running a workload through the C ABI, running the same workload through the
oracle, and the normwise error metric."""
from __future__ import annotations

import sys
from typing import Dict, List, Optional

import numpy as np

import oracle
import synth
from synth.device import device_params, stack_layers, to_dev, to_f64  # noqa: F401

TOL = {"f32": dict(out=1e-4, grad=1e-4), "bf16": dict(out=2e-2, grad=5e-2)}


def normwise(a, r) -> float:
    """max_i |a_i - r_i| / max_i |r_i| (absolute error when r is all zero)."""
    a = np.asarray(a, dtype=np.float64)
    r = np.asarray(r, dtype=np.float64)
    den = float(np.max(np.abs(r))) if r.size else 0.0
    num = float(np.max(np.abs(a - r))) if r.size else 0.0
    return num / den if den > 0 else num


def announce(msg: str):
    print(f"[gpu-case] {msg}", flush=True)
    sys.stdout.flush()


def oracle_layers(prob: synth.Problem) -> List[oracle.LayerDef]:
    out = []
    for li, L in enumerate(prob.wl.layers):
        dirs = []
        for d, p in enumerate(prob.params[li]):
            prm = dict(W=p.W.f64, R=p.R.f64, b=p.b64)
            if p.P is not None:
                prm["P"] = p.P.f64
            h0 = prob.h0[li][d]
            c0 = prob.c0[li][d]
            if h0 is not None:
                prm["h0"] = h0.f64
            if c0 is not None:
                prm["c0"] = c0.astype(np.float64)
            dirs.append(prm)
        out.append(oracle.LayerDef(dirs, residual=L.residual))
    return out


def _rows_of(prm: dict, rows) -> dict:
    q = dict(prm)
    for k in ("h0", "c0"):
        if k in q:
            q[k] = q[k][rows]
    return q


def run_oracle(prob: synth.Problem, rows: Optional[np.ndarray] = None) -> Dict:
    """Stack output and all gradients from the oracle, on all batch rows or on
    the selected ones (rows are independent, so the per-row results are the
    full problem's; the weight gradients are those of the selected rows)."""
    layers = oracle_layers(prob)
    x = prob.x.f64
    dy = prob.dy.f64
    if rows is not None:
        x = x[:, rows]
        dy = dy[:, rows]
        layers = [oracle.LayerDef([_rows_of(p, rows) for p in L.dirs], L.residual) for L in layers]
    y, _ = oracle.stack_forward(x, layers)
    g = oracle.stack_backward(x, layers, dy)
    return dict(y=y, dx=g["dx"], layers=g["layers"])


def run_stack_gpu(prob: synth.Problem, stack=None, params=None):
    """Forward + backward of the whole stack through the C ABI (zero initial
    states).  Returns numpy float64 results and the Stack object."""
    import torch
    from paper_1907_13257_amd import Stack
    wl = prob.wl
    if stack is None:
        stack = Stack(wl.T, wl.B, stack_layers(wl), wl.dtype)
    if params is None:
        params = device_params(prob)
    grads = stack.alloc_grads(params)
    x = to_dev(prob.x)
    dy = to_dev(prob.dy)
    y = stack.forward(x, params)
    dx = stack.backward(dy, params, grads)
    st = stack.check()
    torch.cuda.synchronize()
    assert st == 0, f"lstm_check returned {st}"
    res = dict(y=to_f64(y), dx=to_f64(dx),
               layers=[[{k: to_f64(v) for k, v in g.items()} for g in gl] for gl in grads])
    return res, stack


def compare(gpu: Dict, ref: Dict, dtype: str, rows=None, label="") -> Dict[str, float]:
    """Normwise errors of every output and gradient; asserts the tolerances."""
    tol = TOL[dtype]
    errs = {}
    ysel = gpu["y"] if rows is None else gpu["y"][:, rows]
    dxsel = gpu["dx"] if rows is None else gpu["dx"][:, rows]
    errs["y"] = normwise(ysel, ref["y"])
    errs["dx"] = normwise(dxsel, ref["dx"])
    for li, (gl, rl) in enumerate(zip(gpu["layers"], ref["layers"])):
        for d, (g, r) in enumerate(zip(gl, rl)):
            for k in ("dW", "dR", "db", "dP"):
                if k in g:
                    errs[f"L{li}d{d}.{k}"] = normwise(g[k], r[k])
    announce(f"{label} errors: " + ", ".join(f"{k}={v:.2e}" for k, v in errs.items()))
    bad = {k: v for k, v in errs.items() if v > (tol["out"] if k == "y" else tol["grad"])}
    assert not bad, f"{label}: tolerance exceeded {bad}"
    return errs
