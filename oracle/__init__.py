"""fp64 CPU oracle for the stacked LSTM / LSTMP training step.

TEST INFRASTRUCTURE.  Only `tests/`, `__graft_entry__.smoke()` and the
`cpu_baseline` leg of `bench.py` may import this package.  It shares no code
with the GPU library and never imports it.

`layer_forward` / `layer_backward` wrap the plain C loops of
`lstm_oracle.c` (one layer or one direction).  `stack_forward` /
`stack_backward` compose layers the way the GNMT encoder stacks them: a
bidirectional first layer whose two directions are concatenated on the
feature axis, and residual connections (output = y + x) on later layers.
The paper names these networks and their widths (Section 4, "Methodology";
the original GNMT's layout is recalled in Section 4, "Model Parallel
Splitting") without writing out their equations; the composition here is the
standard one.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from typing import Dict, List, Optional, Sequence

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "lstm_oracle.c")
_LIB = os.path.join(_HERE, "liblstm_oracle.so")
_lib = None

_DP = ctypes.POINTER(ctypes.c_double)


def build(force: bool = True) -> str:
    """Compile the oracle with gcc (plain -O2, OpenMP, generic x86-64)."""
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp"
        subprocess.check_call(["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-std=c99",
                               "-Wall", "-Wextra", "-o", tmp, _SRC, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build(force=True)
        lib = ctypes.CDLL(_LIB)
        i = ctypes.c_int
        lib.lstm_oracle_forward.argtypes = [i, i, i, i, i, i] + [_DP] * 13
        lib.lstm_oracle_forward.restype = i
        lib.lstm_oracle_backward.argtypes = [i, i, i, i, i, i] + [_DP] * 17
        lib.lstm_oracle_backward.restype = i
        lib.lstm_oracle_num_threads.argtypes = []
        lib.lstm_oracle_num_threads.restype = i
        lib.lstm_oracle_set_num_threads.argtypes = [i]
        lib.lstm_oracle_set_num_threads.restype = None
        _lib = lib
    return _lib


def num_threads() -> int:
    return int(_load().lstm_oracle_num_threads())


def set_num_threads(n: int) -> None:
    """Threads of the oracle's loops (timing only; results do not depend on it)."""
    _load().lstm_oracle_set_num_threads(int(n))


def _in(a) -> Optional[np.ndarray]:
    if a is None:
        return None
    return np.ascontiguousarray(np.asarray(a, dtype=np.float64))


def _p(a):
    return None if a is None else a.ctypes.data_as(_DP)


def _dims(x, W, R, P):
    T, B, I = x.shape
    G, I2 = W.shape
    if G % 4 or I2 != I:
        raise ValueError("W must be [4H, I]")
    H = G // 4
    Hp = 0 if P is None else P.shape[0]
    Hr = Hp if Hp else H
    if R.shape != (G, Hr):
        raise ValueError("R must be [4H, Hr]")
    if P is not None and P.shape != (Hp, H):
        raise ValueError("P must be [Hp, H]")
    return T, B, I, H, Hp, Hr


def layer_forward(x, W, R, b, P=None, h0=None, c0=None, reverse=False, states=False) -> Dict[str, np.ndarray]:
    """One layer (or one direction) forward.  Returns y[T,B,Hr], hT, cT and,
    with `states`, the activated gates [T,B,4H], c [T,B,H] and m [T,B,H]."""
    x, W, R, b, P, h0, c0 = map(_in, (x, W, R, b, P, h0, c0))
    T, B, I, H, Hp, Hr = _dims(x, W, R, P)
    y = np.empty((T, B, Hr))
    hT = np.empty((B, Hr))
    cT = np.empty((B, H))
    out = dict(y=y, hT=hT, cT=cT)
    g = cs = ms = None
    if states:
        g = out["gates"] = np.empty((T, B, 4 * H))
        cs = out["c"] = np.empty((T, B, H))
        ms = out["m"] = np.empty((T, B, H))
    rc = _load().lstm_oracle_forward(T, B, I, H, Hp, int(bool(reverse)), _p(x), _p(h0), _p(c0), _p(W), _p(R),
                                     _p(b), _p(P), _p(y), _p(hT), _p(cT), _p(g), _p(cs), _p(ms))
    if rc:
        raise RuntimeError("oracle forward failed")
    return out


def layer_backward(x, W, R, b, dy, P=None, h0=None, c0=None, dhT=None, dcT=None, reverse=False) -> Dict[str, np.ndarray]:
    """Gradients of L = sum <dy, y> + <dhT, hT> + <dcT, cT> for one layer."""
    x, W, R, b, P, h0, c0, dy, dhT, dcT = map(_in, (x, W, R, b, P, h0, c0, dy, dhT, dcT))
    T, B, I, H, Hp, Hr = _dims(x, W, R, P)
    if dy.shape != (T, B, Hr):
        raise ValueError("dy must be [T, B, Hr]")
    g = dict(dx=np.empty((T, B, I)), dh0=np.empty((B, Hr)), dc0=np.empty((B, H)),
             dW=np.empty((4 * H, I)), dR=np.empty((4 * H, Hr)), db=np.empty(4 * H))
    if Hp:
        g["dP"] = np.empty((Hp, H))
    rc = _load().lstm_oracle_backward(T, B, I, H, Hp, int(bool(reverse)), _p(x), _p(h0), _p(c0), _p(W), _p(R),
                                      _p(b), _p(P), _p(dy), _p(dhT), _p(dcT), _p(g["dx"]), _p(g["dh0"]),
                                      _p(g["dc0"]), _p(g["dW"]), _p(g["dR"]), _p(g["db"]), _p(g.get("dP")))
    if rc:
        raise RuntimeError("oracle backward failed")
    return g


# ---------------------------------------------------------------------------
# stacks
# ---------------------------------------------------------------------------
class LayerDef:
    """One layer of a stack: a list of one (unidirectional) or two
    (bidirectional: forward, then reverse) parameter dicts with keys W, R, b
    and optionally P, h0, c0; `residual` adds the layer input to its output."""

    def __init__(self, dirs: Sequence[dict], residual: bool = False):
        if len(dirs) not in (1, 2):
            raise ValueError("a layer has one or two directions")
        self.dirs = list(dirs)
        self.residual = residual


def stack_forward(x, layers: List[LayerDef]):
    """Returns the stack output and the input of every layer."""
    inputs = []
    cur = _in(x)
    for L in layers:
        inputs.append(cur)
        ys = []
        for d, prm in enumerate(L.dirs):
            ys.append(layer_forward(cur, prm["W"], prm["R"], prm["b"], prm.get("P"), prm.get("h0"),
                                    prm.get("c0"), reverse=(d == 1))["y"])
        y = ys[0] if len(ys) == 1 else np.concatenate(ys, axis=2)
        if L.residual:
            if y.shape != cur.shape:
                raise ValueError("residual layer needs equal input and output widths")
            y = y + cur
        cur = y
    return cur, inputs


def stack_backward(x, layers: List[LayerDef], d_out) -> Dict[str, object]:
    """Gradients of L = <d_out, stack output>.  Returns dx (input gradient) and
    per layer a list (one entry per direction) of gradient dicts."""
    _, inputs = stack_forward(x, layers)
    g = _in(d_out)
    per_layer: List[List[dict]] = [None] * len(layers)
    for li in range(len(layers) - 1, -1, -1):
        L = layers[li]
        xin = inputs[li]
        grads = []
        dx = None
        off = 0
        for d, prm in enumerate(L.dirs):
            Hr = prm["R"].shape[1]
            dyd = g[:, :, off:off + Hr]
            off += Hr
            gr = layer_backward(xin, prm["W"], prm["R"], prm["b"], dyd, prm.get("P"), prm.get("h0"),
                                prm.get("c0"), reverse=(d == 1))
            grads.append(gr)
            dx = gr["dx"] if dx is None else dx + gr["dx"]
        if L.residual:
            dx = dx + g
        per_layer[li] = grads
        g = dx
    return dict(dx=g, layers=per_layer)
