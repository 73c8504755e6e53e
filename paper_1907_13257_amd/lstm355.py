"""ctypes binding of liblstm355 (include/lstm355.h).

Argument marshalling only: every computation runs in the library's HIP
kernels.  torch supplies device memory (`data_ptr()`) and streams
(`torch.cuda.current_stream().cuda_stream`).  If the shared library is
missing, importing this module raises: there is no fallback path.
"""
from __future__ import annotations

import ctypes
import os
import re
from typing import Dict, List, Optional, Sequence

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "liblstm355.so")
HEADER = os.path.join(os.path.dirname(HERE), "include", "lstm355.h")

LSTM_OK, LSTM_ERR_INVALID_ARG, LSTM_ERR_UNSUPPORTED, LSTM_ERR_WORKSPACE, LSTM_ERR_HIP, LSTM_ERR_TIMEOUT = range(6)
LSTM_F32, LSTM_BF16 = 0, 1


class lstm_desc_t(ctypes.Structure):
    _fields_ = [("T", ctypes.c_int), ("B", ctypes.c_int), ("I", ctypes.c_int), ("H", ctypes.c_int),
                ("Hp", ctypes.c_int), ("dtype", ctypes.c_int), ("reverse", ctypes.c_int),
                ("ldx", ctypes.c_long), ("ldy", ctypes.c_long)]


class lstm_kernel_stat_t(ctypes.Structure):
    _fields_ = [("name", ctypes.c_char * 32), ("launches", ctypes.c_int), ("total_ms", ctypes.c_double),
                ("flops", ctypes.c_double), ("bytes", ctypes.c_double)]


class LSTMError(RuntimeError):
    def __init__(self, status: int, where: str, detail: str):
        super().__init__(f"{where}: status {status} ({detail})")
        self.status = status


_lib = None


def load_library():
    """Loads liblstm355.so (built by paper_1907_13257_amd.build)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is missing: run `python -m paper_1907_13257_amd.build` "
                          "(there is no fallback implementation)")
    lib = ctypes.CDLL(LIB_PATH)
    vp, i, sz = ctypes.c_void_p, ctypes.c_int, ctypes.c_size_t
    H = ctypes.c_void_p  # lstm_handle_t
    sig = {
        "lstm_create": ([ctypes.POINTER(lstm_desc_t), ctypes.POINTER(H)], i),
        "lstm_reserve_size": ([H], sz),
        "lstm_workspace_size": ([H], sz),
        "lstm_forward": ([H] + [vp] * 11 + [sz, vp, sz, vp], i),
        "lstm_backward": ([H] + [vp] * 11 + [sz] + [vp] * 7 + [i, vp, sz, vp], i),
        "lstm_forward_noalloc": ([H] + [vp] * 11 + [sz, vp], i),
        "lstm_forward_stack": ([i] + [vp] * 9 + [sz, vp, sz, vp], i),
        "lstm_backward_stack": ([i] + [vp] * 9 + [sz] + [vp] * 4 + [i, vp, sz, vp], i),
        "lstm_backward_stack_workspace_size": ([i, vp], sz),
        "lstm_check": ([H, vp, vp], i),
        "lstm_destroy": ([H], i),
        "lstm_status_string": ([i], ctypes.c_char_p),
        "lstm_last_error_detail": ([], ctypes.c_char_p),
        "lstm_describe_tiling": ([H, ctypes.POINTER(ctypes.c_int)], i),
        "lstm_add": ([i, sz, vp, vp, vp, vp], i),
        "lstm_profile_enable": ([i], i),
        "lstm_profile_reset": ([], i),
        "lstm_profile_read": ([ctypes.POINTER(lstm_kernel_stat_t), i, ctypes.POINTER(i)], i),
    }
    for name, (args, res) in sig.items():
        fn = getattr(lib, name)
        fn.argtypes = args
        fn.restype = res
    _lib = lib
    return lib


def header_functions() -> List[str]:
    """Names of the functions include/lstm355.h declares."""
    with open(HEADER) as f:
        text = f.read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(lstm_[a-z_0-9]+)\s*\(", text)))


def _check(st: int, where: str):
    if st != LSTM_OK:
        lib = load_library()
        raise LSTMError(st, where, lib.lstm_last_error_detail().decode())


def _ptr(t) -> Optional[int]:
    if t is None:
        return None
    if isinstance(t, int):
        return t
    return t.data_ptr()


def _nbytes(t, given=None) -> int:
    """Size of a buffer: `given` when stated, else a torch tensor's bytes."""
    if given is not None:
        return int(given)
    if t is None or isinstance(t, int):
        raise ValueError("the size of a raw-pointer buffer must be given")
    return t.numel() * t.element_size()


def _stream(stream) -> Optional[int]:
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


# ---------------------------------------------------------------------------
# one-to-one wrappers of the C entry points
# ---------------------------------------------------------------------------
def lstm_create(T, B, I, H, Hp=0, dtype="bf16", reverse=False, ldx=0, ldy=0) -> int:
    lib = load_library()
    d = lstm_desc_t(T, B, I, H, Hp, LSTM_BF16 if dtype == "bf16" else LSTM_F32, int(bool(reverse)), ldx, ldy)
    h = ctypes.c_void_p()
    _check(lib.lstm_create(ctypes.byref(d), ctypes.byref(h)), "lstm_create")
    return h.value


def lstm_reserve_size(h) -> int:
    return load_library().lstm_reserve_size(h)


def lstm_workspace_size(h) -> int:
    return load_library().lstm_workspace_size(h)


def lstm_forward(h, x, h0, c0, W, R, b, P, y, hT, cT, reserve, workspace, stream=None, reserve_bytes=None,
                 workspace_bytes=None):
    _check(load_library().lstm_forward(h, _ptr(x), _ptr(h0), _ptr(c0), _ptr(W), _ptr(R), _ptr(b), _ptr(P), _ptr(y),
                                       _ptr(hT), _ptr(cT), _ptr(reserve), _nbytes(reserve, reserve_bytes),
                                       _ptr(workspace), _nbytes(workspace, workspace_bytes), _stream(stream)),
           "lstm_forward")


def lstm_forward_noalloc(h, x, h0, c0, W, R, b, P, y, hT, cT, reserve, stream=None, reserve_bytes=None):
    _check(load_library().lstm_forward_noalloc(h, _ptr(x), _ptr(h0), _ptr(c0), _ptr(W), _ptr(R), _ptr(b), _ptr(P),
                                               _ptr(y), _ptr(hT), _ptr(cT), _ptr(reserve),
                                               _nbytes(reserve, reserve_bytes), _stream(stream)),
           "lstm_forward_noalloc")


def _residual_args(n, residual, sums):
    if not residual or not any(residual):
        return None, None
    flags = (ctypes.c_int * n)(*[int(bool(r)) for r in residual])
    return flags, (ctypes.c_void_p * n)(*[_ptr(v) for v in sums])


def lstm_forward_stack(handles, x, Ws, Rs, bs, ys, reserves, workspace, stream=None, residual=None,
                       sums=None) -> bool:
    """Layer-wavefront forward of a stack (lstm_forward_stack).  Returns False,
    having computed nothing that counts, when the stack does not fit it
    (LSTM_ERR_UNSUPPORTED); raises on any other error.  residual[l] / sums[l]:
    layer l's output is y_l plus its input, stored in sums[l]."""
    n = len(handles)
    arr = lambda vals: (ctypes.c_void_p * n)(*[_ptr(v) for v in vals])
    rf, sp = _residual_args(n, residual, sums)
    st = load_library().lstm_forward_stack(n, arr(handles), _ptr(x), arr(Ws), arr(Rs), arr(bs), arr(ys), rf, sp,
                                           arr(reserves), min(_nbytes(r) for r in reserves), _ptr(workspace),
                                           _nbytes(workspace), _stream(stream))
    if st == LSTM_ERR_UNSUPPORTED:
        return False
    _check(st, "lstm_forward_stack")
    return True


def lstm_backward_stack_workspace_size(handles) -> int:
    n = len(handles)
    return load_library().lstm_backward_stack_workspace_size(n, (ctypes.c_void_p * n)(*handles))


def lstm_backward_stack(handles, dy, x, Ws, Rs, ys, reserves, dx, dWs, dRs, dbs, accumulate, workspace,
                        stream=None, residual=None, sums=None) -> bool:
    """Layer-wavefront backward of a stack (lstm_backward_stack).  Returns
    False when the stack does not fit it (LSTM_ERR_UNSUPPORTED); raises on
    any other error."""
    n = len(handles)
    arr = lambda vals: (ctypes.c_void_p * n)(*[_ptr(v) for v in vals])
    rf, sp = _residual_args(n, residual, sums)
    st = load_library().lstm_backward_stack(n, arr(handles), _ptr(dy), _ptr(x), arr(Ws), arr(Rs), arr(ys), rf, sp,
                                            arr(reserves), min(_nbytes(r) for r in reserves), _ptr(dx), arr(dWs),
                                            arr(dRs), arr(dbs), int(bool(accumulate)), _ptr(workspace),
                                            _nbytes(workspace), _stream(stream))
    if st == LSTM_ERR_UNSUPPORTED:
        return False
    _check(st, "lstm_backward_stack")
    return True


def lstm_backward(h, dy, dhT, dcT, x, h0, c0, W, R, P, y, reserve, dx, dh0, dc0, dW, dR, db, dP, accumulate,
                  workspace, stream=None, reserve_bytes=None, workspace_bytes=None):
    _check(load_library().lstm_backward(h, _ptr(dy), _ptr(dhT), _ptr(dcT), _ptr(x), _ptr(h0), _ptr(c0), _ptr(W),
                                        _ptr(R), _ptr(P), _ptr(y), _ptr(reserve), _nbytes(reserve, reserve_bytes),
                                        _ptr(dx), _ptr(dh0), _ptr(dc0), _ptr(dW), _ptr(dR), _ptr(db), _ptr(dP),
                                        int(bool(accumulate)), _ptr(workspace), _nbytes(workspace, workspace_bytes),
                                        _stream(stream)),
           "lstm_backward")


def lstm_check(h, workspace, stream=None) -> int:
    return load_library().lstm_check(h, _ptr(workspace), _stream(stream))


def lstm_destroy(h):
    _check(load_library().lstm_destroy(h), "lstm_destroy")


def lstm_status_string(s: int) -> str:
    return load_library().lstm_status_string(s).decode()


def lstm_last_error_detail() -> str:
    return load_library().lstm_last_error_detail().decode()


def lstm_describe_tiling(h) -> List[int]:
    out = (ctypes.c_int * 8)()
    _check(load_library().lstm_describe_tiling(h, out), "lstm_describe_tiling")
    return list(out)


def lstm_add(dtype, n, a, b, out, stream=None):
    _check(load_library().lstm_add(LSTM_BF16 if dtype == "bf16" else LSTM_F32, n, _ptr(a), _ptr(b), _ptr(out),
                                   _stream(stream)), "lstm_add")


def lstm_profile_enable(on: bool):
    _check(load_library().lstm_profile_enable(int(bool(on))), "lstm_profile_enable")


def lstm_profile_reset():
    _check(load_library().lstm_profile_reset(), "lstm_profile_reset")


def lstm_profile_read() -> Dict[str, dict]:
    arr = (lstm_kernel_stat_t * 16)()
    n = ctypes.c_int()
    _check(load_library().lstm_profile_read(arr, 16, ctypes.byref(n)), "lstm_profile_read")
    return {arr[k].name.decode(): dict(launches=arr[k].launches, total_ms=arr[k].total_ms, flops=arr[k].flops,
                                       bytes=arr[k].bytes) for k in range(n.value)}


# ---------------------------------------------------------------------------
# layers and stacks over torch-allocated device memory
# ---------------------------------------------------------------------------
def torch_dtype(dtype: str):
    import torch
    return torch.bfloat16 if dtype == "bf16" else torch.float32


class Layer:
    """One LSTM/LSTMP layer or direction: owns a handle and its reserve; the
    workspace may be shared between layers whose calls are ordered."""

    def __init__(self, T, B, I, H, Hp=0, dtype="bf16", reverse=False, ldx=0, ldy=0, device="cuda",
                 workspace=None):
        import torch
        self.T, self.B, self.I, self.H, self.Hp, self.dtype, self.reverse = T, B, I, H, Hp, dtype, bool(reverse)
        self.Hr = Hp if Hp else H
        self.ldx = ldx or I
        self.ldy = ldy or self.Hr
        self.handle = lstm_create(T, B, I, H, Hp, dtype, reverse, self.ldx, self.ldy)
        self.reserve = torch.empty(lstm_reserve_size(self.handle), dtype=torch.uint8, device=device)
        self.ws_bytes = lstm_workspace_size(self.handle)
        if workspace is None:
            workspace = torch.empty(self.ws_bytes, dtype=torch.uint8, device=device)
        if workspace.numel() < self.ws_bytes:
            raise ValueError("workspace too small")
        self.workspace = workspace
        self.device = device

    def close(self):
        if self.handle:
            lstm_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def forward(self, x, W, R, b, P=None, h0=None, c0=None, y=None, hT=None, cT=None, stream=None):
        lstm_forward(self.handle, x, h0, c0, W, R, b, P, y, hT, cT, self.reserve, self.workspace, stream)

    def backward(self, dy, x, W, R, y, grads, P=None, h0=None, c0=None, dhT=None, dcT=None, dx=None, dh0=None,
                 dc0=None, accumulate=False, stream=None):
        lstm_backward(self.handle, dy, dhT, dcT, x, h0, c0, W, R, P, y, self.reserve, dx, dh0, dc0, grads["dW"],
                      grads["dR"], grads["db"], grads.get("dP"), accumulate, self.workspace, stream)

    def check(self, stream=None) -> int:
        return lstm_check(self.handle, self.workspace, stream)

    def tiling(self) -> List[int]:
        return lstm_describe_tiling(self.handle)


class StackLayer:
    def __init__(self, I, H, Hp=0, bidirectional=False, residual=False):
        self.I, self.H, self.Hp, self.bidirectional, self.residual = I, H, Hp, bidirectional, residual
        self.Hr = Hp if Hp else H
        self.out = self.Hr * (2 if bidirectional else 1)


class Stack:
    """A stack of layers composed through the C ABI: a bidirectional layer
    runs its two directions into the halves of one output buffer (row stride
    2*Hr); a residual layer's output is y + x (lstm_add).  Backward mirrors it:
    the directions' input gradients and the identity path are summed with
    lstm_add.  Initial states are zero and the final states get no gradient.

    params[l][d] = dict(W, R, b[, P]) device tensors; grads likewise with
    dW, dR, db[, dP] (fp32), allocated here."""

    def __init__(self, T, B, layers: Sequence[StackLayer], dtype="bf16", device="cuda", wavefront=True):
        import torch
        self.T, self.B, self.dtype, self.device = T, B, dtype, device
        self.wavefront = wavefront
        self.last_forward = None
        self.last_backward = None
        self.wave_ws = None
        self.layers = list(layers)
        td = torch_dtype(dtype)
        self.dirs: List[List[Layer]] = []
        ws_bytes = 0
        shapes = []
        for L in self.layers:
            if L.residual and L.out != L.I:
                raise ValueError("residual layer needs input width == output width")
            nd = 2 if L.bidirectional else 1
            shapes.append(nd)
            for d in range(nd):
                h = lstm_create(T, B, L.I, L.H, L.Hp, dtype, d == 1, L.I, L.out)
                ws_bytes = max(ws_bytes, lstm_workspace_size(h))
                lstm_destroy(h)
        self.workspace = torch.empty(ws_bytes, dtype=torch.uint8, device=device)
        for L, nd in zip(self.layers, shapes):
            self.dirs.append([Layer(T, B, L.I, L.H, L.Hp, dtype, d == 1, L.I, L.out, device, self.workspace)
                              for d in range(nd)])
        self.y = [torch.empty((T, B, L.out), dtype=td, device=device) for L in self.layers]
        self.xout = [torch.empty((T, B, L.out), dtype=td, device=device) if L.residual else None
                     for L in self.layers]
        self.inputs: List = [None] * len(self.layers)
        self.dxbuf = [[torch.empty((T, B, L.I), dtype=td, device=device) for _ in range(2 if L.bidirectional else 1)]
                      for L in self.layers]
        self.gbuf = [torch.empty((T, B, L.I), dtype=td, device=device) for L in self.layers]

    def alloc_grads(self, params):
        import torch
        grads = []
        for L, prm in zip(self.layers, params):
            gl = []
            for p in prm:
                g = dict(dW=torch.empty(p["W"].shape, dtype=torch.float32, device=self.device),
                         dR=torch.empty(p["R"].shape, dtype=torch.float32, device=self.device),
                         db=torch.empty(p["b"].shape, dtype=torch.float32, device=self.device))
                if L.Hp:
                    g["dP"] = torch.empty(p["P"].shape, dtype=torch.float32, device=self.device)
                gl.append(g)
            grads.append(gl)
        return grads

    def forward(self, x, params, stream=None):
        # a stack of unidirectional LSTM layers (residual ones included) runs
        # as one layer wavefront when the library supports its shape
        # (lstm_forward_stack)
        self.last_forward = "layers"
        if (self.wavefront and 2 <= len(self.layers) <= 4 and self.dtype == "bf16"
                and all(not L.bidirectional and not L.Hp for L in self.layers)):
            lays = [d[0] for d in self.dirs]
            residual = [L.residual for L in self.layers]
            if lstm_forward_stack([l.handle for l in lays], x, [p[0]["W"] for p in params],
                                  [p[0]["R"] for p in params], [p[0]["b"] for p in params], self.y,
                                  [l.reserve for l in lays], self.workspace, stream, residual=residual,
                                  sums=self.xout):
                outs = [self.xout[li] if L.residual else self.y[li] for li, L in enumerate(self.layers)]
                self.inputs = [x] + outs[:-1]
                self.last_forward = "wavefront"
                return outs[-1]
        cur = x
        for li, L in enumerate(self.layers):
            self.inputs[li] = cur
            y = self.y[li]
            for d, lay in enumerate(self.dirs[li]):
                p = params[li][d]
                yd = y[:, :, d * L.Hr:] if d else y
                lay.forward(cur, p["W"], p["R"], p["b"], p.get("P"), y=yd, stream=stream)
            if L.residual:
                lstm_add(self.dtype, y.numel(), y, cur, self.xout[li], stream)
                cur = self.xout[li]
            else:
                cur = y
        return cur

    def backward(self, d_out, params, grads, accumulate=False, stream=None):
        # after a wavefront forward, the backward runs as one too when its
        # shapes allow (lstm_backward_stack)
        self.last_backward = "layers"
        if self.last_forward == "wavefront":
            lays = [d[0] for d in self.dirs]
            hs = [l.handle for l in lays]
            need = lstm_backward_stack_workspace_size(hs)
            if need:
                import torch
                if self.wave_ws is None or self.wave_ws.numel() < need:
                    self.wave_ws = torch.empty(need, dtype=torch.uint8, device=self.device)
                dx = self.dxbuf[0][0]
                if lstm_backward_stack(hs, d_out, self.inputs[0], [p[0]["W"] for p in params],
                                       [p[0]["R"] for p in params], self.y, [l.reserve for l in lays], dx,
                                       [g[0]["dW"] for g in grads], [g[0]["dR"] for g in grads],
                                       [g[0]["db"] for g in grads], accumulate, self.wave_ws, stream,
                                       residual=[L.residual for L in self.layers], sums=self.xout):
                    self.last_backward = "wavefront"
                    return dx
        g = d_out
        for li in range(len(self.layers) - 1, -1, -1):
            L = self.layers[li]
            x = self.inputs[li]
            y = self.y[li]
            for d, lay in enumerate(self.dirs[li]):
                p = params[li][d]
                off = d * L.Hr
                lay.backward(g[:, :, off:] if d else g, x, p["W"], p["R"], y[:, :, off:] if d else y,
                             grads[li][d], P=p.get("P"), dx=self.dxbuf[li][d], accumulate=accumulate,
                             stream=stream)
            dx = self.dxbuf[li][0]
            out = self.gbuf[li]
            if L.bidirectional:
                lstm_add(self.dtype, dx.numel(), dx, self.dxbuf[li][1], out, stream)
                dx = out
            if L.residual:
                lstm_add(self.dtype, dx.numel(), dx, g, out, stream)
                dx = out
            g = dx
        return g

    def check(self, stream=None) -> int:
        return lstm_check(self.dirs[0][0].handle, self.workspace, stream)
