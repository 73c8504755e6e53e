"""Seeded synthetic inputs for the stacked LSTM / LSTMP training step.

This module is shared by the tests, the benchmark and the smoke check.  It
draws random numbers and converts them to the storage formats; it holds none
of the LSTM arithmetic (no gates, no recurrence, no gradients), so the oracle
and the GPU path stay independent of each other while consuming the very same
host arrays.

The workloads follow the per-worker training step of the two recurrent
networks the paper evaluates (Section 4, "Methodology"): the GNMT stacks of
1024-wide LSTM layers and the BigLSTM layers with 8192 cells.  Their datasets
(WMT'16, 1B Word) are replaced by seeded Gaussian inputs: an LSTM step's cost
does not depend on the values, only the gate saturation does.

Generator: numpy's PCG64 (O'Neill 2014) seeded with the config seed.  Draw
order is fixed: for every layer (and every direction of a bidirectional
layer) W, R, b, P; then x, h0, c0; then the upstream gradient.  Values are
drawn in float64, then rounded once to the storage type; the oracle consumes
the rounded values exactly (bf16 and fp32 are exact in fp64).
"""
from __future__ import annotations

import dataclasses
from typing import Dict, List, Optional

import numpy as np

GATES = 4  # rows of W, R and b come in four blocks (i, f, g, o)


# ---------------------------------------------------------------------------
# storage formats
# ---------------------------------------------------------------------------
def f32_to_bf16_bits(a) -> np.ndarray:
    """Round float32 values to bfloat16, round-to-nearest-even, NaN kept quiet.

    Returns the 16-bit patterns as uint16.
    """
    a = np.ascontiguousarray(np.asarray(a, dtype=np.float32))
    u = a.view(np.uint32).astype(np.uint64)
    lsb = (u >> np.uint64(16)) & np.uint64(1)
    r = ((u + np.uint64(0x7FFF) + lsb) >> np.uint64(16)).astype(np.uint16)
    nan = np.isnan(a)
    if nan.any():
        r[nan] = ((u[nan] >> np.uint64(16)).astype(np.uint16)) | np.uint16(0x0040)
    return r


def bf16_bits_to_f64(bits) -> np.ndarray:
    bits = np.ascontiguousarray(np.asarray(bits, dtype=np.uint16))
    return (bits.astype(np.uint32) << np.uint32(16)).view(np.float32).astype(np.float64)


class Tensor:
    """One synthetic tensor in two views: `dev` (the storage bits handed to the
    library: float32, or uint16 bfloat16 patterns) and `f64` (the same values,
    exactly, for the oracle)."""

    __slots__ = ("dev", "f64", "dtype")

    def __init__(self, values64: np.ndarray, dtype: str):
        self.dtype = dtype
        if dtype == "bf16":
            self.dev = f32_to_bf16_bits(values64.astype(np.float32))
            self.f64 = bf16_bits_to_f64(self.dev)
        elif dtype == "f32":
            self.dev = np.ascontiguousarray(values64.astype(np.float32))
            self.f64 = self.dev.astype(np.float64)
        else:
            raise ValueError(dtype)

    @property
    def shape(self):
        return self.dev.shape


# ---------------------------------------------------------------------------
# workload description
# ---------------------------------------------------------------------------
@dataclasses.dataclass
class LayerSpec:
    I: int                   # input width
    H: int                   # cells
    Hp: int = 0              # projection width (0: plain LSTM)
    bidirectional: bool = False
    residual: bool = False   # output is y + x (requires Ho * dirs == I)

    @property
    def Hr(self) -> int:
        return self.Hp if self.Hp else self.H

    @property
    def out_width(self) -> int:
        return self.Hr * (2 if self.bidirectional else 1)


@dataclasses.dataclass
class Workload:
    name: str
    T: int
    B: int
    layers: List[LayerSpec]
    dtype: str                 # "bf16" or "f32"
    seed: int
    x_dist: str = "normal"     # "normal": N(0,1); "uniform1": U(-1,1)
    w_scale: float = 0.1       # W, R, P ~ U(-w_scale, w_scale)
    b_mode: str = "uniform"    # "uniform": U(-w_scale, w_scale); "forget1": 0 except forget gate 1.0
    state: str = "zero"        # "zero": h0 = c0 = 0; "uniform1": U(-1,1)
    loss: str = "dy_all"       # "dy_all": dy ~ N(0,1) for every t; "hT_dot_g": dy only at the last step

    def gemm_flops(self) -> float:
        """Algorithmic FLOPs of one training step: 2*M*N*K over every matrix
        product of forward, BPTT and the weight/input gradients.  Pointwise gate
        math is excluded.  Per layer and direction: forward 2TB*4H*(I+Hr)
        (+ 2TB*H*Hp for the projection), backward twice the forward."""
        tot = 0.0
        for L in self.layers:
            fwd = 2.0 * self.T * self.B * 4 * L.H * (L.I + L.Hr)
            if L.Hp:
                fwd += 2.0 * self.T * self.B * L.H * L.Hp
            dirs = 2 if L.bidirectional else 1
            tot += 3.0 * fwd * dirs
        return tot


def tiny(dtype: str = "f32") -> Workload:
    return Workload("tiny", T=8, B=4, layers=[LayerSpec(32, 64)], dtype=dtype, seed=0,
                    x_dist="uniform1", w_scale=1.0 / 8.0, b_mode="forget1",
                    state="uniform1", loss="hT_dot_g")


def gnmt4(B: int = 128, seed: int = 1, T: int = 50) -> Workload:
    return Workload(f"gnmt4_B{B}", T=T, B=B, layers=[LayerSpec(1024, 1024) for _ in range(4)],
                    dtype="bf16", seed=seed, w_scale=0.1)


def sweep(B: int) -> Workload:
    return gnmt4(B=B, seed=2)


SWEEP_BATCHES = (16, 32, 64, 128, 256, 512)


def biglstm(T: int = 20, B: int = 128) -> Workload:
    return Workload("biglstm", T=T, B=B,
                    layers=[LayerSpec(1024, 8192, Hp=1024) for _ in range(2)],
                    dtype="bf16", seed=3, w_scale=0.05)


def gnmt8(T: int = 50, B: int = 256) -> Workload:
    layers = [LayerSpec(1024, 1024, bidirectional=True), LayerSpec(2048, 1024)]
    layers += [LayerSpec(1024, 1024, residual=True) for _ in range(6)]
    return Workload("gnmt8_bi_residual", T=T, B=B, layers=layers, dtype="bf16", seed=4, w_scale=0.1)


def floor(T: int = 50, B: int = 8) -> Workload:
    """The smallest layer the XCD-local recurrences take (256 cells, one batch
    row per XCD): its per-step time is the kernels' exchange and
    synchronisation floor, with almost no arithmetic or traffic per step."""
    return Workload(f"floor_B{B}", T=T, B=B, layers=[LayerSpec(256, 256)], dtype="bf16", seed=5, w_scale=0.1)


CONFIGS = {
    "tiny": tiny,
    "gnmt4": gnmt4,
    "biglstm": biglstm,
    "gnmt8": gnmt8,
}


# ---------------------------------------------------------------------------
# drawing
# ---------------------------------------------------------------------------
@dataclasses.dataclass
class LayerParams:
    W: Tensor                 # [4H, I]
    R: Tensor                 # [4H, Hr]
    b: np.ndarray             # [4H] float32 (bias is always fp32)
    P: Optional[Tensor]       # [Hp, H] or None

    @property
    def b64(self) -> np.ndarray:
        return self.b.astype(np.float64)


@dataclasses.dataclass
class Problem:
    wl: Workload
    params: List[List[LayerParams]]   # params[layer][direction]
    x: Tensor                         # [T, B, I0]
    h0: List[List[Optional[Tensor]]]  # per layer/direction [B, Hr] or None
    c0: List[List[Optional[np.ndarray]]]  # per layer/direction float32 [B, H] or None
    dy: Tensor                        # [T, B, out] upstream gradient of the top output


def _uniform(rng, a, shape):
    return rng.uniform(-a, a, size=shape)


def draw(wl: Workload, row_mask: Optional[np.ndarray] = None) -> Problem:
    """Draw every tensor of one training step.

    `row_mask` (bool [B]) zeroes the upstream gradient outside the selected
    batch rows after drawing, so the draw itself is identical with and without
    it."""
    rng = np.random.Generator(np.random.PCG64(wl.seed))
    params: List[List[LayerParams]] = []
    for L in wl.layers:
        dirs = []
        for _ in range(2 if L.bidirectional else 1):
            W = Tensor(_uniform(rng, wl.w_scale, (GATES * L.H, L.I)), wl.dtype)
            R = Tensor(_uniform(rng, wl.w_scale, (GATES * L.H, L.Hr)), wl.dtype)
            if wl.b_mode == "forget1":
                b = np.zeros(GATES * L.H, dtype=np.float32)
                b[L.H:2 * L.H] = 1.0
            else:
                b = _uniform(rng, wl.w_scale, (GATES * L.H,)).astype(np.float32)
            P = Tensor(_uniform(rng, wl.w_scale, (L.Hp, L.H)), wl.dtype) if L.Hp else None
            dirs.append(LayerParams(W, R, b, P))
        params.append(dirs)

    I0 = wl.layers[0].I
    if wl.x_dist == "normal":
        x = Tensor(rng.standard_normal((wl.T, wl.B, I0)), wl.dtype)
    else:
        x = Tensor(_uniform(rng, 1.0, (wl.T, wl.B, I0)), wl.dtype)

    h0: List[List[Optional[Tensor]]] = []
    c0: List[List[Optional[np.ndarray]]] = []
    for L in wl.layers:
        hs, cs = [], []
        for _ in range(2 if L.bidirectional else 1):
            if wl.state == "uniform1":
                hs.append(Tensor(_uniform(rng, 1.0, (wl.B, L.Hr)), wl.dtype))
                cs.append(_uniform(rng, 1.0, (wl.B, L.H)).astype(np.float32))
            else:
                hs.append(None)
                cs.append(None)
        h0.append(hs)
        c0.append(cs)

    out = wl.layers[-1].out_width
    if wl.loss == "hT_dot_g":
        g = rng.standard_normal((wl.B, out))
        dyv = np.zeros((wl.T, wl.B, out))
        dyv[wl.T - 1] = g
    else:
        dyv = rng.standard_normal((wl.T, wl.B, out))
    if row_mask is not None:
        dyv[:, ~np.asarray(row_mask, dtype=bool), :] = 0.0
    dy = Tensor(dyv, wl.dtype)
    return Problem(wl, params, x, h0, c0, dy)


def sample_rows_blocks(B: int, seed: int, parts: int = 8, block: int = 16) -> np.ndarray:
    """A seeded sample of batch rows that touches every (part, row block)
    pair of a batch split into `parts` contiguous shares of ceil(B/parts)
    rows, each cut into blocks of `block` rows: per block one random row,
    plus its first row (even blocks) or its last row (odd blocks); the
    batch's first and last rows are always included."""
    rng = np.random.Generator(np.random.PCG64(20_000 + seed))
    share = (B + parts - 1) // parts
    rows = {0, B - 1}
    k = 0
    for p in range(parts):
        lo, hi = p * share, min(B, p * share + share)
        for b0 in range(lo, hi, block):
            b1 = min(hi, b0 + block)
            rows.add(int(rng.integers(b0, b1)))
            rows.add(b0 if k % 2 == 0 else b1 - 1)
            k += 1
    return np.array(sorted(rows), dtype=np.int64)
