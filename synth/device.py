"""Moves seeded synthetic tensors to the GPU and back (torch supplies the
device memory).  Holds no arithmetic of the method and imports nothing from
the oracle, so the benchmark's GPU path can use it."""
from __future__ import annotations

import numpy as np

from . import Problem, Tensor, Workload, bf16_bits_to_f64


def to_dev(t, device="cuda"):
    import torch
    if t is None:
        return None
    if isinstance(t, Tensor):
        if t.dtype == "bf16":
            return torch.from_numpy(t.dev.view(np.int16)).view(torch.bfloat16).to(device)
        return torch.from_numpy(t.dev).to(device)
    return torch.from_numpy(np.ascontiguousarray(t)).to(device)


def to_f64(x) -> np.ndarray:
    import torch
    x = x.detach()
    if x.dtype == torch.bfloat16:
        return bf16_bits_to_f64(x.contiguous().view(torch.int16).cpu().numpy().view(np.uint16))
    return x.double().cpu().numpy()


def stack_layers(wl: Workload):
    from paper_1907_13257_amd import StackLayer
    return [StackLayer(L.I, L.H, L.Hp, L.bidirectional, L.residual) for L in wl.layers]


def device_params(prob: Problem):
    params = []
    for li, L in enumerate(prob.wl.layers):
        dl = []
        for p in prob.params[li]:
            d = dict(W=to_dev(p.W), R=to_dev(p.R), b=to_dev(p.b))
            if p.P is not None:
                d["P"] = to_dev(p.P)
            dl.append(d)
        params.append(dl)
    return params
