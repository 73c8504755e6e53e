"""Hybrid data/model-parallel projection (Section 3 of arXiv 1907.13257,
Equations 1-6), fed with step times measured by this library.

The paper decides between N-way data parallelism (DP) with single-device
workers and N-way DP whose workers are M-way model parallel (MP) by comparing
end-to-end speedups built from three factors: the per-step scaling efficiency
SE_N = T_1 / T_N, the statistical efficiency E_1 / E_N (epochs to converge),
and the per-step MP speedup SU^M.  Epoch counts need the training datasets
and SE_N needs a multi-device all-reduce, so both are inputs here.  SU^M can
be estimated from one device: a 2-stage pipeline over the layer stack
(Section 2, the GPipe-style split the paper uses for GNMT and BigLSTM) runs
its micro-batches at the per-step time this library measures at the
micro-batch size.

    python -m paper_1907_13257_amd.hybrid --sweep bench_B16.json bench_B32.json ...

reads `bench.py` JSON lines of a batch sweep and prints the SU^M estimates.
Host arithmetic only; nothing here touches the GPU.
"""
from __future__ import annotations

import argparse
import json
import math
import sys
from typing import Callable, Dict, Iterable, List, Mapping, Optional, Tuple, Union


def _pos(name: str, v: float) -> float:
    if not (isinstance(v, (int, float)) and math.isfinite(v) and v > 0):
        raise ValueError(f"{name} must be a positive finite number, got {v!r}")
    return float(v)


def training_time(T: float, S: float, E: float) -> float:
    """Equation 1: time to converge = time per step x steps per epoch x epochs."""
    return _pos("T", T) * _pos("S", S) * _pos("E", E)


def dp_speedup_from_times(T1: float, TN: float, S1: float, SN: float, E1: float, EN: float) -> float:
    """Equation 2: N-way DP speedup over one device as the product of the
    per-step, steps-per-epoch and epoch ratios."""
    return (_pos("T1", T1) / _pos("TN", TN)) * (_pos("S1", S1) / _pos("SN", SN)) * (_pos("E1", E1) / _pos("EN", EN))


def dp_speedup(se_n: float, n: int, e1: float, e_n: float) -> float:
    """Equations 3 and 4: SU_N = SE_N x N x E_1 / E_N (constant per-device
    mini-batch, so S_1 / S_N = N)."""
    if int(n) != n or n < 1:
        raise ValueError(f"N must be a positive integer, got {n!r}")
    return _pos("SE_N", se_n) * n * _pos("E_1", e1) / _pos("E_N", e_n)


def hybrid_speedup(su_m: float, se_n: float, n: int, e1: float, e_n: float) -> float:
    """Equation 5: N-way DP of M-way MP workers, SU_N^M = SU^M x SU_N (the
    global batch, and so the epoch count, is that of N-way DP)."""
    return _pos("SU^M", su_m) * dp_speedup(se_n, n, e1, e_n)


def hybrid_threshold(m: int, se_n: float, se_mn: float, e_n: float, e_mn: float) -> float:
    """Right-hand side of Equation 6: the MP speedup above which N x M devices
    are better used as N-way DP of M-way MP workers than as (M x N)-way DP."""
    if int(m) != m or m < 1:
        raise ValueError(f"M must be a positive integer, got {m!r}")
    return m * (_pos("SE_MxN", se_mn) / _pos("SE_N", se_n)) * (_pos("E_N", e_n) / _pos("E_MxN", e_mn))


def hybrid_wins(su_m: float, m: int, se_n: float, se_mn: float, e_n: float, e_mn: float) -> bool:
    """Equation 6: SU^M > M x (SE_{MxN} / SE_N) x (E_N / E_{MxN})."""
    return _pos("SU^M", su_m) > hybrid_threshold(m, se_n, se_mn, e_n, e_mn)


StepTime = Union[Mapping[int, float], Callable[[int], float]]


def _step_time(t: StepTime, b: int) -> float:
    v = t(b) if callable(t) else t.get(b)
    if v is None:
        raise KeyError(f"no step time measured at batch {b}")
    return _pos(f"step time at batch {b}", v)


def pipeline_mp_speedup(step_ms: StepTime, batch: int, micro: int, stages: int = 2, comm_ms: float = 0.0) -> float:
    """SU^M of an M-stage pipeline (M = `stages`) over a stack of equal layers,
    estimated from single-device step times.

    The mini-batch of `batch` rows is cut into `micro` micro-batches.  A stage
    holds 1/M of the layers, so it spends step_ms(batch/micro)/M per
    micro-batch in forward + backward; the schedule fills and drains the
    pipeline once, micro + M - 1 stage slots in all, and `comm_ms` adds the
    activation and gradient transfers between stages on the critical path.
    SU^M = step_ms(batch) / (that time).  With a step time proportional to
    the batch this is micro*M / (micro + M - 1), the pipeline-bubble bound.
    """
    if batch < 1 or micro < 1 or stages < 1 or batch % micro:
        raise ValueError("batch, micro and stages must be positive and micro must divide batch")
    if comm_ms < 0 or not math.isfinite(comm_ms):
        raise ValueError("comm_ms must be finite and non-negative")
    t_full = _step_time(step_ms, batch)
    t_micro = _step_time(step_ms, batch // micro)
    t_pipe = (micro + stages - 1) * t_micro / stages + comm_ms
    return t_full / t_pipe


def best_pipeline(step_ms: Mapping[int, float], batch: int, stages: int = 2,
                  comm_ms: float = 0.0) -> Optional[Tuple[int, float]]:
    """Micro-batch count with the largest estimated SU^M among the measured
    batch sizes (None when no split of `batch` was measured)."""
    best = None
    for micro in range(1, batch + 1):
        if batch % micro or (batch // micro) not in step_ms:
            continue
        su = pipeline_mp_speedup(step_ms, batch, micro, stages, comm_ms)
        if best is None or su > best[1]:
            best = (micro, su)
    return best


def project(epochs: Mapping[int, float], su_m: float, m: int,
            se: Union[float, Mapping[int, float]] = 1.0) -> List[Dict]:
    """For every device count D with E_D known: DP-only speedup SU_D, and the
    hybrid speedup with D/M DP workers of M-way MP when E_{D/M} is known.
    SE defaults to 1, the paper's assumption in its evaluation."""
    if 1 not in epochs:
        raise ValueError("epochs must include E_1")
    e1 = epochs[1]

    def se_of(n: int) -> float:
        return float(se) if not isinstance(se, Mapping) else se[n]

    rows = []
    for d in sorted(epochs):
        row = dict(devices=d, dp=dp_speedup(se_of(d), d, e1, epochs[d]), hybrid=None, hybrid_wins=None)
        if d % m == 0 and (d // m) in epochs:
            n = d // m
            row["hybrid"] = hybrid_speedup(su_m, se_of(n), n, e1, epochs[n])
            row["hybrid_wins"] = hybrid_wins(su_m, m, se_of(n), se_of(d), epochs[n], epochs[d])
        rows.append(row)
    return rows


def step_times_from_bench(lines: Iterable[str]) -> Dict[int, float]:
    """Batch size -> ms per step from `bench.py` JSON lines of one workload
    family (the headline pass without kernel events)."""
    out: Dict[int, float] = {}
    for line in lines:
        line = line.strip()
        if not line.startswith("{"):
            continue
        d = json.loads(line)
        cfg = d.get("config", {})
        if "B" not in cfg or "ms_per_step" not in d:
            continue
        out[int(cfg["B"])] = float(d["ms_per_step"])
    return out


def _parse_epochs(s: str) -> Dict[int, float]:
    out = {}
    for part in s.split(","):
        n, e = part.split(":")
        out[int(n)] = float(e)
    return out


def main(argv: Optional[List[str]] = None) -> int:
    ap = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    ap.add_argument("--sweep", nargs="+", required=True, help="bench.py JSON output files of a batch sweep")
    ap.add_argument("--stages", type=int, default=2, help="M: pipeline stages (devices per worker)")
    ap.add_argument("--comm-ms", type=float, default=0.0, help="inter-stage transfer time per step (ms)")
    ap.add_argument("--epochs", default="", help="epochs to converge per device count, e.g. 1:4,32:4,64:7")
    ap.add_argument("--se", type=float, default=1.0, help="DP scaling efficiency (the paper assumes 1)")
    args = ap.parse_args(argv)
    lines: List[str] = []
    for path in args.sweep:
        with open(path) as f:
            lines.extend(f.read().splitlines())
    t = step_times_from_bench(lines)
    if not t:
        print("no bench results found", file=sys.stderr)
        return 1
    res = {"step_ms": {str(b): t[b] for b in sorted(t)}, "stages": args.stages, "comm_ms": args.comm_ms,
           "su_m": {}}
    for b in sorted(t):
        best = best_pipeline(t, b, args.stages, args.comm_ms)
        if best:
            res["su_m"][str(b)] = {"micro_batches": best[0], "su_m": best[1]}
    if args.epochs:
        ep = _parse_epochs(args.epochs)
        res["projection"] = {}
        for b, v in res["su_m"].items():
            res["projection"][b] = project(ep, v["su_m"], args.stages, args.se)
    print(json.dumps(res, indent=1))
    return 0


if __name__ == "__main__":
    sys.exit(main())
