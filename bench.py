#!/usr/bin/env python3
"""Throughput of the per-worker LSTM training step (forward + BPTT + all
gradients) on one MI355X.

Default workload: the GNMT-shaped encoder stack of 4 unidirectional LSTM
layers, input 1024, hidden 1024, T=50, mini-batch B=128, bf16 storage with
fp32 accumulation (the headline configuration).  Inputs are seeded synthetic
tensors already resident in HBM when timing starts.

Prints one JSON line.  `value` is FLOP/s of the whole step (2*M*N*K over
every matrix product of forward, BPTT and gradients) in TFLOP/s.
`roofline` describes the kernel class with the largest share of the timed
region, timed with HIP events the library records around each launch on
the stream it runs on.  `cpu_baseline` times the fp64 oracle on a bounded
sample of the same workload (a subset of the batch rows) on the host cores.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2516.6     # MI355X dense bf16 matrix peak (256 CUs x 4096 FLOP/clk x 2.4 GHz)
PEAK_F32_TFLOPS = 157.3       # MI355X fp32 matrix peak
PEAK_HBM_GBS = 8000.0         # MI355X HBM3E
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic.json")
GEMM_CLASSES = ("gemm_input_proj", "gemm_dx", "gemm_dw", "gemm_dr", "gemm_dw_dr", "gemm_dp")


def recurrence_model_bytes(wl, cls: str, launches_per_step: float):
    """Algorithmic HBM bytes of one launch of a per-layer recurrence, in the
    byte model of the training step: per step and batch row the forward reads
    Gx_t and writes the activated gates (4H values each, fp32), c_t (fp32)
    and h_t (bf16); the backward reads the gates and c_t (fp32) and dy_t
    (bf16) and writes dz_t (4H, bf16); the recurrent weights are read once
    (bf16).  The kernels keep Gx and the gates in fp16 where the layer allows
    it, so they move fewer bytes than this model counts for the same work
    (their own count is the kernel class's `gbs`).  None where a launch is
    not one plain-LSTM layer (the layer wavefront, LSTMP layers)."""
    if cls not in ("recurrent_fwd", "recurrent_bwd"):
        return None
    dirs = sum(2 if L.bidirectional else 1 for L in wl.layers)
    if any(L.Hp for L in wl.layers) or abs(launches_per_step - dirs) > 1e-9:
        return None
    Hs = {L.H for L in wl.layers}
    if len(Hs) != 1:
        return None
    H = Hs.pop()
    per_row = (4 * H * 4 + 4 * H * 4 + H * 4 + H * 2) if cls == "recurrent_fwd" else \
              (4 * H * 4 + H * 4 + H * 2 + 4 * H * 2)
    return float(wl.T) * wl.B * per_row + 4.0 * H * H * 2


def kernel_source_hash() -> str:
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_1907_13257_amd", "csrc")
    for name in sorted(os.listdir(csrc)):
        with open(os.path.join(csrc, name), "rb") as f:
            h.update(name.encode())
            h.update(f.read())
    return h.hexdigest()[:16]


def make_workload(args):
    import synth
    if args.workload == "gnmt4":
        return synth.gnmt4(B=args.batch or 128, seed=1 if not args.batch or args.batch == 128 else 2)
    if args.workload == "biglstm":
        return synth.biglstm(B=args.batch or 128)
    if args.workload == "gnmt8":
        return synth.gnmt8(B=args.batch or 256)
    if args.workload == "floor":
        return synth.floor(B=args.batch or 8)
    raise SystemExit(f"unknown workload {args.workload}")


def workload_name(wl) -> str:
    L0 = wl.layers[0]
    kinds = {"gnmt4": "gnmt4_lstm", "biglstm": "biglstm_lstmp", "gnmt8": "gnmt8_bi_residual_lstm",
             "floor": "sync_floor_lstm"}
    base = kinds.get(wl.name.split("_B")[0], wl.name)
    hp = f"_P{L0.Hp}" if L0.Hp else ""
    return f"{base}_L{len(wl.layers)}_I{L0.I}_H{L0.H}{hp}_T{wl.T}_B{wl.B}"


def _cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def _oracle_step_seconds(prob, sel):
    """Wall time of one oracle forward + backward of the stack on batch rows `sel`."""
    import oracle
    sys.path.insert(0, os.path.join(ROOT, "tests"))
    from _gpu_helpers import oracle_layers
    layers = oracle_layers(prob)
    if len(sel) < prob.wl.B:
        from _gpu_helpers import _rows_of
        layers = [oracle.LayerDef([_rows_of(p, sel) for p in L.dirs], L.residual) for L in layers]
    x = prob.x.f64[:, sel]
    dy = prob.dy.f64[:, sel]
    t0 = time.perf_counter()
    oracle.stack_forward(x, layers)
    oracle.stack_backward(x, layers, dy)
    return time.perf_counter() - t0


def cpu_baseline(wl, rows: int):
    """The oracle, untuned, on the first `rows` batch rows of the same
    workload (rows are independent, so the work per row is the full
    problem's) with every host core; reported in the same unit as `value`.
    Also one thread on one row of the same workload and on the tiny
    configuration (forward + backward, whole problem)."""
    import numpy as np
    import oracle
    import synth

    prob = synth.draw(wl)
    sel = np.arange(min(rows, wl.B))
    threads = oracle.num_threads()
    dt = _oracle_step_seconds(prob, sel)
    frac = len(sel) / wl.B
    flops = wl.gemm_flops() * frac
    oracle.set_num_threads(1)
    try:
        dt1 = _oracle_step_seconds(prob, np.arange(1))
        tiny = synth.tiny("f32")
        dtt = min(_oracle_step_seconds(synth.draw(tiny), np.arange(tiny.B)) for _ in range(3))
    finally:
        oracle.set_num_threads(threads)
    return {"value": flops / dt / 1e12, "unit": "TFLOP/s", "cores": threads, "kind": "oracle",
            "sample": f"{len(sel)} of {wl.B} batch rows of the same stack (all layers, all {wl.T} steps), "
                      f"forward + backward, fp64; {dt:.1f} s wall",
            "nproc": os.cpu_count(), "cpu_model": _cpu_model(),
            "single_thread": {
                "value": wl.gemm_flops() / wl.B / dt1 / 1e12, "unit": "TFLOP/s",
                "sample": f"1 of {wl.B} batch rows of the same stack, 1 thread; {dt1:.1f} s wall",
                "tiny_config_ms_per_step": dtt * 1e3,
                "tiny_config": "1 layer, T=8, B=4, I=32, H=64, forward + backward, 1 thread"}}


# Kernel classes whose launches are one kernel each, by kernel-name prefixes
# (for attributing the per-dispatch counter values to a class): the XCD-local
# recurrences, or the layer wavefront's at small batches.
CLASS_KERNELS = {"recurrent_fwd": ("lstm_fwd_xcd", "lstm_fwd_wave"), "recurrent_bwd": ("lstm_bwd_xcd", "lstm_bwd_wave")}


def _short_kernel(name: str) -> str:
    import re
    name = name.replace("lstm355::(anonymous namespace)::", "").replace("void ", "")
    return re.sub(r"\(.*$", "", name)


def _counter_avgs(path: str):
    """Per kernel name: (dispatches, average counter value) of a rocprofv3
    counter-collection CSV holding one counter."""
    import collections
    import csv
    agg = collections.defaultdict(list)
    with open(path) as f:
        for r in csv.DictReader(f):
            agg[_short_kernel(r["Kernel_Name"])].append(float(r["Counter_Value"]))
    return {k: (len(v), sum(v) / len(v)) for k, v in agg.items()}


def traffic_from(pmc_dir: str, workload: str, copy_mib: int):
    """Writes profiles/traffic.json from four rocprofv3 --pmc runs under
    pmc_dir: fetch/ and write/ (FETCH_SIZE, WRITE_SIZE of the benchmark
    step) and cfetch/ and cwrite/ (the same counters for a plain copy of
    copy_mib MiB, which fixes the scale of each counter: KiB counted per KiB
    actually moved)."""
    def one(sub):
        import glob
        files = glob.glob(os.path.join(pmc_dir, sub, "**", "*counter_collection.csv"), recursive=True)
        if not files:
            raise SystemExit(f"no counter_collection.csv under {os.path.join(pmc_dir, sub)}")
        return _counter_avgs(files[0])
    fetch, write, cfetch, cwrite = one("fetch"), one("write"), one("cfetch"), one("cwrite")
    copy_kib = copy_mib * 1024.0
    cf = [v for k, (n, v) in cfetch.items() if "copyBuffer" in k]
    cw = [v for k, (n, v) in cwrite.items() if "copyBuffer" in k]
    fetch_factor = copy_kib / max(cf)
    write_factor = copy_kib / max(cw)
    by_name = {}
    for k in fetch:
        if k in write:
            by_name[k] = (fetch[k][1] * fetch_factor + write[k][1] * write_factor) * 1024.0
    kernels = {}
    for cls, prefixes in CLASS_KERNELS.items():
        hits = [v for k, v in by_name.items() if k.startswith(prefixes)]
        if len(hits) == 1:
            kernels[cls] = {"hbm_bytes_per_launch": hits[0]}
    # one record per workload, all taken on the same kernel sources
    out = {"source_hash": kernel_source_hash(), "workloads": {}}
    if os.path.exists(TRAFFIC_FILE):
        with open(TRAFFIC_FILE) as f:
            old = json.load(f)
        if old.get("source_hash") == out["source_hash"]:
            out["workloads"] = old.get("workloads", {})
    out["workloads"][workload] = {"fetch_factor": fetch_factor, "write_factor": write_factor,
                                  "copy_bytes": copy_mib * (1 << 20), "kernels": kernels,
                                  "bytes_per_dispatch_by_kernel": by_name}
    with open(TRAFFIC_FILE, "w") as f:
        json.dump(out, f, indent=1, sort_keys=True)
    print(json.dumps({"traffic_file": TRAFFIC_FILE, "workload": workload, "kernels": kernels,
                      "fetch_factor": fetch_factor, "write_factor": write_factor}))


def traffic_for(workload: str, cls: str):
    """HBM bytes per launch of kernel class `cls` counted for `workload` on the
    current kernel sources, or None."""
    if not os.path.exists(TRAFFIC_FILE):
        return None
    with open(TRAFFIC_FILE) as f:
        tr = json.load(f)
    if tr.get("source_hash") != kernel_source_hash():
        return None
    ent = tr.get("workloads", {}).get(workload, {}).get("kernels", {}).get(cls)
    return ent.get("hbm_bytes_per_launch") if ent else None


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="gnmt4", choices=["gnmt4", "biglstm", "gnmt8", "floor"])
    ap.add_argument("--batch", type=int, default=0)
    ap.add_argument("--cpu-rows", type=int, default=16, help="batch rows for the oracle baseline (0: skip)")
    ap.add_argument("--no-profile", action="store_true", help="time without per-kernel events")
    ap.add_argument("--copy-calibration", type=int, default=0,
                    help="only run a plain torch copy of this many MiB (counter calibration) and exit")
    ap.add_argument("--traffic-from", default="",
                    help="write profiles/traffic.json from rocprofv3 --pmc runs in this directory and exit "
                         "(no GPU needed)")
    args = ap.parse_args()

    if args.traffic_from:
        import synth  # noqa: F401
        traffic_from(args.traffic_from, workload_name(make_workload(args)), 256)
        return

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py measures one GPU only: the library has no multi-GPU path "
              "(the data-parallel all-reduce is out of scope); run with --gpus 1", file=sys.stderr)
        sys.exit(2)

    import torch
    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(2)
    torch.cuda.set_device(0)

    if args.copy_calibration:
        n = args.copy_calibration * (1 << 20) // 4
        a = torch.ones(n, dtype=torch.float32, device="cuda")
        b = torch.empty_like(a)
        for _ in range(5):
            b.copy_(a)
        torch.cuda.synchronize()
        print(json.dumps({"copy_bytes_each_way": n * 4, "launches": 5}))
        return

    import synth
    from paper_1907_13257_amd import Stack, lstm355
    from synth.device import device_params, stack_layers, to_dev

    wl = make_workload(args)
    prob = synth.draw(wl)
    stack = Stack(wl.T, wl.B, stack_layers(wl), wl.dtype)
    params = device_params(prob)
    grads = stack.alloc_grads(params)
    x = to_dev(prob.x)
    dy = to_dev(prob.dy)
    tiling = [L.tiling() for L in stack.dirs[0]]

    def step():
        stack.forward(x, params)
        stack.backward(dy, params, grads)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    st = stack.check()
    if st != 0:
        raise SystemExit(f"watchdog tripped during warmup ({lstm355.lstm_status_string(st)})")

    # uninstrumented timing: wall clock over all steps, and one pair of HIP
    # events per step on the stream the library runs on (median, min, p90)
    cur = torch.cuda.current_stream()
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for e0, e1 in evs:
        e0.record(cur)
        step()
        e1.record(cur)
    torch.cuda.synchronize()
    ms_plain = (time.perf_counter() - t0) * 1e3 / args.steps
    per_step = sorted(e0.elapsed_time(e1) for e0, e1 in evs)

    def pct(q):
        return per_step[min(len(per_step) - 1, int(round(q * (len(per_step) - 1))))]
    step_stats = {"median": pct(0.5), "min": per_step[0], "p90": pct(0.9), "max": per_step[-1]}

    # timed region with per-kernel events
    prof = not args.no_profile
    if prof:
        lstm355.lstm_profile_reset()
        lstm355.lstm_profile_enable(True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    ms = (time.perf_counter() - t0) * 1e3 / args.steps
    stats = {}
    if prof:
        lstm355.lstm_profile_enable(False)
        stats = lstm355.lstm_profile_read()
        lstm355.lstm_profile_reset()
    st = stack.check()
    if st != 0:
        raise SystemExit(f"watchdog tripped ({lstm355.lstm_status_string(st)})")

    flops = wl.gemm_flops()
    peak = PEAK_BF16_TFLOPS if wl.dtype == "bf16" else PEAK_F32_TFLOPS
    # the headline is the uninstrumented pass; the instrumented one gives the
    # per-kernel times (its events cost a few percent of the step)
    tflops = flops / (ms_plain / 1e3) / 1e12

    kernels = {}
    for name, s in stats.items():
        avg = s["total_ms"] / s["launches"]
        kernels[name] = dict(launches_per_step=s["launches"] / args.steps, ms_per_step=s["total_ms"] / args.steps,
                             avg_launch_ms=avg,
                             tflops=(s["flops"] / s["launches"]) / (avg / 1e3) / 1e12 if avg > 0 else None,
                             gbs=(s["bytes"] / s["launches"]) / (avg / 1e3) / 1e9 if avg > 0 else None)
    roofline = None
    gemm_summary = None
    if stats:
        dom = max(stats, key=lambda k: stats[k]["total_ms"])
        s = stats[dom]
        avg_s = s["total_ms"] / s["launches"] / 1e3
        traffic = traffic_for(workload_name(wl), dom)
        if dom in GEMM_CLASSES:
            ach = s["flops"] / s["launches"] / avg_s / 1e12
            roofline = {"kernel": dom, "bound": "mfma", "achieved": ach, "peak": peak, "unit": "TFLOP/s",
                        "frac": ach / peak, "traffic": traffic}
        else:
            kernel_bytes = s["bytes"] / s["launches"]
            alg_bytes = recurrence_model_bytes(wl, dom, s["launches"] / args.steps) or kernel_bytes
            ach = alg_bytes / avg_s / 1e9
            roofline = {"kernel": dom, "bound": "hbm", "achieved": ach, "peak": PEAK_HBM_GBS, "unit": "GB/s",
                        "frac": ach / PEAK_HBM_GBS, "traffic": traffic,
                        "bytes_per_launch": alg_bytes, "kernel_bytes_per_launch": kernel_bytes}
            if dom.startswith("recurrent"):
                # HBM is the only roofline that applies to the recurrences, but
                # their counters (matrix cores and LDS a fraction busy, traffic
                # far below peak) show the per-step wait between workgroups sets
                # their time
                roofline["limited_by"] = "per-step latency of the exchange between workgroups"
        gf = sum(stats[k]["flops"] for k in GEMM_CLASSES if k in stats)
        gt = sum(stats[k]["total_ms"] for k in GEMM_CLASSES if k in stats)
        if gt > 0:
            g_tf = gf / (gt / 1e3) / 1e12
            gemm_summary = {"tflops": g_tf, "frac_of_peak": g_tf / peak, "ms_per_step": gt / args.steps}

    cpu = None
    if args.cpu_rows:
        cpu = cpu_baseline(wl, args.cpu_rows)

    out = {
        "metric": "LSTM fwd+BPTT ms/step and TFLOP/s (% bf16 MFMA peak), 4x1024 B=128 T=50",
        "value": tflops,
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_plain,
        "ms_per_step_events": step_stats,
        "ms_per_step_with_kernel_events": ms,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": wl.dtype,
        "data": "synthetic (seeded; x, dy ~ N(0,1), weights ~ U(-a,a))",
        "config": {"workload": workload_name(wl), "layers": len(wl.layers), "T": wl.T, "B": wl.B,
                   "I": wl.layers[0].I, "H": wl.layers[0].H, "Hp": wl.layers[0].Hp,
                   "step_gflop": flops / 1e9, "parallelism": "single GPU (per-worker step)"},
        "frac_of_peak_whole_step": tflops / peak,
        "gemm": gemm_summary,
        "roofline": roofline,
        "kernels": kernels,
        "tiling_layer0": tiling,
        "cpu_baseline": cpu,
    }
    print(json.dumps(out))


if __name__ == "__main__":
    main()
