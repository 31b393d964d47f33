"""Throughput of the batched predict -> route -> prioritize step on one MI355X.

python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload c3] [--no-cpu-baseline]
python bench.py --calibrate-copy MIB   (plain device copy of MIB mebibytes, for counter calibration)

One step = predict (fused MLP + softmax + expected length + KV bytes) -> route (feasibility,
scores, best node) -> prioritize (chain suffix sums, slack keys, stable sort) over one batch
whose inputs are already resident in device memory. The default workload is the chained
batch: 131,072 workflows of 3..8 stages (719,712 stages), 512 nodes, 16 models, predictor
256-512-512-64 in bfloat16. Prints one JSON line.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "stages predicted+routed/sec on 1 MI355X; % of HBM/MFMA roofline"
PEAK_BF16_TFLOPS = 2500.0      # MI355X dense bf16 MFMA
PEAK_F32_TFLOPS = 157.3        # MI355X dense fp32 MFMA
PEAK_HBM_GBS = 8000.0


TRAFFIC_FILE = os.path.join(ROOT, "profiles", "predict_traffic.json")
PREDICT_SOURCE = os.path.join(ROOT, "paper_2606_12950_amd", "csrc", "predict.hip")


def predict_source_hash() -> str:
    return hashlib.sha256(open(PREDICT_SOURCE, "rb").read()).hexdigest()[:16]


def measured_traffic(workload: str):
    """HBM bytes per predictor launch from the committed counter runs, if they were taken on
    the current kernel source for this workload; else None."""
    try:
        rec = json.load(open(TRAFFIC_FILE))
    except (OSError, ValueError):
        return None
    if rec.get("predict_source_sha256_16") != predict_source_hash() or rec.get("workload") != workload:
        return None
    return rec.get("hbm_bytes_per_launch")


def calibrate_copy(mib: int, reps: int = 5):
    import torch
    src = torch.empty(mib << 20, dtype=torch.uint8, device="cuda")
    dst = torch.empty_like(src)
    src.fill_(1)
    torch.cuda.synchronize()
    for _ in range(reps):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"calibration_copy_bytes": mib << 20, "reps": reps}), flush=True)


def mlp_flop_per_stage(dims):
    return 2 * sum(dims[i] * dims[i + 1] for i in range(len(dims) - 1))


def cpu_baseline(wl, n_workflows_sample: int):
    """Oracle (C, OpenMP over stages) on the first workflows of the batch: predict -> route ->
    prioritize, timed on the host cores."""
    import oracle
    W_ = min(n_workflows_sample, wl.n_workflows) if wl.n_workflows else 0
    if W_:
        S = int(wl.chain_offset[W_])
    else:
        S = min(wl.n, n_workflows_sample * 5)
    rows = np.arange(S)
    threads = oracle.max_threads()
    t0 = time.perf_counter()
    pred, kv = oracle.predict_workload(wl, rows=rows, n_threads=threads)
    idx, sc = oracle.route_workload(wl, pred, kv, rows=rows, n_threads=threads)
    if W_:
        oracle.prioritize(wl.chain_offset[:W_ + 1], sc[:, 0], wl.deadline_us[:W_], wl.now_us)
    dt = time.perf_counter() - t0
    sample = (f"first {W_} workflows ({S} stages) of the same batch: oracle predict + route + prioritize"
              if W_ else f"first {S} stages of the same batch: oracle predict + route")
    return {"value": S / dt, "unit": "stages/s", "cores": int(threads), "kind": "oracle",
            "sample": sample, "seconds": round(dt, 3)}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--workload", default="c3", choices=["c0", "c1", "c2", "c3", "c4"])
    ap.add_argument("--cpu-sample-workflows", type=int, default=65536)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--calibrate-copy", type=int, default=0, metavar="MIB")
    args = ap.parse_args()

    if args.calibrate_copy:
        calibrate_copy(args.calibrate_copy)
        return

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: the batched scheduling step runs on a single "
              "MI355X (see the multi-GPU design notes); run it with --gpus 1.", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2606_12950_amd import pipeline
    from paper_2606_12950_amd import workload as W

    if not torch.cuda.is_available():
        print("no GPU visible", file=sys.stderr)
        sys.exit(1)
    torch.cuda.set_device(0)

    wl = W.workload(args.workload)
    spec = wl.spec
    b = pipeline.to_device(wl)
    o = pipeline.allocate_outputs(b)
    chained = b.chain_offset is not None

    for _ in range(args.warmup):
        pipeline.run_step(b, o)
    torch.cuda.synchronize()

    K = args.steps
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(K)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(K):
        e = ev[i]
        e[0].record()
        pipeline.run_predict(b, o)
        e[1].record()
        pipeline.run_route(b, o)
        e[2].record()
        if chained:
            pipeline.run_prioritize(b, o)
        e[3].record()
    torch.cuda.synchronize()
    t1 = time.perf_counter()

    wall = t1 - t0
    ms_predict = float(np.mean([e[0].elapsed_time(e[1]) for e in ev]))
    ms_route = float(np.mean([e[1].elapsed_time(e[2]) for e in ev]))
    ms_prio = float(np.mean([e[2].elapsed_time(e[3]) for e in ev]))

    n = wl.n
    flop = mlp_flop_per_stage(spec.dims) * n
    peak = PEAK_BF16_TFLOPS if spec.dtype == "bf16" else PEAK_F32_TFLOPS
    achieved = flop / (ms_predict * 1e-3) / 1e12
    line = {
        "metric": METRIC,
        "value": n * K / wall,
        "unit": "stages/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": args.warmup,
        "ms_per_step": wall / K * 1e3,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": spec.dtype,
        "data": "synthetic",
        "config": {
            "workload": f"{spec.name}: {W.DESCRIPTIONS[spec.name]}",
            "n_stages": n, "n_workflows": wl.n_workflows, "n_nodes": spec.n_nodes,
            "n_models": spec.n_models, "predictor": "-".join(map(str, spec.dims)), "route_k": spec.k,
        },
        "roofline": {
            "bound": "mfma", "kernel": "predict (fused MLP + length epilogue)",
            "achieved": round(achieved, 2), "peak": peak, "unit": "TFLOP/s",
            "frac": round(achieved / peak, 4), "traffic": measured_traffic(spec.name),
            "flop_per_launch": flop, "avg_ms": round(ms_predict, 4),
        },
        "step_ms": {"predict": round(ms_predict, 4), "route": round(ms_route, 4),
                    "prioritize": round(ms_prio, 4)},
    }
    if not args.no_cpu_baseline:
        line["cpu_baseline"] = cpu_baseline(wl, args.cpu_sample_workflows)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
