"""Throughput of the batched predict -> route -> prioritize step on one MI355X.

python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload c4] [--no-cpu-baseline] [--no-chained]
python bench.py --calibrate-copy MIB   (plain device copy of MIB mebibytes, for counter calibration)
python bench.py --sweep-prioritize     (slack ordering alone, W = 2^17 .. 2^26 workflows)
python bench.py --route-fitness        (routing by fitness, Eq. 5, on the workload's predictions)
python bench.py --route-fitness --plans   (the same with C_deg from degradation plans, Alg. 2)
python bench.py --route-fitness --readiness  (T_act per (node, model) from readiness tiers, Sec. III-C)
python bench.py --two-phase            (the two-phase predictor, Sec. III-B, beside the bins one)
python bench.py --margin               (the adaptive safety margin rho, Sec. III-D, over windows)
python bench.py --route-tiered         (latency routing with T_act from readiness tiers beside the plain route)

One step = predict (fused MLP + softmax + expected length + KV bytes) -> route (feasibility,
scores, best nodes) -> prioritize (chain suffix sums, slack keys, stable sort) over one batch
whose inputs are already resident in device memory. The default workload is the largest one:
4,194,304 stages, 4,096 nodes, 64 models, predictor 256-1024-1024-64 in bfloat16, top-4 routes.
It has no workflow chains, so its step is predict -> route; the chained batch (131,072
workflows of 3..8 stages, 719,712 stages, 512 nodes, predictor 256-512-512-64) is timed in the
same run as the full three-phase step and reported under "chained_step". Prints one JSON line.
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
# non-packed float32 vector ALU: 256 CUs x 4 SIMDs x 32 lanes per clock x 2.4 GHz = 78.6 T
# lane-operations/s (the 157.3 TFLOP/s fp32 vector peak counts a multiply-add as two); a probe of
# independent non-packed v_add_f32 chains sustains about 65 T lane-ops/s on the chip
PEAK_VALU_LANE_OPS = 256 * 4 * 32 * 2.4e9
# operations the fitness definition needs per (stage, node) pair: the feasibility compare and
# the eight float32 operations of the score (fit product; gamma, (1 - gamma) products and their
# sum; lambda and mu products and the two differences)
FITNESS_OPS_PER_PAIR = 9


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
    if rec.get("predict_source_sha256_16") != predict_source_hash():
        return None
    return rec.get("records", {}).get(workload, {}).get("hbm_bytes_per_launch")


def calibrate_copy(mib: int, reps: int = 5):
    import torch
    src = torch.empty(mib << 20, dtype=torch.uint8, device="cuda")
    dst = torch.empty_like(src)
    src.fill_(1)
    torch.cuda.synchronize()
    d = _time_events(lambda: dst.copy_(src), reps, 1)
    ms = float(np.median(d))
    gbs = 2 * (mib << 20) / (ms * 1e-3) / 1e9   # bytes read + bytes written
    print(json.dumps({"calibration_copy_bytes": mib << 20, "reps": reps, "copy_ms": round(ms, 4),
                      "copy_gbs": round(gbs, 1), "of_peak": round(gbs / PEAK_HBM_GBS, 4)}), flush=True)


def mlp_flop_per_stage(dims):
    return 2 * sum(dims[i] * dims[i + 1] for i in range(len(dims) - 1))


def cpu_model() -> str:
    """The host CPU as lscpu names it (model name, sockets x cores, threads), else /proc/cpuinfo."""
    import subprocess
    try:
        out = subprocess.run(["lscpu"], capture_output=True, text=True, timeout=10).stdout
        f = {}
        for line in out.splitlines():
            if ":" in line:
                k, v = line.split(":", 1)
                f[k.strip()] = v.strip()
        name = f.get("Model name", "unknown")
        return (f"{name}; {f.get('Socket(s)', '?')} socket(s) x {f.get('Core(s) per socket', '?')} cores x "
                f"{f.get('Thread(s) per core', '?')} threads; family {f.get('CPU family', '?')} model "
                f"{f.get('Model', '?')} stepping {f.get('Stepping', '?')}; {f.get('CPU(s)', '?')} CPUs visible")
    except (OSError, subprocess.SubprocessError):
        pass
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def percentiles(ms):
    a = np.asarray(ms)
    return {"p10": round(float(np.percentile(a, 10)), 4), "p50": round(float(np.median(a)), 4),
            "p90": round(float(np.percentile(a, 90)), 4), "mean": round(float(a.mean()), 4)}


def route_bytes(n, m, k):
    """Algorithmic HBM bytes of routing: per stage model id, predicted length and KV bytes in
    (16 B) and k (node, score) pairs out (8k B); node state once (queue, cold, residency, free:
    24 B per node)."""
    return n * (16 + 8 * k) + 24 * m


def walk_entries(wl, pred, kv, rows, chunk=2048):
    """Mean number of list entries the sorted-walk route visits per stage, over ``rows``: the
    walk goes through its model's nodes in (ready time, index) order, skips nodes whose headroom
    cannot admit the stage, and stops at the first admitting node whose score exceeds its k-th
    best once it holds k nodes. Counted on the host from the same inputs (the kernel keeps no
    counter)."""
    n_nodes, k = wl.spec.n_nodes, wl.spec.k
    assert pred.shape == kv.shape == (wl.n,), "pred and kv of every stage of the batch"
    need = kv.astype(np.float64) * (1.0 + wl.spec.rho) if wl.spec.rho else kv.astype(np.float64)
    exec_s = (pred.astype(np.float32) * wl.decode_s_per_token[wl.model_id]).astype(np.float32)
    bits = (wl.resident_mask[:, None] >> np.arange(wl.spec.n_models, dtype=np.uint64)[None, :]) & np.uint64(1)
    total = 0
    for m in range(wl.spec.n_models):
        ready = np.where(bits[:, m] == 1, wl.queue_s + np.float32(0), wl.queue_s + wl.cold_s).astype(np.float32)
        order = np.lexsort((np.arange(n_nodes), ready))
        r_sorted, f_sorted = ready[order], wl.free_bytes[order]
        sel = rows[wl.model_id[rows] == m]
        for c in range(0, sel.size, chunk):
            s = sel[c:c + chunk]
            feas = need[s][:, None] <= f_sorted[None, :]
            sc = (r_sorted[None, :] + exec_s[s][:, None]).astype(np.float32)
            cnt = np.cumsum(feas, axis=1)
            full = cnt[:, -1] >= k
            kth_pos = np.argmax(cnt >= k, axis=1)
            kth = sc[np.arange(s.size), kth_pos]
            stop = feas & (sc > kth[:, None]) & (np.arange(n_nodes)[None, :] > kth_pos[:, None])
            has_stop = stop.any(axis=1) & full
            visited = np.where(has_stop, np.argmax(stop, axis=1) + 1, n_nodes)
            total += int(visited.sum())
    return total / max(rows.size, 1)


def prioritize_bytes(n_stages, n_workflows, passes=4):
    """Algorithmic HBM bytes of the slack ordering: per stage the latency in (4 B) and the
    remaining time out (8 B); per workflow chain offsets, deadline in and key out (16 + 4 B),
    then per radix pass keys and indices read and written (16 B) and the final order (4 B)."""
    return n_stages * 12 + n_workflows * (20 + passes * 16 + 4)


def cpu_baseline(wl, n_workflows_sample: int, n_stages_sample: int):
    """Oracle (C, OpenMP over stages) on the first workflows (chained batch) or the first stages
    of the batch: predict -> route (-> prioritize), timed on the host cores."""
    import oracle
    W_ = min(n_workflows_sample, wl.n_workflows) if wl.n_workflows else 0
    if W_:
        S = int(wl.chain_offset[W_])
    else:
        S = min(wl.n, n_stages_sample)
    rows = np.arange(S)
    threads = oracle.max_threads()
    t0 = time.perf_counter()
    pred, kv = oracle.predict_workload(wl, rows=rows, n_threads=threads)
    idx, sc = oracle.route_workload(wl, pred, kv, rows=rows, n_threads=threads)
    if W_:
        oracle.prioritize(wl.chain_offset[:W_ + 1], sc[:, 0], wl.deadline_us[:W_], wl.now_us)
    dt = time.perf_counter() - t0
    which = "all" if W_ == wl.n_workflows else "first"
    sample = (f"{which} {W_} workflows ({S} stages) of the same batch: oracle predict + route + prioritize"
              if W_ else f"first {S} of {wl.n} stages of the same batch (a deterministic prefix; every node): "
                         f"oracle predict + route")
    return {"value": S / dt, "unit": "stages/s", "cores": int(threads), "kind": "oracle",
            "sample": sample, "seconds": round(dt, 3), "cpu_model": cpu_model()}


def sweep_prioritize(log2_lo: int, log2_hi: int, steps: int, warmup: int):
    """Slack ordering alone (chain suffix sums, slack keys, stable sort) at growing batch sizes,
    inputs resident on the GPU, one JSON line per size. The chains follow the chained batch's
    recipe: lengths uniform in 3..8 stages, arrival U[0, 600] s, SLO U[10, 120] s, now = 600 s;
    stage latencies are uniform in [0, 60) s (the range of the routed scores)."""
    import torch
    from paper_2606_12950_amd import _native
    torch.cuda.set_device(0)
    gen = torch.Generator(device="cuda")
    for lg in range(log2_lo, log2_hi + 1):
        W_ = 1 << lg
        gen.manual_seed(1000 + lg)
        lens = torch.randint(3, 9, (W_,), generator=gen, device="cuda", dtype=torch.int64)
        off = torch.zeros(W_ + 1, dtype=torch.int64, device="cuda")
        torch.cumsum(lens, 0, out=off[1:])
        S = int(off[-1].item())
        lat = torch.rand(S, generator=gen, device="cuda", dtype=torch.float32) * 60.0
        arrival = torch.randint(0, 600_000_001, (W_,), generator=gen, device="cuda", dtype=torch.int64)
        slo = torch.randint(10_000_000, 120_000_001, (W_,), generator=gen, device="cuda", dtype=torch.int64)
        deadline = arrival + slo
        now_us = 600_000_000
        out = (torch.empty(S, dtype=torch.int64, device="cuda"), torch.empty(W_, dtype=torch.int32, device="cuda"),
               torch.empty(W_, dtype=torch.int32, device="cuda"))
        ws = torch.empty(max(1, _native.prioritize_workspace_bytes(W_, S)), dtype=torch.uint8, device="cuda")
        for _ in range(warmup):
            _native.prioritize(off, lat, deadline, now_us, out=out, workspace=ws)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(steps):
            _native.prioritize(off, lat, deadline, now_us, out=out, workspace=ws)
        e1.record()
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / steps
        pb = prioritize_bytes(S, W_)
        print(json.dumps({"sweep": "prioritize", "n_workflows": W_, "n_stages": S, "ms": round(ms, 4),
                          "workflows_per_s": W_ / (ms * 1e-3), "algorithmic_bytes": pb,
                          "achieved_gbs": round(pb / (ms * 1e-3) / 1e9, 2),
                          "hbm_frac": round(pb / (ms * 1e-3) / 1e9 / PEAK_HBM_GBS, 4)}), flush=True)
        del lens, off, lat, arrival, slo, deadline, out, ws
        torch.cuda.empty_cache()


def _time_events(call, steps: int, warmup: int):
    import torch
    for _ in range(warmup):
        call()
    torch.cuda.synchronize()
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(steps)]
    for e0, e1 in ev:
        e0.record()
        call()
        e1.record()
    torch.cuda.synchronize()
    return [e0.elapsed_time(e1) for e0, e1 in ev]


def inputs_hash(wl) -> str:
    """One digest over the sha256 of every generated input array (by field name)."""
    h = hashlib.sha256()
    for name, digest in sorted(wl.sha256().items()):
        h.update(name.encode())
        h.update(digest.encode())
    return h.hexdigest()[:16]


def oracle_timed(fn, units: int, unit: str, sample: str):
    """The oracle on a bounded sample, timed on the host cores: a cpu_baseline record."""
    import oracle
    t0 = time.perf_counter()
    fn()
    dt = time.perf_counter() - t0
    return {"value": units / dt, "unit": unit, "cores": int(oracle.max_threads()), "kind": "oracle",
            "sample": sample, "seconds": round(dt, 3), "cpu_model": cpu_model()}


def route_fitness_bench(name: str, steps: int, warmup: int, plans: bool = False, readiness: bool = False):
    """Routing by fitness over the workload's stages, on the GPU's own predictions; bounds from
    the recent-observation windows (maestro_quantiles). With ``plans`` C_deg comes from the
    nodes' degradation plans (built once, timed on their own). One JSON line."""
    import torch
    from paper_2606_12950_amd import _native, pipeline
    from paper_2606_12950_amd import workload as W
    torch.cuda.set_device(0)
    wl = W.workload(name)
    f = W.fitness_inputs(wl)
    b = pipeline.to_device(wl)
    o = pipeline.allocate_outputs(b)
    pipeline.run_predict(b, o)
    t = lambda a: pipeline._t(a, "cuda")
    fd = dict(src=t(f.src_id), cls=t(f.class_id), queue=t(f.queue_ms), act=t(f.act_ms), deg=t(f.deg_ms),
              rtt=t(f.rtt_ms), weights=t(f.class_weights))
    extra = {}
    plan_t = None
    if plans:
        e = W.engine_inputs(wl)
        eng = [t(e.engine_offset), t(e.level), t(e.freed_bytes), t(e.cost_ms)]
        plan_t = _native.degradation_plans(*eng, e.c_int_ms)
        dp = _time_events(lambda: _native.degradation_plans(*eng, e.c_int_ms, out=plan_t), steps, warmup)
        deg_window = e.deg_window
        extra = {"plans": True, "n_engines": int(e.level.shape[0]), "plan_ms": percentiles(dp)}
    else:
        deg_window = f.deg_window
    act = None
    if readiness:
        r = W.readiness_inputs(wl)
        rin = [t(r.tier), t(r.model_bytes), t(r.tier_bw), t(r.tier_setup_ms)]
        act = _native.activation_latency(*rin)
        da = _time_events(lambda: _native.activation_latency(*rin, out=act), steps, warmup)
        extra.update({"readiness": True, "activation_ms": percentiles(da)})
    bounds = torch.cat([_native.quantiles(t(f.rtt_window)), _native.quantiles(t(f.ready_window)),
                        _native.quantiles(t(deg_window))])
    n, m = wl.n, wl.spec.n_nodes
    out = (torch.empty((n, wl.spec.k), dtype=torch.int32, device="cuda"),
           torch.empty((n, wl.spec.k), dtype=torch.float32, device="cuda"))
    call = lambda: _native.route_fitness(b.model_id, fd["src"], fd["cls"], o.kv_bytes, b.free_bytes, fd["queue"],
                                         None if readiness else fd["act"], None if readiness else b.resident_mask,
                                         None if plans else fd["deg"], fd["rtt"], fd["weights"], bounds,
                                         n_models=wl.spec.n_models, k=wl.spec.k, rho=wl.spec.rho, plans=plan_t,
                                         act_matrix=act, out=out)
    d = _time_events(call, steps, warmup)
    ms = float(np.mean(d))
    if plans:
        need = o.kv_bytes.double() * (1.0 + wl.spec.rho)
        extra["short_pair_frac"] = round(float((need[:, None] > b.free_bytes[None, :]).float().mean().item()), 4)
    pairs = n * m
    achieved = pairs * FITNESS_OPS_PER_PAIR / (ms * 1e-3)
    import oracle
    S = min(n, max(256, 10_000_000_000 // m))   # the whole batch up to 10^10 pairs (seconds of oracle work)
    kv = o.kv_bytes[:S].cpu().numpy()
    eng = (e.engine_offset, e.level, e.freed_bytes, e.cost_ms, e.c_int_ms) if plans else None
    am = None
    if readiness:
        am = oracle.activation_latency(r.tier, r.model_bytes, r.tier_bw, r.tier_setup_ms)
    bnd = bounds.cpu().numpy()
    extra["cpu_baseline"] = oracle_timed(
        lambda: oracle.route_fitness(wl.model_id[:S], f.src_id[:S], f.class_id[:S], kv, wl.free_bytes, f.queue_ms,
                                     f.act_ms, wl.resident_mask, f.deg_ms, f.rtt_ms, f.class_weights, bnd,
                                     k=wl.spec.k, rho=wl.spec.rho, n_models=wl.spec.n_models, engines=eng,
                                     act_matrix=am),
        S, "stages/s", (f"all {S} stages" if S == n else f"first {S} stages") + f" x all {m} nodes, same inputs")
    print(json.dumps({"route_fitness": name, "n_stages": n, "n_nodes": m, "k": wl.spec.k, "ms": round(ms, 4),
                      "phase_ms": percentiles(d), "stages_per_s": n / (ms * 1e-3), "pairs_per_s": pairs / (ms * 1e-3),
                      "roofline": {"bound": "alu", "achieved": achieved / 1e12, "peak": PEAK_VALU_LANE_OPS / 1e12,
                                   "unit": "T lane-ops/s", "frac": round(achieved / PEAK_VALU_LANE_OPS, 4),
                                   "ops_per_pair": FITNESS_OPS_PER_PAIR},
                      "routed_frac": float((out[0][:, 0] >= 0).float().mean().item()), **extra}), flush=True)


def two_phase_bench(name: str, steps: int, warmup: int):
    """The two-phase predictor (calibrated tool intent, per-role log(1 + L) heads), the per-role
    regressors with weights of their own (grouped GEMM over the stages bucketed by role), and the
    bins predictor on the same network and batch, interleaved; MFMA roofline of each. One JSON
    line."""
    import torch
    from paper_2606_12950_amd import _native, pipeline
    from paper_2606_12950_amd import workload as W
    torch.cuda.set_device(0)
    wl = W.workload(name)
    if wl.spec.dtype != "bf16":
        print("the two-phase predictor is built for the bfloat16 networks (c1 .. c4)", file=sys.stderr)
        sys.exit(2)
    tp = W.two_phase_inputs(wl)
    b = pipeline.to_device(wl)
    o = pipeline.allocate_outputs(b)
    t = lambda a: pipeline._t(a, "cuda")
    ws = b.weights[:-1] + [t(tp.head_weight)]
    bs = b.biases[:-1] + [t(tp.head_bias)]
    tabs = [t(tp.role_head), t(tp.tool_coef), t(tp.iso_x), t(tp.iso_y)]
    role, tools = t(wl.role), t(tp.tool_avail)
    n = wl.n
    out = (torch.empty(n, dtype=torch.float32, device="cuda"), torch.empty(n, dtype=torch.float32, device="cuda"),
           torch.empty(n, dtype=torch.float64, device="cuda"))
    two = lambda: _native.predict_two_phase(b.x, ws, bs, *tabs, tp.max_len, b.prompt_len, b.model_id, role, tools,
                                            b.kv_bytes_per_token, out=out)
    bins = lambda: pipeline.run_predict(b, o)
    # the per-role regressors (second phase, grouped GEMM) on the two-phase outputs; they rewrite
    # the lengths of their stages in place, which every call does identically
    rr = W.role_regressor_inputs(wl)
    rw, rb = [t(a) for a in rr.weights], [t(a) for a in rr.biases]
    rg, rc = t(rr.role_group), t(rr.tool_coef)
    rws = torch.empty(max(256, _native.load().maestro_role_lengths_workspace(n, rr.tool_coef.size)), dtype=torch.uint8,
                      device="cuda")
    two()
    torch.cuda.synchronize()
    roles = lambda: _native.predict_role_lengths(b.x, rw, rb, rg, rc, rr.max_len, b.prompt_len, b.model_id, role,
                                                 out[0], b.kv_bytes_per_token, out[1], out[2], workspace=rws)
    d2 = _time_events(two, steps, warmup)
    d1 = _time_events(bins, steps, warmup)
    dr = _time_events(roles, steps, warmup)
    d2 += _time_events(two, steps, 0)
    d1 += _time_events(bins, steps, 0)
    dr += _time_events(roles, steps, 0)
    flop = mlp_flop_per_stage(wl.spec.dims) * n
    g = np.where((wl.role >= 0) & (wl.role < rr.role_group.size), rr.role_group[np.clip(wl.role, 0, rr.role_group.size - 1)], -1)
    n_roles = int(((g >= 0) & (g < rr.tool_coef.size)).sum())
    flop_roles = mlp_flop_per_stage(wl.spec.dims) * n_roles
    res = {"workload": name, "n_stages": n, "predictor": "-".join(map(str, wl.spec.dims)), "flop_per_launch": flop,
           "role_stages": n_roles, "role_flop_per_launch": flop_roles}
    for key, d, f in (("two_phase", d2, flop), ("bins", d1, flop), ("role_regressors", dr, flop_roles)):
        ms = float(np.mean(d))
        res[key] = {"ms": round(ms, 4), "phase_ms": percentiles(d), "stages_per_s": (n_roles if f == flop_roles else n) / (ms * 1e-3),
                    "roofline": {"bound": "mfma", "achieved": round(f / (ms * 1e-3) / 1e12, 2),
                                 "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                                 "frac": round(f / (ms * 1e-3) / 1e12 / PEAK_BF16_TFLOPS, 4)}}
    res["role_regressors"]["note"] = ("bucketing (count, plan, scatter) and the grouped GEMM over the stages of "
                                      "roles with a regressor; FLOP counted for those stages only")
    res["mean_p_tool"] = float(out[0].mean().item())
    res["mean_pred_len"] = float(out[1].mean().item())
    import oracle
    S = min(n, 65536)
    res["cpu_baseline"] = oracle_timed(
        lambda: oracle.predict_two_phase(wl.x[:S], wl.weights[:-1] + [tp.head_weight], wl.biases[:-1] + [tp.head_bias],
                                         tp.role_head, tp.tool_coef, tp.iso_x, tp.iso_y, tp.max_len, wl.prompt_len[:S],
                                         wl.model_id[:S], wl.role[:S], tp.tool_avail[:S], wl.kv_bytes_per_token,
                                         wl.spec.dtype),
        S, "stages/s", f"first {S} stages, same network and inputs")
    print(json.dumps(res), flush=True)


def route_tiered_bench(name: str, steps: int, warmup: int):
    """Latency routing (Alg. 3, Eq. 6) with T_act per (node, model) from readiness tiers beside the
    resident-bit route, on the workload's own predictions, interleaved. One JSON line."""
    import torch
    from paper_2606_12950_amd import _native, pipeline
    from paper_2606_12950_amd import workload as W
    torch.cuda.set_device(0)
    wl = W.workload(name)
    r = W.readiness_inputs(wl)
    b = pipeline.to_device(wl)
    o = pipeline.allocate_outputs(b)
    pipeline.run_predict(b, o)
    t = lambda a: pipeline._t(a, "cuda")
    rin = [t(r.tier), t(r.model_bytes), t(r.tier_bw), t((r.tier_setup_ms / np.float32(1000)).astype(np.float32))]
    act = _native.activation_latency(*rin, unit=1.0)
    da = _time_events(lambda: _native.activation_latency(*rin, out=act, unit=1.0), steps, warmup)
    n, k = wl.n, wl.spec.k
    out = (torch.empty((n, k), dtype=torch.int32, device="cuda"), torch.empty((n, k), dtype=torch.float32, device="cuda"))
    ws = o.route_workspace
    tiered = lambda: _native.route(b.model_id, o.pred_len, o.kv_bytes, b.decode_s_per_token, b.free_bytes, b.queue_s,
                                   None, None, k=k, rho=wl.spec.rho, out=out, workspace=ws, act_s=act)
    plain = lambda: pipeline.run_route(b, o)
    d_t = _time_events(tiered, steps, warmup) + _time_events(tiered, steps, 0)
    d_p = _time_events(plain, steps, warmup) + _time_events(plain, steps, 0)
    res = {"route_tiered": name, "n_stages": n, "n_nodes": wl.spec.n_nodes, "n_models": wl.spec.n_models, "k": k,
           "activation_ms": percentiles(da), "tiered_ms": percentiles(d_t), "plain_ms": percentiles(d_p),
           "tiered_stages_per_s": n / (float(np.mean(d_t)) * 1e-3),
           "routed_frac": float((out[0][:, 0] >= 0).float().mean().item())}
    import oracle
    S = min(n, max(256, 10_000_000_000 // wl.spec.n_nodes))
    act_np = act.cpu().numpy()
    pred, kv = o.pred_len[:S].cpu().numpy(), o.kv_bytes[:S].cpu().numpy()
    res["cpu_baseline"] = oracle_timed(
        lambda: oracle.route(wl.model_id[:S], pred, kv, wl.decode_s_per_token, wl.free_bytes, wl.queue_s, wl.cold_s,
                             wl.resident_mask, k=k, rho=wl.spec.rho, act_matrix=act_np),
        S, "stages/s", (f"all {S} stages" if S == n else f"first {S} stages") + f" x all {wl.spec.n_nodes} nodes, same inputs")
    print(json.dumps(res), flush=True)


def margin_bench(steps: int, warmup: int):
    """The adaptive safety margin (EWMA of the relative underestimation, then its high quantile)
    over windows of recent stages, and the window bounds (maestro_quantiles) over the same
    lengths. Windows of 32,768 values or more select over 256 workgroups in a workspace,
    preallocated here. One JSON line."""
    import torch
    from paper_2606_12950_amd import _native, pipeline
    from paper_2606_12950_amd import workload as W
    torch.cuda.set_device(0)
    res = {"margin": "adaptive rho", "beta": 0.2, "q": 0.95, "windows": []}
    for m in (4096, 65536, 1 << 20, 1 << 22):
        actual, pred = W.margin_window(3, m)
        a, p = pipeline._t(actual, "cuda"), pipeline._t(pred, "cuda")
        ws = torch.empty(max(_native.quantiles_workspace_bytes(m), 16), dtype=torch.uint8, device="cuda")
        out = _native.adaptive_rho(a, p, 0.2, 0.95, workspace=ws)
        d = _time_events(lambda: _native.adaptive_rho(a, p, 0.2, 0.95, out=out, workspace=ws), steps, warmup)
        qv = out[0].clone()
        qo = _native.quantiles(qv, workspace=ws)
        dq = _time_events(lambda: _native.quantiles(qv, out=qo, workspace=ws), steps, warmup)
        res["windows"].append({"m": m, "ms": percentiles(d), "quantiles_ms": percentiles(dq),
                               "rho": float(out[1].item())})
    import oracle
    actual, pred = W.margin_window(3, 1 << 20)
    res["cpu_baseline"] = oracle_timed(lambda: oracle.adaptive_rho(actual, pred, 0.2, 0.95), 1 << 20,
                                       "stages/s", "the 2^20-stage window (sequential EWMA and sort)")
    print(json.dumps(res), flush=True)


def mfma_ceiling_bench(steps: int, warmup: int, rounds: int = 20000):
    """The chip's matrix-core ceilings: nothing but bfloat16 32x32x16 MFMAs on pseudo-random
    operands, one wavefront per SIMD as the predictor runs, from the measurement-only
    libmaestro_calibrate.so -- both operands in registers (a dependent accumulation chain, and four
    independent accumulators), then the A operand read from LDS for every MFMA (the predictor's
    LDS traffic with one row group) or for every second MFMA (two row groups). What the power limit
    leaves of the 2.5 PFLOP/s datasheet figure with no global memory traffic or synchronisation.
    One JSON line."""
    import ctypes
    import torch
    from paper_2606_12950_amd import build as B
    if not os.path.exists(B.CALIBRATE_LIB):
        raise SystemExit(f"{B.CALIBRATE_LIB} is not built (python -m paper_2606_12950_amd.build)")
    lib = ctypes.CDLL(B.CALIBRATE_LIB)
    lib.maestro_calibrate_mfma.argtypes = [ctypes.c_void_p, ctypes.c_int, ctypes.c_int, ctypes.c_int,
                                           ctypes.c_uint32, ctypes.c_void_p]
    lib.maestro_calibrate_mfma.restype = ctypes.c_int
    lib.maestro_calibrate_mfma_count.argtypes = [ctypes.c_int]
    lib.maestro_calibrate_mfma_count.restype = ctypes.c_int64
    torch.cuda.set_device(0)
    out = torch.empty(lib.maestro_calibrate_mfma_outputs(), dtype=torch.float32, device="cuda")
    stream = torch.cuda.current_stream().cuda_stream
    flop = lib.maestro_calibrate_mfma_count(rounds) * 32768.0
    res = {"mfma_ceiling": "bf16 32x32x16, register operands, one wavefront per SIMD", "rounds": rounds,
           "flop_per_launch": flop, "variants": []}
    for n_acc, lds_every in ((1, 0), (4, 0), (1, 1), (1, 2)):
        def call(n_acc=n_acc, lds_every=lds_every):
            if lib.maestro_calibrate_mfma(ctypes.c_void_p(out.data_ptr()), rounds, n_acc, lds_every, 1, stream) != 0:
                raise RuntimeError("maestro_calibrate_mfma failed")
        ms = percentiles(_time_events(call, steps, warmup))
        tf = flop / (ms["mean"] * 1e-3) / 1e12
        res["variants"].append({"accumulators": n_acc,
                                "a_operand": "registers" if lds_every == 0 else f"LDS, one read per {lds_every} MFMA",
                                "ms": ms, "tflops": round(tf, 1), "frac": round(tf / PEAK_BF16_TFLOPS, 4)})
    print(json.dumps(res), flush=True)


def library_gemm_bench(name: str, steps: int, warmup: int):
    """The vendor GEMM library (hipBLASLt through torch.mm, bfloat16) beside the fused predictor on
    the same GPU: a large square GEMM, the predictor's three layers as separate library GEMMs on
    the workload's batch, and the unfused three-layer network (library GEMMs with bias, ReLU by
    torch, no length epilogue). It says how far the chip's MFMA throughput goes under its power
    limit for plain dense products; the fused kernel is timed last, on the workload's own inputs.
    One JSON line."""
    import torch
    import torch.nn.functional as F
    from paper_2606_12950_amd import workload as W
    torch.cuda.set_device(0)
    torch.manual_seed(0)
    wl = W.workload(name)
    spec, n = wl.spec, wl.n
    if spec.dtype != "bf16" or len(spec.dims) != 4:
        raise SystemExit("--library-gemm compares the bfloat16 three-layer predictor (c1 .. c4)")
    d0, d1, d2, d3 = spec.dims
    res = {"library": "hipBLASLt via torch.mm, bf16", "workload": name, "gemms": []}

    def rec(label, m, k, nn, fn):
        ms = percentiles(_time_events(fn, steps, warmup))
        fl = 2.0 * m * k * nn
        res["gemms"].append({"shape": label, "m": m, "k": k, "n": nn, "ms": ms,
                             "tflops": round(fl / (ms["mean"] * 1e-3) / 1e12, 1),
                             "frac": round(fl / (ms["mean"] * 1e-3) / 1e12 / PEAK_BF16_TFLOPS, 4)})

    a = torch.randn(16384, 16384, device="cuda", dtype=torch.bfloat16)
    b = torch.randn(16384, 16384, device="cuda", dtype=torch.bfloat16)
    rec("square 16384^3", 16384, 16384, 16384, lambda: torch.mm(a, b))
    del a, b
    x = torch.randn(n, d0, device="cuda", dtype=torch.bfloat16)
    ws = [torch.randn(o, i, device="cuda", dtype=torch.bfloat16) * (1.0 / i) ** 0.5
          for i, o in ((d0, d1), (d1, d2), (d2, d3))]
    bs = [torch.zeros(o, device="cuda", dtype=torch.bfloat16) for o in (d1, d2, d3)]
    h1 = F.relu(F.linear(x, ws[0], bs[0]))
    h2 = F.relu(F.linear(h1, ws[1], bs[1]))
    rec(f"layer 1 ({d0}->{d1})", n, d0, d1, lambda: F.linear(x, ws[0], bs[0]))
    rec(f"layer 2 ({d1}->{d2})", n, d1, d2, lambda: F.linear(h1, ws[1], bs[1]))
    rec(f"layer 3 ({d2}->{d3})", n, d2, d3, lambda: F.linear(h2, ws[2], bs[2]))
    del h1, h2

    def mlp():
        h = F.relu(F.linear(x, ws[0], bs[0]))
        h = F.relu(F.linear(h, ws[1], bs[1]))
        return F.linear(h, ws[2], bs[2])
    flop = mlp_flop_per_stage(spec.dims) * n
    ms = percentiles(_time_events(mlp, max(1, steps // 2), warmup))
    res["unfused_network"] = {"ms": ms, "frac": round(flop / (ms["mean"] * 1e-3) / 1e12 / PEAK_BF16_TFLOPS, 4)}
    del x, ws, bs
    torch.cuda.empty_cache()
    st = time_step(wl, steps, warmup)
    mp = float(np.mean(st["predict"]))
    res["fused_predictor"] = {"ms": percentiles(st["predict"]),
                              "frac": round(flop / (mp * 1e-3) / 1e12 / PEAK_BF16_TFLOPS, 4)}
    print(json.dumps(res), flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="c4", choices=["c0", "c1", "c2", "c3", "c4"])
    ap.add_argument("--cpu-sample-workflows", type=int, default=131072)
    ap.add_argument("--cpu-sample-stages", type=int, default=262144,
                    help="stages of a batch without chains that the oracle baseline runs (a prefix)")
    ap.add_argument("--no-chained", action="store_true",
                    help="skip the chained batch's three-phase step after a batch without chains")
    ap.add_argument("--chained-steps", type=int, default=200)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--calibrate-copy", type=int, default=0, metavar="MIB")
    ap.add_argument("--sweep-prioritize", nargs="?", const="17:26", default=None, metavar="LO:HI",
                    help="time the slack ordering alone for W = 2^LO .. 2^HI workflows")
    ap.add_argument("--route-fitness", action="store_true",
                    help="time routing by fitness (Eq. 5) on the workload's predictions")
    ap.add_argument("--plans", action="store_true",
                    help="with --route-fitness: C_deg from degradation plans (Alg. 2, Eq. 4)")
    ap.add_argument("--readiness", action="store_true",
                    help="with --route-fitness: T_act per (node, model) from readiness tiers (Sec. III-C)")
    ap.add_argument("--margin", action="store_true", help="time the adaptive safety margin (Sec. III-D)")
    ap.add_argument("--route-tiered", action="store_true",
                    help="time latency routing with T_act from readiness tiers (Sec. III-C, Eq. 6)")
    ap.add_argument("--two-phase", action="store_true",
                    help="time the two-phase predictor (Sec. III-B) beside the bins predictor")
    ap.add_argument("--n-stages", type=int, default=0, metavar="N",
                    help="replace the workload's stage count (one GPU's share of a batch sharded by stage)")
    ap.add_argument("--n-nodes", type=int, default=0, metavar="M",
                    help="replace the workload's node count (one GPU's share of a batch sharded by node)")
    ap.add_argument("--free-scale", type=float, default=1.0, metavar="S",
                    help="divide every node's free HBM by S (S = 48 on c4: most stage-node pairs infeasible)")
    ap.add_argument("--library-gemm", action="store_true",
                    help="time the vendor GEMM library (square and per-layer bf16 GEMMs, the unfused network) "
                         "beside the fused predictor")
    ap.add_argument("--mfma-ceiling", action="store_true",
                    help="time the matrix-core ceiling kernel (register-only bf16 MFMAs)")
    args = ap.parse_args()

    if args.calibrate_copy:
        calibrate_copy(args.calibrate_copy)
        return
    if args.mfma_ceiling:
        mfma_ceiling_bench(steps=max(2, min(args.steps, 20)), warmup=max(1, min(args.warmup, 3)))
        return
    if args.library_gemm:
        library_gemm_bench(args.workload, steps=max(2, min(args.steps, 20)), warmup=max(1, min(args.warmup, 3)))
        return
    if args.route_tiered:
        route_tiered_bench(args.workload, steps=max(1, min(args.steps, 50)), warmup=max(1, min(args.warmup, 5)))
        return
    if args.margin:
        margin_bench(steps=max(1, min(args.steps, 50)), warmup=max(1, min(args.warmup, 5)))
        return
    if args.two_phase:
        two_phase_bench(args.workload, steps=max(1, min(args.steps, 50)), warmup=max(1, min(args.warmup, 5)))
        return
    if args.route_fitness:
        route_fitness_bench(args.workload, steps=max(1, min(args.steps, 50)), warmup=max(1, min(args.warmup, 5)),
                            plans=args.plans, readiness=args.readiness)
        return
    if args.sweep_prioritize:
        lo, hi = (int(v) for v in args.sweep_prioritize.split(":"))
        sweep_prioritize(lo, hi, steps=max(1, min(args.steps, 20)), warmup=max(1, min(args.warmup, 3)))
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

    overrides = {key: v for key, v in (("n_stages", args.n_stages), ("n_nodes", args.n_nodes)) if v}
    wl = W.workload(args.workload, **overrides)
    if args.free_scale != 1.0:
        wl.free_bytes = wl.free_bytes / args.free_scale
    step = time_step(wl, args.steps, args.warmup)
    line = step_record(wl, step, args.steps)
    if overrides:
        line["config"]["overrides"] = overrides
    if args.free_scale != 1.0:
        line["config"]["free_scale"] = args.free_scale
        rows = np.arange(min(wl.n, 16384))
        need = step["kv"][rows][:, None] * (1.0 + wl.spec.rho)
        line["config"]["infeasible_pair_fraction"] = round(float((need > wl.free_bytes[None, :]).mean()), 4)
    line.update({"metric": METRIC, "value": line.pop("stages_per_s"), "unit": "stages/s", "n_gpus": 1,
                 "steps": args.steps, "warmup": args.warmup, "higher_is_better": True, "scaling": "weak",
                 "vs_baseline": None, "dtype": wl.spec.dtype, "data": "synthetic"})
    order = ["metric", "value", "unit", "n_gpus", "steps", "warmup", "ms_per_step", "higher_is_better", "scaling",
             "vs_baseline", "dtype", "data", "config", "roofline"]
    line = {**{key: line[key] for key in order}, **{key: v for key, v in line.items() if key not in order}}
    if not args.no_cpu_baseline:
        line["cpu_baseline"] = cpu_baseline(wl, args.cpu_sample_workflows, args.cpu_sample_stages)
        if line["route"]["algorithm"] == "sorted walk":
            rows = np.arange(min(wl.n, args.cpu_sample_stages))
            line["route"]["walk_entries_per_stage"] = round(walk_entries(wl, step["pred"], step["kv"], rows), 3)
            line["route"]["walk_sample"] = f"first {rows.size} stages, host count of the walk's stopping rule"
    if wl.n_workflows == 0 and not args.no_chained:
        del step, wl
        torch.cuda.empty_cache()
        cw = W.workload("c3")
        cs = time_step(cw, args.chained_steps, args.warmup)
        rec = step_record(cw, cs, args.chained_steps)
        line["chained_step"] = {key: rec[key] for key in ("stages_per_s", "ms_per_step", "config", "roofline",
                                                          "step_ms", "phase_ms", "route", "prioritize")}
        line["chained_step"]["steps"] = args.chained_steps
    print(json.dumps(line), flush=True)


def time_step(wl, steps: int, warmup: int):
    """Times ``steps`` passes of predict -> route (-> prioritize for chained batches) with the
    batch resident on the GPU: the wall clock of the whole run, bracketed by synchronisation, and
    HIP events on the launch stream around each phase."""
    import torch
    from paper_2606_12950_amd import pipeline
    b = pipeline.to_device(wl)
    o = pipeline.allocate_outputs(b)
    chained = b.chain_offset is not None
    for _ in range(warmup):
        pipeline.run_step(b, o)
    torch.cuda.synchronize()
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(steps):
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
    res = {"wall": t1 - t0, "chained": chained,
           "predict": [e[0].elapsed_time(e[1]) for e in ev], "route": [e[1].elapsed_time(e[2]) for e in ev],
           "prioritize": [e[2].elapsed_time(e[3]) for e in ev],
           "pred": o.pred_len.cpu().numpy(), "kv": o.kv_bytes.cpu().numpy()}
    del b, o
    torch.cuda.empty_cache()
    return res


def step_record(wl, step, steps: int):
    """The measured figures of one timed run: throughput, per-phase event times, the predictor's
    MFMA roofline, route and prioritize bytes."""
    from paper_2606_12950_amd import workload as W
    spec, n = wl.spec, wl.n
    ms_predict = float(np.mean(step["predict"]))
    ms_route = float(np.mean(step["route"]))
    ms_prio = float(np.mean(step["prioritize"]))
    flop = mlp_flop_per_stage(spec.dims) * n
    peak = PEAK_BF16_TFLOPS if spec.dtype == "bf16" else PEAK_F32_TFLOPS
    achieved = flop / (ms_predict * 1e-3) / 1e12
    line = {
        "stages_per_s": n * steps / step["wall"],
        "ms_per_step": step["wall"] / steps * 1e3,
        "config": {
            "workload": f"{spec.name}: {W.DESCRIPTIONS[spec.name]}",
            "n_stages": n, "n_workflows": wl.n_workflows, "n_nodes": spec.n_nodes,
            "n_models": spec.n_models, "predictor": "-".join(map(str, spec.dims)), "route_k": spec.k,
            "inputs_sha256": inputs_hash(wl),
        },
        "roofline": {
            "bound": "mfma", "kernel": "predict (fused MLP + length epilogue)",
            "achieved": round(achieved, 2), "peak": peak, "unit": "TFLOP/s",
            "frac": round(achieved / peak, 4), "traffic": measured_traffic(spec.name),
            "flop_per_launch": flop, "avg_ms": round(ms_predict, 4),
        },
        "step_ms": {"predict": round(ms_predict, 4), "route": round(ms_route, 4)},
        "phase_ms": {"predict": percentiles(step["predict"]), "route": percentiles(step["route"])},
    }
    rb = route_bytes(n, spec.n_nodes, spec.k)
    line["route"] = {
        "algorithm": "sorted walk" if spec.n_nodes <= 8192 and n >= 4 * spec.n_models else "scan",
        "stages_per_s": n / (ms_route * 1e-3), "algorithmic_bytes": rb,
        "achieved_gbs": round(rb / (ms_route * 1e-3) / 1e9, 2),
        "hbm_frac": round(rb / (ms_route * 1e-3) / 1e9 / PEAK_HBM_GBS, 4),
    }
    if step["chained"]:
        pb = prioritize_bytes(n, wl.n_workflows)
        line["step_ms"]["prioritize"] = round(ms_prio, 4)
        line["phase_ms"]["prioritize"] = percentiles(step["prioritize"])
        line["prioritize"] = {
            "workflows_per_s": wl.n_workflows / (ms_prio * 1e-3), "algorithmic_bytes": pb,
            "achieved_gbs": round(pb / (ms_prio * 1e-3) / 1e9, 2),
            "hbm_frac": round(pb / (ms_prio * 1e-3) / 1e9 / PEAK_HBM_GBS, 4),
        }
    else:
        line["prioritize"] = None
    return line


if __name__ == "__main__":
    main()
