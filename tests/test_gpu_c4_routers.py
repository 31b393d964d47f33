"""Parity at the largest workload's shape (4,194,304 stages x 4,096 nodes, 64 models, top-4) for
the routers beyond the plain latency route: fitness routing (Eq. 5, Alg. 3) with the nodes'
reported C_deg, with degradation plans (Alg. 2, Eq. 4), with T_act from readiness tiers (Eq. 6),
and with both; and the latency route with T_act from tiers, both algorithms. Each router runs
one full launch on the GPU, in the launch configuration the benchmark times; the oracle checks
20,000 sampled stages plus the first and the last, given the same inputs (the GPU's own
predictions, GPU-computed activation latencies that are first checked bit for bit against the
oracle's). Bars: node indices and fitness or score values bit-exact."""
import numpy as np
import pytest
import torch

import oracle
import paper_2606_12950_amd as M
from paper_2606_12950_amd import pipeline
from paper_2606_12950_amd import workload as W

pytestmark = pytest.mark.gpu


def _t(a):
    return pipeline._t(np.ascontiguousarray(a), "cuda")


def _np(t):
    return t.detach().cpu().numpy()


@pytest.fixture(scope="module")
def c4():
    w = W.workload("c4")
    b = pipeline.to_device(w)
    o = pipeline.allocate_outputs(b)
    pipeline.run_predict(b, o)
    torch.cuda.synchronize()
    pred, kv = _np(o.pred_len), _np(o.kv_bytes)
    del b, o
    torch.cuda.empty_cache()
    rows = np.sort(np.random.default_rng(44).choice(w.n, 20000, replace=False))
    rows = np.unique(np.concatenate([rows, [0, w.n - 1]]))
    print(f"c4: {w.n} stages x {w.free_bytes.size} nodes, {w.spec.n_models} models, k = {w.spec.k}", flush=True)
    return w, pred, kv, rows


def _activation(r, unit, setup):
    act = M.activation_latency(_t(r.tier), _t(r.model_bytes), _t(r.tier_bw), _t(setup), unit=unit)
    torch.cuda.synchronize()
    act = _np(act)
    ref = oracle.activation_latency(r.tier, r.model_bytes, r.tier_bw, setup, unit=unit)
    assert np.array_equal(act.view(np.uint32), ref.view(np.uint32))
    return act


def _assert_rows_equal(gi, gv, ri, rv, what):
    bad = np.flatnonzero((gi != ri).any(axis=1) | (gv.view(np.uint32) != rv.view(np.uint32)).any(axis=1))
    assert bad.size == 0, f"{what}: {bad.size} sampled stages differ, first: gpu {gi[bad[0]]} {gv[bad[0]]} " \
                          f"oracle {ri[bad[0]]} {rv[bad[0]]}"


@pytest.mark.parametrize("plans,readiness", [(False, False), (True, False), (False, True), (True, True)])
def test_fitness_c4_sampled_stages(c4, plans, readiness):
    w, _, kv, rows = c4
    f = W.fitness_inputs(w)
    K, k = w.spec.n_models, w.spec.k
    e = W.engine_inputs(w) if plans else None
    r = W.readiness_inputs(w) if readiness else None
    act = _activation(r, 1000.0, r.tier_setup_ms) if readiness else None
    deg_window = e.deg_window if plans else f.deg_window
    bounds = np.concatenate([oracle.quantiles(f.rtt_window), oracle.quantiles(f.ready_window),
                             oracle.quantiles(deg_window)]).astype(np.float32)
    eng = (e.engine_offset, e.level, e.freed_bytes, e.cost_ms, e.c_int_ms) if plans else None
    gplans = M.degradation_plans(_t(e.engine_offset), _t(e.level), _t(e.freed_bytes), _t(e.cost_ms),
                                 e.c_int_ms) if plans else None
    idx, fit = M.route_fitness(_t(w.model_id), _t(f.src_id), _t(f.class_id), _t(kv), _t(w.free_bytes),
                               _t(f.queue_ms), None if readiness else _t(f.act_ms),
                               None if readiness else _t(w.resident_mask), None if plans else _t(f.deg_ms),
                               _t(f.rtt_ms), _t(f.class_weights), _t(bounds), n_models=K, k=k, rho=w.spec.rho,
                               plans=gplans, act_matrix=_t(act) if readiness else None)
    torch.cuda.synchronize()
    gi, gf = _np(idx)[rows], _np(fit)[rows]
    ri, rf = oracle.route_fitness(w.model_id[rows], f.src_id[rows], f.class_id[rows], kv[rows], w.free_bytes,
                                  f.queue_ms, f.act_ms, w.resident_mask, f.deg_ms, f.rtt_ms, f.class_weights, bounds,
                                  k=k, rho=w.spec.rho, n_models=K, engines=eng, act_matrix=act)
    _assert_rows_equal(gi, gf, ri, rf, f"fitness plans={plans} readiness={readiness}")
    if plans:   # the plan path is exercised: some sampled stages fall short on some node
        assert (kv[rows][:, None] > w.free_bytes[None, :]).any(axis=1).mean() > 0.1
    print(f"fitness c4 plans={plans} readiness={readiness}: {(gi[:, 0] >= 0).mean():.4f} of sampled stages "
          f"routed, {rows.size} stages identical", flush=True)


@pytest.mark.parametrize("algo", ["scan", "sorted"])
def test_route_tiered_c4_sampled_stages(c4, algo):
    w, pred, kv, rows = c4
    r = W.readiness_inputs(w)
    act = _activation(r, 1.0, (r.tier_setup_ms / np.float32(1000)).astype(np.float32))
    k = w.spec.k
    idx, sc = M.route(_t(w.model_id), _t(pred), _t(kv), _t(w.decode_s_per_token), _t(w.free_bytes), _t(w.queue_s),
                      None, None, k=k, rho=w.spec.rho, algo={"scan": M._native.ROUTE_SCAN, "sorted": M._native.ROUTE_SORTED}[algo],
                      act_s=_t(act))
    torch.cuda.synchronize()
    gi, gs = _np(idx)[rows], _np(sc)[rows]
    ri, rs = oracle.route(w.model_id[rows], pred[rows], kv[rows], w.decode_s_per_token, w.free_bytes, w.queue_s,
                          w.cold_s, w.resident_mask, k=k, rho=w.spec.rho, act_matrix=act)
    _assert_rows_equal(gi, gs, ri, rs, f"tiered route {algo}")
