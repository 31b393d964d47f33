"""Stages whose per-stage ids are out of range, through the C-ABI: the model id that Eq. 3 and the
routers (Alg. 3, Eq. 5 and 6) read, and the source and class ids of fitness routing. Each such
stage is flagged -- a NaN KV demand from predict (its length unchanged), no node from the routers
(node -1; score +inf, fitness -inf) -- and every other stage's result equals the oracle's on the
in-range stages alone (routing is stage by stage)."""
import numpy as np
import pytest
import torch

import oracle
import paper_2606_12950_amd as M
from paper_2606_12950_amd import pipeline
from paper_2606_12950_amd import workload as W
from test_gpu_fitness import (GB, _engines, _nodes, assert_same, gpu_fitness, gpu_fitness_act, gpu_fitness_plans,
                              oracle_fitness_act)
from test_gpu_parity import ALGOS, assert_route_equal

pytestmark = pytest.mark.gpu

OUT_OF_RANGE = [-1, -(1 << 31), 1 << 30, (1 << 31) - 1, 64, 100]


def _t(a):
    return pipeline._t(np.ascontiguousarray(a), "cuda")


def _spoil(rng, ids, n_valid, frac=0.125):
    """About one id in eight replaced by a value outside [0, n_valid); returns (ids, mask)."""
    bad = rng.random(ids.size) < frac
    values = np.array(OUT_OF_RANGE + [n_valid, n_valid + 1], np.int64)
    out = ids.astype(np.int64).copy()
    out[bad] = rng.choice(values, int(bad.sum()))
    return out.astype(np.int32), bad


@pytest.mark.parametrize("name", ["c0", "c1"])
def test_predict_flags_out_of_range_models(name):
    # c0: the float32 network; c1: the bfloat16 256-512-512-64 network (ragged last tile)
    w = W.workload(name, n_stages=3001)
    b = pipeline.to_device(w)
    o = pipeline.allocate_outputs(b)
    pipeline.run_predict(b, o)
    torch.cuda.synchronize()
    pred_ok, kv_ok = o.pred_len.cpu().numpy().copy(), o.kv_bytes.cpu().numpy().copy()
    ids, bad = _spoil(np.random.default_rng(11), w.model_id, w.spec.n_models)
    b.model_id = _t(ids)
    pipeline.run_predict(b, o)
    torch.cuda.synchronize()
    pred, kv = o.pred_len.cpu().numpy(), o.kv_bytes.cpu().numpy()
    assert bad.any() and np.array_equal(pred, pred_ok)
    assert np.all(np.isnan(kv[bad])) and np.array_equal(kv[~bad], kv_ok[~bad])


def test_two_phase_flags_out_of_range_models():
    w = W.workload("c1", n_stages=2000)
    tp = W.two_phase_inputs(w)
    ws = [_t(a) for a in w.weights[:-1]] + [_t(tp.head_weight)]
    bs = [_t(a) for a in w.biases[:-1]] + [_t(tp.head_bias)]

    def run(model):
        out = M.predict_two_phase(_t(w.x), ws, bs, _t(tp.role_head), _t(tp.tool_coef), _t(tp.iso_x), _t(tp.iso_y),
                                  tp.max_len, _t(w.prompt_len), _t(model), _t(w.role), _t(tp.tool_avail),
                                  _t(w.kv_bytes_per_token))
        torch.cuda.synchronize()
        return [a.cpu().numpy() for a in out]

    p_ok, l_ok, kv_ok = run(w.model_id)
    ids, bad = _spoil(np.random.default_rng(12), w.model_id, w.spec.n_models)
    p, l, kv = run(ids)
    assert np.array_equal(p, p_ok) and np.array_equal(l, l_ok)
    assert np.all(np.isnan(kv[bad])) and np.array_equal(kv[~bad], kv_ok[~bad])


@pytest.mark.parametrize("tiered", [False, True])
@pytest.mark.parametrize("algo", ["scan", "sorted"])
def test_route_flags_out_of_range_models(algo, tiered):
    w = W.workload("c1", n_stages=4000)
    rng = np.random.default_rng(13)
    n, K, k = w.n, w.spec.n_models, 3
    pred = rng.uniform(10, 2000, n).astype(np.float32)
    kv = rng.uniform(0, 1.5, n) * np.median(w.free_bytes)
    ids, bad = _spoil(rng, w.model_id, K)
    act = rng.uniform(0, 20, (w.spec.n_nodes, K)).astype(np.float32) if tiered else None
    idx, sc = M.route(_t(ids), _t(pred), _t(kv), _t(w.decode_s_per_token), _t(w.free_bytes), _t(w.queue_s),
                      None if tiered else _t(w.cold_s), None if tiered else _t(w.resident_mask), k=k, rho=0.1,
                      algo=ALGOS[algo], act_s=None if act is None else _t(act))
    torch.cuda.synchronize()
    idx, sc = idx.cpu().numpy(), sc.cpu().numpy()
    assert bad.any() and np.all(idx[bad] == -1) and np.all(sc[bad] == np.inf)
    ref = oracle.route(w.model_id[~bad], pred[~bad], kv[~bad], w.decode_s_per_token, w.free_bytes, w.queue_s,
                       w.cold_s, w.resident_mask, k=k, rho=0.1, act_matrix=act)
    assert_route_equal((idx[~bad], sc[~bad]), ref)


@pytest.mark.parametrize("plans", [False, True])
@pytest.mark.parametrize("which", ["model", "src", "cls"])
def test_fitness_flags_out_of_range_ids(which, plans):
    rng = np.random.default_rng(14)
    n, M_, n_src, n_models, k = 1500, 300, 3, 16, 2
    nodes = _nodes(rng, M_, n_src)
    ids = dict(model=rng.integers(0, n_models, n).astype(np.int32), src=rng.integers(0, n_src, n).astype(np.int32),
               cls=rng.integers(0, 2, n).astype(np.int32))
    ids[which], bad = _spoil(rng, ids[which], dict(model=n_models, src=n_src, cls=2)[which])
    kv = rng.uniform(0, 250, n) * GB
    weights, bounds = [[0.25, 1, 1], [0.1, 1, 1]], [0, 80, 0, 25000, 0, 500]
    eng = (*_engines(rng, M_), 2000.0)
    if plans:
        gi, gf = gpu_fitness_plans(ids["model"], ids["src"], ids["cls"], kv, nodes, weights, bounds, eng, k=k,
                                   n_models=n_models)
    else:
        gi, gf = gpu_fitness(ids["model"], ids["src"], ids["cls"], kv, nodes, weights, bounds, k=k, n_models=n_models)
    assert bad.any() and np.all(gi[bad] == -1) and np.all(gf[bad] == -np.inf)
    ok = ~bad
    ref = oracle.route_fitness(ids["model"][ok], ids["src"][ok], ids["cls"][ok], kv[ok], nodes["free_bytes"],
                               nodes["queue_ms"], nodes["act_ms"], nodes["resident_mask"], nodes["deg_ms"],
                               nodes["rtt_ms"], np.asarray(weights, np.float32), np.asarray(bounds, np.float32), k=k,
                               engines=eng if plans else None)
    assert_same((gi[ok], gf[ok]), ref)


@pytest.mark.parametrize("n_models", [16, 40])
@pytest.mark.parametrize("which", ["model", "src", "cls"])
def test_fitness_with_act_matrix_flags_out_of_range_ids(which, n_models):
    # T_act from a [node][model] matrix (both chunk classes: up to 16 and up to 64 models), plans
    rng = np.random.default_rng(15 + n_models)
    n, M_, n_src, k = 1200, 200, 4, 3
    nodes = _nodes(rng, M_, n_src)
    ids = dict(model=rng.integers(0, n_models, n).astype(np.int32), src=rng.integers(0, n_src, n).astype(np.int32),
               cls=rng.integers(0, 2, n).astype(np.int32))
    ids[which], bad = _spoil(rng, ids[which], dict(model=n_models, src=n_src, cls=2)[which])
    kv = rng.uniform(0, 250, n) * GB
    act = rng.uniform(0, 20000, (M_, n_models)).astype(np.float32)
    weights, bounds = [[0.25, 1, 1], [0.1, 1, 1]], [0, 80, 0, 25000, 0, 500]
    eng = (*_engines(rng, M_), 2000.0)
    gi, gf = gpu_fitness_act(ids["model"], ids["src"], ids["cls"], kv, nodes, weights, bounds, act, n_models, k=k,
                             eng=eng)
    assert bad.any() and np.all(gi[bad] == -1) and np.all(gf[bad] == -np.inf)
    ok = ~bad
    ref = oracle_fitness_act(ids["model"][ok], ids["src"][ok], ids["cls"][ok], kv[ok], nodes, weights, bounds, act,
                             n_models, k=k, eng=eng)
    assert_same((gi[ok], gf[ok]), ref)
