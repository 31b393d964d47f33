"""Parity of routing by fitness (Eq. 5, Alg. 3) and of the window quantiles between the HIP path
(through the C-ABI) and the CPU oracle, on seeded inputs.

Bars: quantiles bit-exact; node indices and fitness values bit-exact given the same inputs (both
sides evaluate the same float32 expression in the same order; the argmax is taken on it).
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2606_12950_amd as M
from paper_2606_12950_amd import pipeline
from paper_2606_12950_amd import workload as W

pytestmark = pytest.mark.gpu

GB = 1e9


def _t(a):
    return pipeline._t(np.ascontiguousarray(a), "cuda")


def gpu_quantiles(v, lo=0.05, hi=0.95):
    out = M.quantiles(_t(np.asarray(v, np.float32)), lo, hi)
    torch.cuda.synchronize()
    return out.cpu().numpy()


def gpu_fitness(model, src, cls, kv, nodes, weights, bounds, k=1, rho=0.0, n_models=64):
    idx, fit = M.route_fitness(_t(model.astype(np.int32)), _t(src.astype(np.int32)), _t(cls.astype(np.int32)),
                               _t(kv.astype(np.float64)), _t(nodes["free_bytes"]), _t(nodes["queue_ms"]),
                               _t(nodes["act_ms"]), _t(nodes["resident_mask"]), _t(nodes["deg_ms"]),
                               _t(nodes["rtt_ms"]), _t(np.asarray(weights, np.float32).reshape(-1, 3)),
                               _t(np.asarray(bounds, np.float32)), n_models=n_models, k=k, rho=rho)
    torch.cuda.synchronize()
    return idx.cpu().numpy(), fit.cpu().numpy()


def oracle_fitness(model, src, cls, kv, nodes, weights, bounds, k=1, rho=0.0):
    return oracle.route_fitness(model, src, cls, kv, nodes["free_bytes"], nodes["queue_ms"], nodes["act_ms"],
                                nodes["resident_mask"], nodes["deg_ms"], nodes["rtt_ms"],
                                np.asarray(weights, np.float32).reshape(-1, 3), np.asarray(bounds, np.float32),
                                k=k, rho=rho)


def assert_same(got, ref):
    gi, gf = got
    ri, rf = ref
    bad = np.flatnonzero((gi != ri).any(axis=1) | (gf.view(np.uint32) != rf.view(np.uint32)).any(axis=1))
    assert bad.size == 0, f"{bad.size} stages differ, first {bad[:5]}: gpu {gi[bad[0]]} {gf[bad[0]]} " \
                          f"oracle {ri[bad[0]]} {rf[bad[0]]}"


def _nodes(rng, M_, n_src, n_models=16):
    return dict(
        free_bytes=rng.uniform(0, 300, M_) * GB,
        queue_ms=rng.uniform(0, 5000, M_).astype(np.float32),
        act_ms=rng.uniform(2000, 20000, M_).astype(np.float32),
        # residency over all 64 bits (models past n_models never ask for theirs)
        resident_mask=rng.integers(0, 2 ** 64, M_, dtype=np.uint64),
        deg_ms=np.where(rng.random(M_) < 0.3, rng.uniform(0, 500, M_), 0).astype(np.float32),
        rtt_ms=rng.uniform(0.2, 80, (n_src, M_)).astype(np.float32),
    )


@pytest.mark.parametrize("m", [1, 2, 3, 19, 20, 21, 1000, 4096, 32767, 32768, 40000, 100003])
def test_quantiles_match_oracle(m):
    # 32,768 values and more count into per-lane histogram copies
    rng = np.random.default_rng(m)
    v = np.round(rng.normal(0, 30, m), 1).astype(np.float32)
    v[rng.random(m) < 0.05] = -0.0
    v[rng.random(m) < 0.05] = 0.0
    for lo, hi in [(0.05, 0.95), (0.0, 1.0), (0.5, 0.5), (0.01, 0.99)]:
        got = gpu_quantiles(v, lo, hi)
        ref = oracle.quantiles(v, lo, hi)
        assert got.view(np.uint32).tolist() == ref.view(np.uint32).tolist(), (lo, hi, got, ref)


@pytest.mark.parametrize("m", [32768, 32769, (1 << 20) + 7])
@pytest.mark.parametrize("kind", ["equal", "two", "zeros", "spread"])
def test_quantiles_long_windows_degenerate(m, kind):
    # windows of 32,768 values and more select over 256 workgroups: every pass with all
    # candidates in one bin, two values, signed zeros, and a wide spread
    rng = np.random.default_rng(m + len(kind))
    if kind == "equal":
        v = np.full(m, 3.25, np.float32)
    elif kind == "two":
        v = rng.choice(np.array([-1.5, 7.0], np.float32), m)
    elif kind == "zeros":
        v = rng.choice(np.array([-0.0, 0.0, 1e-30, -1e-30], np.float32), m)
    else:
        v = (rng.standard_normal(m) * 10.0 ** rng.integers(-20, 20, m)).astype(np.float32)
    for lo, hi in [(0.05, 0.95), (0.0, 1.0), (0.5, 0.5)]:
        got = gpu_quantiles(v, lo, hi)
        ref = oracle.quantiles(v, lo, hi)
        assert got.view(np.uint32).tolist() == ref.view(np.uint32).tolist(), (lo, hi, got, ref)


@pytest.mark.parametrize("n,M_,n_src,k", [(1, 1, 1, 1), (257, 64, 3, 1), (1000, 1300, 5, 3),
                                          (3000, 512, 16, 16), (700, 2049, 2, 4)])
def test_fitness_matches_oracle(n, M_, n_src, k):
    # several 512-node chunks with a ragged tail, every source count, route widths 1..16
    rng = np.random.default_rng(n * 7 + M_)
    nodes = _nodes(rng, M_, n_src)
    # 64 models: residency bits in both halves of the 64-bit mask
    model = rng.integers(0, 64, n).astype(np.int32)
    src = rng.integers(0, n_src, n).astype(np.int32)
    cls = rng.integers(0, 3, n).astype(np.int32)
    kv = rng.uniform(0, 250, n) * GB
    weights = [[0.25, 1, 1], [0.1, 1, 1], [0.6, 0.3, 2.0]]
    rw, qw = nodes["rtt_ms"].ravel(), (nodes["queue_ms"] + nodes["act_ms"])
    bounds = [*oracle.quantiles(rw), *oracle.quantiles(qw), *oracle.quantiles(nodes["deg_ms"])]
    for rho in (0.0, 0.2):
        got = gpu_fitness(model, src, cls, kv, nodes, weights, bounds, k=k, rho=rho)
        assert_same(got, oracle_fitness(model, src, cls, kv, nodes, weights, bounds, k=k, rho=rho))


def test_fitness_ties_infeasible_and_degenerate_windows():
    rng = np.random.default_rng(11)
    M_ = 600
    nodes = _nodes(rng, M_, 2)
    # duplicated node states: equal fitness, the lower index must come first
    for key in nodes:
        if key == "rtt_ms":
            nodes[key][:, 300:] = nodes[key][:, :300]
        else:
            nodes[key][300:] = nodes[key][:300]
    n = 2000
    model = rng.integers(0, 16, n).astype(np.int32)
    src = rng.integers(0, 2, n).astype(np.int32)
    cls = np.zeros(n, np.int32)
    kv = rng.uniform(0, 400, n) * GB          # many stages fit nowhere
    kv[::50] = 0.0                            # zero demand
    for bounds in ([0, 100, 0, 30000, 0, 500], [5, 5, 7, 7, 1, 1]):   # normal and degenerate windows
        got = gpu_fitness(model, src, cls, kv, nodes, [[0.25, 1, 1]], bounds, k=5)
        ref = oracle_fitness(model, src, cls, kv, nodes, [[0.25, 1, 1]], bounds, k=5)
        assert_same(got, ref)
    assert (got[0][:, 0] == -1).any() and (got[0][:, 0] >= 0).any()


@pytest.mark.parametrize("name", ["c1", "c3"])
def test_fitness_workload_full(name):
    # the GPU's own predictions feed both sides; every stage is compared
    w = W.workload(name)
    f = W.fitness_inputs(w)
    b = pipeline.to_device(w)
    o = pipeline.allocate_outputs(b)
    pipeline.run_predict(b, o)
    torch.cuda.synchronize()
    kv = o.kv_bytes.cpu().numpy()
    nodes = dict(free_bytes=w.free_bytes, queue_ms=f.queue_ms, act_ms=f.act_ms, resident_mask=w.resident_mask,
                 deg_ms=f.deg_ms, rtt_ms=f.rtt_ms)
    bounds_g = np.concatenate([gpu_quantiles(f.rtt_window), gpu_quantiles(f.ready_window),
                               gpu_quantiles(f.deg_window)])
    bounds_o = np.concatenate([oracle.quantiles(f.rtt_window), oracle.quantiles(f.ready_window),
                               oracle.quantiles(f.deg_window)])
    assert bounds_g.view(np.uint32).tolist() == bounds_o.view(np.uint32).tolist()
    got = gpu_fitness(w.model_id, f.src_id, f.class_id, kv, nodes, f.class_weights, bounds_g, k=w.spec.k,
                      rho=w.spec.rho, n_models=w.spec.n_models)
    ref = oracle_fitness(w.model_id, f.src_id, f.class_id, kv, nodes, f.class_weights, bounds_o, k=w.spec.k,
                         rho=w.spec.rho)
    assert_same(got, ref)
    routed = (got[0][:, 0] >= 0).mean()
    print(f"{name}: {w.n} stages x {w.free_bytes.size} nodes, {routed:.4f} routed, fitness identical")


# ---- degradation plans (Alg. 2, Eq. 4) ----------------------------------------------------------

def _engines(rng, M_, max_e=8, level_p=(0.3, 0.2, 0.1, 0.25, 0.15)):
    count = rng.integers(0, max_e + 1, M_)
    off = np.zeros(M_ + 1, np.int32)
    np.cumsum(count, out=off[1:])
    E = int(off[-1])
    level = (rng.choice(5, size=E, p=level_p) + 1).astype(np.int32)
    freed = rng.uniform(0.2, 40, E) * GB
    freed[rng.random(E) < 0.1] = 0.0                   # an action that frees nothing
    cost = rng.uniform(1, 5000, E).astype(np.float32)
    return off, level, freed, cost


def gpu_plans(off, level, freed, cost, c_int):
    """(record freed [M][8], record cost [M][8], n_engines [M], raw records, step freed [E],
    step cost [E], step engine [E])"""
    p = M.degradation_plans(_t(off), _t(level), _t(freed), _t(cost), c_int)
    torch.cuda.synchronize()
    raw = p.records.cpu().numpy()
    st = p.steps.cpu().numpy()[: int(off[-1])]
    return (raw[:, :64].copy().view(np.float64), raw[:, 64:96].copy().view(np.float32),
            raw[:, 96:100].copy().view(np.int32)[:, 0], raw, st[:, :8].copy().view(np.float64)[:, 0],
            st[:, 8:12].copy().view(np.float32)[:, 0], st[:, 12:16].copy().view(np.int32)[:, 0])


def _plan_answer(pf, pc, ne, R):
    """Cost of the shortest prefix with freed >= R, None when none."""
    for j in range(ne):
        if pf[j] >= R:
            return float(pc[j])
    return None


@pytest.mark.parametrize("max_e", [8, 40])
def test_degradation_plans_match_oracle(max_e):
    # every boundary of every node's plan: R at a prefix's freed bytes is met by that prefix,
    # one ulp above it needs the next one (or fails). Up to 40 engines a node: nodes past the
    # record's eight steps are sorted by rank counting and continue in the step array.
    rng = np.random.default_rng(5 + max_e)
    M_ = 700
    off, level, freed, cost = _engines(rng, M_, max_e=max_e)
    level[off[10]:off[11]] = 4                          # equal levels: engine order decides
    for c_int in (2000.0, 0.0):
        pf, pc, ne, raw, sf, sc, se = gpu_plans(off, level, freed, cost, c_int)
        assert (ne == np.diff(off)).all()
        assert (raw[:, 100:104].copy().view(np.int32)[:, 0] == off[:-1]).all()   # first step
        assert not raw[:, 104:].any()                   # reserved words are zero
        checked = 0
        for j in range(M_):
            lv, fr, co = level[off[j]:off[j + 1]], freed[off[j]:off[j + 1]], cost[off[j]:off[j + 1]]
            jf, jc, je = sf[off[j]:off[j + 1]], sc[off[j]:off[j + 1]], se[off[j]:off[j + 1]]
            # the steps take every engine once, in (level, index) order
            assert je.tolist() == sorted(range(off[j], off[j + 1]), key=lambda e: (level[e], e))
            # the record holds the first eight steps, +inf and 0 past the node's engines
            h = min(ne[j], 8)
            assert np.array_equal(pf[j, :h], jf[:h]) and np.array_equal(pc[j, :h].view(np.uint32),
                                                                        jc[:h].view(np.uint32))
            assert np.isposinf(pf[j, h:]).all() and (pc[j, h:] == 0).all()
            Rs = [1.0, 1e13]
            for e in range(ne[j]):
                Rs += [jf[e], np.nextafter(jf[e], np.inf)]
            for R in Rs:
                if R <= 0:
                    continue
                ref = oracle.degradation_cost(R, lv, fr, co, c_int)
                got = _plan_answer(jf, jc, ne[j], R)
                assert (got is None) == (ref is None), (j, R, got, ref)
                if ref is not None:
                    assert np.float32(got).view(np.uint32) == np.float32(ref).view(np.uint32), (j, R, got, ref)
                checked += 1
        assert checked > 4 * M_
        if max_e > 8:
            assert (ne > 8).sum() > 100


def test_degradation_plans_empty_and_single():
    off = np.array([0, 0, 1, 1], np.int32)              # nodes with 0, 1 and 0 engines
    level = np.array([5], np.int32)
    freed = np.array([3 * GB])
    cost = np.array([40.0], np.float32)
    pf, pc, ne = gpu_plans(off, level, freed, cost, 2000.0)[:3]
    assert ne.tolist() == [0, 1, 0]
    assert pf[1, 0] == 3 * GB and pc[1, 0] == np.float32(2040.0)
    pf, pc, ne = gpu_plans(np.zeros(3, np.int32), np.zeros(0, np.int32), np.zeros(0), np.zeros(0, np.float32),
                           10.0)[:3]
    assert ne.tolist() == [0, 0]


def gpu_fitness_plans(model, src, cls, kv, nodes, weights, bounds, eng, k=1, rho=0.0, n_models=64):
    off, level, freed, cost, c_int = eng
    plans = M.degradation_plans(_t(off), _t(level), _t(freed), _t(cost), c_int)
    idx, fit = M.route_fitness(_t(model.astype(np.int32)), _t(src.astype(np.int32)), _t(cls.astype(np.int32)),
                               _t(kv.astype(np.float64)), _t(nodes["free_bytes"]), _t(nodes["queue_ms"]),
                               _t(nodes["act_ms"]), _t(nodes["resident_mask"]), None,
                               _t(nodes["rtt_ms"]), _t(np.asarray(weights, np.float32).reshape(-1, 3)),
                               _t(np.asarray(bounds, np.float32)), n_models=n_models, k=k, rho=rho, plans=plans)
    torch.cuda.synchronize()
    return idx.cpu().numpy(), fit.cpu().numpy()


@pytest.mark.parametrize("n,M_,n_src,k,max_e", [(1, 1, 1, 1, 8), (300, 255, 2, 1, 8), (1000, 257, 5, 3, 8),
                                                (2000, 1300, 16, 16, 8), (513, 700, 3, 4, 8), (1000, 300, 4, 1, 30),
                                                (777, 1100, 3, 4, 30)])
def test_fitness_with_plans_matches_oracle(n, M_, n_src, k, max_e):
    # several 128-node chunks with ragged tails; most stages fall short on many nodes; with up to
    # 30 engines a node, shortfalls beyond a record's eight steps search the step array
    rng = np.random.default_rng(n * 13 + M_ + max_e)
    nodes = _nodes(rng, M_, n_src)
    nodes["free_bytes"] = rng.uniform(0, 60, M_) * GB
    nodes["free_bytes"][rng.random(M_) < 0.05] = 0.0
    off, level, freed, cost = _engines(rng, M_, max_e=max_e)
    if max_e > 8:
        freed = freed * 0.2                               # small actions: long plans on big nodes
    eng = (off, level, freed, cost, 2000.0)
    model = rng.integers(0, 64, n).astype(np.int32)
    src = rng.integers(0, n_src, n).astype(np.int32)
    cls = rng.integers(0, 3, n).astype(np.int32)
    kv = rng.uniform(0, 120, n) * GB
    kv[::37] = 0.0
    weights = [[0.25, 1, 1], [0.1, 1, 1], [1.0, 0.0, 1.0]]
    bounds = [*oracle.quantiles(nodes["rtt_ms"].ravel()), *oracle.quantiles(nodes["queue_ms"] + nodes["act_ms"]),
              0.0, 12000.0]
    for rho in (0.0, 0.2):
        got = gpu_fitness_plans(model, src, cls, kv, nodes, weights, bounds, eng, k=k, rho=rho)
        ref = oracle.route_fitness(model, src, cls, kv, nodes["free_bytes"], nodes["queue_ms"], nodes["act_ms"],
                                   nodes["resident_mask"], nodes["deg_ms"], nodes["rtt_ms"],
                                   np.asarray(weights, np.float32), np.asarray(bounds, np.float32), k=k, rho=rho,
                                   engines=eng)
        assert_same(got, ref)
    if n > 100:   # the shortfall branch is exercised, on most pairs
        assert (kv[:, None] > nodes["free_bytes"][None, :]).mean() > 0.3


def test_fitness_with_plans_exact_shortfall_boundaries():
    # shortfalls that equal a prefix's freed bytes exactly, and degenerate C_deg window
    rng = np.random.default_rng(23)
    M_ = 300
    nodes = _nodes(rng, M_, 2)
    nodes["free_bytes"] = np.round(rng.uniform(0, 20, M_)) * GB
    off, level, freed, cost = _engines(rng, M_)
    freed = np.round(freed / GB) * GB                   # integral GB: exact sums
    eng = (off, level, freed, cost, 2000.0)
    n = 3000
    kv = np.round(rng.uniform(0, 80, n)) * GB           # shortfalls hit prefix sums exactly
    model = rng.integers(0, 16, n).astype(np.int32)
    src = rng.integers(0, 2, n).astype(np.int32)
    cls = np.zeros(n, np.int32)
    for bounds in ([0, 100, 0, 30000, 0, 8000], [5, 5, 7, 7, 1, 1]):
        got = gpu_fitness_plans(model, src, cls, kv, nodes, [[0.25, 1, 1]], bounds, eng, k=4)
        ref = oracle.route_fitness(model, src, cls, kv, nodes["free_bytes"], nodes["queue_ms"], nodes["act_ms"],
                                   nodes["resident_mask"], nodes["deg_ms"], nodes["rtt_ms"],
                                   np.asarray([[0.25, 1, 1]], np.float32), np.asarray(bounds, np.float32), k=4,
                                   engines=eng)
        assert_same(got, ref)


@pytest.mark.parametrize("name", ["c1", "c3"])
def test_fitness_with_plans_workload_full(name):
    w = W.workload(name)
    f = W.fitness_inputs(w)
    e = W.engine_inputs(w)
    b = pipeline.to_device(w)
    o = pipeline.allocate_outputs(b)
    pipeline.run_predict(b, o)
    torch.cuda.synchronize()
    kv = o.kv_bytes.cpu().numpy()
    nodes = dict(free_bytes=w.free_bytes, queue_ms=f.queue_ms, act_ms=f.act_ms, resident_mask=w.resident_mask,
                 deg_ms=f.deg_ms, rtt_ms=f.rtt_ms)
    bounds = np.concatenate([oracle.quantiles(f.rtt_window), oracle.quantiles(f.ready_window),
                             oracle.quantiles(e.deg_window)])
    eng = (e.engine_offset, e.level, e.freed_bytes, e.cost_ms, e.c_int_ms)
    got = gpu_fitness_plans(w.model_id, f.src_id, f.class_id, kv, nodes, f.class_weights, bounds, eng, k=w.spec.k,
                            rho=w.spec.rho, n_models=w.spec.n_models)
    ref = oracle.route_fitness(w.model_id, f.src_id, f.class_id, kv, nodes["free_bytes"], nodes["queue_ms"],
                               nodes["act_ms"], nodes["resident_mask"], nodes["deg_ms"], nodes["rtt_ms"],
                               f.class_weights, bounds, k=w.spec.k, rho=w.spec.rho, engines=eng)
    assert_same(got, ref)
    print(f"{name}: {w.n} stages x {w.free_bytes.size} nodes with plans, "
          f"{(got[0][:, 0] >= 0).mean():.4f} routed, fitness identical")


# ---- model readiness tiers (Sec. III-C) as T_act(N, M(T)) of Eq. 6 -------------------------------

TIER_BW = np.array([1.0, 25e9, 25e9, 3e9, 1.25e9])
TIER_SETUP = np.array([0.0, 150.0, 2500.0, 2500.0, 4000.0], np.float32)


def gpu_activation(tier, size, bw=TIER_BW, setup=TIER_SETUP):
    out = M.activation_latency(_t(tier.astype(np.uint8)), _t(size.astype(np.float64)), _t(bw.astype(np.float64)),
                               _t(setup.astype(np.float32)))
    torch.cuda.synchronize()
    return out.cpu().numpy()


def test_activation_latency_matches_oracle():
    rng = np.random.default_rng(17)
    for Mn, K in [(1, 1), (513, 16), (3000, 64), (0, 5)]:
        tier = rng.integers(0, 9, (Mn, K)).astype(np.uint8)      # values past 4 count as Remote
        size = rng.uniform(0.5, 30, K) * GB
        size[0] = 0.0
        got = gpu_activation(tier, size)
        ref = oracle.activation_latency(tier, size, TIER_BW, TIER_SETUP)
        assert got.shape == (Mn, K) and np.array_equal(got.view(np.uint32), ref.view(np.uint32))


def gpu_fitness_act(model, src, cls, kv, nodes, weights, bounds, act, n_models, k=1, rho=0.0, eng=None):
    plans = None
    if eng is not None:
        off, level, freed, cost, c_int = eng
        plans = M.degradation_plans(_t(off), _t(level), _t(freed), _t(cost), c_int)
    idx, fit = M.route_fitness(_t(model.astype(np.int32)), _t(src.astype(np.int32)), _t(cls.astype(np.int32)),
                               _t(kv.astype(np.float64)), _t(nodes["free_bytes"]), _t(nodes["queue_ms"]), None, None,
                               None if eng is not None else _t(nodes["deg_ms"]), _t(nodes["rtt_ms"]),
                               _t(np.asarray(weights, np.float32).reshape(-1, 3)), _t(np.asarray(bounds, np.float32)),
                               n_models=n_models, k=k, rho=rho, plans=plans, act_matrix=_t(act))
    torch.cuda.synchronize()
    return idx.cpu().numpy(), fit.cpu().numpy()


def oracle_fitness_act(model, src, cls, kv, nodes, weights, bounds, act, n_models, k=1, rho=0.0, eng=None):
    return oracle.route_fitness(model, src, cls, kv, nodes["free_bytes"], nodes["queue_ms"], nodes["act_ms"],
                                nodes["resident_mask"], nodes["deg_ms"], nodes["rtt_ms"],
                                np.asarray(weights, np.float32).reshape(-1, 3), np.asarray(bounds, np.float32), k=k,
                                rho=rho, n_models=n_models, engines=eng, act_matrix=act)


@pytest.mark.parametrize("n,M_,n_src,k,n_models,plans", [(1, 1, 1, 1, 1, False), (300, 65, 2, 1, 16, False),
                                                         (1000, 700, 5, 3, 64, False), (777, 129, 16, 16, 33, True),
                                                         (2000, 1300, 3, 4, 64, True)])
def test_fitness_with_act_matrix_matches_oracle(n, M_, n_src, k, n_models, plans):
    # several 64-node chunks with ragged tails, up to 64 models, with and without plans
    rng = np.random.default_rng(n + 31 * M_)
    nodes = _nodes(rng, M_, n_src)
    if plans:
        nodes["free_bytes"] = rng.uniform(0, 60, M_) * GB
    tier = rng.integers(0, 5, (M_, n_models)).astype(np.uint8)
    act = oracle.activation_latency(tier, rng.uniform(1, 28, n_models) * GB, TIER_BW, TIER_SETUP)
    eng = None
    if plans:
        off, level, freed, cost = _engines(rng, M_)
        eng = (off, level, freed, cost, 2000.0)
    model = rng.integers(0, n_models, n).astype(np.int32)
    src = rng.integers(0, n_src, n).astype(np.int32)
    cls = rng.integers(0, 3, n).astype(np.int32)
    kv = rng.uniform(0, 120 if plans else 250, n) * GB
    weights = [[0.25, 1, 1], [0.1, 1, 1], [1.0, 1.0, 0.0]]
    bounds = [*oracle.quantiles(nodes["rtt_ms"].ravel()), *oracle.quantiles((nodes["queue_ms"][:, None] + act).ravel()),
              0.0, 12000.0]
    for rho in (0.0, 0.2):
        got = gpu_fitness_act(model, src, cls, kv, nodes, weights, bounds, act, n_models, k=k, rho=rho, eng=eng)
        assert_same(got, oracle_fitness_act(model, src, cls, kv, nodes, weights, bounds, act, n_models, k=k, rho=rho,
                                            eng=eng))


def test_fitness_act_matrix_of_resident_bits_equals_mask_form():
    # the matrix {0 where resident, act_ms otherwise} routes exactly like the residency bits
    rng = np.random.default_rng(29)
    M_, n = 900, 3000
    nodes = _nodes(rng, M_, 4)
    bits = (nodes["resident_mask"][:, None] >> np.arange(16, dtype=np.uint64)[None, :]) & np.uint64(1)
    act = np.where(bits == 1, 0.0, nodes["act_ms"][:, None]).astype(np.float32)
    model = rng.integers(0, 16, n).astype(np.int32)
    src = rng.integers(0, 4, n).astype(np.int32)
    cls = rng.integers(0, 2, n).astype(np.int32)
    kv = rng.uniform(0, 250, n) * GB
    w, b = [[0.25, 1, 1], [0.1, 1, 1]], [0, 80, 0, 25000, 0, 500]
    got = gpu_fitness_act(model, src, cls, kv, nodes, w, b, act, 16, k=4)
    ref = gpu_fitness(model, src, cls, kv, nodes, w, b, k=4, n_models=16)
    assert_same(got, ref)


@pytest.mark.parametrize("name", ["c1", "c3"])
def test_fitness_with_readiness_and_plans_workload_full(name):
    # readiness tiers on the GPU, then fitness with T_act from them and C_deg from plans
    w = W.workload(name)
    f = W.fitness_inputs(w)
    e = W.engine_inputs(w)
    r = W.readiness_inputs(w)
    b = pipeline.to_device(w)
    o = pipeline.allocate_outputs(b)
    pipeline.run_predict(b, o)
    torch.cuda.synchronize()
    kv = o.kv_bytes.cpu().numpy()
    act = gpu_activation(r.tier, r.model_bytes, r.tier_bw, r.tier_setup_ms)
    assert np.array_equal(act.view(np.uint32),
                          oracle.activation_latency(r.tier, r.model_bytes, r.tier_bw, r.tier_setup_ms).view(np.uint32))
    nodes = dict(free_bytes=w.free_bytes, queue_ms=f.queue_ms, act_ms=f.act_ms, resident_mask=w.resident_mask,
                 deg_ms=f.deg_ms, rtt_ms=f.rtt_ms)
    bounds = np.concatenate([oracle.quantiles(f.rtt_window), oracle.quantiles(f.ready_window),
                             oracle.quantiles(e.deg_window)])
    eng = (e.engine_offset, e.level, e.freed_bytes, e.cost_ms, e.c_int_ms)
    K = w.spec.n_models
    got = gpu_fitness_act(w.model_id, f.src_id, f.class_id, kv, nodes, f.class_weights, bounds, act, K, k=w.spec.k,
                          rho=w.spec.rho, eng=eng)
    ref = oracle_fitness_act(w.model_id, f.src_id, f.class_id, kv, nodes, f.class_weights, bounds, act, K,
                             k=w.spec.k, rho=w.spec.rho, eng=eng)
    assert_same(got, ref)
    print(f"{name}: {w.n} stages x {w.free_bytes.size} nodes, readiness tiers + plans, fitness identical")


# ---- adaptive safety margin (Sec. III-D) ---------------------------------------------------------

def _ulp_close(got, ref):
    """Within one float32 unit in the last place (the float64 EWMA is a parallel scan on the GPU
    and a sequential loop in the oracle; rounding to float32 can then differ in the last place)."""
    got, ref = np.asarray(got, np.float32), np.asarray(ref, np.float32)
    return np.all(np.abs(got.astype(np.float64) - ref) <= np.spacing(np.abs(ref)).astype(np.float64))


@pytest.mark.parametrize("m", [1, 2, 1000, 1023, 1024, 1025, 4096, 8192, 8193, 16384, 16385, 16386, 24576,
                               24579, 32767, 32768, 100003, 3000000])
def test_adaptive_rho_matches_oracle(m):
    # tiles of 8,192 stages: up to two tiles in one workgroup, longer windows in three launches
    # (16,385 and 24,579 end in a tile of one and three stages; 16,385 is finished by the
    # composition pass); the selection switches to per-lane histogram copies at 32,768
    actual, pred = W.margin_window(m, m)
    for beta, q in [(0.2, 0.95), (0.05, 0.9), (1.0, 0.95), (0.5, 1.0), (0.2, 0.0)]:
        ew, rho = M.adaptive_rho(_t(actual), _t(pred), beta, q)
        torch.cuda.synchronize()
        ew, rho = ew.cpu().numpy(), rho.cpu().numpy()[0]
        ew_o, rho_o = oracle.adaptive_rho(actual, pred, beta, q)
        assert _ulp_close(ew, ew_o), (beta, q)
        assert np.mean(ew.view(np.uint32) == ew_o.view(np.uint32)) > 0.999
        # rho is an order statistic of the GPU's own values, and within an ulp of the oracle's
        assert rho == np.sort(ew)[int(np.ceil(q * (m - 1)))]
        assert _ulp_close(rho, rho_o), (beta, q, rho, rho_o)
        if (beta, q) == (0.2, 0.95):
            print(f"m={m}: rho(beta 0.2, q 0.95) = {rho:.4f}")


def test_adaptive_rho_exact_cases():
    pred = np.full(5000, 1e9)
    ew, rho = M.adaptive_rho(_t(pred), _t(pred), 0.2, 0.95)
    assert not ew.cpu().numpy().any() and rho.item() == 0.0
    ew, rho = M.adaptive_rho(_t(1.25 * pred), _t(pred), 0.3, 0.9)
    assert np.all(ew.cpu().numpy() == np.float32(0.25)) and rho.item() == np.float32(0.25)
