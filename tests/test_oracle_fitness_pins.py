"""Pins of the oracle's fitness routing (Eq. 5 over the feasible nodes, Alg. 3 argmax) and of
its window bounds (order statistics), against what the definitions fix: limiting weights reduce
the score to one metric whose argmax is a plain argmin/argmax, clipping and degenerate windows,
infeasibility, ordering and tie-breaks, node-permutation equivariance, and numpy's percentile
selection for the bounds. No GPU."""
import numpy as np
import pytest

import oracle

GB = 1e9


def _nodes(rng, M, n_src=3, n_models=8):
    return dict(
        free_bytes=rng.uniform(1, 300, M) * GB,
        queue_ms=rng.uniform(0, 5000, M).astype(np.float32),
        act_ms=rng.uniform(2000, 20000, M).astype(np.float32),
        resident_mask=rng.integers(0, 1 << n_models, M).astype(np.uint64),
        deg_ms=rng.uniform(0, 50, M).astype(np.float32),
        rtt_ms=rng.uniform(0.2, 80, (n_src, M)).astype(np.float32),
    )


def _route(nodes, model_id, src_id, class_id, kv, weights, bounds, k=1, rho=0.0):
    return oracle.route_fitness(model_id, src_id, class_id, kv, nodes["free_bytes"], nodes["queue_ms"],
                                nodes["act_ms"], nodes["resident_mask"], nodes["deg_ms"], nodes["rtt_ms"],
                                np.asarray(weights, np.float32).reshape(-1, 3), np.asarray(bounds, np.float32),
                                k=k, rho=rho)


def _wide_bounds(nodes):
    """bounds strictly outside every value: no clipping"""
    r, q = nodes["rtt_ms"], nodes["queue_ms"] + nodes["act_ms"]
    return [r.min() - 1, r.max() + 1, 0.0, float(q.max()) + 1, -1.0, float(nodes["deg_ms"].max()) + 1]


@pytest.mark.parametrize("m", [1, 2, 19, 20, 21, 1000, 4097])
def test_quantiles_are_numpy_order_statistics(m):
    rng = np.random.default_rng(m)
    v = np.round(rng.normal(0, 10, m), 1).astype(np.float32)     # duplicates on purpose
    lo, hi = oracle.quantiles(v, 0.05, 0.95)
    assert lo == np.percentile(v, 5, method="lower")
    assert hi == np.percentile(v, 95, method="higher")
    assert oracle.quantiles(v, 0.0, 1.0).tolist() == [v.min(), v.max()]
    med = oracle.quantiles(v, 0.5, 0.5)
    assert med[0] == np.percentile(v, 50, method="lower") and med[1] == np.percentile(v, 50, method="higher")


def test_network_weight_one_picks_the_nearest_node():
    rng = np.random.default_rng(1)
    M, N = 64, 500
    nodes = _nodes(rng, M)
    nodes["rtt_ms"] = rng.permutation(np.arange(3 * M, dtype=np.float32)).reshape(3, M) * 0.5 + 0.2
    src = rng.integers(0, 3, N).astype(np.int32)
    kv = rng.uniform(0, 100, N) * GB
    idx, _ = _route(nodes, np.zeros(N, np.int32), src, np.zeros(N, np.int32), kv, [1, 0, 0], _wide_bounds(nodes))
    for i in range(N):
        feas = np.flatnonzero(kv[i] <= nodes["free_bytes"])
        want = feas[np.argmin(nodes["rtt_ms"][src[i], feas])] if feas.size else -1
        assert idx[i, 0] == want


def test_fit_only_is_best_fit_packing():
    # gamma = lambda = mu = 0: the feasible node whose headroom is closest above the demand
    rng = np.random.default_rng(2)
    M, N = 50, 400
    nodes = _nodes(rng, M)
    nodes["free_bytes"] = rng.permutation(np.arange(1, M + 1)) * 5.0 * GB
    kv = rng.uniform(0, 260, N) * GB
    idx, fit = _route(nodes, np.zeros(N, np.int32), np.zeros(N, np.int32), np.zeros(N, np.int32), kv,
                      [0, 0, 0], _wide_bounds(nodes))
    for i in range(N):
        feas = np.flatnonzero(kv[i] <= nodes["free_bytes"])
        want = feas[np.argmin(nodes["free_bytes"][feas])] if feas.size else -1
        assert idx[i, 0] == want
        if want >= 0:
            assert 0.0 < fit[i, 0] <= 1.0


def test_zero_demand_reduces_to_time_to_start_or_disruption():
    # zero demand: fit = 0 on every node and every node is feasible
    rng = np.random.default_rng(3)
    M, N = 40, 300
    nodes = _nodes(rng, M)
    nodes["queue_ms"] = rng.permutation(np.arange(M, dtype=np.float32)) * 100
    nodes["deg_ms"] = rng.permutation(np.arange(M, dtype=np.float32)) * 2
    model = rng.integers(0, 8, N).astype(np.int32)
    kv = np.zeros(N)
    b = _wide_bounds(nodes)
    idx, _ = _route(nodes, model, np.zeros(N, np.int32), np.zeros(N, np.int32), kv, [0, 1, 0], b)
    for i in range(N):
        res = (nodes["resident_mask"] >> np.uint64(model[i])) & np.uint64(1)
        t_ready = nodes["queue_ms"] + np.where(res == 1, 0, nodes["act_ms"])   # T_q + T_act
        assert idx[i, 0] == np.argmin(t_ready)
    idx, _ = _route(nodes, model, np.zeros(N, np.int32), np.zeros(N, np.int32), kv, [0, 0, 1], b)
    assert (idx[:, 0] == np.argmin(nodes["deg_ms"])).all()


def test_values_beyond_the_window_clip_and_degenerate_windows_vanish():
    rng = np.random.default_rng(4)
    M = 6
    nodes = _nodes(rng, M, n_src=1)
    nodes["free_bytes"][:] = 100 * GB
    nodes["rtt_ms"][0] = [5, 50, 100, 500, 1000, 3]
    kv = np.array([10 * GB])
    one = np.zeros(1, np.int32)
    # RTT bounds [10, 100]: 500 and 1000 clip to the bound 100, 5 and 3 to the bound 10
    idx, fit = _route(nodes, one, one, one, kv, [1, 0, 0], [10, 100, 0, 1, 0, 1], k=6)
    assert idx[0].tolist() == [0, 5, 1, 2, 3, 4]
    assert fit[0].tolist() == [1, 1, fit[0, 2], 0, 0, 0] and 0 < fit[0, 2] < 1
    # a degenerate window (hi <= lo) normalises every value to 0: proximity 1 everywhere
    idx, fit = _route(nodes, one, one, one, kv, [1, 0, 0], [7, 7, 0, 1, 0, 1], k=6)
    assert idx[0].tolist() == list(range(6)) and (fit[0] == 1).all()


def test_infeasible_padding_topk_order_and_rho():
    rng = np.random.default_rng(5)
    M, N, k = 30, 200, 5
    nodes = _nodes(rng, M)
    kv = rng.uniform(0, 400, N) * GB                               # some stages fit nowhere
    model, src, cls = (rng.integers(0, 8, N).astype(np.int32), rng.integers(0, 3, N).astype(np.int32),
                       rng.integers(0, 2, N).astype(np.int32))
    w = [[0.25, 1, 1], [0.1, 1, 1]]
    b = _wide_bounds(nodes)
    idx, fit = _route(nodes, model, src, cls, kv, w, b, k=k, rho=0.2)
    for i in range(N):
        feas = set(np.flatnonzero(kv[i] * 1.2 <= nodes["free_bytes"]).tolist())
        got = [j for j in idx[i] if j >= 0]
        assert len(got) == min(k, len(feas)) and set(got) <= feas
        assert all(j == -1 for j in idx[i, len(got):]) and np.all(np.isneginf(fit[i, len(got):]))
        f = fit[i, :len(got)]
        assert all(f[j] > f[j + 1] or (f[j] == f[j + 1] and got[j] < got[j + 1]) for j in range(len(got) - 1))
        if len(got) == k and len(feas) > k:                        # nothing better left out
            ref, _ = _route(nodes, model[i:i + 1], src[i:i + 1], cls[i:i + 1], kv[i:i + 1], w, b, k=M, rho=0.2)
            assert ref[0, :k].tolist() == got


def test_class_weights_are_per_stage():
    # two classes with opposite preferences route the same stage to different nodes
    rng = np.random.default_rng(6)
    M = 2
    nodes = _nodes(rng, M, n_src=1)
    nodes["free_bytes"][:] = [50 * GB, 200 * GB]
    nodes["rtt_ms"][0] = [80, 1]                                  # the tight node is far
    kv = np.full(2, 40 * GB)
    one = np.zeros(2, np.int32)
    idx, _ = _route(nodes, one, one, np.array([0, 1], np.int32), kv, [[1, 0, 0], [0, 0, 0]],
                    [0, 100, 0, 1e6, 0, 1e6])
    assert idx[:, 0].tolist() == [1, 0]


def test_node_permutation_equivariance():
    rng = np.random.default_rng(7)
    M, N = 48, 300
    nodes = _nodes(rng, M)
    kv = rng.uniform(0, 150, N) * GB
    model, src, cls = (rng.integers(0, 8, N).astype(np.int32), rng.integers(0, 3, N).astype(np.int32),
                       rng.integers(0, 2, N).astype(np.int32))
    w = [[0.25, 1, 1], [0.1, 1, 1]]
    b = _wide_bounds(nodes)
    idx, fit = _route(nodes, model, src, cls, kv, w, b)
    perm = rng.permutation(M)
    pn = {key: (v[:, perm] if key == "rtt_ms" else v[perm]) for key, v in nodes.items()}
    idx2, fit2 = _route(pn, model, src, cls, kv, w, b)
    ok = idx[:, 0] >= 0
    assert (ok == (idx2[:, 0] >= 0)).all()
    assert (perm[idx2[ok, 0]] == idx[ok, 0]).all() and (fit2 == fit).all()


# ---- minimum-impact degradation (Alg. 2) and its cost (Eq. 4) ---------------------------------

def test_degradation_plan_closed_forms():
    dc = oracle.degradation_cost
    # one engine: enough frees it alone, too little is a Failure
    assert dc(5.0, [1], [5.0], [7.5], 100.0) == 7.5            # freed == R suffices (stop at >=)
    assert dc(5.1, [1], [5.0], [7.5], 100.0) is None
    # priority order: the level-1 engine (listed second) is taken first and suffices alone
    assert dc(3.0, [2, 1], [10.0, 4.0], [50.0, 2.0], 100.0) == 2.0
    # equal levels: lower index first
    assert dc(3.0, [1, 1], [4.0, 4.0], [2.0, 9.0], 100.0) == 2.0
    # the check comes before each engine: exactly covered by the first two -> the third is not taken
    assert dc(6.0, [1, 2, 3], [2.0, 4.0, 8.0], [1.0, 10.0, 100.0], 1000.0) == 11.0
    # the interrupt penalty is charged only when an active engine (level 4 or 5) is in the plan
    assert dc(2.0, [1, 4], [2.0, 8.0], [1.0, 3.0], 1000.0) == 1.0
    assert dc(3.0, [1, 4], [2.0, 8.0], [1.0, 3.0], 1000.0) == 1004.0
    assert dc(3.0, [1, 5], [2.0, 8.0], [1.0, 3.0], 1000.0) == 1004.0
    assert dc(3.0, [1, 3], [2.0, 8.0], [1.0, 3.0], 1000.0) == 4.0
    # nothing required: an empty plan
    assert dc(0.0, [4], [1.0], [9.0], 1000.0) == 0.0
    assert dc(-1.0, [], [], [], 1000.0) == 0.0
    assert dc(1.0, [], [], [], 1000.0) is None


def test_degradation_plan_is_the_shortest_sufficient_priority_prefix():
    # any number of engines: the definition has no cap
    rng = np.random.default_rng(8)
    for t in range(600):
        ne = int(rng.integers(0, 9)) if t < 400 else int(rng.integers(9, 80))
        level = rng.integers(1, 6, ne).astype(np.int32)
        freed = rng.choice([1.0, 2.0, 3.0, 5.0], ne)             # coarse: many exact coverings
        cost = rng.uniform(0, 100, ne).astype(np.float32)
        R = float(rng.choice([0.5, 1.0, 2.0, 3.0, 4.0, 7.0, 11.0, 30.0, 60.0, 150.0]))
        order = sorted(range(ne), key=lambda i: (level[i], i))
        want = None
        for j in range(1, ne + 1):                               # shortest prefix freeing R
            if sum(freed[order[:j]]) >= R:
                plan = order[:j]
                c = np.float32(0)
                for i in plan:
                    c = np.float32(c + cost[i])
                want = float(np.float32(c + (np.float32(250) if (level[plan] >= 4).any() else np.float32(0))))
                break
        assert oracle.degradation_cost(R, level, freed, cost, 250.0) == want


def test_late_low_level_engine_is_taken_first():
    # a ninth, tenth ... engine of the lowest level comes first in priority order: a plan that
    # truncated the list at eight engines would miss it
    level = np.array([3] * 12 + [1], np.int32)
    freed = np.array([1.0] * 12 + [50.0])
    cost = np.array([10.0] * 12 + [7.0], np.float32)
    assert oracle.degradation_cost(40.0, level, freed, cost, 1000.0) == 7.0
    assert oracle.degradation_cost(52.0, level, freed, cost, 1000.0) == 27.0     # 1-level, then two 3s
    assert oracle.degradation_cost(63.0, level, freed, cost, 1000.0) is None


def _quotient_pairs(rng, n):
    """float32 pairs (a, b), 0 < a <= b, whose correctly rounded quotient a / b differs from the
    product of a with the rounded reciprocal of b"""
    a = rng.uniform(1e8, 3e11, 20 * n).astype(np.float32)
    b = (a * rng.uniform(1.0, 8.0, a.size)).astype(np.float32)
    with np.errstate(all="ignore"):
        q = a / b
        r = a * (np.float32(1) / b)
    sel = np.flatnonzero(q != r)[:n]
    assert sel.size == n
    return a[sel], b[sel], q[sel]


def test_fit_is_the_float32_quotient():
    # gamma = lambda = mu = 0: the fitness is the fit alone, R_need / headroom rounded once
    rng = np.random.default_rng(21)
    a, b, q = _quotient_pairs(rng, 200)
    for ai, bi, qi in zip(a, b, q):
        nodes = dict(free_bytes=np.array([float(bi)]), queue_ms=np.zeros(1, np.float32),
                     act_ms=np.zeros(1, np.float32), resident_mask=np.zeros(1, np.uint64),
                     deg_ms=np.zeros(1, np.float32), rtt_ms=np.zeros((1, 1), np.float32))
        one = np.zeros(1, np.int32)
        idx, fit = _route(nodes, one, one, one, np.array([float(ai)]), [0, 0, 0], [0, 1, 0, 1, 0, 1])
        assert idx[0, 0] == 0 and fit[0, 0].view(np.uint32) == qi.view(np.uint32)


def test_normalisation_is_the_float32_quotient():
    # gamma = 1, lambda = mu = 0: the fitness is 1 - norm(RTT), norm = (x - lo) / (hi - lo)
    rng = np.random.default_rng(22)
    lo = np.float32(0.0)
    a, b, q = _quotient_pairs(rng, 100)
    for ai, bi, qi in zip(a, b, q):
        # x - lo = ai and hi - lo = bi exactly (lo = 0), inside the window
        nodes = dict(free_bytes=np.array([1e12]), queue_ms=np.zeros(1, np.float32),
                     act_ms=np.zeros(1, np.float32), resident_mask=np.zeros(1, np.uint64),
                     deg_ms=np.zeros(1, np.float32), rtt_ms=np.array([[ai]], np.float32))
        one = np.zeros(1, np.int32)
        _, fit = _route(nodes, one, one, one, np.array([1.0]), [1, 0, 0], [lo, bi, 0, 1, 0, 1])
        assert fit[0, 0].view(np.uint32) == (np.float32(1) - qi).view(np.uint32)


def test_penalties_add_before_they_leave_the_affinity():
    # S = A - (lambda T + mu C): with A = 0 (gamma = 1, RTT at the window top) the fitness is the
    # negated float32 sum of the two weighted penalties
    rng = np.random.default_rng(23)
    for _ in range(200):
        t, c = rng.uniform(0, 1, 2).astype(np.float32)
        lam, mu = rng.uniform(0.1, 3, 2).astype(np.float32)
        nodes = dict(free_bytes=np.array([1e12]), queue_ms=np.array([t], np.float32),
                     act_ms=np.zeros(1, np.float32), resident_mask=np.ones(1, np.uint64),
                     deg_ms=np.array([c], np.float32), rtt_ms=np.array([[5.0]], np.float32))
        one = np.zeros(1, np.int32)
        _, fit = _route(nodes, one, one, one, np.array([1.0]), [1, lam, mu], [0, 5, 0, 1, 0, 1])
        want = -(np.float32(lam * t) + np.float32(mu * c))
        assert fit[0, 0].view(np.uint32) == np.float32(want).view(np.uint32)


def test_fitness_with_degradation_plans():
    # node 0 cannot admit the stage and has no plan; node 1 needs a plan; node 2 fits outright
    nodes = dict(free_bytes=np.array([10, 10, 100], float) * GB,
                 queue_ms=np.zeros(3, np.float32), act_ms=np.zeros(3, np.float32),
                 resident_mask=np.zeros(3, np.uint64), deg_ms=np.zeros(3, np.float32),
                 rtt_ms=np.zeros((1, 3), np.float32))
    eng = (np.array([0, 0, 2, 2], np.int32), np.array([1, 4], np.int32), np.array([5, 20], float) * GB,
           np.array([100, 300], np.float32), 1000.0)
    one = np.zeros(1, np.int32)
    b = [0, 1, 0, 1, 0, 2000]
    route = lambda kv, w, k=3: oracle.route_fitness(one, one, one, np.array([kv]), nodes["free_bytes"], nodes["queue_ms"],
                                                    nodes["act_ms"], nodes["resident_mask"], nodes["deg_ms"],
                                                    nodes["rtt_ms"], np.array(w, np.float32).reshape(1, 3),
                                                    np.array(b, np.float32), k=k, engines=eng)
    # gamma = 1 with equal proximity everywhere: S = 1 - norm(C_deg), C_deg window [0, 2000] ms
    # 12 GB: node 1 frees 5 GB (level 1, cost 100) -> feasible with C_deg = 100; node 0 infeasible
    idx, fit = route(12 * GB, [1, 0, 1])
    assert idx[0].tolist() == [2, 1, -1]
    assert fit[0, 0] == 1.0 and abs(fit[0, 1] - (1 - 100 / 2000)) < 1e-6
    # 20 GB: node 1 needs both engines (C_deg = 100 + 300 + interrupt 1000 = 1400)
    idx, fit = route(20 * GB, [1, 0, 1])
    assert idx[0].tolist() == [2, 1, -1] and abs(fit[0, 1] - (1 - 1400 / 2000)) < 1e-6
    # 40 GB: node 1 cannot free enough either; only node 2
    idx, _ = route(40 * GB, [1, 0, 1])
    assert idx[0].tolist() == [2, -1, -1]
    # with mu = 0 feasibility equals "need <= headroom + everything freeable" (node 1: 35 GB)
    rng = np.random.default_rng(9)
    for kv in rng.uniform(0, 120, 200) * GB:
        idx, _ = route(kv, [0, 1, 0])
        feas = {j for j, cap in enumerate([10, 35, 100]) if kv <= cap * GB}
        assert {j for j in idx[0] if j >= 0} == feas
