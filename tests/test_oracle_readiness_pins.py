"""Pins of the oracle's model-readiness inputs (Sec. III-C: five readiness states, T_act from a
profiled bandwidth model, Size / BW_tier) and their use as T_act(N, M(T)) in Eq. 6 -- no GPU."""
import numpy as np

import oracle

GB = 1e9
BW = np.array([1.0, 25.0, 25.0, 3.0, 1.25]) * GB           # bytes/s per tier (tier 0 unused)
SETUP = np.array([0.0, 150.0, 2500.0, 2500.0, 4000.0], np.float32)


def test_activation_latency_closed_forms():
    rng = np.random.default_rng(1)
    M, K = 40, 7
    tier = rng.integers(0, 8, (M, K)).astype(np.uint8)
    size = rng.uniform(1, 30, K) * GB
    act = oracle.activation_latency(tier, size, BW, SETUP)
    assert np.all(act[tier == 0] == 0.0)                    # Running: nothing to activate
    # tiers past Remote count as Remote
    assert np.array_equal(act, oracle.activation_latency(np.minimum(tier, 4), size, BW, SETUP))
    # size 0 leaves the setup; 1 GB over 1 GB/s is 1000 ms exactly
    z = oracle.activation_latency(tier, np.zeros(K), BW, SETUP)
    assert np.array_equal(z, np.where(tier == 0, 0.0, SETUP[np.minimum(tier, 4)]).astype(np.float32))
    one = oracle.activation_latency(np.full((1, 1), 4, np.uint8), np.array([1.25 * GB]), BW, np.zeros(5, np.float32))
    assert one[0, 0] == 1000.0
    # without setup, doubling every bandwidth halves every latency exactly (powers of two)
    a1 = oracle.activation_latency(tier, size, BW, np.zeros(5, np.float32))
    a2 = oracle.activation_latency(tier, size, 2 * BW, np.zeros(5, np.float32))
    assert np.array_equal(a1, 2 * a2)
    # slower tiers of the same model take longer (bandwidths fall, setups rise from tier 1 on)
    for m in range(K):
        lat = oracle.activation_latency(np.arange(5, dtype=np.uint8)[:, None].repeat(1, 1), size[m:m + 1], BW, SETUP)
        assert lat[0, 0] == 0.0 and np.all(np.diff(lat[1:, 0]) > 0)


def _fitness_case(rng, n, M, n_models=16):
    nodes = dict(free_bytes=rng.uniform(0, 300, M) * GB, queue_ms=rng.uniform(0, 5000, M).astype(np.float32),
                 act_ms=rng.uniform(2000, 20000, M).astype(np.float32),
                 resident_mask=rng.integers(0, 1 << n_models, M).astype(np.uint64),
                 deg_ms=rng.uniform(0, 500, M).astype(np.float32), rtt_ms=rng.uniform(0.2, 80, (3, M)).astype(np.float32))
    stages = dict(model=rng.integers(0, n_models, n).astype(np.int32), src=rng.integers(0, 3, n).astype(np.int32),
                  cls=rng.integers(0, 2, n).astype(np.int32), kv=rng.uniform(0, 250, n) * GB)
    return nodes, stages


def _route(nodes, st, weights, bounds, k=3, n_models=16, act_matrix=None):
    return oracle.route_fitness(st["model"], st["src"], st["cls"], st["kv"], nodes["free_bytes"], nodes["queue_ms"],
                                nodes["act_ms"], nodes["resident_mask"], nodes["deg_ms"], nodes["rtt_ms"],
                                np.asarray(weights, np.float32), np.asarray(bounds, np.float32), k=k,
                                n_models=n_models, act_matrix=act_matrix)


def test_matrix_of_resident_bits_equals_the_mask_form():
    # T_act(N, m) = 0 where m is resident on N, the node's activation latency otherwise: the same
    # fitness, bit for bit, as the resident-mask form of Eq. 6
    rng = np.random.default_rng(2)
    nodes, st = _fitness_case(rng, 800, 300)
    bits = (nodes["resident_mask"][:, None] >> np.arange(16, dtype=np.uint64)[None, :]) & np.uint64(1)
    mat = np.where(bits == 1, 0.0, nodes["act_ms"][:, None]).astype(np.float32)
    w, b = [[0.25, 1, 1], [0.1, 1, 1]], [0, 80, 0, 25000, 0, 500]
    i0, f0 = _route(nodes, st, w, b)
    i1, f1 = _route(nodes, st, w, b, act_matrix=mat)
    assert np.array_equal(i0, i1) and np.array_equal(f0.view(np.uint32), f1.view(np.uint32))


def test_readiness_is_per_model():
    # two nodes, equal in everything but which model is warm on which: with proximity equal and
    # lambda = 1, each model's stages go to the node where that model is ready
    M, n_models = 2, 2
    nodes = dict(free_bytes=np.full(M, 100 * GB), queue_ms=np.zeros(M, np.float32), act_ms=np.zeros(M, np.float32),
                 resident_mask=np.zeros(M, np.uint64), deg_ms=np.zeros(M, np.float32),
                 rtt_ms=np.ones((1, M), np.float32))
    tier = np.array([[0, 4], [3, 1]], np.uint8)              # node 0: model 0 running; node 1: model 1 sleeping
    act = oracle.activation_latency(tier, np.array([16 * GB, 16 * GB]), BW, SETUP)
    st = dict(model=np.array([0, 1, 0, 1], np.int32), src=np.zeros(4, np.int32), cls=np.zeros(4, np.int32),
              kv=np.full(4, GB))
    idx, _ = _route(nodes, st, [[1, 1, 0]], [0, 1, 0, 20000, 0, 1], k=1, n_models=n_models, act_matrix=act)
    assert idx[:, 0].tolist() == [0, 1, 0, 1]
    # the same stages with the tiers swapped swap nodes
    act2 = oracle.activation_latency(tier[::-1].copy(), np.array([16 * GB, 16 * GB]), BW, SETUP)
    idx, _ = _route(nodes, st, [[1, 1, 0]], [0, 1, 0, 20000, 0, 1], k=1, n_models=n_models, act_matrix=act2)
    assert idx[:, 0].tolist() == [1, 0, 1, 0]


# ---- adaptive safety margin (Sec. III-D): EWMA of the relative underestimation, high quantile ----

def test_adaptive_rho_closed_forms():
    rng = np.random.default_rng(5)
    m = 2000
    pred = rng.uniform(1, 100, m) * GB
    actual = pred * rng.lognormal(0.0, 0.3, m)
    e = np.maximum(actual / pred - 1.0, 0.0)
    # beta = 1: no smoothing, the EWMA is e itself; rho its "higher" percentile
    ew, rho = oracle.adaptive_rho(actual, pred, 1.0, 0.95)
    assert np.array_equal(ew, e.astype(np.float32))
    assert rho == np.percentile(ew, 95, method="higher")
    # exact or over-estimating predictions: no margin
    ew, rho = oracle.adaptive_rho(pred, pred, 0.2, 0.9)
    assert not ew.any() and rho == 0.0
    ew, rho = oracle.adaptive_rho(0.5 * pred, pred, 0.2, 0.9)
    assert not ew.any() and rho == 0.0
    # a constant underestimation of 25% is its own average and quantile
    ew, rho = oracle.adaptive_rho(1.25 * pred, pred, 0.3, 0.9)
    assert np.all(ew == np.float32(0.25)) and rho == np.float32(0.25)


def test_adaptive_rho_recursion_and_window_quantile():
    # one underestimate followed by exact predictions decays geometrically: e~_i = x (1 - beta)^i
    m, beta, x = 50, 0.2, 0.8
    pred = np.full(m, 1e9)
    actual = pred.copy()
    actual[0] = (1 + x) * 1e9
    ew, rho = oracle.adaptive_rho(actual, pred, beta, 0.5)
    np.testing.assert_allclose(ew, x * (1 - beta) ** np.arange(m), rtol=1e-6)
    assert rho == np.sort(ew)[int(np.ceil(0.5 * (m - 1)))]
    # the quantile is over the smoothed values, not the raw errors: alternating errors smooth out
    pred = np.full(1000, 1e9)
    actual = np.where(np.arange(1000) % 2 == 0, 2e9, 1e9)          # e alternates 1, 0
    ew, rho = oracle.adaptive_rho(actual, pred, 0.1, 0.95)
    assert 0.45 < rho < 0.6                                       # near the mean 0.5, far below 1
    assert rho == np.percentile(ew, 95, method="higher")


def test_activation_latency_units_and_latency_routing():
    # the time unit: 2.5 GB over 1.25 GB/s is 2 s, 2000 ms; setups are taken in the same unit
    tier = np.array([[4, 0]], np.uint8)
    size = np.array([2.5 * GB, 7 * GB])
    assert oracle.activation_latency(tier, size, BW, np.zeros(5, np.float32), unit=1.0)[0].tolist() == [2.0, 0.0]
    assert oracle.activation_latency(tier, size, BW, np.zeros(5, np.float32))[0].tolist() == [2000.0, 0.0]
    assert oracle.activation_latency(tier, size, BW, np.full(5, 0.5, np.float32), unit=1.0)[0, 0] == 2.5
    # latency routing (Alg. 3 with Eq. 6): a {0, cold} matrix in seconds equals the resident-mask form
    rng = np.random.default_rng(6)
    M, n, K = 400, 2000, 16
    free = rng.uniform(0, 300, M) * GB
    q = rng.uniform(0, 5, M).astype(np.float32)
    cold = rng.uniform(2, 20, M).astype(np.float32)
    mask = rng.integers(0, 1 << K, M).astype(np.uint64)
    model = rng.integers(0, K, n).astype(np.int32)
    pred = rng.uniform(10, 2000, n).astype(np.float32)
    kv = rng.uniform(0, 250, n) * GB
    dec = rng.uniform(0.01, 0.04, K).astype(np.float32)
    bits = (mask[:, None] >> np.arange(K, dtype=np.uint64)[None, :]) & np.uint64(1)
    mat = np.where(bits == 1, 0.0, cold[:, None]).astype(np.float32)
    i0, s0 = oracle.route(model, pred, kv, dec, free, q, cold, mask, k=3)
    i1, s1 = oracle.route(model, pred, kv, dec, free, q, cold, mask, k=3, act_matrix=mat)
    assert np.array_equal(i0, i1) and np.array_equal(s0.view(np.uint32), s1.view(np.uint32))
    # with tiers, a stage goes to the node whose ready time for its own model is least
    tier = rng.integers(0, 5, (M, K)).astype(np.uint8)
    act = oracle.activation_latency(tier, rng.uniform(1, 28, K) * GB, BW, SETUP / 1000, unit=1.0)
    i2, s2 = oracle.route(model, pred, kv, dec, np.full(M, 1e15), q, cold, mask, k=1, act_matrix=act)
    ready = q[None, :] + act.T[model]
    best = np.lexsort((np.broadcast_to(np.arange(M), ready.shape), (ready + (pred * dec[model])[:, None]).astype(np.float32)), axis=1)
    assert np.array_equal(i2[:, 0], best[:, 0])
