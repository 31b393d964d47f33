"""Parity of the HIP path (through the C-ABI) with the CPU oracle, on seeded inputs.

Bars (element by element):
  predict    : |pred_gpu - pred_oracle| <= 1e-3 |pred_oracle| (float32 predictor) or
               1e-2 |pred_oracle| (bfloat16 predictor); kv_bytes equal, bit for bit, to
               Eq. 3 evaluated on the GPU's own predicted length.
  route      : node indices and scores bit-exact, given the same pred/kv inputs.
  prioritize : remaining time, slack keys and order bit-exact, given the same latencies.
Full-size workloads are checked on sampled stages (predict) or in full (route, prioritize).
"""
import functools

import numpy as np
import pytest
import torch

import oracle
import paper_2606_12950_amd as M
from paper_2606_12950_amd import pipeline
from paper_2606_12950_amd import workload as W
from route_guard import explain_route_differences

pytestmark = pytest.mark.gpu

PRED_TOL = {"f32": 1e-3, "bf16": 1e-2}


@functools.lru_cache(maxsize=None)
def _wl(name, **kw):
    return W.workload(name, **dict(kw))


def wl(name, **kw):
    return _wl(name, **kw)


def _np(t):
    return t.detach().cpu().numpy()


def gpu_predict(w):
    b = pipeline.to_device(w)
    o = pipeline.allocate_outputs(b)
    pipeline.run_predict(b, o)
    torch.cuda.synchronize()
    return _np(o.pred_len), _np(o.kv_bytes), b, o


def check_pred(w, pred_g, kv_g, rows=None):
    sel = slice(None) if rows is None else rows
    pred_o, _ = oracle.predict_workload(w, rows=rows)
    pg = pred_g[sel]
    rel = np.abs(pg.astype(np.float64) - pred_o) / np.abs(pred_o)
    assert np.all(np.isfinite(pg))
    assert rel.max() <= PRED_TOL[w.spec.dtype], f"max rel err {rel.max():.3e}"
    # Eq. 3 on the GPU's own prediction, exact in float64
    alpha = w.kv_bytes_per_token[w.model_id[sel]].astype(np.float64)
    assert np.array_equal(kv_g[sel], (w.prompt_len[sel].astype(np.float64) + pg.astype(np.float64)) * alpha)
    return rel.max()


def test_library_is_the_in_tree_build():
    lib = M.load()
    assert M.LIBRARY_PATH.endswith("paper_2606_12950_amd/libmaestro.so")
    for f in M._native.EXPORTS:
        assert hasattr(lib, f)


# ----------------------------------------------------------------------------------------------
# predict
# ----------------------------------------------------------------------------------------------

@pytest.mark.parametrize("name,n", [("c0", None), ("c0", 1), ("c0", 129), ("c1", 1), ("c1", 7), ("c1", 257),
                                    ("c1", 1000), ("c1", None), ("c1", 131_149), ("c4", 1), ("c4", 777)])
def test_predict_matches_oracle(name, n):
    w = wl(name) if n is None else wl(name, n_stages=n)
    pred_g, kv_g, _, _ = gpu_predict(w)
    err = check_pred(w, pred_g, kv_g)
    print(f"{name} n={w.n}: predict max rel err {err:.2e}")


@pytest.mark.parametrize("name,sample", [("c2", 3000), ("c4", 2000)])
def test_predict_full_size_sampled(name, sample):
    w = wl(name)
    pred_g, kv_g, _, _ = gpu_predict(w)
    rows = np.sort(np.random.default_rng(99).choice(w.n, sample, replace=False))
    rows = np.unique(np.concatenate([rows, [0, w.n - 1]]))
    err = check_pred(w, pred_g, kv_g, rows=rows)
    assert np.all(np.isfinite(pred_g)) and pred_g.min() >= 32.0 and pred_g.max() <= 4064.0
    print(f"{name}: predict sampled max rel err {err:.2e}")


@pytest.mark.parametrize("name,shift", [("c1", 1000.0), ("c1", -1000.0), ("c4", 1000.0), ("c4", -1000.0)])
def test_predict_shifted_logits(name, shift):
    # the softmax is invariant to a common shift of the logits; +-1000 on every output bias
    # overflows (or underflows) float32 e^z unless the row maximum is subtracted first
    import dataclasses
    w = wl(name, n_stages=2000)
    w = dataclasses.replace(w, biases=w.biases[:-1] + [(w.biases[-1] + np.float32(shift)).astype(np.float32)])
    pred_g, kv_g, _, _ = gpu_predict(w)
    err = check_pred(w, pred_g, kv_g)
    print(f"{name} logits {shift:+.0f}: predict max rel err {err:.2e}")


@pytest.mark.parametrize("name", ["c0", "c1", "c4"])
def test_predict_zero_weights_is_exact_mean_centre(name):
    # uniform softmax: the expected length is the mean of the bin centres, exactly
    w = wl(name, n_stages=300)
    b = pipeline.to_device(w)
    b.weights = [torch.zeros_like(t) for t in b.weights]
    o = pipeline.allocate_outputs(b)
    pipeline.run_predict(b, o)
    torch.cuda.synchronize()
    expect = np.float32(w.bin_centre.astype(np.float64).mean())
    assert np.all(_np(o.pred_len) == expect)


def test_predict_is_deterministic_and_empty_is_noop():
    w = wl("c1", n_stages=5000)
    p1, k1, b, o = gpu_predict(w)
    p2, k2, _, _ = gpu_predict(w)
    assert np.array_equal(p1, p2) and np.array_equal(k1, k2)
    e = torch.empty((0, 256), dtype=torch.bfloat16, device="cuda")
    pr, kv = M.predict(e, b.weights, b.biases, b.bin_centre, b.prompt_len[:0], b.model_id[:0],
                       b.kv_bytes_per_token)
    assert pr.numel() == 0 and kv.numel() == 0


def test_predict_rejects_unsupported_and_bad_args():
    w = wl("c1", n_stages=10)
    b = pipeline.to_device(w)
    # a shape the kernels are not built for
    w_odd = [torch.zeros((96, 256), dtype=torch.bfloat16, device="cuda"),
             torch.zeros((64, 96), dtype=torch.bfloat16, device="cuda")]
    b_odd = [torch.zeros(96, device="cuda"), torch.zeros(64, device="cuda")]
    with pytest.raises(M.MaestroError) as e:
        M.predict(b.x, w_odd, b_odd, b.bin_centre, b.prompt_len, b.model_id, b.kv_bytes_per_token)
    assert e.value.status == 2
    # misaligned feature pointer
    xs = b.x.flatten()[1:1 + 9 * 256].view(9, 256)
    with pytest.raises(M.MaestroError) as e:
        M.predict(xs, b.weights, b.biases, b.bin_centre, b.prompt_len[:9], b.model_id[:9],
                  b.kv_bytes_per_token)
    assert e.value.status == 1


# ----------------------------------------------------------------------------------------------
# route (bit-exact given identical inputs)
# ----------------------------------------------------------------------------------------------

ALGOS = {"scan": M._native.ROUTE_SCAN, "sorted": M._native.ROUTE_SORTED}


def gpu_route(w, pred, kv, free=None, queue=None, cold=None, mask=None, dec=None, k=None, rho=None,
              model=None, algo=0):
    t = lambda a: pipeline._t(a, "cuda")
    model = w.model_id if model is None else model
    args = dict(free=w.free_bytes if free is None else free, queue=w.queue_s if queue is None else queue,
                cold=w.cold_s if cold is None else cold, mask=w.resident_mask if mask is None else mask,
                dec=w.decode_s_per_token if dec is None else dec)
    k = w.spec.k if k is None else k
    rho = w.spec.rho if rho is None else rho
    idx, sc = M.route(t(model), t(pred), t(kv), t(args["dec"]), t(args["free"]), t(args["queue"]),
                      t(args["cold"]), t(args["mask"]), k=k, rho=rho, algo=algo)
    torch.cuda.synchronize()
    ref = oracle.route(model, pred, kv, args["dec"], args["free"], args["queue"], args["cold"],
                       args["mask"], k=k, rho=rho)
    return (_np(idx), _np(sc)), ref


def assert_route_equal(got, ref):
    gi, gs = got
    ri, rs = ref
    bad = np.nonzero(np.any(gi != ri, axis=1) | np.any(gs.view(np.uint32) != rs.view(np.uint32), axis=1))[0]
    assert bad.size == 0, f"{bad.size} stages differ, first {bad[:5]}: gpu {gi[bad[:3]]} {gs[bad[:3]]} " \
                          f"oracle {ri[bad[:3]]} {rs[bad[:3]]}"


@pytest.mark.parametrize("algo", ["scan", "sorted"])
@pytest.mark.parametrize("name", ["c0", "c1", "c2", "c3"])
def test_route_matches_oracle_full(name, algo):
    w = wl(name)
    pred, kv, _, _ = gpu_predict(w)
    got, ref = gpu_route(w, pred, kv, algo=ALGOS[algo])
    assert_route_equal(got, ref)
    infeasible = float(np.mean(ref[0][:, 0] < 0))
    print(f"{name}: {w.n} stages x {w.spec.n_nodes} nodes, routes identical; unroutable {infeasible:.4%}")


@pytest.mark.parametrize("algo", ["scan", "sorted"])
def test_route_c4_top4_sampled_stages(algo):
    # full c4 on the GPU (4,194,304 stages x 4,096 nodes, top-4); oracle on a stage sample
    w = wl("c4")
    pred, kv, b, o = gpu_predict(w)
    pipeline.run_route(b, o, algo=ALGOS[algo])
    torch.cuda.synchronize()
    gi, gs = _np(o.node_idx), _np(o.score)
    rows = np.sort(np.random.default_rng(7).choice(w.n, 20000, replace=False))
    rows = np.unique(np.concatenate([rows, [0, w.n - 1]]))
    ref = oracle.route(w.model_id[rows], pred[rows], kv[rows], w.decode_s_per_token, w.free_bytes,
                       w.queue_s, w.cold_s, w.resident_mask, k=4)
    assert_route_equal((gi[rows], gs[rows]), ref)


@pytest.mark.parametrize("algo", ["scan", "sorted"])
def test_route_c4_contended_sampled_stages(algo):
    # c4 with every node's headroom divided by 48 (U[0, 0.625] GB): most stage-node pairs are
    # infeasible, so the sorted walk skips many nodes per stage and some stages have fewer than k
    # feasible nodes; full launch on the GPU, the oracle on a stage sample
    w = wl("c4")
    pred, kv, b, o = gpu_predict(w)
    free = w.free_bytes / 48.0
    idx, sc = M.route(b.model_id, o.pred_len, o.kv_bytes, b.decode_s_per_token, pipeline._t(free, "cuda"),
                      b.queue_s, b.cold_s, b.resident_mask, k=4, rho=w.spec.rho, algo=ALGOS[algo])
    torch.cuda.synchronize()
    gi, gs = _np(idx), _np(sc)
    rows = np.sort(np.random.default_rng(11).choice(w.n, 20000, replace=False))
    rows = np.unique(np.concatenate([rows, [0, w.n - 1]]))
    assert (kv[rows][:, None] > free[None, :]).mean() > 0.5
    assert (gi[rows] < 0).any()             # some sampled stages fit fewer than 4 nodes
    ref = oracle.route(w.model_id[rows], pred[rows], kv[rows], w.decode_s_per_token, free,
                       w.queue_s, w.cold_s, w.resident_mask, k=4)
    assert_route_equal((gi[rows], gs[rows]), ref)


@pytest.mark.parametrize("algo", ["scan", "sorted"])
@pytest.mark.parametrize("k", [1, 3, 4, 16])
@pytest.mark.parametrize("n,M_", [(1, 1), (7, 3), (300, 64), (2500, 1500), (40000, 37), (3000, 8192)])
def test_route_shapes_and_widths(n, M_, k, algo):
    # ragged stage tiles, node chunks that do not divide, several lanes per stage, k > #nodes
    w = wl("c1", n_stages=n, n_nodes=M_, with_x=False)
    rng = np.random.default_rng(n * 31 + M_)
    pred = rng.uniform(32, 4064, n).astype(np.float32)
    kv = (w.prompt_len + pred.astype(np.float64)) * w.kv_bytes_per_token[w.model_id].astype(np.float64)
    got, ref = gpu_route(w, pred, kv, free=w.free_bytes / 60.0, k=k, algo=ALGOS[algo])
    assert_route_equal(got, ref)


@pytest.mark.parametrize("algo", ["scan", "sorted"])
def test_route_ties_and_boundaries(algo):
    # coarse value grids: many exactly equal scores and free == need boundaries
    rng = np.random.default_rng(5)
    n, M_, K = 5000, 700, 64
    w = wl("c4", n_stages=n, n_nodes=M_, with_x=False)
    model = rng.integers(0, K, n).astype(np.int32)
    pred = rng.choice(np.array([64.0, 128.0, 256.0], np.float32), n)
    kv = rng.choice(np.array([1e9, 2e9, 3e9, 4e9]), n)      # 4e9 fits no node
    free = rng.choice(np.array([0.5e9, 1e9, 2e9, 3e9]), M_)
    q = rng.choice(np.array([0.0, 0.5, 1.0], np.float32), M_)
    cold = rng.choice(np.array([2.0, 4.0], np.float32), M_)
    mask = rng.integers(0, 2 ** 63, M_, dtype=np.int64).astype(np.uint64) | \
        (rng.integers(0, 2, M_).astype(np.uint64) << np.uint64(63))
    dec = rng.choice(np.array([0.015625, 0.03125], np.float32), K)
    for k, rho in [(1, 0.0), (4, 0.0), (5, 0.25)]:
        got, ref = gpu_route(w, pred, kv, free=free, queue=q, cold=cold, mask=mask, dec=dec, k=k,
                             rho=rho, model=model, algo=ALGOS[algo])
        assert_route_equal(got, ref)
        if k == 1:
            assert np.any(ref[0][:, 0] < 0) and np.any(ref[0][:, 0] >= 0)


@pytest.mark.parametrize("algo", ["scan", "sorted"])
def test_route_all_infeasible_and_equal_scores(algo):
    w = wl("c0", n_stages=100, with_x=False)
    pred = np.full(100, 500.0, np.float32)
    kv = np.full(100, 1e12)   # more than any node has
    got, ref = gpu_route(w, pred, kv, k=4, algo=ALGOS[algo])
    assert np.all(got[0] == -1) and np.all(np.isinf(got[1]))
    assert_route_equal(got, ref)
    # identical nodes: lowest feasible index first
    M_ = w.spec.n_nodes
    got, ref = gpu_route(w, pred, np.full(100, 1e9), free=np.full(M_, 1e9), queue=np.ones(M_, np.float32),
                         cold=np.ones(M_, np.float32), mask=np.zeros(M_, np.uint64), k=4, algo=ALGOS[algo])
    assert np.all(got[0] == np.arange(4)[None, :])
    assert_route_equal(got, ref)


# ----------------------------------------------------------------------------------------------
# prioritize (bit-exact given identical latencies)
# ----------------------------------------------------------------------------------------------

def gpu_prioritize(off, lat, dl, now, cursor=None):
    t = lambda a: pipeline._t(a, "cuda")
    rem, key, order = M.prioritize(t(off), t(lat), t(dl), now,
                                   cursor=None if cursor is None else t(cursor))
    torch.cuda.synchronize()
    return _np(rem), _np(key), _np(order)


def assert_prio_equal(got, ref):
    for g, r, what in zip(got, ref, ("remaining_us", "slack_key", "order")):
        bad = np.nonzero(g != r)[0]
        assert bad.size == 0, f"{what}: {bad.size} differ, first {bad[:5]}: {g[bad[:5]]} vs {r[bad[:5]]}"


def test_c3_full_step_matches_oracle():
    # the whole hot path on c3: predict -> route -> prioritize on the routed scores
    w = wl("c3")
    b = pipeline.to_device(w)
    o = pipeline.run_step(b)
    torch.cuda.synchronize()
    pred, kv = _np(o.pred_len), _np(o.kv_bytes)
    rows = np.sort(np.random.default_rng(3).choice(w.n, 3000, replace=False))
    check_pred(w, pred, kv, rows=rows)
    ref_r = oracle.route_workload(w, pred, kv)
    assert_route_equal((_np(o.node_idx), _np(o.score)), ref_r)
    lat = _np(o.score)[:, 0]
    ref_p = oracle.prioritize(w.chain_offset, lat, w.deadline_us, w.now_us)
    assert_prio_equal((_np(o.remaining_us), _np(o.slack_key), _np(o.order)), ref_p)
    print(f"c3: W={w.n_workflows} S={w.n}: route + order identical")


@pytest.mark.parametrize("name,sample", [("c1", None), ("c2", 20000), ("c3", 20000), ("c4", 3000)])
def test_end_to_end_match_rate_with_guard_bands(name, sample):
    # oracle predict -> oracle route against GPU predict -> GPU route. The predictions agree only
    # to the predictor tolerance, so a node choice may legitimately differ; every difference must
    # be explained by one of the two ways a prediction enters routing: some node's feasibility
    # flips between the two predictions (the demand straddles its headroom), or the two choices'
    # scores under the oracle's prediction tie to within float32 rounding (a prediction adds the
    # same decode term to every node of the stage, so it can reorder nodes only through rounding)
    w = wl(name)
    b = pipeline.to_device(w)
    o = pipeline.allocate_outputs(b)
    pipeline.run_predict(b, o)
    pipeline.run_route(b, o)
    torch.cuda.synchronize()
    rows = (np.arange(w.n) if sample is None
            else np.sort(np.random.default_rng(17).choice(w.n, sample, replace=False)))
    kv_g = _np(o.kv_bytes)[rows]
    idx_g = _np(o.node_idx)[rows]
    pred_o, kv_o = oracle.predict_workload(w, rows=rows)
    idx_o, _ = oracle.route_workload(w, pred_o, kv_o, rows=rows)
    rate, flips, ties = explain_route_differences(w, rows, pred_o, kv_o, idx_o, kv_g, idx_g)
    print(f"{name}: {rows.size} stages, node lists identical for {rate:.5%}; "
          f"{flips} feasibility flips, {ties} rounding ties")
    assert rate > 0.99


@pytest.mark.parametrize("W_", [1, 5, 1023, 1024, 1025, 4097, 131072, 131073, 300001, 1 << 20, (1 << 22) + 3])
def test_prioritize_random_chains(W_):
    rng = np.random.default_rng(W_)
    lens = rng.integers(0, 9, W_)
    off = np.zeros(W_ + 1, np.int64)
    off[1:] = np.cumsum(lens)
    S = int(off[-1])
    lat = rng.uniform(0.0, 200.0, S).astype(np.float32)
    lat[rng.random(S) < 0.001] = np.inf
    dl = rng.integers(0, 720 * 10 ** 6, W_).astype(np.int64)
    cur = rng.integers(-1, 10, W_).astype(np.int32)
    got = gpu_prioritize(off, lat, dl, 600 * 10 ** 6, cursor=cur)
    ref = oracle.prioritize(off, lat, dl, 600 * 10 ** 6, cursor=cur)
    assert_prio_equal(got, ref)


def test_prioritize_adversarial_keys():
    rng = np.random.default_rng(11)
    W_ = 50000
    off = np.arange(W_ + 1, dtype=np.int64)
    cases = {
        "all_equal": (np.zeros(W_, np.float32), np.full(W_, 5, np.int64)),
        "sorted": (np.zeros(W_, np.float32), np.arange(W_, dtype=np.int64)),
        "reverse": (np.zeros(W_, np.float32), np.arange(W_, 0, -1, dtype=np.int64)),
        "extremes": (np.zeros(W_, np.float32),
                     rng.choice(np.array([-(2 ** 62), -(2 ** 31), -(2 ** 31) + 1, -1, 0, 1, 2 ** 31 - 2,
                                          2 ** 31 - 1, 2 ** 31, 2 ** 62], np.int64), W_)),
        "nonfinite": (rng.choice(np.array([0.5, np.inf, np.nan, -np.inf, 1e30], np.float32), W_),
                      rng.integers(0, 10 ** 9, W_).astype(np.int64)),
        "few_keys": (np.zeros(W_, np.float32), rng.choice(np.array([7, 3, 7 + 2 ** 20], np.int64), W_)),
    }
    for name, (lat, dl) in cases.items():
        got = gpu_prioritize(off, lat, dl, 0)
        ref = oracle.prioritize(off, lat, dl, 0)
        assert_prio_equal(got, ref)
        if name == "all_equal":
            assert np.array_equal(got[2], np.arange(W_))


def gpu_route_tiered(w, pred, kv, act_s, k=None, rho=None, free=None, algo=0):
    t = lambda a: pipeline._t(a, "cuda")
    k = w.spec.k if k is None else k
    rho = w.spec.rho if rho is None else rho
    free = w.free_bytes if free is None else free
    idx, sc = M.route(t(w.model_id), t(pred), t(kv), t(w.decode_s_per_token), t(free), t(w.queue_s), None, None,
                      k=k, rho=rho, algo=algo, act_s=t(act_s))
    torch.cuda.synchronize()
    ref = oracle.route(w.model_id, pred, kv, w.decode_s_per_token, free, w.queue_s, w.cold_s, w.resident_mask,
                       k=k, rho=rho, act_matrix=act_s)
    return (_np(idx), _np(sc)), ref


@pytest.mark.parametrize("algo", ["scan", "sorted"])
@pytest.mark.parametrize("name", ["c1", "c3"])
def test_route_tiered_full(name, algo):
    # T_act(N, M(T)) of Eq. 6 from readiness tiers (seconds), both algorithms, every stage
    w = wl(name)
    r = W.readiness_inputs(w)
    act = M.activation_latency(pipeline._t(r.tier, "cuda"), pipeline._t(r.model_bytes, "cuda"),
                               pipeline._t(r.tier_bw, "cuda"),
                               pipeline._t((r.tier_setup_ms / np.float32(1000)).astype(np.float32), "cuda"), unit=1.0)
    torch.cuda.synchronize()
    act = _np(act)
    assert np.array_equal(act.view(np.uint32), oracle.activation_latency(
        r.tier, r.model_bytes, r.tier_bw, (r.tier_setup_ms / np.float32(1000)).astype(np.float32), unit=1.0).view(np.uint32))
    pred, kv, _, _ = gpu_predict(w)
    got, ref = gpu_route_tiered(w, pred, kv, act, algo=ALGOS[algo])
    assert_route_equal(got, ref)


@pytest.mark.parametrize("algo", ["scan", "sorted"])
@pytest.mark.parametrize("n,M_,K,k", [(1, 1, 1, 1), (500, 129, 64, 3), (3000, 1100, 33, 4), (777, 2049, 16, 16)])
def test_route_tiered_shapes(n, M_, K, k, algo):
    # ragged node chunks (128 per chunk for the scan), up to 64 models, tie-prone coarse values
    rng = np.random.default_rng(n + M_ + K)
    w = wl("c0", n_stages=n, n_nodes=M_, n_models=K)
    act = np.round(rng.uniform(0, 30, (M_, K)), 0).astype(np.float32)
    act[rng.random((M_, K)) < 0.3] = 0.0
    pred, kv, _, _ = gpu_predict(w)
    got, ref = gpu_route_tiered(w, pred, kv, act, k=k, free=w.free_bytes / 4.0, algo=ALGOS[algo])
    assert_route_equal(got, ref)


def test_route_tiered_of_resident_bits_equals_route():
    # a {0, cold} matrix routes exactly like the residency bits on the GPU too
    w = wl("c1")
    pred, kv, _, _ = gpu_predict(w)
    K = w.spec.n_models
    bits = (w.resident_mask[:, None] >> np.arange(K, dtype=np.uint64)[None, :]) & np.uint64(1)
    act = np.where(bits == 1, 0.0, w.cold_s[:, None]).astype(np.float32)
    for algo in ALGOS.values():
        got, _ = gpu_route_tiered(w, pred, kv, act, algo=algo)
        plain, _ = gpu_route(w, pred, kv, algo=algo)
        assert_route_equal(got, plain)


def test_route_sorted_rejects_too_many_nodes():
    w = wl("c1", n_stages=10, n_nodes=8193, with_x=False)
    pred = np.full(10, 100.0, np.float32)
    kv = np.full(10, 1e9)
    with pytest.raises(M.MaestroError) as e:
        gpu_route(w, pred, kv, algo=ALGOS["sorted"])
    assert e.value.status == 2
    got, ref = gpu_route(w, pred, kv)            # auto falls back to the scan
    assert_route_equal(got, ref)


def test_prioritize_mixed_staging():
    # 1024-workflow blocks whose stage ranges sit exactly at, below and above the 8192-stage
    # LDS staging capacity, in one batch: blocks walk their chains through LDS or in global
    # memory independently
    rng = np.random.default_rng(17)
    lens = np.concatenate([
        np.full(1024, 8),                                     # 8192 stages: at the capacity
        np.concatenate([[5000], np.full(1023, 3)]),          # 8069: below
        np.concatenate([[9000], np.zeros(1023, np.int64)]),  # 9000: above, one long chain
        rng.integers(0, 9, 777),                              # partial last block
    ]).astype(np.int64)
    W_ = lens.size
    off = np.zeros(W_ + 1, np.int64)
    off[1:] = np.cumsum(lens)
    S = int(off[-1])
    lat = rng.uniform(0.0, 30.0, S).astype(np.float32)
    lat[rng.random(S) < 0.002] = np.inf
    dl = rng.integers(0, 720 * 10 ** 6, W_).astype(np.int64)
    cur = rng.integers(0, 4, W_).astype(np.int32)
    got = gpu_prioritize(off, lat, dl, 600 * 10 ** 6, cursor=cur)
    assert_prio_equal(got, oracle.prioritize(off, lat, dl, 600 * 10 ** 6, cursor=cur))


@pytest.mark.parametrize("case", ["staged", "unstaged", "cursors_inf", "mixed_blocks", "very_long"])
def test_prioritize_block_scanned_long_chains(case):
    # chains of more than 1,024 stages are scanned by the whole block (1,024-stage chunks from
    # the end, saturating sums): inside a block staged in LDS, in one walking global memory,
    # with cursors anywhere (also past the end) and infinite latencies at chunk edges, several
    # in one block beside short ones, and one chain of 2^22 stages
    rng = np.random.default_rng(len(case))
    if case == "staged":            # 1,025 + 3,000 + short: the block's 8,192-stage range is staged
        lens = np.concatenate([[1025, 3000], np.full(1022, 3)])
    elif case == "unstaged":
        lens = np.concatenate([[1024, 1025, 2047, 2048, 2049, 9000], rng.integers(0, 9, 1018)])
    elif case == "cursors_inf":
        lens = np.concatenate([[5000, 4097, 1536], rng.integers(0, 6, 2000)])
    elif case == "mixed_blocks":
        lens = np.concatenate([rng.integers(0, 9, 1500), [3000], rng.integers(0, 9, 600), [1100, 1100]])
    else:
        lens = np.array([1 << 22, 5, 0, 7])
    lens = lens.astype(np.int64)
    W_ = lens.size
    off = np.zeros(W_ + 1, np.int64)
    off[1:] = np.cumsum(lens)
    S = int(off[-1])
    lat = rng.uniform(0.0, 30.0, S).astype(np.float32)
    cur = None
    if case == "cursors_inf":
        for j in (off[0] + 5000 - 1024, off[0] + 5000 - 1025, off[1] + 7, off[2] + 1535):
            lat[j] = np.inf         # at chunk edges and inside
        cur = rng.integers(0, 6000, W_).astype(np.int32)
        cur[:3] = [1000, 4097, 0]   # inside, exactly at the end, at the start
    dl = rng.integers(0, 10 ** 12, W_).astype(np.int64)
    got = gpu_prioritize(off, lat, dl, 600 * 10 ** 6, cursor=cur)
    assert_prio_equal(got, oracle.prioritize(off, lat, dl, 600 * 10 ** 6, cursor=cur))


def test_prioritize_long_chain_flag_with_a_reused_workspace():
    # whether a call has chains of more than 1,024 stages is told to the long-chain kernel through a
    # word of the workspace holding the call's number; one workspace serves calls with and without
    # long chains in turn (a stale word from an earlier call must neither skip a long chain nor
    # disturb a call without any), then the same through the static scratch of the allocation-free
    # entry point, and a workspace filled with ones (any stale word) serves one of each
    rng = np.random.default_rng(17)
    t = lambda a: pipeline._t(a, "cuda")

    def batch(long):
        lens = rng.integers(0, 9, 3000)
        if long:
            lens[[7, 1500, 2999]] = [1025, 4000, 2048]
        off = np.zeros(lens.size + 1, np.int64)
        off[1:] = np.cumsum(lens)
        lat = rng.uniform(0.0, 30.0, int(off[-1])).astype(np.float32)
        dl = rng.integers(0, 10 ** 12, lens.size).astype(np.int64)
        return off, lat, dl

    batches = [batch(x) for x in (True, False, True, True, False, False, True)]
    need = max(M.prioritize_workspace_bytes(b[0].size - 1, b[1].size) for b in batches)
    ws = torch.empty(need, dtype=torch.uint8, device="cuda")
    for noalloc in (False, True):
        for off, lat, dl in batches:
            got = M.prioritize(t(off), t(lat), t(dl), 600 * 10 ** 6, workspace=None if noalloc else ws,
                               noalloc=noalloc)
            torch.cuda.synchronize()
            assert_prio_equal(tuple(_np(x) for x in got), oracle.prioritize(off, lat, dl, 600 * 10 ** 6))
    ws.fill_(255)
    for off, lat, dl in batches[:2]:
        got = M.prioritize(t(off), t(lat), t(dl), 600 * 10 ** 6, workspace=ws)
        torch.cuda.synchronize()
        assert_prio_equal(tuple(_np(x) for x in got), oracle.prioritize(off, lat, dl, 600 * 10 ** 6))


def test_prioritize_long_chain_and_empty():
    # one chain spanning every stage, then an empty batch
    S = 100000
    off = np.array([0, S], np.int64)
    lat = np.random.default_rng(1).uniform(0, 1, S).astype(np.float32)
    got = gpu_prioritize(off, lat, np.array([10 ** 9], np.int64), 0)
    assert_prio_equal(got, oracle.prioritize(off, lat, np.array([10 ** 9], np.int64), 0))
    t = lambda a: pipeline._t(a, "cuda")
    rem, key, order = M.prioritize(t(np.zeros(1, np.int64)), t(np.zeros(0, np.float32)),
                                   t(np.zeros(0, np.int64)), 0)
    assert key.numel() == 0 and order.numel() == 0
