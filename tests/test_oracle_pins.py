"""Pins of the CPU oracle against facts fixed by the paper and by mathematics (no GPU).

Each test states what it pins. None of them re-types the oracle's own code: they use closed
forms, independent library routines (PyTorch float64 layers, numpy lexsort / stable argsort),
invariants, degenerate cases and brute force on tiny inputs. The inputs are chosen so that a
plausible slip in the oracle (a dropped bias, a transposed weight, a wrong model index, a
wrong sign in the slack, an off-by-one in the suffix sum, an unstable sort, a wrong
tie-break) fails at least one of them.
"""
import math

import numpy as np
import pytest
import torch

import oracle
from paper_2606_12950_amd import workload as W

INT32_MIN, INT32_MAX = -(2 ** 31), 2 ** 31 - 1
INT64_MAX = 2 ** 63 - 1


def _centres(B):
    return (32.0 + 64.0 * np.arange(B)).astype(np.float32)


def _zero_predictor(dims, dtype):
    store = np.float32 if dtype == "f32" else np.uint16
    ws = [np.zeros((dims[i + 1], dims[i]), store) for i in range(len(dims) - 1)]
    bs = [np.zeros(dims[i + 1], np.float32) for i in range(len(dims) - 1)]
    return ws, bs


# ----------------------------------------------------------------------------------------------
# predict (Sec. III-B stand-in predictor, Eq. 3)
# ----------------------------------------------------------------------------------------------

@pytest.mark.parametrize("dims,dtype,expect", [((64, 128, 32), "f32", 1024.0),
                                               ((256, 512, 512, 64), "bf16", 2048.0)])
def test_zero_weights_give_mean_bin_centre(dims, dtype, expect):
    # All logits equal -> uniform softmax -> expected length = mean of the centres
    # 32 + 64 b, i.e. 32 + 64 (B - 1) / 2: exactly 1024 (B = 32) and 2048 (B = 64).
    rng = np.random.default_rng(0)
    n = 37
    x = rng.standard_normal((n, dims[0])).astype(np.float32)
    if dtype == "bf16":
        x = W.f32_to_bf16_bits(x)
    ws, bs = _zero_predictor(dims, dtype)
    P = rng.integers(16, 8192, n).astype(np.int32)
    m = rng.integers(0, 3, n).astype(np.int32)
    alpha = np.array([65536, 131072, 327680], np.float32)
    pred, kv = oracle.predict(x, ws, bs, _centres(dims[-1]), P, m, alpha, dtype)
    assert np.all(pred == np.float32(expect))
    # Eq. 3 with distinct per-model alpha: a wrong model index changes kv
    assert np.array_equal(kv, (P.astype(np.float64) + expect) * alpha[m].astype(np.float64))


@pytest.mark.parametrize("j", [0, 5, 31])
def test_one_hot_bias_selects_its_bin(j):
    # A +100 logit on bin j puts all but e^-100 of the mass there: expected length = c_j.
    dims = (64, 128, 32)
    ws, bs = _zero_predictor(dims, "f32")
    bs[-1][j] = 100.0
    x = np.random.default_rng(1).standard_normal((5, 64)).astype(np.float32)
    c = _centres(32)
    pred, _ = oracle.predict(x, ws, bs, c, np.full(5, 100, np.int32), np.zeros(5, np.int32),
                             np.ones(1, np.float32), "f32")
    assert np.all(pred == c[j])


def _random_predictor(rng, dims, dtype, scale=3.0, bias_scale=0.5):
    ws, bs = [], []
    for i in range(len(dims) - 1):
        w = (rng.standard_normal((dims[i + 1], dims[i])) * scale / math.sqrt(dims[i])).astype(np.float32)
        ws.append(w if dtype == "f32" else W.f32_to_bf16_bits(w))
        bs.append((rng.standard_normal(dims[i + 1]) * bias_scale).astype(np.float32))
    return ws, bs


def test_expected_length_is_a_convex_combination():
    rng = np.random.default_rng(2)
    dims = (64, 128, 32)
    ws, bs = _random_predictor(rng, dims, "f32", scale=8.0)
    x = rng.standard_normal((200, 64)).astype(np.float32)
    c = _centres(32)
    pred, _ = oracle.predict(x, ws, bs, c, np.full(200, 16, np.int32), np.zeros(200, np.int32),
                             np.ones(1, np.float32), "f32")
    assert np.all(pred >= c[0]) and np.all(pred <= c[-1])
    assert pred.std() > 50.0  # the large weights really move the prediction


def test_shifting_every_centre_shifts_the_prediction():
    # sum_b p_b (c_b + d) = sum_b p_b c_b + d, since the p_b sum to one.
    rng = np.random.default_rng(3)
    dims = (64, 128, 32)
    ws, bs = _random_predictor(rng, dims, "f32")
    x = rng.standard_normal((100, 64)).astype(np.float32)
    c = _centres(32)
    args = (np.full(100, 16, np.int32), np.zeros(100, np.int32), np.ones(1, np.float32), "f32")
    p0, _ = oracle.predict(x, ws, bs, c, *args)
    p1, _ = oracle.predict(x, ws, bs, (c + 1000.0).astype(np.float32), *args)
    diff = p1.astype(np.float64) - p0.astype(np.float64) - 1000.0
    assert np.all(np.abs(diff) <= 2 * np.spacing(p1.astype(np.float32)).astype(np.float64))


def _torch_forward(x, ws, bs, c, dtype):
    """Float64 PyTorch forward pass with the hidden layers rounded to the storage type."""
    as_t = (lambda a: torch.from_numpy(a.astype(np.float64))) if dtype == "f32" else \
        (lambda a: torch.from_numpy(W.bf16_bits_to_f32(a).astype(np.float64)))
    h = as_t(x)
    L = len(ws)
    for i in range(L):
        z = torch.nn.functional.linear(h, as_t(ws[i]), torch.from_numpy(bs[i].astype(np.float64)))
        if i + 1 < L:
            h = torch.relu(z)
            h = h.float().double() if dtype == "f32" else h.float().bfloat16().double()
    p = torch.softmax(z, dim=-1)
    return (p * torch.from_numpy(c.astype(np.float64))).sum(-1).float().numpy()


@pytest.mark.parametrize("dims,dtype", [((64, 128, 32), "f32"), ((48, 80, 40, 16), "bf16"),
                                        ((32, 24, 56, 40, 8), "f32")])
def test_predict_matches_pytorch_float64(dims, dtype):
    # Non-square layers catch a transposed weight, random biases catch a dropped bias.
    rng = np.random.default_rng(4)
    ws, bs = _random_predictor(rng, dims, dtype, scale=4.0)
    n = 300
    x = rng.standard_normal((n, dims[0])).astype(np.float32)
    if dtype == "bf16":
        x = W.f32_to_bf16_bits(x)
    c = _centres(dims[-1])
    P = rng.integers(16, 8192, n).astype(np.int32)
    m = rng.integers(0, 4, n).astype(np.int32)
    alpha = np.array([65536, 131072, 327680, 98304], np.float32)
    pred, kv = oracle.predict(x, ws, bs, c, P, m, alpha, dtype)
    ref = _torch_forward(x, ws, bs, c, dtype)
    # float32 hidden layers: identical rounding points, agreement to float32 rounding.
    # bf16: torch rounds float64 -> float32 -> bf16 (two roundings) where the oracle rounds
    # once, which can move a rare hidden unit by one bf16 step.
    tol = 4e-7 if dtype == "f32" else 2e-4
    assert np.all(np.abs(pred - ref) <= tol * np.abs(ref))
    assert np.array_equal(kv, (P.astype(np.float64) + pred.astype(np.float64)) * alpha[m].astype(np.float64))


def test_round_bf16_matches_torch_on_float32_values():
    rng = np.random.default_rng(5)
    v = np.concatenate([rng.standard_normal(20000).astype(np.float32) * 10.0 ** rng.integers(-30, 30, 20000),
                        np.array([1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, -(1.0 + 2 ** -8), 2 ** -130,
                                  3 * 2 ** -134, 0.0], np.float32)]).astype(np.float32)
    ref = torch.from_numpy(v).bfloat16().float().numpy()
    got = np.array([oracle.round_bf16(float(a)) for a in v], np.float64)
    assert np.array_equal(got.astype(np.float32), ref)
    # ties to even: 1 + 2^-8 sits halfway between 1 and 1 + 2^-7
    assert oracle.round_bf16(1.0 + 2 ** -8) == 1.0
    assert oracle.round_bf16(1.0 + 3 * 2 ** -8) == 1.0 + 2 ** -6


def test_predict_workload_distribution_sanity():
    # c0-shaped draw: N(0, 1/fan_in) weights keep the logits small, so predictions stay near
    # the middle of the bin range and well inside [c_0, c_31].
    wl = W.workload("c0", n_stages=512)
    pred, kv = oracle.predict_workload(wl)
    assert 700.0 < pred.mean() < 1300.0
    assert np.all((pred > 32.0) & (pred < 2016.0))
    assert np.all(kv == (wl.prompt_len + pred.astype(np.float64)) * 131072.0)


# ----------------------------------------------------------------------------------------------
# route (Alg. 3, Eq. 6, Eq. 2 decode term)
# ----------------------------------------------------------------------------------------------

def _route_bruteforce(model, pred, kv, dec, free, q, cold, mask, k, rho):
    """All pairs, feasibility filter, lexicographic (score, index) sort via numpy.lexsort."""
    n, M = model.shape[0], free.shape[0]
    need = kv if rho == 0.0 else kv * (1.0 + rho)
    ks = (pred * dec[model]).astype(np.float32)                                  # float32 product
    res = ((mask[None, :] >> model[:, None].astype(np.uint64)) & np.uint64(1)).astype(bool)
    act = np.where(res, np.float32(0.0), cold[None, :]).astype(np.float32)
    ready = (q[None, :] + act).astype(np.float32)
    s = (ready + ks[:, None]).astype(np.float32)
    feas = need[:, None] <= free[None, :]
    idx = np.full((n, k), -1, np.int32)
    sc = np.full((n, k), np.inf, np.float32)
    for i in range(n):
        cand = np.nonzero(feas[i])[0]
        o = cand[np.lexsort((cand, s[i, cand]))][:k]
        idx[i, :len(o)] = o
        sc[i, :len(o)] = s[i, o]
    return idx, sc


def _tiny_route_case(rng, coarse):
    n, M, K = int(rng.integers(1, 48)), int(rng.integers(1, 17)), int(rng.integers(1, 9))
    model = rng.integers(0, K, n).astype(np.int32)
    if coarse:  # coarse grids make exact score ties and free == need boundaries common
        pred = rng.choice(np.array([64.0, 128.0, 256.0], np.float32), n)
        dec = rng.choice(np.array([0.015625, 0.03125], np.float32), K)
        q = rng.choice(np.array([0.0, 0.5, 1.0], np.float32), M)
        cold = rng.choice(np.array([2.0, 4.0], np.float32), M)
        kv = rng.choice(np.array([1e9, 2e9, 3e9]), n)
        free = rng.choice(np.array([0.5e9, 1e9, 2e9, 3e9]), M)
    else:
        pred = rng.uniform(32, 4064, n).astype(np.float32)
        dec = rng.uniform(0.01, 0.04, K).astype(np.float32)
        q = rng.uniform(0, 5, M).astype(np.float32)
        cold = rng.uniform(2, 20, M).astype(np.float32)
        kv = rng.uniform(0, 4e9, n)
        free = rng.uniform(0, 4e9, M)
    mask = rng.integers(0, 2 ** 63, M, dtype=np.int64).astype(np.uint64) ^ \
        (rng.integers(0, 2, M).astype(np.uint64) << np.uint64(63))
    k = int(rng.choice([1, 2, 4, 7]))
    rho = float(rng.choice([0.0, 0.0, 0.2]))
    return model, pred, kv, dec, free, q, cold, mask, k, rho


@pytest.mark.parametrize("coarse", [False, True])
def test_route_matches_bruteforce_on_tiny_inputs(coarse):
    rng = np.random.default_rng(10 + coarse)
    for _ in range(150):
        model, pred, kv, dec, free, q, cold, mask, k, rho = _tiny_route_case(rng, coarse)
        got = oracle.route(model, pred, kv, dec, free, q, cold, mask, k=k, rho=rho, n_threads=2)
        exp = _route_bruteforce(model, pred, kv, dec, free, q, cold, mask, k, rho)
        assert np.array_equal(got[0], exp[0])
        assert np.array_equal(got[1], exp[1])


def test_route_invariants_at_moderate_size():
    wl = W.workload("c1", n_stages=3000, n_nodes=300, with_x=False, k=4)
    rng = np.random.default_rng(12)
    pred = rng.uniform(500, 3500, wl.n).astype(np.float32)
    kv = (wl.prompt_len + pred.astype(np.float64)) * wl.kv_bytes_per_token[wl.model_id].astype(np.float64)
    # squeeze the free memory so that feasibility binds for a good share of pairs
    free = wl.free_bytes / 100.0
    idx, sc = oracle.route(wl.model_id, pred, kv, wl.decode_s_per_token, free, wl.queue_s,
                           wl.cold_s, wl.resident_mask, k=4)
    dec = wl.decode_s_per_token[wl.model_id]
    ks = (pred * dec).astype(np.float32)
    res = ((wl.resident_mask[None, :] >> wl.model_id[:, None].astype(np.uint64)) & np.uint64(1)).astype(bool)
    s_all = ((wl.queue_s[None, :] + np.where(res, np.float32(0), wl.cold_s[None, :])).astype(np.float32)
             + ks[:, None]).astype(np.float32)
    feas = kv[:, None] <= free[None, :]
    n_feas = feas.sum(1)
    assert 0 < (n_feas < 4).sum() < wl.n  # both regimes occur
    for i in range(wl.n):
        got = [(float(s), int(j)) for s, j in zip(sc[i], idx[i]) if j >= 0]
        assert len(got) == min(4, n_feas[i])                       # -1 only when too few feasible
        assert all(feas[i, j] for _, j in got)                      # chosen nodes are feasible
        assert all(s == s_all[i, j] for s, j in got)                # score is the node's score
        assert got == sorted(got)                                   # lexicographic order
        if got:
            worst = got[-1]
            chosen = {j for _, j in got}
            better = [(float(s_all[i, j]), j) for j in np.nonzero(feas[i])[0]
                      if j not in chosen and (float(s_all[i, j]), int(j)) < worst]
            assert not better                                        # nothing better left out
        assert np.all(idx[i, len(got):] == -1) and np.all(np.isinf(sc[i, len(got):]))


def test_route_degenerate_cases():
    one = np.ones(1)
    # every node infeasible -> -1 / +inf everywhere
    idx, sc = oracle.route(np.zeros(3, np.int32), np.full(3, 100, np.float32), np.full(3, 5e9),
                           np.full(1, 0.02, np.float32), np.full(4, 1e9), np.zeros(4, np.float32),
                           np.ones(4, np.float32), np.zeros(4, np.uint64), k=2)
    assert np.all(idx == -1) and np.all(np.isinf(sc))
    # free == need is feasible (the filter drops a node only when demand exceeds headroom)
    idx, sc = oracle.route(np.zeros(1, np.int32), np.full(1, 100, np.float32), 2e9 * one,
                           np.full(1, 0.02, np.float32), np.array([2e9]), np.zeros(1, np.float32),
                           np.ones(1, np.float32), np.zeros(1, np.uint64))
    assert idx[0, 0] == 0
    # equal scores everywhere -> the lowest feasible index wins (Alg. 3 keeps the first max)
    idx, _ = oracle.route(np.zeros(1, np.int32), np.full(1, 100, np.float32), 1e9 * one,
                          np.full(1, 0.02, np.float32), np.array([0.0, 5e9, 5e9, 5e9]),
                          np.full(4, 1.0, np.float32), np.full(4, 3.0, np.float32),
                          np.zeros(4, np.uint64), k=3)
    assert list(idx[0]) == [1, 2, 3]
    # residency removes the cold-start term for exactly that model's bit
    mask = np.array([0, 1 << 5, 0], np.uint64)
    idx, sc = oracle.route(np.array([5, 4], np.int32), np.full(2, 50, np.float32), np.zeros(2),
                           np.full(8, 0.02, np.float32), np.full(3, 1e9),
                           np.array([1.0, 2.0, 1.5], np.float32), np.full(3, 10.0, np.float32), mask)
    assert list(idx[:, 0]) == [1, 0]
    assert sc[0, 0] == np.float32(np.float32(2.0) + np.float32(np.float32(50) * np.float32(0.02)))
    assert sc[1, 0] == np.float32(np.float32(11.0) + np.float32(np.float32(50) * np.float32(0.02)))
    # bit 63 of the mask belongs to model 63
    idx, _ = oracle.route(np.array([63], np.int32), np.full(1, 50, np.float32), np.zeros(1),
                          np.full(64, 0.02, np.float32), np.full(2, 1e9), np.array([0.0, 1.0], np.float32),
                          np.full(2, 10.0, np.float32), np.array([0, 1 << 63], np.uint64))
    assert idx[0, 0] == 1
    # a safety margin rho > 0 can make a node infeasible: need = (1 + rho) kv
    idx, _ = oracle.route(np.zeros(1, np.int32), np.full(1, 1, np.float32), 1e9 * one,
                          np.full(1, 0.02, np.float32), np.array([1.1e9, 1.3e9]),
                          np.zeros(2, np.float32), np.array([1.0, 2.0], np.float32),
                          np.zeros(2, np.uint64), rho=0.2)
    assert idx[0, 0] == 1


def test_route_node_permutation_equivariance():
    wl = W.workload("c0", n_stages=800, with_x=False, k=3)
    rng = np.random.default_rng(13)
    pred = rng.uniform(500, 1500, wl.n).astype(np.float32)
    kv = (wl.prompt_len + pred.astype(np.float64)) * 131072.0
    args = lambda perm: (wl.model_id, pred, kv, wl.decode_s_per_token, wl.free_bytes[perm],
                         wl.queue_s[perm], wl.cold_s[perm], wl.resident_mask[perm])
    ident = np.arange(wl.spec.n_nodes)
    perm = rng.permutation(wl.spec.n_nodes)
    i0, s0 = oracle.route(*args(ident), k=3)
    i1, s1 = oracle.route(*args(perm), k=3)
    assert np.array_equal(s0, s1)                 # the k smallest scores do not depend on order
    mapped = np.where(i1 >= 0, perm[np.maximum(i1, 0)], -1)
    distinct = np.all(np.diff(s0, axis=1) > 0, axis=1)
    assert np.array_equal(mapped[distinct], i0[distinct])


# ----------------------------------------------------------------------------------------------
# prioritize (Eq. 7, slack, stable order)
# ----------------------------------------------------------------------------------------------

def _chains(rng, W_, lo=0, hi=8):
    lens = rng.integers(lo, hi + 1, W_)
    off = np.zeros(W_ + 1, np.int64)
    off[1:] = np.cumsum(lens)
    return off, lens


def test_unit_latencies_give_closed_form_remaining_time():
    rng = np.random.default_rng(20)
    off, lens = _chains(rng, 500, 1, 9)
    S = int(off[-1])
    dl = rng.integers(0, 10 ** 9, 500).astype(np.int64)
    rem, key, order = oracle.prioritize(off, np.ones(S, np.float32), dl, 5 * 10 ** 8)
    for w in range(500):
        for j in range(off[w], off[w + 1]):
            assert rem[j] == (off[w + 1] - j) * 10 ** 6
        assert key[w] == dl[w] - 5 * 10 ** 8 - lens[w] * 10 ** 6


def test_remaining_time_and_keys_match_bruteforce():
    rng = np.random.default_rng(21)
    off, lens = _chains(rng, 400, 0, 12)
    S = int(off[-1])
    lat = rng.uniform(-1.0, 200.0, S).astype(np.float32)
    dl = rng.integers(-(2 ** 40), 2 ** 40, 400).astype(np.int64)
    cur = rng.integers(-2, 14, 400).astype(np.int32)
    now = int(rng.integers(0, 2 ** 35))
    rem, key, order = oracle.prioritize(off, lat, dl, now, cursor=cur)
    lat_us = np.rint(lat.astype(np.float64) * 1e6).astype(np.int64)   # numpy rint: half to even
    for w in range(400):
        a, b = int(off[w]), int(off[w + 1])
        for j in range(a, b):
            assert rem[j] == sum(int(lat_us[i]) for i in range(j, b))  # O(len^2) brute force
        c = max(int(cur[w]), 0)
        r = sum(int(lat_us[i]) for i in range(a + c, b)) if a + c < b else 0
        assert key[w] == min(max(int(dl[w]) - now - r, INT32_MIN), INT32_MAX)
    assert np.array_equal(order, np.argsort(key, kind="stable"))


def test_order_is_a_stable_sort():
    rng = np.random.default_rng(22)
    Wn = 3000
    off = np.arange(Wn + 1, dtype=np.int64)
    lat = np.zeros(Wn, np.float32)
    # few distinct deadlines -> many equal keys
    dl = rng.choice(np.array([5, 7, 11], np.int64) * 10 ** 6, Wn)
    _, key, order = oracle.prioritize(off, lat, dl, 0)
    assert np.array_equal(np.sort(order), np.arange(Wn))               # a permutation
    assert np.all(np.diff(key[order]) >= 0)                            # ascending keys
    eq = np.diff(key[order]) == 0
    assert np.all(np.diff(order)[eq] > 0)                              # ties keep index order
    assert np.array_equal(order, np.argsort(key, kind="stable"))
    # all keys equal -> identity permutation
    _, _, order = oracle.prioritize(off, lat, np.full(Wn, 42, np.int64), 0)
    assert np.array_equal(order, np.arange(Wn))


def test_latency_quantisation_rounds_half_to_even():
    # 2^-7 s = 7812.5 us and 3 * 2^-7 s = 23437.5 us are exact halves in float64
    assert oracle.latency_us(2 ** -7) == 7812
    assert oracle.latency_us(3 * 2 ** -7) == 23438
    assert oracle.latency_us(-(2 ** -7)) == -7812
    assert oracle.latency_us(1.0) == 10 ** 6
    assert oracle.latency_us(float("inf")) == INT64_MAX
    assert oracle.latency_us(float("nan")) == INT64_MAX
    assert oracle.latency_us(3.0e30) == 2 ** 40                          # clamp of absurd values


def test_slack_clamps_to_int32_and_nonfinite_latency_is_most_urgent():
    off = np.array([0, 2, 4, 6, 6], np.int64)
    lat = np.array([1.0, 2.0, np.inf, 1.0, 1.0, np.nan], np.float32)
    dl = np.array([2 ** 40, 10 ** 8, -(2 ** 40), 7], np.int64)
    rem, key, order = oracle.prioritize(off, lat, dl, 0)
    assert key[0] == INT32_MAX                                           # far deadline clamps up
    assert key[2] == INT32_MIN                                           # far past clamps down
    # an infinite stage latency poisons its own and every earlier suffix of its chain
    assert rem[2] == INT64_MAX and rem[3] == 10 ** 6
    assert key[1] == INT32_MIN
    assert rem[4] == INT64_MAX and rem[5] == INT64_MAX                   # NaN acts like +inf
    assert key[3] == 7                                                   # empty chain: 0 left
    assert list(order) == [1, 2, 3, 0]                                   # ties by index
    # a cursor past the poisoned stage sees only the finite tail
    _, key, _ = oracle.prioritize(off, lat, dl, 0, cursor=np.array([0, 1, 0, 0], np.int32))
    assert key[1] == 10 ** 8 - 10 ** 6


def test_prioritize_empty_and_validation():
    rem, key, order = oracle.prioritize(np.zeros(1, np.int64), np.zeros(0, np.float32),
                                        np.zeros(0, np.int64), 0)
    assert key.size == 0 and order.size == 0
    with pytest.raises(RuntimeError):
        oracle.prioritize(np.array([0, 3, 2], np.int64), np.zeros(2, np.float32), np.zeros(2, np.int64), 0)


def test_generator_bf16_casts_agree():
    # the fast cast used for large feature matrices rounds exactly like the reference cast
    rng = np.random.default_rng(30)
    v = (rng.standard_normal(200000) * 10.0 ** rng.integers(-20, 20, 200000)).astype(np.float32)
    v[:4] = [1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, -(1.0 + 2 ** -8), 0.0]
    assert np.array_equal(W._bf16_bits_fast(v), W.f32_to_bf16_bits(v))


def test_generator_is_deterministic():
    a = W.workload("c3", n_workflows=500)
    b = W.workload("c3", n_workflows=500)
    assert a.sha256() == b.sha256()
    assert a.n == int(a.chain_offset[-1]) and 3 * 500 <= a.n <= 8 * 500
    assert np.all(np.diff(a.chain_offset) >= 3) and np.all(np.diff(a.chain_offset) <= 8)
    c = W.workload("c1", n_stages=100)
    assert c.x.dtype == np.uint16 and c.x.shape == (100, 256)
    assert set(np.unique(c.kv_bytes_per_token)) <= {65536.0, 131072.0, 327680.0}
