"""Pins of the oracle's per-role length regressors (Sec. III-B: a regressor of its own for a role
with training data, the shared global model otherwise; regression on log(1 + L) fed the
calibrated tool probability; Eq. 3) -- no GPU.

Closed forms with zero weights; roles without a regressor keep their inputs bit for bit; each
regressor's output 0 is tied to the already-pinned bins predictor (a two-bin softmax with
centres (0, 1) over logits (0, z) has expectation sigmoid(z), so the bins predictor run on
regressor g's own layers reveals its z), which pins the stacking of the regressors' weights and
the role -> regressor map; clamps at 0 and max_len; Eq. 3 exactly.
"""
import numpy as np
import pytest

import oracle
from paper_2606_12950_amd import workload as W

MAXLEN = 32768.0


def _stack(rng, G, dims, dtype, zero=False):
    """G networks of shape dims (last layer: B outputs), stacked [G][out][in]."""
    ws, bs = [], []
    for i in range(len(dims) - 1):
        w = rng.normal(0, dims[i] ** -0.5, (G, dims[i + 1], dims[i])).astype(np.float32)
        if zero:
            w[:] = 0
        ws.append(w if dtype == "f32" else W.f32_to_bf16_bits(w))
        bs.append(rng.normal(0, 0.3, (G, dims[i + 1])).astype(np.float32))
    return ws, bs


def _x(rng, n, D, dtype):
    x = rng.standard_normal((n, D)).astype(np.float32)
    return x if dtype == "f32" else W.f32_to_bf16_bits(x)


def _inputs(rng, n, n_roles):
    P = rng.integers(16, 4096, n).astype(np.int32)
    m = rng.integers(0, 3, n).astype(np.int32)
    role = rng.integers(-1, n_roles + 2, n).astype(np.int32)          # some roles out of range
    pt = np.where(rng.random(n) < 0.6, rng.random(n), 0.0).astype(np.float32)
    alpha = np.array([65536, 131072, 327680], np.float32)
    pred = rng.uniform(10, 3000, n).astype(np.float32)               # the shared model's lengths
    kv = (P + pred.astype(np.float64)) * alpha[m].astype(np.float64)
    return P, m, role, pt, alpha, pred, kv


def _group_of(role, role_group, G):
    g = np.full(role.shape, -1)
    ok = (role >= 0) & (role < role_group.size)
    g[ok] = role_group[role[ok]]
    g[(g < 0) | (g >= G)] = -1
    return g


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_zero_weights_give_closed_forms_and_other_roles_keep_their_inputs(dtype):
    rng = np.random.default_rng(31)
    G, dims, n = 3, (16, 32, 24, 8), 400
    ws, bs = _stack(rng, G, dims, dtype, zero=True)
    bs[-1][:, 0] = np.array([5.0, 3.5, -1.0], np.float32)             # regressor 2: y < 0 for most p
    coef = np.array([-1.5, 0.75, 0.5], np.float32)
    role_group = np.array([2, 0, -1, 1, 7], np.int32)                 # role 2 and 4: no regressor
    x = _x(rng, n, dims[0], dtype)
    P, m, role, pt, alpha, pred, kv = _inputs(rng, n, role_group.size)
    L, kv2 = oracle.predict_role_lengths(x, ws, bs, role_group, coef, MAXLEN, P, m, role, pt, alpha, dtype,
                                         pred, kv)
    g = _group_of(role, role_group, G)
    own = g >= 0
    assert own.any() and (~own).any()
    assert np.array_equal(L[~own], pred[~own]) and np.array_equal(kv2[~own].view(np.uint64), kv[~own].view(np.uint64))
    y = bs[-1][g[own], 0].astype(np.float64) + coef[g[own]].astype(np.float64) * pt[own].astype(np.float64)
    want = np.minimum(np.expm1(np.maximum(y, 0.0)), MAXLEN).astype(np.float32)
    assert np.array_equal(L[own], want)
    assert (L[own][g[own] == 2] < 1.0).all()                           # clamp at 0: expm1(0) = 0 below
    # Eq. 3 on the new length, exactly
    assert np.array_equal(kv2[own], (P[own] + L[own].astype(np.float64)) * alpha[m[own]].astype(np.float64))


def _regressor_z(x, ws, bs, g, dtype):
    """z_0 of regressor g through the bins predictor on g's own layers: bins (0, z_0), centres (0, 1)."""
    store = np.float32 if dtype == "f32" else np.uint16
    layers = [w[g] for w in ws]
    biases = [b[g] for b in bs]
    w_last = np.zeros((2, layers[-1].shape[1]), store)
    w_last[1] = layers[-1][0]
    b_last = np.array([0.0, biases[-1][0]], np.float32)
    n = x.shape[0]
    s, _ = oracle.predict(x, layers[:-1] + [w_last], biases[:-1] + [b_last], np.array([0.0, 1.0], np.float32),
                          np.zeros(n, np.int32), np.zeros(n, np.int32), np.ones(1, np.float32), dtype)
    s = s.astype(np.float64)
    return np.log(s / (1.0 - s))


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_each_role_uses_its_own_network(dtype):
    rng = np.random.default_rng(32)
    G, dims, n = 4, (16, 40, 24, 8), 300
    ws, bs = _stack(rng, G, dims, dtype)
    for g in range(G):                                                 # keep sigmoid(z_0) well inside (0, 1)
        bs[-1][g, 0] = 0.0
    coef = np.array([-1.0, -0.5, 0.25, 0.8], np.float32)
    role_group = np.array([3, 1, 0, 2], np.int32)                      # a permutation: offsets must match
    x = _x(rng, n, dims[0], dtype)
    P, m, role, pt, alpha, pred, kv = _inputs(rng, n, role_group.size)
    L, _ = oracle.predict_role_lengths(x, ws, bs, role_group, coef, MAXLEN, P, m, role, pt, alpha, dtype,
                                       pred, kv)
    g = _group_of(role, role_group, G)
    for gg in range(G):
        rows = np.flatnonzero(g == gg)
        z = _regressor_z(x[rows], ws, bs, gg, dtype)
        y = z + coef[gg] * pt[rows].astype(np.float64)
        want = np.expm1(np.maximum(y, 0.0))
        # the bins route returns sigmoid(z) rounded to float32: z back within ~1e-6 absolute
        assert np.allclose(L[rows], want, rtol=1e-5, atol=1e-5), gg
        # and another regressor's network would not do
        other = (gg + 1) % G
        z_o = _regressor_z(x[rows], ws, bs, other, dtype)
        assert not np.allclose(z, z_o, rtol=1e-3, atol=1e-3)


def test_clamp_at_max_len():
    rng = np.random.default_rng(33)
    G, dims, n = 1, (8, 16, 16, 8), 50
    ws, bs = _stack(rng, G, dims, "f32", zero=True)
    bs[-1][0, 0] = 12.0                                                # expm1(12) > 1000
    x = _x(rng, n, dims[0], "f32")
    P, m, _, pt, alpha, pred, kv = _inputs(rng, n, 1)
    role = np.zeros(n, np.int32)
    L, kv2 = oracle.predict_role_lengths(x, ws, bs, np.array([0], np.int32), np.zeros(1, np.float32), 1000.0,
                                         P, m, role, pt, alpha, "f32", pred, kv)
    assert (L == 1000.0).all()
    assert np.array_equal(kv2, (P + 1000.0) * alpha[m].astype(np.float64))
