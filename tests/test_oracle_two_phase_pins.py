"""Pins of the oracle's two-phase predictor (Sec. III-B: tool intent, Eq. 1, with isotonic
calibration; per-role log(1 + L) regressors fed the tool probability; Eq. 3) -- no GPU.

The heads are pinned by closed forms (zero weights), by numpy's own routines (interp, expm1, the
logistic function), by the role fallback and the clamps; the trunk that feeds them is tied to
the already-pinned bins predictor: a two-bin softmax with centres (0, 1) over logits (0, z)
has expectation sigmoid(z), so the bins predictor reveals any head's pre-activation z.
"""
import numpy as np
import pytest

import oracle
from paper_2606_12950_amd import workload as W

MAXLEN = 32768.0


def _sigmoid(z):
    return 1.0 / (1.0 + np.exp(-np.asarray(z, np.float64)))


def _net(rng, dims, dtype, B, zero_heads=False):
    """Random trunk (dims[0] -> ... -> dims[-1]) and a head layer of B outputs."""
    store = np.float32 if dtype == "f32" else np.uint16
    ws, bs = [], []
    full = list(dims) + [B]
    for i in range(len(full) - 1):
        w = rng.normal(0, full[i] ** -0.5, (full[i + 1], full[i])).astype(np.float32)
        if i == len(full) - 2 and zero_heads:
            w[:] = 0
        ws.append(w if dtype == "f32" else W.f32_to_bf16_bits(w))
        bs.append(rng.normal(0, 0.3, full[i + 1]).astype(np.float32))
    return ws, bs, store


def _x(rng, n, D, dtype):
    x = rng.standard_normal((n, D)).astype(np.float32)
    return x if dtype == "f32" else W.f32_to_bf16_bits(x)


def _run(x, ws, bs, role_head, coef, kx, ky, P, m, role, tools, alpha, dtype, max_len=MAXLEN):
    return oracle.predict_two_phase(x, ws, bs, role_head, coef, kx, ky, max_len, P, m, role, tools, alpha, dtype)


def _head_preactivation(x, ws, bs, row, dtype):
    """z_row of the head layer through the bins predictor: bins (0, z_row), centres (0, 1)."""
    store = np.float32 if dtype == "f32" else np.uint16
    w_last = np.zeros((2, ws[-1].shape[1]), store)
    w_last[1] = ws[-1][row]
    b_last = np.array([0.0, bs[-1][row]], np.float32)
    n = x.shape[0]
    s, _ = oracle.predict(x, ws[:-1] + [w_last], bs[:-1] + [b_last], np.array([0.0, 1.0], np.float32),
                          np.zeros(n, np.int32), np.zeros(n, np.int32), np.ones(1, np.float32), dtype)
    s = s.astype(np.float64)
    return s, np.log(s / (1.0 - s))


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_zero_head_weights_give_closed_forms(dtype):
    # with a zero head layer every z_g is its bias: p = interp(sigmoid(b_0)), L = expm1(b_g + c_g p)
    rng = np.random.default_rng(1)
    dims, B, n = (24, 40), 8, 300
    ws, bs, _ = _net(rng, dims, dtype, B, zero_heads=True)
    bs[-1][:] = np.array([0.7, 5.0, 4.0, 6.5, 3.0, 2.0, 1.0, 0.5], np.float32)
    kx = np.array([0.0, 0.3, 0.6, 1.0], np.float32)
    ky = np.array([0.1, 0.2, 0.9, 0.95], np.float32)
    coef = np.array([0.0, -1.5, -0.5, 0.25, -3.0, 0.0, 0.0, 0.0], np.float32)
    role_head = np.array([2, 3, 4, 1], np.int32)                 # role 3 uses the shared head
    x = _x(rng, n, dims[0], dtype)
    P = rng.integers(16, 4096, n).astype(np.int32)
    m = rng.integers(0, 3, n).astype(np.int32)
    role = rng.integers(0, 4, n).astype(np.int32)
    tools = (rng.random(n) < 0.5).astype(np.int32)
    alpha = np.array([65536, 131072, 327680], np.float32)
    pt, L, kv = _run(x, ws, bs, role_head, coef, kx, ky, P, m, role, tools, alpha, dtype)
    p = np.interp(_sigmoid(bs[-1][0]), kx.astype(np.float64), ky.astype(np.float64))
    want_p = np.where(tools != 0, p, 0.0)
    assert np.array_equal(pt, want_p.astype(np.float32))
    assert np.all(pt[tools == 0] == 0.0)                          # no tools -> exactly 0
    g = role_head[role]
    y = bs[-1][g].astype(np.float64) + coef[g].astype(np.float64) * want_p
    want_L = np.minimum(np.expm1(np.maximum(y, 0.0)), MAXLEN).astype(np.float32)
    np.testing.assert_allclose(L, want_L, rtol=2e-7, atol=0)
    # Eq. 3 on the float32 length, per-model alpha
    assert np.array_equal(kv, (P.astype(np.float64) + L.astype(np.float64)) * alpha[m].astype(np.float64))


def test_tool_probability_is_the_calibrated_sigmoid_of_the_trunk_logit():
    # identity table: p = sigmoid(z_0); a monotone table: numpy's interp of it
    rng = np.random.default_rng(2)
    dims, B, n = (32, 48, 24), 6, 400
    ws, bs, _ = _net(rng, dims, "f32", B)
    x = _x(rng, n, dims[0], "f32")
    s0, _ = _head_preactivation(x, ws, bs, 0, "f32")
    args = dict(role_head=np.array([1], np.int32), coef=np.zeros(B, np.float32),
                P=np.zeros(n, np.int32), m=np.zeros(n, np.int32), role=np.zeros(n, np.int32),
                tools=np.ones(n, np.int32), alpha=np.ones(1, np.float32), dtype="f32")
    ident = np.array([0.0, 1.0], np.float32)
    pt, _, _ = _run(x, ws, bs, kx=ident, ky=ident, **args)
    np.testing.assert_allclose(pt, s0, rtol=1e-6, atol=1e-7)
    kx = np.sort(rng.uniform(0.05, 0.95, 12)).astype(np.float32)
    ky = np.sort(rng.uniform(0, 1, 12)).astype(np.float32)
    pt, _, _ = _run(x, ws, bs, kx=kx, ky=ky, **args)
    want = np.interp(s0, kx.astype(np.float64), ky.astype(np.float64))
    np.testing.assert_allclose(pt, want, rtol=1e-6, atol=1e-7)
    assert np.all(np.diff(pt[np.argsort(s0)]) >= 0)             # calibration keeps the order


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_length_is_the_roles_head_inverted(dtype):
    # L = expm1(z_g + c_g p) for the role's head g; roles without one, or out of range, use head 1
    rng = np.random.default_rng(3)
    dims, B, n = (16, 64, 32), 7, 500
    ws, bs, _ = _net(rng, dims, dtype, B)
    bs[-1][1:] += 5.0                                             # log(1 + L) around 5
    x = _x(rng, n, dims[0], dtype)
    role_head = np.array([3, 1, 6, 2, 99, 0], np.int32)           # 99 and 0 are not length heads
    role = rng.integers(-2, 8, n).astype(np.int32)
    tools = (rng.random(n) < 0.6).astype(np.int32)
    coef = rng.uniform(-2.5, 1.0, B).astype(np.float32)
    kx = np.array([0.0, 0.5, 1.0], np.float32)
    ky = np.array([0.0, 0.7, 1.0], np.float32)
    P = rng.integers(16, 4096, n).astype(np.int32)
    pt, L, _ = _run(x, ws, bs, role_head, coef, kx, ky, P, np.zeros(n, np.int32), role, tools,
                    np.ones(1, np.float32), dtype)
    g = np.ones(n, np.int64)
    ok = (role >= 0) & (role < role_head.size)
    g[ok] = role_head[role[ok]]
    g[(g < 1) | (g >= B)] = 1
    assert set(np.unique(g)) == {1, 2, 3, 6}
    z = np.stack([_head_preactivation(x, ws, bs, r, dtype)[1] for r in range(B)], axis=1)
    y = z[np.arange(n), g] + coef[g].astype(np.float64) * pt.astype(np.float64)
    want = np.minimum(np.expm1(np.maximum(y, 0.0)), MAXLEN)
    np.testing.assert_allclose(L, want, rtol=5e-5)


def test_length_clamps_and_tool_coefficient_direction():
    rng = np.random.default_rng(4)
    dims, B, n = (8, 16), 3, 64
    ws, bs, _ = _net(rng, dims, "f32", B, zero_heads=True)
    x = _x(rng, n, dims[0], "f32")
    kx = np.array([0.0, 1.0], np.float32)
    args = lambda b1, c1, max_len=MAXLEN: _run(x, ws, bs[:-1] + [np.array([2.0, b1, 0.0], np.float32)],
                                               np.zeros(0, np.int32), np.array([0, c1, 0], np.float32), kx, kx,
                                               np.zeros(n, np.int32), np.zeros(n, np.int32), np.zeros(n, np.int32),
                                               np.ones(n, np.int32), np.ones(1, np.float32), "f32", max_len)
    assert np.all(args(-3.0, 0.0)[1] == 0.0)                      # y < 0 -> L = 0
    assert np.all(args(40.0, 0.0)[1] == np.float32(MAXLEN))       # beyond max_len -> max_len
    assert np.all(args(7.0, 0.0, 100.0)[1] == np.float32(100.0))
    # a negative tool coefficient shortens the predicted output of tool-likely stages
    p = _sigmoid(2.0)
    assert np.allclose(args(6.0, -2.0)[1], np.expm1(6.0 - 2.0 * p), rtol=1e-6)
    assert np.all(args(6.0, -2.0)[1] < args(6.0, 0.0)[1])
