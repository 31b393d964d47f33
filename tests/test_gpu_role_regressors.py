"""Parity of the per-role length regressors (Sec. III-B: a regressor with weights of its own for a
role with training data, the shared model otherwise; one grouped GEMM over the stages bucketed by
role) between the HIP path (through the C-ABI) and the CPU oracle, on seeded inputs.

Both sides take the same first-phase inputs: the GPU two-phase predictor's calibrated tool
probability, lengths and KV bytes. Bars (element by element):
  stages with a regressor : |dL| <= 1e-2 max(L, 1) (the bfloat16 predictor's relative tolerance;
                            the tool term is an identical input on both sides, so only the
                            network's float32-vs-float64 accumulation and bfloat16 hidden
                            rounding differ), and KV bytes equal, bit for bit, to Eq. 3 on the
                            GPU's own length;
  other stages            : lengths and KV bytes bit-identical to the inputs.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2606_12950_amd as M
from paper_2606_12950_amd import pipeline
from paper_2606_12950_amd import workload as W

pytestmark = pytest.mark.gpu

TOL = 1e-2


def _t(a):
    return pipeline._t(np.ascontiguousarray(a), "cuda")


def _first_phase(w, tp, rows=None):
    """GPU two-phase predictor on the workload (p_tool, pred_len, kv_bytes as numpy)."""
    sel = slice(None) if rows is None else rows
    ws = [_t(a) for a in w.weights[:-1]] + [_t(tp.head_weight)]
    bs = [_t(a) for a in w.biases[:-1]] + [_t(tp.head_bias)]
    pt, pl, kv = M.predict_two_phase(_t(w.x[sel]), ws, bs, _t(tp.role_head), _t(tp.tool_coef), _t(tp.iso_x),
                                     _t(tp.iso_y), tp.max_len, _t(w.prompt_len[sel]), _t(w.model_id[sel]),
                                     _t(w.role[sel]), _t(tp.tool_avail[sel]), _t(w.kv_bytes_per_token))
    torch.cuda.synchronize()
    return pt, pl, kv


def gpu_roles(x, rr, P, m, role, pt, alpha, pl, kv, role_regressor=None, coef=None):
    rg = rr.role_group if role_regressor is None else role_regressor
    c = rr.tool_coef if coef is None else coef
    pl_t, kv_t = _t(pl), _t(kv)
    M.predict_role_lengths(_t(x), [_t(a) for a in rr.weights], [_t(a) for a in rr.biases], _t(rg), _t(c), rr.max_len,
                           _t(P), _t(m), _t(role), _t(pt), _t(alpha), pl_t, kv_t)
    torch.cuda.synchronize()
    return pl_t.cpu().numpy(), kv_t.cpu().numpy()


def check(w, rr, role, pt, pl_in, kv_in, got, ref, rows=None, role_regressor=None):
    sel = slice(None) if rows is None else rows
    rg = rr.role_group if role_regressor is None else role_regressor
    G = rr.tool_coef.size
    r = role[sel]
    g = np.full(r.shape, -1)
    ok = (r >= 0) & (r < rg.size)
    g[ok] = rg[r[ok]]
    own = (g >= 0) & (g < G)
    lg, kg = got[0][sel], got[1][sel]
    lo, ko = ref[0][sel], ref[1][sel]
    assert np.array_equal(lg[~own].view(np.uint32), pl_in[sel][~own].view(np.uint32))
    assert np.array_equal(kg[~own].view(np.uint64), kv_in[sel][~own].view(np.uint64))
    rel = np.abs(lg[own].astype(np.float64) - lo[own]) / np.maximum(lo[own].astype(np.float64), 1.0)
    assert rel.size == 0 or rel.max() <= TOL, f"max rel err {rel.max():.3e} at {np.flatnonzero(own)[rel.argmax()]}"
    alpha = w.kv_bytes_per_token[w.model_id[sel][own]].astype(np.float64)
    assert np.array_equal(kg[own], (w.prompt_len[sel][own].astype(np.float64) + lg[own].astype(np.float64)) * alpha)
    changed = (lg[own] != pl_in[sel][own]).mean() if own.any() else 1.0
    print(f"  roles: {own.sum()} of {own.size} stages on their own regressor, max rel dL "
          f"{(rel.max() if rel.size else 0):.2e}, {changed:.3f} changed", flush=True)
    return own


@pytest.mark.parametrize("name,n", [("c1", 1), ("c1", 7), ("c1", 129), ("c1", 1000), ("c1", None), ("c4", 1000),
                                    ("c4", 4097)])
def test_role_regressors_match_oracle(name, n):
    # mid (256-512-512-64) and wide (256-1024-1024-64) regressors; ragged tiles per regressor (256 rows
    # with the two row groups of the mid network, 128 with the one of the wide)
    w = W.workload(name) if n is None else W.workload(name, n_stages=n)
    tp, rr = W.two_phase_inputs(w), W.role_regressor_inputs(w)
    pt, pl, kv = _first_phase(w, tp)
    pt, pl, kv = pt.cpu().numpy(), pl.cpu().numpy(), kv.cpu().numpy()
    got = gpu_roles(w.x, rr, w.prompt_len, w.model_id, w.role, pt, w.kv_bytes_per_token, pl, kv)
    ref = oracle.predict_role_lengths(w.x, rr.weights, rr.biases, rr.role_group, rr.tool_coef, rr.max_len,
                                      w.prompt_len, w.model_id, w.role, pt, w.kv_bytes_per_token, w.spec.dtype,
                                      pl, kv)
    check(w, rr, w.role, pt, pl, kv, got, ref)


@pytest.mark.parametrize("name", ["c3", "c4"])
def test_role_regressors_full_size_sampled(name):
    # the full launch (every stage bucketed, every regressor's tiles), 20,000 sampled stages checked
    w = W.workload(name)
    tp, rr = W.two_phase_inputs(w), W.role_regressor_inputs(w)
    pt, pl, kv = _first_phase(w, tp)
    pt, pl, kv = pt.cpu().numpy(), pl.cpu().numpy(), kv.cpu().numpy()
    got = gpu_roles(w.x, rr, w.prompt_len, w.model_id, w.role, pt, w.kv_bytes_per_token, pl, kv)
    rows = np.sort(np.random.default_rng(55).choice(w.n, 20000, replace=False))
    rows = np.unique(np.concatenate([rows, [0, w.n - 1]]))
    ref_l, ref_k = oracle.predict_role_lengths(w.x[rows], rr.weights, rr.biases, rr.role_group, rr.tool_coef,
                                               rr.max_len, w.prompt_len[rows], w.model_id[rows], w.role[rows],
                                               pt[rows], w.kv_bytes_per_token, w.spec.dtype, pl[rows], kv[rows])
    full_l, full_k = np.array(pl), np.array(kv)
    full_l[rows], full_k[rows] = ref_l, ref_k
    own = check(w, rr, w.role, pt, pl, kv, got, (full_l, full_k), rows=rows)
    assert own.mean() > 0.5


def test_role_map_edge_cases():
    # all sixteen regressors, roles mapped out of range, negative and beyond the map, a regressor
    # no role uses, every stage of one role, and no stage with a regressor at all (no tiles)
    w = W.workload("c1", n_stages=3000)
    rng = np.random.default_rng(56)
    base = W.role_regressor_inputs(w)
    G = 16
    reg = W.RoleRegressorInputs(
        weights=[np.concatenate([a] * 6)[:G] for a in base.weights], biases=[np.concatenate([b] * 6)[:G] for b in base.biases],
        role_group=np.array([15, 3, -1, 99, 0, 7, 7], np.int32), tool_coef=rng.uniform(-2.5, 0.5, G).astype(np.float32),
        max_len=500.0)
    tp = W.two_phase_inputs(w)
    pt, pl, kv = (a.cpu().numpy() for a in _first_phase(w, tp))
    roles = [rng.integers(-3, 10, w.n).astype(np.int32), np.full(w.n, 5, np.int32), np.full(w.n, 2, np.int32)]
    for role in roles:
        got = gpu_roles(w.x, reg, w.prompt_len, w.model_id, role, pt, w.kv_bytes_per_token, pl, kv)
        ref = oracle.predict_role_lengths(w.x, reg.weights, reg.biases, reg.role_group, reg.tool_coef, reg.max_len,
                                          w.prompt_len, w.model_id, role, pt, w.kv_bytes_per_token, w.spec.dtype,
                                          pl, kv)
        check(w, reg, role, pt, pl, kv, got, ref)
    assert (got[0] == pl).all()                      # role 2 has no regressor: nothing changes


@pytest.mark.parametrize("n", [255, 256, 257, 512])
def test_role_tiles_at_tile_boundaries(n):
    # every stage on one regressor (role 0's), so its rows fill whole 256-row tiles of the mid
    # network's two row groups exactly (256, 512) or leave one padding row (255) or one row on a
    # tile of its own (257)
    w = W.workload("c1", n_stages=n)
    rr = W.role_regressor_inputs(w)
    assert rr.role_group[0] >= 0
    tp = W.two_phase_inputs(w)
    pt, pl, kv = (a.cpu().numpy() for a in _first_phase(w, tp))
    role = np.zeros(n, np.int32)
    got = gpu_roles(w.x, rr, w.prompt_len, w.model_id, role, pt, w.kv_bytes_per_token, pl, kv)
    ref = oracle.predict_role_lengths(w.x, rr.weights, rr.biases, rr.role_group, rr.tool_coef, rr.max_len,
                                      w.prompt_len, w.model_id, role, pt, w.kv_bytes_per_token, w.spec.dtype,
                                      pl, kv)
    own = check(w, rr, role, pt, pl, kv, got, ref)
    assert own.all()


def test_two_phase_with_role_regressors_end_to_end():
    # oracle two-phase -> oracle regressors against GPU two-phase -> GPU regressors: the lengths
    # of stages with a regressor within the bar (p_tool now also differs within its own bar)
    w = W.workload("c1", n_stages=5000)
    tp, rr = W.two_phase_inputs(w), W.role_regressor_inputs(w)
    pt, pl, kv = (a.cpu().numpy() for a in _first_phase(w, tp))
    got = gpu_roles(w.x, rr, w.prompt_len, w.model_id, w.role, pt, w.kv_bytes_per_token, pl, kv)
    pto, plo, kvo = oracle.predict_two_phase(w.x, w.weights[:-1] + [tp.head_weight], w.biases[:-1] + [tp.head_bias],
                                             tp.role_head, tp.tool_coef, tp.iso_x, tp.iso_y, tp.max_len, w.prompt_len,
                                             w.model_id, w.role, tp.tool_avail, w.kv_bytes_per_token, w.spec.dtype)
    ref_l, _ = oracle.predict_role_lengths(w.x, rr.weights, rr.biases, rr.role_group, rr.tool_coef, rr.max_len,
                                           w.prompt_len, w.model_id, w.role, pto, w.kv_bytes_per_token, w.spec.dtype,
                                           plo, kvo)
    own = w.role < 3
    rel = np.abs(got[0][own].astype(np.float64) - ref_l[own]) / np.maximum(ref_l[own].astype(np.float64), 1.0)
    assert rel.max() <= 2 * TOL
    assert np.quantile(rel, 0.99) <= 2e-3


def test_role_regressors_reject_bad_args():
    w = W.workload("c1", n_stages=10)
    rr = W.role_regressor_inputs(w)
    pt = np.zeros(w.n, np.float32)
    pl, kv = np.ones(w.n, np.float32), np.ones(w.n)
    with pytest.raises(M.MaestroError, match="invalid"):
        gpu_roles(w.x, rr, w.prompt_len, w.model_id, w.role, pt, w.kv_bytes_per_token, pl, kv,
                  coef=np.zeros(3, np.float32), role_regressor=np.zeros(65, np.int32))
