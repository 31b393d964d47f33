"""Pins of the end-to-end guard bands (tests/route_guard.py) on the oracle alone, no GPU: two
predictions that agree to the bfloat16 predictor tolerance route differently only through a
feasibility flip or a float32 rounding tie (Alg. 3 with Eq. 6: the prediction enters through the
demand R_kv and through the decode term, which is common to all nodes of a stage), and a route
changed any other way is caught."""
import numpy as np
import pytest

import oracle
from paper_2606_12950_amd import workload as W
from route_guard import explain_route_differences


def _perturbed(w, rows, rel, seed):
    pred_a, kv_a = oracle.predict_workload(w, rows=rows)
    f = 1.0 + np.random.default_rng(seed).uniform(-rel, rel, rows.size)
    pred_b = (pred_a.astype(np.float64) * f).astype(np.float32)
    alpha = w.kv_bytes_per_token[w.model_id[rows]].astype(np.float64)
    kv_b = (w.prompt_len[rows].astype(np.float64) + pred_b.astype(np.float64)) * alpha
    return pred_a, kv_a, pred_b, kv_b


@pytest.mark.parametrize("name,n,rel", [("c1", 4000, 1e-2), ("c2", 4000, 1e-2), ("c4", 600, 1e-2)])
def test_perturbed_predictions_route_alike(name, n, rel):
    w = W.workload(name, n_stages=n)
    rows = np.arange(w.n)
    pred_a, kv_a, pred_b, kv_b = _perturbed(w, rows, rel, 5)
    idx_a, _ = oracle.route_workload(w, pred_a, kv_a)
    idx_b, _ = oracle.route_workload(w, pred_b, kv_b)
    rate, _, _ = explain_route_differences(w, rows, pred_a, kv_a, idx_a, kv_b, idx_b)
    assert rate > 0.98


def test_a_feasibility_flip_is_explained():
    # put the chosen node's headroom of some stages between the two demands: prediction b no
    # longer fits there and routes elsewhere, which the guard attributes to the flip
    w = W.workload("c1", n_stages=3000)
    rows = np.arange(w.n)
    pred_a, kv_a, pred_b, kv_b = _perturbed(w, rows, 1e-2, 7)
    idx_a, _ = oracle.route_workload(w, pred_a, kv_a)
    grow = np.nonzero(kv_b > kv_a)[0][:5]
    for i in grow:
        w.free_bytes[idx_a[i, 0]] = 0.5 * (kv_a[i] + kv_b[i])
    idx_a, _ = oracle.route_workload(w, pred_a, kv_a)
    idx_b, _ = oracle.route_workload(w, pred_b, kv_b)
    assert np.any(idx_a[grow, 0] != idx_b[grow, 0])
    _, flips, _ = explain_route_differences(w, rows, pred_a, kv_a, idx_a, kv_b, idx_b)
    assert flips >= 1


class _Nodes:
    """Two nodes whose float32 scores tie under one decode term and not under the other."""
    def __init__(self):
        class S:
            rho = 0.0
        self.spec = S()
        self.model_id = np.zeros(1, np.int32)
        self.decode_s_per_token = np.ones(1, np.float32)
        self.resident_mask = np.ones(2, np.uint64)                 # resident: no cold penalty
        self.free_bytes = np.full(2, 1e12)
        self.queue_s = np.array([1.0 + 2.0 ** -23, 1.0], np.float32)   # one ulp apart at 1
        self.cold_s = np.zeros(2, np.float32)


def test_a_rounding_tie_is_explained():
    w = _Nodes()
    rows = np.arange(1)
    kv = np.array([1e9])
    # decode term 3: both scores round to 4 (ulp 2^-21), the lower index wins; decode term 2^-10:
    # the scores stay apart and node 1 is better
    pa, pb = np.array([3.0], np.float32), np.array([2.0 ** -10], np.float32)
    ia, _ = oracle.route(w.model_id, pa, kv, w.decode_s_per_token, w.free_bytes, w.queue_s, w.cold_s,
                         w.resident_mask)
    ib, _ = oracle.route(w.model_id, pb, kv, w.decode_s_per_token, w.free_bytes, w.queue_s, w.cold_s,
                         w.resident_mask)
    assert ia[0, 0] == 0 and ib[0, 0] == 1
    rate, flips, ties = explain_route_differences(w, rows, pa, kv, ia, kv, ib)
    assert (rate, flips, ties) == (0.0, 0, 1)


def test_a_planted_wrong_choice_is_caught():
    # replace one stage's best node by its feasible node of highest score: no flip, no tie
    w = W.workload("c1", n_stages=2000)
    rows = np.arange(w.n)
    pred_a, kv_a = oracle.predict_workload(w, rows=rows)
    idx_a, _ = oracle.route_workload(w, pred_a, kv_a)
    i = 123
    m = w.model_id[i]
    feas = np.nonzero(kv_a[i] <= w.free_bytes)[0]
    res = (w.resident_mask[feas] >> np.uint64(m)) & np.uint64(1)
    ks = np.float32(pred_a[i] * w.decode_s_per_token[m])
    sc = (np.float32(w.queue_s[feas] + np.where(res == 1, np.float32(0), w.cold_s[feas])) + ks).astype(np.float32)
    worst = int(feas[np.argmax(sc)])
    assert worst != idx_a[i, 0]
    idx_b = idx_a.copy()
    idx_b[i, 0] = worst
    with pytest.raises(AssertionError, match="not a rounding tie"):
        explain_route_differences(w, rows, pred_a, kv_a, idx_a, kv_a, idx_b)
