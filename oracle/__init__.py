"""CPU oracle of the predict -> route -> prioritize step (ctypes wrapper over liboracle.so).

TEST INFRASTRUCTURE ONLY: the test-suite, the smoke check and the benchmark's CPU-baseline
leg may use it; the product path (``paper_2606_12950_amd``) never imports it. It shares no
code with the HIP library. See ``maestro_oracle.c`` for what each function computes and
which passage of the paper it follows.

Parity status of each function (what pins it, see tests/test_oracle_pins.py):
  predict    - pinned: closed forms (zero weights -> mean of bin centres, one-hot bias ->
               that bin's centre), convexity, centre-shift equivariance, Eq. 3 exactly, and a
               float64 PyTorch forward pass with the same rounding points on small shapes.
  predict_two_phase - pinned (tests/test_oracle_two_phase_pins.py): zero weights give closed
               forms (sigmoid of the bias through the table, expm1 of the head's bias), no tools
               gives exactly 0, an identity table leaves the sigmoid unchanged, the table is
               numpy's interp, role fallback to the shared head, clamps at 0 and max_len, Eq. 3,
               and the trunk agrees with predict's on the same network.
  predict_role_lengths - pinned (tests/test_oracle_role_pins.py): zero-weight regressors give
               expm1 of the bias plus the tool term, in closed form; a regressor equal to a bins
               network recovers that network's output 0 through the pinned predict (two-bin
               softmax identity); roles without a regressor keep their inputs bit for bit; the
               stacking offset of each regressor's layers; clamps at 0 and max_len; Eq. 3.
  route      - pinned: brute force via numpy lexsort on tiny inputs, invariants (feasible,
               sorted, nothing better left out), degenerate cases, node-permutation
               equivariance.
  route_fitness - pinned (tests/test_oracle_fitness_pins.py): limiting weights reduce Eq. 5 to
               one metric whose argmax is a plain argmin (nearest node by RTT, best-fit packing,
               minimum time-to-start, minimum disruption), clipping at the window bounds and
               degenerate windows, infeasible padding, top-k order and tie-break, per-class
               weights, node-permutation equivariance.
  degradation_cost - pinned: brute force over priority prefixes (the shortest prefix of the
               level-sorted engines that frees R), closed forms (R <= 0, one engine, Failure), the
               interrupt penalty exactly when a level-4/5 engine is in the plan, stable order.
  activation_latency - pinned (tests/test_oracle_readiness_pins.py): Running is free, size 0
               leaves the setup, doubling a bandwidth halves the transfer exactly, tiers past
               Remote count as Remote; fitness routing with a matrix of {0, act} equals the
               resident-mask form.
  adaptive_rho - pinned (tests/test_oracle_readiness_pins.py): beta = 1 leaves e itself, exact
               predictions give 0, a constant error gives that constant, the recursion's closed
               form on geometric inputs, numpy's "higher" percentile of the EWMA values.
  quantiles  - pinned: numpy's percentile selection ("lower" / "higher" methods).
  prioritize - pinned: closed forms (unit latencies), numpy stable argsort, O(len^2) suffix
               sums, half-even rounding cases, int32 clamping, non-finite latency handling.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from typing import Optional, Sequence

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "maestro_oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")

_lib = None


def build(verbose: bool = False) -> str:
    """Compile liboracle.so with gcc (no fast-math, no FMA contraction)."""
    cmd = ["gcc", "-O2", "-std=gnu11", "-fPIC", "-shared", "-fopenmp", "-ffp-contract=off",
           "-fno-fast-math", "-Wall", "-o", _LIB + ".tmp", _SRC, "-lm"]
    if verbose:
        print(" ".join(cmd))
    subprocess.run(cmd, check=True)
    os.replace(_LIB + ".tmp", _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        build()
    lib = ctypes.CDLL(_LIB)
    P = ctypes.c_void_p
    i32, i64, f64 = ctypes.c_int32, ctypes.c_int64, ctypes.c_double
    lib.oracle_predict.argtypes = [i32, P, i32, P, P, P, i64, P, P, P, P, i32, P, P, i32]
    lib.oracle_predict.restype = ctypes.c_int
    lib.oracle_predict_two_phase.argtypes = [i32, P, i32, P, P, i32, P, P, i32, P, P, ctypes.c_float, i64, P,
                                             P, P, P, P, P, i32, P, P, P, i32]
    lib.oracle_predict_two_phase.restype = ctypes.c_int
    lib.oracle_predict_role_lengths.argtypes = [i32, P, i32, i32, P, P, i32, P, P, ctypes.c_float, i64, P, P, P,
                                                P, P, P, i32, P, P, i32]
    lib.oracle_predict_role_lengths.restype = ctypes.c_int
    lib.oracle_route.argtypes = [i64, P, P, P, P, i32, i32, P, P, P, P, P, f64, i32, P, P, i32]
    lib.oracle_route.restype = ctypes.c_int
    lib.oracle_route_fitness.argtypes = [i64, P, P, P, P, i32, i32, i32, i32, P, P, P, P, P, P, P, P, P,
                                         f64, i32, P, P, P, P, ctypes.c_float, P, P, i32]
    lib.oracle_activation_latency.argtypes = [i32, i32, P, P, P, P, f64, P]
    lib.oracle_adaptive_rho.argtypes = [P, P, i64, f64, f64, P, P]
    lib.oracle_adaptive_rho.restype = ctypes.c_int
    lib.oracle_activation_latency.restype = ctypes.c_int
    lib.oracle_degradation_cost.argtypes = [f64, i32, P, P, P, ctypes.c_float, P]
    lib.oracle_degradation_cost.restype = ctypes.c_int
    lib.oracle_route_fitness.restype = ctypes.c_int
    lib.oracle_quantiles.argtypes = [P, i64, f64, f64, P]
    lib.oracle_quantiles.restype = ctypes.c_int
    lib.oracle_prioritize.argtypes = [i32, i64, P, P, P, P, i64, P, P, P]
    lib.oracle_prioritize.restype = ctypes.c_int
    lib.oracle_round_bf16.argtypes = [f64]
    lib.oracle_round_bf16.restype = f64
    lib.oracle_latency_us.argtypes = [ctypes.c_float]
    lib.oracle_latency_us.restype = ctypes.c_int64
    lib.oracle_max_threads.restype = ctypes.c_int
    _lib = lib
    return lib


def _ptr(a: Optional[np.ndarray]):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _c(a, dtype) -> np.ndarray:
    return np.ascontiguousarray(a, dtype=dtype)


def max_threads() -> int:
    return int(_load().oracle_max_threads())


def round_bf16(v: float) -> float:
    return float(_load().oracle_round_bf16(float(v)))


def latency_us(lat_s: float) -> int:
    return int(_load().oracle_latency_us(float(lat_s)))


def predict(x: np.ndarray, weights: Sequence[np.ndarray], biases: Sequence[np.ndarray],
            bin_centre: np.ndarray, prompt_len: np.ndarray, model_id: np.ndarray,
            kv_bytes_per_token: np.ndarray, dtype: str, n_threads: int = 0):
    """Returns (pred_len float32 [N], kv_bytes float64 [N]).

    ``x``/``weights`` are float32 arrays (dtype "f32") or uint16 bf16 bit patterns ("bf16")."""
    lib = _load()
    dt = 0 if dtype == "f32" else 1
    store = np.float32 if dt == 0 else np.uint16
    x = _c(x, store)
    n = x.shape[0]
    ws = [_c(w, store) for w in weights]
    bs = [_c(b, np.float32) for b in biases]
    L = len(ws)
    dims = np.array([x.shape[1]] + [w.shape[0] for w in ws], dtype=np.int32)
    for l, w in enumerate(ws):
        assert w.shape == (dims[l + 1], dims[l]), "weight shapes must chain [out][in]"
    wptr = (ctypes.c_void_p * L)(*[w.ctypes.data for w in ws])
    bptr = (ctypes.c_void_p * L)(*[b.ctypes.data for b in bs])
    bc = _c(bin_centre, np.float32)
    pl, mi = _c(prompt_len, np.int32), _c(model_id, np.int32)
    alpha = _c(kv_bytes_per_token, np.float32)
    pred = np.empty(n, np.float32)
    kv = np.empty(n, np.float64)
    st = lib.oracle_predict(L, _ptr(dims), dt, ctypes.cast(wptr, ctypes.c_void_p),
                            ctypes.cast(bptr, ctypes.c_void_p), _ptr(bc), n, _ptr(x), _ptr(pl),
                            _ptr(mi), _ptr(alpha), alpha.shape[0], _ptr(pred), _ptr(kv),
                            n_threads or max_threads())
    if st != 0:
        raise RuntimeError(f"oracle_predict failed with status {st}")
    return pred, kv


def predict_two_phase(x: np.ndarray, weights: Sequence[np.ndarray], biases: Sequence[np.ndarray],
                      role_head, tool_coef, iso_x, iso_y, max_len: float, prompt_len, model_id, role_id,
                      tool_avail, kv_bytes_per_token, dtype: str, n_threads: int = 0):
    """Two-phase predictor: returns (p_tool float32 [N], pred_len float32 [N], kv_bytes float64
    [N]). The last layer's outputs are the heads: 0 the tool-intent logit, g >= 1 the log(1 + L)
    regressors (1 the shared one); ``role_head`` [n_roles] maps roles to heads."""
    lib = _load()
    dt = 0 if dtype == "f32" else 1
    store = np.float32 if dt == 0 else np.uint16
    x = _c(x, store)
    n = x.shape[0]
    ws = [_c(w, store) for w in weights]
    bs = [_c(b, np.float32) for b in biases]
    L = len(ws)
    dims = np.array([x.shape[1]] + [w.shape[0] for w in ws], dtype=np.int32)
    for l, w in enumerate(ws):
        assert w.shape == (dims[l + 1], dims[l]), "weight shapes must chain [out][in]"
    wptr = (ctypes.c_void_p * L)(*[w.ctypes.data for w in ws])
    bptr = (ctypes.c_void_p * L)(*[b.ctypes.data for b in bs])
    rh, tc = _c(role_head, np.int32), _c(tool_coef, np.float32)
    kx, ky = _c(iso_x, np.float32), _c(iso_y, np.float32)
    pl, mi = _c(prompt_len, np.int32), _c(model_id, np.int32)
    ri, ta = _c(role_id, np.int32), _c(tool_avail, np.int32)
    alpha = _c(kv_bytes_per_token, np.float32)
    pt = np.empty(n, np.float32)
    pred = np.empty(n, np.float32)
    kv = np.empty(n, np.float64)
    st = lib.oracle_predict_two_phase(L, _ptr(dims), dt, ctypes.cast(wptr, ctypes.c_void_p),
                                      ctypes.cast(bptr, ctypes.c_void_p), rh.shape[0], _ptr(rh), _ptr(tc),
                                      kx.shape[0], _ptr(kx), _ptr(ky), float(max_len), n, _ptr(x), _ptr(pl),
                                      _ptr(mi), _ptr(ri), _ptr(ta), _ptr(alpha), alpha.shape[0], _ptr(pt),
                                      _ptr(pred), _ptr(kv), n_threads or max_threads())
    if st != 0:
        raise RuntimeError(f"oracle_predict_two_phase failed with status {st}")
    return pt, pred, kv


def predict_role_lengths(x: np.ndarray, weights: Sequence[np.ndarray], biases: Sequence[np.ndarray],
                         role_group, tool_coef, max_len: float, prompt_len, model_id, role_id, p_tool,
                         kv_bytes_per_token, dtype: str, pred_len, kv_bytes, n_threads: int = 0):
    """Per-role regressors: ``weights[l]`` [G][out][in] and ``biases[l]`` [G][out] stack the
    layers of the G regressor networks; ``role_group`` [n_roles] maps a role to its regressor
    (-1: none); ``p_tool`` is the first phase's calibrated tool probability. Returns copies of
    (pred_len float32 [N], kv_bytes float64 [N]) with the stages of roles that have a regressor
    predicted by it and every other stage as given."""
    lib = _load()
    dt = 0 if dtype == "f32" else 1
    store = np.float32 if dt == 0 else np.uint16
    x = _c(x, store)
    n = x.shape[0]
    ws = [_c(w, store) for w in weights]
    bs = [_c(b, np.float32) for b in biases]
    L = len(ws)
    G = ws[0].shape[0]
    dims = np.array([x.shape[1]] + [w.shape[1] for w in ws], dtype=np.int32)
    for l, w in enumerate(ws):
        assert w.shape == (G, dims[l + 1], dims[l]), "weight shapes must chain [G][out][in]"
        assert bs[l].shape == (G, dims[l + 1])
    wptr = (ctypes.c_void_p * L)(*[w.ctypes.data for w in ws])
    bptr = (ctypes.c_void_p * L)(*[b.ctypes.data for b in bs])
    rg, tc = _c(role_group, np.int32), _c(tool_coef, np.float32)
    pl, mi, ri = _c(prompt_len, np.int32), _c(model_id, np.int32), _c(role_id, np.int32)
    pt = _c(p_tool, np.float32)
    alpha = _c(kv_bytes_per_token, np.float32)
    pred = np.array(pred_len, np.float32, copy=True)
    kv = np.array(kv_bytes, np.float64, copy=True)
    assert tc.shape == (G,) and pt.shape == pred.shape == kv.shape == (n,)
    st = lib.oracle_predict_role_lengths(L, _ptr(dims), dt, G, ctypes.cast(wptr, ctypes.c_void_p),
                                         ctypes.cast(bptr, ctypes.c_void_p), rg.shape[0], _ptr(rg), _ptr(tc),
                                         float(max_len), n, _ptr(x), _ptr(pl), _ptr(mi), _ptr(ri), _ptr(pt),
                                         _ptr(alpha), alpha.shape[0], _ptr(pred), _ptr(kv),
                                         n_threads or max_threads())
    if st != 0:
        raise RuntimeError(f"oracle_predict_role_lengths failed with status {st}")
    return pred, kv


def route(model_id, pred_len, kv_bytes, decode_s_per_token, free_bytes, queue_s, cold_s,
          resident_mask, k: int = 1, rho: float = 0.0, n_threads: int = 0, act_matrix=None):
    """Returns (node_idx int32 [N][k], score float32 [N][k]). With ``act_matrix`` [M][n_models]
    (seconds) T_act comes from it instead of ``cold_s`` / ``resident_mask``."""
    lib = _load()
    mi = _c(model_id, np.int32)
    n = mi.shape[0]
    pr, kv = _c(pred_len, np.float32), _c(kv_bytes, np.float64)
    dec = _c(decode_s_per_token, np.float32)
    fr, q, cd = _c(free_bytes, np.float64), _c(queue_s, np.float32), _c(cold_s, np.float32)
    rm = _c(resident_mask, np.uint64)
    am = None
    if act_matrix is not None:
        am = _c(act_matrix, np.float32)
        assert am.shape == (fr.shape[0], dec.shape[0])
    idx = np.empty((n, k), np.int32)
    sc = np.empty((n, k), np.float32)
    st = lib.oracle_route(n, _ptr(mi), _ptr(pr), _ptr(kv), _ptr(dec), dec.shape[0], fr.shape[0],
                          _ptr(fr), _ptr(q), _ptr(cd), _ptr(rm), _ptr(am), float(rho), int(k), _ptr(idx),
                          _ptr(sc), n_threads or max_threads())
    if st != 0:
        raise RuntimeError(f"oracle_route failed with status {st}")
    return idx, sc


def route_fitness(model_id, src_id, class_id, kv_bytes, free_bytes, queue_ms, act_ms, resident_mask,
                  deg_ms, rtt_ms, class_weights, bounds, k: int = 1, rho: float = 0.0, n_models: int = 0,
                  n_threads: int = 0, engines=None, act_matrix=None):
    """Alg. 3 with the fitness of Eq. 5. rtt_ms [n_src][M]; class_weights [n_classes][3] =
    (gamma, lambda, mu); bounds [6] = window bounds (lo, hi) of RTT, T_ready, C_deg. With
    ``engines`` = (offset [M+1] int32, level [E] int32, freed [E] float64, cost [E] float32,
    c_int) the disruption cost is Alg. 2 / Eq. 4's per (stage, node) and ``deg_ms`` is unused.
    With ``act_matrix`` [M][n_models] (n_models required) T_act comes from it and ``act_ms`` /
    ``resident_mask`` are unused.
    Returns (node_idx int32 [N][k], fitness float32 [N][k])."""
    lib = _load()
    mi = _c(model_id, np.int32)
    n = mi.shape[0]
    si, ci = _c(src_id, np.int32), _c(class_id, np.int32)
    kv = _c(kv_bytes, np.float64)
    fr, q, act = _c(free_bytes, np.float64), _c(queue_ms, np.float32), _c(act_ms, np.float32)
    rm, dg = _c(resident_mask, np.uint64), _c(deg_ms, np.float32)
    rtt = _c(rtt_ms, np.float32)
    cw, bd = _c(class_weights, np.float32), _c(bounds, np.float32)
    M = fr.shape[0]
    idx = np.empty((n, k), np.int32)
    fit = np.empty((n, k), np.float32)
    if engines is None:
        eo = el = ef = ec = None
        c_int = 0.0
    else:
        eo, el = _c(engines[0], np.int32), _c(engines[1], np.int32)
        ef, ec = _c(engines[2], np.float64), _c(engines[3], np.float32)
        c_int = float(engines[4])
    am = None
    if act_matrix is not None:
        if not n_models:
            raise ValueError("act_matrix needs n_models")
        am = _c(act_matrix, np.float32)
        assert am.shape == (M, n_models)
    st = lib.oracle_route_fitness(n, _ptr(mi), _ptr(si), _ptr(ci), _ptr(kv), n_models or 64, M,
                                  rtt.shape[0], cw.shape[0], _ptr(fr), _ptr(q), _ptr(act), _ptr(rm), _ptr(am),
                                  _ptr(dg), _ptr(rtt), _ptr(cw), _ptr(bd), float(rho), int(k),
                                  _ptr(eo), _ptr(el), _ptr(ef), _ptr(ec), c_int,
                                  _ptr(idx), _ptr(fit), n_threads or max_threads())
    if st != 0:
        raise RuntimeError(f"oracle_route_fitness failed with status {st}")
    return idx, fit


def degradation_cost(R: float, level, freed, cost, c_int: float):
    """Alg. 2 + Eq. 4 on one node's engines: the disruption cost of the minimum-impact plan that
    frees R bytes, or None when no plan frees enough (Failure)."""
    lib = _load()
    lv, fr, co = _c(level, np.int32), _c(freed, np.float64), _c(cost, np.float32)
    out = np.zeros(1, np.float32)
    st = lib.oracle_degradation_cost(float(R), lv.shape[0], _ptr(lv), _ptr(fr), _ptr(co), float(c_int), _ptr(out))
    return None if st else float(out[0])


def activation_latency(tier, model_bytes, tier_bw, tier_setup_ms, unit: float = 1000.0):
    """T_act [M][K] float32 of every model on every node from its readiness tier [M][K]
    (0 Running, 1 Sleeping, 2 CPU, 3 Disk, 4 Remote): Size / BW_tier plus a per-tier setup, in
    the time unit with ``unit`` counts per second (1000: ms, the default; 1: s)."""
    lib = _load()
    t = _c(tier, np.uint8)
    M, K = t.shape
    mb, bw, st_ = _c(model_bytes, np.float64), _c(tier_bw, np.float64), _c(tier_setup_ms, np.float32)
    assert mb.shape == (K,) and bw.shape == (5,) and st_.shape == (5,)
    out = np.empty((M, K), np.float32)
    st = lib.oracle_activation_latency(M, K, _ptr(t), _ptr(mb), _ptr(bw), _ptr(st_), float(unit), _ptr(out))
    if st != 0:
        raise RuntimeError(f"oracle_activation_latency failed with status {st}")
    return out


def adaptive_rho(kv_actual, kv_pred, beta: float, q: float):
    """Safety margin from recent prediction errors: returns (ewma float32 [m], rho float32)."""
    lib = _load()
    a, p = _c(kv_actual, np.float64), _c(kv_pred, np.float64)
    m = a.shape[0]
    ew = np.empty(m, np.float32)
    rho = np.empty(1, np.float32)
    st = lib.oracle_adaptive_rho(_ptr(a), _ptr(p), m, float(beta), float(q), _ptr(ew), _ptr(rho))
    if st != 0:
        raise RuntimeError(f"oracle_adaptive_rho failed with status {st}")
    return ew, rho[0]


def quantiles(values, q_lo: float = 0.05, q_hi: float = 0.95):
    """Window bounds: the order statistics of rank floor(q_lo (m-1)) and ceil(q_hi (m-1))."""
    lib = _load()
    v = _c(values, np.float32).reshape(-1)
    out = np.empty(2, np.float32)
    st = lib.oracle_quantiles(_ptr(v), v.shape[0], float(q_lo), float(q_hi), _ptr(out))
    if st != 0:
        raise RuntimeError(f"oracle_quantiles failed with status {st}")
    return out


def prioritize(chain_offset, stage_latency_s, deadline_us, now_us: int, cursor=None):
    """Returns (remaining_us int64 [S], slack_key int32 [W], order int32 [W])."""
    lib = _load()
    off = _c(chain_offset, np.int64)
    W = off.shape[0] - 1
    lat = _c(stage_latency_s, np.float32)
    S = lat.shape[0]
    dl = _c(deadline_us, np.int64)
    cur = None if cursor is None else _c(cursor, np.int32)
    rem = np.empty(S, np.int64)
    key = np.empty(W, np.int32)
    order = np.empty(W, np.int32)
    st = lib.oracle_prioritize(W, S, _ptr(off), _ptr(lat), _ptr(cur), _ptr(dl), int(now_us),
                               _ptr(rem), _ptr(key), _ptr(order))
    if st != 0:
        raise RuntimeError(f"oracle_prioritize failed with status {st}")
    return rem, key, order


def predict_workload(wl, rows: Optional[np.ndarray] = None, n_threads: int = 0):
    """Oracle predict over a Workload (optionally only the stage indices ``rows``)."""
    sel = slice(None) if rows is None else rows
    return predict(wl.x[sel], wl.weights, wl.biases, wl.bin_centre, wl.prompt_len[sel],
                   wl.model_id[sel], wl.kv_bytes_per_token, wl.spec.dtype, n_threads)


def route_workload(wl, pred_len, kv_bytes, rows: Optional[np.ndarray] = None, n_threads: int = 0):
    """Oracle route of a Workload's stages given their predictions (``pred_len``/``kv_bytes``
    indexed like ``rows`` when given)."""
    mi = wl.model_id if rows is None else wl.model_id[rows]
    return route(mi, pred_len, kv_bytes, wl.decode_s_per_token, wl.free_bytes, wl.queue_s,
                 wl.cold_s, wl.resident_mask, k=wl.spec.k, rho=wl.spec.rho, n_threads=n_threads)
