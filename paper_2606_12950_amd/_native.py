"""Thin ctypes binding of libmaestro's C-ABI (include/maestro.h).

Argument marshalling only: every step of predict / route / prioritize runs in the HIP
kernels of libmaestro.so. PyTorch provides device memory (tensors, workspaces) and the
stream (the current torch stream). There is no fallback: if the library is not built or no
GPU is present, the calls raise.
"""
from __future__ import annotations

import ctypes
import os
from typing import NamedTuple, Optional, Sequence, Tuple

import torch

_PKG = os.path.dirname(os.path.abspath(__file__))
LIBRARY_PATH = os.path.join(_PKG, "libmaestro.so")

MAESTRO_F32, MAESTRO_BF16 = 0, 1
_STATUS = {0: "ok", 1: "invalid argument", 2: "unsupported shape", 3: "workspace too small",
           4: "kernel launch failed"}

# Every function declared in include/maestro.h.
EXPORTS = ("maestro_predict", "maestro_predict_two_phase", "maestro_route", "maestro_route_tiered", "maestro_route_ex", "maestro_route_fitness",
           "maestro_degradation_plans", "maestro_activation_latency", "maestro_adaptive_rho", "maestro_quantiles", "maestro_prioritize", "maestro_predict_workspace",
           "maestro_route_workspace", "maestro_prioritize_workspace", "maestro_status_string",
           "maestro_prioritize_noalloc", "maestro_predict_role_lengths", "maestro_role_lengths_workspace",
           "maestro_route_lists_bytes", "maestro_route_sort_nodes", "maestro_route_walk",
           "maestro_quantiles_workspace")

PRIORITIZE_NOALLOC_MAX_WORKFLOWS = 1 << 20

ROUTE_AUTO, ROUTE_SCAN, ROUTE_SORTED = 0, 1, 2

PLAN_RECORD_STEPS = 8   # steps held in a node's record; more engines continue in the step array
PLAN_BYTES = 128   # one maestro_deg_plan record: freed f64[8], cost f32[8], n_engines, first_step, pad
STEP_BYTES = 16    # one maestro_plan_step: freed f64, cost f32, engine i32


class DegradationPlans(NamedTuple):
    """Output of maestro_degradation_plans: ``records`` uint8 [n_nodes][128] (maestro_deg_plan)
    and ``steps`` uint8 [max(E, 1)][16] (maestro_plan_step, node j's at [engine_offset[j],
    engine_offset[j+1]))."""
    records: torch.Tensor
    steps: torch.Tensor


class MaestroError(RuntimeError):
    def __init__(self, fn: str, status: int):
        super().__init__(f"{fn} failed: {_STATUS.get(status, status)} (status {status})")
        self.status = status


class Predictor(ctypes.Structure):
    """Mirror of ``maestro_predictor``."""
    _fields_ = [("n_layers", ctypes.c_int32), ("dims", ctypes.c_int32 * 5),
                ("dtype", ctypes.c_int32), ("weight", ctypes.c_void_p * 4),
                ("bias", ctypes.c_void_p * 4), ("bin_centre", ctypes.c_void_p)]


class RoleRegressors(ctypes.Structure):
    """Mirror of ``maestro_role_regressors``."""
    _fields_ = [("n_regressors", ctypes.c_int32), ("n_roles", ctypes.c_int32), ("role_regressor", ctypes.c_void_p),
                ("tool_coef", ctypes.c_void_p), ("max_len", ctypes.c_float)]


class TwoPhase(ctypes.Structure):
    """Mirror of ``maestro_two_phase``."""
    _fields_ = [("n_roles", ctypes.c_int32), ("n_knots", ctypes.c_int32), ("role_head", ctypes.c_void_p),
                ("tool_coef", ctypes.c_void_p), ("iso_x", ctypes.c_void_p), ("iso_y", ctypes.c_void_p),
                ("max_len", ctypes.c_float)]


_lib = None


def load():
    """Load libmaestro.so (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIBRARY_PATH):
        raise RuntimeError(f"{LIBRARY_PATH} is missing: build it first "
                           "(python -m paper_2606_12950_amd.build)")
    lib = ctypes.CDLL(LIBRARY_PATH)
    P, i32, i64, f64, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_double, ctypes.c_size_t
    lib.maestro_predict.argtypes = [ctypes.POINTER(Predictor), i64, P, P, P, P, i32, P, P, P, sz, P]
    lib.maestro_predict_two_phase.argtypes = [ctypes.POINTER(Predictor), ctypes.POINTER(TwoPhase), i64, P, P, P,
                                              P, P, P, i32, P, P, P, P]
    lib.maestro_predict_role_lengths.argtypes = [ctypes.POINTER(Predictor), ctypes.POINTER(RoleRegressors), i64, P,
                                                 P, P, P, P, P, i32, P, P, P, sz, P]
    lib.maestro_predict_role_lengths.restype = ctypes.c_int
    lib.maestro_role_lengths_workspace.argtypes = [i64, i32]
    lib.maestro_role_lengths_workspace.restype = sz
    lib.maestro_route.argtypes = [i64, P, P, P, P, i32, i32, P, P, P, P, f64, i32, P, P, P, sz, P]
    lib.maestro_route_ex.argtypes = [i64, P, P, P, P, i32, i32, P, P, P, P, f64, i32, i32, P, P, P, sz, P]
    lib.maestro_route_fitness.argtypes = [i64, P, P, P, P, i32, i32, i32, i32, P, P, P, P, P, P, P, P, P, P, P,
                                          f64, i32, P, P, P]
    lib.maestro_activation_latency.argtypes = [i32, i32, P, P, P, P, f64, P, P]
    lib.maestro_route_tiered.argtypes = [i64, P, P, P, P, i32, i32, P, P, P, f64, i32, i32, P, P, P, sz, P]
    lib.maestro_adaptive_rho.argtypes = [P, P, i64, f64, f64, P, P, P, sz, P]
    lib.maestro_degradation_plans.argtypes = [i32, P, P, P, P, ctypes.c_float, P, P, P]
    lib.maestro_quantiles.argtypes = [P, i64, f64, f64, P, P, sz, P]
    lib.maestro_quantiles_workspace.argtypes = [i64]
    lib.maestro_quantiles_workspace.restype = sz
    lib.maestro_prioritize.argtypes = [i32, i64, P, P, P, P, i64, P, P, P, P, sz, P]
    lib.maestro_prioritize_noalloc.argtypes = [i32, i64, P, P, P, P, i64, P, P, P, P]
    lib.maestro_route_sort_nodes.argtypes = [i32, i32, P, P, P, P, P, P, sz, P]
    lib.maestro_route_sort_nodes.restype = ctypes.c_int
    lib.maestro_route_walk.argtypes = [i64, P, P, P, P, i32, i32, P, sz, f64, i32, P, P, P]
    lib.maestro_route_walk.restype = ctypes.c_int
    lib.maestro_route_lists_bytes.argtypes = [i32, i32]
    lib.maestro_route_lists_bytes.restype = sz
    for f in ("maestro_predict", "maestro_route", "maestro_route_ex", "maestro_prioritize",
              "maestro_prioritize_noalloc"):
        getattr(lib, f).restype = ctypes.c_int
    lib.maestro_predict_workspace.argtypes = [ctypes.POINTER(Predictor), i64]
    lib.maestro_route_workspace.argtypes = [i64, i32, i32, i32]
    lib.maestro_prioritize_workspace.argtypes = [i32, i64]
    for f in ("maestro_predict_workspace", "maestro_route_workspace", "maestro_prioritize_workspace"):
        getattr(lib, f).restype = sz
    lib.maestro_status_string.argtypes = [ctypes.c_int]
    lib.maestro_status_string.restype = ctypes.c_char_p
    _lib = lib
    return lib


def _ptr(t: Optional[torch.Tensor]):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream) -> ctypes.c_void_p:
    s = stream if stream is not None else torch.cuda.current_stream()
    return ctypes.c_void_p(s.cuda_stream)


def _dev(t: torch.Tensor, name: str, dtype: torch.dtype) -> torch.Tensor:
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise TypeError(f"{name} must be a CUDA (HIP) tensor")
    if t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return t


def _shape(t: torch.Tensor, name: str, shape: Tuple[int, ...]) -> torch.Tensor:
    """Raise unless ``t`` has exactly ``shape``: the kernels index every array by the sizes the
    call passes, so a shorter tensor would be read or written past its end."""
    if tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} must have shape {tuple(shape)}, got {tuple(t.shape)}")
    return t


def _workspace(t: Optional[torch.Tensor], name: str = "workspace") -> Optional[torch.Tensor]:
    if t is not None:
        _dev(t, name, torch.uint8)
    return t


def _check(fn: str, status: int):
    if status != 0:
        raise MaestroError(fn, status)


def make_predictor(weights: Sequence[torch.Tensor], biases: Sequence[torch.Tensor],
                   bin_centre: Optional[torch.Tensor]) -> Predictor:
    """Describe a predictor held in device tensors (weights [out][in], bf16 or fp32); the two-phase
    predictor has no bin centres (None)."""
    L = len(weights)
    if not 1 <= L <= 4 or len(biases) != L:
        raise ValueError("1..4 Linear layers with one bias each")
    dt = weights[0].dtype
    if dt not in (torch.float32, torch.bfloat16):
        raise TypeError("weights must be float32 or bfloat16")
    p = Predictor()
    p.n_layers = L
    p.dtype = MAESTRO_F32 if dt == torch.float32 else MAESTRO_BF16
    p.dims[0] = weights[0].shape[1]
    for l, (w, b) in enumerate(zip(weights, biases)):
        _dev(w, f"weight[{l}]", dt)
        _dev(b, f"bias[{l}]", torch.float32)
        if w.dim() != 2 or w.shape[1] != p.dims[l] or b.shape != (w.shape[0],):
            raise ValueError(f"layer {l}: weight must be [out][in] chaining the previous layer")
        p.dims[l + 1] = w.shape[0]
        p.weight[l] = w.data_ptr()
        p.bias[l] = b.data_ptr()
    if bin_centre is not None:
        _dev(bin_centre, "bin_centre", torch.float32)
        if bin_centre.shape != (p.dims[L],):
            raise ValueError("bin_centre must have one entry per output bin")
        p.bin_centre = bin_centre.data_ptr()
    return p


def predict(x: torch.Tensor, weights: Sequence[torch.Tensor], biases: Sequence[torch.Tensor],
            bin_centre: torch.Tensor, prompt_len: torch.Tensor, model_id: torch.Tensor,
            kv_bytes_per_token: torch.Tensor, out: Optional[Tuple[torch.Tensor, torch.Tensor]] = None,
            stream=None) -> Tuple[torch.Tensor, torch.Tensor]:
    """maestro_predict: returns (pred_len float32 [N], kv_bytes float64 [N])."""
    lib = load()
    p = make_predictor(weights, biases, bin_centre)
    _dev(x, "x", weights[0].dtype)
    n = x.shape[0]
    if x.dim() != 2 or x.shape[1] != p.dims[0]:
        raise ValueError("x must be [N][D]")
    _shape(_dev(prompt_len, "prompt_len", torch.int32), "prompt_len", (n,))
    _shape(_dev(model_id, "model_id", torch.int32), "model_id", (n,))
    _dev(kv_bytes_per_token, "kv_bytes_per_token", torch.float32)
    if kv_bytes_per_token.dim() != 1:
        raise ValueError("kv_bytes_per_token must be [n_models]")
    if out is None:
        out = (torch.empty(n, dtype=torch.float32, device=x.device),
               torch.empty(n, dtype=torch.float64, device=x.device))
    pred, kv = out
    _shape(_dev(pred, "pred_len", torch.float32), "pred_len", (n,))
    _shape(_dev(kv, "kv_bytes", torch.float64), "kv_bytes", (n,))
    ws_bytes = lib.maestro_predict_workspace(ctypes.byref(p), n)
    ws = torch.empty(max(ws_bytes, 1), dtype=torch.uint8, device=x.device) if ws_bytes else None
    st = lib.maestro_predict(ctypes.byref(p), n, _ptr(x), _ptr(prompt_len), _ptr(model_id),
                             _ptr(kv_bytes_per_token), kv_bytes_per_token.shape[0], _ptr(pred),
                             _ptr(kv), _ptr(ws), ws_bytes, _stream(stream))
    _check("maestro_predict", st)
    return pred, kv


def predict_two_phase(x: torch.Tensor, weights: Sequence[torch.Tensor], biases: Sequence[torch.Tensor],
                      role_head: torch.Tensor, tool_coef: torch.Tensor, iso_x: torch.Tensor, iso_y: torch.Tensor,
                      max_len: float, prompt_len: torch.Tensor, model_id: torch.Tensor, role_id: torch.Tensor,
                      tool_avail: torch.Tensor, kv_bytes_per_token: torch.Tensor,
                      out: Optional[Tuple[torch.Tensor, torch.Tensor, torch.Tensor]] = None,
                      stream=None) -> Tuple[torch.Tensor, torch.Tensor, torch.Tensor]:
    """maestro_predict_two_phase: returns (p_tool float32 [N], pred_len float32 [N], kv_bytes
    float64 [N]). The last layer's outputs are heads: 0 the tool-intent logit, g >= 1 the
    log(1 + L) regressors (1 the shared one); ``role_head`` [n_roles] int32 maps roles to heads."""
    lib = load()
    p = make_predictor(weights, biases, None)
    _dev(x, "x", weights[0].dtype)
    n = x.shape[0]
    if x.dim() != 2 or x.shape[1] != p.dims[0]:
        raise ValueError("x must be [N][D]")
    for t, name in ((prompt_len, "prompt_len"), (model_id, "model_id"), (role_id, "role_id"),
                    (tool_avail, "tool_avail"), (role_head, "role_head")):
        _dev(t, name, torch.int32)
    for t, name in ((kv_bytes_per_token, "kv_bytes_per_token"), (tool_coef, "tool_coef"), (iso_x, "iso_x"),
                    (iso_y, "iso_y")):
        _dev(t, name, torch.float32)
    if role_id.shape != (n,) or tool_avail.shape != (n,) or prompt_len.shape != (n,) or model_id.shape != (n,):
        raise ValueError("per-stage inputs must have N entries")
    if tool_coef.shape != (p.dims[p.n_layers],) or iso_x.shape != iso_y.shape:
        raise ValueError("tool_coef needs one entry per output; iso_x and iso_y the same length")
    if role_head.dim() != 1 or iso_x.dim() != 1 or kv_bytes_per_token.dim() != 1:
        raise ValueError("role_head, iso_x, iso_y and kv_bytes_per_token must be one-dimensional")
    tp = TwoPhase()
    tp.n_roles = role_head.shape[0]
    tp.n_knots = iso_x.shape[0]
    tp.role_head = role_head.data_ptr() if role_head.numel() else None
    tp.tool_coef = tool_coef.data_ptr()
    tp.iso_x = iso_x.data_ptr()
    tp.iso_y = iso_y.data_ptr()
    tp.max_len = float(max_len)
    if out is None:
        out = (torch.empty(n, dtype=torch.float32, device=x.device), torch.empty(n, dtype=torch.float32, device=x.device),
               torch.empty(n, dtype=torch.float64, device=x.device))
    pt, pred, kv = out
    if pt is not None:
        _shape(_dev(pt, "p_tool", torch.float32), "p_tool", (n,))
    _shape(_dev(pred, "pred_len", torch.float32), "pred_len", (n,))
    _shape(_dev(kv, "kv_bytes", torch.float64), "kv_bytes", (n,))
    st = lib.maestro_predict_two_phase(ctypes.byref(p), ctypes.byref(tp), n, _ptr(x), _ptr(prompt_len),
                                       _ptr(model_id), _ptr(role_id), _ptr(tool_avail), _ptr(kv_bytes_per_token),
                                       kv_bytes_per_token.shape[0], _ptr(pt), _ptr(pred), _ptr(kv), _stream(stream))
    _check("maestro_predict_two_phase", st)
    return pt, pred, kv


def predict_role_lengths(x: torch.Tensor, weights: Sequence[torch.Tensor], biases: Sequence[torch.Tensor],
                         role_regressor: torch.Tensor, tool_coef: torch.Tensor, max_len: float,
                         prompt_len: torch.Tensor, model_id: torch.Tensor, role_id: torch.Tensor, p_tool: torch.Tensor,
                         kv_bytes_per_token: torch.Tensor, pred_len: torch.Tensor, kv_bytes: torch.Tensor,
                         workspace: Optional[torch.Tensor] = None, stream=None) -> Tuple[torch.Tensor, torch.Tensor]:
    """maestro_predict_role_lengths: the per-role regressors over the stages whose role has one,
    written into ``pred_len`` / ``kv_bytes`` in place (returned). ``weights[l]`` [G][out][in] and
    ``biases[l]`` [G][out] stack the G regressors' layers; ``role_regressor`` [n_roles] int32 maps
    a role to its regressor (-1: none); ``p_tool`` is the first phase's calibrated probability."""
    lib = load()
    L = len(weights)
    if not 1 <= L <= 4 or len(biases) != L:
        raise ValueError("1..4 Linear layers with one bias each")
    dt = weights[0].dtype
    G = weights[0].shape[0]
    p = Predictor()
    p.n_layers = L
    p.dtype = MAESTRO_F32 if dt == torch.float32 else MAESTRO_BF16
    p.dims[0] = weights[0].shape[2]
    for l, (w, b) in enumerate(zip(weights, biases)):
        _dev(w, f"weight[{l}]", dt)
        _dev(b, f"bias[{l}]", torch.float32)
        if w.dim() != 3 or w.shape[0] != G or w.shape[2] != p.dims[l] or tuple(b.shape) != (G, w.shape[1]):
            raise ValueError(f"layer {l}: weight must be [G][out][in] chaining the previous layer, bias [G][out]")
        p.dims[l + 1] = w.shape[1]
        p.weight[l] = w.data_ptr()
        p.bias[l] = b.data_ptr()
    _dev(x, "x", dt)
    n = x.shape[0]
    if x.dim() != 2 or x.shape[1] != p.dims[0]:
        raise ValueError("x must be [N][D]")
    for t, name in ((prompt_len, "prompt_len"), (model_id, "model_id"), (role_id, "role_id"),
                    (role_regressor, "role_regressor")):
        _dev(t, name, torch.int32)
    for t, name in ((kv_bytes_per_token, "kv_bytes_per_token"), (tool_coef, "tool_coef"), (p_tool, "p_tool")):
        _dev(t, name, torch.float32)
    for t, name in ((prompt_len, "prompt_len"), (model_id, "model_id"), (role_id, "role_id"), (p_tool, "p_tool")):
        _shape(t, name, (n,))
    _shape(_dev(pred_len, "pred_len", torch.float32), "pred_len", (n,))
    _shape(_dev(kv_bytes, "kv_bytes", torch.float64), "kv_bytes", (n,))
    _shape(tool_coef, "tool_coef", (G,))
    if role_regressor.dim() != 1 or kv_bytes_per_token.dim() != 1:
        raise ValueError("role_regressor and kv_bytes_per_token must be one-dimensional")
    r = RoleRegressors()
    r.n_regressors = G
    r.n_roles = role_regressor.shape[0]
    r.role_regressor = role_regressor.data_ptr() if role_regressor.numel() else None
    r.tool_coef = tool_coef.data_ptr()
    r.max_len = float(max_len)
    need = lib.maestro_role_lengths_workspace(n, G)
    _workspace(workspace)
    if workspace is None:
        workspace = torch.empty(max(need, 256), dtype=torch.uint8, device=x.device)
    st = lib.maestro_predict_role_lengths(ctypes.byref(p), ctypes.byref(r), n, _ptr(x), _ptr(prompt_len),
                                          _ptr(model_id), _ptr(role_id), _ptr(p_tool), _ptr(kv_bytes_per_token),
                                          kv_bytes_per_token.shape[0], _ptr(pred_len), _ptr(kv_bytes),
                                          _ptr(workspace), workspace.numel(), _stream(stream))
    _check("maestro_predict_role_lengths", st)
    return pred_len, kv_bytes


def route(model_id: torch.Tensor, pred_len: torch.Tensor, kv_bytes: torch.Tensor,
          decode_s_per_token: torch.Tensor, free_bytes: torch.Tensor, queue_s: torch.Tensor,
          cold_s: Optional[torch.Tensor], resident_mask: Optional[torch.Tensor], k: int = 1, rho: float = 0.0,
          algo: int = ROUTE_AUTO, out: Optional[Tuple[torch.Tensor, torch.Tensor]] = None,
          workspace: Optional[torch.Tensor] = None, stream=None,
          act_s: Optional[torch.Tensor] = None) -> Tuple[torch.Tensor, torch.Tensor]:
    """maestro_route_ex: returns (node_idx int32 [N][k], score float32 [N][k]); with ``act_s``
    [n_nodes][n_models] (seconds, from readiness tiers) maestro_route_tiered instead, and
    ``cold_s`` / ``resident_mask`` may be None.

    ``resident_mask`` is int64 on the torch side (same bits as the C-ABI's uint64)."""
    lib = load()
    _dev(model_id, "model_id", torch.int32)
    n = model_id.shape[0]
    _dev(pred_len, "pred_len", torch.float32)
    _dev(kv_bytes, "kv_bytes", torch.float64)
    _dev(decode_s_per_token, "decode_s_per_token", torch.float32)
    _dev(free_bytes, "free_bytes", torch.float64)
    _dev(queue_s, "queue_s", torch.float32)
    M = free_bytes.shape[0]
    K = decode_s_per_token.shape[0]
    if model_id.dim() != 1 or free_bytes.dim() != 1 or decode_s_per_token.dim() != 1:
        raise ValueError("model_id, free_bytes and decode_s_per_token must be one-dimensional")
    if pred_len.shape != (n,) or kv_bytes.shape != (n,):
        raise ValueError("per-stage inputs must have the same length")
    if act_s is not None:
        _dev(act_s, "act_s", torch.float32)
        if tuple(act_s.shape) != (M, K):
            raise ValueError("act_s must be [n_nodes][n_models]")
    else:
        _dev(cold_s, "cold_s", torch.float32)
        _dev(resident_mask, "resident_mask", torch.int64)
        if cold_s.shape != (M,) or resident_mask.shape != (M,):
            raise ValueError("per-node inputs must have the same length")
    if queue_s.shape != (M,):
        raise ValueError("per-node inputs must have the same length")
    if out is None:
        out = (torch.empty((n, k), dtype=torch.int32, device=model_id.device),
               torch.empty((n, k), dtype=torch.float32, device=model_id.device))
    idx, sc = out
    _shape(_dev(idx, "node_idx", torch.int32), "node_idx", (n, k))
    _shape(_dev(sc, "score", torch.float32), "score", (n, k))
    _workspace(workspace)
    ws_bytes = route_workspace_bytes(n, decode_s_per_token.shape[0], M, k)
    if ws_bytes and workspace is None:
        workspace = torch.empty(ws_bytes, dtype=torch.uint8, device=model_id.device)
    ws = (_ptr(workspace) if workspace is not None else None, workspace.numel() if workspace is not None else 0)
    if act_s is not None:
        st = lib.maestro_route_tiered(n, _ptr(model_id), _ptr(pred_len), _ptr(kv_bytes), _ptr(decode_s_per_token),
                                      K, M, _ptr(free_bytes), _ptr(queue_s), _ptr(act_s), float(rho), int(k),
                                      int(algo), _ptr(idx), _ptr(sc), ws[0], ws[1], _stream(stream))
        _check("maestro_route_tiered", st)
        return idx, sc
    st = lib.maestro_route_ex(n, _ptr(model_id), _ptr(pred_len), _ptr(kv_bytes),
                              _ptr(decode_s_per_token), K, M,
                              _ptr(free_bytes), _ptr(queue_s), _ptr(cold_s), _ptr(resident_mask),
                              float(rho), int(k), int(algo), _ptr(idx), _ptr(sc), ws[0], ws[1],
                              _stream(stream))
    _check("maestro_route_ex", st)
    return idx, sc


def route_fitness(model_id: torch.Tensor, src_id: torch.Tensor, class_id: torch.Tensor,
                  kv_bytes: torch.Tensor, free_bytes: torch.Tensor, queue_ms: torch.Tensor,
                  act_ms: torch.Tensor, resident_mask: torch.Tensor, deg_ms: Optional[torch.Tensor],
                  rtt_ms: torch.Tensor, class_weights: torch.Tensor, bounds: torch.Tensor,
                  n_models: int, k: int = 1, rho: float = 0.0, plans: Optional[DegradationPlans] = None,
                  act_matrix: Optional[torch.Tensor] = None,
                  out: Optional[Tuple[torch.Tensor, torch.Tensor]] = None,
                  stream=None) -> Tuple[torch.Tensor, torch.Tensor]:
    """maestro_route_fitness: returns (node_idx int32 [N][k], fitness float32 [N][k]).

    ``rtt_ms`` is [n_src][n_nodes], ``class_weights`` [n_classes][3] = (gamma, lambda, mu),
    ``bounds`` [6] = (lo, hi) of RTT, T_ready, C_deg; ``resident_mask`` is int64 on the torch
    side (same bits as the C-ABI's uint64). With ``plans`` (from :func:`degradation_plans`)
    C_deg comes from the node's degradation plan and ``deg_ms`` may be None. With ``act_matrix``
    [n_nodes][n_models] (from :func:`activation_latency`) T_act comes from it and ``act_ms`` /
    ``resident_mask`` may be None."""
    lib = load()
    _dev(model_id, "model_id", torch.int32)
    n = model_id.shape[0]
    _dev(src_id, "src_id", torch.int32)
    _dev(class_id, "class_id", torch.int32)
    _dev(kv_bytes, "kv_bytes", torch.float64)
    _dev(free_bytes, "free_bytes", torch.float64)
    for t, name in ((queue_ms, "queue_ms"), (rtt_ms, "rtt_ms"), (class_weights, "class_weights"),
                    (bounds, "bounds")):
        _dev(t, name, torch.float32)
    M = free_bytes.shape[0]
    if model_id.dim() != 1 or free_bytes.dim() != 1:
        raise ValueError("model_id and free_bytes must be one-dimensional")
    if src_id.shape != (n,) or class_id.shape != (n,) or kv_bytes.shape != (n,):
        raise ValueError("per-stage inputs must have the same length")
    if queue_ms.shape != (M,):
        raise ValueError("per-node inputs must have the same length")
    if act_matrix is not None:
        _dev(act_matrix, "act_matrix", torch.float32)
        if tuple(act_matrix.shape) != (M, n_models):
            raise ValueError("act_matrix must be [n_nodes][n_models]")
    else:
        _dev(act_ms, "act_ms", torch.float32)
        _dev(resident_mask, "resident_mask", torch.int64)
        if act_ms.shape != (M,) or resident_mask.shape != (M,):
            raise ValueError("per-node inputs must have the same length")
    if plans is not None:
        _dev(plans.records, "plans.records", torch.uint8)
        _dev(plans.steps, "plans.steps", torch.uint8)
        if tuple(plans.records.shape) != (M, PLAN_BYTES):
            raise ValueError("plans.records must be uint8 [n_nodes][128]")
        if plans.steps.dim() != 2 or plans.steps.shape[1] != STEP_BYTES:
            raise ValueError("plans.steps must be uint8 [E][16]")
    if deg_ms is not None:
        _dev(deg_ms, "deg_ms", torch.float32)
        if deg_ms.shape != (M,):
            raise ValueError("per-node inputs must have the same length")
    elif plans is None:
        raise ValueError("deg_ms is required without plans")
    if rtt_ms.dim() != 2 or rtt_ms.shape[1] != M:
        raise ValueError("rtt_ms must be [n_src][n_nodes]")
    if class_weights.dim() != 2 or class_weights.shape[1] != 3 or bounds.numel() != 6:
        raise ValueError("class_weights must be [n_classes][3] and bounds hold 6 values")
    if out is None:
        out = (torch.empty((n, k), dtype=torch.int32, device=model_id.device),
               torch.empty((n, k), dtype=torch.float32, device=model_id.device))
    idx, fit = out
    _shape(_dev(idx, "node_idx", torch.int32), "node_idx", (n, k))
    _shape(_dev(fit, "fitness", torch.float32), "fitness", (n, k))
    st = lib.maestro_route_fitness(n, _ptr(model_id), _ptr(src_id), _ptr(class_id), _ptr(kv_bytes),
                                   int(n_models), M, rtt_ms.shape[0], class_weights.shape[0],
                                   _ptr(free_bytes), _ptr(queue_ms), _ptr(act_ms), _ptr(resident_mask),
                                   _ptr(act_matrix),
                                   _ptr(deg_ms) if deg_ms is not None else None,
                                   _ptr(plans.records) if plans is not None else None,
                                   _ptr(plans.steps) if plans is not None else None,
                                   _ptr(rtt_ms), _ptr(class_weights), _ptr(bounds),
                                   float(rho), int(k), _ptr(idx), _ptr(fit), _stream(stream))
    _check("maestro_route_fitness", st)
    return idx, fit


def degradation_plans(engine_offset: torch.Tensor, engine_level: torch.Tensor, engine_freed_bytes: torch.Tensor,
                      engine_cost_ms: torch.Tensor, c_int_ms: float, out: Optional[DegradationPlans] = None,
                      stream=None) -> DegradationPlans:
    """maestro_degradation_plans: the plan records and steps (:class:`DegradationPlans`) of every
    node from its engines in CSR form (``engine_offset`` int32 [n_nodes + 1], any number of
    engines a node; ``engine_level`` int32, ``engine_freed_bytes`` float64, ``engine_cost_ms``
    float32)."""
    lib = load()
    _dev(engine_offset, "engine_offset", torch.int32)
    _dev(engine_level, "engine_level", torch.int32)
    _dev(engine_freed_bytes, "engine_freed_bytes", torch.float64)
    _dev(engine_cost_ms, "engine_cost_ms", torch.float32)
    M = engine_offset.shape[0] - 1
    if M < 0:
        raise ValueError("engine_offset holds n_nodes + 1 entries")
    E = engine_level.shape[0]
    if engine_offset.dim() != 1 or engine_level.dim() != 1:
        raise ValueError("engine_offset and engine_level must be one-dimensional")
    if engine_freed_bytes.shape != (E,) or engine_cost_ms.shape != (E,):
        raise ValueError("per-engine inputs must have the same length")
    if out is None:
        out = DegradationPlans(torch.empty((M, PLAN_BYTES), dtype=torch.uint8, device=engine_offset.device),
                               torch.empty((max(E, 1), STEP_BYTES), dtype=torch.uint8, device=engine_offset.device))
    _dev(out.records, "plans.records", torch.uint8)
    _dev(out.steps, "plans.steps", torch.uint8)
    if tuple(out.records.shape) != (M, PLAN_BYTES):
        raise ValueError("plans.records must be uint8 [n_nodes][128]")
    if out.steps.dim() != 2 or out.steps.shape[1] != STEP_BYTES or out.steps.shape[0] < E:
        raise ValueError("plans.steps must be uint8 [>= E][16]")
    st = lib.maestro_degradation_plans(M, _ptr(engine_offset), _ptr(engine_level) if E else None,
                                       _ptr(engine_freed_bytes) if E else None,
                                       _ptr(engine_cost_ms) if E else None, float(c_int_ms), _ptr(out.records),
                                       _ptr(out.steps), _stream(stream))
    _check("maestro_degradation_plans", st)
    return out


def activation_latency(tier: torch.Tensor, model_bytes: torch.Tensor, tier_bw: torch.Tensor,
                       tier_setup_ms: torch.Tensor, out: Optional[torch.Tensor] = None, stream=None,
                       unit: float = 1000.0) -> torch.Tensor:
    """maestro_activation_latency: T_act [n_nodes][n_models] float32 from the readiness tier
    [n_nodes][n_models] uint8 (0 Running .. 4 Remote), model sizes [n_models] float64 (bytes),
    tier bandwidths [5] float64 (bytes/s) and setup times [5] float32, in the time unit with
    ``unit`` counts per second (1000: ms, the default; 1: s)."""
    lib = load()
    _dev(tier, "tier", torch.uint8)
    _dev(model_bytes, "model_bytes", torch.float64)
    _dev(tier_bw, "tier_bw", torch.float64)
    _dev(tier_setup_ms, "tier_setup_ms", torch.float32)
    if tier.dim() != 2 or model_bytes.shape != (tier.shape[1],) or tier_bw.shape != (5,) or tier_setup_ms.shape != (5,):
        raise ValueError("tier [n_nodes][n_models], model_bytes [n_models], tier_bw and tier_setup_ms [5]")
    M, K = tier.shape
    if out is None:
        out = torch.empty((M, K), dtype=torch.float32, device=tier.device)
    _shape(_dev(out, "act_ms", torch.float32), "act_ms", (M, K))
    st = lib.maestro_activation_latency(M, K, _ptr(tier) if M else None, _ptr(model_bytes), _ptr(tier_bw),
                                        _ptr(tier_setup_ms), float(unit), _ptr(out) if M else None, _stream(stream))
    _check("maestro_activation_latency", st)
    return out


def quantiles_workspace_bytes(m: int) -> int:
    return int(load().maestro_quantiles_workspace(m))


def _select_workspace(m: int, workspace: Optional[torch.Tensor], device) -> Tuple[Optional[int], int]:
    _workspace(workspace)
    need = quantiles_workspace_bytes(m)
    if need and workspace is None:
        workspace = torch.empty(need, dtype=torch.uint8, device=device)
    return (_ptr(workspace), workspace.numel()) if workspace is not None else (None, 0)


def adaptive_rho(kv_actual: torch.Tensor, kv_pred: torch.Tensor, beta: float, q: float,
                 out: Optional[Tuple[torch.Tensor, torch.Tensor]] = None, workspace: Optional[torch.Tensor] = None,
                 stream=None) -> Tuple[torch.Tensor, torch.Tensor]:
    """maestro_adaptive_rho: returns (ewma float32 [m], rho float32 [1]) on the device; the
    workspace (quantiles_workspace_bytes(m), uint8) is allocated when needed and not given."""
    lib = load()
    _dev(kv_actual, "kv_actual", torch.float64)
    _dev(kv_pred, "kv_pred", torch.float64)
    m = kv_actual.shape[0]
    if kv_actual.dim() != 1 or kv_pred.shape != (m,):
        raise ValueError("kv_actual and kv_pred must have the same length")
    if out is None:
        out = (torch.empty(m, dtype=torch.float32, device=kv_actual.device),
               torch.empty(1, dtype=torch.float32, device=kv_actual.device))
    ew, rho = out
    _shape(_dev(ew, "ewma", torch.float32), "ewma", (m,))
    _shape(_dev(rho, "rho", torch.float32), "rho", (1,))
    ws = _select_workspace(m, workspace, kv_actual.device)
    st = lib.maestro_adaptive_rho(_ptr(kv_actual), _ptr(kv_pred), m, float(beta), float(q), _ptr(ew), _ptr(rho),
                                  ws[0], ws[1], _stream(stream))
    _check("maestro_adaptive_rho", st)
    return ew, rho


def quantiles(values: torch.Tensor, q_lo: float = 0.05, q_hi: float = 0.95,
              out: Optional[torch.Tensor] = None, workspace: Optional[torch.Tensor] = None,
              stream=None) -> torch.Tensor:
    """maestro_quantiles: float32 [2] on the device = the order statistics of rank
    floor(q_lo (m-1)) and ceil(q_hi (m-1)) of ``values``; the workspace
    (quantiles_workspace_bytes(m), uint8) is allocated when needed and not given."""
    lib = load()
    _dev(values, "values", torch.float32)
    if out is None:
        out = torch.empty(2, dtype=torch.float32, device=values.device)
    _shape(_dev(out, "out", torch.float32), "out", (2,))
    ws = _select_workspace(values.numel(), workspace, values.device)
    st = lib.maestro_quantiles(_ptr(values), values.numel(), float(q_lo), float(q_hi), _ptr(out), ws[0], ws[1],
                               _stream(stream))
    _check("maestro_quantiles", st)
    return out


def route_workspace_bytes(n: int, n_models: int, n_nodes: int, k: int) -> int:
    return int(load().maestro_route_workspace(n, n_models, n_nodes, k))


def route_lists_bytes(n_models: int, n_nodes: int) -> int:
    """maestro_route_lists_bytes: device bytes of the per-model node lists (0 past 8,192 nodes)."""
    return int(load().maestro_route_lists_bytes(n_models, n_nodes))


def route_sort_nodes(free_bytes: torch.Tensor, queue_s: torch.Tensor, cold_s: Optional[torch.Tensor],
                     resident_mask: Optional[torch.Tensor], n_models: int, act_s: Optional[torch.Tensor] = None,
                     lists: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    """maestro_route_sort_nodes: every model's nodes in (ready time, index) order with their
    headroom, into ``lists`` (uint8, route_lists_bytes(n_models, n_nodes) bytes; allocated when
    None) -- the node half of the sorted route. With ``act_s`` [n_nodes][n_models] (seconds)
    the readiness-tier form; ``cold_s`` / ``resident_mask`` may then be None."""
    lib = load()
    _dev(free_bytes, "free_bytes", torch.float64)
    _dev(queue_s, "queue_s", torch.float32)
    M = free_bytes.shape[0]
    if free_bytes.dim() != 1 or queue_s.shape != (M,):
        raise ValueError("per-node inputs must be one-dimensional and of the same length")
    if act_s is not None:
        _dev(act_s, "act_s", torch.float32)
        if tuple(act_s.shape) != (M, n_models):
            raise ValueError("act_s must be [n_nodes][n_models]")
    else:
        _dev(cold_s, "cold_s", torch.float32)
        _dev(resident_mask, "resident_mask", torch.int64)
        if cold_s.shape != (M,) or resident_mask.shape != (M,):
            raise ValueError("per-node inputs must have the same length")
    need = route_lists_bytes(n_models, M)
    if lists is None:
        lists = torch.empty(max(need, 16), dtype=torch.uint8, device=free_bytes.device)
    _workspace(lists)
    st = lib.maestro_route_sort_nodes(n_models, M, _ptr(free_bytes), _ptr(queue_s),
                                      _ptr(cold_s) if act_s is None else None,
                                      _ptr(resident_mask) if act_s is None else None,
                                      _ptr(act_s) if act_s is not None else None, _ptr(lists), lists.numel(),
                                      _stream(stream))
    _check("maestro_route_sort_nodes", st)
    return lists


def route_walk(model_id: torch.Tensor, pred_len: torch.Tensor, kv_bytes: torch.Tensor,
               decode_s_per_token: torch.Tensor, n_nodes: int, lists: torch.Tensor, k: int = 1, rho: float = 0.0,
               out: Optional[Tuple[torch.Tensor, torch.Tensor]] = None, stream=None) -> Tuple[torch.Tensor, torch.Tensor]:
    """maestro_route_walk: the stage half of the sorted route over lists from route_sort_nodes;
    returns (node_idx int32 [N][k], score float32 [N][k])."""
    lib = load()
    _dev(model_id, "model_id", torch.int32)
    n = model_id.shape[0]
    _dev(pred_len, "pred_len", torch.float32)
    _dev(kv_bytes, "kv_bytes", torch.float64)
    _dev(decode_s_per_token, "decode_s_per_token", torch.float32)
    if model_id.dim() != 1 or decode_s_per_token.dim() != 1 or pred_len.shape != (n,) or kv_bytes.shape != (n,):
        raise ValueError("per-stage inputs must be one-dimensional and of the same length")
    _workspace(lists)
    if out is None:
        out = (torch.empty((n, k), dtype=torch.int32, device=model_id.device),
               torch.empty((n, k), dtype=torch.float32, device=model_id.device))
    idx, sc = out
    _shape(_dev(idx, "node_idx", torch.int32), "node_idx", (n, k))
    _shape(_dev(sc, "score", torch.float32), "score", (n, k))
    st = lib.maestro_route_walk(n, _ptr(model_id), _ptr(pred_len), _ptr(kv_bytes), _ptr(decode_s_per_token),
                                decode_s_per_token.shape[0], int(n_nodes), _ptr(lists), lists.numel(), float(rho),
                                int(k), _ptr(idx), _ptr(sc), _stream(stream))
    _check("maestro_route_walk", st)
    return idx, sc


def prioritize_workspace_bytes(n_workflows: int, n_stages: int) -> int:
    return int(load().maestro_prioritize_workspace(n_workflows, n_stages))


def prioritize(chain_offset: torch.Tensor, stage_latency_s: torch.Tensor, deadline_us: torch.Tensor,
               now_us: int, cursor: Optional[torch.Tensor] = None, want_remaining: bool = True,
               out: Optional[Tuple[Optional[torch.Tensor], torch.Tensor, torch.Tensor]] = None,
               workspace: Optional[torch.Tensor] = None, stream=None, noalloc: bool = False):
    """maestro_prioritize: returns (remaining_us int64 [S] or None, slack_key int32 [W],
    order int32 [W]). With ``noalloc`` maestro_prioritize_noalloc instead: the library's static
    scratch replaces the workspace (at most PRIORITIZE_NOALLOC_MAX_WORKFLOWS workflows; calls
    that overlap in time on one GPU race), so ``out`` preallocated makes the call allocate
    nothing."""
    lib = load()
    _dev(chain_offset, "chain_offset", torch.int64)
    _dev(stage_latency_s, "stage_latency_s", torch.float32)
    _dev(deadline_us, "deadline_us", torch.int64)
    W = chain_offset.shape[0] - 1
    S = stage_latency_s.shape[0]
    if chain_offset.dim() != 1 or W < 0 or stage_latency_s.dim() != 1:
        raise ValueError("chain_offset [W + 1] and stage_latency_s [S] must be one-dimensional")
    if deadline_us.shape != (W,):
        raise ValueError("one deadline per workflow")
    if cursor is not None:
        _dev(cursor, "cursor", torch.int32)
        if cursor.shape != (W,):
            raise ValueError("one cursor per workflow")
    dev = chain_offset.device
    if out is None:
        out = (torch.empty(S, dtype=torch.int64, device=dev) if want_remaining else None,
               torch.empty(W, dtype=torch.int32, device=dev),
               torch.empty(W, dtype=torch.int32, device=dev))
    rem, key, order = out
    if rem is not None:
        _shape(_dev(rem, "remaining_us", torch.int64), "remaining_us", (S,))
    _shape(_dev(key, "slack_key", torch.int32), "slack_key", (W,))
    _shape(_dev(order, "order", torch.int32), "order", (W,))
    if noalloc:
        if workspace is not None:
            raise ValueError("the allocation-free call takes no workspace")
        st = lib.maestro_prioritize_noalloc(W, S, _ptr(chain_offset), _ptr(stage_latency_s), _ptr(cursor),
                                            _ptr(deadline_us), int(now_us), _ptr(rem), _ptr(key), _ptr(order),
                                            _stream(stream))
        _check("maestro_prioritize_noalloc", st)
        return rem, key, order
    _workspace(workspace)
    ws_bytes = prioritize_workspace_bytes(W, S)
    if workspace is None:
        workspace = torch.empty(max(ws_bytes, 256), dtype=torch.uint8, device=dev)
    st = lib.maestro_prioritize(W, S, _ptr(chain_offset), _ptr(stage_latency_s), _ptr(cursor),
                                _ptr(deadline_us), int(now_us), _ptr(rem), _ptr(key), _ptr(order),
                                _ptr(workspace), workspace.numel(), _stream(stream))
    _check("maestro_prioritize", st)
    return rem, key, order
