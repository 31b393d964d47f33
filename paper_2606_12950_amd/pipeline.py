"""One scheduling step on the device: predict -> route -> (for chained batches) prioritize.

``to_device`` copies a generated batch into device tensors once; ``run_step`` enqueues the
three C-ABI calls on the current stream, writing into preallocated outputs. The latency fed to
prioritize is each stage's routed best score (its expected completion time on the chosen
node; +inf when no node can admit it).
"""
from __future__ import annotations

from dataclasses import dataclass
from typing import List, Optional

import numpy as np
import torch

from . import _native
from .workload import Workload


@dataclass
class DeviceBatch:
    n: int
    k: int
    rho: float
    x: torch.Tensor
    prompt_len: torch.Tensor
    model_id: torch.Tensor
    weights: List[torch.Tensor]
    biases: List[torch.Tensor]
    bin_centre: torch.Tensor
    kv_bytes_per_token: torch.Tensor
    decode_s_per_token: torch.Tensor
    free_bytes: torch.Tensor
    queue_s: torch.Tensor
    cold_s: torch.Tensor
    resident_mask: torch.Tensor
    chain_offset: Optional[torch.Tensor]
    deadline_us: Optional[torch.Tensor]
    now_us: int


@dataclass
class StepOutputs:
    pred_len: torch.Tensor
    kv_bytes: torch.Tensor
    node_idx: torch.Tensor
    score: torch.Tensor
    remaining_us: Optional[torch.Tensor]
    slack_key: Optional[torch.Tensor]
    order: Optional[torch.Tensor]
    prio_workspace: Optional[torch.Tensor]
    route_workspace: Optional[torch.Tensor]


def _t(a: np.ndarray, device) -> torch.Tensor:
    a = np.ascontiguousarray(a)
    if a.dtype == np.uint16:      # bf16 bit patterns
        return torch.from_numpy(a.view(np.int16)).to(device).view(torch.bfloat16)
    if a.dtype == np.uint64:      # residency masks: same bits as int64
        return torch.from_numpy(a.view(np.int64)).to(device)
    return torch.from_numpy(a).to(device)


def to_device(wl: Workload, device="cuda") -> DeviceBatch:
    chained = wl.n_workflows > 0
    return DeviceBatch(
        n=wl.n, k=wl.spec.k, rho=wl.spec.rho, x=_t(wl.x, device), prompt_len=_t(wl.prompt_len, device),
        model_id=_t(wl.model_id, device), weights=[_t(w, device) for w in wl.weights],
        biases=[_t(b, device) for b in wl.biases], bin_centre=_t(wl.bin_centre, device),
        kv_bytes_per_token=_t(wl.kv_bytes_per_token, device),
        decode_s_per_token=_t(wl.decode_s_per_token, device), free_bytes=_t(wl.free_bytes, device),
        queue_s=_t(wl.queue_s, device), cold_s=_t(wl.cold_s, device),
        resident_mask=_t(wl.resident_mask, device),
        chain_offset=_t(wl.chain_offset, device) if chained else None,
        deadline_us=_t(wl.deadline_us, device) if chained else None, now_us=int(wl.now_us))


def allocate_outputs(b: DeviceBatch) -> StepOutputs:
    dev = b.x.device
    n = b.n
    chained = b.chain_offset is not None
    W = b.chain_offset.shape[0] - 1 if chained else 0
    ws = None
    if chained:
        ws = torch.empty(max(_native.prioritize_workspace_bytes(W, n), 256), dtype=torch.uint8, device=dev)
    rws_bytes = _native.route_workspace_bytes(n, b.decode_s_per_token.shape[0], b.free_bytes.shape[0], b.k)
    rws = torch.empty(rws_bytes, dtype=torch.uint8, device=dev) if rws_bytes else None
    return StepOutputs(
        pred_len=torch.empty(n, dtype=torch.float32, device=dev),
        kv_bytes=torch.empty(n, dtype=torch.float64, device=dev),
        node_idx=torch.empty((n, b.k), dtype=torch.int32, device=dev),
        score=torch.empty((n, b.k), dtype=torch.float32, device=dev),
        remaining_us=torch.empty(n, dtype=torch.int64, device=dev) if chained else None,
        slack_key=torch.empty(W, dtype=torch.int32, device=dev) if chained else None,
        order=torch.empty(W, dtype=torch.int32, device=dev) if chained else None,
        prio_workspace=ws, route_workspace=rws)


def run_predict(b: DeviceBatch, o: StepOutputs, stream=None):
    _native.predict(b.x, b.weights, b.biases, b.bin_centre, b.prompt_len, b.model_id,
                    b.kv_bytes_per_token, out=(o.pred_len, o.kv_bytes), stream=stream)


def run_route(b: DeviceBatch, o: StepOutputs, stream=None, algo: int = _native.ROUTE_AUTO):
    _native.route(b.model_id, o.pred_len, o.kv_bytes, b.decode_s_per_token, b.free_bytes, b.queue_s,
                  b.cold_s, b.resident_mask, k=b.k, rho=b.rho, algo=algo, out=(o.node_idx, o.score),
                  workspace=o.route_workspace, stream=stream)


def run_prioritize(b: DeviceBatch, o: StepOutputs, stream=None):
    # stage latency = the routed best score (column 0 of the [N][k] score matrix)
    lat = o.score if b.k == 1 else o.score[:, 0].contiguous()
    _native.prioritize(b.chain_offset, lat.reshape(-1), b.deadline_us, b.now_us,
                       out=(o.remaining_us, o.slack_key, o.order), workspace=o.prio_workspace,
                       stream=stream)


def run_step(b: DeviceBatch, o: Optional[StepOutputs] = None, stream=None) -> StepOutputs:
    """Enqueue one full step on the stream (no synchronisation)."""
    if o is None:
        o = allocate_outputs(b)
    run_predict(b, o, stream)
    run_route(b, o, stream)
    if b.chain_offset is not None:
        run_prioritize(b, o, stream)
    return o
