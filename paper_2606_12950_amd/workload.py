"""Seeded synthetic workloads for the batched predict -> route -> prioritize step.

This module only *draws inputs*. It holds none of the method's arithmetic (no MLP, no
softmax, no scoring, no scan, no sort), so both the HIP path and the CPU oracle can be fed
from it without sharing any of the computation under test.

The five named workloads follow the paper's workload structure:
  * skewed (Zipf) model popularity (Sec. II, Observation-2 and its long-tail figure),
  * KV demand that grows with prompt + output length (Sec. II, KV cache memory pressure;
    Eq. 3),
  * sequential agent chains of a few stages each (Sec. IV-A, Table I: 144,524 stages over
    46,769 jobs, about 3.1 stages per job),
  * mixed deadlines (Sec. IV-A, SLOs).
The paper's own trace, its Chatbot-Arena popularity data and its trained predictor are not
available, so these seeded draws stand in for them.

Random streams: ``numpy.random.Generator(PCG64(child))`` where the children come from
``SeedSequence(seed).spawn(len(STREAMS))`` in the fixed order of ``STREAMS``; every array is
drawn from its own stream, so changing one size never perturbs another array. The feature
matrix is drawn in chunks of 65,536 rows, chunk c from the c-th child of the "x" stream.
"""
from __future__ import annotations

import dataclasses
import hashlib
import os
from dataclasses import dataclass, field
from typing import Dict, Optional, Tuple

import numpy as np

STREAMS = ("x", "role", "prompt", "model", "W1", "W2", "W3", "free", "resident",
           "cold", "queue", "alpha", "dec", "half", "chain_len", "arrival", "slo")

GB = 1.0e9  # free HBM is drawn in SI gigabytes and passed as a byte count

# Rows of feature matrix drawn per call to the normal generator; fixed so that the drawn
# matrix is a pure function of (seed, N, D).
_X_CHUNK_ROWS = 1 << 16


@dataclass(frozen=True)
class WorkloadSpec:
    """Shape and distribution parameters of one synthetic scheduling batch."""
    name: str
    seed: int
    n_stages: int                       # ignored when n_workflows > 0 (derived from chains)
    n_nodes: int
    n_models: int
    zipf_s: Optional[float]             # None -> uniform model ids
    dims: Tuple[int, ...]               # (D, H1, [H2,] B): Linear layer widths
    dtype: str                          # "f32" or "bf16" (features, weights, hidden)
    prompt_lognormal: Tuple[float, float, int, int]   # (mu, sigma, lo, hi)
    free_gb: Tuple                      # ("uniform", lo, hi) | ("bimodal", lo1, hi1, lo2, hi2)
    resident_p: float
    alpha: Tuple                        # ("const", v) | ("choice", v0, v1, ...)
    dec: Tuple                          # ("const", v) | ("uniform", lo, hi)
    k: int = 1                          # route width (top-k)
    rho: float = 0.0                    # KV safety margin
    n_workflows: int = 0                # > 0 -> chains of stages (prioritize input)
    chain_len: Tuple[int, int] = (3, 8)
    arrival_s: Tuple[float, float] = (0.0, 600.0)
    slo_s: Tuple[float, float] = (10.0, 120.0)
    now_s: float = 600.0
    bin_start: float = 32.0             # bin centre of bin b = bin_start + bin_width * b
    bin_width: float = 64.0
    cold_s: Tuple[float, float] = (2.0, 20.0)
    queue_s: Tuple[float, float] = (0.0, 5.0)

    @property
    def n_bins(self) -> int:
        return self.dims[-1]

    @property
    def n_layers(self) -> int:
        return len(self.dims) - 1


_ALPHA_CHOICES = ("choice", 65536.0, 131072.0, 327680.0)

SPECS: Dict[str, WorkloadSpec] = {
    # Tiny predict-and-route case.
    "c0": WorkloadSpec(
        name="c0", seed=0, n_stages=4096, n_nodes=64, n_models=8, zipf_s=None,
        dims=(64, 128, 32), dtype="f32", prompt_lognormal=(6.0, 1.0, 16, 8192),
        free_gb=("uniform", 0.0, 288.0), resident_p=0.3,
        alpha=("const", 131072.0), dec=("const", 0.02), k=1),
    # Mid batch.
    "c1": WorkloadSpec(
        name="c1", seed=1, n_stages=65536, n_nodes=512, n_models=16, zipf_s=1.1,
        dims=(256, 512, 512, 64), dtype="bf16", prompt_lognormal=(6.0, 1.0, 16, 8192),
        free_gb=("uniform", 0.0, 288.0), resident_p=0.3,
        alpha=_ALPHA_CHOICES, dec=("uniform", 0.010, 0.040), k=1),
    # Large routing sweep: bimodal free HBM, long prompts.
    "c2": WorkloadSpec(
        name="c2", seed=2, n_stages=1048576, n_nodes=1024, n_models=32, zipf_s=1.1,
        dims=(256, 512, 512, 64), dtype="bf16", prompt_lognormal=(6.5, 1.2, 16, 32768),
        free_gb=("bimodal", 0.0, 40.0, 150.0, 288.0), resident_p=0.25,
        alpha=_ALPHA_CHOICES, dec=("uniform", 0.010, 0.040), k=1),
    # Workflow prioritisation: the mid-batch predictor/route setup over chained stages.
    "c3": WorkloadSpec(
        name="c3", seed=3, n_stages=0, n_nodes=512, n_models=16, zipf_s=1.1,
        dims=(256, 512, 512, 64), dtype="bf16", prompt_lognormal=(6.0, 1.0, 16, 8192),
        free_gb=("uniform", 0.0, 288.0), resident_p=0.3,
        alpha=_ALPHA_CHOICES, dec=("uniform", 0.010, 0.040), k=1,
        n_workflows=131072),
    # High contention: top-4 routing, wide predictor.
    "c4": WorkloadSpec(
        name="c4", seed=4, n_stages=4194304, n_nodes=4096, n_models=64, zipf_s=1.3,
        dims=(256, 1024, 1024, 64), dtype="bf16", prompt_lognormal=(6.0, 1.0, 16, 8192),
        free_gb=("uniform", 0.0, 30.0), resident_p=0.3,
        alpha=_ALPHA_CHOICES, dec=("uniform", 0.010, 0.040), k=4),
}

DESCRIPTIONS = {
    "c0": "tiny predict+route: N=4096 stages, M=64 nodes, 8 models, MLP 64-128-32 fp32",
    "c1": "mid batch: N=65536, M=512, 16 models Zipf(1.1), MLP 256-512-512-64 bf16",
    "c2": "large routing sweep: N=1048576, M=1024, 32 models, bimodal free HBM",
    "c3": "workflow prioritisation: W=131072 chains of 3..8 stages, M=512, "
          "MLP 256-512-512-64 bf16, then slack ordering",
    "c4": "high contention: N=4194304, M=4096, 64 models Zipf(1.3), top-4, "
          "MLP 256-1024-1024-64 bf16",
}


def f32_to_bf16_bits(a: np.ndarray) -> np.ndarray:
    """Round finite float32 values to bfloat16 (round to nearest, ties to even).

    This is a storage cast of drawn data, returned as the raw uint16 bit patterns.
    """
    a = np.ascontiguousarray(a, dtype=np.float32)
    u = a.view(np.uint32)
    r = (u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))) >> np.uint32(16)
    return r.astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    """Exact widening of bfloat16 bit patterns to float32."""
    b = np.ascontiguousarray(b, dtype=np.uint16)
    return (b.astype(np.uint32) << np.uint32(16)).view(np.float32)


@dataclass
class Workload:
    """All inputs of one batch. Array layouts match the C-ABI (row-major, one row per stage
    or node). bf16 arrays are stored as uint16 bit patterns."""
    spec: WorkloadSpec
    # stages
    x: Optional[np.ndarray]             # [N][D] float32, or uint16 (bf16 bits)
    role: np.ndarray                    # [N] int32 (metadata, not read by the predictor)
    prompt_len: np.ndarray              # [N] int32
    model_id: np.ndarray                # [N] int32
    # predictor
    weights: list                       # per layer [out][in]: float32 or uint16 (bf16 bits)
    biases: list                        # per layer [out] float32
    bin_centre: np.ndarray              # [B] float32
    # per model
    kv_bytes_per_token: np.ndarray      # [K] float32 (alpha)
    decode_s_per_token: np.ndarray      # [K] float32
    # nodes
    free_bytes: np.ndarray              # [M] float64
    queue_s: np.ndarray                 # [M] float32
    cold_s: np.ndarray                  # [M] float32
    resident_mask: np.ndarray           # [M] uint64, bit m set <=> model m resident
    # workflows (prioritize); empty when the batch has no chains
    chain_offset: np.ndarray = field(default_factory=lambda: np.zeros(1, np.int64))
    deadline_us: np.ndarray = field(default_factory=lambda: np.zeros(0, np.int64))
    now_us: int = 0

    @property
    def n(self) -> int:
        return int(self.model_id.shape[0])

    @property
    def n_workflows(self) -> int:
        return int(self.chain_offset.shape[0] - 1)

    def sha256(self) -> Dict[str, str]:
        out = {}
        for f in dataclasses.fields(self):
            v = getattr(self, f.name)
            if isinstance(v, np.ndarray):
                out[f.name] = hashlib.sha256(np.ascontiguousarray(v).tobytes()).hexdigest()
            elif isinstance(v, list):
                h = hashlib.sha256()
                for a in v:
                    h.update(np.ascontiguousarray(a).tobytes())
                out[f.name] = h.hexdigest()
        return out


def _seeds(seed: int) -> Dict[str, np.random.SeedSequence]:
    children = np.random.SeedSequence(seed).spawn(len(STREAMS))
    return dict(zip(STREAMS, children))


def _streams(seed: int) -> Dict[str, np.random.Generator]:
    return {name: np.random.Generator(np.random.PCG64(c)) for name, c in _seeds(seed).items()}


def _model_ids(rng: np.random.Generator, n: int, k: int, zipf_s: Optional[float]) -> np.ndarray:
    if zipf_s is None:
        return rng.integers(0, k, size=n, dtype=np.int64).astype(np.int32)
    # truncated Zipf over ids 0..k-1, id 0 the most popular
    p = np.arange(1, k + 1, dtype=np.float64) ** (-zipf_s)
    p /= p.sum()
    return rng.choice(k, size=n, p=p).astype(np.int32)


def _bf16_bits_fast(block: np.ndarray) -> np.ndarray:
    """Same rounding as f32_to_bf16_bits (nearest, ties to even), via PyTorch's multithreaded
    CPU cast; used only for the large feature matrices."""
    import torch
    t = torch.from_numpy(np.ascontiguousarray(block, dtype=np.float32)).to(torch.bfloat16)
    return t.view(torch.int16).numpy().view(np.uint16)


def draw_features(seq: np.random.SeedSequence, n: int, d: int, dtype: str) -> np.ndarray:
    """N(0, 1) features, row chunk c drawn from its own child stream seq.spawn(...)[c] so that
    chunks can be drawn in parallel threads (numpy releases the GIL while drawing)."""
    out = np.empty((n, d), dtype=np.float32 if dtype == "f32" else np.uint16)
    starts = list(range(0, n, _X_CHUNK_ROWS))
    kids = seq.spawn(len(starts))

    def fill(c):
        r0 = starts[c]
        r1 = min(n, r0 + _X_CHUNK_ROWS)
        block = np.random.Generator(np.random.PCG64(kids[c])).standard_normal((r1 - r0, d), dtype=np.float32)
        out[r0:r1] = block if dtype == "f32" else _bf16_bits_fast(block)

    if len(starts) <= 1:
        for c in range(len(starts)):
            fill(c)
    else:
        from concurrent.futures import ThreadPoolExecutor
        with ThreadPoolExecutor(max_workers=min(16, os.cpu_count() or 1)) as ex:
            list(ex.map(fill, range(len(starts))))
    return out


def generate(spec: WorkloadSpec, with_x: bool = True) -> Workload:
    """Draw every input of ``spec``. ``with_x=False`` skips the (large) feature matrix."""
    seeds = _seeds(spec.seed)
    rs = {name: np.random.Generator(np.random.PCG64(c)) for name, c in seeds.items()}
    K, M = spec.n_models, spec.n_nodes

    # workflows first: they fix the number of stages
    if spec.n_workflows > 0:
        W = spec.n_workflows
        lo, hi = spec.chain_len
        lens = rs["chain_len"].integers(lo, hi + 1, size=W, dtype=np.int64)
        chain_offset = np.zeros(W + 1, dtype=np.int64)
        np.cumsum(lens, out=chain_offset[1:])
        n = int(chain_offset[-1])
        arrival = rs["arrival"].uniform(spec.arrival_s[0], spec.arrival_s[1], size=W)
        slo = rs["slo"].uniform(spec.slo_s[0], spec.slo_s[1], size=W)
        deadline_us = np.rint((arrival + slo) * 1.0e6).astype(np.int64)
        now_us = int(round(spec.now_s * 1.0e6))
        # role id cycles along each chain (planner/solver/critic-style); metadata only
        pos = np.arange(n, dtype=np.int64) - np.repeat(chain_offset[:-1], lens)
        role = (pos % 5).astype(np.int32)
    else:
        n = spec.n_stages
        chain_offset = np.zeros(1, dtype=np.int64)
        deadline_us = np.zeros(0, dtype=np.int64)
        now_us = 0
        role = rs["role"].integers(0, 5, size=n, dtype=np.int64).astype(np.int32)

    D = spec.dims[0]
    x = draw_features(seeds["x"], n, D, spec.dtype) if with_x else None

    mu, sigma, plo, phi = spec.prompt_lognormal
    prompt = np.clip(np.rint(rs["prompt"].lognormal(mu, sigma, size=n)), plo, phi).astype(np.int32)
    model = _model_ids(rs["model"], n, K, spec.zipf_s)

    weights, biases = [], []
    for li in range(spec.n_layers):
        fan_in, fan_out = spec.dims[li], spec.dims[li + 1]
        w = rs[("W1", "W2", "W3")[li]].normal(0.0, fan_in ** -0.5, size=(fan_out, fan_in))
        w32 = w.astype(np.float32)
        weights.append(w32 if spec.dtype == "f32" else f32_to_bf16_bits(w32))
        biases.append(np.zeros(fan_out, dtype=np.float32))
    B = spec.n_bins
    bin_centre = (spec.bin_start + spec.bin_width * np.arange(B, dtype=np.float64)).astype(np.float32)

    if spec.alpha[0] == "const":
        alpha = np.full(K, spec.alpha[1], dtype=np.float32)
    else:
        alpha = rs["alpha"].choice(np.asarray(spec.alpha[1:], dtype=np.float64), size=K).astype(np.float32)
    if spec.dec[0] == "const":
        dec = np.full(K, spec.dec[1], dtype=np.float32)
    else:
        dec = rs["dec"].uniform(spec.dec[1], spec.dec[2], size=K).astype(np.float32)

    if spec.free_gb[0] == "uniform":
        free = rs["free"].uniform(spec.free_gb[1], spec.free_gb[2], size=M) * GB
    else:
        _, lo1, hi1, lo2, hi2 = spec.free_gb
        low_half = np.zeros(M, dtype=bool)
        low_half[rs["half"].permutation(M)[: M // 2]] = True
        u = rs["free"].random(size=M)
        free = np.where(low_half, lo1 + u * (hi1 - lo1), lo2 + u * (hi2 - lo2)) * GB
    free = free.astype(np.float64)

    bits = rs["resident"].random(size=(M, K)) < spec.resident_p
    mask = np.zeros(M, dtype=np.uint64)
    for m in range(K):
        mask |= bits[:, m].astype(np.uint64) << np.uint64(m)

    cold = rs["cold"].uniform(spec.cold_s[0], spec.cold_s[1], size=M).astype(np.float32)
    queue = rs["queue"].uniform(spec.queue_s[0], spec.queue_s[1], size=M).astype(np.float32)

    return Workload(spec=spec, x=x, role=role, prompt_len=prompt, model_id=model,
                    weights=weights, biases=biases, bin_centre=bin_centre,
                    kv_bytes_per_token=alpha, decode_s_per_token=dec,
                    free_bytes=free, queue_s=queue, cold_s=cold, resident_mask=mask,
                    chain_offset=chain_offset, deadline_us=deadline_us, now_us=now_us)


# ---------------------------------------------------------------------------------------------
# Extra inputs of routing by fitness (Eq. 5), drawn for an existing Workload
# ---------------------------------------------------------------------------------------------

FITNESS_STREAMS = ("cluster", "src", "class", "rtt", "deg", "rtt_window", "ready_window",
                   "ready_window_cold", "deg_window")

N_CLUSTERS = 5            # three local and two remote clusters, as in the paper's simulator
N_LOCAL = 3
WINDOW = 4096             # recent observations per normalised metric


@dataclass
class FitnessInputs:
    """Per-stage source and class, per-node metrics in milliseconds, the source x node RTT
    matrix, per-class weights (gamma, lambda, mu) and windows of recent observations from
    which the normalisation bounds are taken."""
    src_id: np.ndarray            # [N] int32 source cluster of each stage
    class_id: np.ndarray          # [N] int32: 0 interactive, 1 background
    queue_ms: np.ndarray          # [M] float32 queueing delay T_q
    act_ms: np.ndarray            # [M] float32 activation latency T_act (model not resident)
    deg_ms: np.ndarray            # [M] float32 disruption penalty C_deg
    rtt_ms: np.ndarray            # [N_CLUSTERS][M] float32
    class_weights: np.ndarray     # [2][3] float32
    rtt_window: np.ndarray        # [WINDOW] float32
    ready_window: np.ndarray      # [WINDOW] float32
    deg_window: np.ndarray        # [WINDOW] float32


def _rtt_draw(rng: np.random.Generator, a: np.ndarray, b: np.ndarray) -> np.ndarray:
    """RTT in ms between source cluster a and node cluster b: same cluster U[0.2, 1],
    both local U[1, 5], across regions U[20, 80]."""
    same = a == b
    both_local = (a < N_LOCAL) & (b < N_LOCAL)
    lo = np.where(same, 0.2, np.where(both_local, 1.0, 20.0))
    hi = np.where(same, 1.0, np.where(both_local, 5.0, 80.0))
    return rng.uniform(lo, hi).astype(np.float32)


def fitness_inputs(wl: Workload) -> FitnessInputs:
    """Fitness-routing inputs for the stages and nodes of ``wl`` (seeded by its spec's seed).

    Nodes are spread uniformly over the clusters; 30% of stages are interactive; class weights
    are (gamma, lambda, mu) = (0.25, 1, 1) for interactive stages -- the paper's latency weight
    and default lambda = mu = 1 -- and (0.1, 1, 1) for background ones; the queueing delay and
    activation latency are the workload's own (in ms); 20% of nodes report a disruption penalty
    U[1, 500] ms. Windows hold recent observations of each metric from the same distributions."""
    children = np.random.SeedSequence([wl.spec.seed, 0xF17]).spawn(len(FITNESS_STREAMS))
    r = {name: np.random.Generator(np.random.PCG64(c)) for name, c in zip(FITNESS_STREAMS, children)}
    M, N = wl.free_bytes.shape[0], wl.n
    cluster = r["cluster"].integers(0, N_CLUSTERS, M)
    src = r["src"].integers(0, N_CLUSTERS, N).astype(np.int32)
    cls = (r["class"].random(N) >= 0.3).astype(np.int32)
    rtt = _rtt_draw(r["rtt"], np.arange(N_CLUSTERS)[:, None], cluster[None, :])
    deg = np.where(r["deg"].random(M) < 0.2, r["deg"].uniform(1.0, 500.0, M), 0.0).astype(np.float32)
    wa = r["rtt_window"].integers(0, N_CLUSTERS, WINDOW)
    wb = r["rtt_window"].integers(0, N_CLUSTERS, WINDOW)
    rtt_window = _rtt_draw(r["rtt_window"], wa, wb)
    ready_window = (r["ready_window"].uniform(0.0, 5000.0, WINDOW)
                    + np.where(r["ready_window_cold"].random(WINDOW) < 0.7,
                               r["ready_window_cold"].uniform(2000.0, 20000.0, WINDOW), 0.0)).astype(np.float32)
    deg_window = np.where(r["deg_window"].random(WINDOW) < 0.2,
                          r["deg_window"].uniform(1.0, 500.0, WINDOW), 0.0).astype(np.float32)
    weights = np.array([[0.25, 1.0, 1.0], [0.1, 1.0, 1.0]], np.float32)
    return FitnessInputs(src_id=src, class_id=cls,
                         queue_ms=(wl.queue_s * np.float32(1000.0)).astype(np.float32),
                         act_ms=(wl.cold_s * np.float32(1000.0)).astype(np.float32),
                         deg_ms=deg, rtt_ms=rtt, class_weights=weights, rtt_window=rtt_window,
                         ready_window=ready_window, deg_window=deg_window)


ENGINE_STREAMS = ("count", "level", "size", "kv", "cost", "deg_window")
# levels of Alg. 2's actions: 1 put an idle-running model to sleep, 2 evict a sleeping model,
# 3 stop a pending sleep, 4 swap out an active model's KV, 5 abort an active execution
ENGINE_LEVEL_P = (0.30, 0.20, 0.10, 0.25, 0.15)
HOST_BW = 25e9           # bytes/s, host <-> GPU reload bandwidth of the stand-in cost model
C_INT_MS = 2000.0        # interrupt penalty: an interactive SLO threshold (ms)


@dataclass
class EngineInputs:
    """The resident engines of every node (CSR over nodes) with the action Alg. 2 would take
    on each, the bytes it frees and its restoration cost, plus c_int and a window of recent
    C_deg reports."""
    engine_offset: np.ndarray     # [M + 1] int32
    level: np.ndarray             # [E] int32 in 1..5
    freed_bytes: np.ndarray       # [E] float64
    cost_ms: np.ndarray           # [E] float32
    c_int_ms: float
    deg_window: np.ndarray        # [WINDOW] float32


def engine_inputs(wl: Workload, max_engines: int = 8, crowded: float = 0.1, max_crowded: int = 20) -> EngineInputs:
    """Stand-in engine lists for the nodes of ``wl`` (seeded by its spec's seed).

    Each node hosts U{0..max_engines} engines, except a fraction ``crowded`` of nodes packed
    with many small models, which host U{max_engines+1..max_crowded}; the action level is drawn
    with probabilities
    ENGINE_LEVEL_P. Model sizes are bf16 weights of 0.6B-14B parameters (1.2-28 GB). Freed
    bytes: the weights for levels 1 and 3, the retained runtime context (194-286 MB, the
    paper's measured range) for level 2, the KV in use (U[1, 40] GB) for levels 4 and 5. Cost
    (ms): reloading from host at HOST_BW for levels 1-3 (plus U[0.5, 3] s of context rebuild
    for level 2), the KV reload at HOST_BW for level 4, and U[1, 10] s of KV regeneration for
    level 5. The C_deg window is 80% zeros (stages that fit) and 20% U[100, 30000] ms."""
    children = np.random.SeedSequence([wl.spec.seed, 0xDE6]).spawn(len(ENGINE_STREAMS))
    r = {name: np.random.Generator(np.random.PCG64(c)) for name, c in zip(ENGINE_STREAMS, children)}
    M = wl.free_bytes.shape[0]
    count = np.where(r["count"].random(M) < crowded, r["count"].integers(max_engines + 1, max_crowded + 1, M),
                     r["count"].integers(0, max_engines + 1, M))
    offset = np.zeros(M + 1, np.int32)
    np.cumsum(count, out=offset[1:])
    E = int(offset[-1])
    level = (r["level"].choice(5, size=E, p=ENGINE_LEVEL_P) + 1).astype(np.int32)
    weights = r["size"].uniform(0.6e9, 14e9, E) * 2.0
    ctx = r["size"].uniform(194e6, 286e6, E)
    kv = r["kv"].uniform(1e9, 40e9, E)
    freed = np.where((level == 1) | (level == 3), weights, np.where(level == 2, ctx, kv))
    reload_ms = np.where(level <= 3, weights, kv) / HOST_BW * 1e3
    extra_ms = np.where(level == 2, r["cost"].uniform(500.0, 3000.0, E), 0.0)
    cost = np.where(level == 5, r["cost"].uniform(1000.0, 10000.0, E), reload_ms + extra_ms)
    deg_window = np.where(r["deg_window"].random(WINDOW) < 0.2,
                          r["deg_window"].uniform(100.0, 30000.0, WINDOW), 0.0).astype(np.float32)
    return EngineInputs(engine_offset=offset, level=level, freed_bytes=freed.astype(np.float64),
                        cost_ms=cost.astype(np.float32), c_int_ms=C_INT_MS, deg_window=deg_window)


def margin_window(seed: int, m: int = 4096) -> Tuple[np.ndarray, np.ndarray]:
    """A window of m recent stages' (actual, predicted) KV bytes for the adaptive margin:
    predictions U[1, 100] GB, actual = prediction x lognormal(-0.05, 0.25) (about 40% of the
    stages underestimated, by up to ~2x)."""
    r = np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, 0x4A0])))
    pred = r.uniform(1.0, 100.0, m) * GB
    actual = pred * r.lognormal(-0.05, 0.25, m)
    return actual, pred


READINESS_STREAMS = ("tier", "size")
# readiness tiers (Sec. III-C): 0 Running, 1 Sleeping, 2 CPU-resident, 3 Disk-resident, 4 Remote
TIER_P = (0.3, 0.3, 0.3, 0.1)               # tiers 1..4 of a model that is not running on a node
TIER_BW = (1.0, 25e9, 25e9, 3e9, 1.25e9)    # bytes/s: host link, host link, NVMe, network
TIER_SETUP_MS = (0.0, 150.0, 2500.0, 2500.0, 4000.0)


@dataclass
class ReadinessInputs:
    """Per-(node, model) readiness tier and the profiled bandwidth model T_act = Size / BW_tier."""
    tier: np.ndarray              # [M][K] uint8
    model_bytes: np.ndarray       # [K] float64
    tier_bw: np.ndarray           # [5] float64
    tier_setup_ms: np.ndarray     # [5] float32


def readiness_inputs(wl: Workload) -> ReadinessInputs:
    """Readiness tiers for ``wl`` (seeded by its spec's seed): a model resident on a node (the
    workload's residency bits) is Running there; otherwise Sleeping, CPU-resident, Disk-resident
    or Remote with probabilities TIER_P. Model sizes are bf16 weights of 0.6B-14B parameters
    (1.2-28 GB). Tiers load over a 25 GB/s host link (Sleeping keeps its runtime context: 150 ms
    setup; CPU-resident rebuilds it: 2.5 s), 3 GB/s NVMe (2.5 s) and a 1.25 GB/s network (4 s)."""
    children = np.random.SeedSequence([wl.spec.seed, 0x7E1]).spawn(len(READINESS_STREAMS))
    r = {name: np.random.Generator(np.random.PCG64(c)) for name, c in zip(READINESS_STREAMS, children)}
    M, K = wl.free_bytes.shape[0], wl.spec.n_models
    bits = (wl.resident_mask[:, None] >> np.arange(K, dtype=np.uint64)[None, :]) & np.uint64(1)
    cold = (r["tier"].choice(4, size=(M, K), p=TIER_P) + 1).astype(np.uint8)
    tier = np.where(bits == 1, 0, cold).astype(np.uint8)
    size = r["size"].uniform(0.6e9, 14e9, K) * 2.0
    return ReadinessInputs(tier=tier, model_bytes=size, tier_bw=np.array(TIER_BW, np.float64),
                           tier_setup_ms=np.array(TIER_SETUP_MS, np.float32))


TWO_PHASE_STREAMS = ("head", "head_bias", "coef", "iso", "tools")


@dataclass
class TwoPhaseInputs:
    """Stand-in weights of the two-phase predictor's heads (the last layer of the workload's
    network, read as heads) and its per-stage inputs."""
    head_weight: np.ndarray       # [B][H] float32 or uint16 (bf16 bits): row 0 tool intent, g >= 1 length heads
    head_bias: np.ndarray         # [B] float32
    role_head: np.ndarray         # [n_roles] int32
    tool_coef: np.ndarray         # [B] float32
    iso_x: np.ndarray             # [K] float32, strictly increasing
    iso_y: np.ndarray             # [K] float32, non-decreasing
    max_len: float
    tool_avail: np.ndarray        # [N] int32


def two_phase_inputs(wl: Workload, n_knots: int = 16, max_len: float = 32768.0) -> TwoPhaseInputs:
    """Two-phase predictor inputs for ``wl`` (seeded by its spec's seed).

    Heads: row 0 (tool intent) N(0, 1/H) weights and bias 0; rows g >= 1 (log(1 + L)
    regressors) N(0, 1/H) weights and biases U[4.5, 6.5] (outputs of e^4.5 - e^6.5 tokens
    before the feature terms). Roles 0, 1, 2 have their own heads (2, 3, 4); the others use the
    shared head 1. The tool probability shortens the prediction: coefficients U[-2.5, -1.5].
    The calibration map has n_knots knots from 0 to 1 with sorted uniform values. 60% of stages
    have tools available."""
    children = np.random.SeedSequence([wl.spec.seed, 0x2FA5E]).spawn(len(TWO_PHASE_STREAMS))
    r = {name: np.random.Generator(np.random.PCG64(c)) for name, c in zip(TWO_PHASE_STREAMS, children)}
    B, H = wl.weights[-1].shape
    w = r["head"].normal(0.0, H ** -0.5, size=(B, H)).astype(np.float32)
    bias = np.zeros(B, np.float32)
    bias[1:] = r["head_bias"].uniform(4.5, 6.5, B - 1)
    coef = np.zeros(B, np.float32)
    coef[1:] = r["coef"].uniform(-2.5, -1.5, B - 1)
    x = np.concatenate([[0.0], np.sort(r["iso"].uniform(0.0, 1.0, n_knots - 2)), [1.0]]).astype(np.float32)
    y = np.sort(r["iso"].uniform(0.0, 1.0, n_knots)).astype(np.float32)
    tools = (r["tools"].random(wl.n) < 0.6).astype(np.int32)
    return TwoPhaseInputs(head_weight=w if wl.spec.dtype == "f32" else f32_to_bf16_bits(w), head_bias=bias,
                          role_head=np.array([2, 3, 4], np.int32), tool_coef=coef, iso_x=x, iso_y=y,
                          max_len=max_len, tool_avail=tools)


ROLE_STREAMS = ("w1", "w2", "w3", "bias", "coef")


@dataclass
class RoleRegressorInputs:
    """Stand-in weights of per-role length regressors: G networks of the workload predictor's
    shape, stacked [G][out][in], and the role -> regressor map."""
    weights: list                 # per layer [G][out][in], float32 or uint16 (bf16 bits)
    biases: list                  # per layer [G][out] float32
    role_group: np.ndarray        # [n_roles] int32, -1 = the shared model
    tool_coef: np.ndarray         # [G] float32
    max_len: float


def role_regressor_inputs(wl: Workload, max_len: float = 32768.0) -> RoleRegressorInputs:
    """Per-role regressors for ``wl`` (seeded by its spec's seed): roles 0, 1 and 2 of the five
    have regressors of their own (0, 1, 2); roles 3 and 4 keep the shared model. Each regressor
    is a network of the predictor's shape with N(0, 1/fan_in) weights and zero hidden biases;
    output 0 regresses log(1 + L) (bias U[4.5, 6.5], e^4.5 - e^6.5 tokens before the feature
    terms) and the other outputs are zero. Tool coefficients U[-2.5, -1.5]: tool-invoking stages
    produce short structured outputs (Sec. III-B)."""
    children = np.random.SeedSequence([wl.spec.seed, 0x201E5]).spawn(len(ROLE_STREAMS))
    r = {name: np.random.Generator(np.random.PCG64(c)) for name, c in zip(ROLE_STREAMS, children)}
    G = 3
    dims = wl.spec.dims
    ws, bs = [], []
    for l, key in enumerate(("w1", "w2", "w3")):
        din, dout = dims[l], dims[l + 1]
        w = r[key].normal(0.0, din ** -0.5, size=(G, dout, din)).astype(np.float32)
        b = np.zeros((G, dout), np.float32)
        if l == len(dims) - 2:
            w[:, 1:, :] = 0.0
            b[:, 0] = r["bias"].uniform(4.5, 6.5, G)
        ws.append(w if wl.spec.dtype == "f32" else f32_to_bf16_bits(w))
        bs.append(b)
    coef = r["coef"].uniform(-2.5, -1.5, G).astype(np.float32)
    return RoleRegressorInputs(weights=ws, biases=bs, role_group=np.array([0, 1, 2, -1, -1], np.int32),
                               tool_coef=coef, max_len=max_len)


def workload(name: str, with_x: bool = True, **overrides) -> Workload:
    """Named workload, optionally with fields of its spec replaced (e.g. ``n_stages=5000``)."""
    spec = SPECS[name]
    if overrides:
        spec = dataclasses.replace(spec, **overrides)
    return generate(spec, with_x=with_x)
