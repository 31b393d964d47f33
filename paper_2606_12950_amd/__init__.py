"""MI355X (gfx950) hot path of Maestro's scheduler: batched predict -> route -> prioritize.

The computation lives in libmaestro.so (hand-written HIP kernels behind the C-ABI of
include/maestro.h); this package is its thin Python binding plus the seeded workload
generator. PyTorch supplies device memory and streams only.
"""
from ._native import (LIBRARY_PATH, MaestroError, Predictor, TwoPhase, load, make_predictor, predict,
                      predict_two_phase, predict_role_lengths,
                      activation_latency, adaptive_rho, degradation_plans, prioritize, prioritize_workspace_bytes, quantiles, route,
                      route_fitness, route_lists_bytes, route_sort_nodes, route_walk)
from .pipeline import DeviceBatch, StepOutputs, run_step, to_device

__all__ = ["LIBRARY_PATH", "MaestroError", "Predictor", "TwoPhase", "load", "make_predictor", "predict",
           "predict_two_phase", "predict_role_lengths", "activation_latency", "adaptive_rho", "degradation_plans",
           "prioritize", "prioritize_workspace_bytes", "quantiles", "route", "route_fitness", "route_lists_bytes",
           "route_sort_nodes", "route_walk",
           "DeviceBatch", "StepOutputs",
           "run_step", "to_device"]
