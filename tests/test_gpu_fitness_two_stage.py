"""Parity of routing by fitness (Eq. 5, Alg. 3) with the oracle at the batch sizes where each
lane of the kernel takes two stages that share its node reads: from 2^19 stages without
degradation plans, from 2^20 with them (Alg. 2, Eq. 4). Every stage is compared.

The batches are ragged (the last workgroup's second stage row is partly empty), node counts
span several 128-node chunks (32 with 64-model readiness rows) with a ragged tail, and the route
widths 1..4 all take two stages per lane. With plans, one stage class has mu < 0 and one C_deg
window starts below 0: there the bound that drops short pairs before their plan lookup does not
hold and must not be applied.

Between the split-lane sizes and those, each lane takes one stage of its own (and at any size
when the list is longer than four); those launches, with 64-bit residency masks, are compared
here as well.

Bars: node indices and fitness values bit-exact (both sides evaluate the same float32
expression in the same order).
"""
import numpy as np
import pytest

import oracle
from test_gpu_fitness import (GB, TIER_BW, TIER_SETUP, _engines, _nodes, assert_same, gpu_fitness, gpu_fitness_act,
                              gpu_fitness_plans, oracle_fitness, oracle_fitness_act)

pytestmark = pytest.mark.gpu

N_DEG = (1 << 19) + 333      # two stages per lane without plans
N_PLANS = (1 << 20) + 777    # two stages per lane with plans
N_ONE = 200_003              # one lane, one stage (above 2^17, below 2^19)
N_ONE_PLANS = 600_011        # one lane, one stage with plans (below 2^20)


def _stages(rng, n, n_models, n_src, n_cls, kv_gb):
    model = rng.integers(0, n_models, n).astype(np.int32)
    src = rng.integers(0, n_src, n).astype(np.int32)
    cls = rng.integers(0, n_cls, n).astype(np.int32)
    kv = rng.uniform(0, kv_gb, n) * GB
    kv[::41] = 0.0
    return model, src, cls, kv


@pytest.mark.parametrize("k,n_models", [(1, 16), (2, 64), (3, 16), (4, 64)])
def test_two_stage_fitness_matches_oracle(k, n_models):
    rng = np.random.default_rng(100 + 10 * k + n_models)
    M_, n_src = 300, 5
    nodes = _nodes(rng, M_, n_src)
    model, src, cls, kv = _stages(rng, N_DEG, n_models, n_src, 3, 250)
    weights = [[0.25, 1, 1], [0.1, 1, 1], [0.6, 0.3, 2.0]]
    bounds = [*oracle.quantiles(nodes["rtt_ms"].ravel()), *oracle.quantiles(nodes["queue_ms"] + nodes["act_ms"]),
              *oracle.quantiles(nodes["deg_ms"])]
    rho = 0.2 if k == 3 else 0.0
    got = gpu_fitness(model, src, cls, kv, nodes, weights, bounds, k=k, rho=rho, n_models=n_models)
    assert_same(got, oracle_fitness(model, src, cls, kv, nodes, weights, bounds, k=k, rho=rho))


@pytest.mark.parametrize("k,max_e,deg_lo", [(1, 8, 0.0), (4, 30, 0.0), (2, 8, -500.0)])
def test_two_stage_fitness_with_plans_matches_oracle(k, max_e, deg_lo):
    rng = np.random.default_rng(200 + 10 * k + max_e)
    M_, n_src = 200, 4
    nodes = _nodes(rng, M_, n_src)
    nodes["free_bytes"] = rng.uniform(0, 60, M_) * GB
    nodes["free_bytes"][rng.random(M_) < 0.05] = 0.0
    off, level, freed, cost = _engines(rng, M_, max_e=max_e)
    if max_e > 8:
        freed = freed * 0.2
    eng = (off, level, freed, cost, 2000.0)
    model, src, cls, kv = _stages(rng, N_PLANS, 64, n_src, 3, 120)
    # class 2 penalises C_deg negatively (mu < 0): no fitness bound from C_deg = 0 there
    weights = [[0.25, 1, 1], [0.1, 1, 1], [0.5, 0.5, -1.0]]
    bounds = [*oracle.quantiles(nodes["rtt_ms"].ravel()), *oracle.quantiles(nodes["queue_ms"] + nodes["act_ms"]),
              deg_lo, 12000.0]
    got = gpu_fitness_plans(model, src, cls, kv, nodes, weights, bounds, eng, k=k)
    ref = oracle.route_fitness(model, src, cls, kv, nodes["free_bytes"], nodes["queue_ms"], nodes["act_ms"],
                               nodes["resident_mask"], nodes["deg_ms"], nodes["rtt_ms"], np.asarray(weights, np.float32),
                               np.asarray(bounds, np.float32), k=k, engines=eng)
    assert_same(got, ref)
    short = (kv[:, None] > nodes["free_bytes"][None, :]).mean()
    assert short > 0.3, short


@pytest.mark.parametrize("n_models,plans", [(16, False), (64, False), (33, True)])
def test_two_stage_fitness_with_act_matrix_matches_oracle(n_models, plans):
    rng = np.random.default_rng(300 + n_models)
    M_, n_src = 150, 3
    nodes = _nodes(rng, M_, n_src)
    if plans:
        nodes["free_bytes"] = rng.uniform(0, 60, M_) * GB
    tier = rng.integers(0, 5, (M_, n_models)).astype(np.uint8)
    act = oracle.activation_latency(tier, rng.uniform(1, 28, n_models) * GB, TIER_BW, TIER_SETUP)
    eng = None
    if plans:
        off, level, freed, cost = _engines(rng, M_)
        eng = (off, level, freed, cost, 2000.0)
    n = N_PLANS if plans else N_DEG
    model, src, cls, kv = _stages(rng, n, n_models, n_src, 3, 120 if plans else 250)
    weights = [[0.25, 1, 1], [0.1, 1, 1], [1.0, 1.0, 0.0]]
    bounds = [*oracle.quantiles(nodes["rtt_ms"].ravel()),
              *oracle.quantiles((nodes["queue_ms"][:, None] + act).ravel()), 0.0, 12000.0]
    k = 4 if plans else 2
    got = gpu_fitness_act(model, src, cls, kv, nodes, weights, bounds, act, n_models, k=k, eng=eng)
    assert_same(got, oracle_fitness_act(model, src, cls, kv, nodes, weights, bounds, act, n_models, k=k, eng=eng))


@pytest.mark.parametrize("k,n_models", [(1, 64), (4, 64), (8, 33)])
def test_one_stage_per_lane_fitness_matches_oracle(k, n_models):
    rng = np.random.default_rng(400 + 10 * k + n_models)
    M_, n_src = 300, 5
    nodes = _nodes(rng, M_, n_src)
    model, src, cls, kv = _stages(rng, N_ONE, n_models, n_src, 3, 250)
    weights = [[0.25, 1, 1], [0.1, 1, 1], [0.6, 0.3, 2.0]]
    bounds = [*oracle.quantiles(nodes["rtt_ms"].ravel()), *oracle.quantiles(nodes["queue_ms"] + nodes["act_ms"]),
              *oracle.quantiles(nodes["deg_ms"])]
    got = gpu_fitness(model, src, cls, kv, nodes, weights, bounds, k=k, n_models=n_models)
    assert_same(got, oracle_fitness(model, src, cls, kv, nodes, weights, bounds, k=k))


@pytest.mark.parametrize("k", [1, 4])
def test_one_stage_per_lane_fitness_with_plans_matches_oracle(k):
    rng = np.random.default_rng(500 + k)
    M_, n_src = 200, 4
    nodes = _nodes(rng, M_, n_src)
    nodes["free_bytes"] = rng.uniform(0, 60, M_) * GB
    off, level, freed, cost = _engines(rng, M_, max_e=30)
    eng = (off, level, freed * 0.2, cost, 2000.0)
    model, src, cls, kv = _stages(rng, N_ONE_PLANS, 64, n_src, 3, 120)
    weights = [[0.25, 1, 1], [0.1, 1, 1], [0.5, 0.5, -1.0]]
    bounds = [*oracle.quantiles(nodes["rtt_ms"].ravel()), *oracle.quantiles(nodes["queue_ms"] + nodes["act_ms"]),
              0.0, 12000.0]
    got = gpu_fitness_plans(model, src, cls, kv, nodes, weights, bounds, eng, k=k)
    ref = oracle.route_fitness(model, src, cls, kv, nodes["free_bytes"], nodes["queue_ms"], nodes["act_ms"],
                               nodes["resident_mask"], nodes["deg_ms"], nodes["rtt_ms"], np.asarray(weights, np.float32),
                               np.asarray(bounds, np.float32), k=k, engines=eng)
    assert_same(got, ref)
