"""The sorted route (Sec. III-D; Alg. 3; Eq. 6) in its two halves through the C-ABI:
maestro_route_sort_nodes (every model's nodes in (ready time, index) order, with headroom) and
maestro_route_walk (each stage's k best feasible nodes from its model's list).

Bars: the lists bit-exact against numpy's stable lexicographic sort of the definition's ready
times fl32(T_q + T_act); the walk's node indices and score bits identical to the oracle's route
and to maestro_route_ex with the sorted algorithm, also when one set of lists serves two batches.
Node counts cover every launch shape of the sort (256 .. 8,192 positions, a power of two: 256, 512
or 1,024 threads with 1 key each, then 2, 4 and 8 keys per thread) and non-powers of two.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2606_12950_amd as M
from paper_2606_12950_amd import pipeline

pytestmark = pytest.mark.gpu

GB = 1e9


def _t(a):
    return pipeline._t(np.ascontiguousarray(a), "cuda")


def _nodes(rng, M_, K, coarse=False):
    if coarse:   # many equal ready times: the index must order them
        q = rng.choice(np.array([0.0, 0.5, 1.0], np.float32), M_)
        cold = rng.choice(np.array([2.0, 4.0], np.float32), M_)
    else:
        q = rng.uniform(0, 5, M_).astype(np.float32)
        cold = rng.uniform(1, 20, M_).astype(np.float32)
    mask = rng.integers(0, 2 ** 63, M_, dtype=np.int64).astype(np.uint64) | \
        (rng.integers(0, 2, M_).astype(np.uint64) << np.uint64(63))
    free = rng.uniform(0, 80, M_) * GB
    return free, q, cold, mask


def _lists(buf, K, M_):
    rec = np.dtype([("ready", "<f4"), ("node", "<i4"), ("free", "<f8")])
    return buf[: K * M_ * 16].cpu().numpy().view(rec).reshape(K, M_)


def _expected_lists(free, q, cold, mask, K, act=None):
    M_ = free.shape[0]
    out = []
    for m in range(K):
        if act is None:
            res = ((mask >> np.uint64(m)) & np.uint64(1)) == 1
            ready = np.where(res, q + np.float32(0.0), q + cold).astype(np.float32)
        else:
            ready = (q + act[:, m]).astype(np.float32)
        order = np.lexsort((np.arange(M_), ready))   # ready first, then index
        out.append((ready[order], order.astype(np.int32), free[order]))
    return out


@pytest.mark.parametrize("M_,K", [(1, 1), (37, 16), (64, 3), (65, 64), (700, 16), (1500, 8), (4096, 64),
                                  (5000, 2), (8192, 5)])
def test_sorted_lists_match_definition(M_, K):
    rng = np.random.default_rng(M_ * 7 + K)
    for coarse in (False, True):
        free, q, cold, mask = _nodes(rng, M_, K, coarse)
        lists = M.route_sort_nodes(_t(free), _t(q), _t(cold), _t(mask), K)
        torch.cuda.synchronize()
        # largest headroom per 8 / 64 / 512 entries, rounded up to float32
        blocks = sum((M_ + (1 << b) - 1) >> b for b in (3, 6, 9))
        assert lists.numel() >= M.route_lists_bytes(K, M_) == K * (M_ * 16 + blocks * 4)
        skip = lists[K * M_ * 16: K * (M_ * 16 + blocks * 4)].cpu().numpy().view(np.float32).reshape(K, blocks)
        got = _lists(lists, K, M_)
        for m, (ready, node, fr) in enumerate(_expected_lists(free, q, cold, mask, K)):
            assert np.array_equal(got["ready"][m].view(np.uint32), ready.view(np.uint32)), (m, coarse)
            assert np.array_equal(got["node"][m], node), (m, coarse)
            assert np.array_equal(got["free"][m], fr), (m, coarse)
            for b, off in ((3, 0), (6, (M_ + 7) >> 3), (9, ((M_ + 7) >> 3) + ((M_ + 63) >> 6))):
                nb = (M_ + (1 << b) - 1) >> b
                padded = np.full(nb << b, -np.inf)
                padded[:M_] = fr
                want = padded.reshape(nb, 1 << b).max(axis=1)
                got_b = skip[m, off: off + nb].astype(np.float64)
                # the float32 value at or above the float64 block maximum, and the nearest such
                assert np.all(got_b >= want), (m, b)
                assert np.all((want == -np.inf) | (np.nextafter(got_b.astype(np.float32), np.float32(-np.inf))
                                                   .astype(np.float64) < want)), (m, b)


def test_sorted_lists_readiness_form():
    rng = np.random.default_rng(41)
    M_, K = 2049, 33
    free, q, _, _ = _nodes(rng, M_, K)
    act = rng.choice(np.array([0.0, 0.15, 2.5, 4.0], np.float32), (M_, K))
    lists = M.route_sort_nodes(_t(free), _t(q), None, None, K, act_s=_t(act))
    torch.cuda.synchronize()
    got = _lists(lists, K, M_)
    for m, (ready, node, fr) in enumerate(_expected_lists(free, q, None, None, K, act=act)):
        assert np.array_equal(got["ready"][m].view(np.uint32), ready.view(np.uint32)), m
        assert np.array_equal(got["node"][m], node), m


@pytest.mark.parametrize("n,M_,K,k", [(1, 1, 1, 1), (300, 64, 16, 4), (5000, 700, 64, 3), (40000, 4096, 64, 4),
                                      (20000, 8192, 8, 16), (777, 1500, 5, 1)])
def test_walk_matches_oracle_and_one_call_route(n, M_, K, k):
    rng = np.random.default_rng(n + M_ + K)
    free, q, cold, mask = _nodes(rng, M_, K, coarse=(n % 2 == 0))
    dec = rng.choice(np.array([0.015625, 0.03125, 0.02], np.float32), K)
    lists = M.route_sort_nodes(_t(free), _t(q), _t(cold), _t(mask), K)
    for batch in range(2):   # the same lists serve two batches
        model = rng.integers(0, K, n).astype(np.int32)
        pred = rng.uniform(32, 4064, n).astype(np.float32)
        kv = rng.uniform(0, 60, n) * GB
        rho = 0.2 if batch else 0.0
        gi, gs = M.route_walk(_t(model), _t(pred), _t(kv), _t(dec), M_, lists, k=k, rho=rho)
        oi, os_ = M.route(_t(model), _t(pred), _t(kv), _t(dec), _t(free), _t(q), _t(cold), _t(mask), k=k, rho=rho,
                          algo=M._native.ROUTE_SORTED)
        torch.cuda.synchronize()
        ri, rs = oracle.route(model, pred, kv, dec, free, q, cold, mask, k=k, rho=rho)
        gi, gs = gi.cpu().numpy(), gs.cpu().numpy()
        assert np.array_equal(gi, ri) and np.array_equal(gs.view(np.uint32), rs.view(np.uint32)), batch
        assert np.array_equal(gi, oi.cpu().numpy()) and np.array_equal(gs.view(np.uint32),
                                                                        os_.cpu().numpy().view(np.uint32))


def test_walk_rejects_lists_of_the_wrong_size():
    M_, K = 100, 4
    lists = torch.empty(M.route_lists_bytes(K, M_) - 16, dtype=torch.uint8, device="cuda")
    one = torch.zeros(1, dtype=torch.int32, device="cuda")
    with pytest.raises(M.MaestroError) as e:
        M.route_walk(one, torch.ones(1, device="cuda"), torch.ones(1, dtype=torch.float64, device="cuda"),
                     torch.ones(K, device="cuda"), M_, lists)
    assert e.value.status == 3


@pytest.mark.parametrize("M_,K,k", [(9, 3, 4), (520, 8, 4), (4100, 16, 3), (8192, 4, 16)])
def test_walk_with_few_admitting_nodes(M_, K, k):
    # most nodes admit almost no stage: the walk skips blocks of 8 / 64 / 512 entries whose largest
    # headroom is below the stage's demand; stages that fit nowhere, in one or two nodes only (at
    # any list position, block edges included), and the usual ones; against the oracle and the scan
    rng = np.random.default_rng(M_ + 3 * K + k)
    free, q, cold, mask = _nodes(rng, M_, K)
    free = rng.uniform(0, 1, M_) * GB
    big = rng.choice(M_, min(M_, 5), replace=False)
    free[big] = rng.uniform(40, 80, big.size) * GB
    n = 6000
    model = rng.integers(0, K, n).astype(np.int32)
    pred = rng.uniform(32, 4064, n).astype(np.float32)
    kv = rng.choice(np.array([0.5, 10.0, 60.0, 90.0]), n) * GB      # fits many, a few, one or two, none
    dec = rng.choice(np.array([0.015625, 0.03125, 0.02], np.float32), K)
    lists = M.route_sort_nodes(_t(free), _t(q), _t(cold), _t(mask), K)
    gi, gs = M.route_walk(_t(model), _t(pred), _t(kv), _t(dec), M_, lists, k=k)
    si, ss = M.route(_t(model), _t(pred), _t(kv), _t(dec), _t(free), _t(q), _t(cold), _t(mask), k=k,
                     algo=M._native.ROUTE_SCAN)
    torch.cuda.synchronize()
    ri, rs = oracle.route(model, pred, kv, dec, free, q, cold, mask, k=k)
    gi, gs = gi.cpu().numpy(), gs.cpu().numpy()
    assert (gi[:, 0] < 0).any() and (gi[:, 0] >= 0).any()
    assert np.array_equal(gi, ri) and np.array_equal(gs.view(np.uint32), rs.view(np.uint32))
    assert np.array_equal(gi, si.cpu().numpy()) and np.array_equal(gs.view(np.uint32), ss.cpu().numpy().view(np.uint32))
