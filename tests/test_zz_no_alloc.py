"""The allocation-free slack ordering (maestro_prioritize_noalloc, static scratch) against the
workspace form (maestro_prioritize) through the C-ABI: two calls in a row on the same GPU, the
second with a smaller batch (the static scratch keeps the first call's contents), remaining
times, keys and orders bit for bit; the largest batch it takes and the first one beyond it."""
import numpy as np
import pytest
import torch

import paper_2606_12950_amd as M
from paper_2606_12950_amd import _native, pipeline

pytestmark = pytest.mark.gpu


def _chains(rng, W, max_len=8):
    lens = rng.integers(1, max_len + 1, W)
    off = np.zeros(W + 1, np.int64)
    np.cumsum(lens, out=off[1:])
    lat = rng.uniform(0.0, 30.0, int(off[-1])).astype(np.float32)
    lat[rng.random(lat.size) < 1e-3] = np.inf
    deadline = rng.integers(0, 10**9, W).astype(np.int64)
    return off, lat, deadline


def _run(off, lat, deadline, noalloc):
    t = lambda a: pipeline._t(np.ascontiguousarray(a), "cuda")
    co, la, dl = t(off), t(lat), t(deadline)
    W, S = deadline.size, lat.size
    out = (torch.full((S,), -1, dtype=torch.int64, device="cuda"), torch.full((W,), -1, dtype=torch.int32, device="cuda"),
           torch.full((W,), -1, dtype=torch.int32, device="cuda"))
    rem, key, order = M.prioritize(co, la, dl, 5 * 10**8, out=out, noalloc=noalloc)
    torch.cuda.synchronize()
    return rem.cpu().numpy(), key.cpu().numpy(), order.cpu().numpy()


def _same(a, b):
    for x, y in zip(a, b):
        assert np.array_equal(x, y)


def test_noalloc_matches_workspace_form_twice_then_smaller():
    rng = np.random.default_rng(71)
    # 300,000 workflows: the large-batch sort path; then 5,000: the small-tile path, over
    # scratch that still holds the first call's buffers
    for W in (300_000, 5_000):
        off, lat, dl = _chains(rng, W)
        print(f"noalloc W={W} S={lat.size}", flush=True)
        _same(_run(off, lat, dl, True), _run(off, lat, dl, False))


def test_noalloc_largest_batch_and_limit():
    rng = np.random.default_rng(72)
    W = _native.PRIORITIZE_NOALLOC_MAX_WORKFLOWS
    off, lat, dl = _chains(rng, W, max_len=3)
    print(f"noalloc W={W} S={lat.size}", flush=True)
    _same(_run(off, lat, dl, True), _run(off, lat, dl, False))
    off, lat, dl = _chains(rng, W + 1, max_len=1)
    with pytest.raises(_native.MaestroError, match="workspace"):
        _run(off, lat, dl, True)
    _same(_run(off[:1], lat[:0], dl[:0], True), _run(off[:1], lat[:0], dl[:0], False))   # empty: no-op
