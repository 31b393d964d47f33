"""The measurement-only matrix-core probe behind bench.py --mfma-ceiling: it runs, is
deterministic for a seed, and its one- and four-accumulator forms sum the same products (the
register-operand form issues the same 16 MFMAs per round either way)."""
import ctypes
import os

import pytest
import torch

from paper_2606_12950_amd import build as B

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def probe():
    if not os.path.exists(B.CALIBRATE_LIB):
        pytest.fail("libmaestro_calibrate.so is not built (python -m paper_2606_12950_amd.build)")
    c = ctypes.CDLL(B.CALIBRATE_LIB)
    c.maestro_calibrate_mfma.argtypes = [ctypes.c_void_p, ctypes.c_int, ctypes.c_int, ctypes.c_int,
                                         ctypes.c_uint32, ctypes.c_void_p]
    c.maestro_calibrate_mfma.restype = ctypes.c_int
    c.maestro_calibrate_mfma_outputs.restype = ctypes.c_int
    torch.cuda.set_device(0)

    def run(rounds, n_acc, lds_every, seed):
        out = torch.full((c.maestro_calibrate_mfma_outputs(),), float("nan"), dtype=torch.float32, device="cuda")
        stream = torch.cuda.current_stream().cuda_stream
        assert c.maestro_calibrate_mfma(ctypes.c_void_p(out.data_ptr()), rounds, n_acc, lds_every, seed,
                                        ctypes.c_void_p(stream)) == 0
        torch.cuda.synchronize()
        return out.cpu()
    return run


@pytest.mark.parametrize("n_acc,lds_every", [(1, 0), (4, 0), (1, 1), (1, 2)])
def test_probe_is_finite_and_deterministic(probe, n_acc, lds_every):
    a = probe(8, n_acc, lds_every, 7)
    b = probe(8, n_acc, lds_every, 7)
    assert torch.isfinite(a).all()
    assert torch.equal(a, b)
    assert not torch.equal(a, probe(8, n_acc, lds_every, 8))


def test_one_and_four_accumulators_sum_the_same_products(probe):
    one, four = probe(4, 1, 0, 11), probe(4, 4, 0, 11)
    scale = float(one.abs().max())
    assert scale > 0
    assert float((one - four).abs().max()) <= 1e-4 * scale
