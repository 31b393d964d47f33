"""Host-side checks of the Python binding, without a GPU: the kernels index every array by the
sizes a call passes, so the binding checks each tensor's shape against them before the C-ABI
call (a short output tensor would otherwise be written past its end). CPU tensors stand in for
device tensors and a recording stub stands in for the library, so nothing is ever launched."""
import pytest
import torch

from paper_2606_12950_amd import _native


class _StubLib:
    """Records the entry points called; workspace queries report 0 bytes."""

    def __init__(self):
        self.calls = []

    def __getattr__(self, name):
        if name.endswith("_workspace"):
            return lambda *args: 0

        def entry(*args):
            self.calls.append(name)
            return 0
        return entry


@pytest.fixture
def stub(monkeypatch):
    lib = _StubLib()
    monkeypatch.setattr(_native, "_lib", lib)

    def dev(t, name, dtype):   # the real check minus the device test
        if t.dtype != dtype:
            raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
        if not t.is_contiguous():
            raise ValueError(f"{name} must be contiguous")
        return t
    monkeypatch.setattr(_native, "_dev", dev)
    monkeypatch.setattr(_native, "_stream", lambda s: None)
    return lib


def _e(*shape, dtype=torch.float32):
    return torch.zeros(shape, dtype=dtype)


N, M, K, k = 10, 6, 3, 2


def _predict_args():
    ws = [_e(8, 4), _e(5, 8)]
    bs = [_e(8), _e(5)]
    return dict(x=_e(N, 4), weights=ws, biases=bs, bin_centre=_e(5), prompt_len=_e(N, dtype=torch.int32),
                model_id=_e(N, dtype=torch.int32), kv_bytes_per_token=_e(K))


def test_predict_shapes(stub):
    _native.predict(**_predict_args())
    assert stub.calls == ["maestro_predict"]
    for bad in ((_e(N - 1), _e(N, dtype=torch.float64)), (_e(N), _e(N + 1, dtype=torch.float64))):
        with pytest.raises(ValueError):
            _native.predict(**_predict_args(), out=bad)
    a = _predict_args()
    a["model_id"] = _e(N - 1, dtype=torch.int32)
    with pytest.raises(ValueError):
        _native.predict(**a)
    assert stub.calls == ["maestro_predict"]


def test_predict_two_phase_shapes(stub):
    a = _predict_args()
    del a["bin_centre"]
    a.update(role_head=_e(4, dtype=torch.int32), tool_coef=_e(5), iso_x=_e(3), iso_y=_e(3), max_len=100.0,
             role_id=_e(N, dtype=torch.int32), tool_avail=_e(N, dtype=torch.int32))
    _native.predict_two_phase(**a)
    _native.predict_two_phase(**a, out=(None, _e(N), _e(N, dtype=torch.float64)))   # no p_tool output
    assert stub.calls == ["maestro_predict_two_phase"] * 2
    with pytest.raises(ValueError):
        _native.predict_two_phase(**a, out=(_e(N - 1), _e(N), _e(N, dtype=torch.float64)))
    assert len(stub.calls) == 2


def _route_args():
    return (_e(N, dtype=torch.int32), _e(N), _e(N, dtype=torch.float64), _e(K), _e(M, dtype=torch.float64), _e(M),
            _e(M), _e(M, dtype=torch.int64))


def test_route_shapes(stub):
    _native.route(*_route_args(), k=k)
    _native.route(*_route_args()[:6], None, None, k=k, act_s=_e(M, K))
    assert stub.calls == ["maestro_route_ex", "maestro_route_tiered"]
    for out in ((_e(N, k + 1, dtype=torch.int32), _e(N, k)), (_e(N, k, dtype=torch.int32), _e(N - 1, k))):
        with pytest.raises(ValueError):
            _native.route(*_route_args(), k=k, out=out)
    with pytest.raises(TypeError):   # a workspace counts bytes: it must be uint8
        _native.route(*_route_args(), k=k, workspace=_e(64))
    args = list(_route_args())
    args[6] = _e(M - 1)              # cold_s one node short
    with pytest.raises(ValueError):
        _native.route(*args, k=k)
    assert len(stub.calls) == 2


def _fitness_kwargs():
    return dict(model_id=_e(N, dtype=torch.int32), src_id=_e(N, dtype=torch.int32), class_id=_e(N, dtype=torch.int32),
                kv_bytes=_e(N, dtype=torch.float64), free_bytes=_e(M, dtype=torch.float64), queue_ms=_e(M),
                act_ms=_e(M), resident_mask=_e(M, dtype=torch.int64), deg_ms=_e(M), rtt_ms=_e(2, M),
                class_weights=_e(2, 3), bounds=_e(6), n_models=K, k=k)


def test_route_fitness_shapes(stub):
    _native.route_fitness(**_fitness_kwargs())
    assert stub.calls == ["maestro_route_fitness"]
    with pytest.raises(ValueError):
        _native.route_fitness(**_fitness_kwargs(), out=(_e(N, k, dtype=torch.int32), _e(N, 1)))
    bad = _fitness_kwargs()
    bad["deg_ms"] = _e(M + 1)
    with pytest.raises(ValueError):
        _native.route_fitness(**bad)
    assert len(stub.calls) == 1


def test_small_entry_points_shapes(stub):
    _native.adaptive_rho(_e(N, dtype=torch.float64), _e(N, dtype=torch.float64), 0.2, 0.9)
    _native.quantiles(_e(N))
    _native.activation_latency(_e(M, K, dtype=torch.uint8), _e(K, dtype=torch.float64), _e(5, dtype=torch.float64),
                               _e(5))
    assert len(stub.calls) == 3
    with pytest.raises(ValueError):
        _native.adaptive_rho(_e(N, dtype=torch.float64), _e(N, dtype=torch.float64), 0.2, 0.9,
                             out=(_e(N - 1), _e(1)))
    with pytest.raises(ValueError):
        _native.quantiles(_e(N), out=_e(1))
    with pytest.raises(ValueError):
        _native.activation_latency(_e(M, K, dtype=torch.uint8), _e(K, dtype=torch.float64),
                                   _e(5, dtype=torch.float64), _e(5), out=_e(M, K - 1))
    assert len(stub.calls) == 3


def test_prioritize_shapes(stub):
    W, S = 4, 9
    off = torch.tensor([0, 2, 5, 5, 9], dtype=torch.int64)
    args = (off, _e(S), _e(W, dtype=torch.int64), 0)
    _native.prioritize(*args)
    _native.prioritize(*args, want_remaining=False)
    assert stub.calls == ["maestro_prioritize"] * 2
    for out in ((_e(S - 1, dtype=torch.int64), _e(W, dtype=torch.int32), _e(W, dtype=torch.int32)),
                (None, _e(W, dtype=torch.int32), _e(W - 1, dtype=torch.int32)),
                (None, _e(W + 1, dtype=torch.int32), _e(W, dtype=torch.int32))):
        with pytest.raises(ValueError):
            _native.prioritize(*args, out=out)
    with pytest.raises(TypeError):
        _native.prioritize(*args, out=(None, _e(W), _e(W, dtype=torch.int32)))   # keys are int32
    with pytest.raises(ValueError):
        _native.prioritize(*args, cursor=_e(W - 1, dtype=torch.int32))
    assert len(stub.calls) == 2
