"""The C-ABI library loads, exports every symbol the header declares, and rejects bad
arguments on the host before anything is launched (no GPU needed: none of these calls reach
a kernel)."""
import ctypes
import os
import re

import pytest

import paper_2606_12950_amd as M
from paper_2606_12950_amd import _native

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "maestro.h")

OK, INVALID, UNSUPPORTED, WORKSPACE = 0, 1, 2, 3


def declared_functions():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"MAESTRO_API\s+[\w\s\*]+?\b(maestro_\w+)\s*\(", text)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(M.LIBRARY_PATH):
        pytest.fail("libmaestro.so is not built (python -m paper_2606_12950_amd.build)")
    return M.load()


def test_every_declared_symbol_is_exported(lib):
    names = declared_functions()
    assert len(names) == 22
    assert sorted(_native.EXPORTS) == names
    for n in names:
        assert hasattr(lib, n), n


def test_status_strings(lib):
    assert lib.maestro_status_string(0) == b"ok"
    assert lib.maestro_status_string(2) == b"unsupported shape"
    assert lib.maestro_status_string(99) == b"unknown status"


# Host addresses that are valid-looking (non-null, aligned) but never dereferenced: every call
# below fails validation before any launch.
_buf = (ctypes.c_double * 64)()
FAKE = ctypes.c_void_p(ctypes.addressof(_buf))
MISALIGNED = ctypes.c_void_p(ctypes.addressof(_buf) + 4)    # misaligned for 8-byte elements
MISALIGNED4 = ctypes.c_void_p(ctypes.addressof(_buf) + 2)   # misaligned for 4-byte elements
FAKE16 = ctypes.c_void_p(ctypes.addressof(_buf) + (-ctypes.addressof(_buf) % 16))   # 16-byte aligned
MISALIGNED16 = ctypes.c_void_p(FAKE16.value + 8)            # 8- but not 16-byte aligned


def _pred(dims, dtype, layers):
    p = M.Predictor()
    p.n_layers = layers
    for i, d in enumerate(dims):
        p.dims[i] = d
    p.dtype = dtype
    for l in range(layers):
        p.weight[l] = FAKE.value
        p.bias[l] = FAKE.value
    p.bin_centre = FAKE.value
    return p


def test_predict_validation(lib):
    call = lambda p, n=10, x=FAKE: lib.maestro_predict(ctypes.byref(p) if p is not None else None, n, x,
                                                       FAKE, FAKE, FAKE, 4, FAKE, FAKE, None, 0, None)
    assert call(None) == INVALID
    assert call(_pred((256, 512, 512, 64), 1, 3), n=-1) == INVALID
    assert call(_pred((256, 512, 512, 64), 7, 3)) == INVALID                   # bad dtype
    assert call(_pred((256, 512, 512, 64), 1, 3), x=None) == INVALID          # null features
    assert call(_pred((256, 512, 512, 64), 1, 3), x=MISALIGNED) == INVALID    # misaligned
    p = _pred((256, 512, 512, 64), 1, 3)
    p.weight[1] = None
    assert call(p) == INVALID                                                 # missing layer
    assert call(_pred((256, 512, 0, 64), 1, 3)) == INVALID                    # zero width
    assert call(_pred((256, 384, 512, 64), 1, 3)) == UNSUPPORTED              # not built
    assert call(_pred((64, 128, 32), 1, 2)) == UNSUPPORTED                    # wrong dtype
    assert lib.maestro_predict_workspace(ctypes.byref(_pred((64, 128, 32), 0, 2)), 100) == 0


def test_predict_two_phase_validation(lib):
    def tp(n_roles=3, n_knots=16, max_len=32768.0, coef=FAKE16, head=FAKE, kx=FAKE, ky=FAKE):
        return M.TwoPhase(n_roles=n_roles, n_knots=n_knots, role_head=head.value if head else None,
                          tool_coef=coef.value if coef else None, iso_x=kx.value if kx else None,
                          iso_y=ky.value if ky else None, max_len=max_len)

    def call(p, t, n=10, x=FAKE, role=FAKE, tools=FAKE):
        return lib.maestro_predict_two_phase(ctypes.byref(p) if p is not None else None,
                                             ctypes.byref(t) if t is not None else None, n, x, FAKE, FAKE, role,
                                             tools, FAKE, 4, None, FAKE, FAKE, None)
    good = _pred((256, 512, 512, 64), 1, 3)
    assert call(None, tp()) == INVALID
    assert call(good, None) == INVALID
    assert call(good, tp(), n=-1) == INVALID
    assert call(good, tp(n_knots=1)) == INVALID                                 # a map needs two knots
    assert call(good, tp(n_knots=65)) == INVALID
    assert call(good, tp(n_roles=65)) == INVALID
    assert call(good, tp(n_roles=-1)) == INVALID
    assert call(good, tp(head=None)) == INVALID                                 # roles without a table
    assert call(good, tp(max_len=0.0)) == INVALID
    assert call(good, tp(max_len=float("inf"))) == INVALID
    assert call(good, tp(max_len=float("nan"))) == INVALID
    assert call(good, tp(coef=None)) == INVALID
    assert call(good, tp(coef=MISALIGNED16)) == INVALID                         # 16-byte aligned table
    assert call(good, tp(kx=None)) == INVALID
    assert call(good, tp(), role=None) == INVALID                              # per-stage roles missing
    assert call(good, tp(), tools=MISALIGNED4) == INVALID
    assert call(_pred((64, 128, 32), 0, 2), tp()) == UNSUPPORTED                # float32 network: not built
    assert call(_pred((256, 384, 512, 64), 1, 3), tp()) == UNSUPPORTED
    assert call(good, tp(n_roles=0, head=None), n=0, x=None, role=None, tools=None) == OK   # empty batch


def test_route_validation(lib):
    def call(n=10, n_models=8, n_nodes=16, k=1, rho=0.0, model=FAKE, free=FAKE):
        return lib.maestro_route(n, model, FAKE, FAKE, FAKE, n_models, n_nodes, free, FAKE, FAKE, FAKE,
                                 rho, k, FAKE, FAKE, None, 0, None)
    def call_ex(algo, n_nodes=16, ws=None, ws_bytes=0):
        return lib.maestro_route_ex(10, FAKE, FAKE, FAKE, FAKE, 8, n_nodes, FAKE, FAKE, FAKE, FAKE, 0.0, 1,
                                    algo, FAKE, FAKE, ws, ws_bytes, None)
    assert call_ex(3) == INVALID                                              # unknown algorithm
    assert call_ex(-1) == INVALID
    assert call_ex(2) == WORKSPACE                                            # sorted lists need space
    # sorted lists: one 16-byte entry per (model, node); none beyond 8192 nodes
    # per model: 16 bytes per node, then the float32 largest headroom of every 8 / 64 / 512 nodes
    assert lib.maestro_route_workspace(10, 8, 16, 1) == 8 * (16 * 16 + 4 * (2 + 1 + 1))
    assert lib.maestro_route_workspace(10, 8, 8193, 1) == 0
    assert call(n=-1) == INVALID
    assert call(n_models=0) == INVALID
    assert call(n_models=65) == INVALID
    assert call(n_nodes=0) == INVALID
    assert call(k=0) == INVALID
    assert call(k=17) == INVALID
    assert call(rho=-0.1) == INVALID
    assert call(rho=float("nan")) == INVALID
    assert call(rho=float("inf")) == INVALID
    assert call(model=None) == INVALID
    assert call(free=MISALIGNED) == INVALID


def test_route_split_validation(lib):
    # the node half and the stage half of the sorted route, rejected before any launch
    assert lib.maestro_route_lists_bytes(8, 16) == 8 * (16 * 16 + 4 * (2 + 1 + 1))
    assert lib.maestro_route_lists_bytes(64, 8192) == 64 * (8192 * 16 + 4 * (1024 + 128 + 16))
    assert lib.maestro_route_lists_bytes(8, 8193) == 0
    assert lib.maestro_route_lists_bytes(0, 16) == 0 and lib.maestro_route_lists_bytes(65, 16) == 0
    need = 8 * 16 * 16

    def sort(n_models=8, n_nodes=16, free=FAKE, queue=FAKE, cold=FAKE, mask=FAKE, act=None, lists=FAKE16,
             nbytes=need):
        return lib.maestro_route_sort_nodes(n_models, n_nodes, free, queue, cold, mask, act, lists, nbytes, None)
    assert sort(n_models=0) == INVALID and sort(n_models=65) == INVALID and sort(n_nodes=0) == INVALID
    assert sort(free=None) == INVALID and sort(free=MISALIGNED) == INVALID and sort(queue=MISALIGNED4) == INVALID
    assert sort(cold=None) == INVALID and sort(mask=MISALIGNED) == INVALID    # residency form incomplete
    assert sort(lists=None) == WORKSPACE and sort(lists=MISALIGNED16) == WORKSPACE
    assert sort(nbytes=need - 1) == WORKSPACE
    assert sort(n_nodes=8193, nbytes=1 << 30) == UNSUPPORTED
    assert sort(cold=None, mask=None, act=MISALIGNED4) == INVALID            # readiness form misaligned

    def walk(n=10, n_models=8, n_nodes=16, k=1, rho=0.0, model=FAKE, lists=FAKE16, nbytes=need, dec=FAKE):
        return lib.maestro_route_walk(n, model, FAKE, FAKE, dec, n_models, n_nodes, lists, nbytes, rho, k, FAKE,
                                      FAKE, None)
    assert walk(n=-1) == INVALID and walk(n_models=0) == INVALID and walk(n_nodes=0) == INVALID
    assert walk(k=0) == INVALID and walk(k=17) == INVALID
    assert walk(rho=-1.0) == INVALID and walk(rho=float("nan")) == INVALID
    assert walk(model=None) == INVALID and walk(model=MISALIGNED4) == INVALID and walk(dec=None) == INVALID
    assert walk(lists=None) == WORKSPACE and walk(nbytes=need - 16) == WORKSPACE
    assert walk(n_nodes=9000, nbytes=1 << 30) == UNSUPPORTED
    assert walk(n=1 << 38, nbytes=need) == UNSUPPORTED


def test_route_tiered_validation(lib):
    def call(n=10, n_models=8, n_nodes=16, k=1, act=FAKE, algo=0, ws=None, ws_bytes=0):
        return lib.maestro_route_tiered(n, FAKE, FAKE, FAKE, FAKE, n_models, n_nodes, FAKE, FAKE, act, 0.0, k, algo,
                                        FAKE, FAKE, ws, ws_bytes, None)
    assert call(act=None) == INVALID                                          # T_act from nowhere
    assert call(act=MISALIGNED4) == INVALID
    assert call(n_models=65) == INVALID
    assert call(k=17) == INVALID
    assert call(algo=2) == WORKSPACE                                          # sorted lists need room
    assert call(n=0, algo=1) == OK                                           # empty batch, scan: no-op


def test_route_fitness_and_quantiles_validation(lib):
    def call(n=10, n_models=8, n_nodes=16, n_src=2, n_classes=2, k=1, rho=0.0, src=FAKE, rtt=FAKE, bounds=FAKE,
             deg=FAKE, plans=None, steps=None, act=FAKE, mask=FAKE, mat=None):
        return lib.maestro_route_fitness(n, FAKE, src, FAKE, FAKE, n_models, n_nodes, n_src, n_classes,
                                         FAKE, FAKE, act, mask, mat, deg, plans, steps, rtt, FAKE, bounds, rho, k,
                                         FAKE, FAKE, None)
    assert call(n=-1) == INVALID
    assert call(n_models=0) == INVALID
    assert call(n_models=65) == INVALID
    assert call(n_nodes=0) == INVALID
    assert call(n_src=0) == INVALID
    assert call(n_src=17) == INVALID                                          # at most 16 sources
    assert call(n_classes=17) == INVALID
    assert call(k=17) == INVALID
    assert call(rho=float("nan")) == INVALID
    assert call(src=None) == INVALID                                          # per-stage input missing
    assert call(rtt=None) == INVALID
    assert call(bounds=MISALIGNED4) == INVALID
    assert call(n=0, src=None) == OK                                          # empty batch: no-op
    assert call(deg=None) == INVALID                                          # C_deg from nowhere
    assert call(deg=None, plans=MISALIGNED16, steps=FAKE16) == INVALID        # plan records are 16-aligned
    assert call(deg=None, plans=FAKE16, steps=None) == INVALID                # records need their steps
    assert call(deg=None, plans=FAKE16, steps=MISALIGNED16) == INVALID
    assert call(deg=None, plans=FAKE16, steps=FAKE16, rtt=None) == INVALID
    assert call(n=0, deg=None, plans=FAKE16, steps=FAKE16) == OK              # plans replace deg_ms
    assert call(act=None) == INVALID                                          # T_act from nowhere
    assert call(mask=MISALIGNED) == INVALID
    assert call(act=None, mask=None, mat=MISALIGNED4) == INVALID
    assert call(n=0, act=None, mask=None, mat=FAKE) == OK                     # a T_act matrix replaces both
    q = lambda m=10, lo=0.05, hi=0.95, v=FAKE, out=FAKE, ws=None, wb=0: lib.maestro_quantiles(v, m, lo, hi, out, ws,
                                                                                              wb, None)
    assert q(m=0) == INVALID
    assert q(lo=0.6, hi=0.5) == INVALID
    assert q(lo=-0.1) == INVALID
    assert q(hi=1.5) == INVALID
    assert q(lo=float("nan")) == INVALID
    assert q(v=None) == INVALID
    assert q(out=MISALIGNED4) == INVALID
    assert q(m=1 << 32) == UNSUPPORTED
    # long windows select over several workgroups in a workspace: 256 histograms of 512 words
    need = lib.maestro_quantiles_workspace(32768)
    assert lib.maestro_quantiles_workspace(32767) == 0 and need >= 256 * 512 * 4
    assert lib.maestro_quantiles_workspace(0) == 0 and lib.maestro_quantiles_workspace(1 << 32) == 0
    assert q(m=32768) == WORKSPACE
    assert q(m=32768, ws=FAKE16, wb=need - 1) == WORKSPACE
    assert q(m=32768, ws=MISALIGNED16, wb=need) == WORKSPACE


def test_activation_latency_validation(lib):
    def call(M=4, K=3, tier=FAKE, size=FAKE, bw=FAKE, setup=FAKE, out=FAKE, unit=1000.0):
        return lib.maestro_activation_latency(M, K, tier, size, bw, setup, unit, out, None)
    assert call(M=-1) == INVALID
    assert call(K=0) == INVALID
    assert call(K=65) == INVALID
    assert call(tier=None) == INVALID
    assert call(size=MISALIGNED) == INVALID
    assert call(bw=None) == INVALID
    assert call(out=MISALIGNED4) == INVALID
    assert call(unit=0.0) == INVALID
    assert call(unit=float("inf")) == INVALID
    assert call(M=0, tier=None, out=None) == OK                               # no nodes: no-op


def test_adaptive_rho_validation(lib):
    def call(m=100, beta=0.2, q=0.95, a=FAKE, p=FAKE, ew=FAKE, rho=FAKE, ws=None, wb=0):
        return lib.maestro_adaptive_rho(a, p, m, beta, q, ew, rho, ws, wb, None)
    assert call(m=0) == INVALID
    assert call(beta=0.0) == INVALID                                          # no weight on new errors
    assert call(beta=1.5) == INVALID
    assert call(beta=float("nan")) == INVALID
    assert call(q=-0.1) == INVALID
    assert call(q=1.01) == INVALID
    assert call(a=None) == INVALID
    assert call(p=MISALIGNED) == INVALID
    assert call(rho=MISALIGNED4) == INVALID
    assert call(m=1 << 32) == UNSUPPORTED
    assert call(m=1 << 20) == WORKSPACE                                       # long windows need one
    assert call(m=1 << 20, ws=FAKE16, wb=lib.maestro_quantiles_workspace(1 << 20) - 16) == WORKSPACE


def test_degradation_plans_validation(lib):
    def call(n_nodes=4, off=FAKE, level=FAKE, freed=FAKE, cost=FAKE, c_int=2000.0, plans=FAKE16, steps=FAKE16):
        return lib.maestro_degradation_plans(n_nodes, off, level, freed, cost, c_int, plans, steps, None)
    assert call(n_nodes=-1) == INVALID
    assert call(c_int=float("nan")) == INVALID
    assert call(off=None) == INVALID
    assert call(plans=None) == INVALID
    assert call(plans=MISALIGNED16) == INVALID
    assert call(steps=None) == INVALID
    assert call(steps=MISALIGNED16) == INVALID
    assert call(level=MISALIGNED4) == INVALID
    assert call(freed=MISALIGNED) == INVALID
    assert call(n_nodes=0, off=None, plans=None, steps=None) == OK            # no nodes: no-op
    assert ctypes.sizeof(ctypes.c_double) * 8 + 4 * 8 + 4 * 8 == _native.PLAN_BYTES
    assert ctypes.sizeof(ctypes.c_double) + 4 + 4 == _native.STEP_BYTES


def test_prioritize_validation_and_workspace(lib):
    ws = lib.maestro_prioritize_workspace(131072, 720000)
    # four key/value arrays padded to 1024-key tiles plus a 256-entry count table per tile, and
    # 256 bytes for the word that tells whether a call has long chains
    tiles = 131072 // 1024
    assert ws == 4 * 4 * tiles * 1024 + 4 * 256 * tiles + 256
    assert lib.maestro_prioritize_workspace(0, 0) == 0
    assert lib.maestro_prioritize_workspace(1, 3) == 4 * 4 * 1024 + 4 * 256 + 256
    # beyond 128 such tiles: 4096-key tiles, plus a 256-entry offset table per group of tiles
    # (16 .. 256 tiles, a power of two, at most 64 groups up to 2^26 keys)
    tiles = (200000 + 4095) // 4096
    assert lib.maestro_prioritize_workspace(200000, 10**6) == 4 * 4 * tiles * 4096 + 4 * 256 * tiles + 4 * 256 * 4 + 256
    tiles = (1 << 26) // 4096
    assert lib.maestro_prioritize_workspace(1 << 26, 0) == 4 * 4 * tiles * 4096 + 4 * 256 * tiles + 4 * 256 * 64 + 256
    call = lambda W=4, S=8, off=FAKE, ws=FAKE, ws_bytes=1 << 20: lib.maestro_prioritize(
        W, S, off, FAKE, None, FAKE, 0, None, FAKE, FAKE, ws, ws_bytes, None)
    assert call(W=-1) == INVALID
    assert call(S=-1) == INVALID
    assert call(off=None) == INVALID
    assert call(ws_bytes=100) == WORKSPACE
    assert call(ws=None) == WORKSPACE
    assert call(W=0) == OK                                                   # empty: no-op


def test_prioritize_noalloc_validation(lib):
    call = lambda W=4, S=8, off=FAKE, key=FAKE: lib.maestro_prioritize_noalloc(
        W, S, off, FAKE, None, FAKE, 0, None, key, FAKE, None)
    assert call(W=-1) == INVALID
    assert call(S=-1) == INVALID
    assert call(off=None) == INVALID
    assert call(key=MISALIGNED4) == INVALID
    assert call(W=_native.PRIORITIZE_NOALLOC_MAX_WORKFLOWS + 1) == WORKSPACE   # beyond the static scratch
    assert call(W=0) == OK                                                   # empty: no-op


def test_binding_fails_loudly_without_library(monkeypatch, tmp_path):
    monkeypatch.setattr(_native, "_lib", None)
    monkeypatch.setattr(_native, "LIBRARY_PATH", str(tmp_path / "missing.so"))
    with pytest.raises(RuntimeError, match="missing"):
        _native.load()


def test_calibrate_library_sizes_and_argument_checks():
    """The measurement-only matrix-core probe (libmaestro_calibrate.so, timed by bench.py
    --mfma-ceiling): its sizing calls, and argument checks that return -1 before any launch."""
    from paper_2606_12950_amd import build as B
    if not os.path.exists(B.CALIBRATE_LIB):
        pytest.fail("libmaestro_calibrate.so is not built (python -m paper_2606_12950_amd.build)")
    c = ctypes.CDLL(B.CALIBRATE_LIB)
    c.maestro_calibrate_mfma.argtypes = [ctypes.c_void_p, ctypes.c_int, ctypes.c_int, ctypes.c_int,
                                         ctypes.c_uint32, ctypes.c_void_p]
    c.maestro_calibrate_mfma.restype = ctypes.c_int
    c.maestro_calibrate_mfma_outputs.restype = ctypes.c_int
    c.maestro_calibrate_mfma_count.argtypes = [ctypes.c_int]
    c.maestro_calibrate_mfma_count.restype = ctypes.c_int64
    assert c.maestro_calibrate_mfma_outputs() == 256 * 256          # one float per thread
    assert c.maestro_calibrate_mfma_count(1000) == 16 * 1000 * 4 * 256   # per wavefront x 4 x 256 workgroups
    buf = ctypes.c_void_p(FAKE16.value)
    assert c.maestro_calibrate_mfma(None, 10, 1, 0, 1, None) == -1
    assert c.maestro_calibrate_mfma(buf, 0, 1, 0, 1, None) == -1
    assert c.maestro_calibrate_mfma(buf, 10, 2, 0, 1, None) == -1
    assert c.maestro_calibrate_mfma(buf, 10, 1, 3, 1, None) == -1
    assert c.maestro_calibrate_mfma(buf, 10, 1, -1, 1, None) == -1
