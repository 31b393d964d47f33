"""The fitness kernel evaluates the best fit fl32(a / b) of float32 operands as the float64
product of a with the float64 reciprocal of b, rounded once to float32. This checks, on the CPU
with numpy's IEEE arithmetic, that the method returns the correctly rounded float32 quotient:
random operands over the ranges of KV demands and headrooms, operands with all-ones and
power-of-two significands, quotients near 1, and pairs whose float32 reciprocal-multiply is
off by one unit in the last place. No GPU."""
import numpy as np


def _method(a, b):
    with np.errstate(over="ignore"):       # quotients past float32's range round to infinity
        return (a.astype(np.float64) * (1.0 / b.astype(np.float64))).astype(np.float32)


def _assert_exact(a, b):
    with np.errstate(all="ignore"):
        want = a / b
    got = _method(a, b)
    bad = np.flatnonzero(got.view(np.uint32) != want.view(np.uint32))
    assert bad.size == 0, (a[bad[:3]], b[bad[:3]])


def test_random_operands():
    rng = np.random.default_rng(0)
    for lo, hi in ((1e6, 1e12), (1e-30, 1e30), (0.5, 2.0)):
        a = np.exp(rng.uniform(np.log(lo), np.log(hi), 2_000_000)).astype(np.float32)
        b = np.exp(rng.uniform(np.log(lo), np.log(hi), a.size)).astype(np.float32)
        _assert_exact(a, b)
        _assert_exact(np.minimum(a, b), np.maximum(a, b))     # fits: quotients in (0, 1]


def test_extreme_significands_and_near_one():
    rng = np.random.default_rng(1)
    e = rng.integers(-20, 40, 500_000)
    ones = np.ldexp(np.float32(2) - np.float32(2) ** -23, e).astype(np.float32)     # 1.111...1 x 2^e
    pow2 = np.ldexp(np.float32(1), e).astype(np.float32)
    other = np.exp(rng.uniform(-10, 30, e.size)).astype(np.float32)
    for a, b in ((other, ones), (ones, other), (ones, np.roll(ones, 1)), (other, pow2), (pow2, other)):
        _assert_exact(a, b)
    b = np.exp(rng.uniform(0, 30, 1_000_000)).astype(np.float32)
    a = np.nextafter(b, np.float32(0)).astype(np.float32)                            # just below 1
    _assert_exact(a, b)
    _assert_exact(b, b)


def test_pairs_where_the_float32_reciprocal_is_wrong():
    rng = np.random.default_rng(2)
    a = rng.uniform(1e8, 3e11, 4_000_000).astype(np.float32)
    b = (a * rng.uniform(1.0, 8.0, a.size)).astype(np.float32)
    with np.errstate(all="ignore"):
        sel = (a / b) != a * (np.float32(1) / b)
    assert sel.sum() > 10_000
    _assert_exact(a[sel], b[sel])
