"""Pins of the oracle's bfloat16 tables: the rounding against torch's float32
to bfloat16 conversion and against exact rational rounding, special values,
the initial rows, and the bf16 step against the float step on the same
(widened) values: the same loss, rows equal to the float step's rounded to
bf16 except where rounding twice differs from rounding once, never more
than one bf16 step apart."""
import math
import os
import sys
from fractions import Fraction

import numpy as np
import pytest

sys.path.insert(0, os.path.join(os.path.dirname(__file__), ".."))
from oracle import oracle as orc  # noqa: E402

torch = pytest.importorskip("torch")


def torch_bf16_bits(x32):
    t = torch.from_numpy(np.asarray(x32, np.float32)).to(torch.bfloat16)
    return t.view(torch.int16).numpy().view(np.uint16)


def test_rounding_matches_torch_on_floats():
    rng = np.random.default_rng(1)
    with np.errstate(invalid="ignore"):
        x = _samples(rng)
    x = x[np.isfinite(x)]
    # exact ties: bf16 values plus half a bf16 step
    base = torch_bf16_bits(rng.normal(0, 1, 3000).astype(np.float32)).astype(np.uint32) << 16
    ties = (base | 0x8000).view(np.float32)
    # subnormals
    sub = (rng.integers(1, 1 << 23, 3000).astype(np.uint32)).view(np.float32)
    allx = np.concatenate([x, ties, sub, -sub])
    want = torch_bf16_bits(allx)
    got = np.array([orc.bf16_from_double(float(v)) for v in allx], np.uint16)
    assert np.array_equal(got, want)


def _samples(rng):
    return np.concatenate([
        rng.normal(0, 1, 20000), rng.normal(0, 1e-3, 5000), rng.uniform(-3e38, 3e38, 2000),
        (rng.integers(0, 2**32, 5000, dtype=np.uint64).astype(np.uint32)).view(np.float32)
        .astype(np.float64),
    ]).astype(np.float32)


def exact_bf16(x: float) -> float:
    """Round-half-even of x onto the bf16 grid, in exact rationals."""
    if x == 0:
        return 0.0
    m, e = math.frexp(abs(x))
    E = max(e - 1, -126)
    q = Fraction(2) ** (E - 7)
    n = round(Fraction(abs(x)) / q)          # Python rounds halves to even
    v = n * q
    if v >= Fraction(2) ** 128:
        return math.copysign(math.inf, x)
    return math.copysign(float(v), x)


def test_rounding_of_doubles_against_exact_rationals():
    rng = np.random.default_rng(2)
    xs = list(rng.normal(0, 1, 3000)) + list(rng.normal(0, 1e-39, 500)) + \
        [1.0 + 2 ** -8 + 2 ** -40, 1.0 + 2 ** -8 - 2 ** -40, 3.3895313892515355e38,
         3.3961775292304652e38, -1e-45]
    for x in xs:
        got = orc.bf16_to_float([orc.bf16_from_double(x)])[0]
        want = exact_bf16(float(x))
        assert float(got) == want or (math.isinf(want) and math.isinf(float(got))), x


def test_special_values():
    assert orc.bf16_from_double(0.0) == 0x0000
    assert orc.bf16_from_double(-0.0) == 0x8000
    assert orc.bf16_from_double(math.inf) == 0x7F80
    assert orc.bf16_from_double(-math.inf) == 0xFF80
    assert orc.bf16_from_double(math.nan) & 0x7FC0 == 0x7FC0
    big = float(orc.bf16_to_float([0x7F7F])[0])          # largest finite bf16
    half_ulp = 2.0 ** (127 - 8)
    assert orc.bf16_from_double(big) == 0x7F7F
    assert orc.bf16_from_double(big + half_ulp * 0.999) == 0x7F7F
    assert orc.bf16_from_double(big + half_ulp) == 0x7F80  # tie to the even "mantissa" rounds up
    assert orc.bf16_from_double(1.0 + 2 ** -8) == 0x3F80     # tie to even, down
    assert orc.bf16_from_double(1.0 + 3 * 2 ** -8) == 0x3F82  # tie to even, up


def test_initial_rows_are_the_float_rows_rounded():
    rows = np.array([0, 5, 99, 2 ** 33 + 7], np.int64)
    f = orc.init_rows(7, 1, rows, 36, 0.01)
    b = orc.init_rows_bf16(7, 1, rows, 36, 0.01)
    assert np.array_equal(b, torch_bf16_bits(f).reshape(b.shape))


def _setup(seed=3, N=300, D=16, K=3, n=700):
    rng = np.random.default_rng(seed)
    src = rng.integers(0, N, n).astype(np.int32)
    dst = rng.integers(0, N, n).astype(np.int32)
    neg = rng.integers(0, N, (n, K)).astype(np.int32)
    cc = rng.integers(0, 8, n).astype(np.int32)
    S = torch_bf16_bits(rng.normal(0, 0.2, (N, D)).astype(np.float32)).reshape(N, D)
    T = torch_bf16_bits(rng.normal(0, 0.2, (N, D)).astype(np.float32)).reshape(N, D)
    return src, dst, neg, cc, S, T


def test_bf16_step_against_the_float_step():
    src, dst, neg, cc, S, T = _setup()
    Sb, Tb = S.copy(), T.copy()
    Sf, Tf = orc.bf16_to_float(S).copy(), orc.bf16_to_float(T).copy()
    lb = orc.step_dense_bf16(Sb, Tb, src, dst, cc, neg, 0.05)
    lf = orc.step_dense(Sf, Tf, src, dst, cc, neg, 0.05)
    assert lb == lf                       # the loss is taken at the same pre-step values
    for got, flt in ((Sb, Sf), (Tb, Tf)):
        once = got
        twice = torch_bf16_bits(flt).reshape(got.shape)
        same = once == twice
        assert same.mean() > 0.999
        # where they differ, by one bf16 step
        g = orc.bf16_to_float(once).astype(np.float64)
        w = orc.bf16_to_float(twice).astype(np.float64)
        step = np.abs(w) * 2.0 ** -7
        assert np.all(np.abs(g - w) <= step + 1e-45)


def test_bf16_step_with_zero_rate_changes_nothing():
    src, dst, neg, cc, S, T = _setup(seed=4)
    Sb, Tb = S.copy(), T.copy()
    orc.step_dense_bf16(Sb, Tb, src, dst, cc.astype(np.float32), neg, 0.0)
    assert np.array_equal(Sb, S) and np.array_equal(Tb, T)
