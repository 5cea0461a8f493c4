"""Pins of the oracle's weighted co-occurrences (Sec. 3.2: co_counts is a
histogram over the walk distance; a weight per distance turns it into one
weight per positive): the weights against exact rational arithmetic, the
weighted step against the integer step where the weights are the integer
counts, a zero weight against removing the positive, the loss's linearity in
the weights, and invalid weights rejected."""
import math
import os
import sys
from fractions import Fraction

import numpy as np
import pytest

sys.path.insert(0, os.path.join(os.path.dirname(__file__), ".."))
from oracle import oracle as orc  # noqa: E402


def test_weights_of_unit_distance_weights_are_the_counts():
    rng = np.random.default_rng(1)
    hist = rng.integers(0, 50, size=(500, 5)).astype(np.int32)
    w = orc.cocount_weights(hist, np.ones(5, np.float32))
    assert np.array_equal(w, hist.sum(axis=1).astype(np.float32))


def test_weights_against_exact_rationals():
    rng = np.random.default_rng(2)
    wd = np.array([1.0, 0.5, 0.25, 0.125, 1 / 3], np.float32)   # 1/3 is not exact in float
    hist = rng.integers(0, 1 << 20, size=(300, 5)).astype(np.int32)
    got = orc.cocount_weights(hist, wd)
    for i in range(hist.shape[0]):
        exact = sum(Fraction(float(wd[d])) * int(hist[i, d]) for d in range(5))
        # double sum of 5 products of < 2^44: within a few double ulps of the
        # exact value, so its float rounding is the float nearest to it (or,
        # at a float tie, a neighbour)
        want = np.float32(float(exact))
        assert abs(float(got[i]) - float(exact)) <= abs(float(want) - float(exact)) + \
            2.0 ** -52 * float(exact)
    # small values are exact
    h = np.array([[3, 1, 0, 2, 0]], np.int32)
    assert orc.cocount_weights(h, wd)[0] == np.float32(3 + 0.5 + 0.25)


def _batch(rng, N, n, K):
    src = rng.integers(0, N, n).astype(np.int32)
    dst = rng.integers(0, N, n).astype(np.int32)
    neg = rng.integers(0, N, (n, K)).astype(np.int32)
    return src, dst, neg


def test_weighted_step_with_integer_weights_equals_the_integer_step():
    rng = np.random.default_rng(3)
    N, D, K, n = 300, 16, 3, 800
    src, dst, neg = _batch(rng, N, n, K)
    cc = rng.integers(0, 20, n).astype(np.int32)
    S0 = rng.uniform(-0.1, 0.1, (N, D)).astype(np.float32)
    T0 = rng.uniform(-0.1, 0.1, (N, D)).astype(np.float32)
    S1, T1 = S0.copy(), T0.copy()
    S2, T2 = S0.copy(), T0.copy()
    l1 = orc.step_dense(S1, T1, src, dst, cc, neg, 0.05)
    l2 = orc.step_dense(S2, T2, src, dst, cc.astype(np.float32), neg, 0.05)
    assert l1 == l2
    assert np.array_equal(S1, S2) and np.array_equal(T1, T2)


def test_zero_weight_removes_the_positive():
    rng = np.random.default_rng(4)
    N, D, K, n = 200, 8, 2, 300
    src, dst, neg = _batch(rng, N, n, K)
    w = rng.uniform(0.1, 3.0, n).astype(np.float32)
    drop = np.arange(n) % 7 == 3
    w[drop] = 0.0
    S0 = rng.uniform(-0.2, 0.2, (N, D)).astype(np.float32)
    T0 = rng.uniform(-0.2, 0.2, (N, D)).astype(np.float32)
    S1, T1 = S0.copy(), T0.copy()
    S2, T2 = S0.copy(), T0.copy()
    l1 = orc.step_dense(S1, T1, src, dst, w, neg, 0.1)
    keep = ~drop
    l2 = orc.step_dense(S2, T2, src[keep], dst[keep], w[keep], neg[keep], 0.1)
    assert l1 == pytest.approx(l2, rel=1e-14)
    # rows touched only by dropped positives are rewritten unchanged by the
    # weighted step (a zero gradient); every row agrees to rounding
    assert np.allclose(S1, S2, rtol=0, atol=1e-7) and np.allclose(T1, T2, rtol=0, atol=1e-7)


def test_loss_is_linear_in_the_weights():
    rng = np.random.default_rng(5)
    N, D, K, n = 100, 8, 4, 60
    src, dst, neg = _batch(rng, N, n, K)
    S = rng.normal(0, 0.3, (N, D)).astype(np.float32)
    T = rng.normal(0, 0.3, (N, D)).astype(np.float32)
    w = rng.uniform(0, 5, n).astype(np.float32)
    total = orc.loss_dense(S, T, src, dst, w, neg)
    parts = [orc.loss_dense(S, T, src[i:i + 1], dst[i:i + 1], np.ones(1, np.float32),
                            neg[i:i + 1]) for i in range(n)]
    assert total == pytest.approx(sum(float(w[i]) * parts[i] for i in range(n)), rel=1e-12)
    # and the weighted loss at unit weights is the integer loss at unit counts
    assert orc.loss_dense(S, T, src, dst, np.ones(n, np.float32), neg) == \
        orc.loss_dense(S, T, src, dst, np.ones(n, np.int32), neg)


@pytest.mark.parametrize("bad", [-1.0, float("nan"), float("inf")])
def test_invalid_weights_are_rejected(bad):
    rng = np.random.default_rng(6)
    src, dst, neg = _batch(rng, 50, 10, 2)
    w = np.ones(10, np.float32)
    w[4] = bad
    S = np.zeros((50, 4), np.float32)
    T = np.zeros((50, 4), np.float32)
    with pytest.raises(Exception):
        orc.step_dense(S, T, src, dst, w, neg, 0.1)
    with pytest.raises(Exception):
        orc.cocount_weights(np.ones((2, 3), np.int32), [1.0, bad, 1.0])
    assert math.isfinite(orc.loss_dense(S, T, src, dst, np.ones(10, np.float32), neg))
