"""The LWSGD learning-rate schedule (Table 2) against its definition: the
paper's four numbers at the knots, exact values in between, piecewise
linearity, and agreement of the product's helper with the oracle's."""
import numpy as np
import pytest

from oracle import oracle as orc
from paper_2307_14490_amd.schedule import PAPER_LWSGD, lwsgd


def test_paper_parameters():
    assert PAPER_LWSGD == (5_000, 0.01, 100_000, 0.001)


@pytest.mark.parametrize("f", [lwsgd, lambda t, *a: orc.lwsgd_lr(t, *a)])
def test_knots_and_hand_values(f):
    W, P, Dk, F = PAPER_LWSGD
    assert f(0, W, P, Dk, F) == pytest.approx(P / W, rel=1e-15)           # 2e-6
    assert f(2_499, W, P, Dk, F) == pytest.approx(0.005, rel=1e-15)       # half-way up
    assert f(W - 1, W, P, Dk, F) == pytest.approx(P, rel=1e-15)           # end of warm-up
    assert f(W + 49_999, W, P, Dk, F) == pytest.approx(0.0055, rel=1e-13)  # half-way down
    assert f(W + Dk - 1, W, P, Dk, F) == pytest.approx(F, rel=1e-15)      # end of decay
    assert f(W + Dk, W, P, Dk, F) == F
    assert f(10**9, W, P, Dk, F) == F


@pytest.mark.parametrize("W,P,Dk,F", [(4, 1.0, 3, 0.25), (1, 0.5, 1, 0.1), (10, 0.05, 20, 0.01),
                                      (0, 0.3, 5, 0.1), (7, 0.2, 0, 0.2)])
def test_piecewise_linear_and_equal_to_oracle(W, P, Dk, F):
    ts = np.arange(0, W + Dk + 5)
    a = np.array([lwsgd(int(t), W, P, Dk, F) for t in ts])
    b = np.array([orc.lwsgd_lr(int(t), W, P, Dk, F) for t in ts])
    np.testing.assert_allclose(a, b, rtol=1e-14, atol=0)
    # second differences vanish inside each segment
    for lo, hi in ((0, W), (W, W + Dk)):
        seg = a[lo:hi]
        if seg.size >= 3:
            np.testing.assert_allclose(np.diff(seg, 2), 0.0, atol=1e-15)
    assert np.all(a[W + Dk - 1 if W + Dk > 0 else 0:] == F) or W + Dk == 0


def test_rejects_bad_arguments():
    with pytest.raises(ValueError):
        lwsgd(-1)
    with pytest.raises(ValueError):
        lwsgd(0, warmup=-1)
