"""Checks of the synthetic input generators (no method arithmetic involved)."""
import numpy as np
import pytest

from synth import gen


def test_affine_relabelling_is_a_bijection():
    for n in (1, 2, 10, 997, 10_000):
        perm = gen.affine_permutation(n, 3)
        x = gen.relabel(np.arange(n), n, perm)
        assert np.array_equal(np.sort(x), np.arange(n))


def test_exact_sbm_degrees_match_expectation():
    rng = np.random.default_rng(0)
    n, blocks, din, dout = 10_000, 10, 20.0, 1.0
    E = gen.sbm_edges(n, blocks, din, dout, rng)
    assert np.all(E[:, 0] < E[:, 1])
    assert np.unique(E, axis=0).shape[0] == E.shape[0]
    B = n // blocks
    same = (E[:, 0] // B) == (E[:, 1] // B)
    # 2 m / n is the mean degree of each class; binomial spread is ~1%
    assert 2 * same.sum() / n == pytest.approx(din, rel=0.03)
    assert 2 * (~same).sum() / n == pytest.approx(dout, rel=0.1)


def test_csr_walks_follow_edges():
    rng = np.random.default_rng(1)
    E = gen.sbm_edges(2000, 4, 6.0, 1.0, rng)
    off, nbr = gen.csr_from_edges(2000, E)
    edges = set(map(tuple, E.tolist())) | set((b, a) for a, b in E.tolist())
    W = gen.walk_csr(off, nbr, np.arange(2000), 8, rng)
    for row in W[:300]:
        for a, b in zip(row[:-1], row[1:]):
            if b < 0:
                break
            assert (int(a), int(b)) in edges


def test_window_pair_count_closed_form():
    # distinct nodes in every walk: 2 * sum_{d=1..w} (L + 1 - d) pairs per walk
    L, w, m = 10, 3, 5
    W = np.arange(m * (L + 1)).reshape(m, L + 1)
    s, d = gen.window_pairs(W, w)
    assert s.size == m * 2 * sum(L + 1 - k for k in range(1, w + 1))
    s2, d2, c = gen.aggregate_pairs(s, d, W.size)
    assert c.sum() == s.size and np.all(c == 1)


def test_annealed_sbm_stays_in_block_at_the_sbm_rate():
    n, blocks = 100_000, 100
    step = gen.annealed_sbm_step(n, blocks, 25.0, 2.0)
    rng = np.random.default_rng(2)
    cur = rng.integers(0, n, 200_000)
    nxt = step(cur, rng)
    B = n // blocks
    assert np.all(nxt != cur) and nxt.min() >= 0 and nxt.max() < n
    assert np.mean(cur // B == nxt // B) == pytest.approx(25 / 27, abs=0.005)


def test_tiny_epoch_and_streamed_batches():
    wl = gen.make_workload("tiny", 0)
    s, d, c = wl.epoch()
    assert s.size > 500_000
    assert np.all(s != d) and np.all(c >= 1)
    assert s.min() >= 0 and s.max() < 10_000
    # pairs are unique after aggregation
    key = s.astype(np.int64) * 10_000 + d
    assert np.unique(key).size == key.size
    b0 = wl.batch(0)
    b0_again = wl.batch(0)
    assert all(np.array_equal(x, y) for x, y in zip(b0, b0_again))
    assert b0[0].size == 1024 and np.all(b0[0] != b0[1]) and np.all(b0[2] >= 1)


def test_chung_lu_weights_power_law_tail():
    w = gen.chung_lu_weights(1_000_000, 2.1, 30.0)
    assert w.mean() == pytest.approx(30.0)
    # rank-size slope -1/(gamma-1)
    slope = np.log(w[9999] / w[99]) / np.log(10000 / 100)
    assert slope == pytest.approx(-1 / 1.1, rel=1e-9)
