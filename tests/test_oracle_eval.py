"""Pins of the oracle's embedding metrics (Sec. 4's unsupervised evaluation):
closed forms of the normalised distance, percentiles against numpy, the
pair samplers against brute-force adjacency and uniformity, the nearest
neighbours against points on a circle whose order is known, and recall on
graphs built to give 0, 1/2 and 1."""
import math
import os
import sys

import numpy as np
import pytest

sys.path.insert(0, os.path.join(os.path.dirname(__file__), ".."))
from oracle import oracle as orc  # noqa: E402


def _csr(n, edges):
    """Sorted CSR lists of the directed edge list."""
    adj = [[] for _ in range(n)]
    for a, b in edges:
        adj[a].append(b)
    off = np.zeros(n + 1, np.int64)
    for i in range(n):
        off[i + 1] = off[i] + len(adj[i])
    nbr = np.array([b for i in range(n) for b in sorted(adj[i])], np.int32)
    return off, nbr


# --------------------------------------------------------------------------- distances
def test_distance_closed_forms():
    T = np.array([[3.0, 0, 0, 0],      # 0: e1 scaled
                  [0, 0.5, 0, 0],      # 1: e2 scaled
                  [6.0, 0, 0, 0],      # 2: same direction as 0
                  [-1.0, 0, 0, 0],     # 3: opposite of 0
                  [0, 0, 0, 0],        # 4: zero row
                  [1.0, 1.0, 0, 0]],   # 5: 45 degrees from 0
                 np.float32)
    u = np.array([0, 0, 0, 0, 4, 0, 4])
    v = np.array([1, 2, 3, 4, 4, 5, 1])
    d = orc.pair_distances(T, u, v)
    want = [math.sqrt(2), 0.0, 2.0, 1.0, 0.0, math.sqrt(2 - math.sqrt(2)), 1.0]
    assert np.allclose(d, want, atol=1e-15)


def test_distance_is_scale_invariant_and_symmetric():
    rng = np.random.default_rng(1)
    T = rng.normal(size=(50, 16))
    u = rng.integers(0, 50, 200)
    v = rng.integers(0, 50, 200)
    d = orc.pair_distances(T, u, v)
    T2 = T * rng.uniform(0.1, 10, size=(50, 1))
    assert np.allclose(orc.pair_distances(T2, u, v), d, atol=1e-12)
    assert np.allclose(orc.pair_distances(T, v, u), d, atol=1e-15)
    # |a - b|^2 = 2 - 2 cos for unit rows
    cos = np.sum(orc.normalize_rows(T)[u] * orc.normalize_rows(T)[v], axis=1)
    assert np.allclose(d ** 2, 2 - 2 * cos, atol=1e-12)
    assert np.all(np.isnan(orc.pair_distances(T, [-1, 3], [-1, -1])))


# --------------------------------------------------------------------------- summary
def test_percentiles_match_numpy_linear():
    rng = np.random.default_rng(2)
    for n in (1, 2, 5, 100, 1001):
        x = rng.normal(size=n)
        for q in (0, 1, 10, 25, 50, 75, 90, 99, 100, 33.3):
            assert orc.percentile_linear(x, q) == pytest.approx(
                float(np.percentile(x, q, method="linear")), abs=1e-15)
    assert orc.percentile_linear([1, 2, 3, 4], 50) == 2.5
    assert orc.percentile_linear([4, 1, 3, 2], 0) == 1
    assert orc.percentile_linear([4, 1, 3, 2], 100) == 4


def test_summary_on_a_built_example():
    # edges at distances 0.5 (x3) and 1.0, non-edges at 1.5 and 2.0, one failed draw
    s = orc.eval_summary([0.5, 0.5, 0.5, 1.0], [1.5, 2.0, np.nan], [0, 50, 100])
    assert (s.count_edge, s.count_non) == (4, 2)
    assert s.mean_edge == 0.625 and s.mean_non == 1.75
    assert s.snr == pytest.approx(2.8)
    assert s.pct_edge == [0.5, 0.5, 1.0]
    assert s.pct_non == [1.5, 1.75, 2.0]


# --------------------------------------------------------------------------- pairs
def _small_graph(seed=3, n=40, m=150):
    rng = np.random.default_rng(seed)
    edges = set()
    while len(edges) < m:
        a, b = rng.integers(0, n, 2)
        if a != b:
            edges.add((int(a), int(b)))
    return n, sorted(edges)


def test_edge_pairs_are_edges_and_uniform():
    n, edges = _small_graph()
    off, nbr = _csr(n, edges)
    ne = 150 * 400
    u, v = orc.eval_pairs(off, nbr, n, seed=11, n_edge=ne, n_non=0)
    es = set(edges)
    assert all((int(a), int(b)) in es for a, b in zip(u, v))
    # each directed edge equally likely: chi-square over the 150 edges
    idx = {e: i for i, e in enumerate(edges)}
    cnt = np.bincount([idx[(int(a), int(b))] for a, b in zip(u, v)], minlength=len(edges))
    exp = ne / len(edges)
    chi2 = float(np.sum((cnt - exp) ** 2 / exp))
    assert chi2 < 149 + 6 * math.sqrt(2 * 149), chi2


def test_non_edge_pairs_avoid_edges_and_self_and_are_uniform():
    n, edges = _small_graph(seed=4)
    off, nbr = _csr(n, edges)
    adj = np.zeros((n, n), bool)
    for a, b in edges:
        adj[a, b] = True
    nn = 100_000
    u, v = orc.eval_pairs(off, nbr, n, seed=12, n_edge=0, n_non=nn, max_tries=64)
    assert np.all(u >= 0)
    assert not np.any(u == v)
    assert not np.any(adj[u, v])
    # uniform over the n(n-1) - |E| ordered non-edges
    cells = (~adj) & ~np.eye(n, dtype=bool)
    cnt = np.zeros((n, n))
    np.add.at(cnt, (u, v), 1)
    k = int(cells.sum())
    exp = nn / k
    chi2 = float(np.sum((cnt[cells] - exp) ** 2 / exp))
    assert chi2 < (k - 1) + 6 * math.sqrt(2 * (k - 1)), chi2


def test_non_edge_draws_fail_on_a_complete_graph_and_edges_need_edges():
    n = 6
    off, nbr = _csr(n, [(a, b) for a in range(n) for b in range(n) if a != b])
    u, v = orc.eval_pairs(off, nbr, n, seed=1, n_edge=3, n_non=20, max_tries=16)
    assert np.all(u[3:] == -1) and np.all(v[3:] == -1)
    assert np.all(u[:3] != v[:3]) and np.all(u[:3] >= 0)
    off0, nbr0 = _csr(n, [])
    with pytest.raises(Exception):
        orc.eval_pairs(off0, nbr0, n, seed=1, n_edge=1, n_non=0)
    u0, v0 = orc.eval_pairs(off0, nbr0, n, seed=1, n_edge=0, n_non=5)
    assert np.all(u0 != v0) and np.all(u0 >= 0)


def test_edge_pair_source_rows_include_high_ids_and_skip_empty_lists():
    # rows 0 and 2 empty, row 3 (the last) holds most edges
    off = np.array([0, 0, 1, 1, 5], np.int64)
    nbr = np.array([3, 0, 1, 2, 3], np.int32)
    u, v = orc.eval_pairs(off, nbr, 4, seed=5, n_edge=2000, n_non=0)
    assert set(np.unique(u).tolist()) == {1, 3}
    assert np.mean(u == 3) == pytest.approx(0.8, abs=0.05)


# --------------------------------------------------------------------------- neighbours
def test_knn_on_a_circle():
    n, D = 36, 8
    rng = np.random.default_rng(6)
    ang = 2 * math.pi * np.arange(n) / n
    T = np.zeros((n, D))
    T[:, 0] = np.cos(ang)
    T[:, 1] = np.sin(ang)
    T *= rng.uniform(0.5, 3.0, size=(n, 1))  # normalisation removes the scale
    q = [0, 5, 35]
    ids, d = orc.knn(T, q, 4)
    for qi, u in enumerate(q):
        # nearest: the two at one step, then the two at two steps (within a
        # shell the order follows the rounding of cos and sin)
        assert set(ids[qi][:2].tolist()) == {(u - 1) % n, (u + 1) % n}
        assert set(ids[qi][2:].tolist()) == {(u - 2) % n, (u + 2) % n}
        assert d[qi][0] == pytest.approx(2 * math.sin(math.pi / n), abs=1e-12)
        assert d[qi][2] == pytest.approx(2 * math.sin(2 * math.pi / n), abs=1e-12)


def test_knn_matches_brute_force_loops():
    rng = np.random.default_rng(7)
    n, D, k = 60, 5, 7
    T = rng.normal(size=(n, D))
    T[13] = 0.0  # a zero row: distance 1 to every other row
    T[20] = T[21] * 4  # equal directions: distance 0, tie broken by id
    q = [0, 13, 20, 21, 59]
    ids, d = orc.knn(T, q, k)
    for qi, u in enumerate(q):
        cand = []
        nu = math.sqrt(sum(float(x) ** 2 for x in T[u]))
        for w in range(n):
            if w == u:
                continue
            nw = math.sqrt(sum(float(x) ** 2 for x in T[w]))
            s = 0.0
            for c in range(D):
                a = T[u][c] / nu if nu > 0 else 0.0
                b = T[w][c] / nw if nw > 0 else 0.0
                s += (a - b) ** 2
            cand.append((math.sqrt(s), w))
        cand.sort()
        want = cand[:k]
        assert ids[qi].tolist() == [w for _, w in want]
        assert np.allclose(d[qi], [x for x, _ in want], atol=1e-12)


def test_recall_on_built_graphs():
    n = 36
    ang = 2 * math.pi * np.arange(n) / n
    T = np.stack([np.cos(ang), np.sin(ang), np.zeros(n), np.zeros(n)], axis=1)
    # each node linked to its two nearest on the circle, its antipode, and itself
    edges = []
    for u in range(n):
        edges += [(u, (u - 1) % n), (u, (u + 1) % n), (u, (u + n // 2) % n), (u, u)]
    off, nbr = _csr(n, edges)
    q = [0, 7, 20]
    ids, _ = orc.knn(T, q, 4)
    r4 = orc.recall_at_k(off, nbr, q, ids, 4)
    assert np.allclose(r4, 0.5)          # 2 of the 4 nearest are neighbours
    r2 = orc.recall_at_k(off, nbr, q, ids, 2)
    assert np.allclose(r2, 1.0)          # the 2 nearest are both neighbours
    far = np.array([[(u + n // 2 + 3) % n, (u + n // 2 - 3) % n] for u in q])
    assert np.allclose(orc.recall_at_k(off, nbr, q, far, 2), 0.0)
    # duplicate list entries count once
    off2, nbr2 = _csr(3, [(0, 1), (0, 1), (0, 2)])
    assert orc.recall_at_k(off2, nbr2, [0], np.array([[1, 2]]), 2)[0] == 1.0


def test_knn_with_fewer_rows_than_k_pads():
    T = np.eye(4)[:3]
    ids, d = orc.knn(T, [0], 5)
    assert ids[0].tolist()[:2] == [1, 2] and ids[0].tolist()[2:] == [-1, -1, -1]
    assert np.allclose(d[0][:2], math.sqrt(2)) and np.all(np.isnan(d[0][2:]))
