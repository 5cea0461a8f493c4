"""Pins of the oracle's random-walk co-occurrence sampler (Sec. 3.2, Alg. 1)
against what the graph and the definition fix without running the sampler:
deterministic walks (out-degree 1) have closed-form triples, enumerated here
by brute force over walk positions; alternating walks drop their self pairs;
the neighbour choice is uniform (chi-square); walks stop at nodes without
neighbours; a bad graph is an error; the output does not depend on how the
seed range is split."""
import itertools

import numpy as np
import pytest
from scipy import stats

from oracle import oracle as orc


def _csr(n, edges):
    edges = sorted(edges)
    off = np.zeros(n + 1, np.int64)
    for a, _ in edges:
        off[a + 1] += 1
    off = np.cumsum(off)
    nbr = np.array([b for _, b in edges], np.int32)
    return off, nbr


def _expected_from_walk(walk, window, seed_only, walks):
    """Triples of `walks` identical walks, by brute force over positions."""
    agg = {}
    L = len(walk) - 1
    for a, b in itertools.product(range(L + 1), repeat=2):
        d = abs(a - b)
        if d < 1 or d > window or walk[a] == walk[b]:
            continue
        if seed_only and (a != 0 or b < a):
            continue
        h = agg.setdefault((walk[a], walk[b]), [0] * window)
        h[d - 1] += walks
    keys = sorted(agg)
    return ([k[0] for k in keys], [k[1] for k in keys], [sum(agg[k]) for k in keys],
            [agg[k] for k in keys])


@pytest.mark.parametrize("seed_only", [True, False])
@pytest.mark.parametrize("k,window", [(1, 1), (4, 2), (6, 6), (9, 3)])
def test_directed_cycle_closed_form(seed_only, k, window):
    n, gamma = 13, 5
    off, nbr = _csr(n, [(i, (i + 1) % n) for i in range(n)])
    src, dst, cc, hist = orc.sample_walks(off, nbr, n, gamma, k, window, seed_only, seed=7)
    exp = [[], [], [], []]
    for s in range(n):
        walk = [(s + t) % n for t in range(k + 1)]
        for part, vals in zip(exp, _expected_from_walk(walk, window, seed_only, gamma)):
            part.extend(vals)
    assert src.tolist() == exp[0] and dst.tolist() == exp[1]
    assert cc.tolist() == exp[2] and hist.tolist() == exp[3]


@pytest.mark.parametrize("seed_only", [True, False])
def test_perfect_matching_drops_self_pairs(seed_only):
    """Walks alternate s, m(s), s, ...: every even distance is a self pair."""
    n, gamma, k, window = 8, 4, 7, 5
    edges = [(2 * i, 2 * i + 1) for i in range(n // 2)] + [(2 * i + 1, 2 * i) for i in range(n // 2)]
    off, nbr = _csr(n, edges)
    src, dst, cc, hist = orc.sample_walks(off, nbr, n, gamma, k, window, seed_only, seed=3)
    exp = [[], [], [], []]
    for s in range(n):
        m = s ^ 1
        walk = [s if t % 2 == 0 else m for t in range(k + 1)]
        for part, vals in zip(exp, _expected_from_walk(walk, window, seed_only, gamma)):
            part.extend(vals)
    assert src.tolist() == exp[0] and dst.tolist() == exp[1]
    assert cc.tolist() == exp[2] and hist.tolist() == exp[3]
    assert np.all(hist[:, 1::2] == 0)  # even distances never count


def test_first_step_is_uniform_over_neighbours():
    """Complete graph K_40: the first step of 20,000 walks of one seed is
    uniform over its 39 neighbours."""
    n, gamma = 40, 20_000
    edges = [(a, b) for a in range(n) for b in range(n) if a != b]
    off, nbr = _csr(n, edges)
    src, dst, cc, hist = orc.sample_walks(off, nbr, n, gamma, 1, 1, True, seed=11,
                                          first_seed=5, num_seeds=1)
    assert np.all(src == 5) and 5 not in dst.tolist()
    counts = np.zeros(n, np.int64)
    counts[dst] = cc
    counts = np.delete(counts, 5)
    assert counts.sum() == gamma
    assert stats.chisquare(counts).pvalue > 1e-4


def test_second_step_from_a_star_leaf_is_uniform():
    """Star with centre 0 and 30 leaves: from a leaf, step 1 is the centre
    (all walks), step 2 a uniform leaf (a return to the seed is dropped)."""
    leaves = 30
    n = leaves + 1
    edges = [(0, j) for j in range(1, n)] + [(j, 0) for j in range(1, n)]
    off, nbr = _csr(n, edges)
    gamma = 30_000
    src, dst, cc, hist = orc.sample_walks(off, nbr, n, gamma, 2, 2, True, seed=5,
                                          first_seed=4, num_seeds=1)
    centre = dst.tolist().index(0)
    assert hist[centre].tolist() == [gamma, 0]
    second = np.zeros(n, np.int64)
    for d, h in zip(dst, hist):
        second[d] += h[1]
    returns = gamma - second.sum()       # walks that came back to the seed at step 2
    obs = second[1:].copy()
    obs[4 - 1] = returns                 # the seed's share, dropped from the output
    assert stats.chisquare(obs).pvalue > 1e-4


def test_walks_stop_at_nodes_without_neighbours():
    # 0 -> 1 -> 2 -> 3 (3 has no out-edges); 4 isolated
    off, nbr = _csr(5, [(0, 1), (1, 2), (2, 3)])
    src, dst, cc, hist = orc.sample_walks(off, nbr, 5, 2, 6, 6, True, seed=1)
    triples = list(zip(src.tolist(), dst.tolist(), cc.tolist()))
    assert triples == [(0, 1, 2), (0, 2, 2), (0, 3, 2), (1, 2, 2), (1, 3, 2), (2, 3, 2)]
    assert hist[2].tolist() == [0, 0, 2, 0, 0, 0]


def test_bad_graph_is_an_error():
    off = np.array([0, 1, 2], np.int64)
    nbr = np.array([1, 5], np.int32)  # neighbour 5 does not exist
    with pytest.raises(orc.OracleError):
        orc.sample_walks(off, nbr, 2, 1, 3, 1, True, seed=0)


@pytest.mark.parametrize("seed_only", [True, False])
def test_seed_range_split_invariance(seed_only):
    rng = np.random.default_rng(4)
    n = 200
    edges = {(int(a), int(b)) for a, b in rng.integers(0, n, (1200, 2)) if a != b}
    off, nbr = _csr(n, list(edges))
    whole = orc.sample_walks(off, nbr, n, 3, 5, 3, seed_only, seed=9)
    parts = [orc.sample_walks(off, nbr, n, 3, 5, 3, seed_only, seed=9, first_seed=a,
                              num_seeds=b - a) for a, b in ((0, 77), (77, 150), (150, 200))]
    for i in range(4):
        assert np.array_equal(whole[i], np.concatenate([p[i] for p in parts]))
