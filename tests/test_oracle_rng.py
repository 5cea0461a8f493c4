"""Pins for the oracle's random streams: Philox4x32-10, the negative sampler,
the alias table and the table initialiser.

Everything here checks the oracle against facts that do not come from the
oracle itself: published known-answer vectors, an independent open-source
Philox (rocRAND's host-callable engine), exact integer enumeration of alias
probabilities, and goodness-of-fit statistics.
"""
import os
import shutil
import subprocess

import numpy as np
import pytest
from scipy import stats

from oracle import oracle as orc

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _kat_rows():
    rows = []
    with open(os.path.join(GOLDEN, "philox4x32_10_kat.txt")) as f:
        for line in f:
            if line.startswith("#") or not line.strip():
                continue
            v = [int(x, 16) for x in line.split()]
            rows.append((v[0:4], v[4:6], v[6:10]))
    return rows


@pytest.mark.parametrize("ctr,key,expect", _kat_rows())
def test_philox_known_answers(ctr, key, expect):
    assert list(orc.philox4x32_10(ctr, key)) == expect


_ROCRAND_PROG = r"""
#include <cstdio>
#include <cstdlib>
#include <rocrand/rocrand_philox4x32_10.h>
int main(int argc, char** argv) {
  // Prints Philox4x32-10 blocks for counters (lo(c), hi(c), lo(s), hi(s))
  // under key (lo(seed), hi(seed)), via rocRAND's engine:
  // subsequence s sets counter words 2..3, offset 4*c sets words 0..1.
  unsigned long long seed = strtoull(argv[1], 0, 0);
  for (int a = 2; a + 1 < argc; a += 2) {
    unsigned long long c = strtoull(argv[a], 0, 0), s = strtoull(argv[a + 1], 0, 0);
    rocrand_device::philox4x32_10_engine e(seed, s, 4ull * c);
    unsigned w0 = e.next(), w1 = e.next(), w2 = e.next(), w3 = e.next();
    printf("%u %u %u %u\n", w0, w1, w2, w3);
  }
  return 0;
}
"""


@pytest.mark.slow
def test_philox_matches_rocrand_host_engine(tmp_path):
    """Independent implementation: rocRAND's open-source header, host side."""
    hipcc = shutil.which("hipcc")
    if hipcc is None or not os.path.exists("/opt/rocm/include/rocrand/rocrand_philox4x32_10.h"):
        pytest.skip("hipcc / rocRAND headers not available")
    src = tmp_path / "p.cpp"
    src.write_text(_ROCRAND_PROG)
    exe = tmp_path / "p"
    r = subprocess.run([hipcc, "--offload-host-only", "-O1", "-o", str(exe), str(src)],
                       capture_output=True, text=True)
    if r.returncode != 0:
        pytest.skip("could not build rocRAND host probe: " + r.stderr[-400:])
    seed = 0x0123456789ABCDEF
    rng = np.random.default_rng(7)
    # the engine takes a number offset of 4 c, so c stays below 2^62
    cases = [(int(c), int(s)) for c, s in zip(rng.integers(0, 2**62, 20),
                                               rng.integers(0, 2**63, 20))]
    cases += [(0, 0), (2**62 - 1, 2**64 - 1), (5, 1), (12345, 3)]
    args = [str(exe), str(seed)]
    for c, s in cases:
        args += [str(c), str(s)]
    out = subprocess.run(args, capture_output=True, text=True, check=True).stdout.split("\n")
    key = [seed & 0xFFFFFFFF, seed >> 32]
    for (c, s), line in zip(cases, out):
        ctr = [c & 0xFFFFFFFF, c >> 32, s & 0xFFFFFFFF, s >> 32]
        assert list(orc.philox4x32_10(ctr, key)) == [int(x) for x in line.split()]


# --------------------------------------------------------------------------- #
# Uniform negatives
# --------------------------------------------------------------------------- #
def test_uniform_negatives_power_of_two_is_top_bits():
    """For N = 2^b the bucket floor(x N / 2^64) is the top b bits of x."""
    seed, N, b = 99, 1 << 10, 10
    key = [seed & 0xFFFFFFFF, seed >> 32]
    neg = orc.sample_negatives(seed, 1000, 50, 3, N)
    for i in range(50):
        for k in range(3):
            r = orc.philox4x32_10([1000 + i, 0, k, 1], key)
            x = (int(r[1]) << 32) | int(r[0])
            assert neg[i, k] == x >> (64 - b)


def test_uniform_negatives_chi_square_and_range():
    N = 1000
    neg = orc.sample_negatives(12345, 0, 200_000, 5, N).reshape(-1)
    assert neg.min() >= 0 and neg.max() < N
    counts = np.bincount(neg, minlength=N)
    chi2, p = stats.chisquare(counts)
    assert p > 1e-4, (chi2, p)


def test_negatives_depend_only_on_global_position():
    """Splitting a batch differently does not change any negative."""
    full = orc.sample_negatives(7, 10, 100, 4, 977)
    a = orc.sample_negatives(7, 10, 37, 4, 977)
    b = orc.sample_negatives(7, 47, 63, 4, 977)
    assert np.array_equal(full, np.concatenate([a, b]))
    # slots and positions are distinct streams
    assert not np.array_equal(full[:, 0], full[:, 1])
    other_seed = orc.sample_negatives(8, 10, 100, 4, 977)
    assert not np.array_equal(full, other_seed)


def test_uniform_negatives_large_n_range():
    N = 100_000_000
    neg = orc.sample_negatives(3, 2**40, 20000, 5, N)
    assert neg.min() >= 0 and neg.max() < N
    # roughly uniform over [0, N): deciles
    h = np.histogram(neg, bins=10, range=(0, N))[0]
    assert stats.chisquare(h).pvalue > 1e-4


# --------------------------------------------------------------------------- #
# Alias table
# --------------------------------------------------------------------------- #
def _alias_counts(thr, alias):
    """Exact number of (bucket, coin) pairs out of N * 2^32 that yield each id."""
    N = thr.size
    one = 1 << 32
    counts = [0] * N
    for j in range(N):
        t = int(thr[j])
        counts[j] += t                     # coin r < thr[j] -> j
        counts[int(alias[j])] += one - t   # otherwise -> alias[j]
    return counts


@pytest.mark.parametrize("weights", [
    [1.0, 2.0, 3.0, 4.0],
    [0.0, 5.0, 0.0, 1.0, 1.0],
    [1.0] * 7,
    [3.0],
    list(np.random.default_rng(0).pareto(1.5, 300) + 0.01),
    list((np.arange(1, 501) ** -1.1) ** 0.75),
])
def test_alias_table_exact_probabilities(weights):
    w = np.asarray(weights, np.float64)
    thr, alias = orc.build_alias(w)
    N = w.size
    one = 1 << 32
    counts = _alias_counts(thr, alias)
    assert sum(counts) == N * one
    ideal = w / w.sum() * N * one
    err = np.abs(np.asarray(counts, np.float64) - ideal)
    # truncation leaves each bucket within one unit of the ideal mass except the
    # largest one, which absorbs the total residue (at most N units).
    big = int(np.argmax(ideal))
    others = np.delete(err, big)
    assert np.all(others <= 2.0 + 1e-6 * ideal.max())
    assert err[big] <= N + 2 + 1e-6 * ideal.max()
    # zero weights are never produced
    for j in np.nonzero(w == 0)[0]:
        assert counts[j] == 0
    assert np.all((alias >= 0) & (alias < N))


def test_alias_uniform_weights_are_identity():
    thr, alias = orc.build_alias(np.ones(16))
    assert np.all(thr == 0xFFFFFFFF)
    assert np.array_equal(alias, np.arange(16))


def test_alias_sampler_chi_square():
    rng = np.random.default_rng(5)
    w = rng.integers(1, 50, 200).astype(np.float64) ** 0.75
    thr, alias = orc.build_alias(w)
    neg = orc.sample_negatives(11, 0, 100_000, 4, w.size, thr, alias).reshape(-1)
    counts = np.bincount(neg, minlength=w.size)
    exp = w / w.sum() * neg.size
    chi2, p = stats.chisquare(counts, exp)
    assert p > 1e-4, (chi2, p)


def test_alias_rejects_bad_weights():
    with pytest.raises(orc.OracleError):
        orc.build_alias(np.zeros(4))
    with pytest.raises(orc.OracleError):
        orc.build_alias(np.array([1.0, -1.0]))
    with pytest.raises(orc.OracleError):
        orc.build_alias(np.array([1.0, np.nan]))


# --------------------------------------------------------------------------- #
# Initialiser
# --------------------------------------------------------------------------- #
@pytest.mark.parametrize("dim", [32, 128, 36])
def test_init_range_grid_and_uniformity(dim):
    a = 0.5 / dim
    rows = np.arange(0, 4000, 7)
    S = orc.init_rows(3, 0, rows, dim, np.float32(a))
    T = orc.init_rows(3, 1, rows, dim, np.float32(a))
    a32 = float(np.float32(a))
    for X in (S, T):
        assert X.min() >= -a32 and X.max() < a32
        # every value is fp32(j * scale) for an integer j in [-2^23, 2^23) and
        # scale = fp32(a) * 2^-23; when a is a power of two the product is exact
        scale = np.float32(a32 * 2.0 ** -23)
        q = X.astype(np.float64) / float(scale)
        j = np.round(q)
        assert np.array_equal((j.astype(np.float32) * scale).astype(np.float32), X)
        assert j.min() >= -2**23 and j.max() < 2**23
        if dim & (dim - 1) == 0:
            assert np.all(q == j)
        # uniform on [-a, a): KS test per column position within a Philox block
        for w in range(4):
            col = X[:, w::4].reshape(-1)
            assert stats.kstest(col, stats.uniform(loc=-a32, scale=2 * a32).cdf).pvalue > 1e-4
    assert not np.array_equal(S, T)
    assert abs(np.corrcoef(S.reshape(-1), T.reshape(-1))[0, 1]) < 0.05


def test_init_is_position_addressed():
    a = np.float32(0.01)
    r1 = orc.init_rows(9, 1, [5, 1_000_000_007, 5], 8, a)
    assert np.array_equal(r1[0], r1[2])
    assert not np.array_equal(r1[0], r1[1])
    assert orc.init_value(9, 1, 1_000_000_007, 6, float(a)) == r1[1, 6]
    # rows past 2^32 use the high counter word
    hi = orc.init_rows(9, 0, [5 + (1 << 32)], 8, a)
    lo = orc.init_rows(9, 0, [5], 8, a)
    assert not np.array_equal(hi, lo)


def test_init_rows_agree_with_elementwise_definition():
    rows = np.array([0, 3, 77, 2**33 + 5])
    for dim in (4, 10, 32):
        R = orc.init_rows(17, 1, rows, dim, np.float32(0.02))
        for a, r in enumerate(rows):
            for c in range(dim):
                assert R[a, c] == np.float32(orc.init_value(17, 1, int(r), c, 0.02))
