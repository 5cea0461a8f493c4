"""Weighted co-occurrences on the GPU (Sec. 3.2: co_counts is a histogram over
the walk distance): weights from distance histograms bit-exact with the
oracle; the step with float weights against the oracle's weighted step
(sorted and atomic scatter, same tolerance as the integer step); integer-
valued weights bitwise equal to the integer step; prepared weighted steps
bitwise equal to the direct ones; invalid weights rejected as a no-op; and
the sampler's histograms weighted and trained end to end."""
import numpy as np
import pytest

torch = pytest.importorskip("torch")

from oracle import oracle as orc  # noqa: E402
import paper_2307_14490_amd as P  # noqa: E402
from gpu_common import assert_close, dev, say  # noqa: E402

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    yield
    torch.cuda.synchronize()


def _half(D):
    return float(np.float32(0.5 / D))


@pytest.mark.parametrize("n,window,hmax", [(5000, 3, 50), (777, 1, 10), (2000, 32, 1 << 30),
                                           (1, 7, 3)])
def test_cocount_weights_bit_exact(n, window, hmax):
    rng = np.random.default_rng(n + window)
    hist = rng.integers(0, hmax, size=(n, window)).astype(np.int32)
    hist[::5] = 0
    for wd in (np.ones(window), 1.0 / np.arange(1, window + 1),
               rng.uniform(0, 3, window), np.linspace(0, 1, window)):
        wd = wd.astype(np.float32)
        say(f"weights n={n} window={window} wd={wd[:3]}")
        got = P.cocount_weights(dev(hist, torch), wd).cpu().numpy()
        ref = orc.cocount_weights(hist, wd)
        assert np.array_equal(got.view(np.uint32), ref.view(np.uint32))


def _weighted_step(N, D, K, n, scatter, w, seed=5, lr=0.05):
    rng = np.random.default_rng(N + n)
    src = rng.integers(0, N, n).astype(np.int32)
    dst = rng.integers(0, N, n).astype(np.int32)
    first = 321
    tr = P.Trainer(N, D, K, n, seed=seed, scatter=scatter)
    loss = tr.step(dev(src, torch), dev(dst, torch), dev(w, torch), first, lr).item()
    assert tr.check() == 0
    ids = np.arange(N)
    S = orc.init_rows(seed, 0, ids, D, _half(D))
    T = orc.init_rows(seed, 1, ids, D, _half(D))
    neg = orc.sample_negatives(seed, first, n, K, N)
    ref = orc.step_dense(S, T, src, dst, w, neg, lr)
    return tr, (src, dst, neg), (S, T, ref, loss)


@pytest.mark.parametrize("scatter", ["sorted", "atomic"])
@pytest.mark.parametrize("N,D,K,n", [(3000, 32, 5, 2000), (200, 128, 3, 1500), (50, 8, 10, 500)])
def test_weighted_step_matches_oracle(scatter, N, D, K, n):
    rng = np.random.default_rng(N * 3 + K)
    w = (rng.gamma(0.7, 2.0, n)).astype(np.float32)
    w[::9] = 0.0
    say(f"weighted step {scatter} N={N} D={D} K={K} n={n}")
    tr, _, (S, T, ref, loss) = _weighted_step(N, D, K, n, scatter, w)
    if scatter == "sorted":
        assert_close(tr.S.cpu().numpy(), S, "S weighted")
        assert_close(tr.T.cpu().numpy(), T, "T weighted")
    else:
        # the atomic scatter adds in arbitrary order: rows hit many times are
        # held to the bound of the integer atomic tests (1e-4 of the update)
        gS, gT = tr.S.cpu().numpy(), tr.T.cpu().numpy()
        S0 = orc.init_rows(5, 0, np.arange(N), D, _half(D))
        T0 = orc.init_rows(5, 1, np.arange(N), D, _half(D))
        for name, G, R, R0 in (("S", gS, S, S0), ("T", gT, T, T0)):
            upd = np.linalg.norm(R.astype(np.float64) - R0, axis=1)
            err = np.linalg.norm(G.astype(np.float64) - R, axis=1)
            assert np.all(err <= 1e-4 * upd + 1e-5), name
    assert loss == pytest.approx(ref, rel=1e-5, abs=1e-6)


def test_integer_valued_weights_equal_the_integer_step():
    N, D, K, n = 1000, 64, 5, 3000
    rng = np.random.default_rng(8)
    src = rng.integers(0, N, n).astype(np.int32)
    dst = rng.integers(0, N, n).astype(np.int32)
    cc = rng.integers(0, 30, n).astype(np.int32)
    a = P.Trainer(N, D, K, n, seed=2)
    b = P.Trainer(N, D, K, n, seed=2)
    la = a.step(dev(src, torch), dev(dst, torch), dev(cc, torch), 0, 0.05).item()
    lb = b.step(dev(src, torch), dev(dst, torch), dev(cc.astype(np.float32), torch), 0, 0.05).item()
    assert la == lb
    assert torch.equal(a.S, b.S) and torch.equal(a.T, b.T)
    ea = a.eval_loss(dev(src, torch), dev(dst, torch), dev(cc, torch), 7).item()
    eb = b.eval_loss(dev(src, torch), dev(dst, torch), dev(cc.astype(np.float32), torch), 7).item()
    assert ea == eb


def test_prepared_weighted_steps_equal_direct_ones():
    N, D, K, n = 2000, 32, 4, 1500
    rng = np.random.default_rng(9)
    batches = [(rng.integers(0, N, n).astype(np.int32), rng.integers(0, N, n).astype(np.int32),
                rng.uniform(0, 4, n).astype(np.float32)) for _ in range(4)]
    ref = P.Trainer(N, D, K, n, seed=3)
    for k, (s, d, w) in enumerate(batches):
        ref.step_no_loss(dev(s, torch), dev(d, torch), dev(w, torch), k * n, 0.05)
    tr = P.Trainer(N, D, K, n, seed=3)
    side = torch.cuda.Stream()
    db = [tuple(dev(x, torch) for x in b) for b in batches]
    tr.prepare(*db[0], 0, stream=side)
    for k in range(len(db)):
        if k + 1 < len(db):
            tr.prepare(*db[k + 1], (k + 1) * n, stream=side)
        tr.train_prepared(0.05, with_loss=False)
    torch.cuda.synchronize()
    assert tr.check() == 0 and ref.check() == 0
    assert torch.equal(tr.S, ref.S) and torch.equal(tr.T, ref.T)


@pytest.mark.parametrize("bad", [-0.5, float("nan"), float("inf")])
def test_invalid_weights_make_the_step_a_no_op(bad):
    N, D, K, n = 100, 16, 3, 64
    rng = np.random.default_rng(10)
    src = rng.integers(0, N, n).astype(np.int32)
    dst = rng.integers(0, N, n).astype(np.int32)
    w = np.ones(n, np.float32)
    w[13] = bad
    tr = P.Trainer(N, D, K, n, seed=1)
    S0, T0 = tr.S.clone(), tr.T.clone()
    loss = tr.step(dev(src, torch), dev(dst, torch), dev(w, torch), 0, 0.1).item()
    assert np.isnan(loss)
    assert torch.equal(tr.S, S0) and torch.equal(tr.T, T0)
    assert tr.check() == P.binding.HUGE_ERR_BAD_COUNT


def test_sampler_histograms_weighted_and_trained():
    """Walk triples with their distance histograms (Alg. 1), weighted 1/d,
    trained for a step: tables and loss match the oracle's weighted step on
    the oracle's own triples."""
    from synth import csr_from_edges, sbm_edges
    n_nodes, D, K = 2000, 32, 5
    e = sbm_edges(n_nodes, 10, 8.0, 1.0, np.random.default_rng(4))
    off, nbr = csr_from_edges(n_nodes, e)
    src, dst, cc, hist = P.sample_walks(dev(off, torch), dev(nbr, torch), n_nodes, 4, 10, 3,
                                        False, 11)
    osrc, odst, occ, ohist = orc.sample_walks(off, nbr, n_nodes, 4, 10, 3, False, 11)
    assert np.array_equal(src.cpu().numpy(), osrc) and np.array_equal(hist.cpu().numpy(), ohist)
    wd = np.array([1.0, 0.5, 1.0 / 3.0], np.float32)
    w = P.cocount_weights(hist, wd)
    ow = orc.cocount_weights(ohist, wd)
    assert np.array_equal(w.cpu().numpy(), ow)
    m = min(src.numel(), 20000)
    tr = P.Trainer(n_nodes, D, K, m, seed=6)
    loss = tr.step(src[:m], dst[:m], w[:m], 0, 0.025).item()
    ids = np.arange(n_nodes)
    S = orc.init_rows(6, 0, ids, D, _half(D))
    T = orc.init_rows(6, 1, ids, D, _half(D))
    neg = orc.sample_negatives(6, 0, m, K, n_nodes)
    ref = orc.step_dense(S, T, osrc[:m], odst[:m], ow[:m], neg, 0.025)
    assert_close(tr.S.cpu().numpy(), S, "S")
    assert_close(tr.T.cpu().numpy(), T, "T")
    assert loss == pytest.approx(ref, rel=1e-5, abs=1e-6)
