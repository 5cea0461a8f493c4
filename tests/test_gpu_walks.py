"""GPU random-walk sampler (Sec. 3.2, Alg. 1) against the CPU oracle, through
the C ABI: triples, co_counts and distance histograms bit-exact, in the same
order, on SBM, random and deterministic graphs, for the paper's seed pairs
and for window pairs; errors (a malformed graph, too small a capacity) are
reported and write nothing; the triples feed the training step."""
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


def _graph(kind, n, seed=0):
    rng = np.random.default_rng(seed)
    if kind == "sbm":
        from synth import csr_from_edges, sbm_edges
        edges = sbm_edges(n, 10, 8.0, 1.0, rng)
        off, nbr = csr_from_edges(n, edges)
    elif kind == "random_with_sinks":
        # directed edges; a tenth of the nodes have no out-edges
        m = 6 * n
        a = rng.integers(0, n, m)
        b = rng.integers(0, n, m)
        keep = (a % 10) != 3
        a, b = a[keep], b[keep]
        order = np.lexsort((b, a))
        a, b = a[order], b[order]
        off = np.zeros(n + 1, np.int64)
        np.add.at(off, a + 1, 1)
        off = np.cumsum(off)
        nbr = b.astype(np.int32)
    elif kind == "cycle":
        off = np.arange(n + 1, dtype=np.int64)
        nbr = ((np.arange(n) + 1) % n).astype(np.int32)
    else:
        raise ValueError(kind)
    return np.asarray(off, np.int64), np.asarray(nbr, np.int32)


CASES = [
    # graph, n, walks, steps, window, seed_only, note
    ("sbm", 3000, 128, 3, 3, True, "the paper's sampler: 128 walks of 3 steps per node"),
    ("sbm", 2000, 4, 10, 2, False, "tiny workload's walks: window pairs"),
    ("random_with_sinks", 5000, 8, 20, 3, False, "dead ends, window 3"),
    ("random_with_sinks", 5000, 16, 12, 12, True, "dead ends, seed pairs"),
    ("cycle", 257, 3, 64, 32, True, "deterministic walks, longest walk and window"),
    ("sbm", 1500, 1024, 3, 1, True, "most walks per seed"),
    ("sbm", 1000, 1, 40, 5, False, "one long walk per seed"),
]


@pytest.mark.parametrize("kind,n,walks,steps,window,seed_only,note", CASES)
def test_walk_triples_bit_exact(kind, n, walks, steps, window, seed_only, note):
    say(f"walks {kind} n={n} walks={walks} steps={steps} window={window} seed_only={seed_only}")
    off, nbr = _graph(kind, n, seed=n)
    first, count = 17, n - 40
    ref = orc.sample_walks(off, nbr, n, walks, steps, window, seed_only, seed=99,
                           first_seed=first, num_seeds=count)
    got = P.sample_walks(dev(off, torch), dev(nbr, torch), n, walks, steps, window, seed_only,
                         seed=99, first_seed=first, num_seeds=count)
    for name, g, r in zip(("src", "dst", "cc", "hist"), got, ref):
        g = g.cpu().numpy()
        assert g.shape == r.shape, (name, g.shape, r.shape)
        assert np.array_equal(g, r), name


def test_capacity_and_malformed_graph_are_reported():
    n = 500
    off, nbr = _graph("sbm", n, seed=1)
    doff, dnbr = dev(off, torch), dev(nbr, torch)
    src, dst, cc, hist = P.sample_walks(doff, dnbr, n, 8, 5, 2, True, seed=3)
    need = src.numel()
    with pytest.raises(P.HugeError) as e:
        P.sample_walks(doff, dnbr, n, 8, 5, 2, True, seed=3, capacity=need - 1)
    assert e.value.status == -4
    bad = nbr.copy()
    v = int(np.argmax(np.diff(off) > 0))     # a seed with neighbours: its first step is bad
    bad[off[v]:off[v + 1]] = n + 5
    with pytest.raises(P.HugeError) as e:
        P.sample_walks(doff, dev(bad, torch), n, 8, 5, 2, True, seed=3)
    assert e.value.status == -2
    # host-side argument checks
    with pytest.raises(P.HugeError):
        P.sample_walks(doff, dnbr, n, 2000, 5, 2, True)       # too many walks per seed
    with pytest.raises(P.HugeError):
        P.sample_walks(doff, dnbr, n, 8, 5, 6, True)          # window > steps
    with pytest.raises(P.HugeError):
        P.sample_walks(doff, dnbr, n, 8, 5, 2, True, first_seed=400, num_seeds=200)


def test_walk_triples_train_like_the_oracle():
    """Triples produced on the GPU train one step; the oracle produces its own
    triples from the same graph and takes the same step."""
    n, D, K = 4000, 32, 5
    off, nbr = _graph("sbm", n, seed=5)
    src, dst, cc, _ = P.sample_walks(dev(off, torch), dev(nbr, torch), n, 16, 4, 2, False,
                                     seed=8, with_hist=False)
    m = 3000
    tr = P.Trainer(n, D, K, m, seed=4)
    loss = tr.step(src[:m], dst[:m], cc[:m], 0, 0.05).item()
    assert tr.check() == 0
    rs, rd, rc, _ = orc.sample_walks(off, nbr, n, 16, 4, 2, False, seed=8)
    ids = np.arange(n)
    a = float(np.float32(0.5 / D))
    S = orc.init_rows(4, 0, ids, D, a)
    T = orc.init_rows(4, 1, ids, D, a)
    neg = orc.sample_negatives(4, 0, m, K, n)
    ref = orc.step_dense(S, T, rs[:m], rd[:m], rc[:m], neg, 0.05)
    assert loss == pytest.approx(ref, rel=1e-5)
    assert_close(tr.S.cpu().numpy(), S, "S")
    assert_close(tr.T.cpu().numpy(), T, "T")
