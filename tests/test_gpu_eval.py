"""GPU embedding evaluation (Sec. 4's unsupervised metrics) against the CPU
oracle, through the C ABI:
  - edge and non-edge pairs bit-exact (same Philox counters);
  - distances of normalised rows within the fp32 bound
    |d_gpu - d| <= (D + 16) 2^-24 max(d, 1) + 1e-6 (the norm, the scaling
    and the sum of squares each round once per element);
  - the summary of the GPU's own distances: counts exact, means and
    percentiles within 1e-12 relative of the oracle's on the same values;
  - the k nearest rows: fp32 distances from the expansion of d^2, within
    |d^2_gpu - d^2| <= 4 D 2^-24 + 1e-6; every returned row is among the
    exact k nearest up to that bound, and where the exact k-th and (k+1)-th
    distances are further apart than twice the bound, the ids equal the
    oracle's in order of (distance, id);
  - recall@k exact, from the GPU's ids;
  - ragged shapes (dimensions not a multiple of 128, several query passes,
    fewer rows than k) and bad ids reported by the status word."""
import math

import numpy as np
import pytest

torch = pytest.importorskip("torch")

from oracle import oracle as orc  # noqa: E402
import paper_2307_14490_amd as P  # noqa: E402
from gpu_common import dev, say  # noqa: E402

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    yield
    torch.cuda.synchronize()


def sorted_csr(n, a, b):
    """CSR of the directed edges a -> b, each list in ascending order."""
    order = np.lexsort((b, a))
    a, b = a[order], b[order]
    off = np.zeros(n + 1, np.int64)
    np.add.at(off, a + 1, 1)
    return np.cumsum(off).astype(np.int64), b.astype(np.int32)


def sbm_graph(n, seed=0):
    from synth import sbm_edges
    e = sbm_edges(n, 10, 8.0, 1.0, np.random.default_rng(seed))
    return sorted_csr(n, np.concatenate([e[:, 0], e[:, 1]]), np.concatenate([e[:, 1], e[:, 0]]))


def random_graph(n, m, seed=0):
    rng = np.random.default_rng(seed)
    a = rng.integers(0, n, m)
    b = rng.integers(0, n, m)
    keep = a != b
    return sorted_csr(n, a[keep], b[keep])


def dist_tol(D, d):
    return (D + 16) * 2.0 ** -24 * np.maximum(d, 1.0) + 1e-6


# --------------------------------------------------------------------------- pairs
@pytest.mark.parametrize("kind,n,ne,nn,tries", [
    ("sbm", 2000, 20000, 20000, 64),
    ("random", 5000, 7777, 3333, 8),
    ("dense", 30, 500, 2000, 4),      # most draws are edges: many failed non-edge pairs
])
def test_pairs_bit_exact(kind, n, ne, nn, tries):
    if kind == "sbm":
        off, nbr = sbm_graph(n)
    elif kind == "random":
        off, nbr = random_graph(n, 8 * n)
    else:
        a, b = np.meshgrid(np.arange(n), np.arange(n), indexing="ij")
        keep = (a != b) & ((a + b) % 7 != 0)
        off, nbr = sorted_csr(n, a[keep], b[keep])
    say(f"pairs {kind} n={n} edges={nbr.size} ne={ne} nn={nn}")
    u0, v0 = orc.eval_pairs(off, nbr, n, 99, ne, nn, tries)
    ev = P.Evaluator(n, 8, ne + nn)
    u, v = ev.pairs(dev(off, torch), dev(nbr, torch), n, 99, ne, nn, tries)
    assert np.array_equal(u.cpu().numpy(), u0)
    assert np.array_equal(v.cpu().numpy(), v0)
    if kind == "dense":
        assert np.any(u0[ne:] < 0)


def test_pairs_report_a_malformed_graph():
    n = 100
    off, nbr = random_graph(n, 500)
    bad = nbr.copy()
    bad[7] = n + 5                       # a neighbour id out of range
    ev = P.Evaluator(n, 8, 10000)
    with pytest.raises(P.HugeError):
        ev.pairs(dev(off, torch), dev(bad, torch), n, 1, 10000, 0)
    with pytest.raises(P.HugeError):
        ev.pairs(dev(off, torch), dev(nbr, torch)[:0], n, 1, 10, 0)   # edges requested, none


# --------------------------------------------------------------------------- distances
@pytest.mark.parametrize("N,D", [(1000, 4), (3000, 12), (3000, 128), (500, 512), (200, 1024)])
def test_distances_of_normalised_rows(N, D):
    rng = np.random.default_rng(N + D)
    T = rng.normal(size=(N, D)).astype(np.float32)
    T[5] = 0.0                            # a zero row
    T[6] = T[7] * 8.0                     # same direction
    n = 20000
    u = rng.integers(0, N, n).astype(np.int32)
    v = rng.integers(0, N, n).astype(np.int32)
    u[:4] = [5, 6, 5, -1]
    v[:4] = [9, 7, 5, -1]
    say(f"distances N={N} D={D}")
    ev = P.Evaluator(N, D, n)
    d = ev.distances(dev(T, torch), dev(u, torch), dev(v, torch)).cpu().numpy().astype(np.float64)
    ref = orc.pair_distances(T, u, v)
    assert np.isnan(d[3]) and np.isnan(ref[3])
    ok = ~np.isnan(ref)
    assert np.all(np.abs(d[ok] - ref[ok]) <= dist_tol(D, ref[ok]))
    assert d[0] == pytest.approx(1.0, abs=1e-6) and d[1] == pytest.approx(0.0, abs=1e-3)
    assert d[2] == 0.0


def test_distances_report_ids_out_of_range():
    T = torch.zeros((10, 8), device="cuda")
    ev = P.Evaluator(10, 8, 4)
    with pytest.raises(P.HugeError):
        ev.distances(T, dev(np.array([1, 10], np.int32), torch),
                     dev(np.array([2, 3], np.int32), torch))


# --------------------------------------------------------------------------- summary
@pytest.mark.parametrize("ne,nn,nan_frac", [(20000, 30000, 0.0), (1, 1, 0.0), (9000, 7000, 0.1),
                                            (0, 500, 0.0), (300, 0, 0.5), (1, 2, 1.0)])
def test_summary_of_the_gpus_distances(ne, nn, nan_frac):
    rng = np.random.default_rng(ne * 7 + nn)
    d = rng.uniform(0, 2, ne + nn).astype(np.float32)
    d[: (ne + nn) // 3] = np.round(d[: (ne + nn) // 3], 1)     # ties
    d[rng.random(ne + nn) < nan_frac] = np.nan
    q = [0, 1, 5, 10, 25, 33.3, 50, 75, 90, 99, 100]
    say(f"summary ne={ne} nn={nn} nan={nan_frac}")
    ev = P.Evaluator(10, 8, ne + nn)
    s = ev.summary(dev(d, torch), ne, nn, q)
    ref = orc.eval_summary(d[:ne].astype(np.float64), d[ne:].astype(np.float64), q)
    assert s["count_edge"] == ref.count_edge and s["count_non"] == ref.count_non
    for a, b in [(s["mean_edge"], ref.mean_edge), (s["mean_non"], ref.mean_non),
                 (s["snr"], ref.snr)] + list(zip(s["pct_edge"], ref.pct_edge)) + \
            list(zip(s["pct_non"], ref.pct_non)):
        if math.isnan(b):
            assert math.isnan(a)
        else:
            assert a == pytest.approx(b, rel=1e-12, abs=1e-15)


def test_summary_large_sort():
    """Several radix tiles per set: percentiles are order statistics of
    exactly the GPU's values."""
    rng = np.random.default_rng(5)
    ne, nn = 300_000, 700_001
    d = np.abs(rng.normal(1.0, 0.4, ne + nn)).astype(np.float32)
    q = list(np.linspace(0, 100, 101))
    ev = P.Evaluator(10, 8, ne + nn)
    s = ev.summary(dev(d, torch), ne, nn, q)
    ref = orc.eval_summary(d[:ne].astype(np.float64), d[ne:].astype(np.float64), q)
    assert s["pct_edge"] == pytest.approx(ref.pct_edge, rel=1e-12)
    assert s["pct_non"] == pytest.approx(ref.pct_non, rel=1e-12)
    assert s["mean_non"] == pytest.approx(ref.mean_non, rel=1e-12)


# --------------------------------------------------------------------------- nearest rows
def check_knn(T, queries, k, ids, dist):
    """The GPU's k nearest against exact (double) distances."""
    N, D = T.shape
    tol2 = 4 * D * 2.0 ** -24 + 1e-6
    Xn = orc.normalize_rows(T)
    oid, od = orc.knn(T, queries, k)
    for qi, u in enumerate(queries):
        got = ids[qi]
        m = min(k, N - 1)
        assert np.all(got[m:] == -1)
        g = got[:m].astype(np.int64)
        assert len(set(g.tolist())) == m and u not in g
        exact2 = np.sum((Xn[g] - Xn[u]) ** 2, axis=1)
        assert np.all(np.abs(dist[qi][:m].astype(np.float64) ** 2 - exact2) <= tol2 + 1e-6)
        kth2 = od[qi][m - 1] ** 2
        assert np.all(exact2 <= kth2 + 2 * tol2), (u, exact2.max(), kth2)
        # where no near-tie straddles the k-th place, the answer is unique
        all2 = np.sum((Xn - Xn[u]) ** 2, axis=1)
        all2[u] = np.inf
        srt = np.sort(all2)
        gaps = np.diff(srt[: m + 1])
        if m < N - 1 and np.all(gaps > 2 * tol2):
            assert g.tolist() == oid[qi][:m].tolist()


@pytest.mark.parametrize("N,D,nq,k,note", [
    (5000, 128, 100, 10, "the paper's 100 sampled nodes"),
    (20000, 128, 256, 16, "about 1.6% of rows hold a value that falls on an exact fp16 tie "
                          "once normalised and scaled: the split into two fp16 parts"),
    (4099, 32, 37, 32, "ragged tiles, k = 32, one block of queries"),
    (3000, 100, 70, 5, "dimensions not a multiple of 128, three blocks padded to four"),
    (2000, 256, 150, 8, "two query passes of 64 + 64 + 22"),
    (700, 512, 40, 16, "four dimension chunks"),
    (20, 16, 20, 32, "fewer rows than k: trailing -1"),
    (33, 8, 1, 1, "one query, one neighbour"),
    (9000, 128, 40, 7, "two query blocks of full-width rows, two threshold scans"),
    (12000, 128, 20, 12, "one query block of full-width rows, two threshold scans"),
    (300000, 64, 33, 32, "k = 32 over three threshold scans, half-width rows, two blocks"),
])
def test_knn_and_recall(N, D, nq, k, note):
    rng = np.random.default_rng(N + D + nq)
    T = rng.normal(size=(N, D)).astype(np.float32)
    T[3] = 0.0                                  # zero row
    T[4] = T[5] * 2.0                           # exact tie in direction
    if N > 12:
        T[10] = T[11]                           # identical rows
    queries = np.unique(np.concatenate([[0, 3, 4, N - 1], rng.integers(0, N, nq)]))[:nq]
    queries = queries.astype(np.int32)
    say(f"knn N={N} D={D} nq={queries.size} k={k} ({note})")
    ev = P.Evaluator(N, D, 8, k=max(k, 1))
    ids, dist = ev.knn(dev(T, torch), dev(queries, torch), k)
    ids = ids.cpu().numpy()
    dist = dist.cpu().numpy()
    check_knn(T, queries, k, ids, dist)
    # the per-wave list search computes the same distances: the same answer, bit for bit
    ids_l, dist_l = ev.knn(dev(T, torch), dev(queries, torch), k, lists=True)
    assert np.array_equal(ids, ids_l.cpu().numpy())
    assert np.array_equal(dist.view(np.int32), dist_l.cpu().numpy().view(np.int32))
    off, nbr = random_graph(N, 6 * N, seed=N)
    rec = ev.recall(dev(off, torch), dev(nbr, torch), N, dev(queries, torch),
                    dev(ids, torch)).cpu().numpy()
    m = min(k, N - 1)
    want = orc.recall_at_k(off, nbr, queries, ids[:, :m], k) if m == k else None
    if want is not None:
        assert np.array_equal(rec, want)
    else:
        # fewer rows than k: the -1 entries are not neighbours; divided by k
        want = orc.recall_at_k(off, nbr, queries, ids[:, :m], m) * m / k
        assert np.allclose(rec, want, rtol=0, atol=1e-15)


def test_recall_on_an_embedding_that_reconstructs_the_graph():
    """Points on a circle linked to their 2 nearest: recall@2 = 1 for every
    query, recall@4 = 1/2."""
    n, D = 720, 8
    ang = 2 * np.pi * np.arange(n) / n
    T = np.zeros((n, D), np.float32)
    T[:, 0] = np.cos(ang)
    T[:, 1] = np.sin(ang)
    a = np.repeat(np.arange(n), 2)
    b = np.stack([(np.arange(n) - 1) % n, (np.arange(n) + 1) % n], 1).reshape(-1)
    off, nbr = sorted_csr(n, a, b)
    q = np.arange(0, n, 7).astype(np.int32)
    ev = P.Evaluator(n, D, 8, k=4)
    ids2, _ = ev.knn(dev(T, torch), dev(q, torch), 2)
    r2 = ev.recall(dev(off, torch), dev(nbr, torch), n, dev(q, torch), ids2).cpu().numpy()
    assert np.all(r2 == 1.0)
    ids4, _ = ev.knn(dev(T, torch), dev(q, torch), 4)
    r4 = ev.recall(dev(off, torch), dev(nbr, torch), n, dev(q, torch), ids4).cpu().numpy()
    assert np.all(r4 == 0.5)


@pytest.mark.parametrize("n_others", [99, 20])
def test_knn_falls_back_to_the_list_search_when_a_candidate_list_overflows(n_others):
    """18,000 copies of row 5 lie at one distance from query 5, so its last
    threshold scan keeps more candidates than a list holds (8192): that pass is
    computed again by the list search (four query blocks with 99 other
    queries, one with 20).  Its answer for the other queries equals both
    searches' answer without query 5, bit for bit, and query 5's k nearest are
    the copies with the smallest ids."""
    N, D, k = 30000, 128, 10
    rng = np.random.default_rng(77)
    T = rng.normal(size=(N, D)).astype(np.float32)
    T[12000:] = T[5]
    others = np.setdiff1d(rng.choice(12000, 120, replace=False), [5])[:n_others]
    others = others.astype(np.int32)
    with_5 = np.concatenate([[5], others]).astype(np.int32)
    say(f"knn overflow N={N} D={D} k={k} queries={with_5.size}")
    ev = P.Evaluator(N, D, 8, k=k)
    Td = dev(T, torch)
    ids_a, dist_a = (a.cpu().numpy() for a in ev.knn(Td, dev(with_5, torch), k))
    ids_b, dist_b = (a.cpu().numpy() for a in ev.knn(Td, dev(others, torch), k))
    ids_c, dist_c = (a.cpu().numpy() for a in ev.knn(Td, dev(others, torch), k, lists=True))
    assert ids_a[0].tolist() == list(range(12000, 12000 + k))
    for ids, dist in ((ids_b, dist_b), (ids_c, dist_c)):
        assert np.array_equal(ids_a[1:], ids)
        assert np.array_equal(dist_a[1:].view(np.int32), dist.view(np.int32))
    check_knn(T, others[:20], k, ids_b[:20], dist_b[:20])


def test_knn_threshold_scans_at_a_million_rows():
    """1e6 x 128 rows, 100 queries, k = 10: three threshold scans (31, 977 and
    31,250 tiles of 32 rows).  Bit for bit the list search's answer; the
    first 4 queries against exact double distances."""
    N, D, k, nq = 1_000_000, 128, 10, 100
    g = torch.Generator(device="cuda")
    g.manual_seed(11)
    Td = torch.randn((N, D), generator=g, device="cuda", dtype=torch.float32)
    rng = np.random.default_rng(12)
    queries = rng.choice(N, nq, replace=False).astype(np.int32)
    say(f"knn N={N} D={D} nq={nq} k={k}")
    ev = P.Evaluator(N, D, 8, k=k)
    ids, dist = (a.cpu().numpy() for a in ev.knn(Td, dev(queries, torch), k))
    ids_l, dist_l = (a.cpu().numpy() for a in ev.knn(Td, dev(queries, torch), k, lists=True))
    assert np.array_equal(ids, ids_l)
    assert np.array_equal(dist.view(np.int32), dist_l.view(np.int32))
    check_knn(Td.cpu().numpy(), queries[:4], k, ids[:4], dist[:4])


def test_knn_reports_bad_query_ids():
    T = torch.randn((100, 16), device="cuda")
    ev = P.Evaluator(100, 16, 8, k=4)
    with pytest.raises(P.HugeError):
        ev.knn(T, dev(np.array([3, 100], np.int32), torch), 4)
    with pytest.raises(P.HugeError):
        ev.knn(T, dev(np.array([-1], np.int32), torch), 4)


# --------------------------------------------------------------------------- end to end
def test_evaluation_of_trained_embeddings_matches_the_oracle():
    """The tiny SBM workload trained for three epochs on the GPU, then evaluated:
    SNR and percentiles of the GPU path equal the oracle's evaluation of the
    same tables within the distance bound, and training has separated edges
    from non-edges (SNR well above 1, edges nearer than non-edges at every
    percentile)."""
    from synth import gen
    wl = gen.make_workload("tiny")
    cfg = wl.cfg
    N = cfg.num_nodes
    tr = P.Trainer(N, cfg.dim, cfg.num_neg, cfg.batch, seed=3)
    es, ed, ec = (dev(x, torch) for x in wl.epoch())
    pos = 0
    for _ in range(3):
        for i0 in range(0, es.numel(), cfg.batch):
            i1 = min(i0 + cfg.batch, es.numel())
            tr.step_no_loss(es[i0:i1], ed[i0:i1], ec[i0:i1], pos, cfg.lr)
            pos += i1 - i0
    assert tr.check() == 0
    # the graph in the trained id space (the batches' ids are relabelled)
    off0, nbr0 = wl.csr
    a = gen.relabel(np.repeat(np.arange(N), np.diff(off0)), N, wl.perm)
    b = gen.relabel(np.asarray(nbr0, np.int64), N, wl.perm)
    off, nbr = sorted_csr(N, a, b)
    S = tr.S
    ne, nn = 20000, 20000
    ev = P.Evaluator(N, cfg.dim, ne + nn, k=10)
    u, v = ev.pairs(dev(off, torch), dev(nbr, torch), N, 5, ne, nn)
    d = ev.distances(S, u, v)
    q = [0, 10, 25, 50, 75, 90, 100]
    s = ev.summary(d, ne, nn, q)
    Sh = S.cpu().numpy()
    ref_d = orc.pair_distances(Sh, u.cpu().numpy(), v.cpu().numpy())
    ref = orc.eval_summary(ref_d[:ne], ref_d[ne:], q)
    tol = dist_tol(cfg.dim, 2.0)
    assert s["count_edge"] == ref.count_edge and s["count_non"] == ref.count_non
    assert abs(s["mean_edge"] - ref.mean_edge) <= tol
    assert abs(s["mean_non"] - ref.mean_non) <= tol
    assert np.all(np.abs(np.array(s["pct_edge"]) - ref.pct_edge) <= tol)
    assert np.all(np.abs(np.array(s["pct_non"]) - ref.pct_non) <= tol)
    assert s["snr"] > 2.0
    assert np.all(np.array(s["pct_edge"][1:-1]) < np.array(s["pct_non"][1:-1]))
    say(f"trained tiny: SNR {s['snr']:.3f}, edge median {s['pct_edge'][3]:.3f}, "
        f"non-edge median {s['pct_non'][3]:.3f}")
