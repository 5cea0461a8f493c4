"""GPU parity of libhuge against the CPU oracle, through the C ABI.

Bit-exact: initial tables, sampled negatives, rows a step does not touch, the
row counts of the grouping, run-to-run results of the sorted scatter.
Within |gpu - oracle| <= 1e-6 + 1e-5 |oracle|: every touched table element
after a step, for both scatter variants.  Loss sums within 1e-5 relative.
"""
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


def _trainer(N, D, K, nmax, seed=0, weights=None, scatter="sorted", a=0.0):
    tr = P.Trainer(N, D, K, nmax, seed=seed, init_half_width=a, alias_weights=weights,
                   scatter=scatter)
    torch.cuda.synchronize()
    return tr


def _half(D, a=0.0):
    return float(np.float32(a if a else 0.5 / D))


def _random_batch(rng, N, n, cmax=5, hub_frac=0.0):
    src = rng.integers(0, N, n).astype(np.int32)
    dst = rng.integers(0, N, n).astype(np.int32)
    cc = rng.integers(0, cmax + 1, n).astype(np.int32)
    if hub_frac > 0:
        k = int(n * hub_frac)
        src[:k] = 1 % N
        dst[k // 2:k] = 0
    return src, dst, cc


# --------------------------------------------------------------------------- #
# Bit-exact random streams
# --------------------------------------------------------------------------- #
@pytest.mark.parametrize("N,D,a", [(10_000, 32, 0.0), (777, 36, 0.0), (50, 1024, 0.3)])
def test_init_tables_bit_exact(N, D, a):
    say(f"init N={N} D={D}")
    tr = _trainer(N, D, 5, 16, seed=1234, a=a)
    S = tr.S.cpu().numpy()
    T = tr.T.cpu().numpy()
    ids = np.arange(N)
    assert np.array_equal(S, orc.init_rows(1234, 0, ids, D, _half(D, a)))
    assert np.array_equal(T, orc.init_rows(1234, 1, ids, D, _half(D, a)))


@pytest.mark.parametrize("kind", ["uniform", "alias"])
@pytest.mark.parametrize("N,n,first", [(10_000, 1024, 0), (99_991, 1037, 2**33 + 5),
                                       (3, 513, 7), (100_000_000, 4096, 12345)])
def test_negatives_bit_exact(kind, N, n, first):
    say(f"negatives {kind} N={N} n={n} first={first}")
    w = None
    thr = alias = None
    if kind == "alias":
        # at N = 1e8 the host alias tables (library and oracle) take a few
        # seconds and a few GB of host memory each
        rng = np.random.default_rng(N)
        w = (rng.pareto(1.1, N) + 0.1) ** 0.75
        w[::7] = 0.0
        thr, alias = orc.build_alias(w)
    tr = _trainer(N, 8, 7, max(n, 1), seed=99, weights=w)
    got = tr.sample_negatives(n, first).cpu().numpy()
    ref = orc.sample_negatives(99, first, n, 7, N, thr, alias)
    assert np.array_equal(got, ref)


# --------------------------------------------------------------------------- #
# One step against the dense oracle
# --------------------------------------------------------------------------- #
STEP_CASES = [
    # N, D, K, n, note
    (10_000, 32, 5, 1024, "tiny shape"),
    (1_000, 36, 3, 777, "D/4 not a power of two, ragged n"),
    (500, 512, 2, 300, "two float4 per lane"),
    (300, 1024, 1, 100, "widest row, K=1"),
    (50, 4, 20, 64, "narrowest row, several negative blocks"),
    (2, 8, 5, 50, "two nodes: every row repeats"),
    (1_000, 128, 64, 100, "largest K"),
    (3_000, 32, 13, 2_000, "K = 13: two negative blocks, indices staged, ragged last workgroup"),
    (20_000, 128, 5, 9000, "several sort tiles"),
    (100_000, 16, 5, 20_000, "keys of 18 bits: 9-bit digit, 18 radix tiles"),
    (300_000, 16, 4, 30_000, "keys of 20 bits: 10-bit digit, 22 radix tiles"),
]


def _one_step(N, D, K, n, scatter, seed=7, weights=None, hub=0.0, cmax=5, lr=0.025,
              heavy=None, batch=None):
    rng = np.random.default_rng(N * 31 + D * 7 + K)
    if batch is None:
        src, dst, cc = _random_batch(rng, N, n, cmax=cmax, hub_frac=hub)
    else:
        src, dst, cc = batch
    first = 1000
    tr = _trainer(N, D, K, n, seed=seed, weights=weights, scatter=scatter)
    loss = tr.step(dev(src, torch), dev(dst, torch), dev(cc, torch), first, lr).item()
    assert tr.check() == 0
    S = tr.S.cpu().numpy()
    T = tr.T.cpu().numpy()
    ids = np.arange(N)
    a = _half(D)
    S0 = orc.init_rows(seed, 0, ids, D, a)
    T0 = orc.init_rows(seed, 1, ids, D, a)
    thr = alias = None
    if weights is not None:
        thr, alias = orc.build_alias(weights)
    neg = orc.sample_negatives(seed, first, n, K, N, thr, alias)
    Sr, Tr = S0.copy(), T0.copy()
    ref_loss = orc.step_dense(Sr, Tr, src, dst, cc, neg, lr)
    tS = np.zeros(N, bool)
    tS[src] = True
    tT = np.zeros(N, bool)
    tT[dst] = True
    tT[neg.reshape(-1)] = True
    assert np.array_equal(S[~tS], S0[~tS]), "untouched source rows changed"
    assert np.array_equal(T[~tT], T0[~tT]), "untouched context rows changed"
    if heavy is not None:
        # Rows hit more than `heavy` times: fp32 atomics add thousands of
        # cancelling terms in arbitrary order, so only the update as a whole
        # is held to 1e-4 of its own size; every other row keeps the strict
        # element-wise bound.
        mS = np.bincount(src, minlength=N)
        mT = np.bincount(np.concatenate([dst, neg.reshape(-1)]), minlength=N)
        for name, G, R0, Rr, mult in (("S", S, S0, Sr, mS), ("T", T, T0, Tr, mT)):
            hv = mult > heavy
            for r in np.nonzero(hv)[0]:
                upd = np.linalg.norm(Rr[r].astype(np.float64) - R0[r])
                err = np.linalg.norm(G[r].astype(np.float64) - Rr[r])
                assert err <= 1e-4 * upd + 1e-6, (name, r, err, upd)
            tS = tS & ~hv if name == "S" else tS
            tT = tT & ~hv if name == "T" else tT
    assert_close(S[tS], Sr[tS], f"S {scatter}")
    assert_close(T[tT], Tr[tT], f"T {scatter}")
    assert loss == pytest.approx(ref_loss, rel=1e-5, abs=1e-6)
    return tr, (src, dst, cc, neg)


@pytest.mark.parametrize("scatter", ["sorted", "atomic"])
@pytest.mark.parametrize("N,D,K,n,note", STEP_CASES)
def test_one_step_matches_oracle(scatter, N, D, K, n, note):
    say(f"step {scatter} N={N} D={D} K={K} n={n} ({note})")
    tr, (src, dst, cc, neg) = _one_step(N, D, K, n, scatter)
    if scatter == "sorted":
        _check_counts(tr, N, src, dst, neg)


@pytest.mark.parametrize("scatter", ["sorted", "atomic"])
def test_hub_rows_and_large_counts(scatter):
    """Half the batch shares one source row, a quarter one destination row,
    co_counts up to 1000: long runs summed in pieces and combined.  The
    sorted scatter sums repeated rows in double and meets the element-wise
    bound everywhere; the atomic one is held to it on rows hit <= 64 times."""
    say(f"hub {scatter}")
    _one_step(5_000, 64, 4, 6000, scatter, hub=0.5, cmax=1000,
              heavy=None if scatter == "sorted" else 64)


def _check_counts(tr, N, src, dst, neg):
    uS, uT, dup = tr.stats()
    keys = np.concatenate([src.astype(np.int64) + N, dst, neg.reshape(-1)])
    u, cnt = np.unique(keys, return_counts=True)
    assert uS == np.unique(src).size
    assert uT == np.unique(np.concatenate([dst, neg.reshape(-1)])).size
    assert dup == int(cnt[cnt > 1].sum())


@pytest.mark.parametrize("N,n,hub,note", [
    (5_000, 8_000, 0.75, "hub rows of 6000 and 1500 occurrences: pieces and combined sums"),
    (5_000, 16_000, 0.9, "a bucket of > 14400 keys: grouped over several chunks"),
    (1_100_000, 8_000, 0.75, "hub rows among mostly distinct keys"),
    (1_100_000, 16_000, 0.9, "several chunks, long runs, distinct tail"),
])
@pytest.mark.parametrize("table_bits", [None, 12, 14])
def test_grouping_regimes(N, n, hub, note, table_bits, monkeypatch):
    """Grouping with hub rows and buckets of every size; tables and the
    distinct / repeated counts must match the oracle and numpy.  table_bits
    forces the hash-table grouping of every key with that table size (by
    default a bitmap of the bucket's keys lets only repeated keys in)."""
    if table_bits is not None:
        monkeypatch.setenv("HUGE_GROUP_TABLE_BITS", str(table_bits))
    say(f"grouping regimes N={N} n={n} hub={hub} table_bits={table_bits} ({note})")
    tr, (src, dst, cc, neg) = _one_step(N, 8, 2, n, "sorted", hub=hub)
    _check_counts(tr, N, src, dst, neg)


@pytest.mark.parametrize("table_bits", [None, 12, 13])
def test_bucket_with_more_distinct_rows_than_one_table(table_bits, monkeypatch):
    """Every source and destination key has the same lowest 10 bits (the
    bucket digit for N = 8e6, whose keys have 24 bits), so about 9000
    distinct keys share one bucket, about 6700 of them repeated: more than
    one LDS table holds, and the bucket is grouped key range by key range
    (with the bitmap of repeated keys or, with table_bits, without)."""
    if table_bits is not None:
        monkeypatch.setenv("HUGE_GROUP_TABLE_BITS", str(table_bits))
    N, D, K, n = 8_000_000, 8, 1, 12_000
    ids = np.arange(N, dtype=np.int64)
    cand_s = ids[((ids + N) & 1023) == 7][:4500]
    cand_d = ids[(ids & 1023) == 7][:4500]
    rng = np.random.default_rng(23)
    src = rng.choice(cand_s, n).astype(np.int32)   # with replacement: repeats
    dst = rng.choice(cand_d, n).astype(np.int32)
    cc = rng.integers(0, 6, n).astype(np.int32)
    say(f"one crowded bucket: {np.unique(src).size + np.unique(dst).size} distinct keys, "
        f"table_bits={table_bits}")
    tr, (src, dst, cc, neg) = _one_step(N, D, K, n, "sorted", batch=(src, dst, cc))
    _check_counts(tr, N, src, dst, neg)


def test_alias_negatives_step():
    say("alias step")
    rng = np.random.default_rng(3)
    w = rng.integers(1, 60, 4000).astype(np.float64) ** 0.75
    _one_step(4000, 64, 6, 3000, "sorted", weights=w)


def test_sorted_scatter_is_bitwise_reproducible():
    say("determinism")
    N, D, K, n = 3000, 64, 5, 5000
    rng = np.random.default_rng(11)
    batches = [_random_batch(rng, N, n, hub_frac=0.3) for _ in range(3)]
    out = []
    for _ in range(2):
        tr = _trainer(N, D, K, n, seed=5)
        for b, (s, d, c) in enumerate(batches):
            tr.step(dev(s, torch), dev(d, torch), dev(c, torch), b * n, 0.05)
        out.append((tr.S.cpu().numpy(), tr.T.cpu().numpy()))
        del tr
    assert np.array_equal(out[0][0], out[1][0]) and np.array_equal(out[0][1], out[1][1])


# --------------------------------------------------------------------------- #
# Boundary behaviour
# --------------------------------------------------------------------------- #
@pytest.mark.parametrize("scatter", ["sorted", "atomic"])
def test_empty_batch_is_a_no_op(scatter):
    tr = _trainer(100, 16, 3, 10, scatter=scatter)
    S0, T0 = tr.S.clone(), tr.T.clone()
    e = torch.zeros(0, dtype=torch.int32, device="cuda")
    loss = torch.full((1,), 7.0, dtype=torch.float64, device="cuda")
    tr.step(e, e, e, 0, 0.1, loss_out=loss)
    assert loss.item() == 0.0
    assert torch.equal(tr.S, S0) and torch.equal(tr.T, T0)
    assert tr.check() == 0


@pytest.mark.parametrize("scatter", ["sorted", "atomic"])
@pytest.mark.parametrize("bad", ["src", "dst", "neg_src", "count"])
def test_invalid_batch_is_a_no_op_and_reported(scatter, bad):
    N = 1000
    tr = _trainer(N, 32, 4, 256, scatter=scatter)
    rng = np.random.default_rng(1)
    src, dst, cc = _random_batch(rng, N, 256)
    if bad == "src":
        src[100] = N
    elif bad == "dst":
        dst[5] = N + 7
    elif bad == "neg_src":
        src[0] = -1
    else:
        cc[17] = -2
    S0, T0 = tr.S.clone(), tr.T.clone()
    loss = tr.step(dev(src, torch), dev(dst, torch), dev(cc, torch), 0, 0.1).item()
    assert np.isnan(loss)
    assert tr.check() == (-3 if bad == "count" else -2)
    assert tr.check() == 0  # cleared
    assert torch.equal(tr.S, S0) and torch.equal(tr.T, T0)
    # the next valid batch is applied normally
    s2, d2, c2 = _random_batch(rng, N, 256)
    loss = tr.step(dev(s2, torch), dev(d2, torch), dev(c2, torch), 256, 0.1).item()
    assert np.isfinite(loss) and tr.check() == 0
    assert not torch.equal(tr.S, S0)


def test_batch_larger_than_max_is_rejected_on_host():
    tr = _trainer(100, 16, 3, 10)
    x = torch.zeros(11, dtype=torch.int32, device="cuda")
    with pytest.raises(P.HugeError):
        tr.step(x, x, x, 0, 0.1)


def test_get_rows_and_out_of_range_ids():
    tr = _trainer(500, 40, 2, 8, seed=3)
    ids = torch.tensor([0, 499, 17, 500, -1], dtype=torch.int64, device="cuda")
    rows = tr.get_rows(1, ids).cpu().numpy()
    ref = orc.init_rows(3, 1, [0, 499, 17], 40, _half(40))
    assert np.array_equal(rows[:3], ref)
    assert np.all(np.isnan(rows[3:]))
    assert tr.check() == -2


@pytest.mark.parametrize("D,K", [(128, 5), (36, 11), (1024, 2)])
def test_probe_rows_leaves_tables_bitwise_unchanged(D, K):
    """The bandwidth probe reads and rewrites every row a step would touch
    (hub rows included) and must leave both tables bit for bit as they were;
    an out-of-range id is reported and skipped."""
    N, n = 3000, 2000
    rng = np.random.default_rng(D + K)
    src, dst, cc = _random_batch(rng, N, n, hub_frac=0.3)
    tr = _trainer(N, D, K, n, seed=6)
    tr.step(dev(src, torch), dev(dst, torch), dev(cc, torch), 0, 0.05)  # non-initial values
    S0, T0 = tr.S.clone(), tr.T.clone()
    for rep in range(3):
        tr.probe_rows(dev(src, torch), dev(dst, torch), n * (rep + 1))
    assert tr.check() == 0
    assert torch.equal(tr.S, S0) and torch.equal(tr.T, T0)
    bad = src.copy()
    bad[7] = N
    tr.probe_rows(dev(bad, torch), dev(dst, torch), 0)
    assert tr.check() == -2
    assert torch.equal(tr.S, S0) and torch.equal(tr.T, T0)


def test_eval_loss_matches_oracle_and_writes_nothing():
    N, D, K, n = 2000, 48, 6, 1500
    rng = np.random.default_rng(5)
    src, dst, cc = _random_batch(rng, N, n)
    tr = _trainer(N, D, K, n, seed=8)
    S0, T0 = tr.S.clone(), tr.T.clone()
    got = tr.eval_loss(dev(src, torch), dev(dst, torch), dev(cc, torch), 77).item()
    assert torch.equal(tr.S, S0) and torch.equal(tr.T, T0)
    neg = orc.sample_negatives(8, 77, n, K, N)
    ref = orc.loss_dense(S0.cpu().numpy(), T0.cpu().numpy(), src, dst, cc, neg)
    assert got == pytest.approx(ref, rel=1e-5)
    # it also agrees with the step's own loss on the same batch
    step_loss = tr.step(dev(src, torch), dev(dst, torch), dev(cc, torch), 77, 0.1).item()
    assert step_loss == pytest.approx(got, rel=1e-6)


# --------------------------------------------------------------------------- #
# Several steps: resume equals straight run; an epoch of the tiny workload
# --------------------------------------------------------------------------- #
def test_resume_from_saved_tables_is_bitwise_equal():
    N, D, K, n = 4000, 32, 5, 2048
    rng = np.random.default_rng(2)
    batches = [_random_batch(rng, N, n, hub_frac=0.2) for _ in range(4)]
    straight = _trainer(N, D, K, n, seed=21)
    for b, (s, d, c) in enumerate(batches):
        straight.step(dev(s, torch), dev(d, torch), dev(c, torch), b * n, 0.05)
    first = _trainer(N, D, K, n, seed=21)
    for b, (s, d, c) in enumerate(batches[:2]):
        first.step(dev(s, torch), dev(d, torch), dev(c, torch), b * n, 0.05)
    saved = (first.S.cpu().clone(), first.T.cpu().clone())
    del first
    resumed = P.Trainer(N, D, K, n, seed=21,
                        tables=(saved[0].cuda().contiguous(), saved[1].cuda().contiguous()),
                        init=False)
    for b, (s, d, c) in enumerate(batches[2:], start=2):
        resumed.step(dev(s, torch), dev(d, torch), dev(c, torch), b * n, 0.05)
    assert torch.equal(resumed.S, straight.S) and torch.equal(resumed.T, straight.T)


@pytest.mark.parametrize("scatter", ["sorted", "atomic"])
def test_tiny_epoch_loss_curve(scatter):
    """The tiny SBM workload for one epoch: per-step mean loss within 1e-3."""
    from synth import make_workload
    wl = make_workload("tiny", 0)
    cfg = wl.cfg
    src, dst, cc = wl.epoch()
    nb = (src.size + cfg.batch - 1) // cfg.batch
    say(f"tiny epoch {scatter}: {src.size} positives, {nb} steps")
    tr = _trainer(cfg.num_nodes, cfg.dim, cfg.num_neg, cfg.batch, seed=0, scatter=scatter)
    losses = torch.zeros(nb, dtype=torch.float64, device="cuda")
    ds, dd, dc = dev(src, torch), dev(dst, torch), dev(cc, torch)
    for b in range(nb):
        lo, hi = b * cfg.batch, min(src.size, (b + 1) * cfg.batch)
        tr.step(ds[lo:hi], dd[lo:hi], dc[lo:hi], lo, cfg.lr, loss_out=losses[b:b + 1])
    gl = losses.cpu().numpy()
    a = _half(cfg.dim)
    ids = np.arange(cfg.num_nodes)
    S = orc.init_rows(0, 0, ids, cfg.dim, a)
    T = orc.init_rows(0, 1, ids, cfg.dim, a)
    ol = np.zeros(nb)
    csum = np.zeros(nb)
    for b in range(nb):
        lo, hi = b * cfg.batch, min(src.size, (b + 1) * cfg.batch)
        neg = orc.sample_negatives(0, lo, hi - lo, cfg.num_neg, cfg.num_nodes)
        ol[b] = orc.step_dense(S, T, src[lo:hi], dst[lo:hi], cc[lo:hi], neg, cfg.lr)
        csum[b] = cc[lo:hi].sum()
    gm, om = gl / csum, ol / csum
    err = np.abs(gm - om) / np.maximum(1.0, np.abs(om))
    say(f"  mean loss first {om[0]:.5f} last {om[-1]:.5f}; max rel err {err.max():.2e}")
    assert err.max() <= 1e-3
    assert om[-1] < om[0]  # it learns
    # tables after the epoch stay close to the oracle's
    assert_close(tr.S.cpu().numpy(), S, "S after epoch", abs_tol=1e-4, rel_tol=1e-3)
    assert_close(tr.T.cpu().numpy(), T, "T after epoch", abs_tol=1e-4, rel_tol=1e-3)


def test_lwsgd_schedule_over_tiny_steps():
    """60 steps of the tiny workload under a scaled LWSGD schedule (warm-up
    15, peak 0.05, decay 30, final 0.01): the GPU takes each step's rate from
    the library's helper, the oracle from its own definition of the schedule;
    per-step losses and the final tables must agree."""
    from paper_2307_14490_amd.schedule import lwsgd
    from synth import make_workload
    wl = make_workload("tiny", 0)
    cfg = wl.cfg
    src, dst, cc = wl.epoch()
    steps, sched = 60, (15, 0.05, 30, 0.01)
    tr = _trainer(cfg.num_nodes, cfg.dim, cfg.num_neg, cfg.batch, seed=3)
    losses = torch.zeros(steps, dtype=torch.float64, device="cuda")
    ds, dd, dc = dev(src, torch), dev(dst, torch), dev(cc, torch)
    for b in range(steps):
        lo, hi = b * cfg.batch, (b + 1) * cfg.batch
        tr.step(ds[lo:hi], dd[lo:hi], dc[lo:hi], lo, lwsgd(b, *sched), loss_out=losses[b:b + 1])
    gl = losses.cpu().numpy()
    a = _half(cfg.dim)
    ids = np.arange(cfg.num_nodes)
    S = orc.init_rows(3, 0, ids, cfg.dim, a)
    T = orc.init_rows(3, 1, ids, cfg.dim, a)
    ol = np.zeros(steps)
    for b in range(steps):
        lo, hi = b * cfg.batch, (b + 1) * cfg.batch
        neg = orc.sample_negatives(3, lo, hi - lo, cfg.num_neg, cfg.num_nodes)
        ol[b] = orc.step_dense(S, T, src[lo:hi], dst[lo:hi], cc[lo:hi], neg,
                               orc.lwsgd_lr(b, *sched))
    np.testing.assert_allclose(gl, ol, rtol=1e-5)
    assert_close(tr.S.cpu().numpy(), S, "S after LWSGD steps", abs_tol=1e-5, rel_tol=1e-4)
    assert_close(tr.T.cpu().numpy(), T, "T after LWSGD steps", abs_tol=1e-5, rel_tol=1e-4)


# --------------------------------------------------------------------------- #
# Grouping on one stream while the previous batch is applied on another
# --------------------------------------------------------------------------- #
def test_prepared_steps_on_two_streams_equal_train_step_bitwise():
    N, D, K, n = 5000, 64, 5, 3000
    rng = np.random.default_rng(17)
    batches = [_random_batch(rng, N, n, hub_frac=0.2, cmax=50) for _ in range(5)]
    ref = _trainer(N, D, K, n, seed=4)
    ref_losses = []
    for b, (s, d, c) in enumerate(batches):
        ref_losses.append(ref.step(dev(s, torch), dev(d, torch), dev(c, torch), b * n, 0.05).item())
    tr = _trainer(N, D, K, n, seed=4)
    main = torch.cuda.current_stream()
    side = torch.cuda.Stream()
    dbs = [tuple(dev(x, torch) for x in b) for b in batches]
    losses = torch.zeros(len(batches), dtype=torch.float64, device="cuda")
    tr.prepare(*dbs[0], 0, stream=side)
    for k in range(len(batches)):
        tr.train_prepared(0.05, loss_out=losses[k:k + 1], stream=main)
        if k + 1 < len(batches):
            tr.prepare(*dbs[k + 1], (k + 1) * n, stream=side)
    torch.cuda.synchronize()
    assert tr.check() == 0
    assert torch.equal(tr.S, ref.S) and torch.equal(tr.T, ref.T)
    assert losses.cpu().tolist() == ref_losses


def test_prepared_steps_with_long_groupings_equal_train_step_bitwise():
    """Batches large enough that the grouping of batch k+1 runs beside the
    update of batch k for a long while: the events that order the two halves
    (recorded by the grouping and finish kernels' completion) must hold."""
    N, D, K, n = 200_000, 128, 10, 60_000
    rng = np.random.default_rng(23)
    batches = [_random_batch(rng, N, n, hub_frac=0.3, cmax=20) for _ in range(6)]
    ref = _trainer(N, D, K, n, seed=8)
    ref_losses = []
    for b, (s, d, c) in enumerate(batches):
        ref_losses.append(ref.step(dev(s, torch), dev(d, torch), dev(c, torch), b * n,
                                   0.02).item())
    tr = _trainer(N, D, K, n, seed=8)
    main = torch.cuda.current_stream()
    side = torch.cuda.Stream()
    dbs = [tuple(dev(x, torch) for x in b) for b in batches]
    losses = torch.zeros(len(batches), dtype=torch.float64, device="cuda")
    tr.prepare(*dbs[0], 0, stream=side)
    for k in range(len(batches)):
        if k + 1 < len(batches):
            tr.prepare(*dbs[k + 1], (k + 1) * n, stream=side)
        tr.train_prepared(0.02, loss_out=losses[k:k + 1], stream=main)
    torch.cuda.synchronize()
    assert tr.check() == 0
    assert torch.equal(tr.S, ref.S) and torch.equal(tr.T, ref.T)
    assert losses.cpu().tolist() == ref_losses


def test_prepared_steps_in_irregular_orders_equal_train_step_bitwise():
    """Applies alternate between two streams, preparations run two batches
    ahead on a third, and side calls (a loss evaluation, a row read) on a
    fourth come between them.  An apply's completion is recorded only where a
    wait needs it (by a finish kernel, or on demand): every such wait must
    hold, so tables, losses and the side calls' results equal those of
    sequential steps bit for bit."""
    N, D, K, n, nb = 50_000, 64, 5, 20_000, 9
    rng = np.random.default_rng(31)
    batches = [_random_batch(rng, N, n, hub_frac=0.05, cmax=5) for _ in range(nb)]
    deb = tuple(dev(x, torch) for x in _random_batch(rng, N, 4000))
    ids = torch.from_numpy(rng.integers(0, N, 500)).to("cuda")  # int64: read as given
    ref = _trainer(N, D, K, n, seed=6)
    ref_losses, ref_eval, ref_rows = [], {}, {}
    for b, (s, d, c) in enumerate(batches):
        ref_losses.append(ref.step(dev(s, torch), dev(d, torch), dev(c, torch), b * n,
                                   0.005).item())
        if b % 3 == 1:
            ref_eval[b] = ref.eval_loss(*deb, 7).item()
            ref_rows[b] = ref.get_rows(b % 2, ids).cpu()
    tr = _trainer(N, D, K, n, seed=6)
    applies = [torch.cuda.current_stream(), torch.cuda.Stream()]
    prep, side = torch.cuda.Stream(), torch.cuda.Stream()
    dbs = [tuple(dev(x, torch) for x in b) for b in batches]
    losses = torch.zeros(nb, dtype=torch.float64, device="cuda")
    evals = torch.zeros(nb, dtype=torch.float64, device="cuda")
    rows = {}
    tr.prepare(*dbs[0], 0, stream=prep)
    tr.prepare(*dbs[1], n, stream=prep)
    for k in range(nb):
        tr.train_prepared(0.005, loss_out=losses[k:k + 1], stream=applies[k % 2])
        if k % 3 == 1:
            tr.eval_loss(*deb, 7, loss_out=evals[k:k + 1], stream=side)
            rows[k] = tr.get_rows(k % 2, ids, stream=side)
        if k + 2 < nb:
            tr.prepare(*dbs[k + 2], (k + 2) * n, stream=prep)
    torch.cuda.synchronize()
    assert tr.check() == 0
    assert bool(torch.isfinite(tr.S).all()) and bool(torch.isfinite(tr.T).all())
    assert torch.equal(tr.S, ref.S) and torch.equal(tr.T, ref.T)
    assert losses.cpu().tolist() == ref_losses
    for k in ref_eval:
        assert evals[k].item() == ref_eval[k]
        assert torch.equal(rows[k].cpu(), ref_rows[k])


def test_prepared_call_order_is_checked_on_host():
    tr = _trainer(100, 16, 3, 64)
    rng = np.random.default_rng(3)
    s, d, c = (dev(x, torch) for x in _random_batch(rng, 100, 64))
    with pytest.raises(P.HugeError):
        tr.train_prepared(0.1)
    tr.prepare(s, d, c, 0)
    tr.prepare(s, d, c, 64)
    with pytest.raises(P.HugeError):
        tr.prepare(s, d, c, 128)  # both slots pending
    with pytest.raises(P.HugeError):
        tr.step(s, d, c, 128, 0.1)  # a prepared batch is pending
    tr.train_prepared(0.1)
    tr.train_prepared(0.1)
    tr.step(s, d, c, 128, 0.1)
    assert tr.check() == 0


def test_invalid_prepared_batch_is_a_no_op():
    N = 500
    tr = _trainer(N, 16, 3, 64)
    rng = np.random.default_rng(4)
    s, d, c = _random_batch(rng, N, 64)
    bad = s.copy()
    bad[3] = N
    S0 = tr.S.clone()
    # the batch arrays must outlive their apply: keep them referenced
    b1 = (dev(bad, torch), dev(d, torch), dev(c, torch))
    b2 = (dev(s, torch), dev(d, torch), dev(c, torch))
    tr.prepare(*b1, 0)
    tr.prepare(*b2, 64)
    l1 = tr.train_prepared(0.1, loss_out=torch.zeros(1, dtype=torch.float64, device="cuda"))
    assert np.isnan(l1.item())
    assert torch.equal(tr.S, S0)
    l2 = tr.train_prepared(0.1, loss_out=torch.zeros(1, dtype=torch.float64, device="cuda"))
    assert np.isfinite(l2.item())
    assert tr.check() == -2


def test_batches_of_the_wrong_type_are_refused():
    tr = _trainer(100, 8, 3, 16)
    src = torch.zeros(16, dtype=torch.int64, device="cuda")
    dst = torch.zeros(16, dtype=torch.int32, device="cuda")
    cc = torch.ones(16, dtype=torch.int32, device="cuda")
    with pytest.raises(TypeError, match="src"):
        tr.step(src, dst, cc, 0, 0.1)
    with pytest.raises(ValueError, match="length"):
        tr.step(dst, dst[:8], cc, 0, 0.1)
    with pytest.raises(TypeError, match="counts"):
        tr.step(dst, dst, cc.double(), 0, 0.1)
    assert tr.check() == 0
