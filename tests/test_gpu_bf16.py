"""bfloat16 tables on the GPU against the oracle's bf16 step (widened to
double, each written element rounded once to the nearest bf16, ties to even):

- initial tables bit-exact (the float values rounded);
- one step within one bf16 step of the oracle for every element (plus the
  float step's absolute tolerance) and equal for nearly all of them. The
  kernels compute in fp32 and round each written value once more, so a value
  within a few fp32 ulps of a rounding boundary may land on the other side.
  This covers in-place rows, short runs, pieces and combined hub rows,
  integer counts and float weights;
- the loss at pre-step values within the float step's tolerance;
- prepared steps bitwise equal to direct ones;
- row gather widening exactly;
- the probe leaving the tables bit for bit;
- two epochs of training tracking the float tables' loss.
"""
import numpy as np
import pytest

torch = pytest.importorskip("torch")

from oracle import oracle as orc  # noqa: E402
import paper_2307_14490_amd as P  # noqa: E402
from gpu_common import assert_bf16_close, dev, say  # noqa: E402

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    yield
    torch.cuda.synchronize()


def _half(D):
    return float(np.float32(0.5 / D))


def _bits(t):
    return t.view(torch.int16).cpu().numpy().view(np.uint16)


def _batch(rng, N, n, cmax=5, hub=0.0, weights=False):
    src = rng.integers(0, N, n).astype(np.int32)
    dst = rng.integers(0, N, n).astype(np.int32)
    if weights:
        cc = rng.gamma(0.7, 2.0, n).astype(np.float32)
    else:
        cc = rng.integers(0, cmax + 1, n).astype(np.int32)
    if hub > 0:
        k = int(n * hub)
        src[:k] = 1 % N
        dst[k // 2:k] = 0
    return src, dst, cc


@pytest.mark.parametrize("N,D,a", [(1000, 128, 0.0), (257, 36, 0.01), (64, 1024, 0.5)])
def test_init_tables_bit_exact(N, D, a):
    say(f"bf16 init N={N} D={D} a={a}")
    tr = P.Trainer(N, D, 5, 16, seed=11, init_half_width=a, dtype="bf16")
    ids = np.arange(N)
    hw = float(np.float32(a)) if a else _half(D)
    assert np.array_equal(_bits(tr.S), orc.init_rows_bf16(11, 0, ids, D, hw))
    assert np.array_equal(_bits(tr.T), orc.init_rows_bf16(11, 1, ids, D, hw))


STEP_CASES = [
    # N, D, K, n, hub, cmax, weights, note
    (3000, 128, 5, 4000, 0.0, 5, False, "mostly distinct rows, in place"),
    (200, 32, 3, 3000, 0.0, 5, False, "short runs"),
    (5000, 64, 4, 6000, 0.5, 1000, False, "hub rows: pieces and combined sums"),
    (1000, 8, 10, 2000, 0.2, 5, True, "float weights, narrow rows"),
    (500, 260, 6, 1500, 0.1, 3, False, "D = 260: 4-element chunks, several per lane, ragged"),
    (300, 1024, 3, 500, 0.1, 3, False, "D = 1024: two 8-element units per lane"),
    (400, 520, 4, 800, 0.0, 5, False, "D = 520: 65 units, those past the row masked"),
    (800, 16, 9, 1200, 0.3, 7, False, "D = 16: two lanes per row, K = 9 in two blocks"),
]


@pytest.mark.parametrize("N,D,K,n,hub,cmax,weights,note", STEP_CASES)
def test_one_step_matches_oracle(N, D, K, n, hub, cmax, weights, note):
    rng = np.random.default_rng(N + D + K)
    src, dst, cc = _batch(rng, N, n, cmax, hub, weights)
    seed, first, lr = 9, 777, 0.025
    say(f"bf16 step N={N} D={D} K={K} n={n} ({note})")
    tr = P.Trainer(N, D, K, n, seed=seed, dtype="bf16")
    loss = tr.step(dev(src, torch), dev(dst, torch), dev(cc, torch), first, lr).item()
    assert tr.check() == 0
    ids = np.arange(N)
    S = orc.init_rows_bf16(seed, 0, ids, D, _half(D))
    T = orc.init_rows_bf16(seed, 1, ids, D, _half(D))
    neg = orc.sample_negatives(seed, first, n, K, N)
    ref = orc.step_dense_bf16(S, T, src, dst, cc, neg, lr)
    assert_bf16_close(_bits(tr.S), S, "S")
    assert_bf16_close(_bits(tr.T), T, "T")
    assert loss == pytest.approx(ref, rel=1e-5, abs=1e-6)


def test_eval_loss_matches_oracle():
    N, D, K, n = 2000, 64, 5, 3000
    rng = np.random.default_rng(3)
    src, dst, cc = _batch(rng, N, n)
    tr = P.Trainer(N, D, K, n, seed=4, dtype="bf16")
    S0, T0 = tr.S.clone(), tr.T.clone()
    got = tr.eval_loss(dev(src, torch), dev(dst, torch), dev(cc, torch), 55).item()
    assert torch.equal(tr.S, S0) and torch.equal(tr.T, T0)
    Sf = orc.bf16_to_float(_bits(S0)).reshape(N, D)
    Tf = orc.bf16_to_float(_bits(T0)).reshape(N, D)
    ref = orc.loss_dense(Sf, Tf, src, dst, cc, orc.sample_negatives(4, 55, n, K, N))
    assert got == pytest.approx(ref, rel=1e-5, abs=1e-6)


def test_prepared_steps_equal_direct_ones_bitwise():
    N, D, K, n = 3000, 128, 5, 2500
    rng = np.random.default_rng(5)
    batches = [_batch(rng, N, n, cmax=50, hub=0.2) for _ in range(4)]
    ref = P.Trainer(N, D, K, n, seed=3, dtype="bf16")
    for k, (s, d, c) in enumerate(batches):
        ref.step_no_loss(dev(s, torch), dev(d, torch), dev(c, torch), k * n, 0.05)
    tr = P.Trainer(N, D, K, n, seed=3, dtype="bf16")
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


def test_get_rows_widens_exactly():
    N, D = 500, 40
    tr = P.Trainer(N, D, 3, 8, seed=2, dtype="bf16")
    ids = torch.tensor([0, 499, 7, 7, 250], dtype=torch.int64)
    for t, tab in ((0, tr.S), (1, tr.T)):
        got = tr.get_rows(t, ids)
        assert got.dtype == torch.float32
        assert torch.equal(got, tab[ids.to(tab.device)].float())


@pytest.mark.parametrize("D", [128, 520, 36])
def test_probe_rows_leaves_bf16_tables_unchanged(D):
    N, K, n = 1000, 5, 4000
    rng = np.random.default_rng(6)
    src, dst, _ = _batch(rng, N, n, hub=0.3)
    tr = P.Trainer(N, D, K, n, seed=1, dtype="bf16")
    S0, T0 = tr.S.clone(), tr.T.clone()
    tr.probe_rows(dev(src, torch), dev(dst, torch), 10)
    torch.cuda.synchronize()
    assert tr.check() == 0
    assert torch.equal(tr.S, S0) and torch.equal(tr.T, T0)


def test_atomic_scatter_with_bf16_is_rejected():
    with pytest.raises(P.binding.HugeError):
        P.Trainer(100, 16, 3, 8, scatter="atomic", dtype="bf16")


def test_training_tracks_the_float_tables():
    """The tiny SBM workload trained for two epochs with float and with bf16
    tables (the same initial values, rounded): the loss falls, and the bf16
    run's loss over the second epoch is within 2% of the float run's."""
    from synth import gen
    wl = gen.make_workload("tiny")
    cfg = wl.cfg
    es, ed, ec = (dev(x, torch) for x in wl.epoch())
    runs = {}
    for dt in ("f32", "bf16"):
        tr = P.Trainer(cfg.num_nodes, cfg.dim, cfg.num_neg, cfg.batch, seed=3, dtype=dt)
        pos, per_epoch = 0, []
        for _ in range(2):
            total = 0.0
            for i0 in range(0, es.numel(), cfg.batch):
                i1 = min(i0 + cfg.batch, es.numel())
                total += tr.step(es[i0:i1], ed[i0:i1], ec[i0:i1], pos, cfg.lr).item()
                pos += i1 - i0
            per_epoch.append(total)
        assert tr.check() == 0
        runs[dt] = per_epoch
    say(f"  epoch losses f32 {runs['f32']}, bf16 {runs['bf16']}")
    assert runs["f32"][1] < runs["f32"][0] and runs["bf16"][1] < runs["bf16"][0]
    assert runs["bf16"][1] == pytest.approx(runs["f32"][1], rel=0.02)


def test_evaluator_refuses_a_bf16_table():
    """The evaluators read fp32 rows; a bf16 table is refused by the binding
    (its rows go through get_rows, which widens them)."""
    tr = P.Trainer(100, 16, 3, 8, seed=1, dtype="bf16")
    ev = P.Evaluator(100, 16, 8)
    u = torch.zeros(4, dtype=torch.int32, device="cuda")
    with pytest.raises(TypeError, match="float32"):
        ev.distances(tr.S, u, u)
    ids = torch.arange(100, dtype=torch.int64)
    d = ev.distances(tr.get_rows(0, ids), u, u)   # a row against itself
    assert torch.all(d.abs() < 1e-3)


@pytest.mark.parametrize("bad", ["src", "count"])
def test_invalid_batch_is_a_no_op_on_bf16_tables(bad):
    """The same all-or-nothing rule as for fp32 tables: an out-of-range id or
    a negative count leaves the bf16 tables bit for bit and is reported; an
    empty batch changes nothing; the next valid batch is applied."""
    N, D, K, n = 1000, 128, 5, 256
    tr = P.Trainer(N, D, K, n, seed=2, dtype="bf16")
    rng = np.random.default_rng(7)
    src, dst, cc = _batch(rng, N, n)
    if bad == "src":
        src[100] = N
    else:
        cc[17] = -2
    S0, T0 = tr.S.clone(), tr.T.clone()
    loss = tr.step(dev(src, torch), dev(dst, torch), dev(cc, torch), 0, 0.1).item()
    assert np.isnan(loss)
    assert tr.check() == (-2 if bad == "src" else -3)
    assert torch.equal(tr.S, S0) and torch.equal(tr.T, T0)
    e = torch.empty(0, dtype=torch.int32, device="cuda")
    assert tr.step(e, e, e, 0, 0.1).item() == 0.0
    assert tr.check() == 0 and torch.equal(tr.S, S0) and torch.equal(tr.T, T0)
    s2, d2, c2 = _batch(rng, N, n)
    loss = tr.step(dev(s2, torch), dev(d2, torch), dev(c2, torch), n, 0.1).item()
    assert np.isfinite(loss) and tr.check() == 0
    assert not torch.equal(tr.S, S0)


def test_alias_negatives_step_on_bf16_tables():
    """Negatives from an alias table over degree^0.75-like weights (the
    medium, power-law and hub-stress workloads' sampler), bf16 tables."""
    N, D, K, n = 2000, 128, 6, 3000
    rng = np.random.default_rng(12)
    w = (rng.pareto(1.1, N) + 0.1) ** 0.75
    w[::9] = 0.0
    src, dst, cc = _batch(rng, N, n, hub=0.2)
    seed, first, lr = 4, 99, 0.025
    tr = P.Trainer(N, D, K, n, seed=seed, alias_weights=w, dtype="bf16")
    loss = tr.step(dev(src, torch), dev(dst, torch), dev(cc, torch), first, lr).item()
    assert tr.check() == 0
    thr, alias = orc.build_alias(w)
    neg = orc.sample_negatives(seed, first, n, K, N, thr, alias)
    assert np.array_equal(tr.sample_negatives(n, first).cpu().numpy(), neg)
    ids = np.arange(N)
    S = orc.init_rows_bf16(seed, 0, ids, D, _half(D))
    T = orc.init_rows_bf16(seed, 1, ids, D, _half(D))
    ref = orc.step_dense_bf16(S, T, src, dst, cc, neg, lr)
    assert_bf16_close(_bits(tr.S), S, "S")
    assert_bf16_close(_bits(tr.T), T, "T")
    assert loss == pytest.approx(ref, rel=1e-5, abs=1e-6)
