"""Parity at the full sizes of the benchmark workloads (GPU).

One step from freshly initialised tables on batch 0 of each workload, in the
launch configuration the benchmark times (sorted scatter; the medium workload
also with the atomic scatter).  The oracle holds only the rows the batch
touches (its own sampler picks the negatives, its own initialiser the
pre-step values), so every touched element is checked against it; a random
sample of untouched rows must still equal the oracle's initial values bit for
bit, and the step's row counts must equal the oracle's exactly.  SBM-100M
also runs on bf16 tables against the oracle's bf16 step.
"""
import time

import numpy as np
import pytest

torch = pytest.importorskip("torch")

from oracle import oracle as orc  # noqa: E402
import paper_2307_14490_amd as P  # noqa: E402
from gpu_common import assert_bf16_close, assert_close, dev, say  # noqa: E402

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    yield
    torch.cuda.synchronize()
    torch.cuda.empty_cache()


# One step from the initial values at a fixed rate (the workloads' own rates
# keep long runs finite; a single step at 0.025 moves every touched element
# well above float32 resolution).
PARITY_LR = 0.025

CASES = [("medium", "sorted"), ("medium", "atomic"), ("powerlaw", "sorted"),
         ("sbm100m", "sorted"), ("hubstress", "sorted"), ("sbm100m_k31", "sorted")]


@pytest.mark.timeout(600)
@pytest.mark.parametrize("name,scatter", CASES)
def test_full_size_step(name, scatter):
    from synth import make_workload
    t0 = time.time()
    wl = make_workload(name, 0)
    cfg = wl.cfg
    src, dst, cc = wl.batch(0)
    say(f"[{name}/{scatter}] N={cfg.num_nodes} D={cfg.dim} K={cfg.num_neg} n={src.size} "
        f"inputs {time.time() - t0:.1f}s")
    seed = 2024
    first = 3 * cfg.batch
    a = float(np.float32(cfg.init_half_width))
    thr = alias = None
    if cfg.neg_kind == "alias":
        thr, alias = orc.build_alias(wl.weights)
    tr = P.Trainer(cfg.num_nodes, cfg.dim, cfg.num_neg, cfg.batch, seed=seed,
                   alias_weights=wl.weights, scatter=scatter)
    loss = tr.step(dev(src, torch), dev(dst, torch), dev(cc, torch), first, PARITY_LR).item()
    assert tr.check() == 0
    say(f"[{name}/{scatter}] gpu step done {time.time() - t0:.1f}s")

    ref = orc.step_sparse(seed, cfg.num_nodes, cfg.dim, cfg.num_neg, a, src, dst, cc, first,
                          PARITY_LR, thr, alias)
    say(f"[{name}/{scatter}] oracle done {time.time() - t0:.1f}s "
        f"rows S {ref.rows_S.size} T {ref.rows_T.size}")
    # negatives: the device sampler must give the oracle's draws
    negs = tr.sample_negatives(src.size, first).cpu().numpy()
    assert np.array_equal(negs, ref.neg)
    if scatter == "sorted":
        uS, uT, dup = tr.stats()
        keys = np.concatenate([src.astype(np.int64) + cfg.num_nodes, dst, ref.neg.reshape(-1)])
        _, cnt = np.unique(keys, return_counts=True)
        assert (uS, uT) == (ref.rows_S.size, ref.rows_T.size)
        assert dup == int(cnt[cnt > 1].sum())
    gS = tr.get_rows(0, torch.from_numpy(ref.rows_S)).cpu().numpy()
    assert_close(gS, ref.S, f"{name} S")
    del gS
    gT = tr.get_rows(1, torch.from_numpy(ref.rows_T)).cpu().numpy()
    assert_close(gT, ref.T, f"{name} T")
    del gT
    assert loss == pytest.approx(ref.loss, rel=1e-5)
    # untouched rows keep their initial values exactly
    rng = np.random.default_rng(1)
    for table, rows in ((0, ref.rows_S), (1, ref.rows_T)):
        cand = rng.integers(0, cfg.num_nodes, 6000)
        cand = np.setdiff1d(cand, rows)[:4096]
        got = tr.get_rows(table, torch.from_numpy(cand)).cpu().numpy()
        assert np.array_equal(got, orc.init_rows(seed, table, cand, cfg.dim, a))
    say(f"[{name}/{scatter}] checked {time.time() - t0:.1f}s")
    tr.close()
    del tr


def _bf16_bits(rows_f32):
    """bf16 bit patterns of float32 rows that hold widened bf16 values."""
    b = np.ascontiguousarray(rows_f32, np.float32).view(np.uint32)
    assert not np.any(b & 0xFFFF), "a widened bf16 value has no low half"
    return (b >> 16).astype(np.uint16)


@pytest.mark.timeout(600)
def test_full_size_step_bf16():
    """SBM-100M on bf16 tables, one step in the benchmark's launch
    configuration: the touched rows against the oracle's bf16 step on the
    compact set of those rows (initial rows rounded to bf16, the step in
    double, each element rounded once), untouched rows bit-exact."""
    from synth import make_workload
    t0 = time.time()
    wl = make_workload("sbm100m", 0)
    cfg = wl.cfg
    src, dst, cc = wl.batch(0)
    seed, first = 2024, 3 * cfg.batch
    a = float(np.float32(cfg.init_half_width))
    tr = P.Trainer(cfg.num_nodes, cfg.dim, cfg.num_neg, cfg.batch, seed=seed, dtype="bf16")
    loss = tr.step(dev(src, torch), dev(dst, torch), dev(cc, torch), first, PARITY_LR).item()
    assert tr.check() == 0
    say(f"[sbm100m/bf16] gpu step done {time.time() - t0:.1f}s")

    n, K = src.size, cfg.num_neg
    neg = orc.sample_negatives(seed, first, n, K, cfg.num_nodes)
    rows_S = np.unique(src.astype(np.int64))
    rows_T = np.unique(np.concatenate([dst.astype(np.int64), neg.reshape(-1).astype(np.int64)]))
    S = orc.init_rows_bf16(seed, 0, rows_S, cfg.dim, a)
    T = orc.init_rows_bf16(seed, 1, rows_T, cfg.dim, a)
    ref_loss = orc.step_dense_bf16(
        S, T, np.searchsorted(rows_S, src).astype(np.int32),
        np.searchsorted(rows_T, dst).astype(np.int32), cc,
        np.searchsorted(rows_T, neg.reshape(-1)).astype(np.int32).reshape(n, K), PARITY_LR)
    say(f"[sbm100m/bf16] oracle done {time.time() - t0:.1f}s rows S {rows_S.size} T {rows_T.size}")
    uS, uT, _ = tr.stats()
    assert (uS, uT) == (rows_S.size, rows_T.size)
    assert_bf16_close(_bf16_bits(tr.get_rows(0, torch.from_numpy(rows_S)).cpu().numpy()), S,
                      "sbm100m bf16 S")
    assert_bf16_close(_bf16_bits(tr.get_rows(1, torch.from_numpy(rows_T)).cpu().numpy()), T,
                      "sbm100m bf16 T")
    assert loss == pytest.approx(ref_loss, rel=1e-5)
    rng = np.random.default_rng(1)
    for table, rows in ((0, rows_S), (1, rows_T)):
        cand = np.setdiff1d(rng.integers(0, cfg.num_nodes, 6000), rows)[:4096]
        got = _bf16_bits(tr.get_rows(table, torch.from_numpy(cand)).cpu().numpy())
        assert np.array_equal(got, orc.init_rows_bf16(seed, table, cand, cfg.dim, a))
    say(f"[sbm100m/bf16] checked {time.time() - t0:.1f}s")
    tr.close()
    del tr
