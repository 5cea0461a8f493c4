"""Pins for the oracle's loss, gradient and SGD step.

Independent checks, none of which retypes the oracle's code:
  * closed form: with every dot product zero the loss is ln 2 (1+K) sum c and
    the coefficients are -c/2 and c/2;
  * brute force on a 5-node path graph, term by term in plain Python;
  * central finite differences of the loss;
  * a third implementation: PyTorch CPU autograd in float64;
  * invariants: linearity in co_counts, duplicates equal summed weight,
    synchronous reads, untouched rows unchanged, error handling.
"""
import math

import numpy as np
import pytest
import torch

from oracle import oracle as orc


def _rand_problem(rng, ns, nt, dim, n, K, scale=0.5, cmax=4):
    S = rng.normal(0, scale, (ns, dim))
    T = rng.normal(0, scale, (nt, dim))
    src = rng.integers(0, ns, n).astype(np.int32)
    dst = rng.integers(0, nt, n).astype(np.int32)
    cc = rng.integers(0, cmax + 1, n).astype(np.int32)
    neg = rng.integers(0, nt, (n, K)).astype(np.int32)
    return S, T, src, dst, cc, neg


# --------------------------------------------------------------------------- #
# Closed form at zero dot products
# --------------------------------------------------------------------------- #
def test_zero_context_table_closed_form():
    rng = np.random.default_rng(1)
    ns, nt, dim, n, K = 6, 9, 4, 5, 3
    S = rng.uniform(-1, 1, (ns, dim)).astype(np.float32)
    T = np.zeros((nt, dim), np.float32)
    src = np.array([0, 1, 2, 3, 4], np.int32)
    dst = np.array([0, 1, 2, 3, 4], np.int32)
    cc = np.array([1, 2, 3, 1, 5], np.int32)
    neg = np.array([[5, 6, 7], [5, 6, 8], [6, 7, 8], [5, 7, 8], [6, 5, 8]], np.int32)
    lr = np.float32(0.1)
    S0 = S.copy()
    loss = orc.step_dense(S, T, src, dst, cc, neg, float(lr))
    assert loss == pytest.approx(math.log(2) * (1 + K) * cc.sum(), rel=1e-14)
    # dS = g T[v] + sum h T[m] = 0 -> S unchanged (rewritten with the same value)
    assert np.array_equal(S, S0)
    # dT[v] = g S[u] with g = -c/2 ; dT[m] += c/2 S[u]
    gT = np.zeros((nt, dim))
    for i in range(n):
        gT[dst[i]] += -cc[i] / 2.0 * S0[src[i]].astype(np.float64)
        for k in range(K):
            gT[neg[i, k]] += cc[i] / 2.0 * S0[src[i]].astype(np.float64)
    expect = (0.0 - float(lr) * gT).astype(np.float32)
    assert np.allclose(T, expect, rtol=1e-6, atol=1e-9)


# --------------------------------------------------------------------------- #
# Brute force on a 5-node path graph
# --------------------------------------------------------------------------- #
def _sigmoid(z):
    return 1.0 / (1.0 + math.exp(-z))


def test_five_node_path_brute_force():
    """Path 0-1-2-3-4: positives are its edges in both directions with window 1.

    The loss is enumerated term by term with scalar Python arithmetic.  For
    every positive (u, v, c) with negatives m_1..m_K it adds
    c * log(1 + exp(-<S_u, T_v>)) and c * log(1 + exp(<S_u, T_m>)), i.e. minus
    the log-likelihood of word2vec negative sampling weighted by co_counts.
    """
    rng = np.random.default_rng(3)
    dim, K = 3, 2
    S = rng.normal(0, 0.7, (5, dim))
    T = rng.normal(0, 0.7, (5, dim))
    edges = [(0, 1), (1, 2), (2, 3), (3, 4)]
    pos = [(a, b) for a, b in edges] + [(b, a) for a, b in edges]
    src = np.array([p[0] for p in pos], np.int32)
    dst = np.array([p[1] for p in pos], np.int32)
    cc = np.array([1, 2, 1, 3, 2, 1, 1, 2], np.int32)
    neg = np.array([[(u + 2) % 5, (u + 3) % 5] for u in src], np.int32)

    expect = 0.0
    for i in range(len(pos)):
        u, v, c = int(src[i]), int(dst[i]), float(cc[i])
        x = sum(S[u, d] * T[v, d] for d in range(dim))
        expect += c * math.log(1.0 + math.exp(-x))
        for k in range(K):
            m = int(neg[i, k])
            y = sum(S[u, d] * T[m, d] for d in range(dim))
            expect += c * math.log(1.0 + math.exp(y))
    got = orc.loss_d(S, T, src, dst, cc, neg)
    assert got == pytest.approx(expect, rel=1e-13)
    loss, gS, gT = orc.grad_d(S, T, src, dst, cc, neg)
    assert loss == pytest.approx(expect, rel=1e-13)
    # gradient of the source row of node 2, written out by hand
    g_expect = np.zeros(dim)
    for i in range(len(pos)):
        if src[i] != 2:
            continue
        c = float(cc[i])
        x = float(S[2] @ T[dst[i]])
        g_expect += c * (_sigmoid(x) - 1.0) * T[dst[i]]
        for k in range(K):
            y = float(S[2] @ T[neg[i, k]])
            g_expect += c * _sigmoid(y) * T[neg[i, k]]
    assert np.allclose(gS[2], g_expect, rtol=1e-12, atol=1e-14)


# --------------------------------------------------------------------------- #
# Finite differences
# --------------------------------------------------------------------------- #
def test_gradient_matches_central_differences():
    rng = np.random.default_rng(4)
    S, T, src, dst, cc, neg = _rand_problem(rng, 5, 5, 3, 6, 2)
    # include a repeated source, a destination that is also a negative
    src[1] = src[0]
    neg[2, 0] = dst[2]
    loss, gS, gT = orc.grad_d(S, T, src, dst, cc, neg)
    h = 1e-6
    for X, G in ((S, gS), (T, gT)):
        for idx in np.ndindex(X.shape):
            old = X[idx]
            X[idx] = old + h
            lp = orc.loss_d(S, T, src, dst, cc, neg)
            X[idx] = old - h
            lm = orc.loss_d(S, T, src, dst, cc, neg)
            X[idx] = old
            fd = (lp - lm) / (2 * h)
            assert abs(fd - G[idx]) <= 1e-7 * max(1.0, abs(G[idx])), (idx, fd, G[idx])


# --------------------------------------------------------------------------- #
# Third implementation: PyTorch CPU autograd (float64)
# --------------------------------------------------------------------------- #
def test_gradient_matches_torch_autograd():
    rng = np.random.default_rng(5)
    S, T, src, dst, cc, neg = _rand_problem(rng, 20, 30, 8, 64, 4)
    src[:10] = 3  # heavy duplicates
    neg[5, :] = dst[5]
    loss, gS, gT = orc.grad_d(S, T, src, dst, cc, neg)

    St = torch.tensor(S, dtype=torch.float64, requires_grad=True)
    Tt = torch.tensor(T, dtype=torch.float64, requires_grad=True)
    s = St[torch.from_numpy(src.astype(np.int64))]
    tp = Tt[torch.from_numpy(dst.astype(np.int64))]
    tn = Tt[torch.from_numpy(neg.astype(np.int64))]
    c = torch.from_numpy(cc.astype(np.float64))
    x = (s * tp).sum(-1)
    y = torch.einsum("nd,nkd->nk", s, tn)
    L = (c * (torch.nn.functional.softplus(-x) + torch.nn.functional.softplus(y).sum(-1))).sum()
    L.backward()
    assert loss == pytest.approx(L.item(), rel=1e-12)
    assert np.allclose(gS, St.grad.numpy(), rtol=1e-11, atol=1e-13)
    assert np.allclose(gT, Tt.grad.numpy(), rtol=1e-11, atol=1e-13)


# --------------------------------------------------------------------------- #
# Invariants
# --------------------------------------------------------------------------- #
def test_gradient_linear_in_co_counts():
    rng = np.random.default_rng(6)
    S, T, src, dst, cc, neg = _rand_problem(rng, 10, 10, 5, 20, 3)
    _, gS1, gT1 = orc.grad_d(S, T, src, dst, cc, neg)
    l1 = orc.loss_d(S, T, src, dst, cc, neg)
    _, gS2, gT2 = orc.grad_d(S, T, src, dst, 2 * cc, neg)
    l2 = orc.loss_d(S, T, src, dst, 2 * cc, neg)
    # scaling by a power of two commutes with every rounding: bitwise
    assert np.array_equal(gS2, 2 * gS1) and np.array_equal(gT2, 2 * gT1)
    assert l2 == 2 * l1
    c_a = rng.integers(0, 5, cc.size).astype(np.int32)
    c_b = rng.integers(0, 5, cc.size).astype(np.int32)
    _, gSa, gTa = orc.grad_d(S, T, src, dst, c_a, neg)
    _, gSb, gTb = orc.grad_d(S, T, src, dst, c_b, neg)
    _, gSs, gTs = orc.grad_d(S, T, src, dst, c_a + c_b, neg)
    assert np.allclose(gSs, gSa + gSb, rtol=1e-12, atol=1e-14)
    assert np.allclose(gTs, gTa + gTb, rtol=1e-12, atol=1e-14)
    # zero co_count contributes nothing
    _, gS0, gT0 = orc.grad_d(S, T, src, dst, np.zeros_like(cc), neg)
    assert not gS0.any() and not gT0.any()


def test_duplicate_positive_equals_summed_weight():
    rng = np.random.default_rng(7)
    S, T, _, _, _, _ = _rand_problem(rng, 6, 6, 4, 1, 2)
    m = 5
    src = np.full(m, 2, np.int32)
    dst = np.full(m, 4, np.int32)
    cc = np.full(m, 3, np.int32)
    neg = np.tile(np.array([[1, 5]], np.int32), (m, 1))
    l_rep, gS_rep, gT_rep = orc.grad_d(S, T, src, dst, cc, neg)
    l_one, gS_one, gT_one = orc.grad_d(S, T, src[:1], dst[:1], cc[:1] * m, neg[:1])
    assert l_rep == pytest.approx(l_one, rel=1e-14)
    assert np.allclose(gS_rep, gS_one, rtol=1e-13, atol=1e-15)
    assert np.allclose(gT_rep, gT_one, rtol=1e-13, atol=1e-15)


def test_synchronous_reads_when_destination_is_also_negative():
    """T[v] is read once per occurrence at its pre-step value; contributions add."""
    S = np.array([[0.3, -0.2]], np.float64)
    T = np.array([[0.5, 0.1], [0.0, 0.0]], np.float64)
    src = np.array([0], np.int32)
    dst = np.array([0], np.int32)
    cc = np.array([2], np.int32)
    neg = np.array([[0, 1]], np.int32)
    _, gS, gT = orc.grad_d(S, T, src, dst, cc, neg)
    x = float(S[0] @ T[0])
    g = 2 * (_sigmoid(x) - 1)
    h0 = 2 * _sigmoid(x)          # same dot: negative 0 is row 0 again
    h1 = 2 * _sigmoid(0.0)
    assert np.allclose(gT[0], (g + h0) * S[0], rtol=1e-14)
    assert np.allclose(gT[1], h1 * S[0], rtol=1e-14)
    assert np.allclose(gS[0], g * T[0] + h0 * T[0] + h1 * T[1], rtol=1e-14)
    # the step applies exactly that sum once, from the pre-step value
    Sf, Tf = S.astype(np.float32), T.astype(np.float32)
    orc.step_dense(Sf, Tf, src, dst, cc, neg, 0.5)
    assert np.allclose(Tf[0], (T[0] - 0.5 * (g + h0) * S[0]).astype(np.float32), rtol=1e-6)


def test_step_touches_only_batch_rows_and_matches_gradient():
    rng = np.random.default_rng(8)
    S, T, src, dst, cc, neg = _rand_problem(rng, 40, 50, 6, 12, 3, scale=0.2)
    S32, T32 = S.astype(np.float32), T.astype(np.float32)
    S0, T0 = S32.copy(), T32.copy()
    lr = 0.05
    loss = orc.step_dense(S32, T32, src, dst, cc, neg, lr)
    l_ref, gS, gT = orc.grad_d(S0.astype(np.float64), T0.astype(np.float64), src, dst, cc, neg)
    assert loss == l_ref
    touched_S = np.zeros(40, bool)
    touched_S[src] = True
    touched_T = np.zeros(50, bool)
    touched_T[dst] = True
    touched_T[neg.reshape(-1)] = True
    assert np.array_equal(S32[~touched_S], S0[~touched_S])
    assert np.array_equal(T32[~touched_T], T0[~touched_T])
    exp_S = (S0.astype(np.float64) - np.float64(np.float32(lr)) * gS).astype(np.float32)
    exp_T = (T0.astype(np.float64) - np.float64(np.float32(lr)) * gT).astype(np.float32)
    assert np.array_equal(S32[touched_S], exp_S[touched_S])
    assert np.array_equal(T32[touched_T], exp_T[touched_T])
    assert orc.loss_dense(S0, T0, src, dst, cc, neg) == pytest.approx(loss, rel=1e-15)


def test_errors_leave_tables_untouched():
    rng = np.random.default_rng(9)
    S, T, src, dst, cc, neg = _rand_problem(rng, 8, 8, 4, 6, 2)
    S32, T32 = S.astype(np.float32), T.astype(np.float32)
    S0, T0 = S32.copy(), T32.copy()
    bad = dst.copy()
    bad[3] = 8
    with pytest.raises(orc.OracleError, match="-2"):
        orc.step_dense(S32, T32, src, bad, cc, neg, 0.1)
    badc = cc.copy()
    badc[0] = -1
    with pytest.raises(orc.OracleError, match="-3"):
        orc.step_dense(S32, T32, src, dst, badc, neg, 0.1)
    badn = neg.copy()
    badn[1, 1] = -4
    with pytest.raises(orc.OracleError, match="-2"):
        orc.step_dense(S32, T32, src, dst, cc, badn, 0.1)
    assert np.array_equal(S32, S0) and np.array_equal(T32, T0)


def test_empty_batch_is_a_no_op():
    S = np.ones((3, 4), np.float32)
    T = np.ones((3, 4), np.float32)
    e = np.zeros(0, np.int32)
    loss = orc.step_dense(S, T, e, e, e, np.zeros((0, 2), np.int32), 0.1)
    assert loss == 0.0 and np.all(S == 1) and np.all(T == 1)


def test_sparse_step_equals_dense_step_from_init():
    seed, N, dim, K, a = 21, 300, 8, 3, np.float32(0.5 / 8)
    rng = np.random.default_rng(10)
    n = 200
    src = rng.integers(0, N, n).astype(np.int32)
    dst = rng.integers(0, N, n).astype(np.int32)
    cc = rng.integers(1, 4, n).astype(np.int32)
    S = orc.init_rows(seed, 0, np.arange(N), dim, a)
    T = orc.init_rows(seed, 1, np.arange(N), dim, a)
    neg = orc.sample_negatives(seed, 1000, n, K, N)
    loss = orc.step_dense(S, T, src, dst, cc, neg, 0.025)
    sp = orc.step_sparse(seed, N, dim, K, float(a), src, dst, cc, 1000, 0.025)
    assert sp.loss == loss
    assert np.array_equal(sp.neg, neg)
    assert np.array_equal(sp.S, S[sp.rows_S])
    assert np.array_equal(sp.T, T[sp.rows_T])
