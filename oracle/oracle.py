"""CPU oracle for the HUGE embedding training step (test infrastructure only).

Only the test suite, ``__graft_entry__.smoke()`` and the benchmark's CPU
baseline may import this module.  It loads ``liboracle.so`` built from
``huge_oracle.c`` with gcc (no GPU code, nothing shared with the product
library) and adds numpy glue:

* :func:`step_dense`   -- one synchronous SGD step on whole float32 tables;
* :func:`sample_walks` -- co-occurrence triples from uniform random walks grouped
  by seed (Sec. 3.2, Alg. 1);
* :func:`lwsgd_lr`     -- the LWSGD learning-rate schedule (Table 2), as the
  piecewise-linear curve through its knots;
* :func:`eval_pairs`, :func:`pair_distances`, :func:`eval_summary`,
  :func:`knn`, :func:`recall_at_k` -- the unsupervised embedding metrics of
  Sec. 4 (edge SNR, edge and non-edge distance percentiles, sampled edge
  recall) on L2-normalised rows;
* :func:`step_sparse`  -- the same step on the rows a batch touches only, with
  every other row left at its initial value.  Tables too large for host memory
  (up to 1e8 x 128 floats) are represented by the rows the batch reads; each
  such row is produced by the oracle's own initialiser, so nothing here reads
  the GPU's tables.

Readings and formulas are stated in the header of ``huge_oracle.c``.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from dataclasses import dataclass

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "huge_oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")

_i32p = ctypes.POINTER(ctypes.c_int32)
_u32p = ctypes.POINTER(ctypes.c_uint32)
_i64p = ctypes.POINTER(ctypes.c_int64)
_f32p = ctypes.POINTER(ctypes.c_float)
_f64p = ctypes.POINTER(ctypes.c_double)


def build(force: bool = True) -> str:
    """Compile liboracle.so with gcc (plain -O2, no fast-math, no FMA contraction)."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp%d" % os.getpid()
        cmd = ["gcc", "-O2", "-std=gnu99", "-fPIC", "-shared", "-ffp-contract=off",
               "-fno-fast-math", "-Wall", "-o", tmp, _SRC, "-lm"]
        subprocess.check_call(cmd)
        os.replace(tmp, _LIB)
    return _LIB


_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
            build(force=True)
        L = ctypes.CDLL(_LIB)
        L.oracle_philox4x32_10.argtypes = [_u32p, _u32p, _u32p]
        L.oracle_philox4x32_10.restype = None
        L.oracle_init_value.argtypes = [ctypes.c_uint64, ctypes.c_int32, ctypes.c_int64,
                                        ctypes.c_int32, ctypes.c_float]
        L.oracle_init_value.restype = ctypes.c_float
        L.oracle_init_rows.argtypes = [ctypes.c_uint64, ctypes.c_int32, _i64p, ctypes.c_int64,
                                       ctypes.c_int32, ctypes.c_float, _f32p]
        L.oracle_build_alias.argtypes = [_f64p, ctypes.c_int64, _u32p, _i32p]
        L.oracle_sample_negative.argtypes = [ctypes.c_uint64, ctypes.c_uint64, ctypes.c_int32,
                                             ctypes.c_int64, _u32p, _i32p]
        L.oracle_sample_negative.restype = ctypes.c_int64
        L.oracle_sample_negatives.argtypes = [ctypes.c_uint64, ctypes.c_uint64, ctypes.c_int64,
                                              ctypes.c_int32, ctypes.c_int64, _u32p, _i32p, _i32p]
        grad_args = [_f64p, _f64p, ctypes.c_int64, ctypes.c_int64, ctypes.c_int32,
                     ctypes.c_int64, ctypes.c_int32, _i32p, _i32p, _i32p, _i32p]
        L.oracle_sgns_grad_d.argtypes = grad_args + [_f64p, _f64p, _f64p]
        L.oracle_sgns_loss_d.argtypes = grad_args + [_f64p]
        f_args = [_f32p, _f32p, ctypes.c_int64, ctypes.c_int64, ctypes.c_int32,
                  ctypes.c_int64, ctypes.c_int32, _i32p, _i32p, _i32p, _i32p]
        L.oracle_sgns_step.argtypes = f_args + [ctypes.c_float, _f64p]
        L.oracle_sgns_loss.argtypes = f_args + [_f64p]
        w_args = [_f32p, _f32p, ctypes.c_int64, ctypes.c_int64, ctypes.c_int32,
                  ctypes.c_int64, ctypes.c_int32, _i32p, _i32p, _f32p, _i32p]
        L.oracle_sgns_step_w.argtypes = w_args + [ctypes.c_float, _f64p]
        L.oracle_sgns_loss_w.argtypes = w_args + [_f64p]
        L.oracle_cocount_weights.argtypes = [_i32p, ctypes.c_int64, ctypes.c_int32, _f32p, _f32p]
        _u16p = ctypes.POINTER(ctypes.c_uint16)
        L.oracle_bf16_from_double.argtypes = [ctypes.c_double]
        L.oracle_bf16_from_double.restype = ctypes.c_uint16
        L.oracle_bf16_to_double.argtypes = [ctypes.c_uint16]
        L.oracle_bf16_to_double.restype = ctypes.c_double
        L.oracle_init_rows_bf16.argtypes = [ctypes.c_uint64, ctypes.c_int32, _i64p,
                                            ctypes.c_int64, ctypes.c_int32, ctypes.c_float, _u16p]
        L.oracle_sgns_step_bf16.argtypes = [_u16p, _u16p, ctypes.c_int64, ctypes.c_int64,
                                            ctypes.c_int32, ctypes.c_int64, ctypes.c_int32,
                                            _i32p, _i32p, _i32p, _f32p, _i32p, ctypes.c_float,
                                            _f64p]
        L.oracle_sample_walks.argtypes = [_i64p, _i32p, ctypes.c_int64, ctypes.c_int64,
                                          ctypes.c_int32, ctypes.c_int32, ctypes.c_int32,
                                          ctypes.c_int32, ctypes.c_uint64, ctypes.c_int64,
                                          ctypes.c_int64, _i32p, _i32p, _i32p, _i32p,
                                          ctypes.c_int64, _i64p]
        L.oracle_eval_pairs.argtypes = [_i64p, _i32p, ctypes.c_int64, ctypes.c_int64,
                                        ctypes.c_uint64, ctypes.c_int64, ctypes.c_int64,
                                        ctypes.c_int32, _i32p, _i32p]
        for name in ("oracle_init_rows", "oracle_build_alias", "oracle_sample_negatives",
                     "oracle_sample_walks", "oracle_eval_pairs",
                     "oracle_sgns_grad_d", "oracle_sgns_loss_d", "oracle_sgns_step",
                     "oracle_sgns_loss", "oracle_sgns_step_w", "oracle_sgns_loss_w",
                     "oracle_cocount_weights", "oracle_init_rows_bf16", "oracle_sgns_step_bf16"):
            getattr(L, name).restype = ctypes.c_int
        _lib = L
    return _lib


class OracleError(RuntimeError):
    pass


def _ptr(a: np.ndarray, t):
    if a is None:
        return None
    return a.ctypes.data_as(t)


def _check(rc: int, what: str):
    if rc != 0:
        raise OracleError(f"{what} failed with code {rc}")


def _c(a, dtype):
    return np.ascontiguousarray(a, dtype=dtype)


def _as_neg(neg, n):
    neg = _c(neg, np.int32)
    if neg.ndim == 2:
        return neg
    return neg.reshape(n, -1)


# --------------------------------------------------------------------------- #
# Random numbers
# --------------------------------------------------------------------------- #
def philox4x32_10(ctr, key) -> np.ndarray:
    c = _c(ctr, np.uint32)
    k = _c(key, np.uint32)
    out = np.zeros(4, np.uint32)
    lib().oracle_philox4x32_10(_ptr(c, _u32p), _ptr(k, _u32p), _ptr(out, _u32p))
    return out


def init_value(seed: int, table: int, row: int, col: int, half_width: float) -> float:
    return float(lib().oracle_init_value(seed, table, row, col, half_width))


def init_rows(seed: int, table: int, rows, dim: int, half_width: float) -> np.ndarray:
    r = _c(rows, np.int64)
    out = np.empty((r.size, dim), np.float32)
    _check(lib().oracle_init_rows(seed, table, _ptr(r, _i64p), r.size, dim, half_width,
                                  _ptr(out, _f32p)), "init_rows")
    return out


def build_alias(weights):
    w = _c(weights, np.float64)
    thr = np.empty(w.size, np.uint32)
    alias = np.empty(w.size, np.int32)
    _check(lib().oracle_build_alias(_ptr(w, _f64p), w.size, _ptr(thr, _u32p),
                                    _ptr(alias, _i32p)), "build_alias")
    return thr, alias


def sample_negatives(seed: int, first_pos: int, n: int, num_neg: int, num_nodes: int,
                     thr=None, alias=None) -> np.ndarray:
    out = np.empty((n, num_neg), np.int32)
    t = None if thr is None else _c(thr, np.uint32)
    a = None if alias is None else _c(alias, np.int32)
    _check(lib().oracle_sample_negatives(seed, first_pos, n, num_neg, num_nodes,
                                         _ptr(t, _u32p), _ptr(a, _i32p), _ptr(out, _i32p)),
           "sample_negatives")
    return out


# --------------------------------------------------------------------------- #
# Loss, gradient and step
# --------------------------------------------------------------------------- #
def grad_d(S, T, src, dst, cc, neg):
    """Loss and gradients in double on double tables (finite-difference pins)."""
    S = _c(S, np.float64)
    T = _c(T, np.float64)
    src, dst, cc = _c(src, np.int32), _c(dst, np.int32), _c(cc, np.int32)
    neg = _c(neg, np.int32)
    n, K = neg.shape
    gS = np.empty_like(S)
    gT = np.empty_like(T)
    loss = ctypes.c_double()
    _check(lib().oracle_sgns_grad_d(_ptr(S, _f64p), _ptr(T, _f64p), S.shape[0], T.shape[0],
                                    S.shape[1], n, K, _ptr(src, _i32p), _ptr(dst, _i32p),
                                    _ptr(cc, _i32p), _ptr(neg, _i32p), _ptr(gS, _f64p),
                                    _ptr(gT, _f64p), ctypes.byref(loss)), "sgns_grad_d")
    return loss.value, gS, gT


def loss_d(S, T, src, dst, cc, neg) -> float:
    S = _c(S, np.float64)
    T = _c(T, np.float64)
    src, dst, cc = _c(src, np.int32), _c(dst, np.int32), _c(cc, np.int32)
    neg = _c(neg, np.int32)
    n, K = neg.shape
    loss = ctypes.c_double()
    _check(lib().oracle_sgns_loss_d(_ptr(S, _f64p), _ptr(T, _f64p), S.shape[0], T.shape[0],
                                    S.shape[1], n, K, _ptr(src, _i32p), _ptr(dst, _i32p),
                                    _ptr(cc, _i32p), _ptr(neg, _i32p), ctypes.byref(loss)),
           "sgns_loss_d")
    return loss.value


def step_dense(S: np.ndarray, T: np.ndarray, src, dst, cc, neg, lr: float) -> float:
    """One step in place on float32 tables S, T (C-contiguous); returns the loss sum.
    cc: integer co_counts, or float32 weights (one per positive)."""
    assert S.dtype == np.float32 and T.dtype == np.float32
    assert S.flags.c_contiguous and T.flags.c_contiguous
    src, dst = _c(src, np.int32), _c(dst, np.int32)
    neg = _as_neg(neg, len(src))
    n, K = neg.shape
    loss = ctypes.c_double()
    if np.asarray(cc).dtype.kind == "f":
        w = _c(cc, np.float32)
        _check(lib().oracle_sgns_step_w(_ptr(S, _f32p), _ptr(T, _f32p), S.shape[0], T.shape[0],
                                        S.shape[1], n, K, _ptr(src, _i32p), _ptr(dst, _i32p),
                                        _ptr(w, _f32p), _ptr(neg, _i32p), lr,
                                        ctypes.byref(loss)), "sgns_step_w")
        return loss.value
    cc = _c(cc, np.int32)
    _check(lib().oracle_sgns_step(_ptr(S, _f32p), _ptr(T, _f32p), S.shape[0], T.shape[0],
                                  S.shape[1], n, K, _ptr(src, _i32p), _ptr(dst, _i32p),
                                  _ptr(cc, _i32p), _ptr(neg, _i32p), lr, ctypes.byref(loss)),
           "sgns_step")
    return loss.value


def loss_dense(S: np.ndarray, T: np.ndarray, src, dst, cc, neg) -> float:
    """Loss sum in double; cc: integer co_counts or float32 weights."""
    S = _c(S, np.float32)
    T = _c(T, np.float32)
    src, dst = _c(src, np.int32), _c(dst, np.int32)
    neg = _as_neg(neg, len(src))
    n, K = neg.shape
    loss = ctypes.c_double()
    if np.asarray(cc).dtype.kind == "f":
        w = _c(cc, np.float32)
        _check(lib().oracle_sgns_loss_w(_ptr(S, _f32p), _ptr(T, _f32p), S.shape[0], T.shape[0],
                                        S.shape[1], n, K, _ptr(src, _i32p), _ptr(dst, _i32p),
                                        _ptr(w, _f32p), _ptr(neg, _i32p), ctypes.byref(loss)),
               "sgns_loss_w")
        return loss.value
    cc = _c(cc, np.int32)
    _check(lib().oracle_sgns_loss(_ptr(S, _f32p), _ptr(T, _f32p), S.shape[0], T.shape[0],
                                  S.shape[1], n, K, _ptr(src, _i32p), _ptr(dst, _i32p),
                                  _ptr(cc, _i32p), _ptr(neg, _i32p), ctypes.byref(loss)),
           "sgns_loss")
    return loss.value


@dataclass
class SparseStep:
    """Result of :func:`step_sparse`: post-step values of every touched row."""
    rows_S: np.ndarray      # int64 ascending ids of touched source-table rows
    S: np.ndarray           # float32 (len(rows_S), dim), post-step
    rows_T: np.ndarray      # int64 ascending ids of touched context-table rows
    T: np.ndarray           # float32 (len(rows_T), dim), post-step
    loss: float             # loss sum over the batch, at pre-step values
    neg: np.ndarray         # int32 (n, K) negatives used


def step_sparse(seed: int, num_nodes: int, dim: int, num_neg: int, half_width: float,
                src, dst, cc, first_pos: int, lr: float, thr=None, alias=None,
                pre_S=None, pre_T=None) -> SparseStep:
    """One step from freshly initialised tables, holding only the touched rows.

    The oracle draws the negatives itself, gathers the ids the batch touches,
    materialises those rows with its own initialiser (or takes them from
    ``pre_S``/``pre_T``: dicts id -> float32 row produced by earlier oracle
    steps), relabels ids to positions in that compact set and runs the dense
    step on it.  Relabelling changes no arithmetic: the per-row accumulation
    order is still positive index, then slot.
    """
    src = _c(src, np.int32)
    dst = _c(dst, np.int32)
    cc = _c(cc, np.int32)
    n = src.size
    neg = sample_negatives(seed, first_pos, n, num_neg, num_nodes, thr, alias)
    if n and (src.min() < 0 or src.max() >= num_nodes or dst.min() < 0
              or dst.max() >= num_nodes):
        raise OracleError("id out of range")
    rows_S = np.unique(src.astype(np.int64))
    rows_T = np.unique(np.concatenate([dst.astype(np.int64), neg.reshape(-1).astype(np.int64)]))
    S = init_rows(seed, 0, rows_S, dim, half_width)
    T = init_rows(seed, 1, rows_T, dim, half_width)
    if pre_S:
        for j, r in enumerate(rows_S):
            if int(r) in pre_S:
                S[j] = pre_S[int(r)]
    if pre_T:
        for j, r in enumerate(rows_T):
            if int(r) in pre_T:
                T[j] = pre_T[int(r)]
    src_c = np.searchsorted(rows_S, src).astype(np.int32)
    dst_c = np.searchsorted(rows_T, dst).astype(np.int32)
    neg_c = np.searchsorted(rows_T, neg.reshape(-1)).astype(np.int32).reshape(n, num_neg)
    loss = step_dense(S, T, src_c, dst_c, cc, neg_c, lr)
    return SparseStep(rows_S, S, rows_T, T, loss, neg)


def cocount_weights(hist, dist_weights) -> np.ndarray:
    """float32 weight per triple from its distance histogram (n x window):
    sum_d dist_weights[d] * hist[:, d] in double (ascending d), rounded once."""
    h = _c(hist, np.int32)
    n, window = h.shape
    wd = _c(dist_weights, np.float32)
    assert wd.size == window
    out = np.empty(n, np.float32)
    _check(lib().oracle_cocount_weights(_ptr(h, _i32p), n, window, _ptr(wd, _f32p),
                                        _ptr(out, _f32p)), "cocount_weights")
    return out


def lwsgd_lr(t: int, warmup: int, peak: float, decay: int, final: float) -> float:
    """LWSGD (Table 2): linear warm-up to `peak` over `warmup` steps, linear
    decay to `final` over `decay` steps, then `final`.  Reading (the paper
    gives only the four numbers): steps count from 0 and the curve is the
    straight line through the knots (-1, 0), (warmup - 1, peak),
    (warmup + decay - 1, final), held constant after the last knot."""
    knots = [(-1.0, 0.0), (warmup - 1.0, peak), (warmup + decay - 1.0, final)]
    if t >= knots[-1][0]:
        return final
    for (x0, y0), (x1, y1) in zip(knots, knots[1:]):
        if x0 <= t <= x1 and x1 > x0:
            return y0 + (y1 - y0) * (t - x0) / (x1 - x0)
    return final


def sample_walks(off, nbr, num_nodes: int, walks_per_node: int, walk_steps: int, window: int,
                 seed_only: bool, seed: int, first_seed: int = 0, num_seeds=None):
    """Co-occurrence triples of the walks of seeds first_seed ..
    first_seed + num_seeds - 1 (see oracle_sample_walks in huge_oracle.c):
    returns (src, dst, cc, hist[n x window]) as int32 arrays."""
    L = lib()
    off = _c(off, np.int64)
    nbr = _c(nbr, np.int32)
    if num_seeds is None:
        num_seeds = num_nodes - first_seed
    count = ctypes.c_int64(0)
    args = (off.ctypes.data_as(_i64p), nbr.ctypes.data_as(_i32p), int(num_nodes),
            int(nbr.size), int(walks_per_node), int(walk_steps), int(window),
            int(bool(seed_only)), int(seed), int(first_seed), int(num_seeds))
    rc = L.oracle_sample_walks(*args, None, None, None, None, 0, ctypes.byref(count))
    if rc not in (0, -4):
        _check(rc, "oracle_sample_walks")
    n = count.value
    src = np.zeros(n, np.int32)
    dst = np.zeros(n, np.int32)
    cc = np.zeros(n, np.int32)
    hist = np.zeros((n, window), np.int32)
    rc = L.oracle_sample_walks(*args, _ptr(src, _i32p), _ptr(dst, _i32p), _ptr(cc, _i32p),
                               _ptr(hist, _i32p), n, ctypes.byref(count))
    _check(rc, "oracle_sample_walks")
    return src, dst, cc, hist


# --------------------------------------------------------------------------- #
# Embedding evaluation (Sec. 4, unsupervised metrics)
#
# Readings: embeddings are L2-normalised and compared by Euclidean distance
# (values in [0, 2], the range of the paper's distance plots); a row of zeros
# stays zero.  SNR = mean non-edge distance / mean edge distance over the
# sampled pairs.  Percentiles interpolate linearly between order statistics.
# recall@k(u) = |N(u) & S| / k, S = the k rows v != u nearest to u (ties:
# smaller id first), N(u) = the distinct ids in u's list other than u.
# --------------------------------------------------------------------------- #
def eval_pairs(off, nbr, num_nodes: int, seed: int, n_edge: int, n_non: int,
               max_tries: int = 64):
    """Edge pairs, then non-edge pairs (see oracle_eval_pairs): (u, v) int32."""
    off = _c(off, np.int64)
    nbr = _c(nbr, np.int32)
    u = np.empty(n_edge + n_non, np.int32)
    v = np.empty(n_edge + n_non, np.int32)
    _check(lib().oracle_eval_pairs(_ptr(off, _i64p), _ptr(nbr, _i32p), int(num_nodes),
                                   int(nbr.size), int(seed), int(n_edge), int(n_non),
                                   int(max_tries), _ptr(u, _i32p), _ptr(v, _i32p)),
           "eval_pairs")
    return u, v


def normalize_rows(X) -> np.ndarray:
    """Rows divided by their Euclidean norm, in double; zero rows stay zero."""
    X = np.asarray(X, dtype=np.float64)
    nrm = np.sqrt(np.sum(X * X, axis=1))
    out = np.zeros_like(X)
    nz = nrm > 0
    out[nz] = X[nz] / nrm[nz, None]
    return out


def pair_distances(table, u, v) -> np.ndarray:
    """|x_u / |x_u| - x_v / |x_v|| in double; NaN where u or v is negative."""
    u = np.asarray(u, np.int64)
    v = np.asarray(v, np.int64)
    out = np.full(u.size, np.nan)
    ok = (u >= 0) & (v >= 0)
    a = normalize_rows(np.asarray(table)[u[ok]])
    b = normalize_rows(np.asarray(table)[v[ok]])
    out[ok] = np.sqrt(np.sum((a - b) ** 2, axis=1))
    return out


def percentile_linear(values, q: float) -> float:
    """The q-th percentile (0 <= q <= 100) of the values: sorted, position
    h = (n - 1) q / 100, linear between the order statistics around h."""
    x = np.sort(np.asarray(values, dtype=np.float64))
    n = x.size
    if n == 0:
        return float("nan")
    h = (n - 1) * (q / 100.0)
    lo = int(np.floor(h))
    hi = min(lo + 1, n - 1)
    return float(x[lo] + (h - lo) * (x[hi] - x[lo]))


@dataclass
class EvalSummary:
    count_edge: int
    count_non: int
    mean_edge: float
    mean_non: float
    snr: float
    pct_edge: list
    pct_non: list


def eval_summary(d_edge, d_non, quantiles) -> EvalSummary:
    """Means over the non-NaN distances, their ratio, and percentiles."""
    e = np.asarray(d_edge, np.float64)
    e = e[~np.isnan(e)]
    m = np.asarray(d_non, np.float64)
    m = m[~np.isnan(m)]
    me = float(np.sum(e) / e.size) if e.size else float("nan")
    mn = float(np.sum(m) / m.size) if m.size else float("nan")
    return EvalSummary(int(e.size), int(m.size), me, mn, mn / me if e.size and m.size else
                       float("nan"), [percentile_linear(e, q) for q in quantiles],
                       [percentile_linear(m, q) for q in quantiles])


def knn(table, queries, k: int):
    """For each query u: the k ids v != u with the smallest distance between
    the normalised rows (ties: smaller id), and those distances; with fewer
    than k other rows, the missing places hold id -1 and distance NaN."""
    Xn = normalize_rows(table)
    ids = np.arange(Xn.shape[0])
    out_ids = np.full((len(queries), k), -1, np.int64)
    out_d = np.full((len(queries), k), np.nan)
    for qi, u in enumerate(queries):
        d = np.sqrt(np.sum((Xn - Xn[u]) ** 2, axis=1))
        keep = ids != u
        order = np.lexsort((ids[keep], d[keep]))[:k]
        out_ids[qi, :order.size] = ids[keep][order]
        out_d[qi, :order.size] = d[keep][order]
    return out_ids, out_d


def recall_at_k(off, nbr, queries, nearest, k: int) -> np.ndarray:
    """|N(u) & S| / k per query, S = the first k ids of its row of `nearest`."""
    off = np.asarray(off, np.int64)
    nbr = np.asarray(nbr)
    out = np.empty(len(queries))
    for qi, u in enumerate(queries):
        nb = set(int(x) for x in nbr[off[u]:off[u + 1]]) - {int(u)}
        S = set(int(x) for x in np.asarray(nearest[qi])[:k])
        out[qi] = len(nb & S) / k
    return out


# --------------------------------------------------------------------------- #
# bfloat16 tables (arrays of uint16: the 16 high bits of a float32)
# --------------------------------------------------------------------------- #
def bf16_from_double(x: float) -> int:
    """The bf16 nearest to x (ties to even), rounded once from x."""
    return int(lib().oracle_bf16_from_double(float(x)))


def bf16_to_float(h) -> np.ndarray:
    """Exact widening of uint16 bf16 values to float32."""
    h = np.asarray(h, np.uint16)
    return (h.astype(np.uint32) << 16).view(np.float32)


def init_rows_bf16(seed: int, table: int, rows, dim: int, half_width: float) -> np.ndarray:
    r = _c(rows, np.int64)
    out = np.empty((r.size, dim), np.uint16)
    _check(lib().oracle_init_rows_bf16(seed, table, _ptr(r, _i64p), r.size, dim, half_width,
                                       out.ctypes.data_as(ctypes.POINTER(ctypes.c_uint16))),
           "init_rows_bf16")
    return out


def step_dense_bf16(S: np.ndarray, T: np.ndarray, src, dst, cc, neg, lr: float) -> float:
    """One step in place on bf16 tables (uint16, C-contiguous); cc: integer
    co_counts or float32 weights.  Returns the loss sum (at pre-step values)."""
    assert S.dtype == np.uint16 and T.dtype == np.uint16
    assert S.flags.c_contiguous and T.flags.c_contiguous
    src, dst = _c(src, np.int32), _c(dst, np.int32)
    neg = _as_neg(neg, len(src))
    n, K = neg.shape
    if np.asarray(cc).dtype.kind == "f":
        ci, wf = None, _c(cc, np.float32)
    else:
        ci, wf = _c(cc, np.int32), None
    u16 = ctypes.POINTER(ctypes.c_uint16)
    loss = ctypes.c_double()
    _check(lib().oracle_sgns_step_bf16(S.ctypes.data_as(u16), T.ctypes.data_as(u16), S.shape[0],
                                       T.shape[0], S.shape[1], n, K, _ptr(src, _i32p),
                                       _ptr(dst, _i32p), _ptr(ci, _i32p), _ptr(wf, _f32p),
                                       _ptr(neg, _i32p), lr, ctypes.byref(loss)),
           "sgns_step_bf16")
    return loss.value
