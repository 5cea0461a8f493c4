"""Graph, walk and co-occurrence generators (numpy, seeded).

Conventions
-----------
* Every random draw comes from ``numpy.random.Generator`` seeded by a
  ``SeedSequence`` built from (workload seed, workload index, batch index), so
  any batch can be regenerated on its own.
* Node ids are relabelled by an affine bijection x -> (A x + B) mod N with
  gcd(A, N) = 1, so that block order or degree order gives no memory locality.
* A walk of ``steps`` steps visits ``steps + 1`` nodes; a walk that reaches a
  node of degree 0 stops (later positions hold -1).
* Window pairs are ordered pairs (w_a, w_b) with 1 <= |a - b| <= window, both
  directions, self pairs (w_a == w_b) dropped.
* ``co_counts`` is the number of times a pair occurs: over the whole corpus
  for the tiny workload, within its own walk for the streamed workloads.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field
from functools import lru_cache
from typing import Callable, Optional

import numpy as np


# --------------------------------------------------------------------------- #
# Workload table
# --------------------------------------------------------------------------- #
@dataclass(frozen=True)
class Config:
    name: str
    index: int
    num_nodes: int
    dim: int
    num_neg: int
    batch: int
    lr: float
    neg_kind: str          # "uniform" or "alias" (weights = degree ** 0.75)
    graph: str             # "sbm", "chung_lu"
    blocks: int = 0        # SBM
    deg_in: float = 0.0    # SBM expected degree inside the block
    deg_out: float = 0.0   # SBM expected degree to other blocks
    exponent: float = 0.0  # Chung-Lu degree exponent
    mean_deg: float = 0.0  # Chung-Lu mean degree
    walks_per_node: int = 0
    walk_steps: int = 0
    window: int = 0
    exact_graph: bool = False
    pairs: str = "walks"   # "walks" or "endpoints" (i.i.d. edge endpoints)
    cc_zipf: float = 0.0   # co_counts ~ Zipf(cc_zipf) capped at cc_cap when > 0
    cc_cap: int = 0

    @property
    def init_half_width(self) -> float:
        return 0.5 / self.dim

    def describe(self) -> dict:
        return {k: v for k, v in self.__dict__.items()}


CONFIGS = {
    "tiny": Config("tiny", 0, 10_000, 32, 5, 1024, 0.025, "uniform", "sbm", blocks=10,
                   deg_in=20.0, deg_out=1.0, walks_per_node=4, walk_steps=10, window=2,
                   exact_graph=True),
    "medium": Config("medium", 1, 1_000_000, 128, 5, 65_536, 0.025, "alias", "sbm", blocks=100,
                     deg_in=20.0, deg_out=2.0, walks_per_node=8, walk_steps=20, window=3,
                     exact_graph=True),
    # learning rates of the Chung-Lu workloads: the largest power of ten (times
    # 1 or 5) whose summed hub-row updates stay finite over a few hundred
    # steps -- a hub row takes thousands of contributions per batch, and the
    # Hub-stress co_counts reach 1000
    "powerlaw": Config("powerlaw", 2, 10_000_000, 128, 10, 131_072, 0.005, "alias", "chung_lu",
                       exponent=2.1, mean_deg=30.0, walks_per_node=4, walk_steps=40, window=5),
    "sbm100m": Config("sbm100m", 3, 100_000_000, 128, 5, 262_144, 0.025, "uniform", "sbm",
                      blocks=1000, deg_in=25.0, deg_out=2.0, walks_per_node=1, walk_steps=20,
                      window=2),
    "hubstress": Config("hubstress", 4, 50_000_000, 256, 20, 262_144, 1e-6, "alias",
                        "chung_lu", exponent=1.9, mean_deg=50.0, pairs="endpoints",
                        cc_zipf=1.5, cc_cap=1000),
    # the SBM-100M graph with the paper's 31 negatives per positive (Table 2)
    "sbm100m_k31": Config("sbm100m_k31", 5, 100_000_000, 128, 31, 262_144, 0.025, "uniform",
                          "sbm", blocks=1000, deg_in=25.0, deg_out=2.0, walks_per_node=1,
                          walk_steps=20, window=2),
}


def _rng(*key: int) -> np.random.Generator:
    return np.random.default_rng(np.random.SeedSequence([int(k) for k in key]))


# --------------------------------------------------------------------------- #
# Relabelling
# --------------------------------------------------------------------------- #
def affine_permutation(n: int, seed: int):
    """Return (A, B) with gcd(A, n) = 1: x -> (A x + B) mod n is a bijection."""
    rng = _rng(seed, 0xAFF1)
    while True:
        A = int(rng.integers(max(2, n // 3), max(3, n - 1))) if n > 3 else 1
        if math.gcd(A, n) == 1:
            break
    B = int(rng.integers(0, n))
    return A, B


def relabel(x: np.ndarray, n: int, perm) -> np.ndarray:
    A, B = perm
    x64 = x.astype(np.int64)
    out = (x64 * A + B) % n  # A < n < 2^31 and x < 2^31: fits in int64
    out[x64 < 0] = -1
    return out


# --------------------------------------------------------------------------- #
# Graphs
# --------------------------------------------------------------------------- #
def _tri_decode(t: np.ndarray):
    """Index t in [0, m(m-1)/2) -> pair (i, j), i < j, row-major over j."""
    t = t.astype(np.int64)
    j = np.floor((1.0 + np.sqrt(1.0 + 8.0 * t.astype(np.float64))) / 2.0).astype(np.int64)
    # fix rounding of the square root
    j -= (j * (j - 1) // 2 > t)
    j += ((j + 1) * j // 2 <= t)
    i = t - j * (j - 1) // 2
    return i, j


def sbm_edges(n: int, blocks: int, deg_in: float, deg_out: float, rng) -> np.ndarray:
    """Exact stochastic block model G(n, blocks, p_in, p_out), equal blocks.

    Each intra-block pair is an edge with p_in = deg_in / (B - 1), each
    inter-block pair with p_out = deg_out / (n - B) (B = n / blocks), all
    independent.  Sampling: the edge count of a pair class is Binomial, the
    edges are a uniform subset of that size.  Returns an (m, 2) int64 array
    with i < j.
    """
    B = n // blocks
    assert B * blocks == n
    p_in = deg_in / (B - 1)
    p_out = deg_out / (n - B)
    out = []
    pairs_in = B * (B - 1) // 2
    for b in range(blocks):
        m = int(rng.binomial(pairs_in, p_in))
        t = rng.choice(pairs_in, size=m, replace=False)
        i, j = _tri_decode(t)
        out.append(np.stack([i + b * B, j + b * B], 1))
    pairs_out = n * (n - 1) // 2 - blocks * pairs_in
    m_out = int(rng.binomial(pairs_out, p_out))
    have = np.zeros((0, 2), np.int64)
    while have.shape[0] < m_out:
        k = int((m_out - have.shape[0]) * 1.2) + 16
        a = rng.integers(0, n, k)
        c = rng.integers(0, n, k)
        ok = (a // B) != (c // B)
        a, c = a[ok], c[ok]
        pr = np.stack([np.minimum(a, c), np.maximum(a, c)], 1)
        have = np.unique(np.concatenate([have, pr]), axis=0)
    if have.shape[0] > m_out:
        have = have[rng.permutation(have.shape[0])[:m_out]]
    out.append(have)
    return np.concatenate(out).astype(np.int64)


def csr_from_edges(n: int, edges: np.ndarray):
    """Symmetric CSR (offsets int64, neighbours int32, sorted by source)."""
    a = np.concatenate([edges[:, 0], edges[:, 1]])
    b = np.concatenate([edges[:, 1], edges[:, 0]])
    order = np.argsort(a, kind="stable")
    a, b = a[order], b[order]
    off = np.zeros(n + 1, np.int64)
    np.add.at(off, a + 1, 1)
    off = np.cumsum(off)
    return off, b.astype(np.int32)


def chung_lu_weights(n: int, exponent: float, mean_deg: float) -> np.ndarray:
    """Expected degrees w_i proportional to (i+1)^(-1/(exponent-1)), mean mean_deg."""
    beta = 1.0 / (exponent - 1.0)
    w = np.arange(1, n + 1, dtype=np.float64) ** (-beta)
    return w * (mean_deg * n / w.sum())


# --------------------------------------------------------------------------- #
# Walks and pairs
# --------------------------------------------------------------------------- #
def walk_csr(off: np.ndarray, nbr: np.ndarray, starts: np.ndarray, steps: int, rng) -> np.ndarray:
    """Uniform random walks on a CSR graph; -1 after a dead end."""
    W = np.full((starts.size, steps + 1), -1, np.int64)
    W[:, 0] = starts
    cur = starts.astype(np.int64)
    for s in range(1, steps + 1):
        alive = cur >= 0
        deg = np.zeros_like(cur)
        deg[alive] = off[cur[alive] + 1] - off[cur[alive]]
        ok = alive & (deg > 0)
        nxt = np.full_like(cur, -1)
        r = (rng.random(cur.size) * deg).astype(np.int64)
        nxt[ok] = nbr[off[cur[ok]] + r[ok]]
        W[:, s] = nxt
        cur = nxt
    return W


def annealed_sbm_step(n: int, blocks: int, deg_in: float, deg_out: float):
    """Next-node law of a walk on an SBM with the edges re-drawn at each step.

    From x the walk moves inside x's block with probability
    deg_in / (deg_in + deg_out), to a uniform other node of the block, else to
    a uniform node of another block: the law of a uniform neighbour in the
    SBM, without the realised graph.
    """
    B = n // blocks
    p_stay = deg_in / (deg_in + deg_out)

    def step(cur: np.ndarray, rng) -> np.ndarray:
        base = (cur // B) * B
        stay = rng.random(cur.size) < p_stay
        r_in = rng.integers(0, B - 1, cur.size)
        in_blk = base + r_in + (r_in >= (cur - base))
        r_out = rng.integers(0, n - B, cur.size)
        out_blk = np.where(r_out < base, r_out, r_out + B)
        return np.where(stay, in_blk, out_blk)

    return step


def annealed_weighted_step(weights: np.ndarray):
    """Next node drawn proportional to weights, never the current node: the
    law of a uniform neighbour in a Chung-Lu multigraph."""
    cdf = np.cumsum(weights)
    cdf /= cdf[-1]

    def draw(size, rng):
        return np.minimum(np.searchsorted(cdf, rng.random(size), side="right"),
                          weights.size - 1).astype(np.int64)

    def step(cur: np.ndarray, rng) -> np.ndarray:
        nxt = draw(cur.size, rng)
        bad = nxt == cur
        while bad.any():
            nxt[bad] = draw(int(bad.sum()), rng)
            bad = nxt == cur
        return nxt

    step.draw = draw
    return step


def walk_step_fn(starts: np.ndarray, steps: int, step: Callable, rng) -> np.ndarray:
    W = np.empty((starts.size, steps + 1), np.int64)
    W[:, 0] = starts
    for s in range(1, steps + 1):
        W[:, s] = step(W[:, s - 1], rng)
    return W


def window_pairs(W: np.ndarray, window: int):
    """All ordered window pairs of every walk (rows of W), self pairs dropped."""
    src, dst = [], []
    for d in range(1, window + 1):
        a, b = W[:, :-d].reshape(-1), W[:, d:].reshape(-1)
        ok = (a >= 0) & (b >= 0) & (a != b)
        src += [a[ok], b[ok]]
        dst += [b[ok], a[ok]]
    return np.concatenate(src), np.concatenate(dst)


def aggregate_pairs(src: np.ndarray, dst: np.ndarray, n: int):
    """Collapse repeated (src, dst) pairs; co_count = multiplicity."""
    key = src.astype(np.int64) * n + dst.astype(np.int64)
    u, cnt = np.unique(key, return_counts=True)
    return (u // n).astype(np.int64), (u % n).astype(np.int64), cnt.astype(np.int64)


def _position_pairs(steps: int, window: int) -> np.ndarray:
    P = [(a, b) for a in range(steps + 1) for b in range(steps + 1) if 1 <= abs(a - b) <= window]
    return np.asarray(P, np.int64)


def tuples_from_walks(n_tuples: int, steps: int, window: int, make_walks: Callable, rng):
    """Draw triples as a uniformly shuffled per-walk-aggregated corpus would hold them.

    Each triple comes from its own walk: a uniformly chosen ordered window
    pair of that walk, accepted with probability 1 / multiplicity so that
    every distinct pair of a walk is equally likely; co_count = multiplicity
    of the pair within the walk.  Self pairs and positions past a dead end
    are rejected and drawn again.
    """
    P = _position_pairs(steps, window)
    got_s, got_d, got_c = [], [], []
    need = n_tuples
    while need > 0:
        m = int(need * 1.25) + 64
        W = make_walks(m, rng)
        pick = P[rng.integers(0, len(P), m)]
        rows = np.arange(m)
        xa = W[rows, pick[:, 0]]
        xb = W[rows, pick[:, 1]]
        valid = (xa >= 0) & (xb >= 0) & (xa != xb)
        mult = np.zeros(m, np.int64)
        for d in range(1, window + 1):
            A, B = W[:, :-d], W[:, d:]
            mult += ((A == xa[:, None]) & (B == xb[:, None])).sum(1)
            mult += ((B == xa[:, None]) & (A == xb[:, None])).sum(1)
        acc = valid & (rng.random(m) * np.maximum(mult, 1) < 1.0)
        idx = np.nonzero(acc)[0][:need]
        got_s.append(xa[idx])
        got_d.append(xb[idx])
        got_c.append(mult[idx])
        need -= idx.size
    return np.concatenate(got_s), np.concatenate(got_d), np.concatenate(got_c)


# --------------------------------------------------------------------------- #
# Workloads
# --------------------------------------------------------------------------- #
@lru_cache(maxsize=2)
def _exact_sbm(name: str, seed: int):
    cfg = CONFIGS[name]
    edges = sbm_edges(cfg.num_nodes, cfg.blocks, cfg.deg_in, cfg.deg_out, _rng(seed, cfg.index, 0xE))
    off, nbr = csr_from_edges(cfg.num_nodes, edges)
    return edges, off, nbr


@dataclass
class Workload:
    cfg: Config
    seed: int
    perm: tuple
    weights: Optional[np.ndarray] = None       # float64 per (relabelled) node id, or None
    _walks: Optional[Callable] = field(default=None, repr=False)
    _endpoint: Optional[Callable] = field(default=None, repr=False)
    csr: Optional[tuple] = field(default=None, repr=False)  # (off, nbr) before relabelling

    def batch(self, b: int, n: Optional[int] = None):
        """Batch b of n triples (default: the configured batch size), int32 arrays."""
        cfg = self.cfg
        n = cfg.batch if n is None else n
        rng = _rng(self.seed, cfg.index, 1000 + b)
        if cfg.pairs == "endpoints":
            s = np.empty(0, np.int64)
            d = np.empty(0, np.int64)
            while s.size < n:
                k = int((n - s.size) * 1.05) + 16
                a = self._endpoint(k, rng)
                c = self._endpoint(k, rng)
                ok = a != c
                s = np.concatenate([s, a[ok]])
                d = np.concatenate([d, c[ok]])
            s, d = s[:n], d[:n]
            cc = np.minimum(rng.zipf(cfg.cc_zipf, n), cfg.cc_cap)
        else:
            s, d, cc = tuples_from_walks(n, cfg.walk_steps, cfg.window, self._walks, rng)
        N = cfg.num_nodes
        return (relabel(s, N, self.perm).astype(np.int32),
                relabel(d, N, self.perm).astype(np.int32),
                cc.astype(np.int32))

    def epoch(self):
        """Tiny workload only: the whole corpus, aggregated over all walks and
        shuffled once (seeded Fisher-Yates)."""
        cfg = self.cfg
        assert cfg.exact_graph and cfg.num_nodes <= 100_000, "epoch() is for small graphs"
        off, nbr = self.csr
        rng = _rng(self.seed, cfg.index, 0xEE)
        starts = np.repeat(np.arange(cfg.num_nodes), cfg.walks_per_node)
        W = walk_csr(off, nbr, starts, cfg.walk_steps, rng)
        s, d = window_pairs(W, cfg.window)
        s, d, c = aggregate_pairs(s, d, cfg.num_nodes)
        order = rng.permutation(s.size)
        N = cfg.num_nodes
        return (relabel(s[order], N, self.perm).astype(np.int32),
                relabel(d[order], N, self.perm).astype(np.int32),
                c[order].astype(np.int32))


def make_workload(name: str, seed: int = 0) -> Workload:
    cfg = CONFIGS[name]
    N = cfg.num_nodes
    perm = affine_permutation(N, seed * 7919 + cfg.index)
    wl = Workload(cfg, seed, perm)
    if cfg.graph == "sbm" and cfg.exact_graph:
        edges, off, nbr = _exact_sbm(name, seed)
        wl.csr = (off, nbr)

        def walks(m, rng, off=off, nbr=nbr):
            return walk_csr(off, nbr, rng.integers(0, N, m), cfg.walk_steps, rng)

        wl._walks = walks
        deg = np.diff(off).astype(np.float64)
    elif cfg.graph == "sbm":
        step = annealed_sbm_step(N, cfg.blocks, cfg.deg_in, cfg.deg_out)

        def walks(m, rng, step=step):
            return walk_step_fn(rng.integers(0, N, m), cfg.walk_steps, step, rng)

        wl._walks = walks
        deg = None
    else:
        w = chung_lu_weights(N, cfg.exponent, cfg.mean_deg)
        step = annealed_weighted_step(w)
        wl._endpoint = step.draw

        def walks(m, rng, step=step):
            return walk_step_fn(rng.integers(0, N, m), cfg.walk_steps, step, rng)

        wl._walks = walks
        deg = w
    if cfg.neg_kind == "alias":
        # negatives ~ degree^0.75 (expected degree for the annealed graphs)
        wrel = np.zeros(N, np.float64)
        wrel[relabel(np.arange(N), N, perm)] = deg ** 0.75
        wl.weights = wrel
    return wl
