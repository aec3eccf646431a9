"""Seeded synthetic inputs for the GCN aggregation SpMM ``Y = A_hat @ X``.

This module only builds inputs: CSR adjacency matrices (int32 row pointer and
column indices, float32 values) and dense float32 feature matrices. It holds
none of the method's arithmetic (no degree sort, no partition, no SpMM), and
both the device path's tests and the oracle's tests draw their inputs from it.

The graphs stand in for the public graphs the paper evaluates on (its Table I);
their shapes follow the five workloads below:

* ``tiny_er``          N=4096 directed Erdos-Renyi, mean out-degree 8, plus
                       self-loops; X is N x 16, uniform[-1, 1].
* ``medium_powerlaw``  N=170,000 Chung-Lu, Zipf(2.1) expected degrees, mean
                       14, cap 5000, symmetric, self-loops; X N x 32, N(0,1).
                       Shaped like ogbn-arxiv (169,343 nodes).
* ``sweep_powerlaw``   N=230,000 Chung-Lu, Zipf(2.0), mean 50, cap
                       floor(sqrt(N*50)); X N x F, N(0,1), F in 16..256.
                       Node count of Collab / Reddit.
* ``large_powerlaw``   N=2,400,000 Chung-Lu, Zipf(2.3), mean 50, cap
                       floor(sqrt(N*50)), ~120M nnz; X N x 128, uniform[-1,1].
                       Shaped like ogbn-products (2,449,029 nodes, 123.7M edges).
* ``skewed_hubs``      N=1,000,000: 999,000 rows of degree U{1..8} and 1000
                       hub rows of degree U{20,000..200,000}, uniform random
                       distinct columns, no extra self-loops; X N x 64, N(0,1).

Values follow the symmetric GCN normalisation a_ij = 1/sqrt(d_i * d_j) where
d is the final row nnz (self-loop included). For the directed graphs d_j is
j's own row nnz (every node has at least a self-loop in ``tiny_er``; in
``skewed_hubs`` every row has degree >= 1).
"""
from __future__ import annotations

import dataclasses
import time

import numpy as np

__all__ = [
    "Graph", "CONFIGS", "make", "features", "random_csr", "identity_csr",
    "permute_rows", "stats",
]


@dataclasses.dataclass
class Graph:
    name: str
    n_rows: int
    n_cols: int
    rowptr: np.ndarray   # int32 [n_rows + 1]
    colidx: np.ndarray   # int32 [nnz]
    vals: np.ndarray     # float32 [nnz]

    @property
    def nnz(self) -> int:
        return int(self.colidx.shape[0])

    @property
    def degrees(self) -> np.ndarray:
        return np.diff(self.rowptr.astype(np.int64))


# name -> (graph seed, feature seed, default F list, feature distribution)
CONFIGS = {
    "tiny_er": dict(graph_seed=1, x_seed=101, F=[16], dist="uniform"),
    "medium_powerlaw": dict(graph_seed=2, x_seed=102, F=[32], dist="normal"),
    "sweep_powerlaw": dict(graph_seed=3, x_seed=103, F=[16, 32, 64, 128, 256], dist="normal"),
    "large_powerlaw": dict(graph_seed=4, x_seed=104, F=[128], dist="uniform"),
    "skewed_hubs": dict(graph_seed=5, x_seed=105, F=[64], dist="normal"),
}


def _finish_csr(name, n, rows, cols, dedupe=True):
    """Sort (row, col) pairs, optionally de-duplicate, build CSR with GCN values."""
    key = (rows.astype(np.int64) << 32) | cols.astype(np.int64)
    del rows, cols
    key.sort()
    if dedupe and key.size:
        keep = np.empty(key.size, dtype=bool)
        keep[0] = True
        np.not_equal(key[1:], key[:-1], out=keep[1:])
        key = key[keep]
        del keep
    r = (key >> 32).astype(np.int32)
    c = (key & 0xFFFFFFFF).astype(np.int32)
    del key
    counts = np.bincount(r, minlength=n)
    rowptr = np.zeros(n + 1, dtype=np.int64)
    np.cumsum(counts, out=rowptr[1:])
    deg = counts.astype(np.float64)
    # a_ij = 1 / sqrt(d_i d_j), computed in float64, stored as float32.
    vals = (1.0 / np.sqrt(deg[r] * deg[c])).astype(np.float32)
    del r
    if rowptr[-1] >= 2**31:
        raise ValueError("nnz does not fit int32")
    return Graph(name, n, n, rowptr.astype(np.int32), c, vals)


def _powerlaw_weights(rng, n, alpha, mean, cap):
    """Zipf(alpha) expected degrees, clipped to [1, cap] and rescaled to `mean` (3 rounds)."""
    w = rng.zipf(alpha, n).astype(np.float64)
    for _ in range(3):
        w *= mean / w.mean()
        np.clip(w, 1.0, cap, out=w)
    return w


def _chung_lu(name, n, alpha, mean, cap, seed):
    """Fast Chung-Lu: n*mean/2 endpoint pairs drawn proportionally to the
    expected-degree weights, self pairs dropped, de-duplicated, symmetrised,
    then one self-loop per node."""
    rng = np.random.default_rng(seed)
    w = _powerlaw_weights(rng, n, alpha, mean, cap)
    m = int(round(n * mean / 2))
    # Endpoint multiplicities ~ Multinomial(2m, w / sum w), then a random matching.
    counts = rng.multinomial(2 * m, w / w.sum())
    ep = np.repeat(np.arange(n, dtype=np.int32), counts)
    del counts
    rng.shuffle(ep)
    a, b = ep[:m], ep[m:]
    lo = np.minimum(a, b)
    hi = np.maximum(a, b)
    del ep, a, b
    off = lo != hi
    lo, hi = lo[off], hi[off]
    und = np.unique((lo.astype(np.int64) << 32) | hi.astype(np.int64))
    del lo, hi
    lo = (und >> 32).astype(np.int32)
    hi = (und & 0xFFFFFFFF).astype(np.int32)
    del und
    diag = np.arange(n, dtype=np.int32)
    rows = np.concatenate([lo, hi, diag])
    cols = np.concatenate([hi, lo, diag])
    del lo, hi, diag
    return _finish_csr(name, n, rows, cols, dedupe=False)


def _tiny_er(seed, n=4096, mean=8):
    rng = np.random.default_rng(seed)
    p = mean / (n - 1)
    k = rng.binomial(n - 1, p, size=n)
    rows, cols = [], []
    for i in range(n):
        j = rng.choice(n - 1, size=int(k[i]), replace=False)
        j = j + (j >= i)                 # skip the diagonal
        rows.append(np.full(j.size + 1, i, dtype=np.int32))
        cols.append(np.concatenate([j.astype(np.int32), [i]]).astype(np.int32))
    return _finish_csr("tiny_er", n, np.concatenate(rows), np.concatenate(cols), dedupe=False)


def _distinct_uniform_rows(rng, n_cols, row_ids, degs):
    """For each row in `row_ids`, `degs[k]` distinct uniform columns in [0, n_cols)."""
    total = int(degs.sum())
    rows = np.repeat(row_ids.astype(np.int32), degs)
    cols = rng.integers(0, n_cols, size=total, dtype=np.int64).astype(np.int32)
    # Redraw duplicates inside a row until every row holds distinct columns.
    for _ in range(64):
        key = (rows.astype(np.int64) << 32) | cols.astype(np.int64)
        order = np.argsort(key, kind="stable")
        ks = key[order]
        dup = np.zeros(total, dtype=bool)
        dup[order[1:]] = ks[1:] == ks[:-1]
        nd = int(dup.sum())
        if nd == 0:
            return rows, cols
        cols[dup] = rng.integers(0, n_cols, size=nd, dtype=np.int64).astype(np.int32)
    raise RuntimeError("could not draw distinct columns")


def _skewed_hubs(seed, n=1_000_000, n_hubs=1000, lo=20_000, hi=200_000):
    rng = np.random.default_rng(seed)
    hub_ids = np.sort(rng.choice(n, size=n_hubs, replace=False))
    is_hub = np.zeros(n, dtype=bool)
    is_hub[hub_ids] = True
    small_ids = np.nonzero(~is_hub)[0]
    small_deg = rng.integers(1, 9, size=small_ids.size)
    r1, c1 = _distinct_uniform_rows(rng, n, small_ids, small_deg)
    hub_deg = rng.integers(lo, hi + 1, size=n_hubs)
    hr, hc = [], []
    for h, d in zip(hub_ids, hub_deg):
        # Distinct columns: a sorted sample without replacement.
        c = rng.choice(n, size=int(d), replace=False).astype(np.int32)
        hr.append(np.full(c.size, h, dtype=np.int32))
        hc.append(c)
    rows = np.concatenate([r1] + hr)
    cols = np.concatenate([c1] + hc)
    return _finish_csr("skewed_hubs", n, rows, cols, dedupe=False)


def make(name: str, seed: int | None = None, verbose: bool = False) -> Graph:
    """Build the named workload graph (deterministic for a given seed)."""
    if name not in CONFIGS:
        raise KeyError(f"unknown workload {name!r}; choose from {sorted(CONFIGS)}")
    s = CONFIGS[name]["graph_seed"] if seed is None else seed
    t0 = time.time()
    if name == "tiny_er":
        g = _tiny_er(s)
    elif name == "medium_powerlaw":
        g = _chung_lu(name, 170_000, 2.1, 14.0, 5000.0, s)
    elif name == "sweep_powerlaw":
        n = 230_000
        g = _chung_lu(name, n, 2.0, 50.0, float(int(np.sqrt(n * 50))), s)
    elif name == "large_powerlaw":
        n = 2_400_000
        g = _chung_lu(name, n, 2.3, 50.0, float(int(np.sqrt(n * 50))), s)
    else:
        g = _skewed_hubs(s)
    if verbose:
        print(f"[graphgen] {name}: {stats(g)} ({time.time() - t0:.1f}s)", flush=True)
    return g


def features(n_rows: int, F: int, seed: int, dist: str = "normal") -> np.ndarray:
    """Dense row-major float32 feature matrix, n_rows x F."""
    rng = np.random.default_rng(seed)
    if dist == "normal":
        return rng.standard_normal((n_rows, F), dtype=np.float32)
    if dist == "uniform":
        return rng.uniform(-1.0, 1.0, size=(n_rows, F)).astype(np.float32)
    raise ValueError(dist)


def weights(fin: int, fout: int, seed: int) -> np.ndarray:
    """A layer weight matrix fin x fout, float32, Glorot-uniform
    U[-sqrt(6 / (fin + fout)), +sqrt(6 / (fin + fout))] (the usual GCN init)."""
    rng = np.random.default_rng(seed)
    lim = np.sqrt(6.0 / max(1, fin + fout))
    return rng.uniform(-lim, lim, size=(fin, fout)).astype(np.float32)


def workload_features(name: str, g: Graph, F: int) -> np.ndarray:
    """Features for a named workload: drawn once at the widest F of that
    workload and column-sliced, so narrower F see the same leading columns."""
    cfg = CONFIGS[name]
    fmax = max(max(cfg["F"]), F)
    X = features(g.n_cols, fmax, cfg["x_seed"], cfg["dist"])
    return np.ascontiguousarray(X[:, :F])


def stats(g: Graph) -> dict:
    d = g.degrees
    out = dict(n=g.n_rows, nnz=g.nnz, avg_deg=round(float(d.mean()), 3) if d.size else 0.0,
               max_deg=int(d.max()) if d.size else 0)
    if d.size:
        for q in (50, 90, 99, 99.9):
            out[f"p{q}"] = float(np.percentile(d, q))
    return out


# ----------------------------------------------------------------------------
# Small graphs for tests
# ----------------------------------------------------------------------------

def random_csr(n_rows: int, n_cols: int, degrees, seed: int, dupes: bool = False,
               value_dist: str = "normal", sort_cols: bool = True) -> Graph:
    """CSR with the given per-row degrees (array) and random columns.

    With ``dupes`` the columns are drawn with replacement (repeated column
    entries inside a row are allowed, plain CSR semantics sums them); without
    it each row holds distinct columns (needs degree <= n_cols).
    """
    rng = np.random.default_rng(seed)
    deg = np.asarray(degrees, dtype=np.int64)
    assert deg.shape == (n_rows,)
    rowptr = np.zeros(n_rows + 1, dtype=np.int64)
    np.cumsum(deg, out=rowptr[1:])
    cols = []
    for i in range(n_rows):
        d = int(deg[i])
        if d == 0:
            cols.append(np.zeros(0, np.int32))
            continue
        if dupes:
            c = rng.integers(0, n_cols, size=d)
        else:
            c = rng.choice(n_cols, size=d, replace=False)
        if sort_cols:
            c = np.sort(c)
        cols.append(c.astype(np.int32))
    colidx = np.concatenate(cols) if cols else np.zeros(0, np.int32)
    colidx = colidx.astype(np.int32)
    if value_dist == "normal":
        vals = rng.standard_normal(colidx.size).astype(np.float32)
    elif value_dist == "ones":
        vals = np.ones(colidx.size, dtype=np.float32)
    else:
        vals = rng.uniform(-1, 1, colidx.size).astype(np.float32)
    return Graph("random", n_rows, n_cols, rowptr.astype(np.int32), colidx, vals)


def identity_csr(n: int) -> Graph:
    return Graph("identity", n, n, np.arange(n + 1, dtype=np.int32),
                 np.arange(n, dtype=np.int32), np.ones(n, dtype=np.float32))


def permute_rows(g: Graph, p: np.ndarray) -> Graph:
    """Row i of the result is row p[i] of g (the matrix P @ A)."""
    p = np.asarray(p, dtype=np.int64)
    deg = g.degrees[p]
    rowptr = np.zeros(g.n_rows + 1, dtype=np.int64)
    np.cumsum(deg, out=rowptr[1:])
    idx = np.concatenate([np.arange(g.rowptr[i], g.rowptr[i + 1]) for i in p]) if g.n_rows else np.zeros(0, np.int64)
    idx = idx.astype(np.int64)
    return Graph(g.name + "_perm", g.n_rows, g.n_cols, rowptr.astype(np.int32),
                 g.colidx[idx].copy(), g.vals[idx].copy())
