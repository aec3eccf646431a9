"""Shared helpers of the GPU tests: device copies, plan creation, and the
oracle comparisons (plan bit-exact, Y within 1e-5 * S + 1e-7 per element,
S = sum_e |a_e| |x|)."""
import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np
import pytest

import graphgen
import oracle

torch = pytest.importorskip("torch")

import paper_2308_11825_amd as agcn  # noqa: E402

DEV = "cuda:0"
RTOL, ATOL = 1e-5, 1e-7


def _dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).to(DEV)


def _plan(g, **kw):
    print(f"[plan] n={g.n_rows} nnz={g.nnz} {kw}", flush=True)
    return agcn.Plan(_dev(g.rowptr), _dev(g.colidx), _dev(g.vals), n_cols=g.n_cols, **kw)


def _params(plan):
    return plan.stats.max_block_waves, plan.stats.max_wave_nzs, plan.stats.hub_chunk_nnz


def assert_plan_matches_oracle(plan, g):
    ex = plan.export()
    W, Z, H = _params(plan)
    ref = oracle.plan(g.rowptr, g.colidx, g.vals, W, Z, H)
    assert np.array_equal(ex["perm"], ref["perm"]), "perm"
    assert np.array_equal(ex["rowptr_s"], ref["rowptr_s"]), "rowptr_s"
    assert np.array_equal(ex["colidx_s"], ref["colidx_s"]), "colidx_s"
    assert np.array_equal(ex["vals_s"].view(np.uint32), ref["vals_s"].view(np.uint32)), "vals_s"
    assert ex["meta"].shape == ref["meta"].shape, (ex["meta"].shape, ref["meta"].shape)
    assert np.array_equal(ex["meta"], ref["meta"]), "meta"
    s = plan.stats
    d = np.diff(ref["rowptr_s"].astype(np.int64))
    hub = d > s.deg_bound
    assert s.n_hub_rows == int(hub.sum())
    assert s.n_entries == len(ref["meta"])
    assert s.max_deg == (int(d.max()) if d.size else 0)
    return ex


def assert_close(Yg, Y, S, what=""):
    """Per element |Yg - Y| <= RTOL * S + ATOL. A NaN or infinity on either
    side must be the same non-finite value on the other (a NaN error would
    otherwise compare as within tolerance)."""
    assert Yg.shape == Y.shape, (what, Yg.shape, Y.shape)
    yg, y = Yg.astype(np.float64), Y.astype(np.float64)
    fin = np.isfinite(yg) & np.isfinite(y)
    same_nonfinite = (np.isnan(yg) & np.isnan(y)) | (~fin & (yg == y))
    with np.errstate(invalid="ignore"):   # inf - inf where not both finite: masked below
        err = np.where(fin, np.abs(yg - y), 0.0)
    tol = RTOL * S + ATOL
    bad = (err > tol) | (~fin & ~same_nonfinite)
    if bad.any():
        i = np.argwhere(bad)[0]
        raise AssertionError(f"{what}: {int(bad.sum())} elements out of tolerance; first at {tuple(i)}: "
                             f"gpu={Yg[tuple(i)]!r} oracle={Y[tuple(i)]!r} S={S[tuple(i)]!r}")


def _mixed(seed, n, n_cols=None, hub_max=3000, dupes=False, empty_frac=0.05):
    rng = np.random.default_rng(seed)
    n_cols = n if n_cols is None else n_cols
    deg = rng.choice([1, 2, 3, 4, 5, 7, 8, 9, 15, 16, 17, 31, 32, 33, 50, 64, 65, 100, 255, 256,
                      257, 383, 384, 385, 511, 512, 513], size=n)
    deg[rng.random(n) < empty_frac] = 0
    hubs = rng.choice(n, size=max(2, n // 400), replace=False)
    deg[hubs] = rng.integers(513, hub_max + 1, size=hubs.size)
    if not dupes:
        deg = np.minimum(deg, n_cols)
    return graphgen.random_csr(n, n_cols, deg, seed=seed + 7, dupes=dupes)


def _spmm_check(plan, g, F, X=None, seed=0):
    if X is None:
        X = np.random.default_rng(seed).standard_normal((g.n_cols, F)).astype(np.float32)
    Y, S = oracle.spmm(g.rowptr, g.colidx, g.vals, X, n_cols=g.n_cols, want_scale=True)
    Yg = plan.spmm(_dev(X)).cpu().numpy()
    assert_close(Yg, Y, S, f"F={F}")
    return Yg



_GRAPHS = {}


def _workload(name):
    if name not in _GRAPHS:
        _GRAPHS.clear()
        _GRAPHS[name] = graphgen.make(name, verbose=True)
    return _GRAPHS[name]


def _sample_rows(g, plan, k=3000, seed=0):
    rng = np.random.default_rng(seed)
    d = g.degrees
    rows = [rng.choice(g.n_rows, size=min(k, g.n_rows), replace=False), [0, g.n_rows - 1]]
    hub = np.nonzero(d > plan.stats.deg_bound)[0]
    if hub.size:
        rows.append(rng.choice(hub, size=min(300, hub.size), replace=False))
    rows.append(np.argsort(d)[-20:])
    return np.unique(np.concatenate(rows)).astype(np.int32)


def _host_workers():
    """Worker threads for the oracle checks: the host's CPU share, at most 16."""
    try:
        n = len(os.sched_getaffinity(0))
    except (AttributeError, OSError):
        n = os.cpu_count() or 1
    return max(1, min(16, n))


def assert_all_rows_close(g, X, Yg, what="", block=32768):
    """Every element of Yg (n_rows x F, original row order) against the
    oracle's definition of A X, within RTOL * S + ATOL. The oracle itself is
    the plain single-threaded function; disjoint blocks of rows are handed to
    it from several host threads (the C call releases the GIL), so that the
    full-size workloads are checked in seconds."""
    n = g.n_rows
    assert Yg.shape == (n, X.shape[1]), (what, Yg.shape)
    X = np.ascontiguousarray(X, dtype=np.float32)

    def check(s):
        rows = np.arange(s, min(n, s + block), dtype=np.int32)
        Yr, Sr = oracle.spmm_rows(g.rowptr, g.colidx, g.vals, X, rows, n_cols=g.n_cols)
        assert_close(Yg[s:s + rows.size], Yr, Sr, f"{what} rows {s}..{s + rows.size - 1}")
        return rows.size

    with ThreadPoolExecutor(_host_workers()) as ex:
        done = sum(f.result() for f in [ex.submit(check, s) for s in range(0, n, block)])
    assert done == n
    return done
