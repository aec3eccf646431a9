"""The plan's degree sorts give the same plan.

Graphs of at most 16384 rows and 2^17 nonzeros are planned by one workgroup up
to the partition (AGCN_TEST_TINY=0 turns that off). Otherwise, with
W * Z >= 255, the plan first sorts by min(degree, 255) in one pass and sorts
the rows of degree >= 255 (the tail, at most 16384 rows) in a single
workgroup; otherwise, or with a larger tail, it runs the multi-pass radix sort
(AGCN_TEST_TAIL_CAP=-1 forces that, after the first short pass, on any graph;
the short sort's second half is then queued all the same and must leave the
plan alone). Graphs of at most 2^24 nonzeros have their column indices checked
before the short sort's last relayout, which then runs after the call returns;
larger ones in the relayout (AGCN_TEST_EARLY_CHECK_NNZ=0 forces that). Every
combination must equal the oracle's plan bit for bit (Sec. III-C: a stable
sort by degree, then Alg. 1 and Alg. 2), at the tail's edges too: degrees 254,
255 and 256, a tail whose degrees are all 255 (no tail pass), degrees that
need three tail passes, W * Z = 255 exactly, and tails of 16384 and 16385 rows.
"""
import contextlib
import os

import numpy as np
import pytest

import graphgen
from gpu_helpers import _mixed, _plan, _spmm_check, assert_plan_matches_oracle

torch = pytest.importorskip("torch")
import paper_2308_11825_amd as agcn  # noqa: E402

pytestmark = pytest.mark.gpu

TAIL_CAP = 16384


@contextlib.contextmanager
def _env(**kv):
    """Sets (value str) or clears (None) the given variables for the block."""
    old = {k: os.environ.get(k) for k in kv}
    try:
        for k, v in kv.items():
            if v is None:
                os.environ.pop(k, None)
            else:
                os.environ[k] = v
        yield
    finally:
        for k, v in old.items():
            if v is None:
                os.environ.pop(k, None)
            else:
                os.environ[k] = v


# (tail cap, early-check limit, tiny plan): the default (the single-workgroup
# plan on a small graph, else the short sort with the early column check); the
# short sort with the early column check and with the relayout's; the
# multi-pass sort after a short attempt under either.
PATHS = [(None, None, None), (None, None, "0"), (None, "0", "0"), ("-1", None, "0"),
         ("-1", "0", "0")]
MULTI = 3  # index of the first multi-pass path


def _both(g, **kw):
    """Plans of g along every path of PATHS, each checked against the oracle
    and against the others; returns the default and a multi-pass plan."""
    out = []
    for cap, early, tiny in PATHS:
        with _env(AGCN_TEST_TAIL_CAP=cap, AGCN_TEST_EARLY_CHECK_NNZ=early, AGCN_TEST_TINY=tiny):
            p = _plan(g, **kw)
        out.append((p, assert_plan_matches_oracle(p, g)))
    p0, e0 = out[0]
    for p, e in out[1:]:
        for k in ("perm", "rowptr_s", "colidx_s", "meta"):
            assert np.array_equal(e0[k], e[k]), k
        assert p0.stats.n_entries == p.stats.n_entries
    for i, (p, _) in enumerate(out):
        if i not in (0, MULTI):
            p.destroy()
    return p0, out[MULTI][0]


@pytest.mark.parametrize("W,Z", [(16, 32), (12, 32), (15, 17), (16, 256), (32, 8)])
@pytest.mark.parametrize("seed", [1, 2])
def test_short_and_multipass_sorts_agree(W, Z, seed):
    g = _mixed(900 + seed, n=20000 + 777 * seed)
    p0, p1 = _both(g, max_block_waves=W, max_wave_nzs=Z)
    _spmm_check(p0, g, 40, seed=seed)
    p0.destroy()
    p1.destroy()


def test_tail_edges():
    rng = np.random.default_rng(31)
    n = 6000
    deg = rng.choice([0, 1, 7, 253, 254, 255, 256, 257, 511, 512, 513, 900], size=n)
    g = graphgen.random_csr(n, 4000, deg, seed=32)
    for p in _both(g):
        p.destroy()
    # every tail row of degree 255: the tail keeps row order with no pass
    deg = rng.choice([3, 254, 255], size=n)
    g = graphgen.random_csr(n, 4000, deg, seed=33)
    p0, p1 = _both(g)
    assert p0.stats.max_deg == 255
    p0.destroy()
    p1.destroy()
    # tail degrees spanning three 8-bit passes (degree - 255 >= 2^16)
    deg = rng.integers(0, 300, size=3000)
    deg[[5, 77, 2999]] = [70000, 66000, 65791]
    g = graphgen.random_csr(3000, 80000, deg, seed=34)
    for p in _both(g):
        p.destroy()


@pytest.mark.parametrize("m", [TAIL_CAP, TAIL_CAP + 1])
def test_tail_at_the_cap(m):
    rng = np.random.default_rng(m)
    n = m + 30000
    deg = rng.integers(0, 255, size=n)
    tail = rng.choice(n, size=m, replace=False)
    deg[tail] = rng.integers(255, 300, size=m)
    deg[tail[:5]] = [255, 600, 1200, 299, 5000]
    g = graphgen.random_csr(n, 60000, deg, seed=m + 1)
    p = _plan(g)
    assert_plan_matches_oracle(p, g)
    _spmm_check(p, g, 16)
    p.destroy()


@pytest.mark.parametrize("cap,early,tiny", PATHS)
def test_invalid_csr_through_the_short_sort(cap, early, tiny):
    g = _mixed(950, n=5000)
    with _env(AGCN_TEST_TAIL_CAP=cap, AGCN_TEST_EARLY_CHECK_NNZ=early, AGCN_TEST_TINY=tiny):
        for where in (0, len(g.colidx) // 2, len(g.colidx) - 1):
            ci = g.colidx.copy()
            ci[where] = g.n_cols if where else -1   # one column out of range
            bad = graphgen.Graph("bad", g.n_rows, g.n_cols, g.rowptr, ci, g.vals)
            with pytest.raises(agcn.AgcnError) as e:
                _plan(bad)
            assert e.value.status == agcn.AGCN_ERR_INVALID_INPUT
            assert "column index" in str(e.value)
        rp = g.rowptr.copy()
        rp[100] = rp[101] + 1             # a decreasing row pointer
        bad = graphgen.Graph("bad", g.n_rows, g.n_cols, rp, g.colidx, g.vals)
        with pytest.raises(agcn.AgcnError) as e:
            _plan(bad)
        assert e.value.status == agcn.AGCN_ERR_INVALID_INPUT
        p = _plan(g)                      # and a valid plan right after
        assert_plan_matches_oracle(p, g)
        p.destroy()


@pytest.mark.parametrize("n", [30000, 3000])
def test_inputs_overwritten_in_stream_order_after_create(n):
    # The last relayout (of the short sort, or after the single-workgroup plan
    # of a small graph) still reads the inputs when the call returns; work
    # queued after it on the same stream may overwrite them.
    g = _mixed(960, n=n)
    dev = torch.device("cuda:0")
    rp = torch.from_numpy(g.rowptr.copy()).to(dev)
    ci = torch.from_numpy(g.colidx.copy()).to(dev)
    va = torch.from_numpy(g.vals.copy()).to(dev)
    torch.cuda.synchronize()
    for _ in range(3):
        p = agcn.Plan(rp, ci, va, n_cols=g.n_cols)
        ci.fill_(-5)
        va.fill_(float("nan"))
        rp.fill_(-3)
        assert_plan_matches_oracle(p, g)
        p.destroy()
        rp.copy_(torch.from_numpy(g.rowptr))
        ci.copy_(torch.from_numpy(g.colidx))
        va.copy_(torch.from_numpy(g.vals))


def test_short_sort_on_a_graph_whose_counts_scan_is_multi_launch():
    # Over 512 K rows: the reduction runs before the short sort's first pass,
    # whose tail (here 700 rows) is read back first.
    rng = np.random.default_rng(41)
    n = 600_000
    deg = rng.integers(0, 20, size=n)
    deg[rng.choice(n, 700, replace=False)] = rng.integers(255, 2000, size=700)
    g = graphgen.random_csr(n, 200_000, deg, seed=42)
    p0, p1 = _both(g)
    _spmm_check(p0, g, 16)
    p0.destroy()
    p1.destroy()


def test_every_row_in_the_tail_and_none():
    rng = np.random.default_rng(51)
    # every row of degree >= 255: no rows below the tail, no lower nonzeros
    deg = rng.integers(255, 700, size=2000)
    g = graphgen.random_csr(2000, 3000, deg, seed=52)
    p0, p1 = _both(g)
    assert p0.stats.n_hub_rows == int((deg > 512).sum())
    _spmm_check(p0, g, 32)
    p0.destroy()
    p1.destroy()
    # no row of degree >= 255, W * Z = 4096 (class starts up to 4097)
    deg = rng.integers(0, 255, size=5000)
    g = graphgen.random_csr(5000, 3000, deg, seed=53)
    for p in _both(g, max_block_waves=16, max_wave_nzs=256):
        p.destroy()


def test_relayout_runs_over_rows_of_one_nonzero():
    """The relayout's runs of tiles look up each tile's rows in rounds of 256
    row starts: a tile of rows of one nonzero needs the most rounds (2,048
    rows), every tile of such rows ends exactly where a row starts (the next
    tile's first row is then the one after the window), and the rows of no
    nonzero sort first. Every plan path must give the oracle's plan (the
    multi-pass sort relays out every row this way), and Y the oracle's."""
    rng = np.random.default_rng(5)
    n = 120_000
    deg = np.ones(n, np.int64)
    u = rng.random(n)
    deg[u < 0.05] = 0
    deg[(u >= 0.05) & (u < 0.15)] = 2
    deg[(u >= 0.15) & (u < 0.20)] = rng.integers(3, 40, size=int(((u >= 0.15) & (u < 0.20)).sum()))
    hubs = rng.choice(n, size=40, replace=False)
    deg[hubs] = rng.integers(300, 5000, size=hubs.size)
    g = graphgen.random_csr(n, n, deg, seed=11, dupes=True)
    p0, pm = _both(g)
    try:
        _spmm_check(p0, g, 16)
        _spmm_check(pm, g, 33)
    finally:
        p0.destroy()
        pm.destroy()
