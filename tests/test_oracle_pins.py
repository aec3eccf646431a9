"""Pins for the CPU oracle against what the paper and the mathematics fix.

Each test checks the oracle against something other than itself: the paper's
worked example, Alg. 1's hand-derived table, library routines (numpy stable
argsort, scipy CSR row indexing and products, dense matmul), closed forms
(identity, all-ones features), invariances (row permutation, linearity) and
the coverage invariants of the block-level partition.
"""
import json
import os

import numpy as np
import pytest
import scipy.sparse as sp
from hypothesis import given, settings, strategies as st

import graphgen
import oracle


def _golden(name):
    from conftest import GOLDEN
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


def _csr_from_rowptr(rowptr, seed=0, n_cols=None):
    rowptr = np.asarray(rowptr, dtype=np.int32)
    nnz = int(rowptr[-1])
    rng = np.random.default_rng(seed)
    n = rowptr.size - 1
    n_cols = n if n_cols is None else n_cols
    colidx = rng.integers(0, n_cols, nnz).astype(np.int32)
    vals = rng.standard_normal(nnz).astype(np.float32)
    return rowptr, colidx, vals


def _scipy(g):
    return sp.csr_matrix((g.vals.astype(np.float64), g.colidx, g.rowptr), shape=(g.n_rows, g.n_cols))


def _mixed_graph(seed, n=300, n_cols=None, max_deg=900, dupes=False):
    """Degrees from several regimes: empty rows, small, mid, and hub rows."""
    rng = np.random.default_rng(seed)
    n_cols = n if n_cols is None else n_cols
    deg = rng.choice([0, 1, 2, 3, 5, 8, 17, 31, 32, 33, 64, 100, 383, 384, 385], size=n)
    hubs = rng.choice(n, size=max(1, n // 50), replace=False)
    deg[hubs] = rng.integers(385, max_deg + 1, size=hubs.size)
    if not dupes:
        deg = np.minimum(deg, n_cols)
    return graphgen.random_csr(n, n_cols, deg, seed=seed + 1, dupes=dupes)


# --------------------------------------------------------------------------
# Worked example of Sec. III-C (golden)
# --------------------------------------------------------------------------

def test_worked_example_sort_relayout_partition():
    g = _golden("worked_example_w2_z2.json")
    W, Z = g["max_block_warps"], g["max_warp_nzs"]
    rowptr, colidx, vals = _csr_from_rowptr(g["rowptr"], seed=3)
    perm = oracle.degree_sort(rowptr)
    assert perm.tolist() == g["expected_perm"]
    rowptr_s, colidx_s, vals_s = oracle.relayout(rowptr, colidx, vals, perm)
    assert rowptr_s.tolist() == g["expected_rowptr_s"]
    # Sorted row 2 is original row 1: its nnz moved to positions 4..7.
    assert colidx_s[4:8].tolist() == colidx[2:6].tolist()
    br, wn = oracle.patterns(W, Z)
    for d, (b, w) in g["expected_patterns"].items():
        assert (br[int(d)], wn[int(d)]) == (b, w), d
    meta = oracle.partition(rowptr_s, W, Z)
    assert meta.tolist() == g["expected_meta"]


def test_worked_example_warp_workloads_and_storage_ratio():
    g = _golden("worked_example_w2_z2.json")
    W, Z = g["max_block_warps"], g["max_warp_nzs"]
    rowptr, colidx, vals = _csr_from_rowptr(g["rowptr"], seed=4)
    p = oracle.plan(rowptr, colidx, vals, W, Z)
    # Replay the metadata with one-hot features so each warp's slice is visible.
    X = np.eye(3, dtype=np.float32)
    Y, cover, row_hits, hub_chunks = oracle.replay_meta(
        p["rowptr_s"], p["colidx_s"], p["vals_s"], p["perm"], p["meta"], W, Z, X)
    assert cover.tolist() == [1] * 8
    assert row_hits.tolist() == [1, 1, 1] and hub_chunks.tolist() == [0, 0, 0]
    # Slices the decode rule assigns, from the entries themselves.
    slices = []
    for deg, loc, row, info in p["meta"].tolist():
        w, rows = info >> 16, info & 0xFFFF
        wpr = -(-deg // w)
        for v in range(rows * wpr):
            rl, part = divmod(v, wpr)
            b = loc + rl * deg + part * w
            slices.append([row + rl, b, b + min(w, deg - part * w)])
    assert slices == g["expected_warp_slices"]
    # Eq. 1: block-level metadata / warp-level metadata = blocks / warps.
    assert len(p["meta"]) / g["warp_level_warps"] == pytest.approx(0.5)


# --------------------------------------------------------------------------
# Alg. 1
# --------------------------------------------------------------------------

def test_patterns_w12_z32_table():
    g = _golden("patterns_w12_z32.json")
    br, wn = oracle.patterns(g["max_block_warps"], g["max_warp_nzs"])
    assert br.size == g["deg_bound"] + 1
    for r in g["ranges"]:
        ds = np.arange(r["deg_lo"], r["deg_hi"] + 1)
        assert np.all(br[ds] == r["block_rows"])
        assert wn[ds].min() == r["warp_nzs_lo"] and wn[ds].max() == r["warp_nzs_hi"]
        # warp_nzs = ceil(deg / factor) across the whole range
        assert np.all(wn[ds] * r["factor"] >= ds) and np.all((wn[ds] - 1) * r["factor"] < ds)
    for d, (b, w) in g["spot_values"].items():
        assert (br[int(d)], wn[int(d)]) == (b, w)


@pytest.mark.parametrize("W,Z", [(1, 1), (2, 2), (12, 32), (16, 32), (8, 64), (12, 2), (6, 3),
                                 (7, 5), (16, 64), (30, 4)])
def test_patterns_cover_properties(W, Z):
    br, wn = oracle.patterns(W, Z)
    factors = [f for f in range(1, W + 1) if W % f == 0]
    for d in range(1, W * Z + 1):
        f = W // br[d]
        assert f * br[d] == W and f in factors
        assert f * Z >= d                      # f warps of Z nnz hold the row
        assert all(g * Z < d for g in factors if g < f)   # no smaller factor would
        assert wn[d] <= Z and f * wn[d] >= d and f * (wn[d] - 1) < d
        assert br[d] * d <= W * Z              # a block holds at most deg_bound nnz


def test_patterns_reject_bad_params():
    with pytest.raises(oracle.OracleError):
        oracle.patterns(0, 4)
    with pytest.raises(oracle.OracleError):
        oracle.patterns(4, 0)


# --------------------------------------------------------------------------
# Degree sort and relayout
# --------------------------------------------------------------------------

@pytest.mark.parametrize("seed", range(6))
def test_degree_sort_is_stable_ascending(seed):
    rng = np.random.default_rng(seed)
    n = int(rng.integers(1, 3000))
    deg = rng.choice([0, 1, 1, 2, 3, 3, 3, 7, 50, 1000], size=n)
    rowptr = np.concatenate([[0], np.cumsum(deg)]).astype(np.int32)
    perm = oracle.degree_sort(rowptr)
    assert perm.tolist() == np.argsort(deg, kind="stable").tolist()


def test_degree_sort_edge_cases():
    assert oracle.degree_sort(np.array([0], np.int32)).size == 0
    assert oracle.degree_sort(np.array([0, 0, 0, 0], np.int32)).tolist() == [0, 1, 2]
    assert oracle.degree_sort(np.array([0, 3, 3, 4], np.int32)).tolist() == [1, 2, 0]
    with pytest.raises(oracle.OracleError):
        oracle.degree_sort(np.array([0, 3, 2], np.int32))
    with pytest.raises(oracle.OracleError):
        oracle.degree_sort(np.array([1, 3], np.int32))


@pytest.mark.parametrize("seed", range(4))
def test_relayout_equals_scipy_row_permutation(seed):
    g = _mixed_graph(seed, n=400, dupes=bool(seed % 2))
    perm = oracle.degree_sort(g.rowptr)
    rowptr_s, colidx_s, vals_s = oracle.relayout(g.rowptr, g.colidx, g.vals, perm)
    A = sp.csr_matrix((g.vals, g.colidx, g.rowptr), shape=(g.n_rows, g.n_cols))
    B = A[perm]       # scipy keeps each row's internal order
    assert rowptr_s.tolist() == B.indptr.tolist()
    assert colidx_s.tolist() == B.indices.tolist()
    assert np.array_equal(vals_s.view(np.uint32), B.data.astype(np.float32).view(np.uint32))


# --------------------------------------------------------------------------
# SpMM by definition
# --------------------------------------------------------------------------

@pytest.mark.parametrize("seed", range(8))
def test_spmm_matches_dense_bruteforce(seed):
    rng = np.random.default_rng(100 + seed)
    n = int(rng.integers(1, 65))
    n_cols = int(rng.integers(1, 65))
    deg = rng.integers(0, 12, size=n)
    deg[rng.random(n) < 0.2] = 0                        # empty rows
    g = graphgen.random_csr(n, n_cols, deg, seed=seed, dupes=True)   # repeated columns
    F = int(rng.integers(1, 20))
    X = rng.standard_normal((n_cols, F)).astype(np.float32)
    Y, Yd, S = oracle.spmm(g.rowptr, g.colidx, g.vals, X, n_cols=n_cols, want_double=True,
                           want_scale=True)
    A = np.zeros((n, n_cols))
    Aabs = np.zeros((n, n_cols))
    for i in range(n):
        for e in range(g.rowptr[i], g.rowptr[i + 1]):
            A[i, g.colidx[e]] += float(g.vals[e])         # repeated entries add up
            Aabs[i, g.colidx[e]] += abs(float(g.vals[e]))
    ref = A @ X.astype(np.float64)
    assert np.allclose(Yd, ref, rtol=0, atol=1e-12 * (1 + np.abs(ref).max()))
    assert np.array_equal(Y, Yd.astype(np.float32))
    assert np.allclose(S, Aabs @ np.abs(X.astype(np.float64)), rtol=1e-12, atol=1e-300)
    assert np.all(S + 1e-300 >= np.abs(Yd))
    assert np.all(Y[deg == 0] == 0)


def test_spmm_matches_scipy_on_mixed_graph():
    g = _mixed_graph(7, n=500)
    rng = np.random.default_rng(8)
    X = rng.standard_normal((g.n_cols, 33)).astype(np.float32)
    Yd = oracle.spmm(g.rowptr, g.colidx, g.vals, X, want_double=True)[1]
    ref = _scipy(g) @ X.astype(np.float64)
    assert np.allclose(Yd, ref, rtol=1e-12, atol=1e-12)


def test_spmm_identity_is_exact():
    n, F = 257, 19
    g = graphgen.identity_csr(n)
    X = np.random.default_rng(1).standard_normal((n, F)).astype(np.float32)
    Y = oracle.spmm(g.rowptr, g.colidx, g.vals, X)
    assert np.array_equal(Y.view(np.uint32), X.view(np.uint32))


def test_spmm_all_ones_gives_row_sums():
    g = graphgen.make("tiny_er")
    X = np.ones((g.n_cols, 3), dtype=np.float32)
    Yd = oracle.spmm(g.rowptr, g.colidx, g.vals, X, want_double=True)[1]
    sums = np.add.reduceat(g.vals.astype(np.float64), g.rowptr[:-1]) if g.nnz else np.zeros(g.n_rows)
    for k in range(3):
        assert np.allclose(Yd[:, k], sums, rtol=1e-14, atol=0)
    # symmetric normalisation: row sums are not all 1
    assert np.abs(sums - 1).max() > 1e-3


def test_spmm_row_permutation_equivariance_bit_exact():
    g = _mixed_graph(11, n=300, dupes=True)
    rng = np.random.default_rng(12)
    X = rng.standard_normal((g.n_cols, 24)).astype(np.float32)
    p = rng.permutation(g.n_rows)
    Y = oracle.spmm(g.rowptr, g.colidx, g.vals, X)
    gp = graphgen.permute_rows(g, p)
    Yp = oracle.spmm(gp.rowptr, gp.colidx, gp.vals, X)
    assert np.array_equal(Yp.view(np.uint32), Y[p].view(np.uint32))


def test_spmm_linearity():
    g = _mixed_graph(13, n=200)
    rng = np.random.default_rng(14)
    X1 = rng.standard_normal((g.n_cols, 8)).astype(np.float32)
    X2 = rng.standard_normal((g.n_cols, 8)).astype(np.float32)
    a, b = 0.75, -2.0          # exact in float32, so a X1 + b X2 rounds once
    _, Y1, S1 = oracle.spmm(g.rowptr, g.colidx, g.vals, X1, want_double=True, want_scale=True)
    _, Y2, S2 = oracle.spmm(g.rowptr, g.colidx, g.vals, X2, want_double=True, want_scale=True)
    X3 = (a * X1.astype(np.float64) + b * X2.astype(np.float64)).astype(np.float32)
    Y3 = oracle.spmm(g.rowptr, g.colidx, g.vals, X3, want_double=True)[1]
    scale = abs(a) * S1 + abs(b) * S2
    assert np.all(np.abs(Y3 - (a * Y1 + b * Y2)) <= 1e-6 * scale + 1e-12)


def test_spmm_column_slice_and_spmv():
    g = _mixed_graph(15, n=150)
    X = np.random.default_rng(16).standard_normal((g.n_cols, 40)).astype(np.float32)
    Y = oracle.spmm(g.rowptr, g.colidx, g.vals, X)
    Y5 = oracle.spmm(g.rowptr, g.colidx, g.vals, np.ascontiguousarray(X[:, :5]))
    assert np.array_equal(Y5, Y[:, :5])
    y1 = oracle.spmm(g.rowptr, g.colidx, g.vals, np.ascontiguousarray(X[:, 7:8]))
    ref = _scipy(g) @ X[:, 7].astype(np.float64)
    assert np.allclose(y1[:, 0], ref, rtol=1e-6, atol=1e-6)


def test_spmm_rows_matches_full():
    g = _mixed_graph(17, n=220)
    X = np.random.default_rng(18).standard_normal((g.n_cols, 12)).astype(np.float32)
    Y, S = oracle.spmm(g.rowptr, g.colidx, g.vals, X, want_scale=True)
    rows = np.array([0, 5, 219, 7, 7, 100], np.int32)
    Yr, Sr = oracle.spmm_rows(g.rowptr, g.colidx, g.vals, X, rows)
    assert np.array_equal(Yr, Y[rows]) and np.array_equal(Sr, S[rows])


def test_spmm_rejects_out_of_range_column():
    g = graphgen.random_csr(4, 4, [1, 1, 1, 1], seed=0)
    g.colidx[2] = 4
    with pytest.raises(oracle.OracleError):
        oracle.spmm(g.rowptr, g.colidx, g.vals, np.zeros((4, 2), np.float32))


# --------------------------------------------------------------------------
# Block-level partition (Alg. 2) invariants
# --------------------------------------------------------------------------

PARAMS = [(12, 32, 0), (16, 32, 0), (8, 64, 0), (2, 2, 0), (12, 2, 0), (6, 3, 0), (16, 32, 100),
          (4, 8, 7), (16, 64, 2048)]


def _check_partition(rowptr_s, meta, W, Z, H):
    deg_s = np.diff(rowptr_s.astype(np.int64))
    n = deg_s.size
    DB = W * Z
    H = H if H > 0 else DB
    br_tab, wn_tab = oracle.patterns(W, Z)
    covered_rows = np.zeros(n, np.int64)
    chunks = np.zeros(n, np.int64)
    prev = None
    for b, (deg, loc, row, info) in enumerate(meta.tolist()):
        if deg <= DB:
            wn, rows = (info >> 16) & 0xFFFF, info & 0xFFFF
            assert rows >= 1                                              # I4
            assert np.all(deg_s[row:row + rows] == deg)                   # I2
            assert loc == rowptr_s[row]
            if deg == 0:
                assert wn == 0 and rows <= W
            else:
                assert wn == wn_tab[deg] and rows <= br_tab[deg]
                assert rows * deg <= DB and rows * (-(-deg // wn)) <= W   # I3
            covered_rows[row:row + rows] += 1
            key = (deg, row, loc)
        else:
            assert deg_s[row] == deg and 1 <= info <= H                   # I4
            assert rowptr_s[row] <= loc and loc + info <= rowptr_s[row + 1]
            chunks[row] += 1
            key = (deg, row, loc)
        if prev is not None:
            assert key > prev                                             # I5
        prev = key
    small = deg_s <= DB
    assert np.all(covered_rows[small] == 1) and np.all(covered_rows[~small] == 0)
    assert np.all(chunks[~small] == -(-deg_s[~small] // H)) and np.all(chunks[small] == 0)  # I7
    # I6: closed-form entry count
    want = 0
    for d in np.unique(deg_s[small]):
        c = int((deg_s == d).sum())
        want += -(-c // (W if d == 0 else int(br_tab[d])))
    want += int((-(-deg_s[~small] // H)).sum())
    assert len(meta) == want


@pytest.mark.parametrize("W,Z,H", PARAMS)
@pytest.mark.parametrize("seed", [0, 1])
def test_partition_invariants_and_replay(W, Z, H, seed):
    g = _mixed_graph(20 + seed, n=350, max_deg=1500, dupes=True)
    p = oracle.plan(g.rowptr, g.colidx, g.vals, W, Z, H)
    _check_partition(p["rowptr_s"], p["meta"], W, Z, H)
    X = np.random.default_rng(seed).standard_normal((g.n_cols, 5)).astype(np.float32)
    Y, cover, row_hits, hub_chunks = oracle.replay_meta(
        p["rowptr_s"], p["colidx_s"], p["vals_s"], p["perm"], p["meta"], W, Z, X)
    assert np.all(cover == 1)                                             # I1
    # Replaying visits each row's nnz in ascending order, so the float64 sums
    # match the definition exactly.
    assert np.array_equal(Y, oracle.spmm(g.rowptr, g.colidx, g.vals, X))


@settings(max_examples=60, deadline=None, derandomize=True)
@given(W=st.integers(1, 32), zf=st.floats(0.0, 1.0), H=st.integers(0, 4096),
       degs=st.lists(st.integers(0, 600), min_size=0, max_size=60))
def test_partition_invariants_for_any_parameters(W, zf, H, degs):
    """I1-I7 and the replay cover for parameters drawn over the whole
    accepted range (1 <= W <= 32, W * Z <= 4096, 0 <= H <= 4096) and
    arbitrary degree lists, including empty ones and rows far above
    deg_bound."""
    Z = 1 + int(zf * (4096 // W - 1))
    n = len(degs)
    g = graphgen.random_csr(n, 700, np.array(degs, dtype=np.int64), seed=n + W, dupes=True)
    p = oracle.plan(g.rowptr, g.colidx, g.vals, W, Z, H)
    _check_partition(p["rowptr_s"], p["meta"], W, Z, H)
    X = np.random.default_rng(n).standard_normal((g.n_cols, 3)).astype(np.float32)
    Y, cover, _, _ = oracle.replay_meta(
        p["rowptr_s"], p["colidx_s"], p["vals_s"], p["perm"], p["meta"], W, Z, X)
    assert np.all(cover == 1)
    assert np.array_equal(Y, oracle.spmm(g.rowptr, g.colidx, g.vals, X))


def test_partition_all_empty_rows():
    rowptr = np.zeros(40, np.int32)       # 39 rows, no nnz
    meta = oracle.partition(rowptr, 16, 32)
    assert meta.tolist() == [[0, 0, 0, 16], [0, 0, 16, 16], [0, 0, 32, 7]]
    assert oracle.partition(np.zeros(1, np.int32), 16, 32).shape == (0, 4)


def test_partition_hub_boundaries():
    W, Z = 4, 8                      # deg_bound 32
    for d, H, want_chunks in [(32, 0, None), (33, 0, [32, 1]), (64, 0, [32, 32]), (65, 0, [32, 32, 1]),
                              (100, 7, [7] * 14 + [2])]:
        rowptr = np.array([0, d], np.int32)
        meta = oracle.partition(rowptr, W, Z, H)
        if want_chunks is None:
            assert meta.tolist() == [[d, 0, 0, (8 << 16) | 1]]
        else:
            assert [m[3] for m in meta.tolist()] == want_chunks
            assert [m[1] for m in meta.tolist()] == list(np.cumsum([0] + want_chunks[:-1]))


def test_metadata_storage_ratio_eq1():
    """Sec. III-C, Eq. 1 and the storage example: with 12 warps per block and
    well-populated degree classes, block metadata is ~1/12 (about 8%) of the
    per-warp metadata."""
    rng = np.random.default_rng(5)
    deg = rng.integers(1, 385, size=200_000)
    rowptr = np.concatenate([[0], np.cumsum(deg)]).astype(np.int32)
    perm = oracle.degree_sort(rowptr)
    rowptr_s = np.concatenate([[0], np.cumsum(deg[perm])]).astype(np.int32)
    meta = oracle.partition(rowptr_s, 12, 32)
    warps = 0
    for deg_, loc, row, info in meta.tolist():
        wn, rows = info >> 16, info & 0xFFFF
        warps += rows * (-(-deg_ // wn))
    ratio = len(meta) / warps
    assert 0.080 <= ratio <= 0.086


def test_partition_rejects_bad_input():
    with pytest.raises(oracle.OracleError):
        oracle.partition(np.array([0, 5, 3], np.int32), 16, 32)
    with pytest.raises(oracle.OracleError):
        oracle.partition(np.array([0, 1], np.int32), 0, 32)


# --------------------------------------------------------------------------
# Warp-level partition (the baseline of Table II)
# --------------------------------------------------------------------------

def test_warp_partition_worked_example():
    g = _golden("worked_example_w2_z2.json")
    meta = oracle.warp_partition(np.array(g["rowptr"], np.int32), g["max_warp_nzs"])
    assert meta.tolist() == g["expected_warp_level_meta"]
    assert len(meta) == g["warp_level_warps"]


@pytest.mark.parametrize("Z", [1, 2, 7, 32, 64])
def test_warp_partition_covers_every_nnz_once(Z):
    g = _mixed_graph(50 + Z, n=300, dupes=True)
    meta = oracle.warp_partition(g.rowptr, Z)
    deg = g.degrees
    assert len(meta) == int(np.maximum(1, -(-deg // Z)).sum())
    cover = np.zeros(g.nnz, np.int64)
    prev = (-1, -1)
    for row, loc, ln, pad in meta.tolist():
        assert pad == 0 and 0 <= ln <= Z
        assert g.rowptr[row] <= loc and loc + ln <= g.rowptr[row + 1]
        assert (row, loc) > prev
        prev = (row, loc)
        cover[loc:loc + ln] += 1
        if ln == 0:
            assert deg[row] == 0
    assert np.all(cover == 1)
    # every row, empty or not, owns at least one group
    assert set(meta[:, 0].tolist()) == set(range(g.n_rows))


# --------------------------------------------------------------------------
# GCNConv layer of Sec. II-A: linear transformation, aggregation, activation
# --------------------------------------------------------------------------

def _ulp_close(a, b, ulps=1):
    """|a - b| <= ulps units in the last place of float32 at |b| (plus the
    smallest normal, for values that round to zero)."""
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    return np.all(np.abs(a - b) <= ulps * np.spacing(np.abs(b).astype(np.float32)).astype(np.float64)
                  + np.finfo(np.float32).tiny)


@pytest.mark.parametrize("n,fin,fout", [(7, 5, 3), (33, 64, 17), (1, 1, 1), (50, 3, 130)])
def test_linear_matches_numpy_float64(n, fin, fout):
    rng = np.random.default_rng(n * 1000 + fin * 10 + fout)
    X = rng.standard_normal((n, fin)).astype(np.float32)
    W = rng.standard_normal((fin, fout)).astype(np.float32)
    H = oracle.linear(X, W)
    ref = X.astype(np.float64) @ W.astype(np.float64)
    assert H.shape == (n, fout) and H.dtype == np.float32
    assert _ulp_close(H, ref)


def test_linear_closed_forms():
    rng = np.random.default_rng(1)
    X = rng.standard_normal((40, 6)).astype(np.float32)
    assert np.array_equal(oracle.linear(X, np.eye(6, dtype=np.float32)), X)
    # W selects and scales columns: H[:, c] = 2 * X[:, p[c]] exactly
    p = np.array([4, 0, 5, 5, 1])
    W = np.zeros((6, 5), np.float32)
    W[p, np.arange(5)] = 2.0
    assert np.array_equal(oracle.linear(X, W), 2.0 * X[:, p])
    assert oracle.linear(np.zeros((0, 6), np.float32), W).shape == (0, 5)
    assert np.array_equal(oracle.linear(X, np.zeros((6, 0), np.float32)), np.zeros((40, 0)))


@pytest.mark.parametrize("seed", range(4))
def test_gcn_layer_matches_dense_bruteforce(seed):
    """act(A (X W)) against a dense float64 evaluation of the same formula,
    with repeated columns and empty rows; non-square W catches a transposed
    operand."""
    rng = np.random.default_rng(seed)
    n, n_cols, fin, fout = 23, 19, 7, 5
    deg = rng.integers(0, 9, size=n)
    g = graphgen.random_csr(n, n_cols, deg, seed=seed + 40, dupes=True)
    A = np.zeros((n, n_cols))
    Aabs = np.zeros((n, n_cols))      # entry-wise |a|: repeated columns add magnitudes
    for i in range(n):
        for e in range(g.rowptr[i], g.rowptr[i + 1]):
            A[i, g.colidx[e]] += float(g.vals[e])
            Aabs[i, g.colidx[e]] += abs(float(g.vals[e]))
    X = rng.standard_normal((n_cols, fin)).astype(np.float32)
    W = rng.standard_normal((fin, fout)).astype(np.float32)
    Z = A @ (X.astype(np.float64) @ W.astype(np.float64))
    for act, ref in (("none", Z), ("relu", np.maximum(Z, 0.0))):
        Y, S2 = oracle.gcn_layer(g.rowptr, g.colidx, g.vals, X, W, act=act, want_scale=True)
        assert Y.shape == (n, fout)
        assert np.all(np.abs(Y.astype(np.float64) - ref) <= 1e-6 * S2 + 1e-30), act
        Smag = Aabs @ (np.abs(X.astype(np.float64)) @ np.abs(W.astype(np.float64)))
        assert np.allclose(S2, Smag, rtol=1e-12, atol=0)


def test_gcn_layer_reduces_to_spmm_with_identity_weights():
    g = _mixed_graph(5, n=120, max_deg=500, dupes=True)
    X = np.random.default_rng(6).standard_normal((g.n_cols, 9)).astype(np.float32)
    Y = oracle.gcn_layer(g.rowptr, g.colidx, g.vals, X, np.eye(9, dtype=np.float32), act="none")
    Ys = oracle.spmm(g.rowptr, g.colidx, g.vals, X)
    assert np.array_equal(Y.view(np.uint32), Ys.view(np.uint32))


def test_gcn_layer_relu_rows_and_nonnegative_case():
    g = _mixed_graph(7, n=90, max_deg=400)
    rng = np.random.default_rng(8)
    X = rng.standard_normal((g.n_cols, 6)).astype(np.float32)
    W = rng.standard_normal((6, 4)).astype(np.float32)
    Yn = oracle.gcn_layer(g.rowptr, g.colidx, g.vals, X, W, act="none")
    Yr = oracle.gcn_layer(g.rowptr, g.colidx, g.vals, X, W, act="relu")
    assert np.array_equal(Yr, np.maximum(Yn, 0.0))
    rows = np.array([5, 0, 89, 5], np.int32)
    assert np.array_equal(oracle.gcn_layer(g.rowptr, g.colidx, g.vals, X, W, rows=rows), Yr[rows])
    # all inputs non-negative: the scale is the value itself
    Xa, Wa, va = np.abs(X), np.abs(W), np.abs(g.vals)
    Y, S2 = oracle.gcn_layer(g.rowptr, g.colidx, va, Xa, Wa, want_scale=True)
    assert _ulp_close(Y, S2)


def test_gcn_layer_rejects_bad_input():
    g = graphgen.random_csr(4, 4, np.array([1, 2, 0, 1]), seed=1)
    X = np.ones((4, 3), np.float32)
    with pytest.raises(oracle.OracleError):
        oracle.gcn_layer(g.rowptr, g.colidx, g.vals, X, np.ones((2, 2), np.float32))
    bad = g.colidx.copy()
    bad[0] = 4
    with pytest.raises(oracle.OracleError):
        oracle.gcn_layer(g.rowptr, bad, g.vals, X, np.ones((3, 2), np.float32))
