"""CPU oracle for the Accel-GCN aggregation path -- TEST INFRASTRUCTURE ONLY.

The plain, slow, single-threaded statement of what the device path computes
(C++ in ``agcn_oracle.cpp``, float64 accumulation), wrapped with numpy. Only
the tests, the package smoke check and the benchmark's CPU-baseline leg may
import this module; the device library and its Python binding never do.

Functions and the passages of the paper they follow:

* ``degree_sort``   Sec. III-C "Degree Sorting", steps (1)-(2)
* ``relayout``      Sec. III-C "Degree Sorting", step (3)
* ``patterns``      Alg. 1 (get partition patterns)
* ``partition``     Alg. 2 (block-level partitioning) + the metadata format
* ``spmm``          Sec. II-A / II-B, the aggregation A' Y by definition
* ``spmm_rows``     the same for selected rows
* ``replay_meta``   Sec. III-C, last paragraph (warp workload from metadata)
* ``warp_partition`` Sec. III-C panel (b): the warp-level partition baseline
* ``plan``          degree_sort + relayout + partition in one call
* ``linear``        Sec. II-A, the linear transformation H = X W
* ``gcn_layer``     Sec. II-A, a GCNConv forward act(A' (X W)), optionally for
                    selected rows

The readings taken where the paper is silent are listed in agcn_oracle.h.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "liboracle_agcn.so")
SRC_PATH = os.path.join(_HERE, "agcn_oracle.cpp")

_i32p = ctypes.POINTER(ctypes.c_int32)
_f32p = ctypes.POINTER(ctypes.c_float)
_f64p = ctypes.POINTER(ctypes.c_double)
_lib = None


def build(force: bool = True) -> str:
    """Compile the oracle with g++ (single-threaded, -O2, no FP contraction)."""
    if force or not os.path.exists(LIB_PATH):
        tmp = LIB_PATH + ".tmp"
        cmd = ["g++", "-O2", "-std=c++17", "-ffp-contract=off", "-fno-fast-math", "-Wall",
               "-shared", "-fPIC", SRC_PATH, "-o", tmp]
        subprocess.run(cmd, check=True)
        os.replace(tmp, LIB_PATH)
    return LIB_PATH


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        build(force=False)
    lib = ctypes.CDLL(LIB_PATH)
    lib.oracle_degree_sort.argtypes = [ctypes.c_int32, _i32p, _i32p]
    lib.oracle_degree_sort.restype = ctypes.c_int
    lib.oracle_relayout.argtypes = [ctypes.c_int32, _i32p, _i32p, _f32p, _i32p, _i32p, _i32p, _f32p]
    lib.oracle_relayout.restype = ctypes.c_int
    lib.oracle_patterns.argtypes = [ctypes.c_int32, ctypes.c_int32, _i32p, _i32p]
    lib.oracle_patterns.restype = ctypes.c_int
    lib.oracle_partition.argtypes = [ctypes.c_int32, _i32p, ctypes.c_int32, ctypes.c_int32,
                                     ctypes.c_int32, _i32p, ctypes.c_int64]
    lib.oracle_partition.restype = ctypes.c_int64
    lib.oracle_warp_partition.argtypes = [ctypes.c_int32, _i32p, ctypes.c_int32, _i32p,
                                          ctypes.c_int64]
    lib.oracle_warp_partition.restype = ctypes.c_int64
    lib.oracle_spmm.argtypes = [ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, _i32p, _i32p,
                                _f32p, _f32p, ctypes.c_int64, _f32p, ctypes.c_int64, _f64p, _f64p]
    lib.oracle_spmm.restype = ctypes.c_int
    lib.oracle_spmm_rows.argtypes = [ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, _i32p, _i32p,
                                     _f32p, _f32p, ctypes.c_int64, _i32p, ctypes.c_int32, _f32p,
                                     _f64p]
    lib.oracle_spmm_rows.restype = ctypes.c_int
    lib.oracle_replay_meta.argtypes = [ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, _i32p,
                                       _i32p, _f32p, _i32p, _i32p, ctypes.c_int64, ctypes.c_int32,
                                       ctypes.c_int32, _f32p, ctypes.c_int64, _f32p, _i32p, _i32p,
                                       _i32p]
    lib.oracle_replay_meta.restype = ctypes.c_int
    lib.oracle_linear.argtypes = [ctypes.c_int64, ctypes.c_int32, ctypes.c_int32, _f32p,
                                  ctypes.c_int64, _f32p, ctypes.c_int64, _f32p, ctypes.c_int64]
    lib.oracle_linear.restype = ctypes.c_int
    lib.oracle_gcn_layer_rows.argtypes = [ctypes.c_int32, ctypes.c_int32, ctypes.c_int32,
                                          ctypes.c_int32, _i32p, _i32p, _f32p, _f32p,
                                          ctypes.c_int64, _f32p, ctypes.c_int64, ctypes.c_int32,
                                          _i32p, ctypes.c_int32, _f32p, _f64p]
    lib.oracle_gcn_layer_rows.restype = ctypes.c_int
    _lib = lib
    return lib


def _p(a, t):
    return a.ctypes.data_as(t) if a is not None else None


def _i32(a):
    return np.ascontiguousarray(a, dtype=np.int32)


def _f32(a):
    return np.ascontiguousarray(a, dtype=np.float32)


class OracleError(RuntimeError):
    pass


def degree_sort(rowptr) -> np.ndarray:
    rowptr = _i32(rowptr)
    n = rowptr.size - 1
    perm = np.empty(n, dtype=np.int32)
    if _load().oracle_degree_sort(n, _p(rowptr, _i32p), _p(perm, _i32p)) != 0:
        raise OracleError("degree_sort: invalid row pointer")
    return perm


def relayout(rowptr, colidx, vals, perm):
    rowptr, colidx, vals, perm = _i32(rowptr), _i32(colidx), _f32(vals), _i32(perm)
    n = rowptr.size - 1
    nnz = int(rowptr[-1]) if n >= 0 else 0
    rowptr_s = np.empty(n + 1, dtype=np.int32)
    colidx_s = np.empty(nnz, dtype=np.int32)
    vals_s = np.empty(nnz, dtype=np.float32)
    rc = _load().oracle_relayout(n, _p(rowptr, _i32p), _p(colidx, _i32p), _p(vals, _f32p),
                                 _p(perm, _i32p), _p(rowptr_s, _i32p), _p(colidx_s, _i32p),
                                 _p(vals_s, _f32p))
    if rc != 0:
        raise OracleError("relayout: invalid input")
    return rowptr_s, colidx_s, vals_s


def patterns(max_block_warps: int, max_warp_nzs: int):
    """Alg. 1: arrays block_rows[d], warp_nzs[d] for d = 0..W*Z (index 0 unused)."""
    n = max_block_warps * max_warp_nzs + 1
    br = np.zeros(n, dtype=np.int32)
    wn = np.zeros(n, dtype=np.int32)
    if _load().oracle_patterns(max_block_warps, max_warp_nzs, _p(br, _i32p), _p(wn, _i32p)) != 0:
        raise OracleError("patterns: invalid parameters")
    return br, wn


def partition(rowptr_s, max_block_warps: int, max_warp_nzs: int, hub_chunk_nnz: int = 0):
    """Alg. 2: metadata entries as an (n_entries, 4) int32 array {deg, loc, row, info}."""
    rowptr_s = _i32(rowptr_s)
    n = rowptr_s.size - 1
    lib = _load()
    cnt = lib.oracle_partition(n, _p(rowptr_s, _i32p), max_block_warps, max_warp_nzs,
                               hub_chunk_nnz, None, 0)
    if cnt < 0:
        raise OracleError("partition: invalid input")
    meta = np.zeros((max(cnt, 1), 4), dtype=np.int32)
    got = lib.oracle_partition(n, _p(rowptr_s, _i32p), max_block_warps, max_warp_nzs,
                               hub_chunk_nnz, _p(meta, _i32p), cnt)
    if got != cnt:
        raise OracleError("partition: count mismatch")
    return meta[:cnt]


def warp_partition(rowptr, max_warp_nzs: int):
    """Warp-level partition: (n_groups, 4) int32 {row, first nnz, nnz count, 0}."""
    rowptr = _i32(rowptr)
    n = rowptr.size - 1
    lib = _load()
    cnt = lib.oracle_warp_partition(n, _p(rowptr, _i32p), max_warp_nzs, None, 0)
    if cnt < 0:
        raise OracleError("warp_partition: invalid input")
    meta = np.zeros((max(cnt, 1), 4), dtype=np.int32)
    if lib.oracle_warp_partition(n, _p(rowptr, _i32p), max_warp_nzs, _p(meta, _i32p), cnt) != cnt:
        raise OracleError("warp_partition: count mismatch")
    return meta[:cnt]


def spmm(rowptr, colidx, vals, X, n_cols=None, want_double=False, want_scale=False):
    """Y = A X by definition; optionally the float64 sums and the |a||x| scale S."""
    rowptr, colidx, vals = _i32(rowptr), _i32(colidx), _f32(vals)
    X = _f32(X)
    n = rowptr.size - 1
    F = X.shape[1]
    n_cols = X.shape[0] if n_cols is None else n_cols
    Y = np.empty((n, F), dtype=np.float32)
    Yd = np.empty((n, F), dtype=np.float64) if want_double else None
    S = np.empty((n, F), dtype=np.float64) if want_scale else None
    rc = _load().oracle_spmm(n, n_cols, F, _p(rowptr, _i32p), _p(colidx, _i32p), _p(vals, _f32p),
                             _p(X, _f32p), F, _p(Y, _f32p), F, _p(Yd, _f64p), _p(S, _f64p))
    if rc != 0:
        raise OracleError("spmm: invalid input")
    out = [Y]
    if want_double:
        out.append(Yd)
    if want_scale:
        out.append(S)
    return out[0] if len(out) == 1 else tuple(out)


def spmm_rows(rowptr, colidx, vals, X, rows, n_cols=None):
    """(Y_rows, S_rows) for the selected original rows."""
    rowptr, colidx, vals, X, rows = _i32(rowptr), _i32(colidx), _f32(vals), _f32(X), _i32(rows)
    n = rowptr.size - 1
    F = X.shape[1]
    n_cols = X.shape[0] if n_cols is None else n_cols
    Y = np.empty((rows.size, F), dtype=np.float32)
    S = np.empty((rows.size, F), dtype=np.float64)
    rc = _load().oracle_spmm_rows(n, n_cols, F, _p(rowptr, _i32p), _p(colidx, _i32p),
                                  _p(vals, _f32p), _p(X, _f32p), F, _p(rows, _i32p), rows.size,
                                  _p(Y, _f32p), _p(S, _f64p))
    if rc != 0:
        raise OracleError("spmm_rows: invalid input")
    return Y, S


def replay_meta(rowptr_s, colidx_s, vals_s, perm, meta, max_block_warps, max_warp_nzs, X,
                n_cols=None):
    """Walk every entry with the warp-workload rule; returns (Y, cover, row_hits, hub_chunks)."""
    rowptr_s, colidx_s, vals_s, perm = _i32(rowptr_s), _i32(colidx_s), _f32(vals_s), _i32(perm)
    meta = _i32(meta).reshape(-1, 4)
    X = _f32(X)
    n = rowptr_s.size - 1
    F = X.shape[1]
    n_cols = X.shape[0] if n_cols is None else n_cols
    Y = np.empty((n, F), dtype=np.float32)
    cover = np.empty(int(rowptr_s[-1]), dtype=np.int32)
    row_hits = np.empty(n, dtype=np.int32)
    hub_chunks = np.empty(n, dtype=np.int32)
    rc = _load().oracle_replay_meta(n, n_cols, F, _p(rowptr_s, _i32p), _p(colidx_s, _i32p),
                                    _p(vals_s, _f32p), _p(perm, _i32p), _p(meta, _i32p),
                                    meta.shape[0], max_block_warps, max_warp_nzs, _p(X, _f32p), F,
                                    _p(Y, _f32p), _p(cover, _i32p), _p(row_hits, _i32p),
                                    _p(hub_chunks, _i32p))
    if rc != 0:
        raise OracleError("replay_meta: an entry decodes outside the sorted CSR")
    return Y, cover, row_hits, hub_chunks


def plan(rowptr, colidx, vals, max_block_warps, max_warp_nzs, hub_chunk_nnz=0):
    """Degree sort, relayout and partition: dict(perm, rowptr_s, colidx_s, vals_s, meta)."""
    perm = degree_sort(rowptr)
    rowptr_s, colidx_s, vals_s = relayout(rowptr, colidx, vals, perm)
    meta = partition(rowptr_s, max_block_warps, max_warp_nzs, hub_chunk_nnz)
    return dict(perm=perm, rowptr_s=rowptr_s, colidx_s=colidx_s, vals_s=vals_s, meta=meta)


def linear(X, W):
    """H = X W (float32 result of float64 sums)."""
    X, W = _f32(X), _f32(W)
    n, fin = X.shape
    fin2, fout = W.shape
    if fin2 != fin:
        raise OracleError("linear: inner dimensions differ")
    H = np.empty((n, fout), dtype=np.float32)
    if _load().oracle_linear(n, fin, fout, _p(X, _f32p), max(fin, 1), _p(W, _f32p), max(fout, 1),
                             _p(H, _f32p), max(fout, 1)) != 0:
        raise OracleError("linear: invalid input")
    return H


def gcn_layer(rowptr, colidx, vals, X, W, act="relu", rows=None, n_cols=None, want_scale=False):
    """act(A' (X W)) for all rows or for `rows`; optionally the scale S2."""
    rowptr, colidx, vals = _i32(rowptr), _i32(colidx), _f32(vals)
    X, W = _f32(X), _f32(W)
    n = rowptr.size - 1
    fin, fout = W.shape
    if X.shape[1] != fin:
        raise OracleError("gcn_layer: X and W disagree on fin")
    n_cols = X.shape[0] if n_cols is None else n_cols
    a = {"none": 0, "relu": 1}[act]
    rows_a = None if rows is None else _i32(rows)
    m = n if rows_a is None else rows_a.size
    Y = np.empty((m, fout), dtype=np.float32)
    S2 = np.empty((m, fout), dtype=np.float64) if want_scale else None
    rc = _load().oracle_gcn_layer_rows(n, n_cols, fin, fout, _p(rowptr, _i32p), _p(colidx, _i32p),
                                       _p(vals, _f32p), _p(X, _f32p), max(fin, 1), _p(W, _f32p),
                                       max(fout, 1), a, _p(rows_a, _i32p), m, _p(Y, _f32p),
                                       _p(S2, _f64p))
    if rc != 0:
        raise OracleError("gcn_layer: invalid input")
    return (Y, S2) if want_scale else Y
