"""The small-plan path of the aggregation (no hub rows, every degree <= 32,
at most 2^18 nnz and 2^16 rows): one vwarp per sorted row reading its CSR
pairs directly. Y against the oracle within 1e-5 * S + 1e-7 for aligned,
unaligned (scalar) and strided layouts, the ReLU epilogue and empty rows; and
bit for bit against k_spmm, which runs for the same rows inside a graph too
large for the small path (with every degree <= Z each row is one vwarp in
both kernels)."""
import numpy as np
import pytest

import graphgen
import oracle
from gpu_helpers import DEV, _dev, _plan, _spmm_check, assert_close, assert_plan_matches_oracle

torch = pytest.importorskip("torch")
import paper_2308_11825_amd as agcn  # noqa: E402

pytestmark = pytest.mark.gpu


def _light(seed, n, n_cols=None, max_deg=32, empty_frac=0.1):
    rng = np.random.default_rng(seed)
    n_cols = n if n_cols is None else n_cols
    deg = rng.integers(1, max_deg + 1, size=n)
    deg[rng.random(n) < empty_frac] = 0
    deg[rng.choice(n, 3, replace=False)] = [0, 1, max_deg]
    return graphgen.random_csr(n, n_cols, np.minimum(deg, n_cols), seed=seed + 1)


@pytest.mark.parametrize("F", [1, 4, 16, 17, 32, 33, 64, 100, 256])
def test_small_path_matches_oracle(F):
    g = _light(701, n=5000)
    plan = _plan(g)
    assert plan.stats.n_hub_rows == 0 and plan.stats.max_deg <= 32 and g.nnz <= 1 << 18
    if F == 16:
        assert_plan_matches_oracle(plan, g)
    _spmm_check(plan, g, F, seed=F)
    plan.destroy()


def test_small_path_strides_relu_and_rectangular():
    g = _light(711, n=3000, n_cols=700)
    plan = _plan(g)
    X = np.random.default_rng(3).standard_normal((700, 40)).astype(np.float32)
    Xd = _dev(np.pad(X, ((0, 0), (0, 9))))[:, :40]          # row stride 49
    Yd = torch.full((3000, 45), float("nan"), device=DEV)
    plan.spmm(Xd, out=Yd[:, :40], act="relu")
    Y, S = oracle.spmm(g.rowptr, g.colidx, g.vals, X, n_cols=700, want_scale=True)
    assert_close(Yd[:, :40].cpu().numpy(), np.maximum(Y, 0), S, "small path, strided, relu")
    assert torch.isnan(Yd[:, 40:]).all()                     # untouched past F
    plan.destroy()


def test_small_path_equals_k_spmm_bit_for_bit():
    small = _light(721, n=4000)
    n_big = 40000                                            # nnz > 2^18: k_spmm runs
    rng = np.random.default_rng(722)
    deg_extra = rng.integers(1, 33, size=n_big - small.n_rows)
    extra = graphgen.random_csr(n_big - small.n_rows, small.n_cols, deg_extra, seed=723)
    rowptr = np.concatenate([small.rowptr, extra.rowptr[1:] + small.rowptr[-1]]).astype(np.int32)
    big = graphgen.Graph("big", n_big, small.n_cols, rowptr,
                         np.concatenate([small.colidx, extra.colidx]),
                         np.concatenate([small.vals, extra.vals]))
    assert big.nnz > 1 << 18
    ps, pb = _plan(small), _plan(big)
    for F in (16, 64, 18):
        X = _dev(np.random.default_rng(F).standard_normal((small.n_cols, F)).astype(np.float32))
        ys = ps.spmm(X).cpu().numpy()
        yb = pb.spmm(X).cpu().numpy()[: small.n_rows]
        assert np.array_equal(ys.view(np.uint32), yb.view(np.uint32)), F
    ps.destroy()
    pb.destroy()


def test_small_path_all_empty_and_one_row():
    g = graphgen.random_csr(64, 64, np.zeros(64, np.int64), seed=5)
    plan = _plan(g)
    Y = plan.spmm(_dev(np.ones((64, 8), np.float32))).cpu().numpy()
    assert np.array_equal(Y, np.zeros((64, 8), np.float32))
    plan.destroy()
    g = graphgen.random_csr(1, 10, np.array([7]), seed=6)
    plan = _plan(g)
    _spmm_check(plan, g, 12)
    plan.destroy()
