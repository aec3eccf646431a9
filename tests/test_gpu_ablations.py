"""GPU parity of the two ablation baselines of Table II, through the C ABI.

* AGCN_PLAN_WARP_LEVEL: the warp-level partition (no degree sort, groups of
  <= Z nnz in row order). Plan: identity permutation, the input CSR, and
  metadata bit-exact against oracle.warp_partition. Y within the same
  per-element bound as the main path.
* AGCN_PLAN_COLUMN_LOOP: the block-level plan (bit-exact against oracle.plan,
  it is the same plan) executed by a single-warp column loop. Y within the
  same bound.
"""
import numpy as np
import pytest

import graphgen
import oracle

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

import paper_2308_11825_amd as agcn  # noqa: E402

from gpu_helpers import (DEV, _dev, _mixed, _plan, _spmm_check, assert_all_rows_close,  # noqa: E402
                         _workload, assert_close, assert_plan_matches_oracle)

WL = agcn.AGCN_PLAN_WARP_LEVEL
CL = agcn.AGCN_PLAN_COLUMN_LOOP


def assert_warp_plan_matches_oracle(plan, g):
    ex = plan.export()
    s = plan.stats
    assert s.flags == WL
    ref = oracle.warp_partition(g.rowptr, s.max_wave_nzs)
    assert np.array_equal(ex["perm"], np.arange(g.n_rows, dtype=np.int32)), "perm"
    assert np.array_equal(ex["rowptr_s"], g.rowptr), "rowptr_s"
    assert np.array_equal(ex["colidx_s"], g.colidx), "colidx_s"
    assert np.array_equal(ex["vals_s"].view(np.uint32), g.vals.view(np.uint32)), "vals_s"
    assert ex["meta"].shape == ref.shape, (ex["meta"].shape, ref.shape)
    assert np.array_equal(ex["meta"], ref), "meta"
    assert s.n_entries == len(ref) and s.n_hub_rows == 0 and s.n_hub_chunks == 0
    d = np.diff(g.rowptr.astype(np.int64))
    assert s.max_deg == (int(d.max()) if d.size else 0)
    return ex


# ---------------------------------------------------------------------------
# Warp-level partition
# ---------------------------------------------------------------------------

WL_PARAMS = [dict(max_block_waves=16, max_wave_nzs=32), dict(max_block_waves=12, max_wave_nzs=32),
             dict(max_block_waves=4, max_wave_nzs=2), dict(max_block_waves=32, max_wave_nzs=64),
             dict(max_block_waves=1, max_wave_nzs=5), dict(max_block_waves=7, max_wave_nzs=3)]


@pytest.mark.parametrize("kw", WL_PARAMS)
def test_warp_level_plan_and_spmm(kw):
    g = _mixed(51, n=7000, hub_max=5000, dupes=True)
    plan = _plan(g, flags=WL, **kw)
    assert_warp_plan_matches_oracle(plan, g)
    for F in (1, 3, 16, 17, 64, 100):
        _spmm_check(plan, g, F, seed=F)
    plan.destroy()


@pytest.fixture(scope="module")
def wl_plan():
    g = _mixed(53, n=12000, hub_max=6000)
    plan = _plan(g, flags=WL)
    yield g, plan
    plan.destroy()


@pytest.mark.parametrize("F", [4, 8, 32, 33, 96, 128, 256, 257, 512])
def test_warp_level_spmm_matches_oracle(wl_plan, F):
    g, plan = wl_plan
    _spmm_check(plan, g, F, seed=F)


def test_warp_level_rows_spanning_many_workgroups():
    """Rows of thousands of nnz cut into groups of 2 cover hundreds of
    workgroups: the boundary fix-up adds runs of 16 partials in order."""
    deg = np.array([0, 1, 5000, 3, 0, 2999, 64, 0, 7], np.int64)
    g = graphgen.random_csr(deg.size, 6000, deg, seed=5)
    plan = _plan(g, flags=WL, max_block_waves=4, max_wave_nzs=2)
    assert_warp_plan_matches_oracle(plan, g)
    for F in (1, 4, 16, 40):
        _spmm_check(plan, g, F, seed=F)
    plan.destroy()


def test_warp_level_deterministic_and_unaligned(wl_plan):
    g, plan = wl_plan
    X = np.random.default_rng(9).standard_normal((g.n_cols, 64)).astype(np.float32)
    Xd = _dev(X)
    Y1 = plan.spmm(Xd).cpu().numpy()
    Y2 = plan.spmm(Xd).cpu().numpy()
    assert np.array_equal(Y1.view(np.uint32), Y2.view(np.uint32))
    Y, S = oracle.spmm(g.rowptr, g.colidx, g.vals, X, want_scale=True)
    buf = torch.empty(g.n_cols * 64 + 1, dtype=torch.float32, device=DEV)
    Xu = buf[1:].view(g.n_cols, 64)
    Xu.copy_(Xd)
    assert_close(plan.spmm(Xu).cpu().numpy(), Y, S, "unaligned X (32-bit path)")


def test_warp_level_identity_and_edge_cases():
    g = graphgen.identity_csr(3000)
    plan = _plan(g, flags=WL)
    assert_warp_plan_matches_oracle(plan, g)
    X = np.random.default_rng(2).standard_normal((3000, 20)).astype(np.float32)
    assert np.array_equal(plan.spmm(_dev(X)).cpu().numpy().view(np.uint32), X.view(np.uint32))
    plan.destroy()
    for deg in ([0] * 37, [5], [3, 40, 0, 7, 33]):
        g = graphgen.random_csr(len(deg), 100, np.array(deg), seed=3, dupes=True)
        plan = _plan(g, flags=WL, max_block_waves=4, max_wave_nzs=8)
        assert_warp_plan_matches_oracle(plan, g)
        for F in (1, 8, 17):
            _spmm_check(plan, g, F)
        plan.destroy()


def test_warp_level_empty_matrix_and_invalid_csr():
    g = graphgen.Graph("empty", 0, 0, np.zeros(1, np.int32), np.zeros(0, np.int32),
                       np.zeros(0, np.float32))
    plan = _plan(g, flags=WL)
    assert plan.stats.n_entries == 0
    assert plan.spmm(torch.zeros((0, 8), device=DEV)).shape == (0, 8)
    plan.destroy()
    g = graphgen.random_csr(100, 100, np.full(100, 3), seed=1)
    bad = g.colidx.copy()
    bad[57] = -1
    with pytest.raises(agcn.AgcnError) as ei:
        agcn.Plan(_dev(g.rowptr), _dev(bad), _dev(g.vals), n_cols=100, flags=WL)
    assert ei.value.status == agcn.AGCN_ERR_INVALID_INPUT
    rp = g.rowptr.copy()
    rp[40] = rp[41] + 1
    with pytest.raises(agcn.AgcnError) as ei:
        agcn.Plan(_dev(rp), _dev(g.colidx), _dev(g.vals), n_cols=100, flags=WL)
    assert ei.value.status == agcn.AGCN_ERR_INVALID_INPUT


# ---------------------------------------------------------------------------
# Column loop (block-level partition without the combined warp)
# ---------------------------------------------------------------------------

@pytest.fixture(scope="module")
def cl_plan():
    g = _mixed(57, n=12000, hub_max=6000)
    plan = _plan(g, flags=CL)
    yield g, plan
    plan.destroy()


def test_column_loop_plan_is_the_block_level_plan(cl_plan):
    g, plan = cl_plan
    assert plan.stats.flags == CL
    assert_plan_matches_oracle(plan, g)


@pytest.mark.parametrize("F", [1, 3, 4, 17, 32, 64, 65, 128, 200, 256])
def test_column_loop_spmm_matches_oracle(cl_plan, F):
    g, plan = cl_plan
    _spmm_check(plan, g, F, seed=F)


@pytest.mark.parametrize("kw", [dict(max_block_waves=4, max_wave_nzs=8),
                                dict(max_block_waves=16, max_wave_nzs=32, hub_chunk_nnz=1000),
                                dict(max_block_waves=2, max_wave_nzs=2)])
def test_column_loop_other_params(kw):
    g = _mixed(59, n=5000, hub_max=3000, dupes=True)
    plan = _plan(g, flags=CL, **kw)
    assert_plan_matches_oracle(plan, g)
    for F in (1, 16, 70):
        _spmm_check(plan, g, F, seed=F)
    plan.destroy()


def test_column_loop_matches_main_path_bit_exact_when_unsplit():
    """Rows held by one vwarp sum in the same order on both paths (fp32 FMA
    in nnz order), so the two paths agree bit for bit on them."""
    deg = np.random.default_rng(3).integers(1, 9, size=4000)
    g = graphgen.random_csr(deg.size, deg.size, deg, seed=4)
    pa = _plan(g, max_block_waves=16, max_wave_nzs=32)
    pb = _plan(g, max_block_waves=16, max_wave_nzs=32, flags=CL)
    X = _dev(np.random.default_rng(5).standard_normal((g.n_cols, 64)).astype(np.float32))
    Ya, Yb = pa.spmm(X).cpu().numpy(), pb.spmm(X).cpu().numpy()
    assert np.array_equal(Ya.view(np.uint32), Yb.view(np.uint32))
    pa.destroy()
    pb.destroy()


def test_column_loop_lds_limit_is_an_error(cl_plan):
    g, plan = cl_plan
    F = 4096              # W * F * 4 bytes of partial rows > 64 KiB
    X = torch.zeros((g.n_cols, F), device=DEV)
    with pytest.raises(agcn.AgcnError) as ei:
        plan.spmm(X)
    assert ei.value.status == agcn.AGCN_ERR_UNSUPPORTED


# ---------------------------------------------------------------------------
# Full-size workload, the configuration the benchmark's ablation lines time
# ---------------------------------------------------------------------------

@pytest.mark.slow
@pytest.mark.parametrize("flags", [WL, CL])
def test_ablation_workload_parity(flags):
    name = "sweep_powerlaw"
    g = _workload(name)
    plan = _plan(g, flags=flags)
    if flags == WL:
        assert_warp_plan_matches_oracle(plan, g)
    else:
        assert_plan_matches_oracle(plan, g)
    for F in graphgen.CONFIGS[name]["F"]:
        X = graphgen.workload_features(name, g, F)
        Yg = plan.spmm(_dev(X)).cpu().numpy()
        n = assert_all_rows_close(g, X, Yg, f"{name} flags={flags} F={F}")
        print(f"[parity] {name} flags={flags} F={F} ok (all {n} rows checked)", flush=True)
    plan.destroy()
