"""GPU parity: the HIP path, called through the C ABI, against the CPU oracle.

* Plan (permutation, sorted CSR, metadata): bit-exact.
* Y: |Y_gpu - Y_oracle| <= 1e-5 * S + 1e-7 per element, S = sum_e |a_e| |x|.
* Determinism, row-permutation equivariance and the identity case: bit-exact.
"""
import numpy as np
import pytest

import graphgen
import oracle

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

import paper_2308_11825_amd as agcn  # noqa: E402

from gpu_helpers import (DEV, _dev, _mixed, _plan, _sample_rows, _spmm_check, assert_all_rows_close,  # noqa: E402
                         _workload, assert_close, assert_plan_matches_oracle)


# ---------------------------------------------------------------------------
# Plan parity
# ---------------------------------------------------------------------------

PARAM_SETS = [dict(), dict(max_block_waves=12, max_wave_nzs=32), dict(max_block_waves=8,
              max_wave_nzs=64), dict(max_block_waves=16, max_wave_nzs=32, hub_chunk_nnz=1000),
              dict(max_block_waves=2, max_wave_nzs=2), dict(max_block_waves=6, max_wave_nzs=3)]

# Parameter extremes: the widest block (W = 32), the largest block (W Z = 4096),
# the largest hub chunk, a single vwarp per block.
EXTREME_PARAMS = [dict(max_block_waves=32, max_wave_nzs=64), dict(max_block_waves=4, max_wave_nzs=1024),
                  dict(max_block_waves=16, max_wave_nzs=32, hub_chunk_nnz=4096),
                  dict(max_block_waves=1, max_wave_nzs=1), dict(max_block_waves=1, max_wave_nzs=512)]


@pytest.mark.parametrize("kw", EXTREME_PARAMS)
def test_parameter_extremes_plan_and_spmm(kw):
    g = _mixed(13, n=6000, hub_max=9000, dupes=True)
    plan = _plan(g, **kw)
    assert_plan_matches_oracle(plan, g)
    for F in (2, 5, 32, 48, 100):
        _spmm_check(plan, g, F, seed=F)
    plan.destroy()


@pytest.mark.parametrize("kw", PARAM_SETS)
@pytest.mark.parametrize("seed", [0, 1])
def test_plan_bit_exact_random(kw, seed):
    g = _mixed(seed, n=9000 + 1777 * seed, dupes=bool(seed))
    plan = _plan(g, **kw)
    assert_plan_matches_oracle(plan, g)
    plan.destroy()


def test_plan_bit_exact_drawn_parameters():
    """Device plan against the oracle, and the SpMM, for 24 (W, Z, H) drawn
    over the whole accepted range (1 <= W <= 32, W * Z <= 4096,
    0 <= H <= 4096) on small graphs with empty, short and hub rows."""
    rng = np.random.default_rng(2024)
    ran = 0
    for i in range(24):
        W = int(rng.integers(1, 33))
        Z = int(rng.integers(1, 4096 // W + 1))
        H = int(rng.choice([0, int(rng.integers(1, 4097))]))
        g = _mixed(100 + i, n=int(rng.integers(50, 3000)), hub_max=6000, dupes=bool(i % 2))
        print(f"[drawn] W={W} Z={Z} H={H} n={g.n_rows} nnz={g.nnz}", flush=True)
        try:
            plan = _plan(g, max_block_waves=W, max_wave_nzs=Z, hub_chunk_nnz=H)
        except agcn.AgcnError as e:   # the one further limit: one entry's staging in 64 KiB of LDS
            assert e.status == agcn.AGCN_ERR_INVALID_ARGUMENT and "LDS" in str(e), str(e)
            continue
        assert_plan_matches_oracle(plan, g)
        _spmm_check(plan, g, int(rng.choice([3, 16, 40])), seed=i)
        plan.destroy()
        ran += 1
    assert ran >= 12


@pytest.mark.parametrize("n", [64 * 4096 - 1, 64 * 4096, 64 * 4096 + 1])
def test_plan_at_the_single_pass_scan_limit(n):
    """The row-pointer scan has n values: up to 64 tiles of 4096 run in one
    pass (decoupled look-back), more in two passes. Both sides of the limit
    give the oracle's plan bit for bit and a matching SpMM."""
    deg = np.random.default_rng(n).integers(0, 6, size=n)
    g = graphgen.random_csr(n, n, deg, seed=n % 1000)
    plan = _plan(g)
    assert_plan_matches_oracle(plan, g)
    _spmm_check(plan, g, 32, seed=3)
    plan.destroy()


@pytest.mark.parametrize("case", ["one_row", "all_empty", "deg_eq_bound", "deg_multiple_bound",
                                  "deg_bound_plus_one", "single_hub", "no_nnz_cols", "rect"])
def test_plan_and_spmm_edge_cases(case):
    W, Z = 4, 8
    DB = W * Z
    n_cols = None
    if case == "one_row":
        deg = [5]
    elif case == "all_empty":
        deg = [0] * 37
    elif case == "deg_eq_bound":
        deg = [DB] * 11 + [1] * 3
    elif case == "deg_multiple_bound":
        deg = [3 * DB] * 3 + [2] * 5
    elif case == "deg_bound_plus_one":
        deg = [DB + 1] * 4 + [DB - 1] * 4
    elif case == "single_hub":
        deg = [0] * 3 + [1] * 100 + [5000]
    elif case == "no_nnz_cols":
        deg = [0, 0, 0]
        n_cols = 0
    else:  # rectangular: more columns than rows
        deg = [3, 40, 0, 7, 33]
        n_cols = 6000
    n = len(deg)
    nc = n_cols if n_cols is not None else max(n, max(deg) + 1 if deg else 1)
    g = graphgen.random_csr(n, nc, np.array(deg), seed=3, dupes=True)
    plan = _plan(g, max_block_waves=W, max_wave_nzs=Z)
    assert_plan_matches_oracle(plan, g)
    for F in (1, 4, 16, 17):
        if nc == 0:
            X = np.zeros((0, F), np.float32)
            Yg = plan.spmm(_dev(X)).cpu().numpy()
            assert np.all(Yg == 0)
        else:
            _spmm_check(plan, g, F)
    plan.destroy()


def test_empty_matrix():
    g = graphgen.Graph("empty", 0, 0, np.zeros(1, np.int32), np.zeros(0, np.int32),
                       np.zeros(0, np.float32))
    plan = _plan(g)
    assert plan.stats.n_entries == 0
    Y = plan.spmm(torch.zeros((0, 8), device=DEV))
    assert Y.shape == (0, 8)
    plan.destroy()


# ---------------------------------------------------------------------------
# SpMM parity across F and layouts
# ---------------------------------------------------------------------------

@pytest.fixture(scope="module")
def mixed_plan():
    g = _mixed(11, n=12000, hub_max=6000)
    plan = _plan(g)
    yield g, plan
    plan.destroy()


@pytest.mark.parametrize("F", [1, 2, 3, 4, 5, 8, 16, 17, 32, 33, 48, 64, 96, 128, 256, 257, 320,
                               512, 1024])
def test_spmm_matches_oracle(mixed_plan, F):
    g, plan = mixed_plan
    _spmm_check(plan, g, F, seed=F)


def test_spmm_unaligned_and_strided(mixed_plan):
    g, plan = mixed_plan
    rng = np.random.default_rng(5)
    F = 64
    X = rng.standard_normal((g.n_cols, F)).astype(np.float32)
    Y, S = oracle.spmm(g.rowptr, g.colidx, g.vals, X, want_scale=True)
    # X starting one float past an aligned address: the 32-bit path.
    buf = torch.empty(g.n_cols * F + 1, dtype=torch.float32, device=DEV)
    Xu = buf[1:].view(g.n_cols, F)
    Xu.copy_(_dev(X))
    assert Xu.data_ptr() % 16 != 0
    assert_close(plan.spmm(Xu).cpu().numpy(), Y, S, "unaligned X")
    # Row strides larger than F for both X and Y.
    Xs = torch.zeros((g.n_cols, F + 12), dtype=torch.float32, device=DEV)
    Xs[:, :F] = _dev(X)
    Ys = torch.full((g.n_rows, F + 8), 7.0, dtype=torch.float32, device=DEV)
    plan.spmm(Xs[:, :F], out=Ys[:, :F])
    assert_close(Ys[:, :F].cpu().numpy(), Y, S, "strided")
    assert torch.all(Ys[:, F:] == 7.0)      # padding untouched
    # ldy not a multiple of 4 -> 32-bit path
    Ys2 = torch.empty((g.n_rows, F + 1), dtype=torch.float32, device=DEV)
    plan.spmm(_dev(X), out=Ys2[:, :F])
    assert_close(Ys2[:, :F].cpu().numpy(), Y, S, "odd ldy")


def test_spmm_deterministic_and_column_slicing(mixed_plan):
    g, plan = mixed_plan
    X = np.random.default_rng(9).standard_normal((g.n_cols, 128)).astype(np.float32)
    Xd = _dev(X)
    Y1 = plan.spmm(Xd).cpu().numpy()
    Y2 = plan.spmm(Xd).cpu().numpy()
    assert np.array_equal(Y1.view(np.uint32), Y2.view(np.uint32))
    Y16 = plan.spmm(_dev(X[:, :16])).cpu().numpy()
    _, S = oracle.spmm(g.rowptr, g.colidx, g.vals, X[:, :16], want_scale=True)
    assert_close(Y16, Y1[:, :16], 2 * S, "column slice")


def test_identity_is_exact():
    n, F = 5000, 36
    g = graphgen.identity_csr(n)
    plan = _plan(g)
    X = np.random.default_rng(2).standard_normal((n, F)).astype(np.float32)
    Yg = plan.spmm(_dev(X)).cpu().numpy()
    assert np.array_equal(Yg.view(np.uint32), X.view(np.uint32))
    plan.destroy()


def test_row_permutation_equivariance_bit_exact():
    g = _mixed(21, n=6000)
    p = np.random.default_rng(22).permutation(g.n_rows)
    gp = graphgen.permute_rows(g, p)
    X = _dev(np.random.default_rng(23).standard_normal((g.n_cols, 48)).astype(np.float32))
    pa, pb = _plan(g), _plan(gp)
    Ya = pa.spmm(X).cpu().numpy()
    Yb = pb.spmm(X).cpu().numpy()
    assert np.array_equal(Yb.view(np.uint32), Ya[p].view(np.uint32))
    pa.destroy()
    pb.destroy()


def test_symmetric_relabel_within_tolerance():
    """Relabelling the nodes, (P A P^T)(P X) = P (A X): the relabelled graph
    has other degrees per position, other columns and so another partition
    and summation order, so the two agree within the tolerance (twice the
    bound: each side carries its own rounding)."""
    g = _mixed(24, n=7000, hub_max=5000)
    p = np.random.default_rng(25).permutation(g.n_rows)
    pinv = np.empty_like(p)
    pinv[p] = np.arange(p.size)
    gp = graphgen.permute_rows(g, p)
    gp.colidx[:] = pinv[gp.colidx].astype(np.int32)      # column j of A is column pinv[j] of P A P^T
    X = np.random.default_rng(26).standard_normal((g.n_cols, 64)).astype(np.float32)
    Y, S = oracle.spmm(g.rowptr, g.colidx, g.vals, X, want_scale=True)
    pb = _plan(gp)
    Yb = pb.spmm(_dev(X[p])).cpu().numpy()
    assert_close(Yb, Y[p], 2 * S[p], "P A P^T P X against P (A X)")
    pb.destroy()


def test_linearity_within_tolerance(mixed_plan):
    """A (a X1 + b X2) = a (A X1) + b (A X2): each of the three products is
    within the bound of its own scale, so the two sides differ by at most
    the sum of the bounds."""
    g, plan = mixed_plan
    rng = np.random.default_rng(27)
    F, a, b = 32, np.float32(0.75), np.float32(-1.5)
    X1 = rng.standard_normal((g.n_cols, F)).astype(np.float32)
    X2 = rng.standard_normal((g.n_cols, F)).astype(np.float32)
    Z = a * X1 + b * X2
    _, S1 = oracle.spmm(g.rowptr, g.colidx, g.vals, X1, want_scale=True)
    _, S2 = oracle.spmm(g.rowptr, g.colidx, g.vals, X2, want_scale=True)
    _, SZ = oracle.spmm(g.rowptr, g.colidx, g.vals, Z, want_scale=True)
    lhs = plan.spmm(_dev(Z)).cpu().numpy()
    rhs = (a * plan.spmm(_dev(X1)) + b * plan.spmm(_dev(X2))).cpu().numpy()
    # Bound of |lhs - rhs| in units of the tolerance's 1e-5: the three products'
    # bounds (each with its 1e-7 absolute term), plus the float32 roundings of
    # a * y1, b * y2 and their sum (2^-24 relative each).
    u = 2.0 ** -24 / 1e-5
    S = (SZ + (abs(a) * S1 + abs(b) * S2) * (1 + u) + 2 * u * np.abs(rhs).astype(np.float64)
         + (abs(a) + abs(b)) * 1e-7 / 1e-5)
    assert_close(lhs, rhs, S, "linearity")


def test_non_finite_features_propagate_like_the_oracle(mixed_plan):
    """NaN and infinite X rows reach exactly the Y elements the definition
    says (NaN anywhere -> NaN, +inf with -inf -> NaN, +inf alone -> +inf),
    also through the ReLU epilogue (NaN kept, -inf -> 0)."""
    g, plan = mixed_plan
    rng = np.random.default_rng(17)
    F = 12
    X = rng.standard_normal((g.n_cols, F)).astype(np.float32)
    X[rng.choice(g.n_cols, 40, replace=False)] = np.nan
    X[rng.choice(g.n_cols, 40, replace=False), :6] = np.inf
    X[rng.choice(g.n_cols, 40, replace=False), 3:9] = -np.inf
    Y, S = oracle.spmm(g.rowptr, g.colidx, g.vals, X, want_scale=True)
    assert np.isnan(Y).any() and np.isinf(Y).any()
    Xd = _dev(X)
    assert_close(plan.spmm(Xd).cpu().numpy(), Y, np.nan_to_num(S), "non-finite")
    Yr = np.where(Y < 0, np.float32(0), Y)
    assert_close(plan.spmm(Xd, act="relu").cpu().numpy(), Yr, np.nan_to_num(S), "non-finite relu")


def test_ones_gives_row_sums(mixed_plan):
    g, plan = mixed_plan
    X = np.ones((g.n_cols, 4), np.float32)
    Y, S = oracle.spmm(g.rowptr, g.colidx, g.vals, X, want_scale=True)
    assert_close(plan.spmm(_dev(X)).cpu().numpy(), Y, S, "ones")


def test_plan_reused_across_streams(mixed_plan):
    g, plan = mixed_plan
    X = _dev(np.random.default_rng(4).standard_normal((g.n_cols, 32)).astype(np.float32))
    ref = plan.spmm(X).cpu().numpy()
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        ws = torch.empty(max(1, plan.workspace_bytes(32) // 4), device=DEV)
        Y = plan.spmm(X, ws=ws if plan.workspace_bytes(32) else None, stream=s)
    s.synchronize()
    assert np.array_equal(Y.cpu().numpy(), ref)


def test_concurrent_executes_of_one_plan_on_two_streams(mixed_plan):
    """The plan is read-only during an execute: two executes of one plan
    queued on two streams at once (each with its own Y and workspace, the
    second with another F) both match their single-stream results bit for
    bit."""
    g, plan = mixed_plan
    rng = np.random.default_rng(31)
    Xa = _dev(rng.standard_normal((g.n_cols, 64)).astype(np.float32))
    Xb = _dev(rng.standard_normal((g.n_cols, 96)).astype(np.float32))
    ref_a, ref_b = plan.spmm(Xa).cpu().numpy(), plan.spmm(Xb).cpu().numpy()
    sa, sb = torch.cuda.Stream(), torch.cuda.Stream()
    wsa, wsb = plan.workspace(64), plan.workspace(96)
    Ya = torch.empty((g.n_rows, 64), device=DEV)
    Yb = torch.empty((g.n_rows, 96), device=DEV)
    torch.cuda.synchronize()
    for _ in range(4):
        with torch.cuda.stream(sa):
            plan.spmm(Xa, out=Ya, ws=wsa, stream=sa)
        with torch.cuda.stream(sb):
            plan.spmm(Xb, out=Yb, ws=wsb, stream=sb)
    torch.cuda.synchronize()
    assert np.array_equal(Ya.cpu().numpy().view(np.uint32), ref_a.view(np.uint32))
    assert np.array_equal(Yb.cpu().numpy().view(np.uint32), ref_b.view(np.uint32))


def test_plan_on_a_side_stream_used_at_once():
    """agcn_plan_create returns once the device has written the plan's
    summary; its last kernels may still run on the plan's stream. An export
    right away, an execute on another stream, and the next plans that reuse
    the cached plan memory (on the same stream, then on another) all see the
    finished plan: bit-exact plans, executes equal bit for bit."""
    g = _mixed(77, n=6000, hub_max=4000)
    rng = np.random.default_rng(78)
    X = _dev(rng.standard_normal((g.n_cols, 64)).astype(np.float32))
    Y, S = oracle.spmm(g.rowptr, g.colidx, g.vals, X.cpu().numpy(), want_scale=True)
    rp, ci, va = _dev(g.rowptr), _dev(g.colidx), _dev(g.vals)
    side, other = torch.cuda.Stream(), torch.cuda.Stream()
    torch.cuda.synchronize()
    first = None
    for rep in range(3):
        print(f"[side stream] rep {rep}", flush=True)
        p1 = agcn.Plan(rp, ci, va, n_cols=g.n_cols, stream=side)
        assert_plan_matches_oracle(p1, g)
        with torch.cuda.stream(other):
            Y1 = p1.spmm(X, stream=other)
        other.synchronize()
        Y1 = Y1.cpu().numpy()
        assert_close(Y1, Y, S, "execute on another stream")
        first = Y1 if first is None else first
        assert np.array_equal(Y1.view(np.uint32), first.view(np.uint32))
        p1.destroy()
        p2 = agcn.Plan(rp, ci, va, n_cols=g.n_cols, stream=side)
        with torch.cuda.stream(side):
            Y2 = p2.spmm(X, stream=side)
        side.synchronize()
        assert np.array_equal(Y2.cpu().numpy().view(np.uint32), first.view(np.uint32))
        p2.destroy()
        p3 = agcn.Plan(rp, ci, va, n_cols=g.n_cols, stream=other)
        assert_plan_matches_oracle(p3, g)
        p3.destroy()
    torch.cuda.synchronize()


# ---------------------------------------------------------------------------
# Input validation on the device and host-side errors with a live plan
# ---------------------------------------------------------------------------

def test_invalid_csr_rejected_on_device():
    g = graphgen.random_csr(100, 100, np.full(100, 3), seed=1)
    bad = g.colidx.copy()
    bad[57] = 100
    with pytest.raises(agcn.AgcnError) as ei:
        agcn.Plan(_dev(g.rowptr), _dev(bad), _dev(g.vals), n_cols=100)
    assert ei.value.status == agcn.AGCN_ERR_INVALID_INPUT and "column" in str(ei.value)
    rp = g.rowptr.copy()
    rp[40] = rp[41] + 1
    with pytest.raises(agcn.AgcnError) as ei:
        agcn.Plan(_dev(rp), _dev(g.colidx), _dev(g.vals), n_cols=100)
    assert ei.value.status == agcn.AGCN_ERR_INVALID_INPUT
    # the next plan on this thread reads its own results, not the failed ones'
    ok = _plan(g)
    assert_plan_matches_oracle(ok, g)
    ok.destroy()
    rp = g.rowptr.copy()
    rp[-1] -= 1
    with pytest.raises(agcn.AgcnError) as ei:
        agcn.Plan(_dev(rp), _dev(g.colidx), _dev(g.vals), n_cols=100)
    assert ei.value.status == agcn.AGCN_ERR_INVALID_INPUT


def test_spmm_argument_errors(mixed_plan):
    g, plan = mixed_plan
    X = torch.zeros((g.n_cols, 16), device=DEV)
    Y = torch.zeros((g.n_rows, 16), device=DEV)
    h = plan.handle
    ws = plan.workspace(16)
    wsp = ws.data_ptr() if ws is not None else None
    for args, status in [((h, 0, X.data_ptr(), 16, Y.data_ptr(), 16, wsp), 1),
                         ((h, 16, X.data_ptr(), 8, Y.data_ptr(), 16, wsp), 1),
                         ((h, 16, X.data_ptr(), 16, X.data_ptr(), 16, wsp), 1),
                         ((h, 16, X.data_ptr(), 16, None, 16, wsp), 1)]:
        with pytest.raises(agcn.AgcnError) as ei:
            agcn.agcn_spmm(*args)
        assert ei.value.status == status
    if plan.stats.n_hub_chunks:
        with pytest.raises(agcn.AgcnError):
            agcn.agcn_spmm(h, 16, X.data_ptr(), 16, Y.data_ptr(), 16, None)


# ---------------------------------------------------------------------------
# Full-size workloads (default parameters, the launch configuration the
# benchmark times): plan bit-exact, and every element of Y against the oracle
# at every feature width of the workload.
# ---------------------------------------------------------------------------

@pytest.mark.slow
@pytest.mark.parametrize("name", list(graphgen.CONFIGS))
def test_workload_parity(name):
    g = _workload(name)
    plan = _plan(g)
    assert_plan_matches_oracle(plan, g)
    for F in graphgen.CONFIGS[name]["F"]:
        X = graphgen.workload_features(name, g, F)
        Yg = plan.spmm(_dev(X)).cpu().numpy()
        n = assert_all_rows_close(g, X, Yg, f"{name} F={F}")
        print(f"[parity] {name} F={F} ok (all {n} rows x {F} columns checked)", flush=True)
    plan.destroy()


def test_plan_memory_reused_across_plans():
    """A destroyed plan's device block is reused by the next plan; stale
    contents must not leak into the new plan."""
    g1 = _mixed(31, n=8000)
    g2 = _mixed(32, n=7900)
    p1 = _plan(g1)
    assert_plan_matches_oracle(p1, g1)
    p1.destroy()
    p2 = _plan(g2)
    assert_plan_matches_oracle(p2, g2)
    _spmm_check(p2, g2, 64)
    p2.destroy()
    agcn.agcn_release_cached_memory()
    p3 = _plan(g1)
    assert_plan_matches_oracle(p3, g1)
    p3.destroy()


@pytest.mark.parametrize("plan_stream", ["exec", "other"])
def test_destroy_while_executing_then_reuse_on_another_stream(plan_stream):
    """agcn_plan_destroy does not block; a plan that reuses the destroyed
    plan's cached memory on another stream must wait for the work still
    queued with the old plan (it would otherwise overwrite the sorted CSR the
    running execute reads). The executes run on the plan's own stream (marked
    at release) or on another stream (marked by each call)."""
    g1 = _mixed(81, n=40000, hub_max=8000)
    g2 = _mixed(82, n=39000, hub_max=8000)
    s1, s2, s0 = torch.cuda.Stream(), torch.cuda.Stream(), torch.cuda.Stream()
    agcn.agcn_release_cached_memory()
    p1 = _plan(g1, stream=s1 if plan_stream == "exec" else s0)
    F = 512
    X1 = np.random.default_rng(83).standard_normal((g1.n_cols, F)).astype(np.float32)
    X1d = _dev(X1)
    ws1 = p1.workspace(F)
    torch.cuda.synchronize()
    with torch.cuda.stream(s1):
        Y1 = torch.empty((g1.n_rows, F), device=DEV)
        for _ in range(3):      # several launches keep s1 busy for a while
            p1.spmm(X1d, out=Y1, ws=ws1, stream=s1)
    p1.destroy()
    p2 = _plan(g2, stream=s2)   # reuses p1's block: s2 waits on s1's last execute
    assert_plan_matches_oracle(p2, g2)
    torch.cuda.synchronize()
    Y, S = oracle.spmm(g1.rowptr, g1.colidx, g1.vals, X1, want_scale=True)
    assert_close(Y1.cpu().numpy(), Y, S, "execute of the destroyed plan")
    _spmm_check(p2, g2, 64)
    p2.destroy()


def test_long_hub_rows_column_ordered_launch():
    """Hub rows of tens of thousands of nnz (many chunks each) take the
    column-ordered launch path; Y must still match the oracle everywhere."""
    rng = np.random.default_rng(41)
    n = 60000
    deg = rng.integers(1, 9, size=n)
    hubs = rng.choice(n, size=24, replace=False)
    deg[hubs] = rng.integers(20000, 50001, size=hubs.size)
    g = graphgen.random_csr(n, n, deg, seed=42)
    plan = _plan(g)
    st = plan.stats
    assert st.n_hub_chunks >= 8 * st.n_hub_rows      # the sorted-order path is taken
    assert_plan_matches_oracle(plan, g)
    for F in (16, 64, 100):
        Yg = _spmm_check(plan, g, F, seed=F)
    X = _dev(np.random.default_rng(1).standard_normal((n, 64)).astype(np.float32))
    assert np.array_equal(plan.spmm(X).cpu().numpy(), plan.spmm(X).cpu().numpy())
    plan.destroy()


@pytest.mark.slow
@pytest.mark.parametrize("flags", [0, agcn.AGCN_PLAN_WARP_LEVEL])
def test_nnz_just_below_the_int32_limit(flags):
    """The largest matrix the int32 format holds: nnz = 2^31 - 3 over about
    1.9 M rows of mixed degree (empty, small, the deg_bound edges, hubs of
    several chunks). Entry counts checked against the closed forms, every
    element of Y against the oracle."""
    pattern = np.array([0, 1, 7, 64, 511, 512, 513, 2000, 4000], np.int64)
    n_cols = 1 << 20
    target = (1 << 31) - 3
    reps = target // int(pattern.sum())
    deg = np.tile(pattern, reps)
    deg = np.append(deg, target - int(deg.sum()))          # last row takes the remainder
    n = deg.size
    rowptr = np.zeros(n + 1, np.int64)
    np.cumsum(deg, out=rowptr[1:])
    assert rowptr[-1] == target
    rowptr = rowptr.astype(np.int32)
    rng = np.random.default_rng(97)
    colidx = rng.integers(0, n_cols, size=target, dtype=np.int32)
    vals = rng.random(target, dtype=np.float32)
    print(f"[max] n={n} nnz={target} flags={flags}", flush=True)
    d_rp, d_ci, d_v = _dev(rowptr), _dev(colidx), _dev(vals)
    plan = agcn.Plan(d_rp, d_ci, d_v, n_cols=n_cols, flags=flags)
    s = plan.stats
    assert s.nnz == target and s.max_deg == int(deg.max())
    Z = s.max_wave_nzs
    if flags:
        assert s.n_entries == int(np.maximum(1, -(-deg // Z)).sum())
    else:
        assert s.n_hub_rows == int((deg > s.deg_bound).sum())
        assert s.n_hub_chunks == int(-(-deg[deg > s.deg_bound] // s.hub_chunk_nnz).sum())
    del d_ci, d_v
    F = 8
    X = rng.standard_normal((n_cols, F)).astype(np.float32)
    Yg = plan.spmm(_dev(X)).cpu().numpy()
    g = graphgen.Graph("max", n, n_cols, rowptr, colidx, vals)
    checked = assert_all_rows_close(g, X, Yg, f"nnz=2^31-3 flags={flags}", block=65536)
    print(f"[max] ok (all {checked} rows checked)", flush=True)
    plan.destroy()
    agcn.agcn_release_cached_memory()
