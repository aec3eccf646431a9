"""The hub rows' column windows.

When the hub rows (degree above deg_bound) average at least 16 nonzeros per
window of 512 columns, the plan keeps, for every hub row and window, where the
row's nonzeros of that window start; executes at F >= 64 on the float4 path
then aggregate the hub rows window by window from X staged in LDS, one partial
row per (hub row, window group), added in window order. Y must match the
oracle's A X (Sec. II-B) within 1e-5 * S + 1e-7 on every element: at one and
several 64-column slices and a partial last slice, with the ReLU epilogue,
over several workgroup row batches, with hub rows only, and with hub rows
whose columns do not ascend (their pairs outside the current window are added
from X by the reduction). F < 64, a scalar-path F and plans built with
AGCN_HUB_WINDOWS=0 take the hub chunks, which must agree; agcn_spmm_noalloc
uses the windows when their partials fit its fixed workspace and the hub
chunks otherwise.
"""
import contextlib
import os

import numpy as np
import pytest

import graphgen
import oracle
from gpu_helpers import DEV, _dev, _plan, assert_all_rows_close, assert_close

torch = pytest.importorskip("torch")
import paper_2308_11825_amd as agcn  # noqa: E402

pytestmark = pytest.mark.gpu

WIN = 512


@contextlib.contextmanager
def _no_windows():
    old = os.environ.get("AGCN_HUB_WINDOWS")
    os.environ["AGCN_HUB_WINDOWS"] = "0"
    try:
        yield
    finally:
        if old is None:
            os.environ.pop("AGCN_HUB_WINDOWS", None)
        else:
            os.environ["AGCN_HUB_WINDOWS"] = old


def _hub_graph(seed, n, n_cols, n_hub, lo, hi, sort_cols=True):
    rng = np.random.default_rng(seed)
    deg = rng.integers(1, 9, size=n)
    hubs = rng.choice(n, size=n_hub, replace=False)
    deg[hubs] = rng.integers(lo, hi + 1, size=n_hub)
    return graphgen.random_csr(n, n_cols, deg, seed=seed + 1, sort_cols=sort_cols)


def _stray_flags(plan, F):
    """The stray flags k_hub_win leaves after the window partials in the
    workspace of the last execute at F: one int32 per (hub row, window group),
    n_grp = ceil(n_win / G) with G chosen for about 512 workgroups over
    ceil(F / 64) slices and ceil(n_hub / 1024) row batches."""
    st = plan.stats
    n_hub, n_win = st.n_hub_rows, st.hub_windows
    per = max(1, -(-F // 64) * -(-n_hub // 1024))
    G = max(1, -(-n_win // max(1, -(-512 // per))))
    n_grp = -(-n_win // G)
    ws = plan.workspace(F)
    assert ws.numel() * 4 >= n_hub * n_grp * (4 * F + 4)
    off = n_hub * n_grp * F
    return ws[off:off + n_hub * n_grp].view(torch.int32).cpu().numpy()


def _X(g, F, seed):
    return np.random.default_rng(seed).standard_normal((g.n_cols, F)).astype(np.float32)


def _windowed(g):
    p = _plan(g)
    assert p.stats.hub_windows == -(-g.n_cols // WIN), p.stats.as_dict()
    return p


@pytest.fixture(scope="module")
def hub_case():
    g = _hub_graph(1100, n=20000, n_cols=40000, n_hub=200, lo=1500, hi=4000)
    p = _windowed(g)
    with _no_windows():
        pc = _plan(g)
    assert pc.stats.hub_windows == 0
    yield g, p, pc
    p.destroy()
    pc.destroy()


@pytest.mark.parametrize("F", [64, 96, 128, 256, 512])
def test_windows_match_the_oracle(hub_case, F):
    g, p, pc = hub_case
    X = _X(g, F, F)
    Xd = _dev(X)
    Y = p.spmm(Xd).cpu().numpy()
    assert_all_rows_close(g, X, Y, f"windows F={F}")
    assert np.array_equal(Y.view(np.uint32), p.spmm(Xd).cpu().numpy().view(np.uint32))
    # sorted rows: every pair lies in the window the table gives it (a table
    # off by one anywhere would flag a stray; Y would still be right)
    flags = _stray_flags(p, F)
    assert flags.size > 0 and np.all(flags == 0), int(np.count_nonzero(flags))
    Yc = pc.spmm(Xd).cpu().numpy()
    _, S = oracle.spmm(g.rowptr, g.colidx, g.vals, X, n_cols=g.n_cols, want_scale=True)
    assert_close(Y, Yc, 2 * S, f"windows against hub chunks F={F}")


def test_windows_relu_and_strided_y(hub_case):
    g, p, _ = hub_case
    F = 64
    X = _X(g, F, 5)
    Y, S = oracle.spmm(g.rowptr, g.colidx, g.vals, X, n_cols=g.n_cols, want_scale=True)
    out = torch.full((g.n_rows, F + 12), 7.0, device=DEV)
    p.spmm(_dev(X), out=out[:, :F], act="relu")
    Yg = out.cpu().numpy()
    assert_close(Yg[:, :F], np.where(Y < 0, 0.0, Y), S, "relu")
    assert np.all(Yg[:, F:] == 7.0)


@pytest.mark.parametrize("F", [32, 66])
def test_hub_chunks_below_64_columns_and_on_the_scalar_path(hub_case, F):
    g, p, _ = hub_case
    X = _X(g, F, 10 + F)
    assert_all_rows_close(g, X, p.spmm(_dev(X)).cpu().numpy(), f"chunks F={F}")


def test_windows_with_columns_out_of_order():
    # Unsorted rows: the windows still partition each row; a pair outside its
    # window is left to the reduction.
    g = _hub_graph(1200, n=8000, n_cols=30000, n_hub=120, lo=1500, hi=3500, sort_cols=False)
    ci = g.colidx.copy()
    d = g.degrees
    hub_rows = np.nonzero(d > 512)[0]
    for r in hub_rows[:10]:               # some rows sorted, some descending
        s, e = g.rowptr[r], g.rowptr[r + 1]
        ci[s:e] = np.sort(ci[s:e])[::-1] if r % 2 else np.sort(ci[s:e])
    g = graphgen.Graph("unsorted", g.n_rows, g.n_cols, g.rowptr, ci, g.vals)
    p = _windowed(g)
    for F in (64, 128):
        X = _X(g, F, 20 + F)
        assert_all_rows_close(g, X, p.spmm(_dev(X)).cpu().numpy(), f"unsorted F={F}")
        flags = _stray_flags(p, F)
        assert np.all((flags == 0) | (flags == 1)) and np.count_nonzero(flags) > 0
    p.destroy()


def test_windows_over_two_row_batches():
    # 1500 hub rows: two workgroup row batches of 1024.
    g = _hub_graph(1300, n=30000, n_cols=20000, n_hub=1500, lo=1600, hi=2400)
    p = _windowed(g)
    assert p.stats.n_hub_rows == 1500
    for F in (64, 192):
        X = _X(g, F, 30 + F)
        assert_all_rows_close(g, X, p.spmm(_dev(X)).cpu().numpy(), f"two batches F={F}")
    p.destroy()


def test_windows_with_hub_rows_only():
    rng = np.random.default_rng(1400)
    n, n_cols = 300, 8000
    deg = rng.integers(1000, 3001, size=n)
    g = graphgen.random_csr(n, n_cols, deg, seed=1401)
    p = _windowed(g)
    assert p.stats.n_hub_rows == n
    F = 64
    X = _X(g, F, 41)
    Xd = _dev(X)
    assert_all_rows_close(g, X, p.spmm(Xd).cpu().numpy(), "hub rows only")
    # the timed call's marks still frame the (empty) aggregation
    Y = torch.empty((n, F), device=DEV)
    ws = p.workspace(F)
    b, m = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    for e in (b, m):
        e.record()  # creates the underlying event, which the library records again
    agcn.agcn_spmm_timed(p.handle, F, Xd.data_ptr(), F, Y.data_ptr(), F, ws.data_ptr(),
                         torch.cuda.current_stream().cuda_stream, b.cuda_event, m.cuda_event, None)
    torch.cuda.synchronize()
    assert b.elapsed_time(m) >= 0.0
    assert_all_rows_close(g, X, Y.cpu().numpy(), "hub rows only, timed")
    p.destroy()


def _noalloc(plan, Xd, F):
    Y = torch.full((plan.n_rows, F), float("nan"), device=DEV)
    rc = agcn.load_library().agcn_spmm_noalloc(plan.handle, F, Xd.data_ptr(), F, Y.data_ptr(), F,
                                                torch.cuda.current_stream().cuda_stream,
                                                agcn.AGCN_EPILOGUE_NONE)
    assert rc == agcn.AGCN_OK, agcn.agcn_last_error()
    return Y.cpu().numpy()


def test_noalloc_takes_the_windows_only_when_they_fit():
    # 1000 hub rows over 137 windows: at F = 64 the window partials (about
    # 36 MB) fit the fixed 64 MiB workspace, at F = 256 (about 71 MB) they do not.
    g = _hub_graph(1500, n=20000, n_cols=70000, n_hub=1000, lo=3000, hi=5000)
    p = _windowed(g)
    with _no_windows():
        pc = _plan(g)
    limit = agcn.AGCN_NOALLOC_MAX_WORKSPACE
    assert p.workspace_bytes(64) <= limit < p.workspace_bytes(256)
    assert pc.workspace_bytes(256) <= limit
    for F, chunks in ((64, False), (256, True)):
        X = _X(g, F, 50 + F)
        Xd = _dev(X)
        Yn = _noalloc(p, Xd, F)
        ref = (pc if chunks else p).spmm(Xd).cpu().numpy()
        assert np.array_equal(Yn.view(np.uint32), ref.view(np.uint32)), F
        assert_all_rows_close(g, X, Yn, f"noalloc F={F}")
    p.destroy()
    pc.destroy()


def test_window_plan_destroyed_while_its_execute_runs_on_another_stream():
    g = _hub_graph(1600, n=20000, n_cols=40000, n_hub=300, lo=2000, hi=4000)
    X = _X(g, 128, 61)
    Xd = _dev(X)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    p = _windowed(g)
    with torch.cuda.stream(side):
        Y = torch.empty((g.n_rows, 128), device=DEV)
        p.spmm(Xd, out=Y, stream=side)
    p.destroy()                       # the table is freed after the side stream's execute
    torch.cuda.synchronize()
    assert_all_rows_close(g, X, Y.cpu().numpy(), "execute on another stream")


def test_windows_with_empty_ranges():
    # Half the hub rows keep their columns in the first 8 windows, so most of
    # their (row, window) ranges are empty: a group's preloaded batch is then
    # empty and it moves on to its next row's.
    rng = np.random.default_rng(1700)
    n, n_cols = 12000, 40000
    deg = rng.integers(1, 9, size=n)
    hubs = rng.choice(n, size=200, replace=False)
    deg[hubs] = rng.integers(2500, 3500, size=200)
    g = graphgen.random_csr(n, n_cols, deg, seed=1701)
    ci = g.colidx.copy()
    for r in hubs[:100]:
        s, e = g.rowptr[r], g.rowptr[r + 1]
        ci[s:e] = np.sort(rng.choice(8 * WIN, size=e - s, replace=False))
    g = graphgen.Graph("clustered", g.n_rows, g.n_cols, g.rowptr, ci, g.vals)
    p = _windowed(g)
    for F in (64, 128):
        X = _X(g, F, 70 + F)
        assert_all_rows_close(g, X, p.spmm(_dev(X)).cpu().numpy(), f"empty ranges F={F}")
        assert np.all(_stray_flags(p, F) == 0)
    p.destroy()


@pytest.mark.parametrize("cap,early,tiny", [(None, None, None), ("-1", None, "0"), (None, "0", "0")])
def test_windows_after_every_degree_sort(cap, early, tiny):
    # The table lies over the plan's working buffers whichever sort built the
    # plan: the single-workgroup plan of a small graph, the short sort with
    # the column check early or in the relayout, the multi-pass sort.
    rng = np.random.default_rng(1800)
    n, n_cols = 2000, 4096
    deg = rng.integers(1, 9, size=n)
    hubs = rng.choice(n, size=64, replace=False)
    deg[hubs] = rng.integers(1200, 1700, size=64)
    g = graphgen.random_csr(n, n_cols, deg, seed=1801)
    assert g.nnz <= 1 << 17            # small enough for the single-workgroup plan
    old = {k: os.environ.get(k) for k in ("AGCN_TEST_TAIL_CAP", "AGCN_TEST_EARLY_CHECK_NNZ",
                                           "AGCN_TEST_TINY")}
    try:
        for k, v in zip(old, (cap, early, tiny)):
            if v is None:
                os.environ.pop(k, None)
            else:
                os.environ[k] = v
        p = _windowed(g)
    finally:
        for k, v in old.items():
            if v is None:
                os.environ.pop(k, None)
            else:
                os.environ[k] = v
    X = _X(g, 64, 81)
    assert_all_rows_close(g, X, p.spmm(_dev(X)).cpu().numpy(), f"windows cap={cap} early={early}")
    assert np.all(_stray_flags(p, 64) == 0)
    p.destroy()


def test_windows_captured_in_a_hip_graph_replay_like_eager(hub_case):
    """The window execute (k_spmm over the other rows, k_hub_win,
    k_hub_win_reduce) launches kernels only: captured into a HIP graph, every
    replay with new X (copied in eagerly, the device synchronised between
    replays) equals the eager call bit for bit."""
    g, p, _ = hub_case
    F = 64
    X = torch.zeros((g.n_cols, F), device=DEV)
    Y = torch.empty((g.n_rows, F), device=DEV)
    ws = torch.empty(p.workspace_bytes(F) // 4 + 1, device=DEV)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        with torch.cuda.graph(graph, stream=s):
            p.spmm(X, out=Y, ws=ws, stream=s)
    torch.cuda.synchronize()
    rng = np.random.default_rng(93)
    for r in range(3):
        Xr = rng.standard_normal((g.n_cols, F)).astype(np.float32)
        X.copy_(_dev(Xr))
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        Ye = p.spmm(_dev(Xr))
        torch.cuda.synchronize()
        assert torch.equal(Y, Ye), f"replay {r}"
        if r == 0:
            assert_all_rows_close(g, Xr, Y.cpu().numpy(), "graph replay")
    del graph


def test_gcn_layer_over_the_windows(hub_case):
    # agcn_gcn_layer passes its SpMM the layer workspace, sized with the
    # window partials: fout = 64 takes the windows.
    from test_gpu_layer import _check_layer
    g, p, _ = hub_case
    X = np.random.default_rng(95).standard_normal((g.n_cols, 32)).astype(np.float32)
    W = graphgen.weights(32, 64, seed=96)
    _check_layer(p, g, X, W, "relu")
    H = agcn.linear(_dev(X), _dev(W))
    Y = p.spmm(H, act="relu")
    assert torch.equal(Y, p.gcn_layer(_dev(X), _dev(W), act="relu"))
