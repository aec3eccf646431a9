"""GPU parity of the GCNConv layer (Sec. II-A) through the C ABI:
agcn_linear (H = X W on the matrix cores), agcn_spmm_ex (the aggregation
with the ReLU epilogue) and agcn_gcn_layer (both in one call), against the
CPU oracle.

Tolerances, from the rounding depth of the device arithmetic (u = 2^-24):
* linear: |H - H_oracle| <= (fin + 2) u |X||W| + 1e-30 (fp32 products and a
  chain of at most fin additions per element, the oracle rounded once);
* aggregation with ReLU: the SpMM bound 1e-5 S + 1e-7 (ReLU is 1-Lipschitz);
* layer: (1e-5 + (fin + 3) u) S2 + 1e-7, S2 = sum_e |a_e| sum_k |x||w|: the
  linear step's error carried through A, plus the SpMM bound over the
  computed H, plus the oracle's single rounding.
"""
import numpy as np
import pytest

import graphgen
import oracle

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

import paper_2308_11825_amd as agcn  # noqa: E402

from gpu_helpers import DEV, _dev, _mixed, _plan, _sample_rows, _workload, assert_close  # noqa: E402

U = 2.0 ** -24


def _check_linear(X, W, H, what=""):
    fin = W.shape[0]
    Hr = oracle.linear(X, W)
    S = np.abs(X.astype(np.float64)) @ np.abs(W.astype(np.float64))
    err = np.abs(H.astype(np.float64) - Hr.astype(np.float64))
    tol = (fin + 2) * U * S + 1e-30
    bad = ~(err <= tol)                    # NaN counts as out of tolerance
    assert not bad.any(), (f"{what}: {int(bad.sum())} out of tolerance; first "
                           f"{tuple(np.argwhere(bad)[0])}")


@pytest.mark.parametrize("n,fin,fout", [(1000, 128, 128), (777, 33, 17), (5000, 64, 16),
                                        (130, 1, 1), (300, 256, 300), (2000, 100, 40),
                                        (129, 32, 32), (64, 0, 8), (4097, 12, 200),
                                        (20011, 128, 256), (5003, 64, 300), (3000, 128, 132)])
def test_linear_matches_oracle(n, fin, fout):
    rng = np.random.default_rng(n + fin + fout)
    X = rng.standard_normal((n, fin)).astype(np.float32)
    W = graphgen.weights(fin, fout, seed=fin * 1000 + fout)
    print(f"[linear] n={n} fin={fin} fout={fout}", flush=True)
    H = agcn.linear(_dev(X), _dev(W)).cpu().numpy()
    _check_linear(X, W, H, f"n={n} fin={fin} fout={fout}")


def _resident_waves():
    # Waves the W-resident kernel runs at the widths below: one workgroup of 4
    # waves per compute unit.
    return torch.cuda.get_device_properties(0).multi_processor_count * 4


_LAST_ROUND = {"one": lambda w: 1, "eighth": lambda w: w // 8, "eighth+1": lambda w: w // 8 + 1,
               "quarter+1": lambda w: w // 4 + 1, "half+1": lambda w: w // 2 + 1,
               "all-3": lambda w: w - 3}


@pytest.mark.parametrize("last,fin,fout,short", [("one", 128, 128, 3), ("eighth", 128, 128, 5),
                                                 ("eighth+1", 128, 128, 0), ("eighth", 100, 60, 7),
                                                 ("quarter+1", 128, 128, 1), ("quarter+1", 32, 32, 0),
                                                 ("half+1", 128, 128, 2), ("all-3", 64, 128, 9)])
def test_linear_last_round_split_by_columns(last, fin, fout, short):
    """16-row tiles past the last whole round of waves are cut by output
    columns (1, 2, 4 or 8 ranges, depending on how many are left). Every
    output row stays within the oracle's bound, and is bit-identical to the
    same row computed inside a whole round: the rows are rotated so that the
    last round's rows come first and the outputs compared row by row."""
    waves = _resident_waves()
    rem = _LAST_ROUND[last](waves)
    tiles = 2 * waves + rem
    n = 16 * tiles - short
    rng = np.random.default_rng(tiles + fin + fout + short)
    X = rng.standard_normal((n, fin)).astype(np.float32)
    W = graphgen.weights(fin, fout, seed=fin * 7 + fout)
    print(f"[linear tail] n={n} tiles={tiles} rem={rem} fin={fin} fout={fout}", flush=True)
    H = agcn.linear(_dev(X), _dev(W)).cpu().numpy()
    _check_linear(X, W, H, f"n={n} fin={fin} fout={fout}")
    cut = 16 * 2 * waves
    Xr = np.ascontiguousarray(np.concatenate([X[cut:], X[:cut]]))
    Hr = agcn.linear(_dev(Xr), _dev(W)).cpu().numpy()
    assert np.array_equal(np.concatenate([H[cut:], H[:cut]]), Hr)


def test_linear_strided_unaligned_and_deterministic():
    rng = np.random.default_rng(3)
    n, fin, fout = 3001, 64, 48
    X = rng.standard_normal((n, fin)).astype(np.float32)
    W = graphgen.weights(fin, fout, seed=4)
    Xd, Wd = _dev(X), _dev(W)
    H1 = agcn.linear(Xd, Wd).cpu().numpy()
    H2 = agcn.linear(Xd, Wd).cpu().numpy()
    assert np.array_equal(H1.view(np.uint32), H2.view(np.uint32))
    _check_linear(X, W, H1, "aligned")
    # X one float past an aligned address, W with a padded row stride, H strided: 32-bit path
    buf = torch.empty(n * fin + 1, device=DEV)
    Xu = buf[1:].view(n, fin)
    Xu.copy_(Xd)
    Wp = torch.zeros((fin, fout + 3), device=DEV)
    Wp[:, :fout] = Wd
    Hs = torch.full((n, fout + 5), 9.0, device=DEV)
    agcn.linear(Xu, Wp[:, :fout], out=Hs[:, :fout])
    _check_linear(X, W, Hs[:, :fout].cpu().numpy(), "unaligned/strided")
    assert torch.all(Hs[:, fout:] == 9.0)


@pytest.mark.parametrize("offset,pad", [(1, 4), (0, 3), (1, 3)])
def test_linear_output_rows_not_16_byte_aligned(offset, pad):
    """fin, fout <= 128 with X and W aligned, but H's rows not all 16-byte
    aligned (H one float past an aligned address, or a row stride that is not
    a multiple of 4): the resident-W kernel writes 16-byte pieces, so the
    tiled kernel runs instead. Within the bound; padding untouched."""
    rng = np.random.default_rng(21 + offset + pad)
    n, fin, fout = 3001, 128, 128
    X = rng.standard_normal((n, fin)).astype(np.float32)
    W = graphgen.weights(fin, fout, seed=22)
    ld = fout + pad
    buf = torch.full((n * ld + offset,), 5.0, device=DEV)
    Hs = buf[offset:].view(n, ld)
    agcn.linear(_dev(X), _dev(W), out=Hs[:, :fout])
    _check_linear(X, W, Hs[:, :fout].cpu().numpy(), f"offset={offset} ldh={ld}")
    assert torch.all(Hs[:, fout:] == 5.0) and torch.all(buf[:offset] == 5.0)


def test_linear_wide_output_in_column_launches():
    """fin <= 128 and fout > 128 run as one W-resident launch per 128 output
    columns: within the bound, padding columns of a strided H untouched, and
    each column bit-identical to the same column computed alone."""
    rng = np.random.default_rng(41)
    n, fin, fout = 3001, 96, 260
    X = rng.standard_normal((n, fin)).astype(np.float32)
    W = graphgen.weights(fin, fout, seed=42)
    Hp = torch.full((n, fout + 12), 3.0, device=DEV)
    agcn.linear(_dev(X), _dev(W), out=Hp[:, :fout])
    H = Hp[:, :fout].cpu().numpy()
    _check_linear(X, W, H, "wide output")
    assert torch.all(Hp[:, fout:] == 3.0)
    Hc = agcn.linear(_dev(X), _dev(np.ascontiguousarray(W[:, 128:256]))).cpu().numpy()
    assert np.array_equal(H[:, 128:256].view(np.uint32), Hc.view(np.uint32))


def test_linear_identity_is_exact():
    X = np.random.default_rng(5).standard_normal((1000, 96)).astype(np.float32)
    H = agcn.linear(_dev(X), _dev(np.eye(96, dtype=np.float32))).cpu().numpy()
    assert np.array_equal(H.view(np.uint32), X.view(np.uint32))


@pytest.fixture(scope="module")
def layer_graph():
    return _mixed(61, n=9000, hub_max=5000)


@pytest.mark.parametrize("flags", [0, agcn.AGCN_PLAN_WARP_LEVEL, agcn.AGCN_PLAN_COLUMN_LOOP])
@pytest.mark.parametrize("F", [1, 16, 17, 64, 128])
def test_spmm_relu_epilogue(layer_graph, flags, F):
    g = layer_graph
    plan = _plan(g, flags=flags)
    X = np.random.default_rng(F).standard_normal((g.n_cols, F)).astype(np.float32)
    Y, S = oracle.spmm(g.rowptr, g.colidx, g.vals, X, want_scale=True)
    Yg = plan.spmm(_dev(X), act="relu").cpu().numpy()
    assert np.all(Yg >= 0)
    assert_close(Yg, np.maximum(Y, 0.0), S, f"relu flags={flags} F={F}")
    # the epilogue only touches negative values
    Yn = plan.spmm(_dev(X)).cpu().numpy()
    assert np.array_equal(Yg, np.where(Yn < 0, np.float32(0), Yn))
    plan.destroy()


def _check_layer(plan, g, X, W, act, rows=None, Yg=None):
    fin = W.shape[0]
    if Yg is None:
        Yg = plan.gcn_layer(_dev(X), _dev(W), act=act).cpu().numpy()
    Yr, S2 = oracle.gcn_layer(g.rowptr, g.colidx, g.vals, X, W, act=act, rows=rows,
                              n_cols=g.n_cols, want_scale=True)
    Yc = Yg if rows is None else Yg[rows]
    err = np.abs(Yc.astype(np.float64) - Yr.astype(np.float64))
    tol = (1e-5 + (fin + 3) * U) * S2 + 1e-7
    bad = ~(err <= tol)                    # NaN counts as out of tolerance
    assert not bad.any(), (f"layer act={act}: {int(bad.sum())} out of tolerance; first "
                           f"{tuple(np.argwhere(bad)[0])}")
    return Yg


@pytest.mark.parametrize("flags", [0, agcn.AGCN_PLAN_WARP_LEVEL, agcn.AGCN_PLAN_COLUMN_LOOP])
@pytest.mark.parametrize("fin,fout", [(32, 16), (64, 64), (48, 17), (128, 128)])
def test_gcn_layer_matches_oracle(layer_graph, flags, fin, fout):
    g = layer_graph
    plan = _plan(g, flags=flags)
    X = np.random.default_rng(fin).standard_normal((g.n_cols, fin)).astype(np.float32)
    W = graphgen.weights(fin, fout, seed=fout)
    print(f"[layer] flags={flags} fin={fin} fout={fout}", flush=True)
    Y1 = _check_layer(plan, g, X, W, "relu")
    Y2 = plan.gcn_layer(_dev(X), _dev(W), act="relu").cpu().numpy()
    assert np.array_equal(Y1.view(np.uint32), Y2.view(np.uint32))
    _check_layer(plan, g, X, W, "none")
    plan.destroy()


def test_gcn_layer_equals_linear_then_spmm(layer_graph):
    """The fused call runs the same kernels as linear followed by spmm_ex."""
    g = layer_graph
    plan = _plan(g)
    X = _dev(np.random.default_rng(1).standard_normal((g.n_cols, 64)).astype(np.float32))
    W = _dev(graphgen.weights(64, 32, seed=2))
    Y1 = plan.gcn_layer(X, W, act="relu")
    Y2 = plan.spmm(agcn.linear(X, W), act="relu")
    assert torch.equal(Y1, Y2)
    plan.destroy()


def test_gcn_layer_argument_errors(layer_graph):
    g = layer_graph
    plan = _plan(g)
    X = torch.zeros((g.n_cols, 8), device=DEV)
    W = torch.zeros((8, 16), device=DEV)
    Y = torch.zeros((g.n_rows, 16), device=DEV)
    nb = agcn.agcn_gcn_workspace_size(plan.handle, 16)
    assert nb >= g.n_cols * 16 * 4
    ws = torch.empty(nb // 4 + 8, device=DEV)
    h = plan.handle
    cases = [((h, 8, 16, X.data_ptr(), 8, W.data_ptr(), 16, Y.data_ptr(), 16, None, None, 1), 1),
             ((h, 8, 16, X.data_ptr(), 8, W.data_ptr(), 16, Y.data_ptr(), 16, ws.data_ptr(), None, 2), 1),
             ((h, 8, 16, X.data_ptr(), 8, W.data_ptr(), 16, Y.data_ptr(), 16, ws.data_ptr() + 4, None, 1), 1),
             ((h, 8, 16, X.data_ptr(), 8, W.data_ptr(), 16, X.data_ptr(), 16, ws.data_ptr(), None, 1), 1),
             ((h, 8, 0, X.data_ptr(), 8, W.data_ptr(), 16, Y.data_ptr(), 16, ws.data_ptr(), None, 1), 1)]
    for args, status in cases:
        with pytest.raises(agcn.AgcnError) as ei:
            agcn.agcn_gcn_layer(*args)
        assert ei.value.status == status
    with pytest.raises(agcn.AgcnError):
        agcn.agcn_spmm_ex(h, 16, W.data_ptr(), 16, Y.data_ptr(), 16, None, None, 5)
    plan.destroy()


@pytest.mark.slow
def test_gcn_layer_workload_parity():
    """The layer at the benchmark's size: sweep_powerlaw graph, fin = fout = 128."""
    name = "sweep_powerlaw"
    g = _workload(name)
    plan = _plan(g)
    X = graphgen.workload_features(name, g, 128)
    W = graphgen.weights(128, 128, seed=7)
    rows = _sample_rows(g, plan, k=1500)
    _check_layer(plan, g, X, W, "relu", rows=rows)
    print(f"[layer] {name} fin=fout=128 ok ({rows.size} rows checked)", flush=True)
    plan.destroy()


def test_layer_captured_in_a_hip_graph_replays_like_eager():
    """A GCNConv layer (linear, aggregation with ReLU, hub-row reduction)
    captured into a HIP graph: every replay, with new X copied in eagerly
    and the device synchronised between replays, equals the eager call bit
    for bit. The library launches kernels only (no memsets, no allocations)."""
    g = _mixed(91, n=8000, hub_max=4000)
    plan = _plan(g)
    assert plan.stats.n_hub_rows > 0
    fin, fout = 32, 48
    W = _dev(graphgen.weights(fin, fout, seed=5))
    X = torch.zeros((g.n_cols, fin), device=DEV)
    Y = torch.empty((g.n_rows, fout), device=DEV)
    nb = agcn.agcn_gcn_workspace_size(plan.handle, fout)
    ws = torch.empty(nb // 4 + 1, device=DEV)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        with torch.cuda.graph(graph, stream=s):
            plan.gcn_layer(X, W, act="relu", out=Y, ws=ws, stream=s)
    torch.cuda.synchronize()
    rng = np.random.default_rng(92)
    for r in range(4):
        Xr = rng.standard_normal((g.n_cols, fin)).astype(np.float32)
        X.copy_(_dev(Xr))
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        Ye = plan.gcn_layer(_dev(Xr), W, act="relu")
        torch.cuda.synchronize()
        assert torch.equal(Y, Ye), f"replay {r}"
        if r == 0:
            _check_layer(plan, g, Xr, W.cpu().numpy(), "relu", Yg=Y.cpu().numpy())
    del graph
    plan.destroy()


def test_linear_padded_strides_and_x_past_4_gib():
    """The resident-W kernel (fin, fout <= 128, 16-byte aligned rows) with
    padded leading dimensions: X's padding columns hold infinities that must
    never be read, H's padding columns stay untouched. X spanning 4 GiB or
    more takes the tiled kernel: same tolerance."""
    rng = np.random.default_rng(11)
    n, fin, fout = 2051, 100, 44
    X = rng.standard_normal((n, fin)).astype(np.float32)
    W = graphgen.weights(fin, fout, seed=12)
    Xp = torch.full((n, fin + 8), float("inf"), device=DEV)
    Xp[:, :fin] = _dev(X)
    Wp = torch.full((fin, fout + 4), float("inf"), device=DEV)
    Wp[:, :fout] = _dev(W)
    Hp = torch.full((n, fout + 12), 7.0, device=DEV)
    agcn.linear(Xp[:, :fin], Wp[:, :fout], out=Hp[:, :fout])
    _check_linear(X, W, Hp[:, :fout].cpu().numpy(), "padded strides")
    assert torch.all(Hp[:, fout:] == 7.0)
    n2, ld2 = 60_000, 18_000                  # n2 * ld2 * 4 bytes > 4 GiB
    X2 = rng.standard_normal((n2, 64)).astype(np.float32)
    W2 = graphgen.weights(64, 128, seed=13)
    big = torch.empty((n2, ld2), device=DEV)
    big[:, :64] = _dev(X2)
    H2 = agcn.linear(big[:, :64], _dev(W2)).cpu().numpy()
    del big
    _check_linear(X2, W2, H2, "X past 4 GiB")
