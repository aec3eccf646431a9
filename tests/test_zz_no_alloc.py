"""agcn_spmm_noalloc, the execute for callers that cannot allocate: called
through the C ABI, its Y must equal agcn_spmm_ex's bit for bit (same kernels,
the fixed device workspace in place of the caller's) and the oracle's within
1e-5 * S + 1e-7, on consecutive calls whose second input is smaller (the
workspace then holds the first call's partials), on both partitions and on
the scalar path; workspaces beyond the fixed size are refused before any
launch."""
import ctypes

import numpy as np
import pytest

import graphgen
import oracle
from gpu_helpers import DEV, _dev, _mixed, _plan, assert_close

torch = pytest.importorskip("torch")
import paper_2308_11825_amd as agcn  # noqa: E402

pytestmark = pytest.mark.gpu


def _stream(s=None):
    return (s or torch.cuda.current_stream()).cuda_stream


def _reference(plan, Xd, F, act):
    """agcn_spmm_ex with a workspace from the caller."""
    Y = torch.full((plan.n_rows, F), float("nan"), device=DEV)
    ws = plan.workspace(F)
    agcn.agcn_spmm_ex(plan.handle, F, Xd.data_ptr(), F, Y.data_ptr(), F,
                      ws.data_ptr() if ws is not None else None, _stream(), act)
    return Y


def _noalloc(plan, Xd, F, act, stream=None):
    Y = torch.full((plan.n_rows, F), float("nan"), device=DEV)
    rc = agcn.load_library().agcn_spmm_noalloc(plan.handle, F, Xd.data_ptr(), F, Y.data_ptr(), F,
                                                _stream(stream), act)
    assert rc == agcn.AGCN_OK, agcn.agcn_last_error()
    return Y


def _case(g, F, seed):
    X = np.random.default_rng(seed).standard_normal((g.n_cols, F)).astype(np.float32)
    return X, _dev(X)


@pytest.mark.parametrize("flags", [0, agcn.AGCN_PLAN_WARP_LEVEL, agcn.AGCN_PLAN_COLUMN_LOOP])
def test_noalloc_matches_the_workspace_call_twice_in_a_row(flags):
    big = _mixed(601, n=40000, hub_max=8000)
    small = _mixed(602, n=6000, hub_max=3000)
    pb, ps = _plan(big, flags=flags), _plan(small, flags=flags)
    assert pb.workspace_bytes(96) > 0 and ps.workspace_bytes(40) > 0
    assert pb.workspace_bytes(96) <= agcn.AGCN_NOALLOC_MAX_WORKSPACE
    cases = [(pb, big, 96, agcn.AGCN_EPILOGUE_NONE, 1), (ps, small, 40, agcn.AGCN_EPILOGUE_RELU, 2),
             (ps, small, 33, agcn.AGCN_EPILOGUE_NONE, 3)]     # F = 33: the scalar path
    outs = []
    for plan, g, F, act, seed in cases:     # consecutive calls on one stream, no sync between
        X, Xd = _case(g, F, seed)
        outs.append((plan, g, F, act, X, Xd, _noalloc(plan, Xd, F, act)))
    for plan, g, F, act, X, Xd, Y in outs:
        Yn = Y.cpu().numpy()
        Yr = _reference(plan, Xd, F, act).cpu().numpy()
        assert np.array_equal(Yn.view(np.uint32), Yr.view(np.uint32)), (flags, F)
        if act == agcn.AGCN_EPILOGUE_NONE:
            Yo, S = oracle.spmm(g.rowptr, g.colidx, g.vals, X, want_scale=True)
            assert_close(Yn, Yo, S, f"noalloc flags={flags} F={F}")
        print(f"[noalloc] flags={flags} n={g.n_rows} F={F} act={act} ok", flush=True)
    pb.destroy()
    ps.destroy()


def test_noalloc_on_another_stream_then_destroy():
    g = _mixed(611, n=20000, hub_max=6000)
    plan = _plan(g)
    F = 64
    X, Xd = _case(g, F, 5)
    s = torch.cuda.Stream()
    torch.cuda.synchronize()
    with torch.cuda.stream(s):
        Y = _noalloc(plan, Xd, F, agcn.AGCN_EPILOGUE_NONE, stream=s)
        Y2 = _noalloc(plan, Xd, F, agcn.AGCN_EPILOGUE_NONE, stream=s)
    plan.destroy()          # waits for the device: the stream was never tracked by an event
    torch.cuda.synchronize()
    Yo, S = oracle.spmm(g.rowptr, g.colidx, g.vals, X, want_scale=True)
    assert_close(Y.cpu().numpy(), Yo, S, "noalloc on a side stream")
    assert np.array_equal(Y.cpu().numpy(), Y2.cpu().numpy())
    again = _plan(g)        # reuses the destroyed plan's memory
    Yn = _noalloc(again, Xd, F, agcn.AGCN_EPILOGUE_NONE).cpu().numpy()
    assert np.array_equal(Yn, Y.cpu().numpy())
    again.destroy()


def test_noalloc_refuses_workspaces_beyond_the_fixed_size():
    n = 60000
    deg = np.full(n, 3)
    deg[:40] = 50000
    g = graphgen.random_csr(n, n, deg, seed=621)
    plan = _plan(g)
    F = 8192
    need = plan.workspace_bytes(F)
    assert need > agcn.AGCN_NOALLOC_MAX_WORKSPACE
    lib = agcn.load_library()
    # refused on the host before any launch: the arrays are never touched
    rc = lib.agcn_spmm_noalloc(plan.handle, F, ctypes.c_void_p(1 << 44), F,
                               ctypes.c_void_p(2 << 44), F, None, 0)
    assert rc == agcn.AGCN_ERR_UNSUPPORTED
    assert "fixed workspace" in agcn.agcn_last_error()
    # a width that fits runs
    F = 64
    assert plan.workspace_bytes(F) <= agcn.AGCN_NOALLOC_MAX_WORKSPACE
    X, Xd = _case(g, F, 7)
    Yn = _noalloc(plan, Xd, F, agcn.AGCN_EPILOGUE_NONE).cpu().numpy()
    Yo, S = oracle.spmm(g.rowptr, g.colidx, g.vals, X, want_scale=True)
    assert_close(Yn, Yo, S, "noalloc after a refused call")
    plan.destroy()
