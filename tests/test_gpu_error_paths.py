"""Error paths of agcn_plan_create on the device, forced from the host.

* An allocation that fails (AGCN_TEST_FAIL_ALLOC=k: the k-th allocation
  attempt of the call fails as out of memory): the call returns
  AGCN_ERR_OUT_OF_MEMORY, sets *out to NULL and leaves no device memory
  behind once the plan-memory cache is emptied.
* The hub-chunk launch-order sort runs after the host has read the plan's
  summary, so a failure inside it (AGCN_TEST_FAIL_ORDER_SORT=1 raises the
  internal-error flag before it, as a scan that gives up its bounded wait
  would) must leave a valid launch order: every entry launched once, Y equal
  to the normally planned one bit for bit and to the oracle within tolerance.

Every kernel still runs to its normal end: the failures are injected on the
host or as a flag the kernels read.
"""
import ctypes
import threading

import numpy as np
import pytest

import graphgen
from gpu_helpers import DEV, _dev, _plan, _spmm_check, assert_plan_matches_oracle, _mixed

torch = pytest.importorskip("torch")
import paper_2308_11825_amd as agcn  # noqa: E402

pytestmark = pytest.mark.gpu


def _raw_create(g, d):
    """agcn_plan_create through the raw C call: (status, handle value)."""
    lib = agcn.load_library()
    h = ctypes.c_void_p(0x1234)   # poisoned: the call must overwrite it
    rc = lib.agcn_plan_create(ctypes.byref(h), g.n_rows, g.n_cols, g.nnz, d[0].data_ptr(),
                              d[1].data_ptr(), d[2].data_ptr(), None, None)
    return rc, h.value


def _in_thread(fn):
    """Runs fn in a fresh host thread (a thread's first plan allocates its
    pinned read-back buffer) and returns its result."""
    out = {}

    def run():
        try:
            out["r"] = fn()
        except BaseException as e:  # noqa: BLE001 -- re-raised below
            out["e"] = e
    t = threading.Thread(target=run)
    t.start()
    t.join()
    if "e" in out:
        raise out["e"]
    return out["r"]


def _free_bytes():
    torch.cuda.synchronize()
    return torch.cuda.mem_get_info()[0]


SLACK = 2 << 20   # the runtime's own small allocations (a new thread's first call)


def test_plan_allocation_failure_unwinds(monkeypatch):
    g = _mixed(501, n=20000)
    d = (_dev(g.rowptr), _dev(g.colidx), _dev(g.vals))
    torch.cuda.synchronize()
    probe = _plan(g)
    block = probe.stats.device_bytes
    probe.destroy()
    assert block > 8 * SLACK
    # one injected failure first, so that anything the runtime sets up lazily
    # on such a call is in place before the baseline is taken
    agcn.agcn_release_cached_memory()
    free_pre = _free_bytes()
    monkeypatch.setenv("AGCN_TEST_FAIL_ALLOC", "1")
    assert _raw_create(g, d)[0] == agcn.AGCN_ERR_OUT_OF_MEMORY
    agcn.agcn_release_cached_memory()
    free0 = _free_bytes()
    print(f"[alloc-fail] free before the first injected failure {free_pre}, after {free0}", flush=True)

    def leaked():
        """Device bytes lost since the baseline (a leak lowers free memory)."""
        f = _free_bytes()
        print(f"[alloc-fail] free {f} baseline {free0} lost {free0 - f}", flush=True)
        return free0 - f

    # 1: the plan's device block
    monkeypatch.setenv("AGCN_TEST_FAIL_ALLOC", "1")
    rc, h = _raw_create(g, d)
    assert rc == agcn.AGCN_ERR_OUT_OF_MEMORY, agcn.agcn_status_string(rc)
    assert h is None
    assert "hipMalloc" in agcn.agcn_last_error()
    agcn.agcn_release_cached_memory()
    assert leaked() <= SLACK

    # 2 in a fresh thread: the device block is allocated, then the thread's
    # pinned read-back buffer fails; the block goes back to the cache
    monkeypatch.setenv("AGCN_TEST_FAIL_ALLOC", "2")
    rc, h = _in_thread(lambda: _raw_create(g, d))
    assert rc == agcn.AGCN_ERR_OUT_OF_MEMORY, agcn.agcn_status_string(rc)
    assert h is None
    agcn.agcn_release_cached_memory()
    assert leaked() <= SLACK

    # 3 in a fresh thread: there is no third attempt, the plan is built
    monkeypatch.setenv("AGCN_TEST_FAIL_ALLOC", "3")
    rc, h = _in_thread(lambda: _raw_create(g, d))
    assert rc == agcn.AGCN_OK and h is not None
    agcn.agcn_plan_destroy(h)

    # unset: normal plans again, bit-exact, and the memory comes back
    monkeypatch.delenv("AGCN_TEST_FAIL_ALLOC")
    plan = _plan(g)
    assert_plan_matches_oracle(plan, g)
    _spmm_check(plan, g, 32)
    plan.destroy()
    agcn.agcn_release_cached_memory()
    assert leaked() <= SLACK


def test_hub_order_sort_failure_keeps_a_valid_order(monkeypatch):
    rng = np.random.default_rng(43)
    n = 60000
    deg = rng.integers(1, 9, size=n)
    hubs = rng.choice(n, size=24, replace=False)
    deg[hubs] = rng.integers(20000, 50001, size=hubs.size)
    g = graphgen.random_csr(n, n, deg, seed=44)
    X = np.random.default_rng(45).standard_normal((n, 64)).astype(np.float32)
    Xd = _dev(X)

    ref = _plan(g)
    st = ref.stats
    assert st.n_hub_chunks >= 8 * st.n_hub_rows      # the column-ordered launch is used
    Y_ref = ref.spmm(Xd).cpu().numpy()
    ref.destroy()

    monkeypatch.setenv("AGCN_TEST_FAIL_ORDER_SORT", "1")
    plan = _plan(g)
    monkeypatch.delenv("AGCN_TEST_FAIL_ORDER_SORT")
    assert_plan_matches_oracle(plan, g)
    Y = plan.spmm(Xd).cpu().numpy()
    assert np.array_equal(Y.view(np.uint32), Y_ref.view(np.uint32))
    _spmm_check(plan, g, 64, X=X)
    plan.destroy()

    # the next plan on the same memory (error word cleared by its first kernels)
    again = _plan(g)
    assert np.array_equal(again.spmm(Xd).cpu().numpy().view(np.uint32), Y_ref.view(np.uint32))
    again.destroy()
