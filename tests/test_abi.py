"""C-ABI checks that need no GPU: the library loads, exports every function
include/agcn.h declares, and rejects bad arguments on the host before any HIP
call is made."""
import ctypes
import os
import re

import pytest

import paper_2308_11825_amd as agcn
from conftest import ROOT

HEADER = os.path.join(ROOT, "include", "agcn.h")


def _declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(agcn_[a-z_]+)\s*\(", text)))


@pytest.fixture(scope="module")
def lib():
    return agcn.load_library()


def test_library_exports_every_declared_function(lib):
    names = _declared_functions()
    assert len(names) >= 10
    for n in names:
        assert hasattr(lib, n), n
    assert sorted(agcn.EXPORTED_SYMBOLS) == names


def test_header_compiles_as_c(tmp_path):
    src = tmp_path / "t.c"
    src.write_text('#include "agcn.h"\nint main(void){agcn_plan_params p; agcn_default_params(&p); '
                   'return p.max_block_waves > 0 ? 0 : 1;}\n')
    import subprocess
    r = subprocess.run(["gcc", "-std=c99", "-Wall", "-Werror", "-fsyntax-only",
                        "-I", os.path.join(ROOT, "include"), str(src)], capture_output=True, text=True)
    assert r.returncode == 0, r.stderr


def test_default_params_and_status_strings(lib):
    p = agcn.agcn_default_params()
    assert p.max_block_waves >= 1 and p.max_wave_nzs >= 1 and p.hub_chunk_nnz >= 0 and p.flags == 0
    assert p.max_block_waves * p.max_wave_nzs <= 4096
    for code, name in [(0, "AGCN_OK"), (1, "AGCN_ERR_INVALID_ARGUMENT"), (2, "AGCN_ERR_INVALID_INPUT"),
                       (3, "AGCN_ERR_UNSUPPORTED"), (4, "AGCN_ERR_OUT_OF_MEMORY"), (5, "AGCN_ERR_HIP")]:
        assert agcn.agcn_status_string(code) == name
    assert agcn.agcn_status_string(99) == "AGCN_ERR_UNKNOWN"


def _create(lib, n_rows=4, n_cols=4, nnz=4, rowptr=0x1000, colidx=0x2000, vals=0x3000, params=None,
            out=True):
    h = ctypes.c_void_p(0xdead)
    rc = lib.agcn_plan_create(ctypes.byref(h) if out else None, n_rows, n_cols, nnz, rowptr, colidx,
                              vals, ctypes.byref(params) if params is not None else None, None)
    return rc, h


def _params(W=16, Z=32, H=0, flags=0):
    p = agcn.PlanParams()
    p.max_block_waves, p.max_wave_nzs, p.hub_chunk_nnz, p.flags = W, Z, H, flags
    return p


@pytest.mark.parametrize("kw,status", [
    (dict(out=False), 1),
    (dict(n_rows=-1), 1),
    (dict(n_cols=-1), 1),
    (dict(nnz=-1), 1),
    (dict(n_rows=0, nnz=5), 1),
    (dict(nnz=2**31), 3),
    (dict(rowptr=None), 1),
    (dict(colidx=None), 1),
    (dict(vals=None), 1),
    (dict(params=_params(W=0)), 1),
    (dict(params=_params(W=33)), 1),
    (dict(params=_params(Z=0)), 1),
    (dict(params=_params(W=16, Z=257)), 1),
    (dict(params=_params(H=-1)), 1),
    (dict(params=_params(H=4097)), 1),
    (dict(params=_params(flags=4)), 1),             # unknown flag
    (dict(params=_params(flags=3)), 1),             # the two ablations are exclusive
    (dict(params=_params(W=32, Z=128)), 1),         # needs > 64 KiB of LDS
    (dict(n_rows=2**31 - 2, nnz=2**31 - 1, params=_params(H=1)), 3),
])
def test_plan_create_rejects_on_host(lib, kw, status):
    rc, h = _create(lib, **kw)
    assert rc == status, agcn.agcn_last_error()
    if kw.get("out", True):
        assert h.value is None
    assert agcn.agcn_last_error() != ""


def test_null_plan_calls(lib):
    assert lib.agcn_spmm_ex(None, 16, 0x1000, 16, 0x2000, 16, None, None, 1) == 1
    n = ctypes.c_size_t()
    assert lib.agcn_gcn_workspace_size(None, 16, ctypes.byref(n)) == 1
    assert lib.agcn_gcn_layer(None, 8, 16, 0x1000, 8, 0x2000, 16, 0x3000, 16, 0x4000, None, 1) == 1
    assert lib.agcn_spmm(None, 16, 0x1000, 16, 0x2000, 16, None, None) == 1
    assert lib.agcn_spmm_timed(None, 16, 0x1000, 16, 0x2000, 16, None, None, None, None, None) == 1
    n = ctypes.c_size_t()
    assert lib.agcn_spmm_workspace_size(None, 16, ctypes.byref(n)) == 1
    assert lib.agcn_plan_info(None, ctypes.byref(agcn.PlanStats())) == 1
    assert lib.agcn_plan_export(None, None, None, None, None, None) == 1
    lib.agcn_plan_destroy(None)        # ignored
    with pytest.raises(agcn.AgcnError) as ei:
        agcn.agcn_spmm(None, 4, 1, 4, 2, 4)
    assert ei.value.status == agcn.AGCN_ERR_INVALID_ARGUMENT


def test_stats_struct_layout_matches_header():
    # int32 x2, int64 x4, int32 x8, size_t, int32 (+4 bytes of tail padding)
    assert ctypes.sizeof(agcn.PlanStats) == 8 + 32 + 32 + 8 + 8
    assert agcn.PlanStats.hub_windows.offset == 80
    assert ctypes.sizeof(agcn.PlanParams) == 16


def test_product_package_does_not_reference_the_oracle():
    pkg = os.path.join(ROOT, "paper_2308_11825_amd")
    for dirpath, _, files in os.walk(pkg):
        for f in files:
            if f.endswith((".py", ".hip", ".hpp", ".cpp", ".h")):
                text = open(os.path.join(dirpath, f)).read()
                assert "import oracle" not in text and "from oracle" not in text, f
                assert "agcn_oracle" not in text, f


@pytest.mark.parametrize("args,status", [
    ((-1, 4, 4, 0x1000, 4, 0x2000, 4, 0x3000, 4), 1),          # negative n
    ((8, -1, 4, 0x1000, 4, 0x2000, 4, 0x3000, 4), 1),          # negative fin
    ((8, 4, -2, 0x1000, 4, 0x2000, 4, 0x3000, 4), 1),          # negative fout
    ((8, 4, 4, 0x1000, 3, 0x2000, 4, 0x3000, 4), 1),           # ldx < fin
    ((8, 4, 4, 0x1000, 4, 0x2000, 3, 0x3000, 4), 1),           # ldw < fout
    ((8, 4, 4, 0x1000, 4, 0x2000, 4, 0x3000, 3), 1),           # ldh < fout
    ((8, 4, 4, None, 4, 0x2000, 4, 0x3000, 4), 1),             # X missing
    ((8, 4, 4, 0x1000, 4, None, 4, 0x3000, 4), 1),             # W missing
    ((8, 4, 4, 0x1000, 4, 0x2000, 4, None, 4), 1),             # H missing
    ((8, 4, 4, 0x1000, 4, 0x2000, 4, 0x1010, 4), 1),           # H overlaps X
    ((0, 4, 4, None, 4, 0x2000, 4, None, 4), 0),               # empty: nothing to launch
    ((8, 4, 0, 0x1000, 4, None, 0, None, 0), 0),               # fout = 0: nothing to launch
])
def test_linear_rejects_on_host(lib, args, status):
    assert lib.agcn_linear(*args, None) == status, agcn.agcn_last_error()
