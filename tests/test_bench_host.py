"""Host-side checks of bench.py that need no GPU: the multi-GPU refusal and
the algorithmic byte model used by its roofline."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402


def test_more_than_one_gpu_is_refused_with_a_message():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode != 0
    assert "one GPU" in r.stderr


class _Stats:
    n_rows, nnz, n_entries, n_hub_rows, n_hub_chunks = 1000, 50_000, 120, 3, 40


@pytest.mark.parametrize("F", [16, 128])
def test_kernel_bytes_model(F):
    st = _Stats()
    b7, b8 = bench.kernel_bytes(st, F, n_ref=900)
    nonhub = st.n_rows - st.n_hub_rows
    assert b7 == (8 * st.nnz + 16 * st.n_entries + 4 * nonhub + 4 * F * 900 + 4 * F * nonhub
                  + 4 * F * st.n_hub_chunks)
    assert b8 == 4 * F * st.n_hub_chunks + 4 * F * st.n_hub_rows + 8 * st.n_hub_rows
    w7, w8 = bench.kernel_bytes(st, F, n_ref=900, variant="warp_level")
    assert w7 == 8 * st.nnz + 16 * st.n_entries + 4 * F * 900 + 4 * F * st.n_rows
    assert w8 == 8 * st.n_rows


def test_kernel_names_match_the_library_dispatch():
    assert bench.spmm_kernel_name(16) == "k_spmm<4, 4>"
    assert bench.spmm_kernel_name(256) == "k_spmm<4, 8>"
    assert bench.spmm_kernel_name(17) == "k_spmm<1, 17>"
    assert bench.spmm_kernel_name(64, "column_loop") == "k_spmm_colloop"
    assert bench.spmm_kernel_name(64, "warp_level") == "k_spmm_wl<4, 8>"


def test_linear_kernel_names_match_the_library_dispatch():
    assert bench.linear_kernel_name(128, 128) == "k_linear_rw<8, 8>"
    assert bench.linear_kernel_name(32, 16) == "k_linear_rw<2, 2>"
    assert bench.linear_kernel_name(64, 100) == "k_linear_rw<8, 4>"
    assert bench.linear_kernel_name(256, 128) == "k_linear<128, true>"
    assert bench.linear_kernel_name(128, 200) == "k_linear<128, true>"
    assert bench.linear_kernel_name(30, 64) == "k_linear<64, false>"


def test_small_path_kernel_name():
    class St:
        n_hub_rows, max_deg, max_wave_nzs, nnz, n_rows = 0, 21, 32, 36844, 4096
    assert bench.small_path(St)
    assert bench.spmm_kernel_name(16, "block", St) == "k_spmm_rows<4, 4>"
    assert bench.spmm_kernel_name(64, "block", St) == "k_spmm_rows<4, 8>"
    St.max_deg = 33
    assert not bench.small_path(St)
    assert bench.spmm_kernel_name(16, "block", St) == "k_spmm<4, 4>"


def test_gather_requests_model():
    class St:
        nnz = 1000
    assert bench.gather_requests(St, 16) == 1000
    assert bench.gather_requests(St, 32) == 1000
    assert bench.gather_requests(St, 256) == 8000
