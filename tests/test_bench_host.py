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


class _WinStats:
    n_rows, nnz, n_hub_rows, hub_first_entry, deg_bound = 1_000_000, 111_640_508, 1000, 270_000, 512
    hub_windows = 1954


def test_window_shape_and_bytes_model():
    # skewed_hubs' shape: 1000 hub rows, 1954 windows of 512 columns; one row
    # batch; F = 64 is one slice, so about 512 workgroups means G = 4 windows
    # per group (489 groups); F = 256 has four slices, so G = 16 (123 groups).
    st = _WinStats()
    assert bench.win_shape(st, 64) == (1, 1, 4, 489)
    assert bench.win_shape(st, 256) == (4, 1, 16, 123)
    assert bench.win_shape(st, 96) == (2, 1, 8, 245)
    hub = {"hub_nnz": 107_144_212, "n_cols": 1_000_000, "low_nnz": 4_496_296,
           "low_entries": 270_000, "low_ref": 990_000}
    b_low, b_hub = bench.window_bytes(st, 64, hub)
    assert b_hub == (8 * hub["hub_nnz"] + 4 * 64 * hub["n_cols"] + 8 * 1000 * 1954
                     + 2 * (4 * 64 + 4) * 1000 * 489 + (4 * 64 + 4) * 1000)
    nonhub = st.n_rows - st.n_hub_rows
    assert b_low == (8 * hub["low_nnz"] + 16 * hub["low_entries"] + 4 * nonhub
                     + 4 * 64 * hub["low_ref"] + 4 * 64 * nonhub)
    # the windows serve F >= 64 on the float4 path of the block-level plan only
    assert bench.windows_used(st, 64) and bench.windows_used(st, 512)
    assert not bench.windows_used(st, 32) and not bench.windows_used(st, 66)
    assert not bench.windows_used(st, 64, "warp_level")
    st.hub_windows = 0
    assert not bench.windows_used(st, 64)
