"""libagcn's host code built with AddressSanitizer and
UndefinedBehaviorSanitizer (hipcc; the flags apply to the host pass only,
the gfx950 device code is built as usual) and driven from a plain C program
through every argument check of the C ABI (tests/c_abi_host_check.c). No GPU
is needed: each call is refused on the host, or fails cleanly for want of a
device."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
CLANG = "/opt/rocm/llvm/bin/clang"


@pytest.mark.skipif(not (os.path.exists(HIPCC) and os.path.exists(CLANG)), reason="needs hipcc")
def test_c_abi_host_code_under_asan_and_ubsan(tmp_path):
    import glob
    lib = str(tmp_path / "libagcn_san.so")
    srcs = sorted(glob.glob(os.path.join(ROOT, "paper_2308_11825_amd", "csrc", "*.hip")))
    host_san = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
                "-Xarch_host", "-fno-sanitize-recover=all"]
    subprocess.run([HIPCC, "--offload-arch=gfx950", "-O1", "-g", "-std=c++17", "-fPIC",
                    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops", *host_san,
                    "-I", os.path.join(ROOT, "include"), "-shared", *srcs, "-o", lib],
                   check=True, capture_output=True, text=True, timeout=600)
    exe = str(tmp_path / "c_abi_host_check")
    subprocess.run([CLANG, "-std=c99", "-O1", "-g", "-fsanitize=address,undefined",
                    "-fno-sanitize-recover=all", "-I", os.path.join(ROOT, "include"),
                    os.path.join(ROOT, "tests", "c_abi_host_check.c"), "-L", str(tmp_path),
                    "-lagcn_san", "-Wl,-rpath," + str(tmp_path), "-o", exe],
                   check=True, capture_output=True, text=True, timeout=300)
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1", UBSAN_OPTIONS="print_stacktrace=1",
               HIP_VISIBLE_DEVICES="")
    r = subprocess.run([exe], capture_output=True, text=True, timeout=300, env=env)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "c abi host check ok" in r.stdout
