"""The C ABI driven from plain C (tests/c_abi_check.c): no Python or torch in
the process. The CPU test compiles it with gcc against include/agcn.h and the
oracle's header; the GPU test runs it (plan bit-exact, SpMM with and without
ReLU, and a GCN layer, each against the oracle)."""
import os
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "tests", "c_abi_check.c")
PKG = os.path.join(ROOT, "paper_2308_11825_amd")
ORACLE = os.path.join(ROOT, "oracle")


def _compile(out):
    import oracle
    import paper_2308_11825_amd as agcn
    if not os.path.exists(agcn.LIB_PATH):
        pytest.fail("libagcn.so is not built (python -m paper_2308_11825_amd.build)")
    oracle.build(force=False)
    cmd = ["gcc", "-std=c11", "-O2", "-Wall", "-Werror", "-D__HIP_PLATFORM_AMD__",
           "-I/opt/rocm/include", "-I" + os.path.join(ROOT, "include"), "-I" + ORACLE, SRC,
           "-o", out, "-L" + PKG, "-lagcn", "-L" + ORACLE, "-loracle_agcn", "-L/opt/rocm/lib",
           "-lamdhip64", "-lm", "-Wl,-rpath," + ":".join([PKG, ORACLE, "/opt/rocm/lib"])]
    r = subprocess.run(cmd, capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, r.stderr
    return out


def test_c_program_compiles_against_the_header(tmp_path):
    _compile(str(tmp_path / "c_abi_check"))


@pytest.mark.gpu
def test_c_program_runs_and_matches_the_oracle(tmp_path):
    exe = _compile(str(tmp_path / "c_abi_check"))
    print("[c-abi] running", exe, flush=True)
    r = subprocess.run([exe], capture_output=True, text=True, timeout=120)
    print(r.stdout, r.stderr, flush=True)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "plan metadata bit-exact: yes" in r.stdout and "C ABI check: ok" in r.stdout
