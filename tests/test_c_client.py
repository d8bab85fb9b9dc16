"""The C ABI from a C program: tests/c_client/ntt_client.c (HIP runtime for device memory, no Python or torch in
the path) is compiled with gcc against include/ckks_mi.h and linked to libckks_mi.so.  Without a GPU it must
build, load the library and report the missing device through the ABI's error text (exit status 2); on a GPU it
checks the NTT against its definition and the inverse round trip (exit status 0)."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "tests", "c_client", "ntt_client.c")
PKG = os.path.join(ROOT, "paper_2609_12378_amd")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")


def build(tmp_path):
    from paper_2609_12378_amd import LIB_PATH, build as b
    if not os.path.exists(LIB_PATH):
        b.build()
    cc = shutil.which("gcc") or shutil.which("cc")
    if cc is None:
        pytest.skip("no C compiler")
    exe = str(tmp_path / "ntt_client")
    cmd = [cc, "-std=c11", "-O2", "-Wall", "-Wextra", "-Werror", "-D__HIP_PLATFORM_AMD__",
           "-I", os.path.join(ROCM, "include"), "-I", os.path.join(ROOT, "include"), SRC,
           "-L", PKG, "-lckks_mi", "-L", os.path.join(ROCM, "lib"), "-lamdhip64",
           "-Wl,-rpath," + PKG, "-Wl,-rpath," + os.path.join(ROCM, "lib"), "-o", exe]
    subprocess.run(cmd, check=True, capture_output=True, text=True)
    return exe


def run(exe):
    return subprocess.run([exe], capture_output=True, text=True, timeout=120)


def test_c_client_builds_and_reports_through_the_abi(tmp_path):
    import torch
    if torch.cuda.is_available():
        pytest.skip("covered by the GPU run of the same client")
    exe = build(tmp_path)
    r = run(exe)
    assert r.returncode == 2, (r.returncode, r.stdout, r.stderr)
    assert "no context" in r.stderr


@pytest.mark.gpu
def test_c_client_ntt_against_definition(tmp_path):
    from gpu_common import require_gpu
    require_gpu()
    exe = build(tmp_path)
    r = run(exe)
    print(r.stdout, r.stderr, flush=True)
    assert r.returncode == 0, (r.returncode, r.stdout, r.stderr)
    assert "ntt_client: ok" in r.stdout
