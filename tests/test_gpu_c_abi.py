"""End to end through the C-ABI alone, from plain C: tests/c_abi/forward_gpu.c
(gcc -std=c99, HIP runtime API for device buffers) quantizes Q, K, V and runs
both forwards on a stream; with V = 2^-3 everywhere every output element is
0.125 up to fp32 summation, whatever Q and K."""
import os
import shutil
import subprocess

import pytest

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
LIB_DIR = os.path.join(ROOT, "paper_2609_04105_amd")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")


@pytest.mark.skipif(shutil.which("gcc") is None, reason="gcc is not installed")
def test_c_client_runs_both_forwards(tmp_path):
    exe = tmp_path / "forward_gpu"
    cmd = ["gcc", "-std=c99", "-Wall", "-Wextra", "-Werror", "-D__HIP_PLATFORM_AMD__",
           "-I", os.path.join(ROCM, "include"), "-I", os.path.join(ROOT, "include"),
           os.path.join(ROOT, "tests", "c_abi", "forward_gpu.c"), "-L", LIB_DIR, "-lfp4attn",
           "-L", os.path.join(ROCM, "lib"), "-lamdhip64", "-lm", f"-Wl,-rpath,{LIB_DIR}", "-o", str(exe)]
    res = subprocess.run(cmd, capture_output=True, text=True)
    assert res.returncode == 0, res.stderr
    print("[c-abi] running the C client", flush=True)
    run = subprocess.run([str(exe)], capture_output=True, text=True, timeout=120)
    print(run.stdout, flush=True)
    assert run.returncode == 0, run.stderr + run.stdout
    assert "all checks held" in run.stdout
