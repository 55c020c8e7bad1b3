"""The header is a plain C99 header and the library a plain C library: a small
C program (tests/c_abi/validation.c) compiled with gcc -std=c99 -Wall -Werror
against include/fp4attn.h and linked against libfp4attn.so runs the documented
error paths (no GPU call) and checks status codes and strings."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
LIB_DIR = os.path.join(ROOT, "paper_2609_04105_amd")


@pytest.mark.skipif(shutil.which("gcc") is None, reason="gcc is not installed")
def test_c_client_compiles_links_and_validates(tmp_path):
    if not os.path.exists(os.path.join(LIB_DIR, "libfp4attn.so")):
        pytest.skip("libfp4attn.so is not built")
    exe = tmp_path / "validation"
    cmd = ["gcc", "-std=c99", "-Wall", "-Wextra", "-Werror", "-I", os.path.join(ROOT, "include"),
           os.path.join(ROOT, "tests", "c_abi", "validation.c"), "-L", LIB_DIR, "-lfp4attn",
           f"-Wl,-rpath,{LIB_DIR}", "-o", str(exe)]
    res = subprocess.run(cmd, capture_output=True, text=True)
    assert res.returncode == 0, res.stderr
    run = subprocess.run([str(exe)], capture_output=True, text=True, timeout=120)
    assert run.returncode == 0, run.stderr + run.stdout
    assert "all checks held" in run.stdout
