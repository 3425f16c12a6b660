"""The C ABI from a plain C program (no Python in the process): build
tests/native/c_client.c against the in-tree library and run it on the GPU."""

import os
import shutil
import subprocess

import pytest

from paper_2008_00325_amd import umap_layout as U

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.mark.skipif(shutil.which("gcc") is None, reason="gcc not available")
def test_c_client(tmp_path):
    lib_dir = os.path.dirname(U.LIB_PATH)
    assert os.path.exists(U.LIB_PATH), "build the library first"
    exe = str(tmp_path / "c_client")
    r = subprocess.run(["gcc", "-std=c11", "-O2", "-Wall", "-I", os.path.join(ROOT, "include"),
                        os.path.join(ROOT, "tests", "native", "c_client.c"), "-L", lib_dir, "-lumap_layout",
                        f"-Wl,-rpath,{lib_dir}", "-lm", "-o", exe], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, r.stderr
    print("[gpu case] c client: 20,000-vertex ring, 60 epochs", flush=True)
    r = subprocess.run([exe], capture_output=True, text=True, timeout=120)
    print(r.stdout, r.stderr, flush=True)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "c client ok" in r.stdout
