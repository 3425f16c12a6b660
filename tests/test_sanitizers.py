"""Sanitizer builds on the CPU: the C oracle and the host code of the C-ABI
library compiled with AddressSanitizer and UndefinedBehaviorSanitizer, each
driven by a small C program under tests/native/ that exits non-zero when an
invariant or an expected error code does not hold.  A sanitizer report aborts
the program (no recovery), so a clean exit is the pass condition.

Only host code is instrumented: the library's sources are compiled for gfx950
as usual, with every sanitizer flag given to the host pass alone; the driver
never launches a kernel (every call it makes fails in argument checking or at
device discovery), so its device code is built without optimisation to keep
the build short."""

import os
import shutil
import subprocess
from concurrent.futures import ThreadPoolExecutor

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
NATIVE = os.path.join(ROOT, "tests", "native")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")
HIPCC = os.path.join(ROCM, "bin", "hipcc")
CLANG = os.path.join(ROCM, "llvm", "bin", "clang")

SAN_ENV = {
    # abort on the first report; the harness may preload its own library first
    "ASAN_OPTIONS": "detect_leaks=1:abort_on_error=0:halt_on_error=1:verify_asan_link_order=0",
    "UBSAN_OPTIONS": "print_stacktrace=1:halt_on_error=1",
}


def _run(cmd, cwd, env=None, timeout=600):
    r = subprocess.run(cmd, cwd=cwd, env=env, capture_output=True, text=True, timeout=timeout)
    return r.returncode, r.stdout + r.stderr


def _san_env():
    env = dict(os.environ)
    env.update(SAN_ENV)
    return env


def _assert_clean(rc, out, what):
    assert rc == 0, f"{what} exited {rc}:\n{out[-4000:]}"
    for marker in ("ERROR: AddressSanitizer", "ERROR: LeakSanitizer", "Sanitizer: WARNING", "runtime error:"):
        assert marker not in out, f"{what} reported a sanitizer finding:\n{out[-4000:]}"


@pytest.mark.skipif(shutil.which("gcc") is None, reason="gcc not available")
def test_oracle_under_address_and_ub_sanitizers(tmp_path):
    exe = str(tmp_path / "oracle_driver")
    rc, out = _run(["gcc", "-std=c11", "-O1", "-g", "-fopenmp", "-fno-omit-frame-pointer",
                    "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
                    os.path.join(ROOT, "oracle", "umap_oracle.c"), os.path.join(NATIVE, "oracle_driver.c"),
                    "-lm", "-o", exe], cwd=ROOT)
    assert rc == 0, out
    env = _san_env()
    env["OMP_NUM_THREADS"] = "4"
    rc, out = _run([exe], cwd=str(tmp_path), env=env, timeout=300)
    _assert_clean(rc, out, "oracle driver")
    assert "oracle driver ok" in out


@pytest.mark.skipif(not (os.path.exists(HIPCC) and os.path.exists(CLANG)), reason="ROCm toolchain not available")
def test_host_library_under_address_and_ub_sanitizers(tmp_path):
    from paper_2008_00325_amd import _build

    objs = []
    jobs = []
    for src in _build.SOURCES:
        obj = str(tmp_path / (src + ".o"))
        objs.append(obj)
        jobs.append([HIPCC, "--offload-arch=gfx950", "-O1", "-g", "-Xarch_device", "-O0", "-std=c++17", "-fPIC",
                     "-c", "-fno-omit-frame-pointer",
                     "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
                     "-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
                     "-Xarch_host", "-fno-sanitize-recover=all",
                     "-Wno-unused-command-line-argument", "-I", os.path.join(ROOT, "include"),
                     os.path.join(_build.CSRC, src), "-o", obj])
    with ThreadPoolExecutor(max_workers=min(len(jobs), os.cpu_count() or 1)) as ex:
        for rc, out in ex.map(lambda c: _run(c, ROOT), jobs):
            assert rc == 0, out
    lib = str(tmp_path / "libumap_layout_san.so")
    rc, out = _run([HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC",
                    "-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
                    *objs, "-o", lib], cwd=ROOT)
    assert rc == 0, out
    exe = str(tmp_path / "api_driver")
    rc, out = _run([CLANG, "-std=c11", "-O1", "-g", "-fno-omit-frame-pointer", "-fsanitize=address,undefined",
                    "-fno-sanitize-recover=all", "-I", os.path.join(ROOT, "include"),
                    os.path.join(NATIVE, "api_driver.c"), lib, f"-Wl,-rpath,{tmp_path}",
                    f"-L{ROCM}/lib", "-lamdhip64", f"-Wl,-rpath,{ROCM}/lib", "-lm", "-o", exe], cwd=ROOT)
    assert rc == 0, out
    rc, out = _run([exe], cwd=str(tmp_path), env=_san_env(), timeout=300)
    _assert_clean(rc, out, "api driver")
    assert "api driver ok" in out
