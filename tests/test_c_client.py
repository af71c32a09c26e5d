"""The C ABI is usable from plain C: tests/c/abi_check.c compiles as C99
with warnings as errors against include/pcpp.h, links to libpcpp.so and runs
its host-side checks (no GPU needed)."""

import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_c_client_builds_and_runs(tmp_path):
    cc = shutil.which("gcc") or shutil.which("cc")
    if cc is None:
        pytest.skip("no C compiler")
    from paper_2412_02962_amd import pcpp
    lib_dir = os.path.dirname(pcpp.LIB_PATH)
    exe = tmp_path / "abi_check"
    cmd = [cc, "-std=c99", "-Wall", "-Wextra", "-Werror", "-I", os.path.join(ROOT, "include"),
           os.path.join(ROOT, "tests", "c", "abi_check.c"), "-L", lib_dir, "-lpcpp", f"-Wl,-rpath,{lib_dir}",
           "-o", str(exe)]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
    r = subprocess.run([str(exe)], capture_output=True, text=True, timeout=60)
    assert r.returncode == 0, f"check {r.returncode} failed: {r.stdout} {r.stderr}"
    assert "C ABI checks passed" in r.stdout
