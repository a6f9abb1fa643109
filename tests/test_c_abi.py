"""The C ABI used from C (no GPU): tests/c/abi_host.c is compiled with gcc
against include/spconv.h as C99 with warnings as errors, linked to
libspconv.so, and run."""

import os
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
LIBDIR = os.path.join(ROOT, "paper_1911_09723_amd")


def test_host_calls_from_c(tmp_path):
    if not os.path.exists(os.path.join(LIBDIR, "libspconv.so")):
        pytest.fail("libspconv.so is not built")
    exe = tmp_path / "abi_host"
    subprocess.check_call(["gcc", "-std=c99", "-Wall", "-Wextra", "-Werror", "-I", os.path.join(ROOT, "include"),
                           os.path.join(ROOT, "tests", "c", "abi_host.c"), "-o", str(exe), "-L", LIBDIR, "-lspconv",
                           "-Wl,-rpath," + LIBDIR])
    out = subprocess.run([str(exe)], capture_output=True, text=True, timeout=120)
    assert out.returncode == 0 and out.stdout.strip().endswith("ok"), out.stdout + out.stderr
