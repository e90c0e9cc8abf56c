"""The public headers compile as strict C99 (gcc -std=c99 -pedantic -Werror)
and a plain C program linked against libssba.so can call the entry points
that need no device: version, status strings, workspace sizes and the
argument checks of the forward, Haar and probe calls (tests/c/abi_from_c.c)."""
import os
import shutil
import subprocess

import pytest

from paper_2605_15684_amd import _lib

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.mark.skipif(shutil.which("gcc") is None, reason="gcc not installed")
def test_c99_caller(tmp_path):
    if not os.path.exists(_lib.LIB_PATH):
        from paper_2605_15684_amd import build
        build.build()
    libdir = os.path.dirname(_lib.LIB_PATH)
    exe = tmp_path / "abi_from_c"
    cmd = ["gcc", "-std=c99", "-Wall", "-Wextra", "-Werror", "-pedantic",
           "-I", os.path.join(ROOT, "include"), os.path.join(ROOT, "tests", "c", "abi_from_c.c"),
           "-L", libdir, "-lssba", f"-Wl,-rpath,{libdir}", "-o", str(exe)]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
    r = subprocess.run([str(exe)], capture_output=True, text=True, timeout=60)
    assert r.returncode == 0, r.stderr
    assert r.stdout.strip() == "ok"
