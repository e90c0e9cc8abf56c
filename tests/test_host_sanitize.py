"""The library's host layer (ssba_api.cpp: descriptor checks, workspace
arithmetic, dispatch, the layer-stack driver; ssba_select.cpp: kernel
selection) built for the CPU under AddressSanitizer and
UndefinedBehaviorSanitizer, with the kernel launchers replaced by recording
stand-ins (tests/sanitize/stub_launch.cpp), and driven by
tests/sanitize/host_driver.cpp: workspace sizes against their formulas, every
size-checked entry point with short and exact buffers, the layer stack's slice
offsets, offset alternation and index cache, and 20 000 descriptors at the
edges of the integer ranges.  No GPU is used; the sanitizers apply to host
code only."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2605_15684_amd", "csrc")
SAN = os.path.join(ROOT, "tests", "sanitize")
HIPCC = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"

# Host-only compilation; each sanitizer flag applies to the host side only.
FLAGS = ["-x", "hip", "--cuda-host-only", "-O1", "-g", "-std=c++17", "-fno-omit-frame-pointer",
         "-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
         "-Xarch_host", "-fno-sanitize-recover=all",
         "-I", os.path.join(ROOT, "include"), "-I", CSRC, "-I", SAN]


@pytest.mark.skipif(not os.path.exists(HIPCC), reason="hipcc not installed")
def test_host_layer_under_asan_ubsan(tmp_path):
    objs = []
    for src in (os.path.join(CSRC, "ssba_api.cpp"), os.path.join(CSRC, "ssba_select.cpp"),
                os.path.join(SAN, "stub_launch.cpp"), os.path.join(SAN, "host_driver.cpp")):
        obj = tmp_path / (os.path.basename(src) + ".o")
        r = subprocess.run([HIPCC, *FLAGS, "-c", src, "-o", str(obj)], capture_output=True, text=True)
        assert r.returncode == 0, r.stderr[-4000:]
        objs.append(str(obj))
    exe = tmp_path / "host_driver"
    r = subprocess.run([HIPCC, "-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
                        *objs, "-o", str(exe)], capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-4000:]
    env = dict(os.environ)
    # The sanitizer runtime need not come first when the environment preloads a library.
    env["ASAN_OPTIONS"] = "verify_asan_link_order=0:detect_leaks=1:abort_on_error=0"
    env["UBSAN_OPTIONS"] = "print_stacktrace=1:halt_on_error=1"
    r = subprocess.run([str(exe)], capture_output=True, text=True, timeout=300, env=env)
    assert r.returncode == 0, (r.stdout + r.stderr)[-4000:]
    assert r.stdout.strip() == "ok"
    assert "runtime error" not in r.stderr and "AddressSanitizer" not in r.stderr, r.stderr[-4000:]
