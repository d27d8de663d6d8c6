"""The host runtime under AddressSanitizer and UndefinedBehaviorSanitizer.

The library's sources are compiled with the sanitizers on the host code
only (the device code is built as usual, at -O1), and every argument check
of the C ABI plus
the host-only calls (model import, export, importance, free, options, timing
tallies) are driven through it by tests/sanitizer_driver.py in a process with
the sanitizer runtime preloaded.  Any invalid memory access or undefined
behaviour aborts that process.  No call reaches a device.
"""
import glob
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_1609_06119_amd", "csrc")


def _runtime():
    libs = sorted(glob.glob("/opt/rocm/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so"))
    return libs[-1] if libs else None


def test_argument_checks_and_host_calls_are_clean_under_sanitizers(tmp_path):
    hipcc = "/opt/rocm/bin/hipcc" if os.path.exists("/opt/rocm/bin/hipcc") else shutil.which("hipcc")
    rt = _runtime()
    if not hipcc or not rt:
        pytest.skip("hipcc or the sanitizer runtime is not installed")
    lib = str(tmp_path / "libfbdt_sanitized.so")
    flags = ["--offload-arch=gfx950", "-O1", "-std=c++17", "-fPIC",
             "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
             "-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
             "-Xarch_host", "-fno-sanitize-recover=all", "-Xarch_host", "-fno-omit-frame-pointer",
             "-I", os.path.join(ROOT, "include"), "-I", CSRC]
    objs, procs = [], []
    for f in ("kernels.hip", "quantiles.hip", "capi.hip"):
        o = str(tmp_path / (f + ".o"))
        objs.append(o)
        procs.append(subprocess.Popen([hipcc, *flags, "-c", "-o", o, os.path.join(CSRC, f)],
                                      stdout=subprocess.PIPE, stderr=subprocess.PIPE, text=True))
    for p in procs:
        out, err = p.communicate()
        assert p.returncode == 0, err[-3000:]
    res = subprocess.run([hipcc, "--offload-arch=gfx950", "-shared", "-Xarch_host",
                          "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined", "-o", lib,
                          *objs], capture_output=True, text=True)
    assert res.returncode == 0, res.stderr[-3000:]
    env = dict(os.environ, LD_PRELOAD=rt,
               ASAN_OPTIONS="detect_leaks=0:abort_on_error=1:halt_on_error=1",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    run = subprocess.run([sys.executable, os.path.join(ROOT, "tests", "sanitizer_driver.py"), lib,
                          ROOT], capture_output=True, text=True, env=env, timeout=300)
    assert run.returncode == 0, (run.stdout[-2000:], run.stderr[-4000:])
    assert "checks ok" in run.stdout
