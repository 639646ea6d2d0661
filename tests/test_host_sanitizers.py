"""Host code under AddressSanitizer and UndefinedBehaviorSanitizer (CPU only).

build.py --sanitize builds a copy of librollout.so whose host code -- the C ABI's argument validation, the
planner, the arena layout and the occupancy controller's metrics and threshold rule -- is instrumented; the
CPU tests of those parts (test_abi_cpu.py, test_occupancy_cpu.py) then run against that copy in a child
process with the sanitizer runtime preloaded.  Any report (out-of-bounds access, use after free, signed
overflow, misaligned or null access, ...) aborts the child and fails this test.  No device code runs."""
import importlib.util
import os
import shutil
import subprocess
import sys

import pytest

from conftest import ROOT

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")


def _build_module():
    spec = importlib.util.spec_from_file_location("_rollout_build_san",
                                                  os.path.join(ROOT, "paper_2608_11226_amd", "build.py"))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


@pytest.mark.skipif(not (shutil.which(HIPCC) or os.path.exists(HIPCC)), reason="needs hipcc to build the library")
def test_host_code_is_clean_under_asan_and_ubsan():
    b = _build_module()
    lib = b.build(verbose=False, sanitize=True)
    runtime = b.sanitizer_runtime()
    assert os.path.exists(runtime), runtime
    syms = subprocess.run(["nm", "-D", lib], capture_output=True, text=True).stdout
    assert "__asan_report" in syms and "__ubsan_handle" in syms, "the host code is not instrumented"
    env = dict(os.environ)
    env.update({
        "LD_PRELOAD": runtime,
        "ASAN_OPTIONS": "detect_leaks=0:abort_on_error=1",
        "UBSAN_OPTIONS": "print_stacktrace=1:halt_on_error=1",
        "ROLLOUT_LIBRARY": lib,
    })
    probe = "import paper_2608_11226_amd as R; print(R.LIB_PATH)"
    res = subprocess.run([sys.executable, "-c", probe], cwd=ROOT, env=env, capture_output=True, text=True)
    assert res.returncode == 0 and res.stdout.strip() == lib, res.stderr[-2000:]
    res = subprocess.run([sys.executable, "-m", "pytest", "-q", "-x", "-p", "no:cacheprovider",
                          "tests/test_abi_cpu.py", "tests/test_occupancy_cpu.py"],
                         cwd=ROOT, env=env, capture_output=True, text=True, timeout=600)
    out = res.stdout[-3000:] + res.stderr[-3000:]
    assert res.returncode == 0, out
    assert "ERROR: AddressSanitizer" not in out and "runtime error:" not in out, out
    assert " passed" in res.stdout
