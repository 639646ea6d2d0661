"""Build librollout.so (HIP for gfx950) in-tree.

    python paper_2608_11226_amd/build.py [--jobs N] [--sanitize]

(run by path: importing the package needs the library this script builds)

Every .hip file under csrc/ is compiled with hipcc for gfx950 only, every .cpp
file there (host code) with the same compiler as plain C++, and all are linked
into paper_2608_11226_amd/librollout.so.  Packed-fp32 instructions are turned
off for the device code (the host pass warns that it does not know the
feature; that is harmless).

--sanitize builds a second copy, paper_2608_11226_amd/_build/sanitize/librollout.so,
whose host code (the C ABI, planner, argument validation, block tables and the
occupancy metrics) is instrumented with AddressSanitizer and
UndefinedBehaviorSanitizer; the device code is built as usual.  Loading it
needs the sanitizer runtime preloaded (SANITIZER_RUNTIME below); the binding
loads it in place of the product library when ROLLOUT_LIBRARY names it.
"""
from __future__ import annotations

import argparse
import glob
import os
import shutil
import subprocess
from concurrent.futures import ThreadPoolExecutor

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
BUILD = os.path.join(PKG, "_build")
LIB = os.path.join(PKG, "librollout.so")

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"
FLAGS = [
    f"--offload-arch={ARCH}",
    "-O3",
    "-std=c++17",
    "-fPIC",
    "-Wall",
    "-Wno-unused-function",
    "-Wno-unused-value",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    f"-I{INCLUDE}",
    f"-I{CSRC}",
]


# host-only instrumentation: each sanitizer flag applies to the host pass alone
SANITIZE_FLAGS = [
    "-Xarch_host", "-fsanitize=address",
    "-Xarch_host", "-fsanitize=undefined",
    "-Xarch_host", "-fno-sanitize-recover=undefined",
    "-Xarch_host", "-fno-omit-frame-pointer",
    "-g",
]
SANITIZE_DIR = os.path.join(BUILD, "sanitize")
SANITIZE_LIB = os.path.join(SANITIZE_DIR, "librollout.so")


def sanitizer_runtime() -> str:
    """Path of the compiler's shared AddressSanitizer runtime (to preload before loading SANITIZE_LIB)."""
    res = subprocess.run([HIPCC, "-print-file-name=libclang_rt.asan-x86_64.so"], capture_output=True, text=True)
    return res.stdout.strip()


def _compile(src: str, sanitize: bool = False) -> str:
    out_dir = SANITIZE_DIR if sanitize else BUILD
    obj = os.path.join(out_dir, os.path.basename(src) + ".o")
    cmd = [HIPCC, *FLAGS, *(SANITIZE_FLAGS if sanitize else []), "-c", src, "-o", obj]
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n{res.stderr}")
    # the host pass does not know the packed-fp32 feature; drop that line only
    noise = "is not a recognized feature for this target"
    warn = "\n".join(l for l in res.stderr.splitlines() if noise not in l)
    if warn.strip():
        print(warn)
    return obj


def build(jobs: int | None = None, verbose: bool = True, sanitize: bool = False) -> str:
    """Compile every source and link the shared library; returns its path."""
    if not shutil.which(HIPCC) and not os.path.exists(HIPCC):
        raise RuntimeError("hipcc not found; the HIP library cannot be built")
    out = SANITIZE_LIB if sanitize else LIB
    os.makedirs(SANITIZE_DIR if sanitize else BUILD, exist_ok=True)
    srcs = sorted(glob.glob(os.path.join(CSRC, "*.hip"))) + sorted(glob.glob(os.path.join(CSRC, "*.cpp")))
    jobs = jobs or min(16, os.cpu_count() or 1)
    with ThreadPoolExecutor(jobs) as ex:
        objs = list(ex.map(lambda src: _compile(src, sanitize), srcs))
    tmp = out + ".tmp"
    cmd = [HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, "-o", tmp, "-L/opt/rocm/lib",
           "-lrocprofiler-sdk-roctx", "-Wl,-rpath,/opt/rocm/lib"]
    if sanitize:
        cmd += ["-shared-libsan", *SANITIZE_FLAGS]
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"link failed:\n{res.stderr}")
    os.replace(tmp, out)
    if verbose:
        print(f"built {out} from {len(srcs)} sources")
    return out


if __name__ == "__main__":
    ap = argparse.ArgumentParser()
    ap.add_argument("--jobs", type=int, default=None)
    ap.add_argument("--sanitize", action="store_true", help="host code under ASan + UBSan, built beside the product")
    a = ap.parse_args()
    build(a.jobs, sanitize=a.sanitize)
