"""The C ABI's host code (argument validation, buffer sizing, weight layout,
KV page planning, the transition-table size checks) under AddressSanitizer
and UndefinedBehaviorSanitizer: tests/abi_sanitize.cpp drives every refusal
path that returns before a kernel launch, linked against the library's
sources with the sanitizers on the host side only.  CPU only."""
import os
import shutil
import subprocess
from concurrent.futures import ThreadPoolExecutor

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2410_13839_amd", "csrc")
OUT = os.path.join(ROOT, "paper_2410_13839_amd", "_build", "sanitize")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
SAN = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
       "-Xarch_host", "-fno-sanitize-recover=undefined", "-fno-omit-frame-pointer"]
FLAGS = ["--offload-arch=gfx950", "-std=c++17", "-O1", "-g", "-Xclang", "-target-feature", "-Xclang",
         "-packed-fp32-ops", *SAN]


def _compile(src):
    obj = os.path.join(OUT, os.path.basename(src) + ".o")
    r = subprocess.run([HIPCC, *FLAGS, "-c", src, "-o", obj], capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-3000:]
    return obj


@pytest.mark.skipif(shutil.which(HIPCC) is None and not os.path.exists(HIPCC), reason="hipcc not available")
def test_abi_host_code_under_asan_and_ubsan():
    os.makedirs(OUT, exist_ok=True)
    build = __import__("paper_2410_13839_amd.build", fromlist=["SOURCES"])
    srcs = [os.path.join(CSRC, s) for s in build.SOURCES] + [os.path.join(ROOT, "tests", "abi_sanitize.cpp")]
    with ThreadPoolExecutor(max_workers=min(8, os.cpu_count() or 1)) as ex:
        objs = list(ex.map(_compile, srcs))
    exe = os.path.join(OUT, "abi_sanitize")
    r = subprocess.run([HIPCC, "--offload-arch=gfx950", *SAN, *objs, "-o", exe], capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-3000:]
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=0:halt_on_error=1:abort_on_error=0",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    r = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=120)
    assert r.returncode == 0 and "abi sanitize ok" in r.stdout, (r.stdout[-2000:], r.stderr[-4000:])
