"""The library's host code under AddressSanitizer and UndefinedBehaviorSanitizer.

Every source of liblst is compiled with the sanitizers on its host side only (device code
as usual, -O1) and linked into tests/host/plan_check.cpp, a host program that exercises
the argument and workspace validation of the C ABI and checks the step's product
descriptors for several hundred shapes against the carved buffers (see that file).  No GPU
is used: every call it makes returns before any device work.
"""
import concurrent.futures as cf
import glob
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_1606_08061_amd", "csrc")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
SAN = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
       "-Xarch_host", "-fno-sanitize-recover=all", "-Xarch_host", "-fno-omit-frame-pointer"]
FLAGS = ["-O1", "-g", "-std=c++17", "--offload-arch=gfx950", "-Xarch_device", "-O1",
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
         "-I", os.path.join(ROOT, "include"), "-I", CSRC]


def _compile(src, out, extra=()):
    r = subprocess.run([HIPCC, *FLAGS, *SAN, *extra, "-c", src, "-o", out],
                       capture_output=True, text=True, timeout=600)
    assert r.returncode == 0, r.stderr[-4000:]
    return out


@pytest.mark.skipif(shutil.which(HIPCC) is None and not os.path.exists(HIPCC),
                    reason="hipcc not available")
def test_host_code_under_sanitizers(tmp_path):
    srcs = sorted(glob.glob(os.path.join(CSRC, "*.hip")))
    with cf.ThreadPoolExecutor(max_workers=min(8, os.cpu_count() or 1)) as ex:
        futs = [ex.submit(_compile, s, str(tmp_path / (os.path.basename(s) + ".o"))) for s in srcs]
        futs.append(ex.submit(_compile, os.path.join(ROOT, "tests", "host", "plan_check.cpp"),
                              str(tmp_path / "plan_check.o"), ("-x", "hip")))
        objs = [f.result() for f in futs]
    exe = str(tmp_path / "plan_check")
    r = subprocess.run([HIPCC, "-fsanitize=address,undefined", *objs, "-o", exe],
                       capture_output=True, text=True, timeout=600)
    assert r.returncode == 0, r.stderr[-4000:]
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=0:abort_on_error=1",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    r = subprocess.run([exe], capture_output=True, text=True, timeout=600, env=env)
    assert r.returncode == 0, (r.stdout[-2000:], r.stderr[-6000:])
    assert "all host checks passed" in r.stdout
