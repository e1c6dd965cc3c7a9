"""Host code of the library under AddressSanitizer (CPU only, opt-in).

Builds every HIP source with the sanitizer on its host code only (device code
is unchanged), links tests/host_planning_check.cpp against the objects and
runs it: random shapes through the planning of every entry point (ragged
tables and launch orders, pyramid schedules, workspace sizes) and the early
argument errors, with leak detection.  Compiling takes a minute or more, so
the test runs only with GRKV_HOST_ASAN=1."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2605_31105_amd", "csrc")
SOURCES = ["attention", "stream", "selection", "merge", "merge_generic", "key", "carrier",
           "frontend", "api"]


@pytest.mark.skipif(os.environ.get("GRKV_HOST_ASAN") != "1", reason="opt-in: GRKV_HOST_ASAN=1")
def test_host_planning_under_asan(tmp_path):
    hipcc = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
    if not os.path.exists(hipcc) or shutil.which("g++") is None:
        pytest.skip("hipcc or g++ missing")
    objs = []
    for src in SOURCES:
        obj = str(tmp_path / (src + ".o"))
        subprocess.run([hipcc, "--offload-arch=gfx950", "-O1", "-g", "-std=c++17", "-fPIC",
                        "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
                        "-Xarch_host", "-fsanitize=address",
                        "-Xarch_host", "-fno-omit-frame-pointer",
                        "-I" + os.path.join(ROOT, "include"), "-I" + CSRC,
                        "-c", os.path.join(CSRC, src + ".hip"), "-o", obj], check=True)
        objs.append(obj)
    drv = str(tmp_path / "drv.o")
    exe = str(tmp_path / "host_planning_check")
    subprocess.run(["g++", "-fsanitize=address", "-fno-omit-frame-pointer", "-g", "-std=c++17",
                    "-I" + os.path.join(ROOT, "include"), "-c",
                    os.path.join(ROOT, "tests", "host_planning_check.cpp"), "-o", drv], check=True)
    subprocess.run(["g++", "-fsanitize=address", drv, *objs, "-L/opt/rocm/lib", "-lamdhip64",
                    "-Wl,-rpath,/opt/rocm/lib", "-o", exe], check=True)
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1")
    r = subprocess.run([exe], env=env, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True,
                       timeout=600)
    print(r.stdout[-2000:])
    assert r.returncode == 0 and "bad = 0" in r.stdout
