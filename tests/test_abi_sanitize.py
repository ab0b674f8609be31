"""The library's host-side argument validation under AddressSanitizer and
UndefinedBehaviorSanitizer.  Every HIP source is built with the sanitizers on
its host pass only (each -fsanitize= behind -Xarch_host; the device code is
the ordinary gfx950 build), linked with a C++ driver (abi_sanitize_driver.cpp)
that calls every entry point with invalid arguments, and run on the CPU: each
call must return its error code before any device work, with no sanitizer
report.  Nothing here launches a kernel."""
import glob
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
HOST_SAN = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
            "-Xarch_host", "-fno-sanitize-recover=all", "-Xarch_host", "-fno-omit-frame-pointer"]


@pytest.mark.slow
def test_host_validation_runs_clean_under_asan_and_ubsan(tmp_path):
    if not os.path.exists(HIPCC):
        pytest.skip("hipcc not available")
    srcs = sorted(glob.glob(os.path.join(ROOT, "paper_2411_03171_amd", "csrc", "*.hip")))
    common = [HIPCC, "-std=c++17", "-O1", "-g", "--offload-arch=gfx950", "-Xclang", "-target-feature",
              "-Xclang", "-packed-fp32-ops", "-I", os.path.join(ROOT, "include")] + HOST_SAN
    objs, procs = [], []
    jobs = max(1, min(len(srcs), int(os.environ.get("MAX_JOBS", "8"))))
    for src in srcs:
        obj = str(tmp_path / (os.path.basename(src) + ".o"))
        objs.append(obj)
        procs.append(subprocess.Popen(common + ["-c", "-o", obj, src], stdout=subprocess.DEVNULL,
                                      stderr=subprocess.PIPE))
        while len([p for p in procs if p.poll() is None]) >= jobs:
            procs[[p.poll() is None for p in procs].index(True)].wait()
    for p in procs:
        _, err = p.communicate()
        assert p.returncode == 0, err.decode()[-2000:]
    drv = str(tmp_path / "driver.o")
    subprocess.check_call(common + ["-c", "-o", drv, os.path.join(ROOT, "tests", "abi_sanitize_driver.cpp")],
                          stdout=subprocess.DEVNULL)
    exe = str(tmp_path / "abi_sanitized")
    subprocess.check_call([HIPCC, "--offload-arch=gfx950"] + HOST_SAN + ["-o", exe, drv] + objs,
                          stdout=subprocess.DEVNULL)
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=1",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    r = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=300)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "0 failures" in r.stdout, r.stdout
    assert "runtime error" not in r.stderr and "AddressSanitizer" not in r.stderr, r.stderr
