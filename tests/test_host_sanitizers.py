"""The host code of the C ABI (validation, planning, workspace layouts of
slim_api.cpp and of the model step) built with AddressSanitizer and
UndefinedBehaviorSanitizer, and driven through every entry point by
tests/host_abi_driver.cpp on the CPU: sizing over a grid of problem
descriptions at the edges of their ranges, and calls that validation must
reject before any device call.  The other translation units are linked as
the regular build compiled them (their host code only launches kernels).
"""

import glob
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
SANITIZED = ("slim_api.cpp", "slim_model.hip")
# host code only: each sanitizer flag applies to the host pass
HOST_SAN = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
            "-Xarch_host", "-fno-sanitize-recover=all"]


def test_host_code_under_sanitizers(tmp_path):
    if not os.path.exists(HIPCC):
        pytest.skip("hipcc not available")
    from paper_2012_11346_amd import build as B

    objs = []
    srcs = B.sources()
    procs = []
    for src in srcs:
        base = os.path.basename(src)
        if base in SANITIZED:
            obj = str(tmp_path / (base + ".san.o"))
            cmd = [HIPCC, *B.CFLAGS, "-O1", "-g", *HOST_SAN, "-x", "hip", "-c", src, "-o", obj, "-I",
                   os.path.join(ROOT, "include")]
            procs.append((src, subprocess.Popen(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)))
        else:
            obj = os.path.join(B.BUILD, base + ".o")
            if not os.path.exists(obj):
                pytest.skip("the regular build's objects are missing (build first)")
        objs.append(obj)
    for src, pr in procs:
        out, _ = pr.communicate(timeout=900)
        assert pr.returncode == 0, f"hipcc failed for {src}:\n{out[-4000:]}"
    drv = str(tmp_path / "driver.o")
    r = subprocess.run([HIPCC, "-O1", "-g", "-std=c++17", *HOST_SAN, "-x", "c++", "-c",
                        os.path.join(ROOT, "tests", "host_abi_driver.cpp"), "-o", drv],
                       capture_output=True, text=True, timeout=300)
    assert r.returncode == 0, r.stdout + r.stderr
    exe = str(tmp_path / "host_abi_driver")
    r = subprocess.run([HIPCC, f"--offload-arch={B.ARCH}", *HOST_SAN, drv, *objs, "-o", exe],
                       capture_output=True, text=True, timeout=300)
    assert r.returncode == 0, r.stdout + r.stderr
    env = dict(os.environ)
    # the HIP runtime keeps allocations until exit; leaks are not what is checked here
    env["ASAN_OPTIONS"] = "detect_leaks=0:abort_on_error=1"
    env["UBSAN_OPTIONS"] = "print_stacktrace=1:halt_on_error=1"
    r = subprocess.run([exe], capture_output=True, text=True, timeout=600, env=env)
    print(r.stdout[-2000:])
    assert r.returncode == 0, (r.stdout + r.stderr)[-6000:]
    assert "0 failures" in r.stdout
