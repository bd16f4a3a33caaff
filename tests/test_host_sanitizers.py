"""The C ABI's host code under AddressSanitizer and UndefinedBehaviorSanitizer.

arckv_host.cpp (validation, workspace planning, budgets, timing) and a driver
that calls every entry point with invalid arguments (tests/sanitize/host_checks.cpp)
are compiled with the sanitizers on the host side only and linked with the
library's kernel objects as built by paper_2609_36835_amd.build; no GPU is
touched (every case fails validation before any HIP call)."""
import os
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
PKG = os.path.join(ROOT, "paper_2609_36835_amd")
BUILD = os.path.join(PKG, "_build")
OUT = os.path.join(BUILD, "sanitize")
HOST_SAN = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
            "-Xarch_host", "-fno-sanitize-recover=undefined", "-fno-omit-frame-pointer", "-g", "-O1"]


def _kernel_objects():
    if not os.path.isdir(BUILD):
        return []
    return sorted(os.path.join(BUILD, f) for f in os.listdir(BUILD) if f.endswith(".hip.o"))


def test_host_code_under_address_and_undefined_sanitizers():
    from paper_2609_36835_amd import build as B
    objs = _kernel_objects()
    if not objs:
        pytest.skip("kernel objects not built (run paper_2609_36835_amd.build first)")
    hipcc = B._hipcc()
    os.makedirs(OUT, exist_ok=True)
    inc = ["-I", os.path.join(ROOT, "include"), "-I", os.path.join(PKG, "csrc")]
    host_o = os.path.join(OUT, "arckv_host_san.o")
    drv_o = os.path.join(OUT, "host_checks.o")
    exe = os.path.join(OUT, "host_checks")
    steps = [
        [hipcc, "-std=c++17", "-fPIC", *HOST_SAN, *inc, "-c", os.path.join(PKG, "csrc", "arckv_host.cpp"), "-o", host_o],
        [hipcc, "-std=c++17", *HOST_SAN, *inc, "-c", os.path.join(ROOT, "tests", "sanitize", "host_checks.cpp"),
         "-o", drv_o],
        [hipcc, f"--offload-arch={B.ARCH}", *HOST_SAN, drv_o, host_o, *objs, "-o", exe],
    ]
    for cmd in steps:
        r = subprocess.run(cmd, capture_output=True, text=True)
        assert r.returncode == 0, (" ".join(cmd), r.stderr[-4000:])
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=0:halt_on_error=1",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1", HIP_VISIBLE_DEVICES="")
    r = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=120)
    print(r.stdout[-2000:])
    assert r.returncode == 0, (r.stdout[-4000:], r.stderr[-4000:])
    assert "ok: 0 failures" in r.stdout
