"""The C ABI's host code under AddressSanitizer and UndefinedBehaviorSanitizer (CPU only).

The library's host translation unit (mca_api.cpp) and a driver of argument checks
(sanitize/abi_checks.cpp) are compiled with the sanitizers on the host side only; the HIP
kernel sources are compiled as in the product build. The driver's calls all return before any
device work, so it runs without a GPU; a sanitizer report aborts it with a non-zero status."""
import os
import shutil
import subprocess

import pytest

from paper_2201_12854_amd import build_lib

HERE = os.path.dirname(os.path.abspath(__file__))


def test_abi_checks_under_host_sanitizers(tmp_path):
    hipcc = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    if not os.path.exists(hipcc):
        pytest.skip("hipcc not available")
    san = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
           "-Xarch_host", "-fno-sanitize-recover=all", "-Xarch_host", "-fno-omit-frame-pointer", "-g"]
    def compile_(src_path, obj, extra):
        cmd = [hipcc, *build_lib.CXXFLAGS, *extra, "-x", "hip", "-c", src_path, "-o", obj]
        r = subprocess.run(cmd, capture_output=True, text=True)
        assert r.returncode == 0, r.stderr[-3000:]
        return obj

    objs = []
    for src in build_lib.SOURCES:
        path = os.path.join(build_lib.CSRC, src)
        if src.endswith(".cpp"):  # the host code under test, with the sanitizers
            objs.append(compile_(path, str(tmp_path / (src + ".o")), san))
            continue
        # kernel sources: the product build's object when it is newer than the source
        built = os.path.join(build_lib.BUILD, src + ".o")
        headers = [os.path.join(build_lib.CSRC, h) for h in ("mca_device.h", "mca_kernels.h")]
        fresh = os.path.exists(built) and all(os.path.getmtime(built) >= os.path.getmtime(f) for f in [path, *headers])
        objs.append(built if fresh else compile_(path, str(tmp_path / (src + ".o")), []))
    drv = compile_(os.path.join(HERE, "sanitize", "abi_checks.cpp"), str(tmp_path / "abi_checks.o"),
                   [*san, "-I", os.path.join(build_lib.ROOT, "include")])
    exe = str(tmp_path / "abi_checks")
    r = subprocess.run([hipcc, f"--offload-arch={build_lib.ARCH}", *san, drv, *objs, "-o", exe],
                       capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-3000:]
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=0:halt_on_error=1:abort_on_error=0",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1", HIP_VISIBLE_DEVICES="")
    r = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=120)
    out = r.stdout + r.stderr
    assert r.returncode == 0, out[-3000:]
    assert "runtime error" not in out and "AddressSanitizer" not in out, out[-3000:]
    assert "all ABI checks passed" in out
