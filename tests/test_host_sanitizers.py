"""The library's host code (argument checks, split planning, workspace sizing)
under AddressSanitizer and UndefinedBehaviorSanitizer, on the CPU.

Builds every source with the sanitizers applied to the host compilation only
(device code is compiled as usual), links the driver in tests/host_abi_driver.cpp
against it, and runs it. The driver makes only calls that stop at a host-side
check or never launch anything, so it needs no GPU.
"""

import os
import shutil
import subprocess

import pytest

from paper_2608_00531_amd import build as pbuild

HERE = os.path.dirname(os.path.abspath(__file__))
SANITIZE = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
            "-Xarch_host", "-fno-sanitize-recover=undefined", "-Xarch_host",
            "-fno-omit-frame-pointer"]


def _run(cmd, cwd):
    res = subprocess.run(cmd, cwd=cwd, capture_output=True, text=True)
    err = "\n".join(l for l in res.stderr.splitlines() if "packed-fp32-ops" not in l)
    assert res.returncode == 0, "%s\n%s\n%s" % (" ".join(cmd), res.stdout, err)
    return res


@pytest.mark.skipif(not os.path.exists(pbuild.hipcc()), reason="hipcc not available")
def test_host_abi_under_asan_and_ubsan(tmp_path):
    rocm = os.path.dirname(os.path.dirname(pbuild.hipcc()))
    clangxx = os.path.join(rocm, "llvm", "bin", "clang++")
    if not os.path.exists(clangxx):
        pytest.skip("ROCm clang++ not available")
    flags = [f for f in pbuild.HIPCC_FLAGS if f not in ("-shared", "-fPIC")]
    objs = []
    for src in pbuild.SOURCES:
        obj = str(tmp_path / (os.path.basename(src) + ".o"))
        _run([pbuild.hipcc()] + flags + SANITIZE + ["-c", "-I", pbuild.INCLUDE, "-I", pbuild.CSRC,
                                                    os.path.join(pbuild.CSRC, src), "-o", obj],
             str(tmp_path))
        objs.append(obj)
    host_san = ["-fsanitize=address", "-fsanitize=undefined", "-fno-sanitize-recover=undefined"]
    drv = str(tmp_path / "driver.o")
    _run([clangxx, "-O1", "-g", "-std=c++17"] + host_san +
         ["-I", pbuild.INCLUDE, "-c", os.path.join(HERE, "host_abi_driver.cpp"), "-o", drv],
         str(tmp_path))
    exe = str(tmp_path / "host_abi_driver")
    _run([clangxx] + host_san + [drv] + objs +
         ["-L", os.path.join(rocm, "lib"), "-lamdhip64", "-Wl,-rpath," + os.path.join(rocm, "lib"),
          "-o", exe], str(tmp_path))
    env = dict(os.environ)
    # The HIP runtime's own allocations at exit are not this library's leaks.
    env["ASAN_OPTIONS"] = "detect_leaks=0:abort_on_error=0"
    env["UBSAN_OPTIONS"] = "print_stacktrace=1:halt_on_error=1"
    res = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=300)
    out = res.stdout + res.stderr
    assert res.returncode == 0, out
    assert "0 failure(s)" in res.stdout, out
    assert "runtime error" not in out and "AddressSanitizer" not in out, out
