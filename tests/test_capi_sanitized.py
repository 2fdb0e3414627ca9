"""The C ABI's host code (csrc/capi.hip) under AddressSanitizer and UBSan.

tests/host_check/capi_host_check.cpp links capi.hip's host object against
stubs of the HIP runtime and of the kernel launchers, with fake device
address ranges: every entry point runs its host logic (validation, workspace
carving, launch sequences, tracing, paging plan, error and release paths)
without a GPU, each launcher checks that its buffers lie inside what the
caller passed, and a launch failure is injected at every position of the
precomputes. Sanitizers apply to host code only (-Xarch_host on the hipcc
line; the driver is plain C++ built with clang++).
"""

import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HIPCC = "/opt/rocm/bin/hipcc"
CLANG = "/opt/rocm/llvm/bin/clang++"


@pytest.mark.skipif(not (os.path.exists(HIPCC) and os.path.exists(CLANG)), reason="ROCm compilers not found")
def test_capi_host_paths_under_asan_and_ubsan(tmp_path):
    capi = os.path.join(ROOT, "paper_2107_03356_amd", "csrc", "capi.hip")
    drv = os.path.join(ROOT, "tests", "host_check", "capi_host_check.cpp")
    san = ["-fsanitize=address", "-fsanitize=undefined", "-fno-sanitize-recover=undefined"]
    host_san = [a for f in san for a in ("-Xarch_host", f)]
    common = ["-std=c++17", "-O1", "-g", "-fno-omit-frame-pointer"]
    cmds = [
        [HIPCC, *common, "--offload-arch=gfx950", "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
         *host_san, "-c", capi, "-o", str(tmp_path / "capi.o")],
        [CLANG, *common, *san, "-I/opt/rocm/include", "-D__HIP_PLATFORM_AMD__", "-c", drv,
         "-o", str(tmp_path / "check.o")],
        [CLANG, *san, str(tmp_path / "capi.o"), str(tmp_path / "check.o"), "-o", str(tmp_path / "check")],
    ]
    for c in cmds:
        r = subprocess.run(c, capture_output=True, text=True)
        assert r.returncode == 0, (" ".join(c), r.stderr[-4000:])
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    r = subprocess.run([str(tmp_path / "check")], capture_output=True, text=True, env=env, timeout=300)
    out = r.stdout + r.stderr
    assert r.returncode == 0, out[-6000:]
    assert "host check ok" in r.stdout, out[-6000:]
    assert "AddressSanitizer" not in out and "runtime error" not in out, out[-6000:]
