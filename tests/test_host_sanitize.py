"""The C-ABI host layer (argument validation, workspace layout and launch
sequencing of jacap_host.hip) built for the CPU with AddressSanitizer and
UndefinedBehaviorSanitizer and driven through every entry point
(tests/sanitize/host_driver.cpp) against host-only stand-ins for the kernel
launchers (tests/sanitize/launch_stubs.cpp). No GPU is used: only host code is
instrumented; device pointers are opaque values the stand-ins never touch."""

import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
CLANG = "/opt/rocm/llvm/bin/clang++"
SAN = os.path.join(ROOT, "tests", "sanitize")
CSRC = os.path.join(ROOT, "paper_2609_08131_amd", "csrc")


@pytest.mark.skipif(not (os.path.exists(HIPCC) and os.path.exists(CLANG)), reason="no ROCm toolchain")
def test_host_layer_under_asan_ubsan(tmp_path):
    # host-only compilation; the sanitizers apply to host code only
    flags = ["-O1", "-g", "-std=c++17", "--offload-host-only", "-x", "hip",
             "-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
             "-Xarch_host", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer",
             f"-I{os.path.join(ROOT, 'include')}", f"-I{CSRC}", f"-I{SAN}"]
    objs = []
    for src in (os.path.join(CSRC, "jacap_host.hip"), os.path.join(SAN, "launch_stubs.cpp"),
                os.path.join(SAN, "host_driver.cpp")):
        obj = str(tmp_path / (os.path.basename(src) + ".o"))
        r = subprocess.run([HIPCC, *flags, "-c", src, "-o", obj], capture_output=True, text=True)
        assert r.returncode == 0, r.stdout + r.stderr
        objs.append(obj)
    exe = str(tmp_path / "host_check")
    r = subprocess.run([CLANG, "-fsanitize=address,undefined", "-fno-sanitize-recover=all", *objs,
                        "-o", exe], capture_output=True, text=True)
    assert r.returncode == 0, r.stdout + r.stderr
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0",
               UBSAN_OPTIONS="print_stacktrace=1")
    r = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=120)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "host layer ok under the sanitizers" in r.stdout
    assert "runtime error" not in r.stderr and "AddressSanitizer" not in r.stderr
