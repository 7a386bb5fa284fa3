"""The library's host-side descriptor validation built with AddressSanitizer
and UndefinedBehaviorSanitizer (host code only; the kernels are the
already-built objects, untouched) and driven through valid, invalid,
aliasing, in-place, empty and large groups (tests/validate_sanitize_driver.cpp):
the expected status for each, and no invalid access, leak or undefined
behaviour. Runs on the CPU; no HIP call is made."""
import glob
import os
import shutil
import subprocess

import pytest

from paper_2607_02945_amd import build as pb

HERE = os.path.dirname(os.path.abspath(__file__))
CLANG = "/opt/rocm/llvm/bin/clang++"
KERNEL_OBJS = sorted(glob.glob(os.path.join(pb.OBJDIR, "kernels_*.o")))


@pytest.mark.skipif(not (os.path.exists(pb.HIPCC) and os.path.exists(CLANG)), reason="ROCm compilers not found")
@pytest.mark.skipif(len(KERNEL_OBJS) != len(pb.SOURCES) - 1, reason="kernel objects not built")
def test_validation_under_sanitizers(tmp_path):
    san = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
           "-Xarch_host", "-fno-omit-frame-pointer"]
    flags = [f for f in pb.FLAGS if f not in ("-O3",)]
    api = str(tmp_path / "api.o")
    subprocess.run([pb.HIPCC, "-O1", "-g", *flags, *san, "-c", os.path.join(pb.CSRC, "optimus_api.hip"), "-o", api],
                   check=True, capture_output=True)
    drv = str(tmp_path / "driver.o")
    host_san = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer"]
    subprocess.run([CLANG, "-O1", "-g", "-std=c++17", *host_san, f"-I{pb.INCLUDE}", "-c",
                    os.path.join(HERE, "validate_sanitize_driver.cpp"), "-o", drv], check=True)
    exe = str(tmp_path / "validate_sanitized")
    subprocess.run([CLANG, *host_san, drv, api, *KERNEL_OBJS, "-L/opt/rocm/lib", "-lamdhip64",
                    "-Wl,-rpath,/opt/rocm/lib", "-o", exe], check=True)
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1", UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    r = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=300)
    assert r.returncode == 0, r.stdout[-2000:] + r.stderr[-6000:]
    assert "runtime error" not in r.stderr and "Sanitizer" not in r.stderr, r.stderr[-6000:]
    assert "ok" in r.stdout
