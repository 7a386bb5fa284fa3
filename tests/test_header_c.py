"""The C ABI from plain C: tests/header_c_driver.c compiles as C11 with
-Wall -Wextra -pedantic -Werror against include/optimus.h, links against the
built liboptimus.so, and its host-only calls (version, descriptor
validation: valid, empty, invalid, aliasing, unknown enum value) return the
documented statuses. Runs on the CPU; no HIP call is made."""
import os
import shutil
import subprocess

import pytest

from paper_2607_02945_amd import binding as B
from paper_2607_02945_amd import build as pb

HERE = os.path.dirname(os.path.abspath(__file__))


@pytest.mark.skipif(shutil.which("gcc") is None, reason="gcc not found")
@pytest.mark.skipif(not os.path.exists(B.LIBPATH), reason="liboptimus.so not built")
def test_header_is_c11_and_links_from_c(tmp_path):
    exe = str(tmp_path / "header_c")
    libdir = os.path.dirname(B.LIBPATH)
    subprocess.run(["gcc", "-std=c11", "-Wall", "-Wextra", "-pedantic", "-Werror", f"-I{pb.INCLUDE}",
                    os.path.join(HERE, "header_c_driver.c"), f"-L{libdir}", "-loptimus",
                    f"-Wl,-rpath,{libdir}", "-Wl,-rpath,/opt/rocm/lib", "-o", exe], check=True)
    r = subprocess.run([exe], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, r.stdout + r.stderr
    assert r.stdout.startswith("ok"), r.stdout
