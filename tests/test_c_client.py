"""The boundary from plain C: tests/c_abi_check.c compiles as C99 against include/treekv.h (warnings
as errors), links against the built libtreekv.so and runs its host-only checks (no GPU)."""
import os
import shutil
import subprocess

import pytest

import paper_2609_39334_amd as tkv

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.mark.skipif(shutil.which("gcc") is None, reason="no C compiler")
def test_c99_client(tmp_path):
    tkv.lib()                                             # raises if the library is not built
    exe = tmp_path / "c_abi_check"
    rocm_lib = os.path.join(os.environ.get("ROCM_PATH", "/opt/rocm"), "lib")
    pkg = os.path.dirname(tkv.LIB_PATH)
    cmd = ["gcc", "-std=c99", "-Wall", "-Wextra", "-pedantic", "-Werror", "-I", os.path.join(ROOT, "include"),
           os.path.join(ROOT, "tests", "c_abi_check.c"), "-o", str(exe), tkv.LIB_PATH,
           f"-Wl,-rpath,{pkg}", f"-Wl,-rpath-link,{rocm_lib}", f"-Wl,-rpath,{rocm_lib}"]
    subprocess.run(cmd, check=True, capture_output=True, text=True)
    out = subprocess.run([str(exe)], capture_output=True, text=True, timeout=60)
    assert out.returncode == 0 and out.stdout.strip() == "ok", out.stderr
