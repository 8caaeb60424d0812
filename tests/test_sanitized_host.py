"""The host half of the library under AddressSanitizer and UndefinedBehaviorSanitizer (no GPU).

The block manager, planner, search controller and C entry points are compiled with g++
-fsanitize=address,undefined and linked with host-only stand-ins for the device entry points
(tests/sanitize/host_stubs.cpp: every device call fails with TKV_EHIP).  The block-manager, planner,
controller and ABI tests then run against that library in a child process with the ASan runtime
preloaded; any sanitizer report fails the test.
"""
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2609_39334_amd", "csrc")
HOST_SOURCES = ["capi.cpp", "bm.cpp", "plan.cpp", "search.cpp"]
SUITES = ["test_bm_parity.py", "test_bm_errors.py", "test_plan.py", "test_plan_update.py", "test_search_parity.py",
          "test_abi.py"]


def _runtime(name):
    path = subprocess.run(["g++", f"-print-file-name={name}"], capture_output=True, text=True).stdout.strip()
    return path if os.path.isabs(path) and os.path.exists(path) else None


@pytest.mark.timeout(900)
def test_host_library_under_asan_and_ubsan(tmp_path):
    asan = _runtime("libasan.so")
    if shutil.which("g++") is None or asan is None or _runtime("libubsan.so") is None:
        pytest.skip("g++ with the ASan/UBSan runtimes is not available")
    lib = tmp_path / "libtreekv_sanitized.so"
    cmd = ["g++", "-std=c++17", "-O1", "-g", "-fPIC", "-shared", "-fvisibility=hidden",
           "-fsanitize=address,undefined", "-fno-sanitize-recover=undefined", "-fno-omit-frame-pointer",
           "-I", CSRC, "-I", os.path.join(ROOT, "include"),
           *[os.path.join(CSRC, s) for s in HOST_SOURCES],
           os.path.join(ROOT, "tests", "sanitize", "host_stubs.cpp"), "-o", str(lib)]
    build = subprocess.run(cmd, capture_output=True, text=True)
    assert build.returncode == 0, build.stdout + build.stderr
    driver = (
        "import sys\n"
        f"sys.path.insert(0, {os.path.join(ROOT, 'tests')!r}); sys.path.insert(0, {ROOT!r})\n"
        "import paper_2609_39334_amd as tkv\n"
        f"tkv.LIB_PATH = {str(lib)!r}\n"
        "import pytest\n"
        "sys.exit(pytest.main(['-x', '-q', '-m', 'not gpu', '-p', 'no:cacheprovider', "
        + ", ".join(repr(os.path.join(ROOT, "tests", s)) for s in SUITES) + "]))\n")
    env = dict(os.environ, LD_PRELOAD=asan, ASAN_OPTIONS="detect_leaks=0:halt_on_error=1",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    run = subprocess.run([sys.executable, "-c", driver], capture_output=True, text=True, env=env, cwd=str(tmp_path))
    out = run.stdout + run.stderr
    print(out[-3000:])
    assert "ERROR: AddressSanitizer" not in out and "runtime error:" not in out
    assert run.returncode == 0, out[-3000:]
    assert " passed" in out
