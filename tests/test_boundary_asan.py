"""The boundary tests again, against the C-ABI layer built for the host with AddressSanitizer
and UndefinedBehaviorSanitizer (g++, host code only; the kernel launchers are stubs that
abort if reached).  An out-of-bounds write in argument validation (such as overrunning the
table of state-tensor ranges) then fails here instead of corrupting the caller's stack."""
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2606_22932_amd", "csrc")


def _libasan():
    out = subprocess.run(["g++", "-print-file-name=libasan.so"], capture_output=True, text=True).stdout.strip()
    return out if os.path.isabs(out) and os.path.exists(out) else None


@pytest.mark.skipif(shutil.which("g++") is None or _libasan() is None, reason="g++ with AddressSanitizer needed")
def test_boundary_suite_under_address_sanitizer(tmp_path):
    lib = str(tmp_path / "libforge_asan.so")
    build = ["g++", "-std=c++17", "-O1", "-g", "-fPIC", "-shared", "-fsanitize=address,undefined",
             "-fno-omit-frame-pointer", "-fno-sanitize-recover=undefined", "-D__HIP_PLATFORM_AMD__",
             "-I", os.path.join(ROOT, "include"), "-I", CSRC, "-I", "/opt/rocm/include",
             os.path.join(CSRC, "forge_api.cpp"), os.path.join(ROOT, "tests", "asan", "launch_stubs.cpp"),
             "-L", "/opt/rocm/lib", "-lamdhip64", "-Wl,-rpath,/opt/rocm/lib", "-o", lib]
    r = subprocess.run(build, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-3000:]
    runner = (
        "import sys, pytest\n"
        "import paper_2606_22932_amd.build as b\n"
        f"b.LIB = {lib!r}\n"
        "sys.exit(pytest.main(['-q', '-s', '-p', 'no:cacheprovider', '-k', 'not query_tile and not status_strings',"
        f" {os.path.join(ROOT, 'tests', 'test_boundary.py')!r}]))\n")
    env = dict(os.environ, LD_PRELOAD=_libasan(), ASAN_OPTIONS="detect_leaks=0:abort_on_error=1",
               UBSAN_OPTIONS="print_stacktrace=1", HIP_VISIBLE_DEVICES="-1", PYTHONPATH=ROOT)
    r = subprocess.run([sys.executable, "-c", runner], cwd=ROOT, env=env, capture_output=True, text=True, timeout=600)
    assert r.returncode == 0, (r.stdout[-3000:] + r.stderr[-3000:])
