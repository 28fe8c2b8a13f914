"""The host layer under AddressSanitizer and UndefinedBehaviorSanitizer (CPU).

The C-ABI layer (fastvr_api.cpp) and the host geometry (geometry.cpp) are built
with g++ -fsanitize=address,undefined into a host-only library whose kernel
launchers are stand-ins that launch nothing (tests/host_stubs.cpp).  Every
validation case of tests/test_abi.py then runs against it in a child Python
process with the sanitizer runtime preloaded, together with valid calls that
pass all checks and reach the launchers; any sanitizer report aborts the child.
The per-CU item-list planner (item_lists.h) runs its own checker
(tests/item_lists_check.cpp: the 480p shape, the plan cache and 400 seeded
shapes) under the same sanitizers."""
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2609_36757_amd", "csrc")
SAN = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer", "-g", "-O1"]
ENV_SAN = {"ASAN_OPTIONS": "detect_leaks=0:abort_on_error=1:halt_on_error=1",
           "UBSAN_OPTIONS": "halt_on_error=1:print_stacktrace=1"}

pytestmark = pytest.mark.skipif(shutil.which("g++") is None or not os.path.isdir("/opt/rocm/include"),
                                reason="needs g++ and the ROCm headers")


def _asan_runtime():
    r = subprocess.run(["g++", "-print-file-name=libasan.so"], capture_output=True, text=True)
    path = r.stdout.strip()
    if r.returncode != 0 or not os.path.isabs(path) or not os.path.exists(path):
        pytest.skip("g++ has no AddressSanitizer runtime")
    return path


def test_c_abi_layer_under_sanitizers(tmp_path):
    lib = str(tmp_path / "libfastvr_hostcheck.so")
    subprocess.run(["g++", "-std=c++17", "-shared", "-fPIC", *SAN, "-D__HIP_PLATFORM_AMD__", "-I/opt/rocm/include",
                    "-I", os.path.join(ROOT, "include"), "-I", CSRC, os.path.join(CSRC, "fastvr_api.cpp"),
                    os.path.join(CSRC, "geometry.cpp"), os.path.join(ROOT, "tests", "host_stubs.cpp"), "-o", lib],
                   check=True, timeout=300)
    env = dict(os.environ, LD_PRELOAD=_asan_runtime(), **ENV_SAN)
    driver = ("import sys, pytest\n"
              "from paper_2609_36757_amd import fastvr\n"
              "fastvr.LIB_PATH = sys.argv[1]\n"
              "sys.exit(pytest.main(['-q', '-p', 'no:cacheprovider', '-x', sys.argv[2], '-k',\n"
              "    'not c_client and not input_generator and not workload_registry']))\n")
    r = subprocess.run([sys.executable, "-c", driver, lib, os.path.join(ROOT, "tests", "test_abi.py")], cwd=ROOT,
                       env=env, capture_output=True, text=True, timeout=600)
    out = r.stdout[-3000:] + r.stderr[-3000:]
    assert r.returncode == 0, out
    assert "ERROR: AddressSanitizer" not in out and "runtime error" not in out, out
    assert " passed" in r.stdout and "skipped" not in r.stdout.splitlines()[-1], out


def test_item_list_planner_under_sanitizers(tmp_path):
    exe = str(tmp_path / "item_lists_check_san")
    subprocess.run(["g++", "-std=c++17", *SAN, "-Wall", "-Werror", "-I", CSRC,
                    os.path.join(ROOT, "tests", "item_lists_check.cpp"), "-o", exe], check=True, timeout=300)
    r = subprocess.run([exe], capture_output=True, text=True, timeout=600, env=dict(os.environ, **ENV_SAN))
    assert r.returncode == 0, r.stdout[-2000:] + r.stderr[-2000:]
    assert "cases ok" in r.stdout and "runtime error" not in r.stderr, r.stderr[-2000:]
