"""CPU test of the forward's per-CU item-list planner (host code in
paper_2609_36757_amd/csrc/item_lists.h): built with g++ into a small checker
(tests/item_lists_check.cpp) that verifies the lists item by item."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.mark.skipif(shutil.which("g++") is None, reason="needs g++")
def test_item_list_planner(tmp_path):
    exe = tmp_path / "item_lists_check"
    subprocess.run(["g++", "-std=c++17", "-O1", "-Wall", "-Werror", "-I",
                    os.path.join(ROOT, "paper_2609_36757_amd", "csrc"),
                    os.path.join(ROOT, "tests", "item_lists_check.cpp"), "-o", str(exe)], check=True, timeout=300)
    r = subprocess.run([str(exe)], capture_output=True, text=True, timeout=300)
    assert r.returncode == 0, r.stdout[-2000:] + r.stderr[-2000:]
    assert "all " in r.stdout and "cases ok" in r.stdout
    # the 480p-shaped call gets lists, and they are at least 3% shorter than dispatch
    first = r.stdout.splitlines()[0].split()
    assert first[first.index("lists") + 1] == "1"
    planned, dispatch = int(first[first.index("planned") + 1]), int(first[first.index("dispatch") + 1])
    assert 100 * planned <= 97 * dispatch
