"""Host-side parts of bench.py that run without a GPU: the single-GPU guard and
the rule that the reported HBM traffic is dropped once the forward kernel's
source no longer matches the one the counters were taken on."""
import importlib.util
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _load_bench():
    spec = importlib.util.spec_from_file_location("bench_under_test", os.path.join(ROOT, "bench.py"))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


@pytest.mark.parametrize("argv,env", [(["--gpus", "2"], {}), (["--gpus", "8"], {}), ([], {"WORLD_SIZE": "4"})])
def test_more_than_one_gpu_is_refused(argv, env):
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py")] + argv, cwd=ROOT,
                       env={**os.environ, **env}, capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    assert r.stdout == ""


def _summary(path, sha, nbytes):
    path.write_text(f"# traffic\n\nkernel_source_sha256_16: {sha}\nhbm_bytes_per_launch: {nbytes}\n")


def test_traffic_follows_the_kernel_source(tmp_path, monkeypatch):
    bench = _load_bench()
    summary = tmp_path / "traffic.md"
    monkeypatch.setattr(bench, "TRAFFIC_SUMMARY", str(summary))
    assert bench.read_traffic() is None                      # no summary
    _summary(summary, bench.kernel_source_hash(), 2.63e9)
    assert bench.read_traffic() == pytest.approx(2.63e9)     # taken on this source
    _summary(summary, "0" * 16, 2.63e9)
    assert bench.read_traffic() is None                      # taken on another source
    summary.write_text("no figures here\n")
    assert bench.read_traffic() is None


def test_source_hash_tracks_the_file(tmp_path, monkeypatch):
    bench = _load_bench()
    src = tmp_path / "k.hip"
    src.write_text("kernel A\n")
    monkeypatch.setattr(bench, "KERNEL_SOURCE", str(src))
    h1 = bench.kernel_source_hash()
    src.write_text("kernel B\n")
    assert bench.kernel_source_hash() != h1
    assert len(h1) == 16 and all(c in "0123456789abcdef" for c in h1)
