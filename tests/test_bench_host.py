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


def test_clock_summary_keeps_refreshes_under_load():
    """bench.py's clock sampler reports only firmware refreshes taken under load
    (activity >= 50%), one entry per distinct refresh, mean over the XCDs."""
    import itertools
    import types

    import bench

    seq = itertools.cycle([
        {"current_gfxclks": [900, 900], "average_gfx_activity": 3, "current_socket_power": 280},
        {"current_gfxclks": [1700, 1800], "average_gfx_activity": 100, "current_socket_power": 1390},
        {"current_gfxclks": [1700, 1800], "average_gfx_activity": 100, "current_socket_power": 1390},
        {"current_gfxclks": [1600, 1600], "average_gfx_activity": 99, "current_socket_power": 1400},
    ])
    fake_smi = types.SimpleNamespace(amdsmi_get_gpu_metrics_info=lambda h: next(seq))
    fake_torch = types.SimpleNamespace(cuda=types.SimpleNamespace(synchronize=lambda: None))
    cs = bench.ClockSampler.__new__(bench.ClockSampler)
    cs.period_s, cs.handle, cs.reason, cs.samples, cs.amdsmi = 0.001, object(), None, [], fake_smi
    cs._stop = cs._thread = None
    r = cs.measure(fake_torch, lambda: None, seconds=0.05, settle=0.0)
    assert r["source"] is not None and r["refreshes"] >= 2
    assert r["gfxclk_mhz_min"] == 1600 and r["gfxclk_mhz_max"] == 1750
    assert 1600 <= r["gfxclk_mhz_mean"] <= 1750
    # refreshes before the settle time are dropped (here: all of them)
    cs.samples = []
    r = cs.measure(fake_torch, lambda: None, seconds=0.02, settle=10.0)
    assert r["source"] is None
    cs2 = bench.ClockSampler.__new__(bench.ClockSampler)
    cs2.handle, cs2.reason = None, "amdsmi unavailable"
    assert cs2.measure(fake_torch, lambda: None)["source"] is None


def test_cpu_baseline_reports_every_configuration():
    """bench.py's oracle baseline on a small sample of the tiny workload: the
    rate, the sample's wall time and the per-configuration extrapolation, which
    scales with the dense work B * H * Nq * Nkv * d of each configuration."""
    import bench
    from paper_2609_36757_amd.workloads import WORKLOADS, make_sequence

    w = WORKLOADS["tiny"]
    q, k, v = make_sequence(w)
    r = bench.cpu_baseline(w, q, k, v, budget_rows=64, seed=1)
    assert r["kind"] == "oracle" and r["value"] > 0 and r["wall_s_sample"] >= 0
    per = r["wall_s_per_config_extrapolated"]
    assert set(per) == set(WORKLOADS)
    dense = {n: c.B * c.H * (c.chunk_len if c.stream_chunk is not None else c.n_tokens) * c.n_tokens * c.d
             for n, c in WORKLOADS.items()}
    # ratios of the extrapolated times follow the dense work (up to the rounding to 0.01 s)
    assert per["wide_sw"] > per["1080p"] > per["1080p_stream"] > per["480p"] >= per["tiny"]
    assert abs(per["wide_sw"] / per["1080p"] - dense["wide_sw"] / dense["1080p"]) < 0.05 * dense["wide_sw"] / dense["1080p"]
