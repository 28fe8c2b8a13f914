"""Benchmark: chunk-causal attention on the 1080p-shaped latent sequence.

One step = the whole hot path on one batch of synthetic input resident in HBM:
  1. the parallel chunk-causal call over the 1080p sequence (B=1, H=12, d=128,
     4 chunks x 16320 tokens, full causal prefix of chunks);
  2. the streaming step for its last chunk: append chunk 3's K/V to a KV cache
     holding chunks 0-2, then attend chunk 3's queries against the 65280-token
     cache (q_chunk_offset = 3).
value = effective (unmasked) TFLOP/s of the whole step: 4 * d * visible pairs
* B * H for both attention calls, divided by the step time.

After the timed steps (and outside them) it reports ms/call and TFLOP/s of
the 480p-shaped and wide sliding-window calls, of the W = 1 ring-cache
streaming step, of the backward of the 1080p call, of the one-step latent
update, of tiled inference with overlapping 64 x 64 latent tiles and of the
parallel calls with cold caches (``other_workloads``), then the fp64 oracle
baseline.

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME] [--no-extra] [--bwd-only]
                      [--no-cpu-baseline] [--no-clock] [--power-probe]
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2516.6  # MI355X dense bf16 MFMA: 256 CU x 2.4 GHz x 4096 flop/clk
TRAFFIC_SUMMARY = os.path.join(ROOT, "profiles", "chunk_attn_fwd_1080p_hbm_traffic.md")
KERNEL_SOURCE = os.path.join(ROOT, "paper_2609_36757_amd", "csrc", "chunk_attn_fwd.hip")
METRIC = "effective TFLOP/s (unmasked) + ms/chunk, 1080p-shaped chunk-causal attention"


def kernel_source_hash() -> str:
    with open(KERNEL_SOURCE, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()[:16]


def read_traffic():
    """HBM bytes per launch from the committed rocprofv3 counter summary, or None
    when the summary is missing or was taken on a different kernel source."""
    if not os.path.exists(TRAFFIC_SUMMARY):
        return None
    text = open(TRAFFIC_SUMMARY).read()
    h = re.search(r"kernel_source_sha256_16:\s*([0-9a-f]+)", text)
    b = re.search(r"hbm_bytes_per_launch:\s*([0-9.eE+]+)", text)
    if not h or not b or h.group(1) != kernel_source_hash():
        return None
    return float(b.group(1))


def cpu_baseline(w, q, k, v, budget_rows: int, seed: int = 0):
    """Time the fp64 oracle on a bounded, seeded sample of query rows of the
    parallel 1080p call and report the effective TFLOP/s it reaches."""
    import numpy as np

    import oracle
    from paper_2609_36757_amd import metrics

    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info() if i.get("user_api") == "blas"] or [1])
    except Exception:  # threadpoolctl missing: report what the environment asks for
        threads = int(os.environ.get("OMP_NUM_THREADS", os.cpu_count() or 1))
    rng = np.random.default_rng(seed)
    rows = np.sort(rng.choice(w.n_tokens, size=budget_rows, replace=False))
    t0 = time.perf_counter()
    oracle.attention(q, k, v, chunk_len=w.chunk_len, window_chunks=w.window_chunks,
                     scale=float(np.float32(w.scale)), rows=rows)
    dt = time.perf_counter() - t0
    vis = 0
    for r in rows:
        lo, hi = metrics.kv_interval(int(r) // w.chunk_len, w.n_tokens, w.chunk_len, w.window_chunks)
        vis += hi - lo
    flops = 4 * w.d * w.B * w.H * vis
    total = metrics.effective_flops(w.B, w.H, w.d, w.n_tokens, w.n_tokens, w.chunk_len, 0, w.window_chunks)
    # The oracle forms every (query, key) score of a row and then masks, so its
    # time scales with the dense work B * H * Nq * Nkv * d of a call; the other
    # configurations are extrapolated from the sample's rate in that measure.
    from paper_2609_36757_amd.workloads import WORKLOADS
    dense_rate = w.B * w.H * budget_rows * w.n_tokens * w.d / dt
    per_cfg = {}
    for name, c in WORKLOADS.items():
        nq = c.chunk_len if c.stream_chunk is not None else c.n_tokens
        per_cfg[name] = round(c.B * c.H * nq * c.n_tokens * c.d / dense_rate, 2)
    return {"value": flops / dt / 1e12, "unit": "TFLOP/s", "cores": int(threads), "kind": "oracle",
            "sample": f"{budget_rows} seeded random query rows of the parallel 1080p call, all {w.H} heads, "
                      f"{dt:.1f} s wall, fp64 NumPy/BLAS ({threads} BLAS threads, 1 process), host "
                      f"os.cpu_count()={os.cpu_count()}",
            "wall_s_sample": round(dt, 2),
            "wall_s_full_call_extrapolated": round(dt * total / flops, 1),
            "wall_s_per_config_extrapolated": per_cfg}


class ClockSampler:
    """Samples the GPU's graphics clock, activity and socket power from amdsmi's
    GPU metrics in a background thread.  The firmware refreshes these metrics
    about once a second, so the sampler runs over a window of about three and a
    half seconds of repeated (untimed) steps after the timed ones, and keeps the
    refreshes taken under load (graphics activity >= 50%) after the first
    second, whose refresh can still describe the ramp from the pause before the
    window.  Under load the firmware holds the chip below its 2.4 GHz peak
    clock, so this is the clock a fraction of the nominal MFMA peak has to be
    read against.  Reports nothing (with the reason) when amdsmi is missing or
    the GPU is not found."""

    def __init__(self, torch, period_s: float = 0.05):
        self.period_s = period_s
        self.handle = None
        self.reason = None
        self.samples = []
        self._stop = None
        self._thread = None
        try:
            import amdsmi
            self.amdsmi = amdsmi
            amdsmi.amdsmi_init()
            handles = amdsmi.amdsmi_get_processor_handles()
            bus = torch.cuda.get_device_properties(0).pci_bus_id
            for h in handles:
                try:
                    if int(amdsmi.amdsmi_get_gpu_device_bdf(h).split(":")[1], 16) == bus:
                        self.handle = h
                        break
                except Exception:
                    continue
            if self.handle is None and len(handles) == 1:
                self.handle = handles[0]
            if self.handle is None:
                self.reason = f"no amdsmi device matches PCI bus {bus:#x} among {len(handles)}"
        except Exception as e:  # amdsmi missing or not usable here
            self.reason = f"amdsmi unavailable: {type(e).__name__}: {e}"[:200]

    def _one(self):
        m = self.amdsmi.amdsmi_get_gpu_metrics_info(self.handle)
        num = lambda x: float(x) if isinstance(x, (int, float)) and x >= 0 else None
        per_xcc = m.get("current_gfxclks")
        clk = None
        if isinstance(per_xcc, (list, tuple)):
            vals = [num(x) for x in per_xcc if num(x)]
            clk = sum(vals) / len(vals) if vals else None
        if clk is None:
            clk = num(m.get("current_gfxclk"))
        power = num(m.get("current_socket_power"))
        if power is None:
            power = num(m.get("average_socket_power"))
        return clk, num(m.get("average_gfx_activity")), power

    def _run(self):
        import time as _t
        while not self._stop.is_set():
            try:
                self.samples.append((_t.perf_counter(),) + self._one())
            except Exception as e:
                self.reason = f"metrics read failed: {type(e).__name__}: {e}"[:200]
                return
            _t.sleep(self.period_s)

    def measure(self, torch, step, seconds: float = 3.5, settle: float = 1.0):
        """Run step() repeatedly for about `seconds` while sampling; summary dict
        over the refreshes seen after the first `settle` seconds."""
        import threading
        import time as _t
        if self.handle is None:
            return {"source": None, "note": self.reason}
        self._stop = threading.Event()
        self._thread = threading.Thread(target=self._run, daemon=True)
        self._thread.start()
        t0 = _t.perf_counter()
        n = 0
        while _t.perf_counter() - t0 < seconds:
            for _ in range(5):
                step()
            torch.cuda.synchronize()
            n += 5
        elapsed = _t.perf_counter() - t0
        self._stop.set()
        self._thread.join(timeout=5)
        loaded, last = [], None
        for t, *smp in self.samples:  # one entry per firmware refresh, taken under load
            if smp != last and t - t0 >= settle and smp[0] and smp[1] is not None and smp[1] >= 50:
                loaded.append(smp)
            last = smp
        if not loaded:
            return {"source": None, "note": self.reason or "no metrics refresh under load during the window"}
        mean = lambda xs: round(sum(xs) / len(xs), 1) if xs else None
        clk = [c for c, _, _ in loaded]
        pw = [p for _, _, p in loaded if p is not None]
        return {"source": "amdsmi GPU metrics (current graphics clock, mean over the 8 XCDs), firmware refreshes "
                          f"under load during {n} further untimed steps after the timed ones (the first "
                          f"{settle:g} s of them excluded)",
                "refreshes": len(loaded), "gfxclk_mhz_mean": mean(clk), "gfxclk_mhz_min": min(clk),
                "gfxclk_mhz_max": max(clk), "socket_power_w_mean": mean(pw),
                "bf16_peak_at_mean_clock_tflops": round(PEAK_BF16_TFLOPS * mean(clk) / 2400.0, 1),
                "window_steps": n, "window_s": round(elapsed, 3)}


def _time_ms(torch, cur, fn, reps: int, warm: int = 2) -> float:
    """Average ms of fn() over reps calls, HIP events on the launch stream."""
    for _ in range(warm):
        fn()
    s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    s.record(cur)
    for _ in range(reps):
        fn()
    e.record(cur)
    torch.cuda.synchronize()
    return s.elapsed_time(e) / reps


def backward_1080p(torch, fastvr, metrics, dev, cur, qd, kd, vd, w, reps: int):
    """ms/call and effective TFLOP/s of the backward (dQ, dK, dV) of the parallel
    1080p call, given its O and LSE, for a seeded upstream gradient."""
    from paper_2609_36757_amd.workloads import randn_bf16
    g = torch.Generator().manual_seed(w.seed + 3000)
    dout = randn_bf16((w.B, w.n_tokens, w.H, w.d), g).to(dev)
    o, lse = fastvr.chunk_attn(qd, kd, vd, chunk_len=w.chunk_len, window_chunks=w.window_chunks, scale=w.scale)
    dq = torch.empty((w.B, w.n_tokens, w.H, w.d), dtype=torch.float32, device=dev)
    dk, dv = torch.empty_like(dq), torch.empty_like(dq)
    rs = torch.empty((w.B, w.H, 2, w.n_tokens), dtype=torch.float32, device=dev)
    ms = _time_ms(torch, cur, lambda: fastvr.chunk_attn_bwd(qd, kd, vd, o, lse, dout, chunk_len=w.chunk_len,
                                                            window_chunks=w.window_chunks, scale=w.scale, dq=dq,
                                                            dk=dk, dv=dv, row_stats=rs), reps)
    f = 2.5 * metrics.effective_flops(w.B, w.H, w.d, w.n_tokens, w.n_tokens, w.chunk_len, 0, w.window_chunks)
    return {"ms": round(ms, 4), "tflops": round(f / (ms * 1e-3) / 1e12, 2),
            "frac_of_bf16_peak": round(f / (ms * 1e-3) / 1e12 / PEAK_BF16_TFLOPS, 4),
            "note": "dQ, dK, dV of the parallel call given O and LSE (two kernels); effective flop = "
                    "10 d per visible pair (5 products); the kernels execute 7 (S and dP are "
                    "recomputed by both)"}


HBM_PEAK_GBS = 8000.0  # MI355X HBM3E


def one_step_update_timing(torch, fastvr, dev, cur):
    """The one-step latent update z_hat = z_LQ - sigma v (fp32 out) on the latent of
    the 1080p sequence (48 channels x 8 latent frames x 68 x 120) and on a
    2^28-element latent, as algorithmic HBM bytes (2 + 2 + 4 per element) per
    second against the 8 TB/s peak."""
    res = {}
    g = torch.Generator().manual_seed(41)
    for name, n, reps in (("one_step_1080p_latent", 48 * 8 * 68 * 120, 200), ("one_step_2e28", 1 << 28, 20)):
        z = torch.randn(n, generator=g).to(torch.bfloat16).to(dev)
        v = torch.randn(n, generator=g).to(torch.bfloat16).to(dev)
        out = torch.empty(n, dtype=torch.float32, device=dev)
        ms = _time_ms(torch, cur, lambda: fastvr.one_step_update(z, v, 0.8, out=out), reps)
        gbs = n * 8 / (ms * 1e-3) / 1e9
        res[name] = {"elements": n, "ms": round(ms, 5), "GB/s": round(gbs, 1),
                     "frac_of_hbm_peak": round(gbs / HBM_PEAK_GBS, 4)}
        del z, v, out
    return res


def tiled_1080p(torch, fastvr, metrics, dev, cur, qd, kd, vd, w):
    """Tiled inference on the 1080p sequence with the paper's overlapping 64 x 64
    latent tiles (overlap 16): gather of the q, k, v tokens (8 latent frames x 68
    x 120 positions, H * d = 1536 channels) into 2 x 3 tiles, one chunk-causal
    attention call over the tile batch (6 x 32768 tokens, chunks of 2 frames =
    8192 tokens), the blend of the per-tile outputs back onto the grid, and the
    blend of 48-channel velocity tiles fused with the one-step update of Eq. 9."""
    T, Hg, Wg, C = 8, 68, 120, w.H * w.d
    tile, ov = 64, 16
    grid = lambda t: t.view(w.B, T, Hg, Wg, C)
    qg, kg, vg = grid(qd), grid(kd), grid(vd)
    tiles = [fastvr.tile_gather(t, tile=tile, overlap=ov) for t in (qg, kg, vg)]
    Bt, nt, _, Ly, Lx, _ = tiles[0].shape
    ms_g = _time_ms(torch, cur, lambda: [fastvr.tile_gather(t, tile=tile, overlap=ov, out=o)
                                         for t, o in zip((qg, kg, vg), tiles)], 10)
    N, L = T * Ly * Lx, 2 * Ly * Lx
    tok = lambda t: t.view(Bt * nt, N, w.H, w.d)
    o = torch.empty((Bt * nt, N, w.H, w.d), dtype=torch.float32, device=dev)
    lse = torch.empty((Bt * nt, w.H, N), dtype=torch.float32, device=dev)
    ms_a = _time_ms(torch, cur, lambda: fastvr.chunk_attn(tok(tiles[0]), tok(tiles[1]), tok(tiles[2]), chunk_len=L,
                                                          window_chunks=w.window_chunks, scale=w.scale, out=o,
                                                          lse=lse), 5)
    f_a = metrics.effective_flops(Bt * nt, w.H, w.d, N, N, L, 0, w.window_chunks)
    out = torch.empty((w.B, T, Hg, Wg, C), dtype=torch.float32, device=dev)
    o6 = o.view(Bt, nt, T, Ly, Lx, C)
    ms_b = _time_ms(torch, cur, lambda: fastvr.tile_blend(o6, Hg, Wg, tile=tile, overlap=ov, out=out), 10)
    g = torch.Generator().manual_seed(43)
    vt = torch.randn((w.B, nt, T, Ly, Lx, 48), generator=g).to(dev)
    z = torch.randn((w.B, T, Hg, Wg, 48), generator=g).to(torch.bfloat16).to(dev)
    zh = torch.empty((w.B, T, Hg, Wg, 48), dtype=torch.float32, device=dev)
    ms_u = _time_ms(torch, cur, lambda: fastvr.tile_blend(vt, Hg, Wg, tile=tile, overlap=ov, z_lq=z, sigma=0.8,
                                                          out=zh), 50)
    gb = lambda nbytes, ms: round(nbytes / (ms * 1e-3) / 1e9, 1)
    tile_bytes = tiles[0].numel() * 2
    return {"tiles": f"{nt} ({Ly} x {Lx}) per frame, {N} tokens per tile",
            "gather_qkv_ms": round(ms_g, 4), "gather_GB/s": gb(3 * 2 * tile_bytes, ms_g),
            "attention_ms": round(ms_a, 4), "attention_tflops": round(f_a / (ms_a * 1e-3) / 1e12, 2),
            "blend_o_ms": round(ms_b, 4), "blend_GB/s": gb(o.numel() * 4 + out.numel() * 4, ms_b),
            "blend_update_latent_ms": round(ms_u, 5),
            "blend_update_GB/s": gb(vt.numel() * 4 + z.numel() * 2 + zh.numel() * 4, ms_u)}


def cold_cache(torch, fastvr, metrics, dev, cur, qd, kd, vd, w1080, reps: int = 5):
    """The 1080p and 480p parallel calls with the caches flushed before every call:
    a 512 MB buffer (twice the Infinity Cache) is overwritten between calls, and
    only the attention call itself is timed (HIP events around each call)."""
    from paper_2609_36757_amd.workloads import WORKLOADS, make_sequence
    flush = torch.empty(512 << 20, dtype=torch.uint8, device=dev)
    res = {}
    for name in ("1080p", "480p"):
        w = WORKLOADS[name]
        if name == "1080p":
            q, k, v = qd, kd, vd
        else:
            q, k, v = (t.to(dev) for t in make_sequence(w))
        o = torch.empty((w.B, w.n_tokens, w.H, w.d), dtype=torch.float32, device=dev)
        lse = torch.empty((w.B, w.H, w.n_tokens), dtype=torch.float32, device=dev)
        call = lambda: fastvr.chunk_attn(q, k, v, chunk_len=w.chunk_len, window_chunks=w.window_chunks,
                                         scale=w.scale, out=o, lse=lse)
        call()
        times = []
        for _ in range(reps):
            flush.fill_(1)
            s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            s.record(cur)
            call()
            e.record(cur)
            torch.cuda.synchronize()
            times.append(s.elapsed_time(e))
        ms = sorted(times)[len(times) // 2]
        f = metrics.effective_flops(w.B, w.H, w.d, w.n_tokens, w.n_tokens, w.chunk_len, 0, w.window_chunks)
        res[name] = {"ms_median": round(ms, 4), "tflops": round(f / (ms * 1e-3) / 1e12, 2)}
    del flush
    return res


def other_workloads(torch, fastvr, metrics, dev, cur, qd, kd, vd, w1080):
    """ms/call and effective TFLOP/s of the other synthetic workloads: the tiny,
    480p-shaped and wide sliding-window parallel calls, and the paper's W = 1
    streaming step with the bounded ring cache at the 1080p chunk shape."""
    from paper_2609_36757_amd.workloads import WORKLOADS, make_sequence
    res = {}
    for name, reps in (("tiny", 200), ("480p", 100), ("wide_sw", 3)):
        w = WORKLOADS[name]
        q, k, v = (t.to(dev) for t in make_sequence(w))
        o = torch.empty((w.B, w.n_tokens, w.H, w.d), dtype=torch.float32, device=dev)
        lse = torch.empty((w.B, w.H, w.n_tokens), dtype=torch.float32, device=dev)
        ms = _time_ms(torch, cur, lambda: fastvr.chunk_attn(q, k, v, chunk_len=w.chunk_len,
                                                            window_chunks=w.window_chunks, scale=w.scale,
                                                            out=o, lse=lse), reps, warm=5)
        f = metrics.effective_flops(w.B, w.H, w.d, w.n_tokens, w.n_tokens, w.chunk_len, 0, w.window_chunks)
        res[name] = {"ms": round(ms, 4), "ms_per_chunk": round(ms / w.n_chunks, 4),
                     "tflops": round(f / (ms * 1e-3) / 1e12, 2), "frac_of_bf16_peak": round(f / (ms * 1e-3) / 1e12
                                                                                          / PEAK_BF16_TFLOPS, 4)}
        del q, k, v, o, lse
    # W = 1 ring step: chunk 3 of the 1080p sequence, chunk 2 already in the ring
    w = w1080
    L, c = w.chunk_len, 3
    ring_k = torch.empty((w.B, 2 * L, w.H, w.d), dtype=torch.bfloat16, device=dev)
    ring_v = torch.empty_like(ring_k)
    s_prev = (c - 1) % 2
    ring_k[:, s_prev * L:(s_prev + 1) * L].copy_(kd[:, (c - 1) * L:c * L])
    ring_v[:, s_prev * L:(s_prev + 1) * L].copy_(vd[:, (c - 1) * L:c * L])
    qn, kn, vn = (t[:, c * L:(c + 1) * L].contiguous() for t in (qd, kd, vd))
    o = torch.empty((w.B, L, w.H, w.d), dtype=torch.float32, device=dev)
    lse = torch.empty((w.B, w.H, L), dtype=torch.float32, device=dev)
    ms = _time_ms(torch, cur, lambda: fastvr.chunk_attn_ring_step(qn, kn, vn, ring_k, ring_v, chunk_len=L,
                                                                  chunk_index=c, window_chunks=1, scale=w.scale,
                                                                  out=o, lse=lse), 20)
    f = metrics.effective_flops(w.B, w.H, w.d, L, 2 * L, L, 1, 1)
    res["ring_step_w1_1080p"] = {"ms": round(ms, 4), "tflops": round(f / (ms * 1e-3) / 1e12, 2),
                                 "note": "chunk 3 vs chunks 2-3, append of chunk 3 fused into the launch"}
    del ring_k, ring_v, qn, kn, vn, o, lse
    res["bwd_1080p"] = backward_1080p(torch, fastvr, metrics, dev, cur, qd, kd, vd, w, 5)
    res.update(one_step_update_timing(torch, fastvr, dev, cur))
    res["tiled_1080p"] = tiled_1080p(torch, fastvr, metrics, dev, cur, qd, kd, vd, w)
    res["cold_cache"] = cold_cache(torch, fastvr, metrics, dev, cur, qd, kd, vd, w)
    return res


def power_probe(torch, fastvr, dev):
    """Clock and socket power under four loads, each run back to back for 3.5 s
    (the first second excluded): a bf16 GEMM 8192^3 through torch.matmul
    (hipBLASLt; a reference load of the same MFMA type), the 1080p and 480p
    parallel forward calls, and the backward of the 1080p call.  Shows which
    loads reach the board's power ceiling and at what clock."""
    from paper_2609_36757_amd import metrics
    from paper_2609_36757_amd.workloads import WORKLOADS, make_sequence, randn_bf16
    out = {}
    sampler = lambda: ClockSampler(torch)

    def entry(r, flop):
        if r.get("source") is None:
            return r
        r = dict(r)
        r.pop("source", None)
        r["tflops"] = round(flop * r["window_steps"] / r["window_s"] / 1e12, 1)
        return r

    a = torch.randn(8192, 8192, device=dev, dtype=torch.bfloat16)
    out["gemm_bf16_8192"] = entry(sampler().measure(torch, lambda: a @ a), 2 * 8192 ** 3)
    del a
    w = WORKLOADS["1080p"]
    q, k, v = (t.to(dev) for t in make_sequence(w))
    o = torch.empty((w.B, w.n_tokens, w.H, w.d), dtype=torch.float32, device=dev)
    lse = torch.empty((w.B, w.H, w.n_tokens), dtype=torch.float32, device=dev)
    fwd = lambda: fastvr.chunk_attn(q, k, v, chunk_len=w.chunk_len, window_chunks=w.window_chunks, scale=w.scale,
                                    out=o, lse=lse)
    f1080 = metrics.effective_flops(w.B, w.H, w.d, w.n_tokens, w.n_tokens, w.chunk_len, 0, w.window_chunks)
    out["fwd_1080p"] = entry(sampler().measure(torch, fwd), f1080)
    g = torch.Generator().manual_seed(w.seed + 3000)
    dout = randn_bf16((w.B, w.n_tokens, w.H, w.d), g).to(dev)
    dq = torch.empty_like(o)
    dk, dv = torch.empty_like(o), torch.empty_like(o)
    rs = torch.empty((w.B, w.H, 2, w.n_tokens), dtype=torch.float32, device=dev)
    bwd = lambda: fastvr.chunk_attn_bwd(q, k, v, o, lse, dout, chunk_len=w.chunk_len, window_chunks=w.window_chunks,
                                        scale=w.scale, dq=dq, dk=dk, dv=dv, row_stats=rs)
    out["bwd_1080p_effective"] = entry(sampler().measure(torch, bwd), 2.5 * f1080)
    del q, k, v, o, lse, dout, dq, dk, dv, rs
    w4 = WORKLOADS["480p"]
    q, k, v = (t.to(dev) for t in make_sequence(w4))
    f480 = metrics.effective_flops(w4.B, w4.H, w4.d, w4.n_tokens, w4.n_tokens, w4.chunk_len, 0, w4.window_chunks)
    out["fwd_480p"] = entry(sampler().measure(torch, lambda: fastvr.chunk_attn(
        q, k, v, chunk_len=w4.chunk_len, window_chunks=w4.window_chunks, scale=w4.scale)), f480)
    return out


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=30)
    ap.add_argument("--warmup", type=int, default=50)
    ap.add_argument("--workload", default="1080p", choices=["1080p", "480p", "wide_sw", "tiny"])
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-clock", action="store_true", help="skip the clock window after the timed steps")
    ap.add_argument("--cpu-rows", type=int, default=2560)
    ap.add_argument("--no-extra", action="store_true", help="skip the 480p / wide_sw / ring-step / backward timings")
    ap.add_argument("--power-probe", action="store_true",
                    help="only report the clock and socket power under a GEMM and the attention calls")
    ap.add_argument("--bwd-only", action="store_true",
                    help="time only the backward of the 1080p call (--steps calls) and print its figures")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py runs on exactly one GPU: this build measures the single-GPU kernel "
              "(multi-GPU sharding is a design note only).", file=sys.stderr)
        sys.exit(2)

    import torch

    from paper_2609_36757_amd import fastvr, metrics
    from paper_2609_36757_amd.workloads import WORKLOADS, make_sequence

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    fastvr.load()
    dev = torch.device("cuda:0")
    w = WORKLOADS[args.workload]
    q, k, v = make_sequence(w)
    qd, kd, vd = q.to(dev), k.to(dev), v.to(dev)
    if args.power_probe:
        print("[bench] clock and power under a GEMM, the 1080p and 480p forward and the backward", flush=True)
        print(json.dumps({"power_probe": power_probe(torch, fastvr, dev)}), flush=True)
        return
    if args.bwd_only:
        w = WORKLOADS["1080p"]
        if args.workload != "1080p":
            q, k, v = make_sequence(w)
            qd, kd, vd = q.to(dev), k.to(dev), v.to(dev)
        print(f"[bench] backward of the 1080p call: {args.steps} calls", flush=True)
        r = backward_1080p(torch, fastvr, metrics, dev, torch.cuda.current_stream(), qd, kd, vd, w, args.steps)
        print(json.dumps({"bwd_1080p": r}), flush=True)
        return
    o = torch.empty((w.B, w.n_tokens, w.H, w.d), dtype=torch.float32, device=dev)
    lse = torch.empty((w.B, w.H, w.n_tokens), dtype=torch.float32, device=dev)

    stream = args.workload == "1080p"
    if stream:
        ws = WORKLOADS["1080p_stream"]
        c = ws.stream_chunk
        lo, hi = c * w.chunk_len, min((c + 1) * w.chunk_len, w.n_tokens)
        kc = torch.empty((w.B, hi, w.H, w.d), dtype=torch.bfloat16, device=dev)
        vc = torch.empty_like(kc)
        kc[:, :lo].copy_(kd[:, :lo])
        vc[:, :lo].copy_(vd[:, :lo])
        k_new, v_new = kd[:, lo:hi].contiguous(), vd[:, lo:hi].contiguous()
        q_new = qd[:, lo:hi].contiguous()
        so = torch.empty((w.B, hi - lo, w.H, w.d), dtype=torch.float32, device=dev)
        sl = torch.empty((w.B, w.H, hi - lo), dtype=torch.float32, device=dev)

    f_full = metrics.effective_flops(w.B, w.H, w.d, w.n_tokens, w.n_tokens, w.chunk_len, 0, w.window_chunks)
    f_stream = (metrics.effective_flops(w.B, w.H, w.d, hi - lo, hi, w.chunk_len, c, w.window_chunks)
                if stream else 0)
    n_chunks_per_step = w.n_chunks + (1 if stream else 0)
    cur = torch.cuda.current_stream()

    def step(ev=None):
        if ev is not None:
            ev[0].record(cur)
        fastvr.chunk_attn(qd, kd, vd, chunk_len=w.chunk_len, window_chunks=w.window_chunks, scale=w.scale,
                          out=o, lse=lse)
        if ev is not None:
            ev[1].record(cur)
        if stream:
            fastvr.kv_cache_append(kc, vc, k_new, v_new, lo)
            if ev is not None:
                ev[2].record(cur)
            fastvr.chunk_attn(q_new, kc, vc, chunk_len=w.chunk_len, q_chunk_offset=c,
                              window_chunks=w.window_chunks, scale=w.scale, out=so, lse=sl)
            if ev is not None:
                ev[3].record(cur)

    print(f"[bench] workload {w.name}: warmup {args.warmup}", flush=True)
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()

    n_ev = 4 if stream else 2
    events = [[torch.cuda.Event(enable_timing=True) for _ in range(n_ev)] for _ in range(args.steps)]
    print(f"[bench] timing {args.steps} steps", flush=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    start = torch.cuda.Event(enable_timing=True)
    end = torch.cuda.Event(enable_timing=True)
    start.record(cur)
    for i in range(args.steps):
        step(events[i])
    end.record(cur)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    clock_info = {"source": None, "note": "--no-clock"} if args.no_clock else ClockSampler(torch).measure(torch, step)
    total_ms = start.elapsed_time(end)
    ms_step = total_ms / args.steps
    per_full = sorted(e[0].elapsed_time(e[1]) for e in events)
    per_str = sorted(e[2].elapsed_time(e[3]) for e in events) if stream else [0.0]
    t_full = sum(per_full) / args.steps
    t_app = sum(e[1].elapsed_time(e[2]) for e in events) / args.steps if stream else 0.0
    t_str = sum(per_str) / args.steps if stream else 0.0
    med = lambda xs: xs[len(xs) // 2] if len(xs) % 2 else 0.5 * (xs[len(xs) // 2 - 1] + xs[len(xs) // 2])
    flops_step = f_full + f_stream
    value = flops_step / (ms_step * 1e-3) / 1e12
    n_launch = 2 if stream else 1
    avg_launch_ms = (t_full + t_str) / n_launch
    achieved = (flops_step / n_launch) / (avg_launch_ms * 1e-3) / 1e12
    traffic = read_traffic()

    out = {
        "metric": METRIC,
        "value": round(value, 2),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {
            "workload": (f"{w.name} chunk-causal attention: parallel call over {w.n_chunks} chunks x {w.chunk_len} "
                         f"tokens" + (f" + streaming step (append chunk {c}, attend {hi - lo} queries against "
                                      f"a {hi}-token KV cache)" if stream else "")),
            "B": w.B, "H": w.H, "head_dim": w.d, "seq_len": w.n_tokens, "chunk_len": w.chunk_len,
            "window_chunks": w.window_chunks, "parallelism": "single GPU",
        },
        "ms_per_chunk": round(ms_step / n_chunks_per_step, 4),
        "calls_ms": {"full": round(t_full, 4), "kv_append": round(t_app, 4), "stream": round(t_str, 4)},
        "calls_ms_median": {"full": round(med(per_full), 4), "stream": round(med(per_str), 4)},
        "calls_ms_min": {"full": round(per_full[0], 4), "stream": round(per_str[0], 4)},
        "calls_tflops": {"full": round(f_full / (t_full * 1e-3) / 1e12, 2),
                         "stream": round(f_stream / (t_str * 1e-3) / 1e12, 2) if stream else None},
        "effective_flop_per_step": flops_step,
        "frac_of_bf16_peak": round(value / PEAK_BF16_TFLOPS, 4),
        "roofline": {"kernel": "chunk_attn_fwd_kernel<128>", "bound": "mfma", "achieved": round(achieved, 2),
                     "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s", "frac": round(achieved / PEAK_BF16_TFLOPS, 4),
                     "traffic": traffic},
        "clock": clock_info,
        "wall_s_timed": round(wall, 3),
    }
    if not args.no_extra:
        print("[bench] other workloads (not part of the step)", flush=True)
        del o, lse
        out["other_workloads"] = other_workloads(torch, fastvr, metrics, dev, cur, qd, kd, vd, w)
    if not args.no_cpu_baseline:
        print("[bench] cpu baseline (fp64 oracle on a row sample)", flush=True)
        out["cpu_baseline"] = cpu_baseline(w, q, k, v, args.cpu_rows)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
