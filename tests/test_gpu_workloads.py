"""Parity at the full sizes of the benchmark workloads, in the launch
configuration the benchmark times.  Coverage per workload, every head each time:

* tiny and 480p: every row against the fp64 oracle;
* 1080p streaming step: every one of its 16320 rows against the oracle, and
  bit for bit against the rows of the parallel call;
* 1080p parallel call and the wide sliding window: a stratified row sample
  against the oracle, holding every row within 2 of each chunk boundary and of
  each 256-row query-tile boundary (the kernel's tile), the last rows of every
  chunk (the ragged tail included) and 4096 seeded random rows;
* every chunk of the tiny, 1080p and wide sliding-window sequences as a
  streaming call, bit for bit against the parallel call.

The oracle runs in host threads, each query chunk against the keys it can see
(parity.run_oracle_parallel)."""
import numpy as np
import pytest
import torch

from paper_2609_36757_amd import fastvr
from paper_2609_36757_amd.workloads import WORKLOADS, make_sequence, streaming_views

from parity import compare, run_oracle_parallel, sample_rows, to_np

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dev():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    fastvr.load()
    return torch.device("cuda:0")


def _announce(label):
    print(f"\n[gpu case] {label}", flush=True)


def _full_call(w, q, k, v, dev):
    qd, kd, vd = q.to(dev), k.to(dev), v.to(dev)
    o, lse = fastvr.chunk_attn(qd, kd, vd, chunk_len=w.chunk_len, window_chunks=w.window_chunks, scale=w.scale)
    torch.cuda.synchronize()
    return qd, kd, vd, o, lse


def _check_rows(w, q, k, v, o, lse, rows, label, q_chunk_offset=0):
    ridx = torch.as_tensor(rows, device=o.device)
    o_s = to_np(o[:, ridx])
    l_s = to_np(lse[:, :, ridx])
    assert torch.isfinite(o).all() and torch.isfinite(lse).all()
    o_ref, l_ref = run_oracle_parallel(q, k, v, w.chunk_len, q_chunk_offset, w.window_chunks, w.scale, rows=rows)
    return compare(o_s, l_s, o_ref, l_ref, label=f"{label} ({len(rows)} rows)")


def test_tiny_all_rows(dev):
    w = WORKLOADS["tiny"]
    _announce("tiny B=1 H=2 d=64 N=1024 L=256")
    q, k, v = make_sequence(w)
    _, _, _, o, lse = _full_call(w, q, k, v, dev)
    o_ref, l_ref = run_oracle_parallel(q, k, v, w.chunk_len, 0, w.window_chunks, w.scale)
    compare(to_np(o), to_np(lse), o_ref, l_ref, label="tiny (all rows)")


def test_480p_all_rows(dev):
    w = WORKLOADS["480p"]
    _announce("480p B=1 H=12 d=128 N=18720 L=3120 (all rows)")
    q, k, v = make_sequence(w)
    _, _, _, o, lse = _full_call(w, q, k, v, dev)
    o_ref, l_ref = run_oracle_parallel(q, k, v, w.chunk_len, 0, w.window_chunks, w.scale)
    compare(to_np(o), to_np(lse), o_ref, l_ref, label="480p (all rows, all heads)")


def test_1080p_full_and_streaming_step(dev):
    w = WORKLOADS["1080p"]
    ws = WORKLOADS["1080p_stream"]
    _announce("1080p B=1 H=12 d=128 N=65280 L=16320 + streaming step chunk 3")
    q, k, v = make_sequence(w)
    qd, kd, vd, o, lse = _full_call(w, q, k, v, dev)
    rows = sample_rows(w.n_tokens, w.chunk_len, n_random=4096, seed=3, band=2, tile=256)
    _check_rows(w, q, k, v, o, lse, rows, "1080p")

    # streaming step: cache holds chunks 0-2, append chunk 3, attend chunk 3
    sv = streaming_views(ws, qd, kd, vd)
    cap = sv["n_kv"]
    kc = torch.empty((w.B, cap, w.H, w.d), dtype=torch.bfloat16, device=dev)
    vc = torch.empty_like(kc)
    kc[:, :sv["cache_len"]].copy_(sv["k_prefix"])
    vc[:, :sv["cache_len"]].copy_(sv["v_prefix"])
    n_kv = fastvr.kv_cache_append(kc, vc, sv["k_new"].contiguous(), sv["v_new"].contiguous(), sv["cache_len"])
    assert n_kv == cap
    so, sl = fastvr.chunk_attn(sv["q_new"].contiguous(), kc, vc, chunk_len=ws.chunk_len,
                               q_chunk_offset=sv["q_chunk_offset"], window_chunks=ws.window_chunks, scale=ws.scale)
    torch.cuda.synchronize()
    lo = sv["cache_len"]
    assert torch.equal(kc, kd) and torch.equal(vc, vd)
    assert torch.equal(so, o[:, lo:lo + so.shape[1]]), "streaming step differs from the parallel call"
    assert torch.equal(sl, lse[:, :, lo:lo + so.shape[1]])
    # every row of the streaming step, every head
    o_ref, l_ref = run_oracle_parallel(q[:, lo:lo + so.shape[1]], k, v, ws.chunk_len, sv["q_chunk_offset"],
                                       ws.window_chunks, ws.scale)
    compare(to_np(so), to_np(sl), o_ref, l_ref,
            label=f"1080p streaming step (all {so.shape[1]} rows, all {w.H} heads)")


def test_wide_sliding_window_sampled(dev):
    w = WORKLOADS["wide_sw"]
    _announce("wide_sw B=1 H=24 d=128 N=138720 L=16320 W=2 outliers")
    q, k, v = make_sequence(w)
    _, _, _, o, lse = _full_call(w, q, k, v, dev)
    rows = sample_rows(w.n_tokens, w.chunk_len, n_random=4096, seed=5, band=2, tile=256)
    _check_rows(w, q, k, v, o, lse, rows, "wide_sw")


@pytest.mark.parametrize("name", ["tiny", "480p", "1080p", "wide_sw"])
def test_streaming_every_chunk_equals_parallel(dev, name):
    """Every chunk of the sequence as a streaming call equals the parallel call's
    rows bit for bit (same key tiles, same arithmetic order).  For 480p the
    parallel call (936 items) runs as per-CU item lists and each streaming call
    (156 items) as plain dispatch, so this also checks the list kernel.  With a window the
    cache is compacted to the W + 1 visible chunks and q_chunk_offset is the new
    chunk's index within it; with W = -1 it holds every earlier chunk."""
    w = WORKLOADS[name]
    _announce(f"{name}: every chunk streamed against the parallel call")
    q, k, v = make_sequence(w)
    qd, kd, vd, o, lse = _full_call(w, q, k, v, dev)
    del q, k, v
    L, N, W = w.chunk_len, w.n_tokens, w.window_chunks
    n_chunks = (N + L - 1) // L
    for c in range(n_chunks):
        c0 = 0 if W < 0 else max(0, c - W)
        lo, hi = c * L, min((c + 1) * L, N)
        kc, vc = kd[:, c0 * L:hi].contiguous(), vd[:, c0 * L:hi].contiguous()
        so, sl = fastvr.chunk_attn(qd[:, lo:hi].contiguous(), kc, vc, chunk_len=L, q_chunk_offset=c - c0,
                                   window_chunks=W, scale=w.scale)
        torch.cuda.synchronize()
        assert torch.equal(so, o[:, lo:hi]), (name, c)
        assert torch.equal(sl, lse[:, :, lo:hi]), (name, c)
        del kc, vc, so, sl
    print(f"[parity] {name}: {n_chunks} streaming calls bit-identical to the parallel call", flush=True)
