"""fastvr_chunk_attn_bwd_noalloc (the backward for callers that cannot allocate:
its row statistics live in the library's static per-device array) against
fastvr_chunk_attn_bwd with a caller workspace, through the C ABI: the same
kernels, so dq, dk and dv must be identical bit for bit.  Two calls in a row,
the second smaller than the first (the array keeps the first call's contents,
which must not leak into the second), then the first shape again; and the
host-side limit on the workspace size."""
import numpy as np
import pytest
import torch

from paper_2609_36757_amd import fastvr
from paper_2609_36757_amd.workloads import make_qkv, randn_bf16

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dev():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    fastvr.load()
    return torch.device("cuda:0")


def _case(dev, B, H, d, nq, nkv, L, off, W, seed):
    q, k, v = (t.to(dev) for t in make_qkv(B, nq, nkv, H, d, seed))
    g = torch.Generator().manual_seed(seed + 1)
    do = randn_bf16((B, nq, H, d), g).to(dev)
    o, lse = fastvr.chunk_attn(q, k, v, chunk_len=L, q_chunk_offset=off, window_chunks=W)
    return q, k, v, do, o, lse


def _both(dev, q, k, v, do, o, lse, L, off, W):
    ref = fastvr.chunk_attn_bwd(q, k, v, o, lse, do, chunk_len=L, q_chunk_offset=off, window_chunks=W)
    B, nq, H, d = q.shape
    nkv = k.shape[1]
    # outputs poisoned first: every element must be written
    dq = torch.full((B, nq, H, d), float("nan"), device=dev)
    dk = torch.full((B, nkv, H, d), float("nan"), device=dev)
    dv = torch.full((B, nkv, H, d), float("nan"), device=dev)
    got = fastvr.chunk_attn_bwd_noalloc(q, k, v, o, lse, do, dq, dk, dv, chunk_len=L, q_chunk_offset=off,
                                        window_chunks=W)
    torch.cuda.synchronize()
    for name, a, b in zip(("dq", "dk", "dv"), got, ref):
        assert torch.equal(a.view(torch.int32), b.view(torch.int32)), name


def test_noalloc_matches_workspace_backward_twice_then_smaller(dev):
    big = (2, 3, 128, 900, 900, 200, 0, -1, 61)
    small = (1, 2, 64, 150, 450, 150, 2, 1, 62)
    for shape in (big, small, big):
        B, H, d, nq, nkv, L, off, W, seed = shape
        print(f"\n[gpu case] bwd_noalloc B={B} H={H} d={d} Nq={nq} Nkv={nkv} L={L} off={off} W={W}", flush=True)
        q, k, v, do, o, lse = _case(dev, B, H, d, nq, nkv, L, off, W, seed)
        _both(dev, q, k, v, do, o, lse, L, off, W)


def test_noalloc_at_the_1080p_shape(dev):
    """The 1080p sequence's backward (2 * 12 * 65280 floats of row statistics)."""
    from paper_2609_36757_amd.workloads import WORKLOADS, make_sequence
    w = WORKLOADS["1080p"]
    print("\n[gpu case] bwd_noalloc 1080p B=1 H=12 d=128 N=65280 L=16320", flush=True)
    q, k, v = (t.to(dev) for t in make_sequence(w))
    g = torch.Generator().manual_seed(w.seed + 3000)
    do = randn_bf16((w.B, w.n_tokens, w.H, w.d), g).to(dev)
    o, lse = fastvr.chunk_attn(q, k, v, chunk_len=w.chunk_len, window_chunks=w.window_chunks, scale=w.scale)
    _both(dev, q, k, v, do, o, lse, w.chunk_len, 0, w.window_chunks)


def test_noalloc_in_a_hip_graph(dev):
    """Captured in a HIP graph (what callers that cannot allocate need it for)
    and replayed three times.  Before each replay an eager call of another shape
    rewrites the static array and the outputs are poisoned: every replay must
    give the eager result bit for bit."""
    B, H, d, nq, nkv, L, off, W, seed = 1, 2, 128, 600, 600, 200, 0, -1, 63
    print(f"\n[gpu case] bwd_noalloc in a HIP graph B={B} H={H} d={d} N={nq} L={L}", flush=True)
    q, k, v, do, o, lse = _case(dev, B, H, d, nq, nkv, L, off, W, seed)
    dq = torch.empty((B, nq, H, d), dtype=torch.float32, device=dev)
    dk, dv = torch.empty((B, nkv, H, d), dtype=torch.float32, device=dev), torch.empty((B, nkv, H, d), device=dev)
    run = lambda: fastvr.chunk_attn_bwd_noalloc(q, k, v, o, lse, do, dq, dk, dv, chunk_len=L, q_chunk_offset=off,
                                                window_chunks=W)
    # another shape, run eagerly between replays (same static array)
    q2, k2, v2, do2, o2, lse2 = _case(dev, 1, 3, 64, 300, 500, 100, 2, 1, seed + 5)
    dq2 = torch.empty((1, 300, 3, 64), dtype=torch.float32, device=dev)
    dk2, dv2 = torch.empty((1, 500, 3, 64), device=dev), torch.empty((1, 500, 3, 64), device=dev)
    other = lambda: fastvr.chunk_attn_bwd_noalloc(q2, k2, v2, o2, lse2, do2, dq2, dk2, dv2, chunk_len=100,
                                                  q_chunk_offset=2, window_chunks=1)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        run()   # eager first: also looks up the array's address outside the capture
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    ref = [t.clone() for t in (dq, dk, dv)]
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        run()
    torch.cuda.synchronize()
    for rep in range(3):
        for t in (dq, dk, dv):
            t.fill_(float("nan"))
        other()
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        for name, a, b in zip(("dq", "dk", "dv"), (dq, dk, dv), ref):
            assert torch.equal(a.view(torch.int32), b.view(torch.int32)), (rep, name)
    print("[parity] bwd_noalloc graph replays x3 bit-identical to eager", flush=True)


def test_noalloc_rejects_workspace_above_the_limit(dev):
    """2 * B * H * Nq above FASTVR_BWD_NOALLOC_MAX_FLOATS is refused on the host
    (no kernel runs; the tensors are never read)."""
    B, H, d, nq = 1, 64, 64, 65537
    x = torch.empty((B, nq, H, d), dtype=torch.bfloat16, device=dev)
    f = torch.empty((B, nq, H, d), dtype=torch.float32, device=dev)
    lse = torch.empty((B, H, nq), dtype=torch.float32, device=dev)
    dk, dv = torch.empty_like(f), torch.empty_like(f)
    with pytest.raises(fastvr.FastVRError) as e:
        fastvr.chunk_attn_bwd_noalloc(x, x, x, f, lse, x, f, dk, dv, chunk_len=1000)
    assert e.value.status == fastvr.ERR_UNSUPPORTED and "at most" in str(e.value)
