"""Re-entrancy on the GPU: the library keeps no global state, so host threads
calling it at the same time, each on a stream of its own, must get exactly the
results of one thread calling it alone (ctypes releases the GIL during the
calls, so the calls really overlap)."""
import threading

import pytest
import torch

from paper_2609_36757_amd import fastvr
from paper_2609_36757_amd.workloads import make_qkv

pytestmark = pytest.mark.gpu

N_THREADS = 4
N_ITERS = 5


@pytest.fixture(scope="module")
def dev():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    fastvr.load()
    return torch.device("cuda:0")


def _problem(i, dev):
    # a different shape, window and scale per thread
    B, H, d, N, L, W = (1, 2, 128, 900 + 37 * i, 150 + 20 * i, [-1, 1, 2, 0][i % 4])
    q, k, v = (t.to(dev) for t in make_qkv(B, N, N, H, d, seed=500 + i))
    g = torch.Generator().manual_seed(600 + i)
    do = torch.randn((B, N, H, d), generator=g).to(torch.bfloat16).to(dev)
    return dict(q=q, k=k, v=v, do=do, L=L, W=W, scale=0.05 + 0.02 * i)


def _run(p):
    o, lse = fastvr.chunk_attn(p["q"], p["k"], p["v"], chunk_len=p["L"], window_chunks=p["W"], scale=p["scale"])
    dq, dk, dv = fastvr.chunk_attn_bwd(p["q"], p["k"], p["v"], o, lse, p["do"], chunk_len=p["L"],
                                       window_chunks=p["W"], scale=p["scale"])
    return o, lse, dq, dk, dv


def test_threads_on_own_streams_match_serial(dev):
    print(f"\n[gpu case] {N_THREADS} host threads x {N_ITERS} forward+backward calls on their own streams", flush=True)
    problems = [_problem(i, dev) for i in range(N_THREADS)]
    serial = [_run(p) for p in problems]
    torch.cuda.synchronize()
    results = [None] * N_THREADS
    errors = []

    def worker(i):
        try:
            s = torch.cuda.Stream()
            with torch.cuda.stream(s):
                out = None
                for _ in range(N_ITERS):
                    out = _run(problems[i])
                s.synchronize()
            results[i] = out
        except Exception as e:  # reported by the main thread
            errors.append((i, repr(e)))

    threads = [threading.Thread(target=worker, args=(i,)) for i in range(N_THREADS)]
    for t in threads:
        t.start()
    for t in threads:
        t.join(timeout=120)
    torch.cuda.synchronize()
    assert not errors, errors
    for i in range(N_THREADS):
        assert results[i] is not None, i
        for name, a, b in zip(("o", "lse", "dq", "dk", "dv"), results[i], serial[i]):
            assert torch.equal(a, b), (i, name)
    print("[parity] concurrent calls bit-identical to serial", flush=True)
