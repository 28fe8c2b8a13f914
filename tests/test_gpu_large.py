"""Far addressing: tensors of several GiB whose checked rows lie past 2 GiB (and,
for the second batch row, past 4 GiB) from their base, so every byte offset the
kernels form for them needs more than 32 bits.  Only the chunks a checked query
sees hold seeded random data.  In the streaming-shaped case every other key row
holds NaN, so a visited chunk that the chunk mask hides (paper Sec. 3.1, Eq. 1:
later chunks, and chunks beyond the window) would show in the output, and the
backward must give those keys gradients of exactly zero.  The oracle runs on the
visible chunks only (the mask depends only on chunk differences)."""
import numpy as np
import pytest
import torch

import oracle
from paper_2609_36757_amd import fastvr
from paper_2609_36757_amd.workloads import make_qkv, randn_bf16

from parity import compare, fp32_scale, run_oracle, to_np
from test_gpu_bwd import _rounding_sigmas, compare_grad

pytestmark = pytest.mark.gpu

D = 128
L = 4096
N_CHUNKS = 2050          # 2050 * 4096 tokens * 256 bytes per key row = 2.15 GB per batch row
N = L * N_CHUNKS


@pytest.fixture(scope="module")
def dev():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    fastvr.load()
    return torch.device("cuda:0")


def test_streaming_chunk_past_4gib_forward_and_backward(dev):
    """B = 2, H = 1: the query chunk is the last of 2050, W = 1, so it sees the
    last two chunks, whose key rows start 2.15 GB (batch 0) and 4.30 GB (batch 1)
    from the base of k and v.  Forward and backward against the oracle on those
    chunks; every other key row is NaN, and its dK, dV must be exactly 0."""
    B, W = 2, 1
    off = N_CHUNKS - 1
    lo = (N_CHUNKS - 2) * L
    print(f"\n[gpu case] far streaming chunk: B={B} H=1 d={D} Nkv={N} L={L} offset={off} W={W}", flush=True)
    q, kc, vc = make_qkv(B, L, 2 * L, 1, D, seed=901)
    do = randn_bf16((B, L, 1, D), torch.Generator().manual_seed(902))
    nan = float("nan")
    kd = torch.full((B, N, 1, D), nan, dtype=torch.bfloat16, device=dev)
    vd = torch.full((B, N, 1, D), nan, dtype=torch.bfloat16, device=dev)
    kd[:, lo:] = kc.to(dev)
    vd[:, lo:] = vc.to(dev)
    qd, dod = q.to(dev), do.to(dev)
    scale = 1.0 / np.sqrt(D)
    o, lse = fastvr.chunk_attn(qd, kd, vd, chunk_len=L, q_chunk_offset=off, window_chunks=W, scale=scale)
    dq, dk, dv = fastvr.chunk_attn_bwd(qd, kd, vd, o, lse, dod, chunk_len=L, q_chunk_offset=off, window_chunks=W,
                                       scale=scale)
    torch.cuda.synchronize()
    # the same mask on the compact key range: the two visible chunks, query chunk 1 of them
    o_ref, l_ref = run_oracle(q, kc, vc, L, 1, W, scale)
    compare(to_np(o), to_np(lse), o_ref, l_ref, label="far streaming chunk (forward)")
    s32 = fp32_scale(scale)
    rq, rk, rv = oracle.attention_bwd(q, kc, vc, do, chunk_len=L, q_chunk_offset=1, window_chunks=W, scale=s32)
    sq, sk, sv = _rounding_sigmas(q, kc, vc, do, L, 1, W, s32)
    compare_grad("dq", to_np(dq), rq, sq, "far streaming chunk")
    compare_grad("dk", to_np(dk[:, lo:]), rk, sk, "far streaming chunk")
    compare_grad("dv", to_np(dv[:, lo:]), rv, sv, "far streaming chunk")
    # keys no query of the call sees (all NaN in k and v): exactly zero gradients
    assert int(torch.count_nonzero(dk[:, :lo])) == 0
    assert int(torch.count_nonzero(dv[:, :lo])) == 0


def test_parallel_rows_past_2gib(dev):
    """B = 1, H = 1, W = 1 over 2050 chunks (8.4 M tokens): rows of the last two
    query chunks lie 2.15 GB into q and 4.3 GB into the fp32 output.  Only the
    last three chunks hold random data (the rest zeros), and the rows of the last
    two query chunks are compared with the oracle on those three chunks."""
    W = 1
    first = N_CHUNKS - 3
    print(f"\n[gpu case] far parallel rows: B=1 H=1 d={D} N={N} L={L} W={W}", flush=True)
    q3, k3, v3 = make_qkv(1, 3 * L, 3 * L, 1, D, seed=903)
    qd = torch.zeros((1, N, 1, D), dtype=torch.bfloat16, device=dev)
    kd, vd = torch.zeros_like(qd), torch.zeros_like(qd)
    qd[:, first * L:] = q3.to(dev)
    kd[:, first * L:] = k3.to(dev)
    vd[:, first * L:] = v3.to(dev)
    scale = 1.0 / np.sqrt(D)
    o, lse = fastvr.chunk_attn(qd, kd, vd, chunk_len=L, window_chunks=W, scale=scale)
    torch.cuda.synchronize()
    rows = np.arange(L, 3 * L)  # query chunks 1 and 2 of the last three
    o_ref, l_ref = run_oracle(q3, k3, v3, L, 0, W, scale, rows=rows)
    got_o = to_np(o[:, (first + 1) * L:])
    got_l = to_np(lse[:, :, (first + 1) * L:])
    compare(got_o, got_l, o_ref, l_ref, label="far parallel rows (last two chunks)")
    assert bool(torch.isfinite(o).all()) and bool(torch.isfinite(lse).all())
