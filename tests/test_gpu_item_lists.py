"""The forward's per-CU item-list kernel in each of its instantiations (head_dim
64 and 128, positive and negative scale).  The 480p shape (B=1, H=12, 6 chunks
of 3120 tokens, 936 uneven items) is one the host packs into per-CU lists
(tests/test_item_lists.py checks that plan on the CPU), while each chunk of it
as a streaming call (156 items) keeps plain dispatch.  So: every row of the
parallel call must equal the streaming calls bit for bit (the same items, run
by the other kernel), and a stratified row sample must match the fp64 oracle."""
import numpy as np
import pytest
import torch

from paper_2609_36757_amd import fastvr
from paper_2609_36757_amd.workloads import make_qkv

from parity import compare, run_oracle, sample_rows, to_np

pytestmark = pytest.mark.gpu

L, N_CHUNKS, H = 3120, 6, 12


@pytest.fixture(scope="module")
def dev():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    fastvr.load()
    return torch.device("cuda:0")


@pytest.mark.parametrize("d,scale,window", [(64, 0.125, -1), (128, -1 / np.sqrt(128), -1), (64, -0.2, -1),
                                            (128, 1 / np.sqrt(128), 1)])
def test_item_lists_equal_plain_dispatch_and_oracle(dev, d, scale, window):
    n = L * N_CHUNKS
    print(f"\n[gpu case] item lists: B=1 H={H} d={d} N={n} L={L} W={window} scale={scale:.4f}", flush=True)
    q, k, v = make_qkv(1, n, n, H, d, seed=700 + d + (window + 1))
    qd, kd, vd = q.to(dev), k.to(dev), v.to(dev)
    o, lse = fastvr.chunk_attn(qd, kd, vd, chunk_len=L, window_chunks=window, scale=scale)
    torch.cuda.synchronize()
    for c in range(N_CHUNKS):
        c0 = 0 if window < 0 else max(0, c - window)
        kc, vc = kd[:, c0 * L:(c + 1) * L].contiguous(), vd[:, c0 * L:(c + 1) * L].contiguous()
        so, sl = fastvr.chunk_attn(qd[:, c * L:(c + 1) * L].contiguous(), kc, vc, chunk_len=L,
                                   q_chunk_offset=c - c0, window_chunks=window, scale=scale)
        torch.cuda.synchronize()
        assert torch.equal(so, o[:, c * L:(c + 1) * L]), (d, scale, window, c)
        assert torch.equal(sl, lse[:, :, c * L:(c + 1) * L]), (d, scale, window, c)
    rows = sample_rows(n, L, n_random=256, seed=17, band=0)
    ridx = torch.as_tensor(rows, device=dev)
    o_ref, l_ref = run_oracle(q, k, v, L, 0, window, scale, rows=rows)
    compare(to_np(o[:, ridx]), to_np(lse[:, :, ridx]), o_ref, l_ref,
            label=f"item lists d={d} scale={scale:.4f} W={window} ({len(rows)} rows)")


def test_item_lists_bf16_output_strided_and_no_lse(dev):
    """The list kernel's other output forms: O as bf16 into a strided view (the
    fp32 result rounded to nearest even, bit for bit, nothing written outside
    the view) and no LSE pointer (O unchanged)."""
    d, n = 128, L * N_CHUNKS
    print(f"\n[gpu case] item lists, bf16 strided O and no LSE: B=1 H={H} d={d} N={n} L={L}", flush=True)
    q, k, v = (t.to(dev) for t in make_qkv(1, n, n, H, d, seed=760))
    o32, l32 = fastvr.chunk_attn(q, k, v, chunk_len=L)
    big = torch.full((1, n + 9, H, d), float("nan"), dtype=torch.bfloat16, device=dev)
    ob = big[:, 3:3 + n]
    _, l16 = fastvr.chunk_attn(q, k, v, chunk_len=L, out=ob)
    o_nl, none = fastvr.chunk_attn(q, k, v, chunk_len=L, return_lse=False)
    torch.cuda.synchronize()
    assert none is None
    assert torch.equal(ob.view(torch.int16), o32.to(torch.bfloat16).view(torch.int16))
    assert torch.isnan(big[:, :3].float()).all() and torch.isnan(big[:, 3 + n:].float()).all()
    assert torch.equal(l16, l32)
    assert torch.equal(o_nl, o32)
