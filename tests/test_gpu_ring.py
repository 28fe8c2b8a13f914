"""GPU tests of the streaming step with a bounded ring KV cache (W + 1 chunk
slots, the append fused into the attention launch), through the C ABI.

Each case streams a sequence chunk by chunk through the ring and checks, for
every chunk: the output rows equal those of the parallel chunk-causal call over
the whole sequence bit for bit (same key tiles, same arithmetic order), the
ring holds the last W + 1 chunks, and sampled steps agree with the fp64 oracle's
ring step."""
import numpy as np
import pytest
import torch

import oracle
from paper_2609_36757_amd import fastvr
from paper_2609_36757_amd.workloads import WORKLOADS, make_qkv, make_sequence

from parity import compare, default_scale, run_oracle, sample_rows, to_np

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dev():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    fastvr.load()
    return torch.device("cuda:0")


def _announce(label):
    print(f"\n[gpu case] {label}", flush=True)


# name, B, H, d, N, chunk_len, W, seed
RING_CASES = [
    ("w1_L64", 2, 2, 128, 64 * 5 + 20, 64, 1, 101),
    ("w1_L100_ragged", 1, 2, 128, 100 * 4 + 37, 100, 1, 102),
    ("w0_L36", 1, 3, 128, 36 * 3 + 5, 36, 0, 103),
    ("w2_L300", 2, 1, 128, 300 * 4 + 128, 300, 2, 104),
    ("w3_L4_tiny_chunks", 1, 2, 128, 4 * 9 + 2, 4, 3, 105),
    ("w1_d64_L72", 2, 2, 64, 72 * 5 + 8, 72, 1, 106),
    ("w7_L24", 1, 1, 128, 24 * 10, 24, 7, 107),
    ("w1_L96_one_tile_per_chunk", 1, 2, 128, 96 * 4 + 50, 96, 1, 108),
    ("w2_L192_d64", 1, 2, 64, 192 * 4 + 10, 192, 2, 109),
    # negative scale: the ring kernels that track the running minimum (optional 9th field: scale)
    ("w1_L100_negative_scale", 1, 2, 128, 100 * 4 + 37, 100, 1, 110, -0.06),
    ("w2_L72_d64_negative_scale", 2, 2, 64, 72 * 5 + 8, 72, 2, 111, -0.2),
]


@pytest.mark.parametrize("case", RING_CASES, ids=[c[0] for c in RING_CASES])
def test_ring_stream_equals_parallel(dev, case):
    name, B, H, d, N, L, W, seed, *opt = case
    scale = opt[0] if opt else default_scale(d)
    _announce(f"ring {name} B={B} H={H} d={d} N={N} L={L} W={W} scale={scale}")
    q, k, v = make_qkv(B, N, N, H, d, seed)
    qd, kd, vd = q.to(dev), k.to(dev), v.to(dev)
    full_o, full_l = fastvr.chunk_attn(qd, kd, vd, chunk_len=L, window_chunks=W, scale=scale)
    ring_k = torch.full((B, (W + 1) * L, H, d), float("nan"), dtype=torch.bfloat16, device=dev)
    ring_v = torch.full_like(ring_k, float("nan"))
    n_chunks = -(-N // L)
    for c in range(n_chunks):
        s = slice(c * L, min((c + 1) * L, N))
        o, lse = fastvr.chunk_attn_ring_step(qd[:, s].contiguous(), kd[:, s].contiguous(), vd[:, s].contiguous(),
                                             ring_k, ring_v, chunk_len=L, chunk_index=c, window_chunks=W,
                                             scale=scale)
        torch.cuda.synchronize()
        assert torch.equal(o, full_o[:, s]), f"chunk {c}: output differs from the parallel call"
        assert torch.equal(lse, full_l[:, :, s]), f"chunk {c}: lse differs from the parallel call"
        # the ring holds chunks c - W .. c in slots chunk mod (W + 1)
        for cc in range(max(0, c - W), c + 1):
            sl = cc % (W + 1)
            n = min(L, N - cc * L)
            assert torch.equal(ring_k[:, sl * L:sl * L + n], kd[:, cc * L:cc * L + n]), f"ring K slot {sl}"
            assert torch.equal(ring_v[:, sl * L:sl * L + n], vd[:, cc * L:cc * L + n]), f"ring V slot {sl}"
    # the parallel call (and so every ring step) against the fp64 oracle
    o_ref, l_ref = run_oracle(q, k, v, L, 0, W, scale)
    compare(to_np(full_o), to_np(full_l), o_ref, l_ref, label=f"ring {name}")


def test_ring_step_matches_oracle_ring_step(dev):
    """One step checked directly against oracle.ring_step (outputs and ring)."""
    B, H, d, L, W, c = 1, 2, 128, 96, 2, 5
    _announce(f"ring step vs oracle B={B} H={H} d={d} L={L} W={W} c={c}")
    g = torch.Generator().manual_seed(7)
    ring_k = torch.randn((B, (W + 1) * L, H, d), generator=g).to(torch.bfloat16)
    ring_v = torch.randn((B, (W + 1) * L, H, d), generator=g).to(torch.bfloat16)
    qn, kn, vn = make_qkv(B, 70, 70, H, d, seed=8)
    o_ref, l_ref, kr_ref, vr_ref = oracle.ring_step(ring_k.float().numpy(), ring_v.float().numpy(),
                                                    qn.float().numpy(), kn.float().numpy(), vn.float().numpy(),
                                                    L, c, W, scale=float(np.float32(default_scale(d))))
    rk, rv = ring_k.to(dev), ring_v.to(dev)
    o, lse = fastvr.chunk_attn_ring_step(qn.to(dev), kn.to(dev), vn.to(dev), rk, rv, chunk_len=L,
                                         chunk_index=c, window_chunks=W)
    torch.cuda.synchronize()
    compare(to_np(o), to_np(lse), o_ref, l_ref, label="ring step vs oracle")
    assert np.array_equal(rk.float().cpu().numpy(), kr_ref)
    assert np.array_equal(rv.float().cpu().numpy(), vr_ref)


def test_ring_1080p_w1_step(dev):
    """The paper's configuration (W = 1) at the 1080p chunk shape: chunk 3 of
    the 1080p sequence with chunk 2 in the ring equals the parallel W = 1 call,
    bit for bit, and a row sample matches the oracle."""
    w = WORKLOADS["1080p"]
    L, W, c = w.chunk_len, 1, 3
    _announce(f"ring 1080p W=1 chunk {c} (L={L}, H={w.H}, d={w.d})")
    q, k, v = make_sequence(w)
    qd, kd, vd = q.to(dev), k.to(dev), v.to(dev)
    lo, hi = c * L, (c + 1) * L
    # parallel W = 1 reference for the rows of chunk c: keys of chunks 2..3 only
    k2, v2 = kd[:, (c - 1) * L:hi].contiguous(), vd[:, (c - 1) * L:hi].contiguous()
    ref_o, ref_l = fastvr.chunk_attn(qd[:, lo:hi].contiguous(), k2, v2, chunk_len=L, q_chunk_offset=1,
                                     window_chunks=W)
    ring_k = torch.empty((w.B, 2 * L, w.H, w.d), dtype=torch.bfloat16, device=dev)
    ring_v = torch.empty_like(ring_k)
    ring_k[:, (c - 1) % 2 * L:((c - 1) % 2 + 1) * L] = kd[:, (c - 1) * L:c * L]
    ring_v[:, (c - 1) % 2 * L:((c - 1) % 2 + 1) * L] = vd[:, (c - 1) * L:c * L]
    o, lse = fastvr.chunk_attn_ring_step(qd[:, lo:hi].contiguous(), kd[:, lo:hi].contiguous(),
                                         vd[:, lo:hi].contiguous(), ring_k, ring_v, chunk_len=L, chunk_index=c,
                                         window_chunks=W, scale=w.scale)
    torch.cuda.synchronize()
    assert torch.equal(o, ref_o) and torch.equal(lse, ref_l)
    assert torch.equal(ring_k[:, c % 2 * L:(c % 2 + 1) * L], kd[:, lo:hi])
    rows = sample_rows(L, L, n_random=64, seed=9, band=0)
    ridx = torch.as_tensor(rows, device=dev)
    o_ref, l_ref = run_oracle(q[:, lo:hi], k[:, (c - 1) * L:hi], v[:, (c - 1) * L:hi], L, 1, W, w.scale, rows=rows)
    compare(to_np(o[:, ridx]), to_np(lse[:, :, ridx]), o_ref, l_ref, label="ring 1080p W=1 (sampled)")
