"""Seeded random shapes for the forward and the backward against the fp64
oracle: batch, heads, head_dim, query and key counts, chunk length, chunk
offset (streaming form), window (the paper's W = 1 among them) and scale are
drawn per case, so ragged chunks, tiles and tails meet in combinations the
hand-picked cases do not list."""
import os

import numpy as np
import pytest
import torch

import oracle
from paper_2609_36757_amd import fastvr
from paper_2609_36757_amd.workloads import make_qkv, randn_bf16

from parity import compare, fp32_scale, run_oracle, to_np

pytestmark = pytest.mark.gpu

# more cases for a longer sweep: FASTVR_FUZZ_CASES=200 pytest tests/test_gpu_fuzz.py
N_CASES = int(os.environ.get("FASTVR_FUZZ_CASES", "24"))


def _case(i):
    rng = np.random.default_rng(9000 + i)
    B = int(rng.integers(1, 3))
    H = int(rng.integers(1, 4))
    d = int(rng.choice([64, 128]))
    L = int(rng.choice([1, 3, 16, 37, 64, 95, 96, 100, 129, 192, 256, 300]))
    n_chunks = int(rng.integers(1, 6))
    off = int(rng.integers(0, 3))
    nq = int(rng.integers(1, n_chunks * L + 1))
    nkv = off * L + nq + int(rng.integers(0, L + 1))   # may hold keys of later chunks (masked)
    W = int(rng.choice([-1, 0, 1, 1, 2, 5]))
    scale = [1.0 / np.sqrt(d), 0.3, 0.05, -0.2][i % 4]
    return B, H, d, L, off, nq, nkv, W, scale


@pytest.fixture(scope="module")
def dev():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    fastvr.load()
    return torch.device("cuda:0")


@pytest.mark.parametrize("i", range(N_CASES))
def test_fuzz_forward_and_backward(dev, i):
    B, H, d, L, off, nq, nkv, W, scale = _case(i)
    print(f"\n[gpu case] fuzz {i}: B={B} H={H} d={d} L={L} off={off} Nq={nq} Nkv={nkv} W={W} scale={scale}",
          flush=True)
    q, k, v = make_qkv(B, nq, nkv, H, d, seed=100 + i)
    qd, kd, vd = q.to(dev), k.to(dev), v.to(dev)
    o, lse = fastvr.chunk_attn(qd, kd, vd, chunk_len=L, q_chunk_offset=off, window_chunks=W, scale=scale)
    g = torch.Generator().manual_seed(200 + i)
    do = randn_bf16((B, nq, H, d), g)
    dq, dk, dv = fastvr.chunk_attn_bwd(qd, kd, vd, o, lse, do.to(dev), chunk_len=L, q_chunk_offset=off,
                                       window_chunks=W, scale=scale)
    torch.cuda.synchronize()
    o_ref, l_ref = run_oracle(q, k, v, L, off, W, scale)
    compare(to_np(o), to_np(lse), o_ref, l_ref, label=f"fuzz {i} forward")
    refs = oracle.attention_bwd(q, k, v, do, chunk_len=L, q_chunk_offset=off, window_chunks=W,
                                scale=fp32_scale(scale))
    for name, got, ref in zip(("dq", "dk", "dv"), (dq, dk, dv), refs):
        g64 = to_np(got)
        assert np.isfinite(g64).all(), (i, name)
        err = float(np.abs(g64 - ref).max())
        if np.linalg.norm(ref) < 1e-6:
            # an exactly vanishing gradient (e.g. a single visible key: dS = 0):
            # the GPU keeps only fp32 rounding noise of dP - D
            print(f"[parity] fuzz {i} {name} reference ~ 0, max_abs={err:.3e}", flush=True)
            assert err <= 1e-4, (i, name, err)
            continue
        rel = float(np.linalg.norm(g64 - ref) / np.linalg.norm(ref))
        print(f"[parity] fuzz {i} {name} rel_fro={rel:.3e} max_abs={err:.3e}", flush=True)
        # bf16 rounding of P and dS: expected about u / sqrt(3) = 2.3e-3 (see test_gpu_bwd.py)
        assert rel <= 1e-2, (i, name, rel)
