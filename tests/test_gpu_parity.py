"""GPU parity of the HIP path (through the C ABI) against the fp64 oracle.

Every case prints its name and shape before touching the GPU."""
import numpy as np
import pytest
import torch

from paper_2609_36757_amd import fastvr
from paper_2609_36757_amd.workloads import make_qkv

from parity import compare, default_scale, run_oracle, to_np

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dev():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    fastvr.load()  # raises if the library is missing: no fallback
    return torch.device("cuda:0")


def _announce(label):
    print(f"\n[gpu case] {label}", flush=True)


# name, B, H, d, Nq, Nkv, chunk_len, q_chunk_offset, window, scale (None: 1/sqrt(d)), seed
CASES = [
    ("tiny_cfg_shape", 1, 2, 64, 1024, 1024, 256, 0, -1, 0.125, 1),
    ("d128_three_chunks_ragged", 2, 3, 128, 700, 700, 300, 0, -1, None, 21),
    ("d64_window1", 1, 2, 64, 900, 900, 128, 0, 1, None, 22),
    ("window0_block_diagonal", 1, 2, 128, 640, 640, 100, 0, 0, None, 23),
    ("window2_ragged", 2, 1, 128, 1000, 1000, 257, 0, 2, None, 24),
    ("chunk1_token_causal", 1, 2, 64, 300, 300, 1, 0, -1, None, 25),
    ("chunk1_window0_diagonal", 1, 1, 128, 130, 130, 1, 0, 0, None, 26),
    ("chunk7_window1", 1, 2, 128, 333, 333, 7, 0, 1, None, 27),
    ("chunk63", 1, 2, 128, 500, 500, 63, 0, -1, None, 28),
    ("chunk64_window2", 1, 2, 128, 512, 512, 64, 0, 2, None, 29),
    ("chunk65_d64", 1, 2, 64, 520, 520, 65, 0, -1, None, 30),
    ("one_chunk_full_attention", 1, 3, 128, 777, 777, 5000, 0, -1, None, 31),
    ("stream_offset3", 2, 2, 128, 300, 1200, 300, 3, -1, None, 32),
    ("stream_offset3_window1", 1, 2, 128, 300, 1200, 300, 3, 1, None, 33),
    ("stream_ragged_chunk", 1, 2, 64, 150, 750, 300, 2, -1, None, 34),
    ("future_keys_masked", 1, 2, 128, 400, 1000, 200, 0, -1, None, 35),
    ("negative_scale", 1, 2, 128, 600, 600, 200, 0, -1, -0.05, 36),
    ("zero_scale", 1, 2, 64, 300, 300, 100, 0, 1, 0.0, 37),
    ("batch3_heads3", 3, 3, 64, 513, 513, 171, 0, -1, None, 38),
    ("single_chunk_six_tiles", 1, 1, 128, 1300, 1300, 1300, 0, -1, None, 39),
    ("single_row", 1, 1, 128, 1, 1, 1, 0, -1, None, 40),
    ("kv_longer_than_tile_window", 1, 2, 128, 260, 2600, 260, 9, 3, None, 41),
    # chunk lengths around the 96-key tile: one key short, exact, one over, two tiles
    ("chunk95", 1, 2, 128, 600, 600, 95, 0, -1, None, 42),
    ("chunk96_window2", 1, 2, 128, 768, 768, 96, 0, 2, None, 43),
    ("chunk97_d64", 1, 2, 64, 700, 700, 97, 0, -1, None, 44),
    ("chunk192_window1", 1, 2, 128, 960, 960, 192, 0, 1, None, 45),
]


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_parity_small(dev, case):
    name, B, H, d, nq, nkv, L, off, W, scale, seed = case
    scale = default_scale(d) if scale is None else scale
    _announce(f"{name} B={B} H={H} d={d} Nq={nq} Nkv={nkv} L={L} off={off} W={W} scale={scale}")
    q, k, v = make_qkv(B, nq, nkv, H, d, seed)
    # guard bands around O and LSE catch out-of-range writes
    g = 1024
    o_buf = torch.full((2 * g + B * nq * H * d,), -7777.0, dtype=torch.float32, device=dev)
    l_buf = torch.full((2 * g + B * H * nq,), -7777.0, dtype=torch.float32, device=dev)
    o = o_buf[g:g + B * nq * H * d].view(B, nq, H, d)
    lse = l_buf[g:g + B * H * nq].view(B, H, nq)
    fastvr.chunk_attn(q.to(dev), k.to(dev), v.to(dev), chunk_len=L, q_chunk_offset=off, window_chunks=W,
                      scale=scale, out=o, lse=lse)
    torch.cuda.synchronize()
    for buf, n in ((o_buf, B * nq * H * d), (l_buf, B * H * nq)):
        assert bool((buf[:g] == -7777.0).all()) and bool((buf[g + n:] == -7777.0).all()), "guard band written"
    o_ref, lse_ref = run_oracle(q, k, v, L, off, W, scale)
    compare(to_np(o), to_np(lse), o_ref, lse_ref, label=name)


def test_window0_chunk1_is_identity(dev):
    """Each token its own chunk and no earlier chunk: O_i = v_i exactly and
    LSE_i = scale * q_i . k_i."""
    _announce("window0 chunk1 identity B=1 H=2 d=128 N=300")
    q, k, v = make_qkv(1, 300, 300, 2, 128, seed=42)
    o, lse = fastvr.chunk_attn(q.to(dev), k.to(dev), v.to(dev), chunk_len=1, window_chunks=0)
    torch.cuda.synchronize()
    torch.testing.assert_close(o.cpu(), v.float(), rtol=1e-6, atol=0)
    s = (q.float() * k.float()).sum(-1).transpose(1, 2) * np.float32(default_scale(128))
    torch.testing.assert_close(lse.cpu(), s, rtol=1e-5, atol=1e-5)


def test_determinism(dev):
    _announce("determinism B=2 H=2 d=128 N=1500 L=500")
    q, k, v = (t.to(dev) for t in make_qkv(2, 1500, 1500, 2, 128, seed=43))
    a = fastvr.chunk_attn(q, k, v, chunk_len=500)
    b = fastvr.chunk_attn(q, k, v, chunk_len=500)
    torch.cuda.synchronize()
    assert torch.equal(a[0], b[0]) and torch.equal(a[1], b[1])


def test_empty_query_set_writes_nothing(dev):
    _announce("empty problem Nq=0")
    q = torch.zeros((1, 0, 2, 64), dtype=torch.bfloat16, device=dev)
    k = torch.zeros((1, 16, 2, 64), dtype=torch.bfloat16, device=dev)
    o, lse = fastvr.chunk_attn(q, k, k, chunk_len=4)
    torch.cuda.synchronize()
    assert o.shape == (1, 0, 2, 64) and lse.shape == (1, 2, 0)


def test_no_lse_pointer(dev):
    _announce("lse=NULL B=1 H=2 d=64 N=300 L=100")
    q, k, v = make_qkv(1, 300, 300, 2, 64, seed=44)
    o, lse = fastvr.chunk_attn(q.to(dev), k.to(dev), v.to(dev), chunk_len=100, return_lse=False)
    torch.cuda.synchronize()
    assert lse is None
    o_ref, _ = run_oracle(q, k, v, 100, 0, -1, default_scale(64))
    assert np.abs(to_np(o) - o_ref).max() <= 1e-2


@pytest.mark.parametrize("B,H,d,cap,cache_len,n_new", [(1, 12, 128, 1000, 0, 300), (2, 3, 64, 777, 301, 222),
                                                       (3, 2, 128, 64, 63, 1), (1, 1, 64, 500, 100, 400)])
def test_kv_append_bit_exact(dev, B, H, d, cap, cache_len, n_new):
    import oracle
    _announce(f"kv_append B={B} H={H} d={d} cap={cap} cache_len={cache_len} n_new={n_new}")
    g = torch.Generator().manual_seed(cap + n_new)
    kc = torch.randn((B, cap, H, d), generator=g).to(torch.bfloat16)
    vc = torch.randn((B, cap, H, d), generator=g).to(torch.bfloat16)
    kn = torch.randn((B, n_new, H, d), generator=g).to(torch.bfloat16)
    vn = torch.randn((B, n_new, H, d), generator=g).to(torch.bfloat16)
    kcd, vcd = kc.to(dev), vc.to(dev)
    new_len = fastvr.kv_cache_append(kcd, vcd, kn.to(dev), vn.to(dev), cache_len)
    torch.cuda.synchronize()
    assert new_len == cache_len + n_new
    k_ref, v_ref = oracle.kv_cache_append(kc.view(torch.int16).numpy(), vc.view(torch.int16).numpy(),
                                          kn.view(torch.int16).numpy(), vn.view(torch.int16).numpy(), cache_len)
    assert np.array_equal(kcd.cpu().view(torch.int16).numpy(), k_ref)
    assert np.array_equal(vcd.cpu().view(torch.int16).numpy(), v_ref)


def test_kv_append_capacity_error(dev):
    kc = torch.zeros((1, 10, 2, 64), dtype=torch.bfloat16, device=dev)
    kn = torch.zeros((1, 4, 2, 64), dtype=torch.bfloat16, device=dev)
    with pytest.raises(fastvr.FastVRError) as e:
        fastvr.kv_cache_append(kc, kc.clone(), kn, kn.clone(), cache_len=7)
    assert e.value.status == fastvr.ERR_CAPACITY


@pytest.mark.parametrize("W", [-1, 1, 2])
def test_streaming_with_cache_equals_parallel(dev, W):
    """Append each chunk to a KV cache (capacity > sequence, B = 2 so the cache
    view is strided) and attend with q_chunk_offset = chunk index: every chunk's
    rows equal the parallel call bit for bit, and a compacted cache holding
    only the W visible earlier chunks gives the same rows."""
    B, H, d, L = 2, 2, 128, 300
    n = 4 * L + 120
    _announce(f"streaming B={B} H={H} d={d} L={L} N={n} W={W}")
    q, k, v = (t.to(dev) for t in make_qkv(B, n, n, H, d, seed=50 + W))
    full_o, full_l = fastvr.chunk_attn(q, k, v, chunk_len=L, window_chunks=W)
    cap = n + 64
    kc = torch.zeros((B, cap, H, d), dtype=torch.bfloat16, device=dev)
    vc = torch.zeros_like(kc)
    cache_len = 0
    for c in range(-(-n // L)):
        s = slice(c * L, min((c + 1) * L, n))
        cache_len = fastvr.kv_cache_append(kc, vc, k[:, s].contiguous(), v[:, s].contiguous(), cache_len)
        so, sl = fastvr.chunk_attn(q[:, s], kc[:, :cache_len], vc[:, :cache_len], chunk_len=L,
                                   q_chunk_offset=c, window_chunks=W)
        torch.cuda.synchronize()
        assert torch.equal(so, full_o[:, s]), f"chunk {c}"
        assert torch.equal(sl, full_l[:, :, s]), f"chunk {c}"
        if W >= 0 and c > W:
            first = c - W
            co, cl_ = fastvr.chunk_attn(q[:, s], kc[:, first * L:cache_len], vc[:, first * L:cache_len],
                                        chunk_len=L, q_chunk_offset=W, window_chunks=W)
            torch.cuda.synchronize()
            assert torch.equal(co, full_o[:, s]), f"compacted chunk {c}"
            assert torch.equal(cl_, full_l[:, :, s]), f"compacted chunk {c}"
    o_ref, l_ref = run_oracle(q.cpu(), k.cpu(), v.cpu(), L, 0, W, default_scale(d))
    compare(to_np(full_o), to_np(full_l), o_ref, l_ref, label=f"streaming W={W}")


@pytest.mark.parametrize("strided", [False, True])
def test_bf16_output_is_the_rounded_fp32_output(dev, strided):
    """fastvr_chunk_attn_fwd_ex with o_bf16 = 1 stores the fp32 result rounded to
    bf16 (nearest even), bit for bit, also into a strided view, and the LSE is
    unchanged."""
    B, H, d, N, L = 2, 3, 128, 500, 120
    print(f"\n[gpu case] bf16 O strided={strided} B={B} H={H} d={d} N={N} L={L}", flush=True)
    q, k, v = (t.to(dev) for t in make_qkv(B, N, N, H, d, seed=44))
    o32, l32 = fastvr.chunk_attn(q, k, v, chunk_len=L, window_chunks=1)
    if strided:
        big = torch.full((B, N + 17, H, d), float("nan"), dtype=torch.bfloat16, device=dev)
        ob = big[:, 5:5 + N]
    else:
        ob = torch.empty((B, N, H, d), dtype=torch.bfloat16, device=dev)
    _, l16 = fastvr.chunk_attn(q, k, v, chunk_len=L, window_chunks=1, out=ob)
    torch.cuda.synchronize()
    assert torch.equal(ob.view(torch.int16), o32.to(torch.bfloat16).view(torch.int16))
    assert torch.equal(l16, l32)
    if strided:
        assert torch.isnan(big[:, :5].float()).all() and torch.isnan(big[:, 5 + N:].float()).all()


@pytest.mark.parametrize("W", [-1, 1])
def test_permuting_keys_within_chunks_leaves_output(dev, W):
    """Eq. 1 makes attention bidirectional inside a chunk: permuting the keys of
    every chunk (values permuted the same way) may change only the summation
    order, so O and LSE move by rounding alone; a stray token-causal mask
    inside a chunk would change them by O(1)."""
    B, H, d, N, L = 1, 2, 128, 1000, 250
    _announce(f"within-chunk key permutation W={W}")
    q, k, v = make_qkv(B, N, N, H, d, seed=77)
    g = torch.Generator().manual_seed(78)
    perm = torch.cat([c * L + torch.randperm(L, generator=g) for c in range(N // L)])
    qd, kd, vd = q.to(dev), k.to(dev), v.to(dev)
    o, lse = fastvr.chunk_attn(qd, kd, vd, chunk_len=L, window_chunks=W)
    op, lp = fastvr.chunk_attn(qd, kd[:, perm.to(dev)].contiguous(), vd[:, perm.to(dev)].contiguous(),
                               chunk_len=L, window_chunks=W)
    torch.cuda.synchronize()
    # bf16 P rounding in a different order: well inside the parity tolerance
    assert float((o - op).abs().max()) <= 2e-3, float((o - op).abs().max())
    assert float((lse - lp).abs().max()) <= 1e-4, float((lse - lp).abs().max())
