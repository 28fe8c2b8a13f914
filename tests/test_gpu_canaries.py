"""Out-of-bounds write checks on the GPU: every output of every entry point is
a view into a larger buffer whose guard regions before and after hold a
sentinel, and must still hold it after the call (ragged sizes, tails of tiles
and of grid-stride loops)."""
import numpy as np
import pytest
import torch

from paper_2609_36757_amd import fastvr
from paper_2609_36757_amd.workloads import make_qkv

pytestmark = pytest.mark.gpu

PAD = 4096  # guard elements on each side (a multiple of 8, so views stay 16-byte aligned)


@pytest.fixture(scope="module")
def dev():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    fastvr.load()
    return torch.device("cuda:0")


def _guarded(shape, dtype, dev):
    n = int(np.prod(shape))
    buf = torch.empty(n + 2 * PAD, dtype=dtype, device=dev)
    if dtype == torch.bfloat16:
        buf.view(torch.int16).fill_(0x7F7F)      # a finite bf16 pattern kernels never produce here
    else:
        buf.fill_(-12345.678)
    return buf, buf[PAD:PAD + n].view(shape)


def _intact(buf, label):
    torch.cuda.synchronize()
    if buf.dtype == torch.bfloat16:
        head, tail = buf[:PAD].view(torch.int16), buf[-PAD:].view(torch.int16)
        ok = bool((head == 0x7F7F).all()) and bool((tail == 0x7F7F).all())
    else:
        ok = bool((buf[:PAD] == -12345.678).all()) and bool((buf[-PAD:] == -12345.678).all())
    assert ok, f"{label}: a guard region was overwritten"


def test_forward_and_backward_guards(dev):
    B, H, d, N, L = 2, 3, 128, 333, 70
    print(f"\n[gpu case] canaries fwd/bwd B={B} H={H} d={d} N={N} L={L}", flush=True)
    q, k, v = (t.to(dev) for t in make_qkv(B, N, N, H, d, seed=9))
    bo, o = _guarded((B, N, H, d), torch.float32, dev)
    bl, lse = _guarded((B, H, N), torch.float32, dev)
    fastvr.chunk_attn(q, k, v, chunk_len=L, window_chunks=1, out=o, lse=lse)
    _intact(bo, "o")
    _intact(bl, "lse")
    do = torch.randn((B, N, H, d), device=dev).to(torch.bfloat16)
    bufs = [_guarded(s, torch.float32, dev) for s in ((B, N, H, d), (B, N, H, d), (B, N, H, d), (B, H, 2, N))]
    fastvr.chunk_attn_bwd(q, k, v, o, lse, do, chunk_len=L, window_chunks=1, dq=bufs[0][1], dk=bufs[1][1],
                          dv=bufs[2][1], row_stats=bufs[3][1])
    for (b, _), name in zip(bufs, ("dq", "dk", "dv", "row_stats")):
        _intact(b, name)


def test_ring_step_and_append_guards(dev):
    B, H, d, L, W = 1, 2, 64, 72, 2
    print(f"\n[gpu case] canaries ring step B={B} H={H} d={d} L={L} W={W}", flush=True)
    q, k, v = (t.to(dev) for t in make_qkv(B, L, L, H, d, seed=10))
    brk, rk = _guarded((B, (W + 1) * L, H, d), torch.bfloat16, dev)
    brv, rv = _guarded((B, (W + 1) * L, H, d), torch.bfloat16, dev)
    bo, o = _guarded((B, L, H, d), torch.float32, dev)
    bl, lse = _guarded((B, H, L), torch.float32, dev)
    for c in range(4):
        fastvr.chunk_attn_ring_step(q, k, v, rk, rv, chunk_len=L, chunk_index=c, window_chunks=W, out=o, lse=lse)
    for b, name in ((brk, "k_ring"), (brv, "v_ring"), (bo, "o"), (bl, "lse")):
        _intact(b, name)
    bkc, kc = _guarded((B, 3 * L, H, d), torch.bfloat16, dev)
    bvc, vc = _guarded((B, 3 * L, H, d), torch.bfloat16, dev)
    fastvr.kv_cache_append(kc, vc, k, v, 2 * L)
    _intact(bkc, "k_cache")
    _intact(bvc, "v_cache")


@pytest.mark.parametrize("n", [7, 4099, 100003])
def test_one_step_guards(dev, n):
    print(f"\n[gpu case] canaries one_step n={n}", flush=True)
    z = torch.randn(n, device=dev).to(torch.bfloat16)
    v = torch.randn(n, device=dev).to(torch.bfloat16)
    bf, of = _guarded((n,), torch.float32, dev)
    fastvr.one_step_update(z, v, 0.5, out=of)
    _intact(bf, "z_hat fp32")
    bb, ob = _guarded((n,), torch.bfloat16, dev)
    fastvr.one_step_update(z, v, 0.5, out=ob)
    _intact(bb, "z_hat bf16")


def test_tile_guards(dev):
    B, T, Hg, Wg, C, tile, ov = 1, 2, 21, 37, 24, 16, 5
    print(f"\n[gpu case] canaries tiles {(B, T, Hg, Wg, C, tile, ov)}", flush=True)
    x = torch.randn((B, T, Hg, Wg, C), device=dev).to(torch.bfloat16)
    ny, Ly = fastvr.tile_axis(Hg, tile, ov)
    nx, Lx = fastvr.tile_axis(Wg, tile, ov)
    bt, t = _guarded((B, ny * nx, T, Ly, Lx, C), torch.bfloat16, dev)
    fastvr.tile_gather(x, tile=tile, overlap=ov, out=t)
    _intact(bt, "tiles")
    bo, o = _guarded((B, T, Hg, Wg, C), torch.float32, dev)
    fastvr.tile_blend(t.float(), Hg, Wg, tile=tile, overlap=ov, out=o)
    _intact(bo, "blend out")
    bu, u = _guarded((B, T, Hg, Wg, C), torch.float32, dev)
    fastvr.tile_blend(t.float(), Hg, Wg, tile=tile, overlap=ov, z_lq=x, sigma=0.3, out=u)
    _intact(bu, "blend-update out")
