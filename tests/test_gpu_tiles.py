"""GPU tests of spatial tiling (Sec. 3 overview, Sec. 4.1 Inference) through the
C ABI: the tile gather bit for bit, the blend and the blend fused with the
one-step update of Eq. 9 against the fp64 oracle, and attention over a tile
batch against the oracle's attention per tile.

Blend tolerance, derived from the arithmetic: the kernel sums at most K tiles
w_k v_k with fp32 fused multiply-adds (integer weights, exact in fp32) and
divides by the weight sum once, so its error is at most (K + 1) u |v|max with
u = 2^-24; K <= 9 for the geometries here, so 2e-6 |v|max bounds it with a
3x margin (plus |z| u for the fused update)."""
import numpy as np
import pytest
import torch

import oracle
from paper_2609_36757_amd import fastvr

from parity import compare, fp32_scale, to_np

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dev():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    fastvr.load()
    return torch.device("cuda:0")


# B, T, Hg, Wg, C, tile, overlap
GEOMS = [
    (1, 2, 68, 120, 48, 64, 16),   # the 1080p latent grid with the paper's 64 x 64 tiles
    (2, 3, 30, 52, 16, 64, 16),    # grid smaller than a tile: one tile
    (1, 1, 40, 33, 8, 16, 5),
    (1, 2, 9, 9, 24, 4, 3),        # heavy overlap: positions covered by several tiles
    (1, 1, 24, 36, 8, 12, 0),      # disjoint tiles
    (1, 1, 20, 70, 1536, 64, 16),  # attention-output width: a blend segment spans under 3 positions
    (1, 1, 1, 65537, 8, 2, 1),     # 65536 tiles along x: n * size > 2^32, the blend's 64-bit index path
    (1, 300, 300, 4, 8, 64, 16),   # 90000 output rows: more rows than blend workgroups along y
]


def _ids(g):
    return "x".join(str(v) for v in g)


@pytest.mark.parametrize("geom", GEOMS, ids=[_ids(g) for g in GEOMS])
def test_tile_gather_bitwise(dev, geom):
    B, T, Hg, Wg, C, tile, ov = geom
    print(f"\n[gpu case] tile_gather {geom}", flush=True)
    g = torch.Generator().manual_seed(sum(geom))
    x = torch.randn((B, T, Hg, Wg, C), generator=g).to(torch.bfloat16)
    t = fastvr.tile_gather(x.to(dev), tile=tile, overlap=ov)
    torch.cuda.synchronize()
    ref = oracle.tile_gather(x.view(torch.int16).numpy(), tile, ov)
    np.testing.assert_array_equal(t.cpu().view(torch.int16).numpy(), ref)


@pytest.mark.parametrize("geom", GEOMS, ids=[_ids(g) for g in GEOMS])
def test_tile_blend_and_update(dev, geom):
    B, T, Hg, Wg, C, tile, ov = geom
    print(f"\n[gpu case] tile_blend {geom}", flush=True)
    g = torch.Generator().manual_seed(1000 + sum(geom))
    ny, Ly = fastvr.tile_axis(Hg, tile, ov)
    nx, Lx = fastvr.tile_axis(Wg, tile, ov)
    tiles = torch.randn((B, ny * nx, T, Ly, Lx, C), generator=g)
    z = torch.randn((B, T, Hg, Wg, C), generator=g).to(torch.bfloat16)
    td = tiles.to(dev)
    out = fastvr.tile_blend(td, Hg, Wg, tile=tile, overlap=ov)
    sigma = 0.8
    upd = fastvr.tile_blend(td, Hg, Wg, tile=tile, overlap=ov, z_lq=z.to(dev), sigma=sigma)
    torch.cuda.synchronize()
    ref = oracle.tile_blend(tiles.numpy(), Hg, Wg, tile, ov)
    vmax = float(tiles.abs().max())
    err = np.abs(to_np(out) - ref).max()
    print(f"[parity] tile_blend {geom} max_abs={err:.3e} bound={2e-6 * vmax:.3e}", flush=True)
    assert err <= 2e-6 * vmax
    ref_u = oracle.one_step_update(z, ref, fp32_scale(sigma))
    err_u = np.abs(to_np(upd) - ref_u).max()
    assert err_u <= 2e-6 * (float(z.float().abs().max()) + sigma * vmax)
    # blending the gathered tiles of a field returns the field
    x = torch.randn((B, T, Hg, Wg, C), generator=g).to(torch.bfloat16)
    back = fastvr.tile_blend(fastvr.tile_gather(x.to(dev), tile=tile, overlap=ov).float(), Hg, Wg, tile=tile,
                             overlap=ov)
    torch.cuda.synchronize()
    assert np.abs(to_np(back) - x.double().numpy()).max() <= 2e-6 * float(x.float().abs().max())


def test_tiled_attention_matches_oracle_per_tile(dev):
    """q, k, v tokens on a 2-frame-per-chunk latent grid are cut into tiles, the
    tile batch runs through one chunk-causal attention call (batch = tiles), and
    every tile's output matches the oracle's attention over that tile's tokens;
    the blended output matches the oracle's blend of those per-tile outputs."""
    B, T, Hg, Wg, H, d, tile, ov, fpc = 1, 4, 20, 28, 2, 64, 16, 4, 2
    print(f"\n[gpu case] tiled attention grid {Hg}x{Wg} T={T} tile={tile} overlap={ov}", flush=True)
    g = torch.Generator().manual_seed(77)
    q, k, v = (torch.randn((B, T, Hg, Wg, H * d), generator=g).to(torch.bfloat16) for _ in range(3))
    qt, kt, vt = (fastvr.tile_gather(t.to(dev), tile=tile, overlap=ov) for t in (q, k, v))
    Bt, nt, _, Ly, Lx, _ = qt.shape
    N, L = T * Ly * Lx, fpc * Ly * Lx
    as_tokens = lambda t: t.view(Bt * nt, N, H, d)
    o, lse = fastvr.chunk_attn(as_tokens(qt), as_tokens(kt), as_tokens(vt), chunk_len=L, window_chunks=1)
    blended = fastvr.tile_blend(o.view(Bt, nt, T, Ly, Lx, H * d), Hg, Wg, tile=tile, overlap=ov)
    torch.cuda.synchronize()
    rq, rk, rv = (oracle.tile_gather(t.float().numpy(), tile, ov).reshape(Bt * nt, N, H, d) for t in (q, k, v))
    o_ref, l_ref = oracle.attention(rq, rk, rv, chunk_len=L, window_chunks=1, scale=fp32_scale(1.0 / np.sqrt(d)))
    compare(to_np(o), to_np(lse), o_ref, l_ref, label="tiled attention")
    b_ref = oracle.tile_blend(o_ref.reshape(Bt, nt, T, Ly, Lx, H * d), Hg, Wg, tile, ov)
    assert np.abs(to_np(blended) - b_ref).max() <= 1e-2


def test_tile_gather_1080p_tokens(dev):
    """The 1080p token grid at full size (8 latent frames x 68 x 120 positions,
    H * d = 1536 channels): the gather in the launch configuration the
    benchmark times, checked bit for bit on every tile's corner rows."""
    shape = (1, 8, 68, 120, 1536)
    print(f"\n[gpu case] tile_gather 1080p tokens {shape}", flush=True)
    g = torch.Generator().manual_seed(5)
    x = torch.randn(shape, generator=g).to(torch.bfloat16)
    t = fastvr.tile_gather(x.to(dev), tile=64, overlap=16).cpu()
    oy, L = oracle.tile_axis(68, 64, 16)
    ox, _ = oracle.tile_axis(120, 64, 16)
    assert t.shape == (1, len(oy) * len(ox), 8, L, L, 1536)
    for ty, ay in enumerate(oy):
        for tx, ax in enumerate(ox):
            for fr in (0, 7):
                for iy in (0, L - 1):
                    assert torch.equal(t[0, ty * len(ox) + tx, fr, iy], x[0, fr, ay + iy, ax:ax + L])
