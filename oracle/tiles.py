"""fp64 CPU oracle for spatial tiling of the latent (FastVR, Sec. 3 overview and
Sec. 4.1, Inference: the DiT runs once per temporal chunk and overlapping
64 x 64 latent tile, and the restored latent is assembled from the tiles).

TEST INFRASTRUCTURE ONLY: used by tests/ and the benchmark's baseline leg; the
HIP library never imports, links or calls it.

The paper fixes the tile size and that tiles overlap; it does not give the
overlap, the tile placement or how overlapping tiles are combined.  Readings:

* Layout: a field over the latent grid is channels-last, x[b, t, y, x, c]; tiles
  span every frame t and cut only the two spatial axes, identically.
* Placement along an axis of `size` positions with tiles of `tile` and a
  requested `overlap`: tile length L = min(tile, size); n = 1 if size <= tile,
  else ceil((size - overlap) / (tile - overlap)); origins evenly spaced,
  a_k = floor((k * (size - L) + floor((n - 1) / 2)) / (n - 1)) (a_0 = 0 and
  a_{n-1} = size - L), so neighbours overlap by at least `overlap`.
* Blend: position i (0 <= i < L) of a tile has the integer axis weight
  min(i + 1, L - i, R), R = max(overlap, 1); a tile's weight at (y, x) is the
  product of its two axis weights, and the assembled value is the
  weight-normalised sum over the tiles that cover the position.  Every weight
  is positive, so the normalisation makes the blend of the tiles of any field
  return that field.
* The assembled velocity may feed the one-step update of Eq. 9 directly.
"""
from __future__ import annotations

import numpy as np


def tile_axis(size: int, tile: int, overlap: int):
    """(origins, L) of the tiles along one axis (see the module docstring)."""
    if size < 1 or tile < 1 or overlap < 0 or overlap >= tile:
        raise ValueError(f"bad tiling: size={size} tile={tile} overlap={overlap}")
    L = min(tile, size)
    if size <= tile:
        return [0], L
    n = -(-(size - overlap) // (tile - overlap))
    origins = [(k * (size - L) + (n - 1) // 2) // (n - 1) for k in range(n)]
    return origins, L


def axis_weights(L: int, overlap: int) -> np.ndarray:
    """Integer feather weights min(i + 1, L - i, R) of the L positions of a tile."""
    R = max(overlap, 1)
    i = np.arange(L)
    return np.minimum(np.minimum(i + 1, L - i), R).astype(np.float64)


def tile_gather(x, tile: int, overlap: int) -> np.ndarray:
    """x [B, T, Hg, Wg, C] -> tiles [B, ny * nx, T, Ly, Lx, C] (tile index ty * nx + tx)."""
    x = np.asarray(x)
    B, T, Hg, Wg, C = x.shape
    oy, Ly = tile_axis(Hg, tile, overlap)
    ox, Lx = tile_axis(Wg, tile, overlap)
    out = np.empty((B, len(oy) * len(ox), T, Ly, Lx, C), dtype=x.dtype)
    for ty, ay in enumerate(oy):
        for tx, ax in enumerate(ox):
            out[:, ty * len(ox) + tx] = x[:, :, ay:ay + Ly, ax:ax + Lx, :]
    return out


def tile_blend(tiles, Hg: int, Wg: int, tile: int, overlap: int) -> np.ndarray:
    """tiles [B, ny * nx, T, Ly, Lx, C] -> the weight-normalised field [B, T, Hg, Wg, C], fp64."""
    tl = np.asarray(tiles, dtype=np.float64)
    B, nt, T, Ly, Lx, C = tl.shape
    oy, Ly2 = tile_axis(Hg, tile, overlap)
    ox, Lx2 = tile_axis(Wg, tile, overlap)
    if (Ly, Lx, nt) != (Ly2, Lx2, len(oy) * len(ox)):
        raise ValueError("tile tensor does not match the grid")
    wy, wx = axis_weights(Ly, overlap), axis_weights(Lx, overlap)
    w2 = wy[:, None] * wx[None, :]
    acc = np.zeros((B, T, Hg, Wg, C))
    wsum = np.zeros((Hg, Wg))
    for ty, ay in enumerate(oy):
        for tx, ax in enumerate(ox):
            acc[:, :, ay:ay + Ly, ax:ax + Lx, :] += w2[None, None, :, :, None] * tl[:, ty * len(ox) + tx]
            wsum[ay:ay + Ly, ax:ax + Lx] += w2
    return acc / wsum[None, None, :, :, None]
