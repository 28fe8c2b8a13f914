"""Shared helpers of the GPU parity tests: tolerances, row sampling, oracle calls."""
from __future__ import annotations

import math

import numpy as np
import torch

import oracle

# Acceptance bar for the fp32 outputs against the fp64 oracle on the same
# bf16-rounded inputs: O max-abs 1e-2 and mean-abs 1e-3, LSE max-abs 1e-3.
# Stricter gate kept here as well: relative Frobenius error of O <= 5e-3
# (O is small on long sequences, so the absolute bounds alone are loose).
O_MAX_ABS = 1e-2
O_MEAN_ABS = 1e-3
LSE_MAX_ABS = 1e-3
O_REL_FRO = 5e-3


def fp32_scale(scale: float) -> float:
    """The value an fp32 `scale` argument carries."""
    return float(np.float32(scale))


def compare(o_gpu, lse_gpu, o_ref, lse_ref, label=""):
    """Element-wise comparison; returns the error statistics, asserts the bar."""
    o_gpu = np.asarray(o_gpu, dtype=np.float64)
    lse_gpu = np.asarray(lse_gpu, dtype=np.float64)
    assert np.isfinite(o_gpu).all(), f"{label}: non-finite O"
    assert np.isfinite(lse_gpu).all(), f"{label}: non-finite LSE"
    err = np.abs(o_gpu - o_ref)
    lerr = np.abs(lse_gpu - lse_ref)
    rel = float(np.linalg.norm(o_gpu - o_ref) / max(np.linalg.norm(o_ref), 1e-300))
    stats = dict(o_max=float(err.max()), o_mean=float(err.mean()), lse_max=float(lerr.max()), o_rel_fro=rel)
    print(f"[parity] {label} {stats}", flush=True)
    assert stats["o_max"] <= O_MAX_ABS, (label, stats)
    assert stats["o_mean"] <= O_MEAN_ABS, (label, stats)
    assert stats["lse_max"] <= LSE_MAX_ABS, (label, stats)
    assert stats["o_rel_fro"] <= O_REL_FRO, (label, stats)
    return stats


def sample_rows(nq: int, chunk_len: int, n_random: int, seed: int, tile: int = 256, band: int = 2):
    """Stratified query-row sample: rows within `band` of every chunk boundary and
    of every tile boundary inside a chunk, the ragged tail, and `n_random`
    uniformly drawn rows (seeded)."""
    rows = set()
    for c0 in range(0, nq, chunk_len):
        c1 = min(c0 + chunk_len, nq)
        for t0 in range(c0, c1, tile):
            for r in range(t0 - band, t0 + band + 1):
                if c0 <= r < c1:
                    rows.add(r)
        for r in range(c1 - band - 1, c1):
            if r >= c0:
                rows.add(r)
    rng = np.random.default_rng(seed)
    rows.update(rng.integers(0, nq, size=n_random).tolist())
    return np.array(sorted(rows), dtype=np.int64)


def run_oracle(q, k, v, chunk_len, q_chunk_offset, window_chunks, scale, rows=None):
    return oracle.attention(q, k, v, chunk_len=chunk_len, q_chunk_offset=q_chunk_offset,
                            window_chunks=window_chunks, scale=fp32_scale(scale), rows=rows)


def to_np(t: torch.Tensor) -> np.ndarray:
    return t.detach().to("cpu", torch.float64).numpy()


def default_scale(d: int) -> float:
    return 1.0 / math.sqrt(d)


def oracle_workers() -> int:
    """Host threads for the oracle: the CPU share of one GPU (16) at most."""
    import os
    return max(1, min(16, os.cpu_count() or 1))


def run_oracle_parallel(q, k, v, chunk_len, q_chunk_offset, window_chunks, scale, rows=None, heads=None,
                        block=1024, workers=None):
    """The fp64 oracle on many rows at once, in host threads (NumPy releases the
    GIL inside BLAS and its element-wise loops; BLAS itself runs one thread per
    worker).  Work units are (head, query chunk, block of rows).  Each unit hands
    the oracle only the keys its chunk can see, [max(0, c - W) L, min((c + 1) L,
    Nkv)), with q_chunk_offset measured from the first of them: the mask depends
    only on chunk differences, so this is the same function (the oracle's
    compacted-cache pin checks exactly that), at the cost of the visible keys.

    Returns (o [B, R, Hs, d], lse [B, Hs, R]) for the rows (sorted, all rows if
    None) and heads (all if None) asked for."""
    from concurrent.futures import ThreadPoolExecutor

    from threadpoolctl import threadpool_limits

    B, nq, H, d = q.shape
    nkv = k.shape[1]
    L = int(chunk_len)
    W = int(window_chunks)
    rows = np.arange(nq, dtype=np.int64) if rows is None else np.asarray(rows, dtype=np.int64)
    assert np.all(np.diff(rows) > 0), "rows must be sorted and distinct"
    heads = list(range(H)) if heads is None else list(heads)
    s32 = fp32_scale(scale)
    units = []
    cl = rows // L
    for local in np.unique(cl):
        idx = np.nonzero(cl == local)[0]
        c = q_chunk_offset + int(local)
        lo = max(0, c - W) * L if W >= 0 else 0
        hi = min((c + 1) * L, nkv)
        for hi_pos, h in enumerate(heads):
            for b0 in range(0, len(idx), block):
                units.append((hi_pos, h, idx[b0:b0 + block], int(local), c, lo, hi))
    o = np.zeros((B, len(rows), len(heads), d))
    lse = np.zeros((B, len(heads), len(rows)))

    def job(u):
        hp, h, idx, local, c, lo, hi = u
        qs = q[:, local * L:min((local + 1) * L, nq), h:h + 1]
        ks, vs = k[:, lo:hi, h:h + 1], v[:, lo:hi, h:h + 1]
        oo, ll = oracle.attention(qs, ks, vs, chunk_len=L, q_chunk_offset=c - lo // L, window_chunks=W,
                                  scale=s32, rows=rows[idx] - local * L)
        o[:, idx, hp] = oo[:, :, 0]
        lse[:, hp, idx] = ll[:, 0]

    with threadpool_limits(1, "blas"):
        with ThreadPoolExecutor(workers or oracle_workers()) as ex:
            for _ in ex.map(job, units):
                pass
    return o, lse
