"""Seeded synthetic inputs for chunk-causal attention.

This module only draws and shapes random tensors; it holds none of the
attention arithmetic, so both the fp64 oracle (through the tests) and the HIP
path can be fed from it.

Latent-token grids follow the paper's 2-latent-frame chunks on a Wan-style
latent: 1080p -> 68 x 120 = 8160 tokens per latent frame, 480p -> 30 x 52 =
1560.  Tokens are flattened frame-major, so a chunk is a contiguous range of
``frames_per_chunk * tokens_per_frame`` tokens.  All tensors are BNHD
(batch, token, head, head_dim), drawn as float32 N(0, 1) from a CPU
``torch.Generator`` and rounded once to bfloat16 (round-to-nearest-even).
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field

import torch


@dataclass(frozen=True)
class Workload:
    name: str
    B: int
    H: int
    d: int
    chunk_len: int          # tokens per chunk
    n_tokens: int           # tokens in the whole latent sequence
    window_chunks: int      # -1: unbounded causal prefix of chunks
    seed: int
    scale: float
    k_head_offset_std: float = 0.0   # per-head mean offset added to every K row
    k_outlier_frac: float = 0.0      # fraction of K token rows scaled by k_outlier_mult
    k_outlier_mult: float = 1.0
    # streaming step: query = chunk `stream_chunk`, KV = chunks 0..stream_chunk
    stream_chunk: int | None = None
    note: str = field(default="", compare=False)

    @property
    def n_chunks(self) -> int:
        return -(-self.n_tokens // self.chunk_len)


WORKLOADS = {
    "tiny": Workload("tiny", B=1, H=2, d=64, chunk_len=256, n_tokens=1024, window_chunks=-1,
                     seed=1, scale=1.0 / 8.0,
                     note="4 chunks x 256 tokens, full causal prefix"),
    "480p": Workload("480p", B=1, H=12, d=128, chunk_len=3120, n_tokens=18720, window_chunks=-1,
                     seed=2, scale=1.0 / math.sqrt(128), k_head_offset_std=0.5,
                     note="30x52 tokens/frame, 2 frames/chunk, 6 chunks, full causal prefix"),
    "1080p": Workload("1080p", B=1, H=12, d=128, chunk_len=16320, n_tokens=65280, window_chunks=-1,
                      seed=3, scale=1.0 / math.sqrt(128),
                      note="68x120 tokens/frame, 2 frames/chunk, 4 chunks, full causal prefix"),
    "1080p_stream": Workload("1080p_stream", B=1, H=12, d=128, chunk_len=16320, n_tokens=65280,
                             window_chunks=-1, seed=3, scale=1.0 / math.sqrt(128), stream_chunk=3,
                             note="chunk 3 of the 1080p sequence against a cache of chunks 0-3"),
    "wide_sw": Workload("wide_sw", B=1, H=24, d=128, chunk_len=16320, n_tokens=138720,
                        window_chunks=2, seed=5, scale=1.0 / math.sqrt(128),
                        k_outlier_frac=0.01, k_outlier_mult=8.0,
                        note="8 x 16320 + 8160 tokens, own chunk + 2 previous, 1% K rows x8"),
}


def randn_bf16(shape, gen: torch.Generator) -> torch.Tensor:
    """float32 N(0,1) draws rounded once to bfloat16."""
    return torch.randn(shape, generator=gen, dtype=torch.float32).to(torch.bfloat16)


def make_qkv(B: int, nq: int, nkv: int, H: int, d: int, seed: int):
    """Independent N(0,1) q [B,nq,H,d], k and v [B,nkv,H,d], bf16, on the CPU."""
    g = torch.Generator(device="cpu").manual_seed(seed)
    q = randn_bf16((B, nq, H, d), g)
    k = randn_bf16((B, nkv, H, d), g)
    v = randn_bf16((B, nkv, H, d), g)
    return q, k, v


def make_sequence(w: Workload):
    """q, k, v for the whole latent sequence of workload ``w`` (bf16, CPU).

    Draw order: Q, K, V (float32 [B, N, H, d]), then the extras:
    * per-head K offset mu_h in R^d, components N(0, std^2), added to every K row
      of head h before rounding;
    * outliers: round(frac * N) token rows chosen without replacement, K scaled
      by ``k_outlier_mult`` in every head (a power of two, so exact in bf16)."""
    g = torch.Generator(device="cpu").manual_seed(w.seed)
    shape = (w.B, w.n_tokens, w.H, w.d)
    q = torch.randn(shape, generator=g, dtype=torch.float32)
    k = torch.randn(shape, generator=g, dtype=torch.float32)
    v = torch.randn(shape, generator=g, dtype=torch.float32)
    if w.k_head_offset_std:
        mu = torch.randn((w.H, w.d), generator=g, dtype=torch.float32) * w.k_head_offset_std
        k += mu[None, None]
    if w.k_outlier_frac:
        n_out = int(round(w.k_outlier_frac * w.n_tokens))
        idx = torch.randperm(w.n_tokens, generator=g)[:n_out]
        k[:, idx] *= w.k_outlier_mult
    return q.to(torch.bfloat16), k.to(torch.bfloat16), v.to(torch.bfloat16)


def streaming_views(w: Workload, q, k, v):
    """For a streaming workload: the new query chunk, the new chunk's K/V, and the
    cached prefix it is appended to, all as slices of the full-sequence tensors."""
    c = w.stream_chunk
    L = w.chunk_len
    lo, hi = c * L, min((c + 1) * L, w.n_tokens)
    return dict(q_new=q[:, lo:hi], k_new=k[:, lo:hi], v_new=v[:, lo:hi],
                k_prefix=k[:, :lo], v_prefix=v[:, :lo], q_chunk_offset=c, cache_len=lo,
                n_kv=hi)
