"""Work accounting for chunk-causal attention.

Effective FLOPs count only visible (query, key) pairs: 2*d flops for the score
and 2*d for the P.V product per pair, over every batch and head.  Masked
chunks and tile padding are not counted."""
from __future__ import annotations


def kv_interval(c: int, nkv: int, chunk_len: int, window_chunks: int):
    """Keys visible to a query in global chunk c form one contiguous range
    [lo, hi): chunk indices max(0, c - W) .. c, clipped to the key count."""
    lo_chunk = 0 if window_chunks < 0 else max(0, c - window_chunks)
    return lo_chunk * chunk_len, min((c + 1) * chunk_len, nkv)


def visible_pairs(nq: int, nkv: int, chunk_len: int, q_chunk_offset: int = 0,
                  window_chunks: int = -1) -> int:
    """Closed-form count of visible (query, key) pairs for one (batch, head)."""
    total = 0
    n_local = -(-nq // chunk_len)
    for cl in range(n_local):
        rows = min((cl + 1) * chunk_len, nq) - cl * chunk_len
        lo, hi = kv_interval(q_chunk_offset + cl, nkv, chunk_len, window_chunks)
        total += rows * max(0, hi - lo)
    return total


def effective_flops(B: int, H: int, d: int, nq: int, nkv: int, chunk_len: int,
                    q_chunk_offset: int = 0, window_chunks: int = -1) -> int:
    return 4 * d * B * H * visible_pairs(nq, nkv, chunk_len, q_chunk_offset, window_chunks)


def algorithmic_bytes(B: int, H: int, d: int, nq: int, nkv: int, with_lse: bool = True) -> int:
    """Compulsory HBM traffic of one attention call: Q, K, V read once (bf16),
    O written once (fp32), LSE written once (fp32)."""
    qkv = 2 * B * H * d * (nq + 2 * nkv)
    o = 4 * B * H * d * nq
    lse = 4 * B * H * nq if with_lse else 0
    return qkv + o + lse
