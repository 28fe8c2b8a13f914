"""Plain fp64 CPU oracle for chunk-wise causal self-attention (FastVR, Sec. 3.1).

TEST INFRASTRUCTURE ONLY.  Nothing on the product path may import, call or link
this module: only the test suite, the smoke check and the benchmark's
``cpu_baseline`` leg use it.  It shares no code with the HIP library.

What is computed (Sec. 3.1, Eq. 1 and the paragraph after it):

* Latent tokens are flattened frame-major, so a chunk of ``k`` latent frames is
  a contiguous token range of ``chunk_len = k * tokens_per_frame`` tokens and
  the frame-level mask of Eq. 1 becomes a token-level mask on
  ``floor(token / chunk_len)``.
* Query row ``i`` belongs to chunk ``cq(i) = q_chunk_offset + i // chunk_len``,
  key row ``j`` to chunk ``ck(j) = j // chunk_len``.  Key ``j`` is visible to
  query ``i`` when ``0 <= cq(i) - ck(j) <= W``.  Eq. 1 is ``W = 1`` ("itself and
  its immediate predecessor"); ``window_chunks = -1`` means no upper bound (an
  unbounded causal prefix of chunks).  Inside a chunk attention is
  bidirectional.
* ``LSE_i = ln sum_{j visible} exp(scale * q_i . k_j)`` and
  ``O_i = sum_{j visible} exp(scale * q_i . k_j - LSE_i) v_j``.
* The parallel (training) form over the whole sequence and the streaming form
  (one query chunk against a KV cache, ``q_chunk_offset`` = its chunk index)
  are the same function (Sec. 3.1, last paragraph).

Everything is evaluated in float64 from the given inputs (bf16 inputs are
widened exactly).  ``scale`` is used exactly as passed; callers that model an
fp32 interface pass the fp32-rounded value.
"""
from __future__ import annotations

import math

import numpy as np


# ---------------------------------------------------------------------------
# Mask (Eq. 1, generalised to a window of W previous chunks)
# ---------------------------------------------------------------------------

def query_chunks(nq: int, chunk_len: int, q_chunk_offset: int = 0) -> np.ndarray:
    """Chunk index of every query row: q_chunk_offset + i // chunk_len."""
    return q_chunk_offset + np.arange(nq, dtype=np.int64) // chunk_len


def key_chunks(nkv: int, chunk_len: int) -> np.ndarray:
    """Chunk index of every key row: j // chunk_len."""
    return np.arange(nkv, dtype=np.int64) // chunk_len


def visibility_mask(nq: int, nkv: int, chunk_len: int, q_chunk_offset: int = 0,
                    window_chunks: int = -1, rows=None) -> np.ndarray:
    """Explicit boolean mask [len(rows), nkv]: True where key j is visible to query i.

    Eq. 1 with the chunk difference allowed in {0..W} (W = -1: any non-negative
    difference)."""
    cq = query_chunks(nq, chunk_len, q_chunk_offset)
    if rows is not None:
        cq = cq[np.asarray(rows, dtype=np.int64)]
    ck = key_chunks(nkv, chunk_len)
    diff = cq[:, None] - ck[None, :]
    vis = diff >= 0
    if window_chunks >= 0:
        vis &= diff <= window_chunks
    return vis


def frame_mask(num_frames: int, frames_per_chunk: int, window_chunks: int = 1) -> np.ndarray:
    """Eq. 1 at the level of latent frames: M[i, j] = 1 iff floor(i/k) - floor(j/k)
    lies in {0..W} (the paper's W is 1)."""
    f = np.arange(num_frames, dtype=np.int64) // frames_per_chunk
    diff = f[:, None] - f[None, :]
    m = diff >= 0
    if window_chunks >= 0:
        m &= diff <= window_chunks
    return m


def count_visible_pairs(nq: int, nkv: int, chunk_len: int, q_chunk_offset: int = 0,
                        window_chunks: int = -1, block: int = 4096) -> int:
    """Number of visible (query, key) pairs, counted from the explicit mask."""
    total = 0
    for r0 in range(0, nq, block):
        rows = np.arange(r0, min(nq, r0 + block))
        total += int(visibility_mask(nq, nkv, chunk_len, q_chunk_offset,
                                     window_chunks, rows=rows).sum())
    return total


# ---------------------------------------------------------------------------
# Masked softmax attention, straight from the definition
# ---------------------------------------------------------------------------

def _as_f64(x) -> np.ndarray:
    if hasattr(x, "detach"):  # a torch tensor; bf16 has no numpy dtype
        import torch
        x = x.detach().to("cpu", torch.float64).numpy()
    return np.asarray(x, dtype=np.float64)


def _head_f64(x, b: int, h: int, rows=None) -> np.ndarray:
    """x[b, rows, h, :] widened to float64 (rows=None: all rows)."""
    if hasattr(x, "detach"):
        import torch
        sl = x[b, :, h, :] if rows is None else x[b, torch.as_tensor(rows), h, :]
        return sl.detach().to("cpu", torch.float64).numpy()
    x = np.asarray(x)
    sl = x[b, :, h, :] if rows is None else x[b, rows, h, :]
    return np.asarray(sl, dtype=np.float64)


def attention(q, k, v, chunk_len: int, q_chunk_offset: int = 0, window_chunks: int = -1,
              scale: float | None = None, rows=None, block: int = 512):
    """Chunk-causal attention in fp64.

    q: [B, Nq, H, d]; k, v: [B, Nkv, H, d] (numpy arrays or CPU torch tensors).
    rows: optional 1-D array of query-row indices to evaluate (all rows if None).
    Returns (o [B, R, H, d] float64, lse [B, H, R] float64) with R = number of rows.

    Per (b, h) and block of query rows: S = scale * Q K^T, S = -inf where the mask
    hides the key, m = rowmax S, P = exp(S - m), l = rowsum P, O = P V / l,
    LSE = m + ln l."""
    B, nq, H, d = q.shape
    nkv = k.shape[1]
    if scale is None:
        scale = 1.0 / math.sqrt(d)
    scale = float(scale)
    rows = np.arange(nq, dtype=np.int64) if rows is None else np.asarray(rows, dtype=np.int64)
    R = rows.shape[0]
    o = np.zeros((B, R, H, d), dtype=np.float64)
    lse = np.zeros((B, H, R), dtype=np.float64)
    for b in range(B):
        for h in range(H):
            kh = _head_f64(k, b, h)
            vh = _head_f64(v, b, h)
            for r0 in range(0, R, block):
                rr = rows[r0:r0 + block]
                vis = visibility_mask(nq, nkv, chunk_len, q_chunk_offset, window_chunks, rows=rr)
                if not vis.any(axis=1).all():
                    raise ValueError("a query row has no visible key")
                s = scale * (_head_f64(q, b, h, rr) @ kh.T)
                s = np.where(vis, s, -np.inf)
                m = s.max(axis=1, keepdims=True)
                p = np.exp(s - m)
                l = p.sum(axis=1, keepdims=True)
                o[b, r0:r0 + len(rr), h, :] = (p @ vh) / l
                lse[b, h, r0:r0 + len(rr)] = (m + np.log(l))[:, 0]
    return o, lse


def softmax_weights(q, k, chunk_len: int, q_chunk_offset: int = 0, window_chunks: int = -1,
                    scale: float | None = None, b: int = 0, h: int = 0) -> np.ndarray:
    """The attention weights P [Nq, Nkv] of one (b, h), masked entries exactly 0.
    For small inputs only (exposes the normalisation invariant)."""
    q = _as_f64(q)
    k = _as_f64(k)
    nq, d = q.shape[1], q.shape[3]
    nkv = k.shape[1]
    if scale is None:
        scale = 1.0 / math.sqrt(d)
    vis = visibility_mask(nq, nkv, chunk_len, q_chunk_offset, window_chunks)
    s = np.where(vis, float(scale) * (q[b, :, h, :] @ k[b, :, h, :].T), -np.inf)
    p = np.exp(s - s.max(axis=1, keepdims=True))
    return p / p.sum(axis=1, keepdims=True)


# ---------------------------------------------------------------------------
# Brute force at the level of latent frames (Eq. 1 exactly as printed)
# ---------------------------------------------------------------------------

def brute_force(q, k, v, tokens_per_frame: int, frames_per_chunk: int,
                q_chunk_offset: int = 0, window_chunks: int = 1,
                scale: float | None = None):
    """Pure-Python loops, for tiny inputs only.

    The token n lies in latent frame n // tokens_per_frame; frames are grouped in
    chunks of ``frames_per_chunk`` (k of Eq. 1).  Query row i lies in frame
    q_chunk_offset * frames_per_chunk + i // tokens_per_frame.  Eq. 1's test
    floor(fi/k) - floor(fj/k) in {0..W} decides visibility.  Dot products and sums
    use math.fsum; the softmax is evaluated with the row maximum subtracted."""
    q = _as_f64(q)
    k = _as_f64(k)
    v = _as_f64(v)
    B, nq, H, d = q.shape
    nkv = k.shape[1]
    if scale is None:
        scale = 1.0 / math.sqrt(d)
    o = np.zeros((B, nq, H, d))
    lse = np.zeros((B, H, nq))
    for b in range(B):
        for h in range(H):
            for i in range(nq):
                fi = q_chunk_offset * frames_per_chunk + i // tokens_per_frame
                ci = fi // frames_per_chunk
                vis_j = []
                for j in range(nkv):
                    cj = (j // tokens_per_frame) // frames_per_chunk
                    delta = ci - cj
                    if delta >= 0 and (window_chunks < 0 or delta <= window_chunks):
                        vis_j.append(j)
                if not vis_j:
                    raise ValueError("a query row has no visible key")
                scores = [scale * math.fsum(q[b, i, h, x] * k[b, j, h, x] for x in range(d))
                          for j in vis_j]
                mx = max(scores)
                w = [math.exp(s - mx) for s in scores]
                tot = math.fsum(w)
                lse[b, h, i] = mx + math.log(tot)
                for x in range(d):
                    o[b, i, h, x] = math.fsum(wj * v[b, j, h, x] for wj, j in zip(w, vis_j)) / tot
    return o, lse


# ---------------------------------------------------------------------------
# KV cache append (streaming inference with KV caching, Sec. 3.1)
# ---------------------------------------------------------------------------

def kv_cache_append(k_cache, v_cache, k_new, v_new, cache_len: int):
    """Return copies of the caches ([B, capacity, H, d]) with the new tokens
    ([B, n_new, H, d]) written at token offset cache_len.  No eviction."""
    kc = np.array(k_cache, copy=True)
    vc = np.array(v_cache, copy=True)
    n_new = np.shape(k_new)[1]
    if cache_len + n_new > kc.shape[1]:
        raise ValueError("append would overflow the cache")
    kc[:, cache_len:cache_len + n_new] = k_new
    vc[:, cache_len:cache_len + n_new] = v_new
    return kc, vc


# ---------------------------------------------------------------------------
# Bounded ring KV cache (streaming with an O(k) cache, Sec. 3.1, last paragraph)
# ---------------------------------------------------------------------------

def ring_slot(chunk_index: int, window_chunks: int) -> int:
    """Slot of chunk ``chunk_index`` in a ring of ``window_chunks + 1`` chunk slots."""
    return chunk_index % (window_chunks + 1)


def ring_step(k_ring, v_ring, q_new, k_new, v_new, chunk_len: int, chunk_index: int,
              window_chunks: int, scale=None):
    """One streaming step with a ring cache of W + 1 chunk slots.

    The ring ([B, (W + 1) * chunk_len, H, d]) holds chunk c in token rows
    ``[slot * chunk_len, slot * chunk_len + chunk_len)`` with
    ``slot = c mod (W + 1)``.  The step writes the new chunk c (``n_new <=
    chunk_len`` tokens of queries, keys and values) into its slot and returns
    the attention of its queries over the keys of chunks ``max(0, c - W) .. c``,
    read from the ring in chunk order, with the chunk-causal mask of Eq. 1
    (queries of chunk c see all of those keys; inside chunk c attention is
    bidirectional).  Earlier chunks are taken as full (``chunk_len`` tokens).

    Returns ``(o, lse, k_ring_after, v_ring_after)``.  The memory of the ring
    stays ``W + 1`` chunks however long the stream is, which is the paper's
    O(k) cache for a fixed chunk size."""
    W = int(window_chunks)
    if W < 0:
        raise ValueError("a ring cache needs a bounded window (window_chunks >= 0)")
    L = int(chunk_len)
    c = int(chunk_index)
    kr = np.array(k_ring, copy=True)
    vr = np.array(v_ring, copy=True)
    n_new = np.shape(k_new)[1]
    if not 1 <= n_new <= L:
        raise ValueError("the new chunk must hold 1 .. chunk_len tokens")
    if kr.shape[1] != (W + 1) * L:
        raise ValueError("the ring must hold (window_chunks + 1) * chunk_len tokens")
    s = ring_slot(c, W)
    kr[:, s * L:s * L + n_new] = k_new
    vr[:, s * L:s * L + n_new] = v_new
    # gather the visible chunks in chunk order: c - n_prev .. c
    n_prev = min(c, W)
    ks, vs = [], []
    for cc in range(c - n_prev, c + 1):
        sc = ring_slot(cc, W)
        rows = L if cc < c else n_new
        ks.append(kr[:, sc * L:sc * L + rows])
        vs.append(vr[:, sc * L:sc * L + rows])
    k_seq = np.concatenate(ks, axis=1)
    v_seq = np.concatenate(vs, axis=1)
    # in the gathered sequence the new chunk has chunk index n_prev
    o, lse = attention(q_new, k_seq, v_seq, chunk_len=L, q_chunk_offset=n_prev,
                       window_chunks=W, scale=scale)
    return o, lse, kr, vr


# ---------------------------------------------------------------------------
# Backward pass (training-mode gradients of the chunk-causal attention)
# ---------------------------------------------------------------------------

def attention_bwd(q, k, v, do, chunk_len: int, q_chunk_offset: int = 0, window_chunks: int = -1,
                  scale: float | None = None, block: int = 512, rows=None):
    """Gradients of O = softmax(scale * Q K^T + mask) V with respect to q, k, v.

    The paper trains the DiT with the whole latent sequence in parallel under
    the chunk mask (Sec. 3.1), so training needs these gradients; the mask is
    fixed, so it only removes terms.  Given the upstream gradient do
    ([B, Nq, H, d]), per (b, h) with P the masked softmax weights:

        dV = P^T dO
        dP = dO V^T
        dS = P * (dP - rowsum(dP * P))      (softmax Jacobian, row by row)
        dQ = scale * dS K
        dK = scale * dS^T Q

    rowsum(dP * P) equals rowsum(dO * O) because O = P V.  Everything in
    float64.  Returns (dq [B, Nq, H, d], dk [B, Nkv, H, d], dv [B, Nkv, H, d]).

    rows: optional 1-D array of query rows.  Then only those rows' terms are
    summed: dq holds the gradient of exactly those rows ([B, R, H, d]; row i of
    dQ depends on query row i alone) and dk / dv hold those rows' contributions
    (the full dK / dV when every query that sees a key is among the rows)."""
    B, nq, H, d = q.shape
    nkv = k.shape[1]
    if scale is None:
        scale = 1.0 / math.sqrt(d)
    scale = float(scale)
    rows = np.arange(nq, dtype=np.int64) if rows is None else np.asarray(rows, dtype=np.int64)
    R = rows.shape[0]
    dq = np.zeros((B, R, H, d))
    dk = np.zeros((B, nkv, H, d))
    dv = np.zeros((B, nkv, H, d))
    for b in range(B):
        for h in range(H):
            kh = _head_f64(k, b, h)
            vh = _head_f64(v, b, h)
            for r0 in range(0, R, block):
                rr = rows[r0:r0 + block]
                vis = visibility_mask(nq, nkv, chunk_len, q_chunk_offset, window_chunks, rows=rr)
                qh = _head_f64(q, b, h, rr)
                doh = _head_f64(do, b, h, rr)
                s = np.where(vis, scale * (qh @ kh.T), -np.inf)
                p = np.exp(s - s.max(axis=1, keepdims=True))
                p /= p.sum(axis=1, keepdims=True)
                dp = doh @ vh.T
                ds = p * (dp - (p * dp).sum(axis=1, keepdims=True))
                dq[b, r0:r0 + len(rr), h] = scale * (ds @ kh)
                dk[b, :, h] += scale * (ds.T @ qh)
                dv[b, :, h] += p.T @ doh
    return dq, dk, dv


def attention_bwd_keys(q, k, v, do, keys, lse, delta, chunk_len: int, q_chunk_offset: int = 0,
                       window_chunks: int = -1, scale: float | None = None):
    """dK and dV of the key rows ``keys`` only, from the per-query row terms.

    For key j, with the queries i that see it (Eq. 1 mask):
        P_ij  = exp(scale * q_i . k_j - LSE_i)
        dS_ij = P_ij * (dO_i . v_j - D_i)
        dV_j  = sum_i P_ij dO_i,      dK_j = scale * sum_i dS_ij q_i
    lse and delta are [B, H, Nq] (LSE_i and D_i = rowsum(dO * O)_i, e.g. from
    ``attention`` and ``attention_bwd_delta``); entries of queries that see none
    of the keys are never read.  Returns (dk, dv), each [B, len(keys), H, d],
    float64."""
    B, nq, H, d = q.shape
    nkv = k.shape[1]
    if scale is None:
        scale = 1.0 / math.sqrt(d)
    scale = float(scale)
    keys = np.asarray(keys, dtype=np.int64)
    cq = query_chunks(nq, chunk_len, q_chunk_offset)
    ck = key_chunks(nkv, chunk_len)[keys]
    diff = cq[None, :] - ck[:, None]                      # [K, Nq]
    vis = diff >= 0
    if window_chunks >= 0:
        vis &= diff <= window_chunks
    lse = np.asarray(lse, dtype=np.float64)
    delta = np.asarray(delta, dtype=np.float64)
    dk = np.zeros((B, len(keys), H, d))
    dv = np.zeros((B, len(keys), H, d))
    for b in range(B):
        for h in range(H):
            for t, j in enumerate(keys):
                ii = np.nonzero(vis[t])[0]
                if ii.size == 0:
                    continue
                qh = _head_f64(q, b, h, ii)
                doh = _head_f64(do, b, h, ii)
                kj = _head_f64(k, b, h, np.array([j]))[0]
                vj = _head_f64(v, b, h, np.array([j]))[0]
                p = np.exp(scale * (qh @ kj) - lse[b, h, ii])
                ds = p * (doh @ vj - delta[b, h, ii])
                dv[b, t, h] = p @ doh
                dk[b, t, h] = scale * (ds @ qh)
    return dk, dv


def attention_bwd_delta(o, do) -> np.ndarray:
    """D[b, h, i] = sum_d dO[b, i, h, d] * O[b, i, h, d] (fp64), the row term of
    the softmax backward, [B, H, Nq]."""
    o64, do64 = _as_f64(o), _as_f64(do)
    return np.einsum("bihd,bihd->bhi", o64, do64)
