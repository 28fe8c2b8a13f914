"""ctypes binding of libfastvr.so (declared in include/fastvr.h).

Argument marshalling only: every step of the computation runs in the HIP
kernels of the library.  torch tensors provide device memory and the stream.
If the library is missing, every call raises; there is no fallback."""
from __future__ import annotations

import ctypes
import math
import os

PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(PKG, "libfastvr.so")

OK = 0
ERR_INVALID_ARGUMENT = 1
ERR_UNSUPPORTED = 2
ERR_CAPACITY = 3
ERR_HIP = 4

EXPORTED = ("fastvr_chunk_attn_fwd", "fastvr_chunk_attn_fwd_ex", "fastvr_kv_cache_append",
            "fastvr_chunk_attn_ring_step", "fastvr_chunk_attn_bwd", "fastvr_chunk_attn_bwd_noalloc",
            "fastvr_one_step_update",
            "fastvr_tile_axis", "fastvr_tile_gather", "fastvr_tile_blend", "fastvr_tile_blend_update",
            "fastvr_status_string", "fastvr_last_error", "fastvr_abi_version")

_i64 = ctypes.c_int64
_vp = ctypes.c_void_p
_LIB = None


class FastVRError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(message)
        self.status = status


def load() -> ctypes.CDLL:
    """Load the in-tree libfastvr.so (built by ``python -m paper_2609_36757_amd.build``)."""
    global _LIB
    if _LIB is not None:
        return _LIB
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is missing: build it with `python -m paper_2609_36757_amd.build`")
    lib = ctypes.CDLL(LIB_PATH)
    lib.fastvr_chunk_attn_fwd.restype = ctypes.c_int
    lib.fastvr_chunk_attn_fwd.argtypes = [_vp, _vp, _vp, _vp, _vp, _i64, _i64, _i64, _i64, _i64, _i64, _i64,
                                          _i64, ctypes.c_float, _vp]
    lib.fastvr_chunk_attn_fwd_ex.restype = ctypes.c_int
    lib.fastvr_chunk_attn_fwd_ex.argtypes = [_vp, _i64, _i64, _vp, _i64, _i64, _vp, _i64, _i64, _vp, _i64, _i64,
                                             ctypes.c_int32, _vp, _i64, _i64, _i64, _i64, _i64, _i64, _i64, _i64,
                                             ctypes.c_float, _vp]
    lib.fastvr_kv_cache_append.restype = ctypes.c_int
    lib.fastvr_kv_cache_append.argtypes = [_vp, _vp, _vp, _vp, _i64, _i64, _i64, _i64, _i64, _i64, _vp]
    lib.fastvr_chunk_attn_ring_step.restype = ctypes.c_int
    lib.fastvr_chunk_attn_ring_step.argtypes = [_vp, _vp, _vp, _vp, _vp, _vp, _vp, _i64, _i64, _i64, _i64, _i64,
                                                _i64, _i64, ctypes.c_float, _vp]
    lib.fastvr_chunk_attn_bwd.restype = ctypes.c_int
    lib.fastvr_chunk_attn_bwd.argtypes = [_vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _i64, _i64, _i64, _i64,
                                          _i64, _i64, _i64, _i64, ctypes.c_float, _vp]
    lib.fastvr_chunk_attn_bwd_noalloc.restype = ctypes.c_int
    lib.fastvr_chunk_attn_bwd_noalloc.argtypes = [_vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _i64, _i64, _i64,
                                                  _i64, _i64, _i64, _i64, _i64, ctypes.c_float, _vp]
    lib.fastvr_one_step_update.restype = ctypes.c_int
    lib.fastvr_one_step_update.argtypes = [_vp, _vp, _vp, _i64, ctypes.c_float, ctypes.c_int32, _vp]
    lib.fastvr_tile_axis.restype = ctypes.c_int
    lib.fastvr_tile_axis.argtypes = [_i64, _i64, _i64, ctypes.POINTER(_i64), ctypes.POINTER(_i64)]
    lib.fastvr_tile_gather.restype = ctypes.c_int
    lib.fastvr_tile_gather.argtypes = [_vp, _vp, _i64, _i64, _i64, _i64, _i64, _i64, _i64, _vp]
    lib.fastvr_tile_blend.restype = ctypes.c_int
    lib.fastvr_tile_blend.argtypes = [_vp, _vp, _i64, _i64, _i64, _i64, _i64, _i64, _i64, _vp]
    lib.fastvr_tile_blend_update.restype = ctypes.c_int
    lib.fastvr_tile_blend_update.argtypes = [_vp, _vp, _vp, ctypes.c_float, _i64, _i64, _i64, _i64, _i64, _i64,
                                             _i64, _vp]
    lib.fastvr_status_string.restype = ctypes.c_char_p
    lib.fastvr_status_string.argtypes = [ctypes.c_int]
    lib.fastvr_last_error.restype = ctypes.c_char_p
    lib.fastvr_last_error.argtypes = []
    lib.fastvr_abi_version.restype = ctypes.c_int
    lib.fastvr_abi_version.argtypes = []
    _LIB = lib
    return lib


def _check(status: int) -> None:
    if status != OK:
        lib = load()
        name = lib.fastvr_status_string(status).decode()
        detail = lib.fastvr_last_error().decode()
        raise FastVRError(status, f"{name}: {detail}")


def last_error() -> str:
    return load().fastvr_last_error().decode()


# ---------------------------------------------------------------------------
# raw entry points (integers for pointers; used by the tests and the bench)
# ---------------------------------------------------------------------------

def fwd_raw(q, k, v, o, lse, B, H, Nq, Nkv, d, chunk_len, q_chunk_offset, window_chunks, scale,
            stream=0) -> int:
    return load().fastvr_chunk_attn_fwd(q, k, v, o, lse, B, H, Nq, Nkv, d, chunk_len, q_chunk_offset,
                                        window_chunks, scale, stream)


def fwd_ex_raw(q, q_sb, q_st, k, k_sb, k_st, v, v_sb, v_st, o, o_sb, o_st, o_bf16, lse, B, H, Nq, Nkv, d,
               chunk_len, q_chunk_offset, window_chunks, scale, stream=0) -> int:
    return load().fastvr_chunk_attn_fwd_ex(q, q_sb, q_st, k, k_sb, k_st, v, v_sb, v_st, o, o_sb, o_st, o_bf16,
                                           lse, B, H, Nq, Nkv, d, chunk_len, q_chunk_offset, window_chunks,
                                           scale, stream)


def append_raw(k_cache, v_cache, k_new, v_new, B, H, d, capacity, cache_len, n_new, stream=0) -> int:
    return load().fastvr_kv_cache_append(k_cache, v_cache, k_new, v_new, B, H, d, capacity, cache_len,
                                         n_new, stream)


def ring_step_raw(q_new, k_new, v_new, k_ring, v_ring, o, lse, B, H, n_new, d, chunk_len, chunk_index,
                  window_chunks, scale, stream=0) -> int:
    return load().fastvr_chunk_attn_ring_step(q_new, k_new, v_new, k_ring, v_ring, o, lse, B, H, n_new, d,
                                              chunk_len, chunk_index, window_chunks, scale, stream)


def bwd_raw(q, k, v, o, lse, dout, dq, dk, dv, row_stats, B, H, Nq, Nkv, d, chunk_len, q_chunk_offset,
            window_chunks, scale, stream=0) -> int:
    return load().fastvr_chunk_attn_bwd(q, k, v, o, lse, dout, dq, dk, dv, row_stats, B, H, Nq, Nkv, d, chunk_len,
                                        q_chunk_offset, window_chunks, scale, stream)


def bwd_noalloc_raw(q, k, v, o, lse, dout, dq, dk, dv, B, H, Nq, Nkv, d, chunk_len, q_chunk_offset, window_chunks,
                    scale, stream=0) -> int:
    return load().fastvr_chunk_attn_bwd_noalloc(q, k, v, o, lse, dout, dq, dk, dv, B, H, Nq, Nkv, d, chunk_len,
                                                q_chunk_offset, window_chunks, scale, stream)


def one_step_raw(z_lq, v, z_hat, n, sigma, out_bf16, stream=0) -> int:
    return load().fastvr_one_step_update(z_lq, v, z_hat, n, sigma, out_bf16, stream)


def tile_axis(size: int, tile: int, overlap: int):
    """(number of tiles, tile length) along one axis, as the library places them."""
    n, L = _i64(0), _i64(0)
    _check(load().fastvr_tile_axis(size, tile, overlap, ctypes.byref(n), ctypes.byref(L)))
    return n.value, L.value


def tile_gather_raw(x, tiles, B, T, Hg, Wg, C, tile, overlap, stream=0) -> int:
    return load().fastvr_tile_gather(x, tiles, B, T, Hg, Wg, C, tile, overlap, stream)


def tile_blend_raw(tiles, out, B, T, Hg, Wg, C, tile, overlap, stream=0) -> int:
    return load().fastvr_tile_blend(tiles, out, B, T, Hg, Wg, C, tile, overlap, stream)


def tile_blend_update_raw(v_tiles, z_lq, z_hat, sigma, B, T, Hg, Wg, C, tile, overlap, stream=0) -> int:
    return load().fastvr_tile_blend_update(v_tiles, z_lq, z_hat, sigma, B, T, Hg, Wg, C, tile, overlap, stream)


# ---------------------------------------------------------------------------
# torch-facing wrappers
# ---------------------------------------------------------------------------

def _stream_handle(stream):
    import torch
    s = torch.cuda.current_stream() if stream is None else stream
    return s.cuda_stream


def _bnhd_strides(t, name):
    """(batch stride, token stride) of a [B, N, H, d] view whose heads and dims
    are packed (stride(3) == 1, stride(2) == d)."""
    if t.dim() != 4:
        raise ValueError(f"{name} must be 4-D [B, N, H, d]")
    if t.stride(3) != 1 or t.stride(2) != t.shape[3]:
        raise ValueError(f"{name}: heads and head_dim must be contiguous (stride(2) == d, stride(3) == 1)")
    return t.stride(0), t.stride(1)


def chunk_attn(q, k, v, *, chunk_len: int, q_chunk_offset: int = 0, window_chunks: int = -1,
               scale: float | None = None, out=None, lse=None, return_lse: bool = True, stream=None):
    """Chunk-causal attention forward (FastVR Sec. 3.1, Eq. 1).

    q [B, Nq, H, d], k/v [B, Nkv, H, d] bf16 GPU tensors (views allowed when
    heads and head_dim are packed).  Returns (o [B, Nq, H, d], lse fp32
    [B, H, Nq] or None); o is fp32 unless ``out`` is a bfloat16 tensor, which
    receives O rounded to bf16."""
    import torch
    for name, t in (("q", q), ("k", k), ("v", v)):
        if t.dtype != torch.bfloat16 or not t.is_cuda:
            raise ValueError(f"{name} must be a bfloat16 GPU tensor")
    B, Nq, H, d = q.shape
    Nkv = k.shape[1]
    if k.shape != (B, Nkv, H, d) or v.shape != k.shape:
        raise ValueError(f"shape mismatch: q {tuple(q.shape)} k {tuple(k.shape)} v {tuple(v.shape)}")
    if scale is None:
        scale = 1.0 / math.sqrt(d)
    if out is None:
        out = torch.empty((B, Nq, H, d), dtype=torch.float32, device=q.device)
    if out.dtype not in (torch.float32, torch.bfloat16) or tuple(out.shape) != (B, Nq, H, d):
        raise ValueError("out must be float32 or bfloat16 [B, Nq, H, d]")
    o_bf16 = 1 if out.dtype == torch.bfloat16 else 0
    if return_lse and lse is None:
        lse = torch.empty((B, H, Nq), dtype=torch.float32, device=q.device)
    if lse is not None and (lse.dtype != torch.float32 or tuple(lse.shape) != (B, H, Nq)
                            or not lse.is_contiguous()):
        raise ValueError("lse must be a contiguous float32 [B, H, Nq] tensor")
    lse_ptr = lse.data_ptr() if lse is not None else None
    st = _stream_handle(stream)
    if not o_bf16 and all(t.is_contiguous() for t in (q, k, v, out)):
        status = fwd_raw(q.data_ptr(), k.data_ptr(), v.data_ptr(), out.data_ptr(), lse_ptr, B, H, Nq, Nkv, d,
                         chunk_len, q_chunk_offset, window_chunks, scale, st)
    else:
        qs, ks, vs, os_ = (_bnhd_strides(t, n) for t, n in ((q, "q"), (k, "k"), (v, "v"), (out, "out")))
        status = fwd_ex_raw(q.data_ptr(), *qs, k.data_ptr(), *ks, v.data_ptr(), *vs, out.data_ptr(), *os_, o_bf16,
                            lse_ptr, B, H, Nq, Nkv, d, chunk_len, q_chunk_offset, window_chunks, scale, st)
    _check(status)
    return out, lse


def kv_cache_append(k_cache, v_cache, k_new, v_new, cache_len: int, stream=None) -> int:
    """Copy k_new/v_new [B, n_new, H, d] into the contiguous caches [B, capacity, H, d]
    at token offset cache_len; returns the new cache length."""
    import torch
    for name, t in (("k_cache", k_cache), ("v_cache", v_cache), ("k_new", k_new), ("v_new", v_new)):
        if t.dtype != torch.bfloat16 or not t.is_cuda or not t.is_contiguous():
            raise ValueError(f"{name} must be a contiguous bfloat16 GPU tensor")
    B, cap, H, d = k_cache.shape
    n_new = k_new.shape[1]
    if v_cache.shape != k_cache.shape or k_new.shape != (B, n_new, H, d) or v_new.shape != k_new.shape:
        raise ValueError("cache / new-chunk shape mismatch")
    _check(append_raw(k_cache.data_ptr(), v_cache.data_ptr(), k_new.data_ptr(), v_new.data_ptr(), B, H, d, cap,
                      cache_len, n_new, _stream_handle(stream)))
    return cache_len + n_new


def chunk_attn_ring_step(q_new, k_new, v_new, k_ring, v_ring, *, chunk_len: int, chunk_index: int,
                         window_chunks: int = 1, scale: float | None = None, out=None, lse=None,
                         return_lse: bool = True, stream=None):
    """One streaming step with a bounded ring KV cache of window_chunks + 1 chunk slots.

    q_new/k_new/v_new [B, n_new, H, d] bf16 hold chunk ``chunk_index`` of the
    stream; k_ring/v_ring [B, (window_chunks + 1) * chunk_len, H, d] bf16 hold
    the earlier chunks (chunk c in slot c mod (window_chunks + 1)).  The library
    writes the new chunk into its slot and returns (o fp32 [B, n_new, H, d],
    lse fp32 [B, H, n_new] or None) over chunks chunk_index - window_chunks ..
    chunk_index.  All tensors contiguous."""
    import torch
    for name, t in (("q_new", q_new), ("k_new", k_new), ("v_new", v_new), ("k_ring", k_ring), ("v_ring", v_ring)):
        if t.dtype != torch.bfloat16 or not t.is_cuda or not t.is_contiguous():
            raise ValueError(f"{name} must be a contiguous bfloat16 GPU tensor")
    B, n_new, H, d = q_new.shape
    if k_new.shape != q_new.shape or v_new.shape != q_new.shape:
        raise ValueError("q_new, k_new and v_new must have the same shape")
    if k_ring.shape != (B, (window_chunks + 1) * chunk_len, H, d) or v_ring.shape != k_ring.shape:
        raise ValueError("k_ring/v_ring must be [B, (window_chunks + 1) * chunk_len, H, d]")
    if scale is None:
        scale = 1.0 / math.sqrt(d)
    if out is None:
        out = torch.empty((B, n_new, H, d), dtype=torch.float32, device=q_new.device)
    if out.dtype != torch.float32 or tuple(out.shape) != (B, n_new, H, d) or not out.is_contiguous():
        raise ValueError("out must be a contiguous float32 [B, n_new, H, d] tensor")
    if return_lse and lse is None:
        lse = torch.empty((B, H, n_new), dtype=torch.float32, device=q_new.device)
    if lse is not None and (lse.dtype != torch.float32 or tuple(lse.shape) != (B, H, n_new)
                            or not lse.is_contiguous()):
        raise ValueError("lse must be a contiguous float32 [B, H, n_new] tensor")
    _check(ring_step_raw(q_new.data_ptr(), k_new.data_ptr(), v_new.data_ptr(), k_ring.data_ptr(), v_ring.data_ptr(),
                         out.data_ptr(), lse.data_ptr() if lse is not None else None, B, H, n_new, d, chunk_len,
                         chunk_index, window_chunks, scale, _stream_handle(stream)))
    return out, lse


def chunk_attn_bwd(q, k, v, o, lse, dout, *, chunk_len: int, q_chunk_offset: int = 0, window_chunks: int = -1,
                   scale: float | None = None, dq=None, dk=None, dv=None, row_stats=None, stream=None):
    """Gradients (dq, dk, dv), fp32, of chunk_attn for the upstream gradient ``dout``.

    q/dout [B, Nq, H, d] and k/v [B, Nkv, H, d] bf16, o fp32 [B, Nq, H, d] and
    lse fp32 [B, H, Nq] from the forward call with the same mask arguments and
    scale; all contiguous.  ``row_stats`` (fp32 [B, H, 2, Nq]) is a workspace the
    call fills with LSE * log2 e (plane 0) and -rowsum(dO * O) (plane 1)."""
    import torch
    for name, t in (("q", q), ("k", k), ("v", v), ("dout", dout)):
        if t.dtype != torch.bfloat16 or not t.is_cuda or not t.is_contiguous():
            raise ValueError(f"{name} must be a contiguous bfloat16 GPU tensor")
    B, Nq, H, d = q.shape
    Nkv = k.shape[1]
    if k.shape != (B, Nkv, H, d) or v.shape != k.shape or dout.shape != q.shape:
        raise ValueError(f"shape mismatch: q {tuple(q.shape)} k {tuple(k.shape)} v {tuple(v.shape)} "
                         f"dout {tuple(dout.shape)}")
    for name, t, shape in (("o", o, (B, Nq, H, d)), ("lse", lse, (B, H, Nq))):
        if t.dtype != torch.float32 or tuple(t.shape) != shape or not t.is_contiguous():
            raise ValueError(f"{name} must be a contiguous float32 {list(shape)} tensor")
    if scale is None:
        scale = 1.0 / math.sqrt(d)
    outs = []
    for name, t, shape in (("dq", dq, (B, Nq, H, d)), ("dk", dk, (B, Nkv, H, d)), ("dv", dv, (B, Nkv, H, d)),
                           ("row_stats", row_stats, (B, H, 2, Nq))):
        if t is None:
            t = torch.empty(shape, dtype=torch.float32, device=q.device)
        if t.dtype != torch.float32 or tuple(t.shape) != shape or not t.is_contiguous():
            raise ValueError(f"{name} must be a contiguous float32 {list(shape)} tensor")
        outs.append(t)
    dq, dk, dv, row_stats = outs
    _check(bwd_raw(q.data_ptr(), k.data_ptr(), v.data_ptr(), o.data_ptr(), lse.data_ptr(), dout.data_ptr(),
                   dq.data_ptr(), dk.data_ptr(), dv.data_ptr(), row_stats.data_ptr(), B, H, Nq, Nkv, d, chunk_len,
                   q_chunk_offset, window_chunks, scale, _stream_handle(stream)))
    return dq, dk, dv


def chunk_attn_bwd_noalloc(q, k, v, o, lse, dout, dq, dk, dv, *, chunk_len: int, q_chunk_offset: int = 0,
                           window_chunks: int = -1, scale: float | None = None, stream=None):
    """chunk_attn_bwd for callers that cannot allocate: the caller passes the
    outputs dq, dk, dv (fp32, contiguous, shapes as in chunk_attn_bwd) and the
    row statistics go to the library's static per-device workspace, so neither
    the library nor this binding allocates.  Calls that overlap in time on one
    device race on that workspace."""
    import torch
    for name, t in (("q", q), ("k", k), ("v", v), ("dout", dout)):
        if t.dtype != torch.bfloat16 or not t.is_cuda or not t.is_contiguous():
            raise ValueError(f"{name} must be a contiguous bfloat16 GPU tensor")
    B, Nq, H, d = q.shape
    Nkv = k.shape[1]
    if k.shape != (B, Nkv, H, d) or v.shape != k.shape or dout.shape != q.shape:
        raise ValueError(f"shape mismatch: q {tuple(q.shape)} k {tuple(k.shape)} v {tuple(v.shape)} "
                         f"dout {tuple(dout.shape)}")
    for name, t, shape in (("o", o, (B, Nq, H, d)), ("lse", lse, (B, H, Nq)), ("dq", dq, (B, Nq, H, d)),
                           ("dk", dk, (B, Nkv, H, d)), ("dv", dv, (B, Nkv, H, d))):
        if t.dtype != torch.float32 or tuple(t.shape) != shape or not t.is_contiguous():
            raise ValueError(f"{name} must be a contiguous float32 {list(shape)} tensor")
    if scale is None:
        scale = 1.0 / math.sqrt(d)
    _check(bwd_noalloc_raw(q.data_ptr(), k.data_ptr(), v.data_ptr(), o.data_ptr(), lse.data_ptr(), dout.data_ptr(),
                           dq.data_ptr(), dk.data_ptr(), dv.data_ptr(), B, H, Nq, Nkv, d, chunk_len, q_chunk_offset,
                           window_chunks, scale, _stream_handle(stream)))
    return dq, dk, dv


def one_step_update(z_lq, v, sigma: float, *, out=None, out_dtype=None, stream=None):
    """One-step latent update z_hat = z_lq - sigma * v (FastVR Eq. 9).

    z_lq, v: contiguous bf16 GPU tensors of one shape.  The result is float32
    (default) or bfloat16 (``out_dtype=torch.bfloat16``; ``out`` may then be
    z_lq or v itself, for an update in place)."""
    import torch
    for name, t in (("z_lq", z_lq), ("v", v)):
        if t.dtype != torch.bfloat16 or not t.is_cuda or not t.is_contiguous():
            raise ValueError(f"{name} must be a contiguous bfloat16 GPU tensor")
    if v.shape != z_lq.shape:
        raise ValueError(f"shape mismatch: z_lq {tuple(z_lq.shape)} v {tuple(v.shape)}")
    if out_dtype is None:
        out_dtype = out.dtype if out is not None else torch.float32
    if out_dtype not in (torch.float32, torch.bfloat16):
        raise ValueError("out_dtype must be float32 or bfloat16")
    if out is None:
        out = torch.empty(z_lq.shape, dtype=out_dtype, device=z_lq.device)
    if out.dtype != out_dtype or out.shape != z_lq.shape or not out.is_contiguous():
        raise ValueError("out must be a contiguous tensor of z_lq's shape and dtype out_dtype")
    _check(one_step_raw(z_lq.data_ptr(), v.data_ptr(), out.data_ptr(), z_lq.numel(), sigma,
                        1 if out_dtype == torch.bfloat16 else 0, _stream_handle(stream)))
    return out


def _tile_shape(B, T, Hg, Wg, C, tile, overlap):
    ny, Ly = tile_axis(Hg, tile, overlap)
    nx, Lx = tile_axis(Wg, tile, overlap)
    return (B, ny * nx, T, Ly, Lx, C)


def tile_gather(x, *, tile: int = 64, overlap: int = 16, out=None, stream=None):
    """Overlapping spatial tiles of a channels-last bf16 field x [B, T, Hg, Wg, C]
    -> [B, ny * nx, T, Ly, Lx, C] (placement as in include/fastvr.h)."""
    import torch
    if x.dtype != torch.bfloat16 or not x.is_cuda or not x.is_contiguous() or x.dim() != 5:
        raise ValueError("x must be a contiguous bfloat16 GPU tensor [B, T, Hg, Wg, C]")
    B, T, Hg, Wg, C = x.shape
    shape = _tile_shape(B, T, Hg, Wg, C, tile, overlap)
    if out is None:
        out = torch.empty(shape, dtype=torch.bfloat16, device=x.device)
    if out.dtype != torch.bfloat16 or tuple(out.shape) != shape or not out.is_contiguous():
        raise ValueError(f"out must be a contiguous bfloat16 tensor of shape {shape}")
    _check(tile_gather_raw(x.data_ptr(), out.data_ptr(), B, T, Hg, Wg, C, tile, overlap, _stream_handle(stream)))
    return out


def tile_blend(tiles, Hg: int, Wg: int, *, tile: int = 64, overlap: int = 16, z_lq=None, sigma: float = 0.0,
               out=None, stream=None):
    """Weight-normalised blend of fp32 tiles [B, ny * nx, T, Ly, Lx, C] into the
    field [B, T, Hg, Wg, C] (fp32).  With z_lq (bf16 [B, T, Hg, Wg, C]) the result
    is the one-step update z_lq - sigma * blend (Eq. 9), fused."""
    import torch
    if tiles.dtype != torch.float32 or not tiles.is_cuda or not tiles.is_contiguous() or tiles.dim() != 6:
        raise ValueError("tiles must be a contiguous float32 GPU tensor [B, ny*nx, T, Ly, Lx, C]")
    B, _, T, _, _, C = tiles.shape
    if tuple(tiles.shape) != _tile_shape(B, T, Hg, Wg, C, tile, overlap):
        raise ValueError("tiles do not match the grid, tile and overlap")
    shape = (B, T, Hg, Wg, C)
    if out is None:
        out = torch.empty(shape, dtype=torch.float32, device=tiles.device)
    if out.dtype != torch.float32 or tuple(out.shape) != shape or not out.is_contiguous():
        raise ValueError(f"out must be a contiguous float32 tensor of shape {shape}")
    st = _stream_handle(stream)
    if z_lq is None:
        _check(tile_blend_raw(tiles.data_ptr(), out.data_ptr(), B, T, Hg, Wg, C, tile, overlap, st))
    else:
        if z_lq.dtype != torch.bfloat16 or tuple(z_lq.shape) != shape or not z_lq.is_contiguous():
            raise ValueError(f"z_lq must be a contiguous bfloat16 tensor of shape {shape}")
        _check(tile_blend_update_raw(tiles.data_ptr(), z_lq.data_ptr(), out.data_ptr(), sigma, B, T, Hg, Wg, C, tile,
                                     overlap, st))
    return out
