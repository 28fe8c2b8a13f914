"""Rows outside a visible key interval contribute nothing, even when the memory
there holds NaN (paper Sec. 3.1, Eq. 1: keys of later chunks, and anything past
the end of the key range, are masked out of every query's softmax).

The kernels stage K/V (forward, ring step, dQ) and Q/dO/row statistics
(dK/dV) in fixed-size tiles whose last tile may run past the valid rows; those
rows must read as zero through the buffer descriptors' range checks, because
the masked softmax weight P = 0 times a NaN value would still be NaN.  Each case
places the tensors at the start of a larger allocation whose tail (at least 256
rows, more than any staged tile) holds NaN in one run and finite random values
in the other; every access stays inside the allocation either way.  The
outputs of the two runs must be identical bit for bit, finite, and (for the
forward) within the parity bar of the fp64 oracle.

Covered: the forward's plain kernel (parallel call with future keys; a
streaming call on a KV cache whose rows past cache_len are poisoned, contiguous
and batch-strided), the per-CU list kernel (a shape the host packs into lists,
see tests/item_lists_check.cpp), the ring step (new chunk in a poisoned buffer,
the slot being replaced poisoned), and both backward kernels (Q, dO, O, K, V and
the row-statistics workspace with poisoned tails)."""
import numpy as np
import pytest
import torch

from paper_2609_36757_amd import fastvr
from paper_2609_36757_amd.workloads import make_qkv, randn_bf16

from parity import compare, default_scale, run_oracle, to_np

pytestmark = pytest.mark.gpu

PAD = 256  # poisoned rows after every tensor: more than one staged tile of any kernel


@pytest.fixture(scope="module")
def dev():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    fastvr.load()
    return torch.device("cuda:0")


def _announce(label):
    print(f"\n[gpu case] {label}", flush=True)


def _tail(t, pad_rows, poison, dev, seed):
    """t [1, n, ...] placed at the start of a device buffer [1, n + pad_rows, ...];
    the tail is NaN (poison) or finite N(0,1) values.  Returns the view of the
    first n rows (contiguous: B = 1)."""
    assert t.shape[0] == 1
    shape = (1, t.shape[1] + pad_rows) + tuple(t.shape[2:])
    if poison:
        buf = torch.full(shape, float("nan"), dtype=t.dtype, device=dev)
    else:
        g = torch.Generator().manual_seed(seed)
        buf = torch.randn(shape, generator=g).to(t.dtype).to(dev)
    buf[:, :t.shape[1]].copy_(t)
    v = buf[:, :t.shape[1]]
    assert v.is_contiguous()
    return v


def _bits(t):
    return t.view(torch.int32) if t.dtype == torch.float32 else t.view(torch.int16)


# name, H, d, Nq, Nkv (keys filled), Nkv_poisoned_after, chunk_len, q_chunk_offset, W
FWD_CASES = [
    # future keys 400..999 never visible; chunk 1's last 96-key tile runs 16 rows into them
    ("future_keys_L200", 2, 128, 400, 400, 600, 200, 0, -1),
    ("ragged_tail_L111_w1_d64", 2, 64, 333, 333, 0, 111, 0, 1),
    ("stream_off2_L150", 2, 128, 150, 450, 0, 150, 2, -1),
    ("stream_off3_w1_L300", 3, 128, 200, 1100, 0, 300, 3, 1),
]


@pytest.mark.parametrize("case", FWD_CASES, ids=[c[0] for c in FWD_CASES])
def test_forward_poisoned_tails(dev, case):
    name, H, d, nq, nkv, extra, L, off, W = case
    _announce(f"zero-fill fwd {name} H={H} d={d} Nq={nq} Nkv={nkv}+{extra} L={L} off={off} W={W}")
    scale = default_scale(d)
    q, k, v = make_qkv(1, nq, nkv, H, d, seed=900 + nq)
    outs = []
    for poison in (True, False):
        qd = _tail(q, PAD, poison, dev, 1)
        # keys: the filled rows, then `extra` never-visible rows and the pad, all poisoned
        kd = _tail(k, extra + PAD, poison, dev, 2)
        vd = _tail(v, extra + PAD, poison, dev, 3)
        if extra:
            kd = kd.as_strided((1, nkv + extra, H, d), kd.stride())
            vd = vd.as_strided((1, nkv + extra, H, d), vd.stride())
        o, lse = fastvr.chunk_attn(qd, kd, vd, chunk_len=L, q_chunk_offset=off, window_chunks=W, scale=scale)
        torch.cuda.synchronize()
        outs.append((o, lse))
    (o_p, l_p), (o_c, l_c) = outs
    assert torch.isfinite(o_p).all() and torch.isfinite(l_p).all(), "NaN from a masked row"
    assert torch.equal(_bits(o_p), _bits(o_c)) and torch.equal(_bits(l_p), _bits(l_c))
    kf = torch.cat([k, torch.zeros((1, extra, H, d), dtype=k.dtype)], dim=1) if extra else k
    vf = torch.cat([v, torch.zeros((1, extra, H, d), dtype=v.dtype)], dim=1) if extra else v
    o_ref, l_ref = run_oracle(q, kf, vf, L, off, W, scale)
    compare(to_np(o_p), to_np(l_p), o_ref, l_ref, label=f"zero-fill {name}")


@pytest.mark.parametrize("B", [1, 2])
def test_kv_cache_rows_past_cache_len_poisoned(dev, B):
    """Streaming call on a KV cache of capacity 1500 holding 1100 tokens (the
    appended chunk 3 is ragged, 200 tokens); rows 1100..1499 of every batch row
    are NaN.  With B = 2 the call reads a strided prefix view of the cache."""
    H, d, L, cap, cache_len, n_new = 2, 128, 300, 1500, 900, 200
    _announce(f"zero-fill kv cache B={B} H={H} d={d} L={L} cap={cap} len={cache_len}+{n_new}")
    q, k, v = make_qkv(B, cache_len + n_new, cache_len + n_new, H, d, seed=950 + B)
    qn = q[:, cache_len:].contiguous()
    outs = []
    for poison in (True, False):
        if poison:
            kc = torch.full((B, cap, H, d), float("nan"), dtype=torch.bfloat16, device=dev)
            vc = torch.full_like(kc, float("nan"))
        else:
            g = torch.Generator().manual_seed(7)
            kc = torch.randn((B, cap, H, d), generator=g).to(torch.bfloat16).to(dev)
            vc = torch.randn((B, cap, H, d), generator=g).to(torch.bfloat16).to(dev)
        kc[:, :cache_len].copy_(k[:, :cache_len])
        vc[:, :cache_len].copy_(v[:, :cache_len])
        n = fastvr.kv_cache_append(kc, vc, k[:, cache_len:].contiguous().to(dev),
                                   v[:, cache_len:].contiguous().to(dev), cache_len)
        for W in (-1, 1):
            o, lse = fastvr.chunk_attn(qn.to(dev), kc[:, :n], vc[:, :n], chunk_len=L, q_chunk_offset=3,
                                       window_chunks=W)
            torch.cuda.synchronize()
            outs.append((W, o, lse))
    for (W, o_p, l_p), (_, o_c, l_c) in zip(outs[:2], outs[2:]):
        assert torch.isfinite(o_p).all() and torch.isfinite(l_p).all(), f"NaN from a masked cache row (W={W})"
        assert torch.equal(_bits(o_p), _bits(o_c)) and torch.equal(_bits(l_p), _bits(l_c)), W
        o_ref, l_ref = run_oracle(qn, k, v, L, 3, W, default_scale(d))
        compare(to_np(o_p), to_np(l_p), o_ref, l_ref, label=f"zero-fill kv cache B={B} W={W}")


def test_list_kernel_poisoned_tail(dev):
    """B=1, H=12, d=128, chunks of 3120 tokens, Nq = Nkv = 4 * 3120 + 770: 672
    uneven items, which the host packs into per-CU lists.  The last chunk's
    interval ends 2 keys into a 96-key tile; the other 94 rows and the rest of
    the allocation are NaN."""
    H, d, L = 12, 128, 3120
    n = 4 * L + 770
    _announce(f"zero-fill list kernel H={H} d={d} N={n} L={L}")
    q, k, v = make_qkv(1, n, n, H, d, seed=960)
    outs = []
    for poison in (True, False):
        qd, kd, vd = (_tail(t, PAD, poison, dev, s) for t, s in ((q, 4), (k, 5), (v, 6)))
        o, lse = fastvr.chunk_attn(qd, kd, vd, chunk_len=L)
        torch.cuda.synchronize()
        outs.append((o, lse))
    (o_p, l_p), (o_c, l_c) = outs
    assert torch.isfinite(o_p).all() and torch.isfinite(l_p).all(), "NaN from a masked row"
    assert torch.equal(_bits(o_p), _bits(o_c)) and torch.equal(_bits(l_p), _bits(l_c))
    rows = np.unique(np.concatenate([np.arange(n - 60, n), np.arange(4 * L - 4, 4 * L + 4), [0, L - 1, 3 * L]]))
    ridx = torch.as_tensor(rows, device=dev)
    o_ref, l_ref = run_oracle(q, k, v, L, 0, -1, default_scale(d), rows=rows)
    compare(to_np(o_p[:, ridx]), to_np(l_p[:, :, ridx]), o_ref, l_ref, label=f"zero-fill list kernel ({len(rows)} rows)")


@pytest.mark.parametrize("W,L,n_chunks,last", [(1, 300, 4, 137), (2, 100, 6, 37)])
def test_ring_step_poisoned(dev, W, L, n_chunks, last):
    """Ring steps whose new chunk sits in a buffer with a NaN tail, and whose
    replaced slot (chunk c - W - 1, not visible) is NaN before the step: every
    step's rows equal the parallel call's bit for bit."""
    H, d = 2, 128
    N = (n_chunks - 1) * L + last
    _announce(f"zero-fill ring W={W} L={L} N={N} H={H} d={d}")
    q, k, v = make_qkv(1, N, N, H, d, seed=970 + W)
    qd, kd, vd = q.to(dev), k.to(dev), v.to(dev)
    full_o, full_l = fastvr.chunk_attn(qd, kd, vd, chunk_len=L, window_chunks=W)
    ring_k = torch.full((1, (W + 1) * L, H, d), float("nan"), dtype=torch.bfloat16, device=dev)
    ring_v = torch.full_like(ring_k, float("nan"))
    for c in range(n_chunks):
        s = slice(c * L, min((c + 1) * L, N))
        slot = c % (W + 1)
        ring_k[:, slot * L:(slot + 1) * L].fill_(float("nan"))
        ring_v[:, slot * L:(slot + 1) * L].fill_(float("nan"))
        qn, kn, vn = (_tail(t[:, s], PAD, True, dev, 0) for t in (q, k, v))
        o, lse = fastvr.chunk_attn_ring_step(qn, kn, vn, ring_k, ring_v, chunk_len=L, chunk_index=c,
                                             window_chunks=W)
        torch.cuda.synchronize()
        assert torch.isfinite(o).all() and torch.isfinite(lse).all(), f"NaN in ring step {c}"
        assert torch.equal(_bits(o), _bits(full_o[:, s])), c
        assert torch.equal(_bits(lse), _bits(full_l[:, :, s])), c
        n_new = s.stop - s.start
        assert torch.equal(ring_k[:, slot * L:slot * L + n_new], kd[:, s]), c
        assert torch.equal(ring_v[:, slot * L:slot * L + n_new], vd[:, s]), c


# name, H, d, Nq, Nkv, chunk_len, q_chunk_offset, W
BWD_CASES = [
    ("ragged_L100", 2, 128, 437, 437, 100, 0, -1),
    ("stream_off2_L150", 2, 128, 150, 450, 150, 2, -1),
    ("w1_L70_d64", 2, 64, 301, 301, 70, 0, 1),
]


@pytest.mark.parametrize("case", BWD_CASES, ids=[c[0] for c in BWD_CASES])
def test_backward_poisoned_tails(dev, case):
    """Q, dO and O with NaN rows past Nq, K and V with NaN rows past Nkv, and the
    row-statistics workspace with a NaN tail: the query tiles the dK/dV kernel
    stages past Nq and the key tiles the dQ kernel stages past the interval
    must read as zero."""
    name, H, d, nq, nkv, L, off, W = case
    _announce(f"zero-fill bwd {name} H={H} d={d} Nq={nq} Nkv={nkv} L={L} off={off} W={W}")
    scale = default_scale(d)
    q, k, v = make_qkv(1, nq, nkv, H, d, seed=980 + nq)
    g = torch.Generator().manual_seed(981)
    do = randn_bf16((1, nq, H, d), g)
    o, lse = fastvr.chunk_attn(q.to(dev), k.to(dev), v.to(dev), chunk_len=L, q_chunk_offset=off, window_chunks=W,
                               scale=scale)
    torch.cuda.synchronize()
    o_cpu = o.cpu()
    grads = []
    for poison in (True, False):
        qd, dod = _tail(q, PAD, poison, dev, 11), _tail(do, PAD, poison, dev, 12)
        kd, vd = _tail(k, PAD, poison, dev, 13), _tail(v, PAD, poison, dev, 14)
        od = _tail(o_cpu, PAD, poison, dev, 15)
        n_rs = H * 2 * nq
        rs_buf = torch.full((n_rs + PAD * 64,), float("nan"), device=dev) if poison else \
            torch.randn((n_rs + PAD * 64,), generator=torch.Generator().manual_seed(16)).to(dev)
        rs = rs_buf[:n_rs].view(1, H, 2, nq)
        dq, dk, dv = fastvr.chunk_attn_bwd(qd, kd, vd, od, lse, dod, chunk_len=L, q_chunk_offset=off,
                                           window_chunks=W, scale=scale, row_stats=rs)
        torch.cuda.synchronize()
        grads.append((dq, dk, dv))
    for name_g, gp, gc in zip(("dq", "dk", "dv"), grads[0], grads[1]):
        assert torch.isfinite(gp).all(), f"{name}: NaN in {name_g}"
        assert torch.equal(_bits(gp), _bits(gc)), f"{name}: {name_g} differs from the run with finite tails"
    print(f"[parity] zero-fill bwd {name}: gradients finite and bit-identical", flush=True)
