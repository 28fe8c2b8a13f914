"""GPU parity tests of the backward pass (dQ, dK, dV) through the C ABI
against the fp64 oracle.

Tolerance, derived from the kernel's arithmetic: the products run on bf16
MFMAs with fp32 accumulation; besides the bf16 inputs (shared with the
oracle) the only roundings of any size are P (operand of dV = P^T dO) and dS
(operand of dQ = scale dS K and dK = scale dS^T Q) to bf16, each a relative
error of at most u = 2^-8 per term.  A gradient element that sums terms t_m
therefore carries an error of standard deviation at most u * sigma (dK:
sqrt(2) u sigma, since its dS is formed from the bf16-rounded P) with
sigma = sqrt(sum_m t_m^2):
    sigma_dV[j, c] = sqrt(sum_i P_ij^2 dO_ic^2)
    sigma_dQ[i, c] = |scale| sqrt(sum_j dS_ij^2 k_jc^2)
    sigma_dK[j, c] = |scale| sqrt(sum_i dS_ij^2 q_ic^2)
Each element must lie within 6 u sigma (+ 1e-5 of the largest reference
entry for the fp32 parts), and the relative Frobenius error of each gradient
within 1e-2 (the expected figure is about u / sqrt(3) = 2.3e-3)."""
import numpy as np
import pytest
import torch

import oracle
from paper_2609_36757_amd import fastvr
from paper_2609_36757_amd.workloads import WORKLOADS, make_qkv, make_sequence, randn_bf16

from parity import default_scale, fp32_scale, to_np

pytestmark = pytest.mark.gpu

U_BF16 = 2.0 ** -8
SIGMAS = 6.0
ABS_FLOOR = 1e-5
REL_FRO = 1e-2
LOG2E = 1.4426950408889634


@pytest.fixture(scope="module")
def dev():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    fastvr.load()
    return torch.device("cuda:0")


def _announce(label):
    print(f"\n[gpu case] {label}", flush=True)


def _draw_do(B, nq, H, d, seed):
    g = torch.Generator().manual_seed(seed)
    return randn_bf16((B, nq, H, d), g)


def _rounding_sigmas(q, k, v, do, L, off, W, scale):
    """Per-element error scales (sigma_dQ, sigma_dK, sigma_dV) of the bf16 P / dS roundings."""
    B, nq, H, d = q.shape
    nkv = k.shape[1]
    sq, sk, sv = np.zeros((B, nq, H, d)), np.zeros((B, nkv, H, d)), np.zeros((B, nkv, H, d))
    q64, k64, v64, do64 = (np.asarray(t.to(torch.float64)) for t in (q, k, v, do))
    for b in range(B):
        for h in range(H):
            p = oracle.softmax_weights(q, k, chunk_len=L, q_chunk_offset=off, window_chunks=W, scale=scale, b=b, h=h)
            dp = do64[b, :, h] @ v64[b, :, h].T
            ds = p * (dp - (p * dp).sum(axis=1, keepdims=True))
            sv[b, :, h] = np.sqrt((p * p).T @ (do64[b, :, h] ** 2))
            sq[b, :, h] = abs(scale) * np.sqrt((ds * ds) @ (k64[b, :, h] ** 2))
            sk[b, :, h] = abs(scale) * np.sqrt((ds * ds).T @ (q64[b, :, h] ** 2))
    return sq, sk, sv


def compare_grad(name, got, ref, sigma, label):
    got = np.asarray(got, dtype=np.float64)
    assert np.isfinite(got).all(), f"{label}: non-finite {name}"
    err = np.abs(got - ref)
    bound = SIGMAS * U_BF16 * sigma + ABS_FLOOR * max(np.abs(ref).max(), 1e-30)
    ratio = float((err / bound).max())
    rel = float(np.linalg.norm(got - ref) / max(np.linalg.norm(ref), 1e-300))
    stats = dict(max_abs=float(err.max()), worst_err_over_bound=ratio, rel_fro=rel)
    print(f"[parity] {label} {name} {stats}", flush=True)
    assert ratio <= 1.0, (label, name, stats)
    assert rel <= REL_FRO, (label, name, stats)
    return stats


def _gpu_fwd_bwd(dev, q, k, v, do, L, off, W, scale):
    qd, kd, vd, dod = (t.to(dev) for t in (q, k, v, do))
    o, lse = fastvr.chunk_attn(qd, kd, vd, chunk_len=L, q_chunk_offset=off, window_chunks=W, scale=scale)
    dq, dk, dv = fastvr.chunk_attn_bwd(qd, kd, vd, o, lse, dod, chunk_len=L, q_chunk_offset=off, window_chunks=W,
                                       scale=scale)
    torch.cuda.synchronize()
    return (qd, kd, vd, dod, o, lse), (dq, dk, dv)


# name, B, H, d, Nq, Nkv, chunk_len, q_chunk_offset, W, scale (None: 1/sqrt(d)), seed
BWD_CASES = [
    ("ragged_L100", 2, 2, 128, 437, 437, 100, 0, -1, None, 11),
    ("w1_L96", 1, 3, 128, 497, 497, 96, 0, 1, None, 12),
    ("w0_L64", 1, 2, 128, 256, 256, 64, 0, 0, None, 13),
    ("stream_off2", 1, 2, 128, 150, 450, 150, 2, -1, None, 14),
    ("stream_off3_w1_d64", 1, 2, 64, 100, 400, 100, 3, 1, None, 15),
    ("L300_w2_d64", 2, 1, 64, 1028, 1028, 300, 0, 2, None, 16),
    ("tiny_chunks_L4", 1, 2, 128, 38, 38, 4, 0, 3, None, 17),
    ("chunk_longer_than_seq", 1, 1, 128, 200, 200, 1000, 0, -1, None, 18),
    ("negative_scale_d64", 1, 2, 64, 300, 300, 70, 0, 1, -0.3, 19),
    ("odd_L257", 1, 1, 128, 600, 600, 257, 0, -1, None, 20),
    ("multi_tile_chunks", 1, 1, 128, 1500, 1500, 700, 0, -1, None, 21),
    ("negative_scale_d128_stream", 1, 2, 128, 200, 600, 200, 2, 1, -0.08, 22),
]


@pytest.mark.parametrize("case", BWD_CASES, ids=[c[0] for c in BWD_CASES])
def test_bwd_matches_oracle(dev, case):
    name, B, H, d, nq, nkv, L, off, W, scale, seed = case
    scale = default_scale(d) if scale is None else scale
    _announce(f"bwd {name} B={B} H={H} d={d} Nq={nq} Nkv={nkv} L={L} off={off} W={W} scale={scale}")
    q, k, v = make_qkv(B, nq, nkv, H, d, seed)
    do = _draw_do(B, nq, H, d, seed + 1000)
    (qd, kd, vd, dod, o, lse), (dq, dk, dv) = _gpu_fwd_bwd(dev, q, k, v, do, L, off, W, scale)
    s32 = fp32_scale(scale)
    rq, rk, rv = oracle.attention_bwd(q, k, v, do, chunk_len=L, q_chunk_offset=off, window_chunks=W, scale=s32)
    sq, sk, sv = _rounding_sigmas(q, k, v, do, L, off, W, s32)
    compare_grad("dq", to_np(dq), rq, sq, name)
    compare_grad("dk", to_np(dk), rk, sk, name)
    compare_grad("dv", to_np(dv), rv, sv, name)
    # keys no query sees get exactly zero
    seen = oracle.visibility_mask(nq, nkv, L, off, W).any(axis=0)
    assert (to_np(dk)[:, ~seen] == 0).all() and (to_np(dv)[:, ~seen] == 0).all()


def test_bwd_row_stats_and_determinism(dev):
    """The workspace holds LSE log2 e and -rowsum(dO * O) per row (two planes),
    and a second call reproduces every output bit for bit (fixed summation
    order)."""
    B, H, d, N, L, W, seed = 2, 3, 128, 700, 160, 1, 31
    _announce(f"bwd row stats / determinism B={B} H={H} d={d} N={N} L={L} W={W}")
    q, k, v = make_qkv(B, N, N, H, d, seed)
    do = _draw_do(B, N, H, d, seed + 1)
    (qd, kd, vd, dod, o, lse), (dq, dk, dv) = _gpu_fwd_bwd(dev, q, k, v, do, L, 0, W, default_scale(d))
    rs = torch.empty((B, H, 2, N), dtype=torch.float32, device=dev)
    dq2, dk2, dv2 = fastvr.chunk_attn_bwd(qd, kd, vd, o, lse, dod, chunk_len=L, window_chunks=W, row_stats=rs)
    torch.cuda.synchronize()
    assert torch.equal(dq, dq2) and torch.equal(dk, dk2) and torch.equal(dv, dv2)
    lse2 = (lse * np.float32(LOG2E)).cpu().numpy()
    np.testing.assert_allclose(rs[:, :, 0].cpu().numpy(), lse2, rtol=2e-7, atol=1e-6)
    dref = oracle.attention_bwd_delta(to_np(o), do)
    np.testing.assert_allclose(-rs[:, :, 1].cpu().numpy(), dref, rtol=1e-5, atol=1e-5)


def test_bwd_no_queries_zeroes_key_gradients(dev):
    """Nq = 0: dK and dV are set to zero."""
    B, H, d, nkv = 1, 2, 128, 300
    _announce(f"bwd Nq=0 B={B} H={H} d={d} Nkv={nkv}")
    k = torch.randn((B, nkv, H, d), device=dev).to(torch.bfloat16)
    q = torch.empty((B, 0, H, d), dtype=torch.bfloat16, device=dev)
    o = torch.empty((B, 0, H, d), dtype=torch.float32, device=dev)
    lse = torch.empty((B, H, 0), dtype=torch.float32, device=dev)
    dk = torch.full((B, nkv, H, d), float("nan"), device=dev)
    dv = torch.full_like(dk, float("nan"))
    fastvr.chunk_attn_bwd(q, k, k, o, lse, q, chunk_len=100, dk=dk, dv=dv)
    torch.cuda.synchronize()
    assert (dk == 0).all() and (dv == 0).all()


def test_bwd_tiny_workload(dev):
    """The tiny configuration (4 chunks x 256 tokens, d = 64, full causal prefix)."""
    w = WORKLOADS["tiny"]
    _announce("bwd tiny workload")
    q, k, v = make_sequence(w)
    do = _draw_do(w.B, w.n_tokens, w.H, w.d, w.seed + 2000)
    _, (dq, dk, dv) = _gpu_fwd_bwd(dev, q, k, v, do, w.chunk_len, 0, w.window_chunks, w.scale)
    s32 = fp32_scale(w.scale)
    rq, rk, rv = oracle.attention_bwd(q, k, v, do, chunk_len=w.chunk_len, window_chunks=w.window_chunks, scale=s32)
    sq, sk, sv = _rounding_sigmas(q, k, v, do, w.chunk_len, 0, w.window_chunks, s32)
    compare_grad("dq", to_np(dq), rq, sq, "tiny")
    compare_grad("dk", to_np(dk), rk, sk, "tiny")
    compare_grad("dv", to_np(dv), rv, sv, "tiny")


def _row_sigmas(q, k, v, do, rows, L, W, scale, h):
    """sigma_dQ (see the module docstring) of the given query rows of head h,
    from the fp64 softmax weights of those rows: [R, d]."""
    q64 = q[0, torch.as_tensor(rows), h].to(torch.float64).numpy()
    do64 = do[0, torch.as_tensor(rows), h].to(torch.float64).numpy()
    k64, v64 = k[0, :, h].to(torch.float64).numpy(), v[0, :, h].to(torch.float64).numpy()
    vis = oracle.visibility_mask(q.shape[1], k.shape[1], L, 0, W, rows=rows)
    s = np.where(vis, scale * (q64 @ k64.T), -np.inf)
    p = np.exp(s - s.max(axis=1, keepdims=True))
    p /= p.sum(axis=1, keepdims=True)
    dp = do64 @ v64.T
    ds = p * (dp - (p * dp).sum(axis=1, keepdims=True))
    return abs(scale) * np.sqrt((ds * ds) @ (k64 ** 2))


def _key_sigmas(q, k, v, do, keys, lse, delta, L, W, scale, h):
    """sigma_dK and sigma_dV of the given key rows of head h, from the fp64
    row statistics (LSE_i, D_i) of every query: ([K, d], [K, d])."""
    nq, nkv = q.shape[1], k.shape[1]
    q64, do64 = q[0, :, h].to(torch.float64).numpy(), do[0, :, h].to(torch.float64).numpy()
    sk, sv = np.zeros((len(keys), q.shape[3])), np.zeros((len(keys), q.shape[3]))
    for t, j in enumerate(keys):
        dc = oracle.query_chunks(nq, L) - j // L
        vis = (dc >= 0) & (dc <= W) if W >= 0 else dc >= 0
        ii = np.nonzero(vis)[0]
        kj, vj = k[0, j, h].to(torch.float64).numpy(), v[0, j, h].to(torch.float64).numpy()
        p = np.exp(scale * (q64[ii] @ kj) - lse[ii])
        ds = p * (do64[ii] @ vj - delta[ii])
        sv[t] = np.sqrt((p * p) @ (do64[ii] ** 2))
        sk[t] = abs(scale) * np.sqrt((ds * ds) @ (q64[ii] ** 2))
    return sk, sv


def test_bwd_1080p_full_size(dev):
    """The 1080p sequence (B=1, H=12, d=128, 4 chunks x 16320 tokens, full causal
    prefix) at full size, in the launch configuration the benchmark times,
    element by element within the per-element bound of the module docstring:
    sampled dQ rows of every head; sampled dK / dV rows of three heads from key
    chunks 0, 1 and 3 (keys of chunk 0 are seen by every query, so their sums run
    over all four query chunks, whose row statistics the oracle computes for
    every query of those heads); and two identities over every output:
    sum_j dV_j = sum_i dO_i (softmax rows sum to one) and sum_j dK_j = 0 (rows
    of dS sum to zero)."""
    from parity import run_oracle_parallel

    w = WORKLOADS["1080p"]
    _announce("bwd 1080p full size")
    q, k, v = make_sequence(w)
    do = _draw_do(w.B, w.n_tokens, w.H, w.d, w.seed + 3000)
    L, N, H = w.chunk_len, w.n_tokens, w.H
    _, (dq, dk, dv) = _gpu_fwd_bwd(dev, q, k, v, do, L, 0, w.window_chunks, w.scale)
    s32 = fp32_scale(w.scale)
    rng = np.random.default_rng(77)
    rows = np.unique(np.concatenate([[0, 255, 256, L - 1, L, 2 * L + 300, N - 1], rng.integers(0, N, 25)]))
    rq, _, _ = oracle.attention_bwd(q, k, v, do, chunk_len=L, window_chunks=w.window_chunks, scale=s32, rows=rows)
    dq_s = to_np(dq[:, rows])
    sq = np.stack([_row_sigmas(q, k, v, do, rows, L, w.window_chunks, s32, h) for h in range(H)], axis=1)[None]
    compare_grad("dq", dq_s, rq, sq, f"1080p sampled rows ({len(rows)} rows, all heads)")
    # dK / dV of sampled keys of chunks 0, 1 and 3, three heads
    heads = [0, 5, 11]
    keys = np.unique(np.concatenate([[0, 127, 128, L - 1, L, L + 127, L + 128, 2 * L - 1, 3 * L, 3 * L + 127,
                                      3 * L + 128, N - 1],
                                     rng.integers(0, L, 5), L + rng.integers(0, L, 5), 3 * L + rng.integers(0, L, 4)]))
    o_ref, lse_ref = run_oracle_parallel(q, k, v, L, 0, w.window_chunks, w.scale, heads=heads)
    for hp, h in enumerate(heads):
        qh, kh, vh, doh = (t[:, :, h:h + 1] for t in (q, k, v, do))
        lse_h = lse_ref[:, hp:hp + 1]
        delta_h = oracle.attention_bwd_delta(o_ref[:, :, hp:hp + 1], doh)
        rk, rv = oracle.attention_bwd_keys(qh, kh, vh, doh, keys, lse_h, delta_h, chunk_len=L,
                                           window_chunks=w.window_chunks, scale=s32)
        sk, sv = _key_sigmas(q, k, v, do, keys, lse_h[0, 0], delta_h[0, 0], L, w.window_chunks, s32, h)
        compare_grad("dk", to_np(dk[:, keys, h:h + 1]), rk, sk[None, :, None], f"1080p keys head {h}")
        compare_grad("dv", to_np(dv[:, keys, h:h + 1]), rv, sv[None, :, None], f"1080p keys head {h}")
    # identities over all outputs, per (b, h, c)
    do64 = do.to(torch.float64)
    sum_do = do64.sum(dim=1)
    sv = dv.to(torch.float64).sum(dim=1).cpu()
    bound_v = SIGMAS * U_BF16 * (do64 ** 2).sum(dim=1).sqrt() + 1e-3
    assert ((sv - sum_do).abs() <= bound_v).all(), float((sv - sum_do).abs().max())
    dk64 = dk.to(torch.float64)
    sk = dk64.sum(dim=1).abs()
    bound_k = 8 * U_BF16 * (dk64 ** 2).sum(dim=1).sqrt() + 1e-3
    assert (sk <= bound_k).all(), float((sk - bound_k).max())
