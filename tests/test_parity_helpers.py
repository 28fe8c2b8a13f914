"""CPU checks of the GPU tests' helpers: the threaded oracle driver gives the
serial oracle's values, and the stratified row sample holds the rows it
promises."""
import numpy as np
import pytest

from paper_2609_36757_amd.workloads import make_qkv

from parity import run_oracle, run_oracle_parallel, sample_rows


@pytest.mark.parametrize("W,off,L,nq,nkv", [(-1, 0, 200, 700, 700), (0, 0, 200, 700, 900), (1, 2, 150, 420, 900),
                                            (2, 1, 96, 500, 700), (-1, 0, 5000, 300, 300), (3, 0, 7, 60, 60)])
def test_parallel_oracle_equals_serial_oracle(W, off, L, nq, nkv):
    q, k, v = make_qkv(2, nq, nkv, 3, 32, seed=5 + W + off)
    rng = np.random.default_rng(W + 10)
    rows = np.unique(rng.integers(0, nq, size=min(nq, 150)))
    o_s, l_s = run_oracle(q, k, v, L, off, W, 0.125, rows=rows)
    o_p, l_p = run_oracle_parallel(q, k, v, L, off, W, 0.125, rows=rows, block=37, workers=4)
    assert np.abs(o_s - o_p).max() <= 1e-12 and np.abs(l_s - l_p).max() <= 1e-12
    heads = [2, 0]
    o_h, l_h = run_oracle_parallel(q, k, v, L, off, W, 0.125, rows=rows, heads=heads, workers=3)
    assert np.abs(o_s[:, :, heads] - o_h).max() <= 1e-12 and np.abs(l_s[:, heads] - l_h).max() <= 1e-12
    o_a, l_a = run_oracle_parallel(q, k, v, L, off, W, 0.125, workers=2)
    o_f, l_f = run_oracle(q, k, v, L, off, W, 0.125)
    assert np.abs(o_a - o_f).max() <= 1e-12 and np.abs(l_a - l_f).max() <= 1e-12


def test_sample_rows_holds_every_band():
    L, n, tile, band = 1000, 3500, 256, 2
    rows = set(sample_rows(n, L, n_random=10, seed=1, tile=tile, band=band).tolist())
    for c0 in range(0, n, L):
        c1 = min(c0 + L, n)
        for t0 in range(c0, c1, tile):
            for r in range(t0 - band, t0 + band + 1):
                if c0 <= r < c1:
                    assert r in rows
        for r in range(c1 - band - 1, c1):
            assert r in rows
    assert n - 1 in rows and 0 in rows


@pytest.mark.parametrize("W", [-1, 1])
def test_sampled_backward_sigmas_equal_the_full_ones(W):
    """The per-row and per-key error scales the full-size backward test uses
    equal the ones computed from the whole softmax on a small case."""
    import oracle
    from test_gpu_bwd import _draw_do, _key_sigmas, _rounding_sigmas, _row_sigmas

    nq, H, d, L, scale = 300, 2, 32, 70, 0.17
    q, k, v = make_qkv(1, nq, nq, H, d, seed=3)
    do = _draw_do(1, nq, H, d, 4)
    sq, sk, sv = _rounding_sigmas(q, k, v, do, L, 0, W, scale)
    rows = np.array([0, 5, 69, 70, 150, 299])
    keys = np.array([0, 1, 69, 140, 299])
    o, lse = oracle.attention(q, k, v, chunk_len=L, window_chunks=W, scale=scale)
    for h in range(H):
        assert np.allclose(_row_sigmas(q, k, v, do, rows, L, W, scale, h), sq[0, rows, h], rtol=1e-10, atol=0)
        delta = oracle.attention_bwd_delta(o[:, :, h:h + 1], do[:, :, h:h + 1])[0, 0]
        ks, vs = _key_sigmas(q, k, v, do, keys, lse[0, h], delta, L, W, scale, h)
        assert np.allclose(ks, sk[0, keys, h], rtol=1e-10, atol=1e-300)
        assert np.allclose(vs, sv[0, keys, h], rtol=1e-10, atol=1e-300)
