"""GPU tests of the one-step latent update (Sec. 3.2, Eq. 9) through the C ABI.

The kernel forms fma(-sigma, v, z) in fp32, i.e. the exact value z - sigma * v
rounded once.  For these inputs (bf16 draws of N(0, 1), |sigma| <= 1000) the
exact value has fewer than 53 significant bits, so the oracle's fp64 result is
exact and its rounding to fp32 is the correctly rounded value: the fp32 output
must equal it bit for bit.  The bf16 output is that fp32 value rounded to
bf16 (nearest even), the same two decisions on both sides."""
import numpy as np
import pytest
import torch

import oracle
from paper_2609_36757_amd import fastvr

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dev():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    fastvr.load()
    return torch.device("cuda:0")


def _draw(n, seed):
    g = torch.Generator().manual_seed(seed)
    z = torch.randn(n, generator=g).to(torch.bfloat16)
    v = torch.randn(n, generator=g).to(torch.bfloat16)
    return z, v


def _expected_f32(z, v, sigma):
    s32 = float(np.float32(sigma))
    return oracle.one_step_update(z, v, s32).astype(np.float32)


@pytest.mark.parametrize("n", [1, 7, 8, 9, 255, 4096 + 5, (1 << 20) + 3])
@pytest.mark.parametrize("sigma", [0.0, 0.3719, -1.5, 1000.0])
def test_one_step_fp32_bitwise(dev, n, sigma):
    print(f"\n[gpu case] one_step fp32 n={n} sigma={sigma}", flush=True)
    z, v = _draw(n, seed=n % 1000 + 7)
    out = fastvr.one_step_update(z.to(dev), v.to(dev), sigma)
    torch.cuda.synchronize()
    exp = _expected_f32(z, v, sigma)
    got = out.cpu().numpy()
    assert got.dtype == np.float32
    np.testing.assert_array_equal(got.view(np.uint32), exp.view(np.uint32))


@pytest.mark.parametrize("n", [5, 64, 100003])
def test_one_step_bf16_bitwise_and_in_place(dev, n):
    print(f"\n[gpu case] one_step bf16 n={n}", flush=True)
    sigma = 0.61
    z, v = _draw(n, seed=300 + n % 97)
    exp = torch.from_numpy(_expected_f32(z, v, sigma)).to(torch.bfloat16)
    zd, vd = z.to(dev), v.to(dev)
    out = fastvr.one_step_update(zd, vd, sigma, out_dtype=torch.bfloat16)
    torch.cuda.synchronize()
    assert torch.equal(out.cpu().view(torch.int16), exp.view(torch.int16))
    # in place on z_lq, then on v: same bits
    fastvr.one_step_update(zd, vd, sigma, out=zd)
    torch.cuda.synchronize()
    assert torch.equal(zd.cpu().view(torch.int16), exp.view(torch.int16))
    zd2 = z.to(dev)
    fastvr.one_step_update(zd2, vd, sigma, out=vd)
    torch.cuda.synchronize()
    assert torch.equal(vd.cpu().view(torch.int16), exp.view(torch.int16))


def test_one_step_1080p_latent(dev):
    """The latent of the 1080p sequence at full size: 48 channels x 8 latent
    frames x 68 x 120, the size the benchmark times."""
    shape = (1, 48, 8, 68, 120)
    print(f"\n[gpu case] one_step 1080p latent {shape}", flush=True)
    g = torch.Generator().manual_seed(11)
    z = torch.randn(shape, generator=g).to(torch.bfloat16)
    v = torch.randn(shape, generator=g).to(torch.bfloat16)
    sigma = 0.8
    out = fastvr.one_step_update(z.to(dev), v.to(dev), sigma)
    torch.cuda.synchronize()
    exp = _expected_f32(z, v, sigma)
    np.testing.assert_array_equal(out.cpu().numpy().view(np.uint32), exp.view(np.uint32))
    # Eq. 4 -> Eq. 9: with the target velocity of a known HQ latent the update
    # returns that latent (up to the bf16 rounding of the velocity)
    z_hq = torch.randn(shape, generator=g).to(torch.bfloat16)
    u = oracle.target_velocity(z, z_hq, float(np.float32(sigma)))
    u_bf = torch.from_numpy(u).to(torch.bfloat16)
    rec = fastvr.one_step_update(z.to(dev), u_bf.to(dev), sigma).cpu().numpy()
    err = np.abs(rec - z_hq.to(torch.float64).numpy())
    bound = float(np.float32(sigma)) * np.abs(u) * 2.0 ** -8 + 1e-6
    assert (err <= bound).all()
