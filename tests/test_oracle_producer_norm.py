"""Pins of the oracle's QK normalization in the producer (the key RMSNorm of
App. B.4 with eps 1e-6 of App. B.2; reading R17): torch's float64 row
statistic with float32 products and its bfloat16 cast, invariance under a
power-of-two scaling of the row, unit RMS with gain 1, and the order
normalization -> rotation -> prescale -> centring."""
import numpy as np
import pytest
import torch

from paper_2609_37852_amd import synth


def rows(B, N, H, D, seed=0, scale=1.0):
    x = np.random.default_rng(seed).standard_normal((B, N, H, D)).astype(np.float32) * np.float32(scale)
    return synth.round_bf16(x)


@pytest.mark.parametrize("D", [64, 128, 192, 256])
def test_norm_matches_torch(orc, D):
    x = rows(2, 64, 3, D, seed=D)
    g = np.random.default_rng(1).uniform(0.5, 2.0, D).astype(np.float32)
    y, _ = orc.producer_ext(x, gain=g)
    xt = torch.from_numpy(x)
    ss = (xt.double() ** 2).sum(-1, keepdim=True)          # bf16 squares: every partial sum is exact
    r = (1.0 / torch.sqrt(ss / D + float(np.float32(1e-6)))).float()
    ref = ((xt * r) * torch.from_numpy(g)).to(torch.bfloat16).double().numpy()
    assert np.array_equal(y, ref)


def test_power_of_two_scaling_and_unit_rms(orc):
    D = 128
    x = rows(1, 32, 2, D, seed=4)
    g = np.ones(D, np.float32)
    # eps does not scale with the row: the invariance is exact without it
    y0, _ = orc.producer_ext(x, gain=g, eps=0.0)
    for s in (0.25, 8.0):
        ys, _ = orc.producer_ext(x * np.float32(s), gain=g, eps=0.0)
        assert np.array_equal(ys, y0)
    y, _ = orc.producer_ext(x, gain=g)
    rms = np.sqrt(np.mean(y ** 2, axis=-1))
    assert np.max(np.abs(rms - 1.0)) < 2 ** -7


def test_order_norm_rope_prescale_centre(orc):
    B, N, H, D = 1, 96, 2, 128
    x = rows(B, N, H, D, seed=6)
    g = np.random.default_rng(2).uniform(0.5, 2.0, D).astype(np.float32)
    tab = synth.rope_table(N, 32, 1e7)
    n, _ = orc.producer_ext(x, gain=g)
    for pre, cen in ((0.125, False), (1.0, True)):
        y, m = orc.producer_ext(x, gain=g, rope=tab, lo=0, R=32, prescale=pre, center=cen)
        y2, m2 = orc.producer_rope(n, tab, 0, 32, prescale=pre, center=cen)
        assert np.array_equal(y, y2) and np.array_equal(m, m2)
    # no gain: the rotary producer itself
    y0, _ = orc.producer_ext(x, rope=tab, lo=0, R=32, prescale=0.3)
    y1, _ = orc.producer_rope(x, tab, 0, 32, prescale=0.3)
    assert np.array_equal(y0, y1)
