"""Pins of the oracle's fused rotary producer (App. B.6.1; reading R16):
torch's float32 products and difference with its bfloat16 cast, untouched
channels and the zero angle, norm preservation of every rotated pair, the
dependence of rotated dot products on relative position only, and the order
rotation -> prescale -> centring."""
import numpy as np
import pytest
import torch

from paper_2609_37852_amd import synth


def bf16_inputs(B, N, H, D, seed=0):
    return synth.round_bf16(np.random.default_rng(seed).standard_normal((B, N, H, D)).astype(np.float32))


@pytest.mark.parametrize("D,lo,R", [(128, 0, 32), (192, 128, 64), (64, 0, 64), (256, 64, 128)])
def test_rotation_matches_torch(orc, D, lo, R):
    B, N, H = 2, 64, 3
    x = bf16_inputs(B, N, H, D)
    tab = synth.rope_table(N, R, 1e4)
    y, _ = orc.producer_rope(x, tab, lo, R)
    h2 = R // 2
    xt = torch.from_numpy(x)
    cs = torch.from_numpy(tab[:, :, 0])[None, :, None, :]
    sn = torch.from_numpy(tab[:, :, 1])[None, :, None, :]
    a, p = xt[..., lo:lo + h2], xt[..., lo + h2:lo + R]
    # separate float32 ops, each rounded once, then torch's bfloat16 cast
    ya = ((a * cs) - (p * sn)).to(torch.bfloat16).to(torch.float64).numpy()
    yp = ((p * cs) + (a * sn)).to(torch.bfloat16).to(torch.float64).numpy()
    assert np.array_equal(y[..., lo:lo + h2], ya)
    assert np.array_equal(y[..., lo + h2:lo + R], yp)
    rest = np.ones(D, bool)
    rest[lo:lo + R] = False
    assert np.array_equal(y[..., rest], x[..., rest].astype(np.float64))
    # position 0: cos 1, sin 0 -> the bf16 input itself
    assert np.array_equal(y[:, 0], x[:, 0].astype(np.float64))


def test_pair_norms_and_relative_position(orc):
    D, lo, R, N = 128, 0, 32, 128
    x = bf16_inputs(1, N, 1, D, seed=3)
    tab = synth.rope_table(N, R, 1e4)
    y, _ = orc.producer_rope(x, tab, lo, R)
    h2 = R // 2
    nx = x[..., :h2].astype(np.float64) ** 2 + x[..., h2:R].astype(np.float64) ** 2
    ny = y[..., :h2] ** 2 + y[..., h2:R] ** 2
    assert np.max(np.abs(ny - nx) / np.maximum(nx, 1e-30)) < 2 ** -6
    # the same query and key vectors placed at positions (m, n) and
    # (m + 40, n + 40): the rotated dot products agree to bf16 rounding
    q = np.repeat(x[:, :1], N, axis=1)
    k = np.repeat(x[:, 1:2], N, axis=1)
    yq, _ = orc.producer_rope(q, tab, lo, R)
    yk, _ = orc.producer_rope(k, tab, lo, R)
    dots = np.einsum("bnhd,bmhd->nm", yq[..., :R], yk[..., :R])
    scale = np.linalg.norm(q[0, 0, 0, :R]) * np.linalg.norm(k[0, 0, 0, :R])
    for m, n in ((10, 3), (50, 50), (70, 20)):
        assert abs(dots[m, n] - dots[m + 40, n + 40]) < 2 ** -6 * scale
    assert abs(dots[10, 3] - dots[10, 60]) > 2 ** -6 * scale   # not position-free


def test_rotation_precedes_prescale_and_centring(orc):
    B, N, H, D = 1, 96, 2, 192
    x = bf16_inputs(B, N, H, D, seed=5) + np.float32(0.75)
    x = synth.round_bf16(x)
    tab = synth.rope_table(N, 64, 1e4)
    r, _ = orc.producer_rope(x, tab, 128, 64)
    for pre, cen in ((0.3, False), (1.0, True), (0.125, True)):
        y, m = orc.producer_rope(x, tab, 128, 64, prescale=pre, center=cen)
        y2, m2 = orc.producer(r, prescale=pre, center=cen)
        assert np.array_equal(y, y2) and np.array_equal(m, m2)
    # no table: the plain producer
    y0, _ = orc.producer_rope(x, np.zeros((N, 0, 2)), 0, 0, prescale=0.3)
    y1, _ = orc.producer(x, prescale=0.3)
    assert np.array_equal(y0, y1)
