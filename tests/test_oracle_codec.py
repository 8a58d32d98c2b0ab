"""Pins of the oracle's FP8/E8M0/bf16 codec against libraries and the format
definitions (App. B.6.1 quantizer; OCP E4M3FN and E8M0 formats)."""
import numpy as np
import pytest
import torch


def _torch_e4m3(y):
    """torch's float32 -> float8_e4m3fn conversion (RNE, non-saturating)."""
    return torch.from_numpy(np.asarray(y, np.float32)).to(torch.float8_e4m3fn).view(torch.uint8).numpy()


def test_decode_table_matches_torch(orc):
    codes = np.arange(256, dtype=np.uint8)
    ours = orc.e4m3_value(codes)
    ref = torch.from_numpy(codes).view(torch.float8_e4m3fn).to(torch.float64).numpy()
    assert np.array_equal(np.isnan(ours), np.isnan(ref))
    ok = ~np.isnan(ref)
    assert np.array_equal(ours[ok], ref[ok])
    assert np.isnan(ours[[0x7F, 0xFF]]).all() and np.sum(np.isnan(ours)) == 2
    assert ours[0x7E] == 448.0 and ours[0x01] == 2.0 ** -9 and ours[0x08] == 2.0 ** -6


def test_round_matches_torch_below_464(orc):
    rng = np.random.default_rng(0)
    vals = orc.e4m3_value(np.arange(0x7F, dtype=np.uint8))
    mids = (vals[1:] + vals[:-1]) / 2
    cand = [vals, mids, np.nextafter(mids.astype(np.float32), np.float32(1e9)),
            np.nextafter(mids.astype(np.float32), np.float32(-1e9)),
            rng.standard_normal(20000) * 30, rng.standard_normal(20000) * 1e-2,
            rng.uniform(0, 464, 20000), np.array([0.0, 1e-30, 1e-45, 2.0 ** -10, 2.0 ** -11])]
    y = np.concatenate([np.asarray(c, np.float32) for c in cand]).astype(np.float32)
    y = np.concatenate([y, -y])
    y = y[np.abs(y) < 464]
    assert np.array_equal(orc.e4m3_round(y.astype(np.float64)), _torch_e4m3(y))


def test_round_ties_and_saturation(orc):
    # ties go to the even mantissa; hand-derived from the E4M3 grid
    cases = {17.0: 16.0, 19.0: 20.0, 2.0 ** -10: 0.0, 3 * 2.0 ** -10: 2.0 ** -8, 5 * 2.0 ** -10: 2.0 ** -8,
             7 * 2.0 ** -10: 2.0 ** -8 * 2, 1.0625: 1.0, 1.1875: 1.25, 240.0: 240.0, 248.0: 256.0,
             232.0: 224.0, 440.0: 448.0}
    for y, v in cases.items():
        assert orc.e4m3_value(orc.e4m3_round([y]))[0] == v, y
    # saturation at +-448 (App. B.6.1: C8 saturates), also beyond the NaN point of torch
    for y in (448.0, 449.0, 464.0, 470.0, 480.0, 1e6, 1e300, np.inf):
        assert orc.e4m3_round([y])[0] == 0x7E and orc.e4m3_round([-y])[0] == 0xFE
    assert orc.e4m3_round([-0.0])[0] == 0x80
    assert orc.e4m3_round([-1e-30])[0] == 0x80
    assert orc.e4m3_round([np.nan])[0] == 0x7F


def test_e8m0_scale_bytes_match_torch():
    b = np.arange(255, dtype=np.uint8)
    ref = torch.from_numpy(b).view(torch.float8_e8m0fnu).to(torch.float64).numpy()
    assert np.array_equal(ref, np.ldexp(1.0, b.astype(np.int64) - 127))


def test_pow2_exponent_brute_force(orc):
    rng = np.random.default_rng(1)
    ks = np.arange(-140, 130)
    a = np.concatenate([448.0 * np.ldexp(1.0, ks), np.nextafter(448.0 * np.ldexp(1.0, ks), np.inf),
                        np.nextafter(448.0 * np.ldexp(1.0, ks), 0), 224.0 * np.ldexp(1.0, ks),
                        np.abs(rng.standard_normal(3000)) * 10.0 ** rng.uniform(-40, 38, 3000),
                        [1e-45, 1.4e-45, 3.4e38, 0.0]])
    a = a[np.isfinite(a)]
    e = orc.pow2_exponent(a)
    for ai, ei in zip(a, e):
        if ai == 0:
            assert ei == -127
            continue
        # brute force over the E8M0 range
        ok = [k for k in range(-127, 128) if ai <= 448.0 * 2.0 ** k]
        assert ei == (min(ok) if ok else 127), (ai, ei)
    # the scaled block max lands in (224, 448] whenever the clamp is inactive
    live = (e > -127) & (e < 127)
    s = a[live] * np.ldexp(1.0, -e[live])
    assert np.all((s > 224) & (s <= 448))


def test_bf16_round(orc):
    rng = np.random.default_rng(2)
    x = (rng.standard_normal(50000) * 10.0 ** rng.uniform(-30, 30, 50000)).astype(np.float32)
    ref = torch.from_numpy(x).to(torch.bfloat16).to(torch.float64).numpy()
    assert np.array_equal(orc.bf16_round(x.astype(np.float64)), ref)
    # direct rounding of the double: just above a bf16 midpoint must round up even
    # when float32 would first round it down onto the midpoint
    mid = 1.0 + 2.0 ** -8                      # midpoint between 1 and 1+2^-7
    assert orc.bf16_round([mid + 2.0 ** -40])[0] == 1.0 + 2.0 ** -7
    assert orc.bf16_round([mid])[0] == 1.0     # tie to even
