"""Pins of the oracle's input quantizer (App. B.6.1 with power-of-two 1x32 /
32x1 blocks) against torch's FP8 cast and the block-scale rule."""
import numpy as np
import torch


def _torch_e4m3_f64(y):
    return torch.from_numpy(np.asarray(y, np.float64)).to(torch.float8_e4m3fn).view(torch.uint8).numpy()


def test_row_copy_matches_library_cast(orc):
    rng = np.random.default_rng(3)
    B, N, H, D = 2, 64, 3, 96
    x = (rng.standard_normal((B, N, H, D)) * np.exp(rng.uniform(-8, 8, (B, N, H, 1)))).astype(np.float32)
    q = orc.quantize(x.astype(np.float64))
    xt = x.transpose(0, 2, 1, 3).astype(np.float64)               # [B,H,N,D]
    blocks = xt.reshape(B, H, N, D // 32, 32)
    amax = np.abs(blocks).max(-1)
    e = q["scale_row"].astype(np.int64) - 127
    # scale rule: smallest power of two with amax <= 448 * 2^e
    assert np.all(amax <= 448.0 * np.ldexp(1.0, e)) and np.all(amax > 448.0 * np.ldexp(1.0, e - 1))
    scaled = blocks * np.ldexp(1.0, -e)[..., None]
    # scaled values never exceed 448, so torch's non-saturating cast applies
    assert np.array_equal(q["code_row"].reshape(B, H, N, D // 32, 32), _torch_e4m3_f64(scaled))


def test_col_copy_is_row_copy_of_transpose(orc):
    rng = np.random.default_rng(4)
    B, N, H, D = 1, 96, 2, 64
    x = rng.standard_normal((B, N, H, D)) * 3
    q = orc.quantize(x)
    qt = orc.quantize(np.ascontiguousarray(x.transpose(0, 3, 2, 1)))   # N <-> D swapped
    assert np.array_equal(q["code_col"], qt["code_row"])
    assert np.array_equal(q["scale_col"], qt["scale_row"])


def test_exactly_representable_roundtrip_and_zero_blocks(orc):
    rng = np.random.default_rng(5)
    B, N, H, D = 1, 64, 1, 64
    grid = orc.e4m3_value(np.arange(0x7F, dtype=np.uint8))
    x = rng.choice(grid, (B, N, H, D)) * rng.choice([-1, 1], (B, N, H, D))
    x[:, :, :, ::7] = 448.0          # every row block and column block has amax 448
    x = x * 2.0 ** -5
    q = orc.quantize(x)
    xr, xc = orc.dequantize(q, B, N, H, D)
    assert np.array_equal(xr, x.transpose(0, 2, 1, 3)) and np.array_equal(xc, x.transpose(0, 2, 1, 3))
    assert np.all(q["scale_row"] == 127 - 5)
    z = np.zeros((1, 32, 1, 32))
    qz = orc.quantize(z)
    assert np.all(qz["scale_row"] == 0) and np.all(qz["code_row"] == 0) and np.all(qz["scale_col"] == 0)


def test_relative_error_bound(orc):
    rng = np.random.default_rng(6)
    B, N, H, D = 1, 128, 2, 128
    x = rng.standard_normal((B, N, H, D)) * np.exp(rng.uniform(-3, 3, (B, N, H, D)))
    q = orc.quantize(x)
    xr, xc = orc.dequantize(q, B, N, H, D)
    xt = x.transpose(0, 2, 1, 3)
    er = np.repeat(q["scale_row"].astype(np.int64) - 127, 32, axis=-1)            # [B,H,N,D]
    ec = np.repeat(q["scale_col"].astype(np.int64) - 127, 32, axis=-1).transpose(0, 1, 3, 2)
    for xh, e in ((xr, er), (xc, ec)):
        # normals: half an ulp is 2^-4 relative; subnormals: half their spacing 2^-10 * 2^e
        bound = np.maximum(2.0 ** -4 * np.abs(xt), np.ldexp(1.0, e - 10))
        assert np.all(np.abs(xh - xt) <= bound)
    assert q["nonfinite"] == 0
    x[0, 0, 0, 0] = np.inf
    assert orc.quantize(x)["nonfinite"] == 1
