"""Pins of the oracle's input producer (App. B.6.1; reading R13): the FP32
query prescale, the FP32 per-(channel, KV head) key mean, the centred key,
and the properties the paper states for them (centering preserves softmax in
exact arithmetic; the straight-through key gradient of App. B.6.3 equals the
true one there, since the key gradient's column sums vanish)."""
import math

import numpy as np
import pytest

from paper_2609_37852_amd import synth


def _x(shape, seed=0, scale=1.0):
    return synth.round_bf16(np.random.default_rng(seed).standard_normal(shape).astype(np.float32) * scale)


def test_identity(orc):
    x = _x((2, 64, 3, 64))
    y, m = orc.producer(x, 1.0, False)
    assert np.array_equal(y, x.astype(np.float64)) and not m.any()


def test_prescale_is_an_fp32_multiply(orc):
    x = _x((1, 96, 2, 128), seed=1)
    s = np.float32(1.0 / math.sqrt(128.0))
    y, _ = orc.producer(x, float(s), False)
    assert np.array_equal(y, (x * s).astype(np.float64))       # numpy float32 product: IEEE RNE


def test_power_of_two_prescale_shifts_the_scales(orc):
    """x 2^-3 is exact, so its codes are x's codes and every block scale
    drops by 3."""
    x = _x((1, 64, 2, 64), seed=2)
    y, _ = orc.producer(x, 0.125, False)
    a, b = orc.quantize(x), orc.quantize(y)
    for f in ("code_row", "code_col"):
        assert np.array_equal(a[f], b[f])
    for f in ("scale_row", "scale_col"):
        assert np.array_equal(a[f].astype(int) - 3, b[f].astype(int))


def test_key_mean_and_centred_values(orc):
    """The mean is the FP32 rounding of the exact mean (the FP64 block sums
    err by far less than an FP32 ulp; near-ties are skipped), and the centred
    value is the FP32 difference (numpy float32 arithmetic)."""
    x = _x((2, 128, 2, 64), seed=3, scale=3.0) + np.float32(0.75)
    s = np.float32(0.3)
    y, m = orc.producer(x, float(s), True)
    xs = (x * s).astype(np.float32)
    checked = 0
    for b in range(2):
        for h in range(2):
            for c in range(64):
                exact = math.fsum(float(v) for v in xs[b, :, h, c]) / 128.0
                r = np.float32(exact)
                lo, hi = np.nextafter(r, np.float32(-np.inf)), np.nextafter(r, np.float32(np.inf))
                if min(abs(exact - (float(r) + float(lo)) / 2), abs(exact - (float(r) + float(hi)) / 2)) < 1e-12 * abs(exact):
                    continue                                 # a near-tie: either rounding is right
                assert m[b, h, c] == float(r), (b, h, c)
                checked += 1
    assert checked > 200
    assert np.array_equal(y, (xs - m.astype(np.float32)[:, None]).astype(np.float64))
    # the centred columns sum to zero up to FP32 rounding of their entries
    assert np.max(np.abs(y.sum(axis=1))) < 128 * np.finfo(np.float32).eps * np.max(np.abs(xs))


def test_centering_preserves_softmax_and_the_key_gradient(orc):
    """Exact arithmetic (no casts, raw inputs): subtracting a per-channel
    key mean adds a per-row constant to the scores, so O and LSE - that
    constant do not change; dQ, dV do not change, and dK for the centred keys
    equals dK for the raw keys (its column sums vanish, so the mean that
    differentiating through the centering would subtract is zero): the
    straight-through key gradient is the true one here."""
    B, N, Hq, Hkv, D = 1, 64, 4, 2, 32
    rng = np.random.default_rng(5)
    q, k = rng.standard_normal((B, N, Hq, D)), rng.standard_normal((B, N, Hkv, D)) + 2.0
    v, do = rng.standard_normal((B, N, Hkv, D)), rng.standard_normal((B, N, Hq, D))
    kc = k - k.mean(axis=1, keepdims=True)
    ex = dict(flags=orc.EXACT_ALL, exact_inputs=True, o_round=orc.ROUND_NONE)
    a, _ = orc.attention_from_inputs(q, k, v, do, 0.2, **ex)
    c, _ = orc.attention_from_inputs(q, kc, v, do, 0.2, **ex)
    for name in ("O", "dQ", "dK", "dV", "delta"):
        assert np.max(np.abs(a[name] - c[name])) < 1e-12 * max(np.max(np.abs(a[name])), 1.0), name
    assert np.max(np.abs(a["dK"].sum(axis=1))) < 1e-12


def test_query_prescale_matches_the_softmax_scale(orc):
    """q tau with softmax scale 1 is attention with scale tau, up to the
    FP32 rounding of q tau (exact arithmetic otherwise)."""
    B, N, Hq, Hkv, D = 1, 64, 2, 1, 64
    rng = np.random.default_rng(6)
    q = synth.round_bf16(rng.standard_normal((B, N, Hq, D)).astype(np.float32))
    k, v, do = (rng.standard_normal(s) for s in ((B, N, Hkv, D), (B, N, Hkv, D), (B, N, Hq, D)))
    tau = float(np.float32(1 / 8.0 / math.sqrt(2)))
    qs, _ = orc.producer(q, tau, False)
    ex = dict(flags=orc.EXACT_ALL, exact_inputs=True, o_round=orc.ROUND_NONE)
    a, _ = orc.attention_from_inputs(q, k, v, do, tau, **ex)
    c, _ = orc.attention_from_inputs(qs, k, v, do, 1.0, **ex)
    assert np.max(np.abs(a["O"] - c["O"])) < 1e-6
    assert np.max(np.abs(a["dK"] - c["dK"])) < 1e-6 * max(np.max(np.abs(a["dK"])), 1.0)


def test_producer_rejects_ragged_sequence(orc):
    with pytest.raises(AssertionError):
        orc.producer(np.zeros((1, 40, 1, 32)))
