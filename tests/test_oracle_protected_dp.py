"""Pins of the oracle's protected-dP variant (App. B.6.3, correction
variants; App. C.4.2): dP = dO V^T from the BF16-rounded dO and V, every
other product on the FP8 copies.

  * the dP it uses, recovered from dS = P (dP - delta) with delta = 0, equals
    a plain numpy product of the BF16-rounded operands (not of their FP8
    copies, not transposed);
  * inputs whose BF16 values are their own FP8 row copies give exactly the
    FP8 path's results (the variant changes the operands of dP and nothing
    else);
  * with BF16 inputs the variant moves dP closer to the exact product of
    the inputs than the FP8 path does."""
import numpy as np
import pytest

import oracle as orc


def _inputs(B, N, Hq, Hkv, D, seed):
    rng = np.random.default_rng(seed)
    q, do = (orc.bf16_round(rng.standard_normal((B, N, Hq, D))) for _ in range(2))
    k, v = (orc.bf16_round(rng.standard_normal((B, N, Hkv, D))) for _ in range(2))
    return q, k, v, do


@pytest.mark.parametrize("causal", [True, False])
def test_dp_is_the_bf16_product(causal):
    B, N, Hq, Hkv, D = 1, 64, 2, 1, 64
    q, k, v, do = _inputs(B, N, Hq, Hkv, D, 1)
    do = do * 3.0 + 0.5          # dP rows of a visible magnitude, BF16 values still
    do = orc.bf16_round(do)
    out, _ = orc.attention_from_inputs(q, k, v, do, 0.125, flags=orc.EXACT_ALL, delta_mode=orc.DELTA_STALE_ROWSUM,
                                       delta_in=np.zeros((B, Hq, N)), want_phat=True, want_ds=True,
                                       protected_dp=True, causal=causal)
    P, dS = out["phat"], out["dsraw"]
    ref = np.einsum("bnhc,bmhc->bhnm", orc.bf16_round(do), np.repeat(orc.bf16_round(v), Hq // Hkv, axis=2))
    live = P > 1e-12
    assert live.sum() > (N * N // 2 if causal else N * N)
    np.testing.assert_allclose(dS[live] / P[live], ref[live], rtol=1e-9, atol=1e-9)
    # the FP8 path's dP differs (its operands are the E4M3 copies)
    f8, _ = orc.attention_from_inputs(q, k, v, do, 0.125, flags=orc.EXACT_ALL, delta_in=np.zeros((B, Hq, N)),
                                      want_phat=True, want_ds=True, causal=causal)
    assert np.max(np.abs(f8["dsraw"][live] / f8["phat"][live] - ref[live])) > 1e-3


@pytest.mark.parametrize("mode", [orc.DELTA_STALE_ROWSUM, orc.DELTA_MATCHING])
def test_fp8_exact_inputs_give_the_fp8_path(mode):
    B, N, Hq, Hkv, D = 1, 96, 2, 2, 64
    q, k, v, do = _inputs(B, N, Hq, Hkv, D, 2)
    # dO and V replaced by their dequantized row copies: FP8 values times
    # powers of two, exact in BF16 and their own row copies again
    for name in ("v", "do"):
        x = {"v": v, "do": do}[name]
        r, _ = orc.dequantize(orc.quantize(x), *x.shape)
        y = np.ascontiguousarray(r.transpose(0, 2, 1, 3))
        assert np.array_equal(orc.bf16_round(y), y)
        if name == "v":
            v = y
        else:
            do = y
    a, _ = orc.attention_from_inputs(q, k, v, do, 0.125, delta_mode=mode, want_rowstats=True)
    b, _ = orc.attention_from_inputs(q, k, v, do, 0.125, delta_mode=mode, want_rowstats=True, protected_dp=True)
    for n in ("O", "LSE", "delta", "dQ", "dK", "dV", "rowstats"):
        assert np.array_equal(a[n], b[n]), n


def test_protected_dp_is_closer_to_the_exact_product():
    B, N, Hq, Hkv, D = 1, 128, 2, 1, 128
    rng = np.random.default_rng(3)
    q = orc.bf16_round(rng.standard_normal((B, N, Hq, D)))
    k = orc.bf16_round(rng.standard_normal((B, N, Hkv, D)))
    v = orc.bf16_round(rng.standard_normal((B, N, Hkv, D)))
    do = orc.bf16_round(rng.standard_normal((B, N, Hq, D)))
    ex = np.einsum("bnhc,bmhc->bhnm", do, np.repeat(v, Hq // Hkv, axis=2))
    errs = {}
    for prot in (False, True):
        out, _ = orc.attention_from_inputs(q, k, v, do, 1 / np.sqrt(D), flags=orc.EXACT_ALL,
                                           delta_in=np.zeros((B, Hq, N)), want_phat=True, want_ds=True,
                                           protected_dp=prot)
        live = out["phat"] > 1e-12
        errs[prot] = np.linalg.norm(out["dsraw"][live] / out["phat"][live] - ex[live]) / np.linalg.norm(ex[live])
    assert errs[True] < 1e-12 < errs[False]
