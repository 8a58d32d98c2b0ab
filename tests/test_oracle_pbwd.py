"""Pins of the backward probability operand P' of dV: the fixed scale of
App. B.6.3 (reading R6: C8(256 P) 2^-8) and the block-scaled variant
(reading R15: one power-of-two scale per aligned 32x32 block, R2's rule on
the block's largest P).  P is recomputed here from the dequantized operands
and the oracle's LSE by the textbook softmax, and each block cast is torch's
FP8 cast; with Q = 0 every row is flat (P_ij = 1/(i+1)) and the operand has a
closed form."""
import numpy as np
import pytest
import torch

from paper_2609_37852_amd import synth


def e4m3(x):
    return torch.tensor(np.asarray(x, np.float64)).to(torch.float8_e4m3fn).to(torch.float64).numpy()


def probabilities(orc, d, w, out):
    """P_ij = min(exp(S_ij - LSE_i), 1) from the row copies of Q and K (causal)."""
    qr, _ = orc.dequantize(orc.quantize(d["q"]), w.B, w.N, w.Hq, w.Dqk)
    kr, _ = orc.dequantize(orc.quantize(d["k"]), w.B, w.N, w.Hkv, w.Dqk)
    G = w.Hq // w.Hkv
    kr = np.repeat(kr, G, axis=1)
    s = w.tau * np.einsum("bhid,bhjd->bhij", qr, kr)
    p = np.minimum(np.exp(s - out["LSE"][..., None]), 1.0)
    return np.where(np.tril(np.ones((w.N, w.N), bool)), p, 0.0)


@pytest.mark.parametrize("mx", [False, True])
def test_block_casts(orc, mx):
    w = synth.with_shape(synth.WORKLOADS["tiny_mha_128"], N=96)
    d = synth.generate(w, seed=3)
    flags = orc.MX_PBWD if mx else 0
    out, _ = orc.attention_from_inputs(d["q"], d["k"], d["v"], d["do"], w.tau, want_ds=True, flags=flags)
    p = probabilities(orc, d, w, out)
    pb = out["pbhat"]
    for b in range(w.B):
        for h in range(w.Hq):
            for i0 in range(0, w.N, 32):
                for j0 in range(0, i0 + 1, 32):
                    blk = p[b, h, i0:i0 + 32, j0:j0 + 32]
                    e = int(orc.pow2_exponent([blk.max()])[0]) if mx else -8
                    ref = e4m3(blk * 2.0 ** -e) * 2.0 ** e
                    # P itself is recomputed here in another order: compare
                    # codes where P is not within 1e-12 of a rounding boundary
                    got = pb[b, h, i0:i0 + 32, j0:j0 + 32]
                    near = np.abs(e4m3(blk * 2.0 ** -e * (1 + 1e-12)) - e4m3(blk * 2.0 ** -e * (1 - 1e-12))) > 0
                    assert np.array_equal(got[~near], ref[~near]), (b, h, i0, j0)


def test_flat_rows_closed_form_and_accuracy(orc):
    """Q = 0: P_ij = 1/(i+1) for j <= i exactly.  The fixed scale keeps
    C8(256/(i+1)) 2^-8, the block scale C8(2^-e/(i+1)) 2^e with e from the
    block's first row 1/(i0+1); dV with the block scale is closer to dV with
    uncast probabilities."""
    w = synth.with_shape(synth.WORKLOADS["tiny_mha_128"], N=1024, Hq=1, Hkv=1)
    d = synth.generate(w, seed=5)
    q = np.zeros_like(d["q"])
    outs = {}
    for name, flags in (("fixed", 0), ("mx", orc.MX_PBWD), ("exact", orc.EXACT_PBWD)):
        outs[name], _ = orc.attention_from_inputs(q, d["k"], d["v"], d["do"], w.tau, flags=flags,
                                                  want_ds=name != "exact")
    i = np.arange(w.N)[:, None]
    p = np.where(np.arange(w.N)[None, :] <= i, 1.0 / (i + 1), 0.0)
    assert np.array_equal(outs["fixed"]["pbhat"][0, 0], e4m3(256 * p) / 256)
    blockmax = np.repeat(1.0 / (np.arange(0, w.N, 32) + 1), 32)[:, None]
    e = orc.pow2_exponent(blockmax).astype(np.float64)
    mxref = np.where(p > 0, e4m3(p * 2.0 ** -e) * 2.0 ** e, 0.0)
    assert np.array_equal(outs["mx"]["pbhat"][0, 0], mxref)
    # P >= 1/1024 keeps 256 P in E4M3's normal range: the two casts agree
    assert np.array_equal(outs["mx"]["dV"], outs["fixed"]["dV"])
    # the forward and dQ/dK do not depend on the dV operand
    for k in ("O", "LSE", "dQ", "dK"):
        assert np.array_equal(outs["mx"][k], outs["fixed"][k]), k


def test_small_probabilities_keep_their_bits(orc):
    """Rows with one dominant key (score about 11.5 above the rest) leave
    P ~ 1e-5 < 2^-14 on every other key: 256 P falls into E4M3's subnormal
    range (steps of 2^-9) under the fixed scale, while the block scale keeps
    three mantissa bits.  dV of the keys in blocks without the dominant key
    is then much closer to dV from uncast probabilities."""
    w = synth.with_shape(synth.WORKLOADS["tiny_mha_128"], N=256, Hq=1, Hkv=1)
    d = synth.generate(w, seed=6)
    q = np.zeros_like(d["q"])
    k = np.zeros_like(d["k"])
    q[..., 0] = 9.5
    k[:, 0, :, 0] = 9.5        # key 0: score 9.5 * 9.5 / 8 = 11.3 for every query
    outs = {}
    for name, flags in (("fixed", 0), ("mx", orc.MX_PBWD), ("exact", orc.EXACT_PBWD)):
        outs[name], _ = orc.attention_from_inputs(q, k, d["v"], d["do"], w.tau, flags=flags)
    ref = outs["exact"]["dV"][:, 32:]
    err = {n: np.linalg.norm(outs[n]["dV"][:, 32:] - ref) / np.linalg.norm(ref) for n in ("fixed", "mx")}
    assert err["mx"] < 0.05 and err["fixed"] > 4 * err["mx"], err
