"""The backward's in-kernel casts of P and dS (App. B.6.3), code by code:
the instrumented backward dumps every pre-cast P and dS with the codes it
formed and the block exponents, and each is checked against torch's own
E4M3FN conversion of the same value at the same power-of-two scale and
against the exponent rule (the smallest scale 2^e with 448 2^e >= the block
maximum, at least 2^-126).  The dumped P is checked against FP64 scores of
the decoded operands, the dumped dS and decoded codes against the kernel's
own FP64 row statistics (same values, another summation order), and blocks
the kernel skips must be left untouched."""
import numpy as np
import pytest
import torch

import oracle as orc
import paper_2609_37852_amd as pk
from paper_2609_37852_amd import synth
from _helpers import say, to_dev

pytestmark = pytest.mark.gpu

SENTINEL = 0xAB


def _e4m3(x):
    """Codes of x (already scaled) by torch's E4M3FN conversion."""
    return torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).to(torch.float8_e4m3fn).view(
        torch.uint8).numpy()


def _decode(c):
    return torch.from_numpy(np.ascontiguousarray(c)).view(torch.float8_e4m3fn).to(torch.float64).numpy()


def _block_exponent(amax):
    """Smallest e >= -126 with 448 2^e >= amax (amax 0: -126)."""
    e = np.full(amax.shape, -126, np.int64)
    pos = amax > 0
    e[pos] = np.frexp(amax[pos])[1] - 10
    for _ in range(4):
        e = np.where(pos & (np.ldexp(448.0, e) < amax), e + 1, e)
    for _ in range(4):
        e = np.where(pos & (np.ldexp(448.0, e - 1) >= amax), e - 1, e)
    return np.maximum(e, -126)


def _blocks(a, nb, nkb):
    B, H = a.shape[:2]
    return a.reshape(B, H, nb, 32, nkb, 32)


CASES = [
    ("causal", synth.with_shape(synth.WORKLOADS["gqa_d128_8k"], B=1, N=256, Hq=2, Hkv=1), 0),
    ("causal_pmx", synth.with_shape(synth.WORKLOADS["gqa_d128_8k"], B=1, N=192, Hq=2, Hkv=1),
     pk.FLAG_PBWD_BLOCK_SCALED),
    ("unmasked", synth.with_shape(synth.WORKLOADS["tiny_mha_128"], B=2, N=96, Nk=160, causal=False), 0),
    # wide heads: two key blocks per workgroup
    ("d192", synth.with_shape(synth.WORKLOADS["mla_d192_4k"], B=1, N=160, Hq=2, Hkv=2), 0),
    ("d256_unmasked", synth.with_shape(synth.WORKLOADS["gqa_d256_8k_qknorm"], B=1, N=96, Nk=128, Hq=2, Hkv=1,
                                       causal=False), 0),
    # the other backward instantiations: three isolated score channels, and
    # the protected dP (dP from BF16 operands, the stale correction)
    ("causal_iso3", synth.with_shape(synth.WORKLOADS["gqa_d128_8k"], B=1, N=128, Hq=2, Hkv=1), pk.FLAG_ISOLATE3),
    ("causal_pdp", synth.with_shape(synth.WORKLOADS["gqa_d128_8k"], B=1, N=128, Hq=2, Hkv=1),
     pk.FLAG_PROTECTED_DP),
]


@pytest.mark.parametrize("name,w,flags", CASES, ids=[c[0] for c in CASES])
def test_cast_dump(name, w, flags):
    d = synth.generate(w, seed=5)
    q, k, v, do = (to_dev(d[n], w.dtype) for n in ("q", "k", "v", "do"))
    mq, mk, mv, mdo = (pk.attn_fp8_quantize(t) for t in (q, k, v, do))
    tau = float(np.float32(w.tau))
    B, N, Nk, Hq, G = w.B, w.N, w.nk, w.Hq, w.Hq // w.Hkv
    p = pk.Problem(B, N, Hq, w.Hkv, w.Dqk, w.Dv, tau, causal=int(w.causal), seqlen_kv=w.Nk, flags=flags)
    o, lse = pk.attn_fp8_fwd(p, mq, mk, mv)
    p.cast_dump = torch.full((p.cast_dump_bytes(),), SENTINEL, dtype=torch.uint8, device="cuda")
    say(f"{name}: {w} flags {flags}, dump {p.cast_dump_bytes()} bytes")
    if flags & pk.FLAG_PROTECTED_DP:
        _, _, _, rs = pk.attn_fp8_bwd_protected_dp(p, mq, mk, mdo, lse, do, v, o, grad_dtype=torch.float32,
                                                   rowstats=True)
    else:
        _, _, _, rs = pk.attn_fp8_bwd(p, pk.DELTA_MATCHING, mq, mk, mv, mdo, lse, do, o, grad_dtype=torch.float32,
                                      rowstats=True)
    torch.cuda.synchronize()
    P, dS, Pc, dSc, eS, eP = (t.cpu().numpy() for t in p.cast_dump_views())
    rs, lse = rs.cpu().numpy(), lse.cpu().numpy().astype(np.float64)
    nb, nkb = N // 32, Nk // 32

    # the blocks the kernel computes: all, or those on and below the diagonal
    want = np.ones((B, Hq, nb, nkb), bool)
    if w.causal:
        want &= np.arange(nkb)[None, :] <= np.arange(nb)[:, None]
    done = eS != SENTINEL
    assert np.array_equal(done, want), name
    untouched = ~np.repeat(np.repeat(want, 32, 2), 32, 3)
    for a in (P, dS):
        assert np.all(a.view(np.uint32)[untouched] == 0xABABABAB)
    for a in (Pc, dSc):
        assert np.all(a[untouched] == SENTINEL)
    ok = ~untouched
    P64, dS64 = P.astype(np.float64), dS.astype(np.float64)
    P64[untouched] = 0.0
    dS64[untouched] = 0.0

    # block exponents and codes
    amax_ds = np.abs(_blocks(dS64, nb, nkb)).max(axis=(3, 5))
    assert np.array_equal(eS[want].astype(np.int64) - 127, _block_exponent(amax_ds)[want])
    es = np.repeat(np.repeat(eS.astype(np.int64) - 127, 32, 2), 32, 3)
    assert np.array_equal(dSc[ok], _e4m3(np.ldexp(dS64, -es)[ok]))
    if flags & pk.FLAG_PBWD_BLOCK_SCALED:
        amax_p = _blocks(P64, nb, nkb).max(axis=(3, 5))
        assert np.array_equal(eP[want].astype(np.int64) - 127, _block_exponent(amax_p)[want])
        ep = np.repeat(np.repeat(eP.astype(np.int64) - 127, 32, 2), 32, 3)
    else:
        assert np.all(eP == SENTINEL)
        ep = np.full(P.shape, -8, np.int64)
    assert np.array_equal(Pc[ok], _e4m3(np.ldexp(P64, -ep)[ok]))
    say(f"  codes equal on {int(ok.sum())} pairs; dS' codes nonzero {int((dSc[ok] & 0x7F).astype(bool).sum())}")

    # P against FP64 scores of the decoded operands (the kernel's LSE): the
    # score's MFMA accumulation is within 2^-8 of the sum of its terms' sizes
    xq = orc.dequantize(orc.quantize(d["q"]), B, N, Hq, w.Dqk)[0]
    xk = orc.dequantize(orc.quantize(d["k"]), B, Nk, w.Hkv, w.Dqk)[0]
    xk = np.repeat(xk, G, axis=1)
    S = tau * (xq @ xk.transpose(0, 1, 3, 2))
    T = tau * (np.abs(xq) @ np.abs(xk).transpose(0, 1, 3, 2))
    Pref = np.exp(S - lse[..., None])
    if w.causal:
        Pref = np.where(np.tril(np.ones((N, Nk), bool)), Pref, 0.0)
    err = np.abs(P64 - Pref)[ok]
    # plus FP32 rounding of the shifted score (relative 2^-22 of its terms)
    bound = (Pref * (2.0 ** -8 * T + 2.0 ** -22 * (1 + np.abs(S) + np.abs(lse[..., None]))) + 1e-7)[ok]
    say(f"  P max abs err {err.max():.2e}, worst err / bound {(err / bound).max():.3f}")
    assert np.all(err <= bound)

    # the dump against the kernel's own FP64 row statistics
    ell = np.abs(dS64).sum(-1)
    assert np.all(np.abs(dS64.sum(-1) - rs[..., pk.RS_SUM_DS]) <= 1e-12 * ell)
    assert np.all(np.abs(ell - rs[..., pk.RS_SUMABS_DS]) <= 1e-12 * ell)
    assert np.array_equal(np.abs(dS64).max(-1), rs[..., pk.RS_MAXABS_DS])
    cast = np.where(ok, _decode(dSc) * np.ldexp(1.0, es), 0.0)
    ellc = np.abs(cast).sum(-1)
    assert np.all(np.abs(cast.sum(-1) - rs[..., pk.RS_SUM_DSCAST]) <= 1e-12 * ellc)
    pcast = np.where(ok, _decode(Pc) * np.ldexp(1.0, ep), 0.0)
    assert np.all(np.abs(pcast.sum(-1) - rs[..., pk.RS_SUM_PCAST]) <= 1e-12 * pcast.sum(-1))


def test_cast_dump_needs_rowstats():
    w = synth.with_shape(synth.WORKLOADS["tiny_mha_128"], B=1, N=64)
    d = synth.generate(w, seed=1)
    q, k, v, do = (to_dev(d[n], w.dtype) for n in ("q", "k", "v", "do"))
    mq, mk, mv, mdo = (pk.attn_fp8_quantize(t) for t in (q, k, v, do))
    p = pk.Problem(w.B, w.N, w.Hq, w.Hkv, w.Dqk, w.Dv, float(np.float32(w.tau)))
    o, lse = pk.attn_fp8_fwd(p, mq, mk, mv)
    p.cast_dump = torch.zeros(p.cast_dump_bytes(), dtype=torch.uint8, device="cuda")
    with pytest.raises(pk.AttnFp8Error) as ei:
        pk.attn_fp8_bwd(p, pk.DELTA_MATCHING, mq, mk, mv, mdo, lse, do, o, grad_dtype=torch.float32)
    assert ei.value.code == -1 and "rowstats" in str(ei.value)
