"""Pins of the oracle's attention forward/correction/backward against what the
paper and the mathematics fix: torch autograd (exact arithmetic), finite
differences, the zero-row-sum invariant (Sec. 3.1/3.4), the stale residual
decomposition (Sec. 3.2, App. A.3), closed forms, and library FP8 casts for the
probability and dS encodings (App. B.6.2/B.6.3)."""
import numpy as np
import pytest
import torch

from paper_2609_37852_amd import synth


def torch_attention(q, k, v, do, tau):
    """Textbook causal attention in float64 with torch autograd (Sec. 2.3)."""
    q, k, v, do = (torch.tensor(np.asarray(t, np.float64)) for t in (q, k, v, do))
    q.requires_grad_(True); k.requires_grad_(True); v.requires_grad_(True)
    B, N, Hq, _ = q.shape
    G = Hq // k.shape[2]
    Q = q.permute(0, 2, 1, 3)
    K = k.repeat_interleave(G, dim=2).permute(0, 2, 1, 3)
    V = v.repeat_interleave(G, dim=2).permute(0, 2, 1, 3)
    S = tau * torch.matmul(Q, K.transpose(-1, -2).contiguous())
    mask = torch.ones(N, N, dtype=torch.bool).triu(1)
    S = S.masked_fill(mask, float("-inf"))
    P = torch.softmax(S, -1)
    O = torch.matmul(P, V).permute(0, 2, 1, 3)
    lse = torch.logsumexp(S, -1)
    O.backward(do)
    return dict(O=O.detach().numpy(), LSE=lse.detach().numpy(), dQ=q.grad.numpy(), dK=k.grad.numpy(),
                dV=v.grad.numpy(), P=P.detach().numpy())


def rel(a, b):
    return np.linalg.norm(a - b) / max(np.linalg.norm(b), 1e-300)


def inputs(B, N, Hq, Hkv, Dqk, Dv, seed=0, scale=1.0):
    rng = np.random.default_rng(seed)
    return (rng.standard_normal((B, N, Hq, Dqk)) * scale, rng.standard_normal((B, N, Hkv, Dqk)) * scale,
            rng.standard_normal((B, N, Hkv, Dv)), rng.standard_normal((B, N, Hq, Dv)))


@pytest.mark.parametrize("shape", [(2, 40, 4, 2, 16, 16), (1, 33, 2, 1, 24, 8), (1, 1, 1, 1, 8, 8)])
def test_exact_mode_matches_torch_autograd(orc, shape):
    B, N, Hq, Hkv, Dqk, Dv = shape
    q, k, v, do = inputs(*shape)
    tau = 1 / np.sqrt(Dqk)
    out, _ = orc.attention_from_inputs(q, k, v, do, tau, flags=orc.EXACT_ALL, exact_inputs=True,
                                       o_round=orc.ROUND_NONE, want_rowstats=True)
    ref = torch_attention(q, k, v, do, tau)
    for name in ("O", "LSE", "dQ", "dK", "dV"):
        assert rel(out[name], ref[name]) < 1e-12, name
    # exact arithmetic: the saved-output shortcut equals the matched correction
    out2, _ = orc.attention_from_inputs(q, k, v, do, tau, flags=orc.EXACT_ALL, exact_inputs=True,
                                        o_round=orc.ROUND_NONE, delta_mode=orc.DELTA_STALE_ROWSUM)
    assert rel(out2["delta"], out["delta"]) < 1e-12
    assert np.max(np.abs(out2["dQ"] - out["dQ"])) < 1e-10 * max(np.max(np.abs(ref["dV"])), 1.0)


def test_finite_differences(orc):
    B, N, Hq, Hkv, D = 1, 6, 2, 1, 4
    q, k, v, do = inputs(B, N, Hq, Hkv, D, D, seed=7)
    tau = 0.7

    def loss(qq, kk, vv):
        o, _ = orc.attention_from_inputs(qq, kk, vv, do, tau, flags=orc.EXACT_ALL, exact_inputs=True,
                                         o_round=orc.ROUND_NONE)
        return float(np.sum(o["O"] * do))
    out, _ = orc.attention_from_inputs(q, k, v, do, tau, flags=orc.EXACT_ALL, exact_inputs=True,
                                       o_round=orc.ROUND_NONE)
    h = 1e-6
    for name, t, g in (("q", q, out["dQ"]), ("k", k, out["dK"]), ("v", v, out["dV"])):
        num = np.zeros_like(t)
        for idx in np.ndindex(t.shape):
            tp, tm = t.copy(), t.copy()
            tp[idx] += h; tm[idx] -= h
            args = {"q": q, "k": k, "v": v}
            args[name] = tp; lp = loss(args["q"], args["k"], args["v"])
            args[name] = tm; lm = loss(args["q"], args["k"], args["v"])
            num[idx] = (lp - lm) / (2 * h)
        assert rel(g, num) < 1e-7, name


def _quantized_case(orc, name="tiny_mha_128", seed=0, **kw):
    w = synth.WORKLOADS[name]
    if kw:
        w = synth.with_shape(w, **kw)
    d = synth.generate(w, seed)
    return w, d


def test_zero_row_sum_matching_and_violation_stale(orc):
    w, d = _quantized_case(orc)
    res = {}
    for mode in (orc.DELTA_MATCHING, orc.DELTA_STALE_ROWSUM):
        out, _ = orc.attention_from_inputs(d["q"], d["k"], d["v"], d["do"], w.tau, delta_mode=mode,
                                           o_round=orc.ROUND_F32, want_rowstats=True)
        st = out["rowstats"].reshape(-1, orc.NSTAT)
        live = st[:, orc.ST_SUMABS_DS] > 0
        res[mode] = np.abs(st[live, orc.ST_SUM_DS]) / st[live, orc.ST_SUMABS_DS]
    # Sec. 3.4: matched correction gives zero row sums up to (here FP64) rounding
    assert res[orc.DELTA_MATCHING].max() < 1e-13
    # Sec. 3.2: the stale correction leaves a measurable residual
    med = np.median(res[orc.DELTA_STALE_ROWSUM])
    assert med > 1e-4 and med > 1e3 * max(np.median(res[orc.DELTA_MATCHING]), 1e-17)


def test_stale_residual_decomposition(orc):
    """App. A.3 decomposition of the stale row sum, extended with the two terms
    this kernel adds (row vs col copy of V, and O storage rounding):
       eps_i = sum_k dOr_ik sum_j (P - Phat)_ij Vr_jk          (probability)
             + sum_k (dOr - dO)_ik sum_j Phat_ij Vr_jk         (gradient)
             + sum_k dO_ik sum_j Phat_ij (Vr - Vc)_jk           (two V copies)
             + sum_k dO_ik (O - O_stored)_ik                    (storage)"""
    w, d = _quantized_case(orc, N=64)
    out, quant = orc.attention_from_inputs(d["q"], d["k"], d["v"], d["do"], w.tau,
                                           delta_mode=orc.DELTA_STALE_ROWSUM, o_round=orc.ROUND_BF16,
                                           want_rowstats=True, want_phat=True)
    B, N, Hq, Hkv, D = w.B, w.N, w.Hq, w.Hkv, w.Dqk
    Qr, _ = orc.dequantize(quant["Q"], B, N, Hq, D)
    Kr, _ = orc.dequantize(quant["K"], B, N, Hkv, D)
    Vr, Vc = orc.dequantize(quant["V"], B, N, Hkv, D)
    dOr, _ = orc.dequantize(quant["dO"], B, N, Hq, D)
    ref = torch_attention(Qr.transpose(0, 2, 1, 3), Kr.transpose(0, 2, 1, 3), Vr.transpose(0, 2, 1, 3),
                          np.zeros((B, N, Hq, D)), w.tau)
    P = ref["P"]                                   # exact probabilities from the same scores
    Ph = out["phat"]
    dO = d["do"].astype(np.float64).transpose(0, 2, 1, 3)
    O = out["O_unrounded"].transpose(0, 2, 1, 3)
    Ost = out["O"].transpose(0, 2, 1, 3)
    G = Hq // Hkv
    Vr_h = np.repeat(Vr, G, axis=1)
    Vc_h = np.repeat(Vc, G, axis=1)
    t1 = np.einsum("bhik,bhik->bhi", dOr, (P - Ph) @ Vr_h)
    t2 = np.einsum("bhik,bhik->bhi", dOr - dO, Ph @ Vr_h)
    t3 = np.einsum("bhik,bhik->bhi", dO, Ph @ (Vr_h - Vc_h))
    t4 = np.einsum("bhik,bhik->bhi", dO, O - Ost)
    eps = out["rowstats"][..., orc.ST_SUM_DS]
    scale = out["rowstats"][..., orc.ST_SUMABS_DS]
    assert np.max(np.abs(eps - (t1 + t2 + t3 + t4)) / np.maximum(scale, 1e-300)) < 1e-10
    assert np.median(np.abs(t1) / scale) > 1e-5 and np.median(np.abs(t2) / scale) > 1e-5


def test_consistent_do_residual_decomposition(orc):
    """Consistent dO (the saved-output correction with dO replaced by its
    dequantized row copy, Sec. 3.4 / App. B.6): the gradient-quantization
    term of the stale decomposition vanishes and what remains is
       eps_i = sum_k dOr_ik sum_j (P - Phat)_ij Vr_jk          (probability)
             + sum_k dOr_ik sum_j Phat_ij (Vr - Vc)_jk          (two V copies)
             + sum_k dOr_ik (O - O_stored)_ik                   (storage)
    (the paper's residual with one V copy and exact O is the first term)."""
    w, d = _quantized_case(orc, N=64)
    outs = {}
    for mode in (orc.DELTA_CONSISTENT_DO, orc.DELTA_STALE_ROWSUM):
        outs[mode], quant = orc.attention_from_inputs(d["q"], d["k"], d["v"], d["do"], w.tau, delta_mode=mode,
                                                      o_round=orc.ROUND_BF16, want_rowstats=True, want_phat=True)
    out = outs[orc.DELTA_CONSISTENT_DO]
    B, N, Hq, Hkv, D = w.B, w.N, w.Hq, w.Hkv, w.Dqk
    Qr, _ = orc.dequantize(quant["Q"], B, N, Hq, D)
    Kr, _ = orc.dequantize(quant["K"], B, N, Hkv, D)
    Vr, Vc = orc.dequantize(quant["V"], B, N, Hkv, D)
    dOr, _ = orc.dequantize(quant["dO"], B, N, Hq, D)
    ref = torch_attention(Qr.transpose(0, 2, 1, 3), Kr.transpose(0, 2, 1, 3), Vr.transpose(0, 2, 1, 3),
                          np.zeros((B, N, Hq, D)), w.tau)
    P, Ph = ref["P"], out["phat"]
    O = out["O_unrounded"].transpose(0, 2, 1, 3)
    Ost = out["O"].transpose(0, 2, 1, 3)
    G = Hq // Hkv
    Vr_h, Vc_h = np.repeat(Vr, G, axis=1), np.repeat(Vc, G, axis=1)
    # the correction itself: <dOr_i, O_stored_i>
    assert np.allclose(out["delta"], np.einsum("bhik,bhik->bhi", dOr, Ost), rtol=1e-12, atol=1e-15)
    t1 = np.einsum("bhik,bhik->bhi", dOr, (P - Ph) @ Vr_h)
    t3 = np.einsum("bhik,bhik->bhi", dOr, Ph @ (Vr_h - Vc_h))
    t4 = np.einsum("bhik,bhik->bhi", dOr, O - Ost)
    eps = out["rowstats"][..., orc.ST_SUM_DS]
    scale = out["rowstats"][..., orc.ST_SUMABS_DS]
    assert np.max(np.abs(eps - (t1 + t3 + t4)) / np.maximum(scale, 1e-300)) < 1e-10
    # a mismatch remains (the probability term), smaller than the stale one
    eps_stale = outs[orc.DELTA_STALE_ROWSUM]["rowstats"][..., orc.ST_SUM_DS]
    assert np.median(np.abs(t1) / scale) > 1e-5
    assert np.median(np.abs(eps) / scale) < np.median(np.abs(eps_stale) / scale)


def test_consistent_do_equals_stale_without_quantization(orc):
    """With exact operands the dequantized dO is the raw dO, so the two
    saved-output corrections coincide."""
    q, k, v, do = inputs(1, 40, 2, 1, 32, 32, seed=4)
    r = {m: orc.attention_from_inputs(q, k, v, do, 0.2, delta_mode=m, exact_inputs=True)[0]["delta"]
         for m in (orc.DELTA_CONSISTENT_DO, orc.DELTA_STALE_ROWSUM)}
    assert np.array_equal(r[orc.DELTA_CONSISTENT_DO], r[orc.DELTA_STALE_ROWSUM])


def test_matched_delta_bilinearity(orc):
    """delta_matched_i = <dOr_i, (P Vr)_i> (the auxiliary-output identity of
    App. C.4.1), computed through a different contraction order."""
    w, d = _quantized_case(orc, N=96)
    out, quant = orc.attention_from_inputs(d["q"], d["k"], d["v"], d["do"], w.tau, want_rowstats=True)
    B, N, Hq, Hkv, D = w.B, w.N, w.Hq, w.Hkv, w.Dqk
    Qr, _ = orc.dequantize(quant["Q"], B, N, Hq, D)
    Kr, _ = orc.dequantize(quant["K"], B, N, Hkv, D)
    Vr, _ = orc.dequantize(quant["V"], B, N, Hkv, D)
    dOr, _ = orc.dequantize(quant["dO"], B, N, Hq, D)
    P = torch_attention(Qr.transpose(0, 2, 1, 3), Kr.transpose(0, 2, 1, 3), Vr.transpose(0, 2, 1, 3),
                        np.zeros((B, N, Hq, D)), w.tau)["P"]
    Ob = P @ np.repeat(Vr, Hq // Hkv, axis=1)
    delta_b = np.einsum("bhik,bhik->bhi", dOr, Ob)
    assert np.max(np.abs(out["delta"] - delta_b)) < 1e-12 * np.max(np.abs(delta_b))
    st = out["rowstats"]
    assert np.max(np.abs(st[..., orc.ST_SUM_P] - 1.0)) < 1e-13


def test_zero_queries_closed_forms(orc):
    """Q = 0: every visible key has P_ij = 1/(i+1), LSE_i = ln(i+1); every
    forward group codes 2^{x-E} = 256 exactly, so O_i is the mean of Vc_0..i;
    dV has the closed form sum_i C8(256/(i+1))/256 dOc_i (torch's FP8 cast)."""
    B, N, H, D = 1, 64, 1, 32
    rng = np.random.default_rng(11)
    q = np.zeros((B, N, H, D)); k = rng.standard_normal((B, N, H, D))
    v = rng.standard_normal((B, N, H, D)); do = rng.standard_normal((B, N, H, D))
    out, quant = orc.attention_from_inputs(q, k, v, do, 0.125, o_round=orc.ROUND_NONE)
    i = np.arange(N)
    assert np.allclose(out["LSE"][0, 0], np.log(i + 1), rtol=0, atol=1e-14)
    _, Vc = orc.dequantize(quant["V"], B, N, H, D)
    mean = np.cumsum(Vc[0, 0], axis=0) / (i + 1)[:, None]
    assert np.max(np.abs(out["O"][0, :, 0] - mean)) < 1e-13
    _, dOc = orc.dequantize(quant["dO"], B, N, H, D)
    pb = torch.tensor(256.0 / (i + 1)).to(torch.float8_e4m3fn).to(torch.float64).numpy() / 256.0
    W = np.tril(np.ones((N, N))) * pb[:, None]          # W[i, j] = Pb_ij for j <= i
    dV_ref = W.T @ dOc[0, 0]
    assert np.max(np.abs(out["dV"][0, :, 0] - dV_ref)) < 1e-12


def test_row_zero_and_dk_column_sums(orc):
    w, d = _quantized_case(orc, N=64)
    out, quant = orc.attention_from_inputs(d["q"], d["k"], d["v"], d["do"], w.tau, want_rowstats=True,
                                           want_ds=True)
    # row 0 sees one key: P_00 = 1 and the matched dS row vanishes
    assert np.all(out["dsraw"][:, :, 0, :] == 0) and np.all(out["rowstats"][:, :, 0, orc.ST_SUMABS_DS] == 0)
    # eq. of the GQA key-sum (App. C.1): sum_j dK_j = tau sum_i Qc_i sum_j dS'_ij
    B, N, Hq, Hkv, D = w.B, w.N, w.Hq, w.Hkv, w.Dqk
    _, Qc = orc.dequantize(quant["Q"], B, N, Hq, D)
    rs = out["rowstats"][..., orc.ST_SUM_DSCAST]                   # [B,Hq,N]
    G = Hq // Hkv
    lhs = out["dK"].sum(axis=1)                                     # [B,Hkv,D]
    rhs = w.tau * np.einsum("bhn,bhnd->bhd", rs, Qc).reshape(B, Hkv, G, D).sum(2)
    assert np.max(np.abs(lhs - rhs)) < 1e-12 * np.max(np.abs(out["dK"]))
    # exact arithmetic (Sec. 3.1 / App. A.3): key gradients sum to zero per channel
    q, k, v, do = inputs(1, 48, 2, 1, 16, 16, seed=3)
    ex, _ = orc.attention_from_inputs(q, k, v, do, 0.25, flags=orc.EXACT_ALL, exact_inputs=True,
                                      o_round=orc.ROUND_NONE)
    assert np.max(np.abs(ex["dK"].sum(axis=1))) < 1e-12 * np.max(np.abs(ex["dK"]))


def test_gqa_group_sum(orc):
    """dK/dV of a shared KV head equal the sum over its query heads of the
    per-head gradients (repeat the KV head, run MHA, sum the group)."""
    q, k, v, do = inputs(1, 64, 4, 2, 32, 32, seed=5)
    a, _ = orc.attention_from_inputs(q, k, v, do, 0.2)
    b, _ = orc.attention_from_inputs(q, np.repeat(k, 2, axis=2), np.repeat(v, 2, axis=2), do, 0.2)
    # quantization of the repeated K/V is identical per head, so all outputs agree
    assert np.array_equal(a["O"], b["O"]) and np.allclose(a["dQ"], b["dQ"], rtol=0, atol=1e-12)
    assert np.allclose(a["dK"], b["dK"].reshape(1, 64, 2, 2, 32).sum(3), rtol=0, atol=1e-12)
    assert np.allclose(a["dV"], b["dV"].reshape(1, 64, 2, 2, 32).sum(3), rtol=0, atol=1e-12)


def test_operand_wiring(orc):
    """Each dequantized copy feeds only the contractions of reading R3:
    perturbing it changes exactly the outputs that depend on it."""
    B, N, Hq, Hkv, D = 1, 64, 2, 1, 32
    q, k, v, do = inputs(B, N, Hq, Hkv, D, D, seed=9)
    ops = {}
    for nm, t in (("Q", q), ("K", k), ("V", v), ("dO", do)):
        xr, xc = orc.dequantize(orc.quantize(t), B, N, t.shape[2], D)
        ops[nm + "r"], ops[nm + "c"] = xr, xc
    def run(o, mode=orc.DELTA_MATCHING):
        return orc.attention(B, N, Hq, Hkv, D, D, 0.2, o, do, delta_mode=mode, o_round=orc.ROUND_NONE)
    base = run(ops)
    expect = {"Qr": {"O", "LSE", "delta", "dQ", "dK", "dV"}, "Kr": {"O", "LSE", "delta", "dQ", "dK", "dV"},
              "Vr": {"delta", "dQ", "dK"}, "dOr": {"delta", "dQ", "dK"}, "Qc": {"dK"}, "Kc": {"dQ"},
              "Vc": {"O"}, "dOc": {"dV"}}
    rng = np.random.default_rng(1)
    for nm, changed in expect.items():
        o2 = dict(ops)
        o2[nm] = ops[nm] + 0.1 * rng.standard_normal(ops[nm].shape)
        r = run(o2)
        got = {k for k in ("O", "LSE", "delta", "dQ", "dK", "dV") if not np.array_equal(r[k], base[k])}
        assert got == changed, (nm, got)
    # in stale mode the stored O (hence Vc) also enters delta, dQ and dK
    base_s = run(ops, orc.DELTA_STALE_ROWSUM)
    o2 = dict(ops); o2["Vc"] = ops["Vc"] * 1.01
    r = run(o2, orc.DELTA_STALE_ROWSUM)
    got = {k for k in ("O", "LSE", "delta", "dQ", "dK", "dV") if not np.array_equal(r[k], base_s[k])}
    assert got == {"O", "delta", "dQ", "dK"}


def test_ds_cast_blocks(orc):
    """dS' is the 32x32-block power-of-two cast of dS (reading R7), checked
    against torch's FP8 cast of each block scaled by its exponent."""
    w, d = _quantized_case(orc, N=96)
    out, _ = orc.attention_from_inputs(d["q"], d["k"], d["v"], d["do"], w.tau, want_ds=True)
    ds, dsh = out["dsraw"], out["dshat"]
    N = w.N
    for b in range(w.B):
        for h in range(w.Hq):
            for i0 in range(0, N, 32):
                for j0 in range(0, i0 + 1, 32):
                    blk = ds[b, h, i0:i0 + 32, j0:j0 + 32]
                    amax = np.abs(blk).max()
                    e = int(orc.pow2_exponent([amax])[0])
                    assert amax <= 448 * 2.0 ** e and (amax > 224 * 2.0 ** e or e == -127)
                    ref = torch.tensor(blk * 2.0 ** -e).to(torch.float8_e4m3fn).to(torch.float64).numpy() * 2.0 ** e
                    assert np.array_equal(dsh[b, h, i0:i0 + 32, j0:j0 + 32], ref)
            assert np.all(np.triu(dsh[b, h], 1) == 0)


def test_forward_probability_codes(orc):
    """Forward probabilities (reading R5): per row and aligned 32-key group,
    phat * ell is a power-of-two multiple of an E4M3 value, equal to torch's
    FP8 cast of 2^{x-E_g} with E_g minimal such that the group max is <= 448."""
    B, N, H, D = 1, 96, 1, 32
    q, k, v, do = inputs(B, N, H, H, D, D, seed=21, scale=1.5)
    tau = 0.3
    out, _ = orc.attention_from_inputs(q, k, v, do, tau, flags=orc.EXACT_PBWD | orc.EXACT_DS,
                                       exact_inputs=True, o_round=orc.ROUND_NONE, want_phat=True)
    S = tau * np.einsum("nd,md->nm", q[0, :, 0], k[0, :, 0])
    x = S * np.log2(np.e)
    for i in range(N):
        M = np.ceil(x[i, :i + 1].max())
        ell = np.sum(np.exp2(x[i, :i + 1] - M))
        for g0 in range(0, i + 1, 32):
            js = np.arange(g0, min(g0 + 32, i + 1))
            xg = x[i, js].max()
            E = int(np.ceil(xg - np.log2(448.0)))
            if np.exp2(xg - (E - 1)) <= 448: E -= 1
            if np.exp2(xg - E) > 448: E += 1
            pre = np.exp2(x[i, js] - E)
            assert 224 < pre.max() <= 448
            codes = torch.tensor(pre).to(torch.float8_e4m3fn).to(torch.float64).numpy()
            want = codes * np.exp2(E - M) / ell
            assert np.allclose(out["phat"][0, 0, i, js], want, rtol=1e-12, atol=0)
    # O = phat @ Vc exactly in this mode (Vc = raw v)
    assert np.allclose(out["O"][0, :, 0], out["phat"][0, 0] @ v[0, :, 0], rtol=1e-12, atol=1e-13)


def test_delta_injection_is_affine(orc):
    """App. C.1 correction-pass consistency: rerunning the gradient pass with
    delta = 0 and delta = 1 gives row sums R(c) = S_PdP - c S_P, and
    delta* = R(0) / (R(0) - R(1)) equals the matched correction."""
    w, d = _quantized_case(orc, N=64)
    kw = dict(want_rowstats=True)
    base, _ = orc.attention_from_inputs(d["q"], d["k"], d["v"], d["do"], w.tau, **kw)
    z = np.zeros((w.B, w.Hq, w.N))
    r0, _ = orc.attention_from_inputs(d["q"], d["k"], d["v"], d["do"], w.tau, delta_in=z, **kw)
    r1, _ = orc.attention_from_inputs(d["q"], d["k"], d["v"], d["do"], w.tau, delta_in=z + 1, **kw)
    R0 = r0["rowstats"][..., orc.ST_SUM_DS]; R1 = r1["rowstats"][..., orc.ST_SUM_DS]
    dstar = R0 / (R0 - R1)
    assert np.max(np.abs(dstar - base["delta"]) / np.maximum(np.abs(base["delta"]), 1e-3)) < 1e-10
    # changing only delta leaves O and dV unchanged (App. C.4.1)
    assert np.array_equal(r0["O"], base["O"]) and np.array_equal(r0["dV"], base["dV"])
    assert not np.array_equal(r0["dQ"], base["dQ"])


def test_probability_clamp_with_injected_lse(orc):
    """Reading R6 (App. B.6.3): the backward's recomputed P is clamped at 1
    and P' = C8(256 P) 2^-8.  An LSE 0.5 below the forward's inflates every
    P by e^0.5, so rows whose largest P exceeds e^-0.5 reach the clamp.
    Pinned against P recomputed here from the dequantized operands (numpy
    matmul) and torch's E4M3 cast: sum_j P_ij and sum_j P'_ij per row, with
    a dropped clamp failing both."""
    w, d = _quantized_case(orc, N=64)
    base, quant = orc.attention_from_inputs(d["q"], d["k"], d["v"], d["do"], w.tau)
    lse_in = base["LSE"] - 0.5
    out, _ = orc.attention_from_inputs(d["q"], d["k"], d["v"], d["do"], w.tau, lse_in=lse_in,
                                       want_rowstats=True)
    B, N, Hq, Hkv, D = w.B, w.N, w.Hq, w.Hkv, w.Dqk
    Qr, _ = orc.dequantize(quant["Q"], B, N, Hq, D)
    Kr, _ = orc.dequantize(quant["K"], B, N, Hkv, D)
    S = w.tau * (Qr @ np.repeat(Kr, Hq // Hkv, axis=1).transpose(0, 1, 3, 2))
    vis = np.tril(np.ones((N, N), dtype=bool))
    P_raw = np.where(vis, np.exp(np.where(vis, S, 0.0) - lse_in[..., None]), 0.0)
    P = np.minimum(P_raw, 1.0)
    assert (P_raw > 1.0).sum() >= B * Hq          # the clamp is reached (row 0 of every head at least)
    st = out["rowstats"]
    assert np.allclose(st[..., orc.ST_SUM_P], P.sum(-1), rtol=1e-12, atol=0)
    assert not np.allclose(st[..., orc.ST_SUM_P], P_raw.sum(-1), rtol=1e-6, atol=0)
    pc = torch.tensor(256.0 * P).to(torch.float8_e4m3fn).to(torch.float64).numpy() / 256.0
    assert np.allclose(st[..., orc.ST_SUM_PCAST], pc.sum(-1), rtol=1e-12, atol=0)
    # the forward does not read the injected LSE
    assert np.array_equal(out["O"], base["O"]) and np.array_equal(out["LSE"], base["LSE"])


def test_row_window_equals_whole_problem(orc):
    """row_lo restricts the oracle to the causal suffix (query rows and keys
    >= row_lo); by causality those outputs do not depend on anything left
    out, so they equal the whole problem's bit for bit (same arithmetic in
    the same order), and everything before row_lo stays zero."""
    w, d = _quantized_case(orc, "gqa_d128_8k", seed=2, B=1, N=160, Hq=4, Hkv=2)
    full, _ = orc.attention_from_inputs(d["q"], d["k"], d["v"], d["do"], w.tau, want_rowstats=True)
    win, _ = orc.attention_from_inputs(d["q"], d["k"], d["v"], d["do"], w.tau, want_rowstats=True, row_lo=96)
    for name in ("O", "dQ", "dK", "dV"):
        assert np.array_equal(win[name][:, 96:], full[name][:, 96:]), name
        assert not np.any(win[name][:, :96]), name
    for name in ("LSE", "delta"):
        assert np.array_equal(win[name][..., 96:], full[name][..., 96:]), name
    assert np.array_equal(win["rowstats"][:, :, 96:], full["rowstats"][:, :, 96:])
    with pytest.raises(ValueError):
        orc.attention_from_inputs(d["q"], d["k"], d["v"], d["do"], w.tau, row_lo=40)


def test_term_magnitude_statistic(orc):
    """ST_SUM_P_ABSTERMS = sum_j P_ij sum_c |dOr_ic Vr_jc| (the scale the FP32
    accumulation of dP works on), against numpy on the dequantized operands;
    it bounds |sum_j P_ij dP_ij| from above."""
    w, d = _quantized_case(orc, N=64)
    out, quant = orc.attention_from_inputs(d["q"], d["k"], d["v"], d["do"], w.tau, want_rowstats=True)
    B, N, Hq, Hkv, D = w.B, w.N, w.Hq, w.Hkv, w.Dqk
    Qr, _ = orc.dequantize(quant["Q"], B, N, Hq, D)
    Kr, _ = orc.dequantize(quant["K"], B, N, Hkv, D)
    Vr, _ = orc.dequantize(quant["V"], B, N, Hkv, D)
    dOr, _ = orc.dequantize(quant["dO"], B, N, Hq, D)
    G = Hq // Hkv
    S = w.tau * (Qr @ np.repeat(Kr, G, axis=1).transpose(0, 1, 3, 2))
    vis = np.tril(np.ones((N, N), dtype=bool))
    P = np.where(vis, np.exp(np.where(vis, S, 0.0) - out["LSE"][..., None]), 0.0)
    T = np.einsum("bhij,bhijk->bhi", P, np.abs(dOr[:, :, :, None, :] * np.repeat(Vr, G, axis=1)[:, :, None, :, :]))
    st = out["rowstats"]
    assert np.allclose(st[..., orc.ST_SUM_P_ABSTERMS], T, rtol=1e-12, atol=0)
    assert np.all(np.abs(st[..., orc.ST_SUM_PDP]) <= st[..., orc.ST_SUM_P_ABSTERMS] * (1 + 1e-12))
