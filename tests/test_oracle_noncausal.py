"""Pins of the oracle without the causal mask and with a key length that
differs from the query length (softmax attention of Sec. 2.3 over all keys):
torch autograd in exact arithmetic, finite differences, invariance under a
permutation of the keys, agreement with the causal problem on the last row
(which sees every key either way), the zero-row-sum invariant of matched
correction (Sec. 3.1, 3.4) and the zero column sums of the key gradient
(App. A.3)."""
import numpy as np
import pytest
import torch

from paper_2609_37852_amd import synth


def torch_full_attention(q, k, v, do, tau):
    """Textbook attention without a mask in float64 with torch autograd."""
    q, k, v, do = (torch.tensor(np.asarray(t, np.float64)) for t in (q, k, v, do))
    q.requires_grad_(True); k.requires_grad_(True); v.requires_grad_(True)
    G = q.shape[2] // k.shape[2]
    Q = q.permute(0, 2, 1, 3)
    K = k.repeat_interleave(G, dim=2).permute(0, 2, 1, 3)
    V = v.repeat_interleave(G, dim=2).permute(0, 2, 1, 3)
    S = tau * torch.matmul(Q, K.transpose(-1, -2).contiguous())
    P = torch.softmax(S, -1)
    O = torch.matmul(P, V).permute(0, 2, 1, 3)
    lse = torch.logsumexp(S, -1)
    O.backward(do)
    return dict(O=O.detach().numpy(), LSE=lse.detach().numpy(), dQ=q.grad.numpy(), dK=k.grad.numpy(),
                dV=v.grad.numpy())


def rel(a, b):
    return np.linalg.norm(a - b) / max(np.linalg.norm(b), 1e-300)


def inputs(B, N, Nk, Hq, Hkv, Dqk, Dv, seed=0, scale=1.0):
    rng = np.random.default_rng(seed)
    return (rng.standard_normal((B, N, Hq, Dqk)) * scale, rng.standard_normal((B, Nk, Hkv, Dqk)) * scale,
            rng.standard_normal((B, Nk, Hkv, Dv)), rng.standard_normal((B, N, Hq, Dv)))


def exact(orc, q, k, v, do, tau, **kw):
    out, _ = orc.attention_from_inputs(q, k, v, do, tau, flags=orc.EXACT_ALL, exact_inputs=True,
                                       o_round=orc.ROUND_NONE, causal=False, **kw)
    return out


@pytest.mark.parametrize("shape", [(2, 40, 72, 4, 2, 16, 16), (1, 33, 33, 2, 1, 24, 8), (1, 1, 5, 1, 1, 8, 8),
                                   (1, 70, 9, 3, 3, 8, 16)])
def test_exact_mode_matches_torch_autograd(orc, shape):
    B, N, Nk, Hq, Hkv, Dqk, Dv = shape
    q, k, v, do = inputs(*shape)
    tau = 1 / np.sqrt(Dqk)
    out = exact(orc, q, k, v, do, tau)
    ref = torch_full_attention(q, k, v, do, tau)
    assert out["dK"].shape == (B, Nk, Hkv, Dqk)
    for name in ("O", "LSE", "dQ", "dK", "dV"):
        assert rel(out[name], ref[name]) < 1e-12, name


def test_finite_differences(orc):
    q, k, v, do = inputs(1, 3, 5, 2, 1, 4, 4, seed=3)
    tau = 0.6

    def loss(qq, kk, vv):
        return float(np.sum(exact(orc, qq, kk, vv, do, tau)["O"] * do))
    out = exact(orc, q, k, v, do, tau)
    h = 1e-6
    for name, t, g in (("q", q, out["dQ"]), ("k", k, out["dK"]), ("v", v, out["dV"])):
        num = np.zeros_like(t)
        for idx in np.ndindex(t.shape):
            tp, tm = t.copy(), t.copy()
            tp[idx] += h
            tm[idx] -= h
            args = {"q": q, "k": k, "v": v}
            args[name] = tp
            lp = loss(args["q"], args["k"], args["v"])
            args[name] = tm
            lm = loss(args["q"], args["k"], args["v"])
            num[idx] = (lp - lm) / (2 * h)
        assert np.max(np.abs(num - g)) < 1e-7, name


def test_key_permutation_invariance(orc):
    """Without a mask the keys form a set: permuting K and V together leaves
    O, LSE and dQ unchanged and permutes dK and dV the same way."""
    q, k, v, do = inputs(1, 24, 40, 2, 1, 16, 8, seed=5)
    perm = np.random.default_rng(1).permutation(40)
    a = exact(orc, q, k, v, do, 0.3)
    b = exact(orc, q, k[:, perm], v[:, perm], do, 0.3)
    for name in ("O", "LSE", "dQ"):
        assert rel(b[name], a[name]) < 1e-13, name
    for name in ("dK", "dV"):
        assert rel(b[name], a[name][:, perm]) < 1e-13, name


@pytest.mark.parametrize("mode", ["matching", "stale"])
def test_last_row_equals_causal(orc, mode):
    """The last query row sees every key with or without the mask, in the
    same aligned 32-key groups: O, LSE and delta of that row agree exactly
    (quantized operands, cast probabilities)."""
    w = synth.with_shape(synth.WORKLOADS["tiny_mha_128"], B=1, N=96, Hq=2, Hkv=1)
    d = synth.generate(w, seed=2)
    dm = orc.DELTA_MATCHING if mode == "matching" else orc.DELTA_STALE_ROWSUM
    kw = dict(delta_mode=dm, o_round=orc.ROUND_NONE)
    c, _ = orc.attention_from_inputs(d["q"], d["k"], d["v"], d["do"], w.tau, causal=True, **kw)
    n, _ = orc.attention_from_inputs(d["q"], d["k"], d["v"], d["do"], w.tau, causal=False, **kw)
    assert np.array_equal(n["O"][:, -1], c["O"][:, -1])
    assert np.array_equal(n["LSE"][..., -1], c["LSE"][..., -1])
    assert np.array_equal(n["delta"][..., -1], c["delta"][..., -1])
    # the other rows see more keys without the mask
    assert not np.allclose(n["O"][:, :-32], c["O"][:, :-32])


def test_matched_invariant_and_stale_violation(orc):
    w = synth.with_shape(synth.WORKLOADS["tiny_mha_128"], B=1, N=64, Hq=2, Hkv=1)
    d = synth.generate(w, seed=4)
    rng = np.random.default_rng(9)
    k = rng.standard_normal((1, 160, 1, w.Dqk)).astype(np.float32)
    v = rng.standard_normal((1, 160, 1, w.Dv)).astype(np.float32)
    outs = {}
    for name, mode in (("m", orc.DELTA_MATCHING), ("s", orc.DELTA_STALE_ROWSUM)):
        outs[name], _ = orc.attention_from_inputs(d["q"], k, v, d["do"], w.tau, causal=False, delta_mode=mode,
                                                  want_rowstats=True)
    st = outs["m"]["rowstats"]
    r = np.abs(st[..., orc.ST_SUM_DS]) / st[..., orc.ST_SUMABS_DS]
    assert r.max() < 1e-13
    ss = outs["s"]["rowstats"]
    rs = np.abs(ss[..., orc.ST_SUM_DS]) / ss[..., orc.ST_SUMABS_DS]
    assert np.median(rs) > 1e-4       # BF16 output and FP8 operands: the stale shortcut misses


def test_key_gradient_column_sums(orc):
    """Matched correction in exact arithmetic: sum_j dS_ij = 0, so the key
    gradient sums to zero over the keys (App. A.3)."""
    q, k, v, do = inputs(2, 20, 44, 2, 2, 8, 8, seed=8)
    out = exact(orc, q, k, v, do, 0.5)
    s = out["dK"].sum(axis=1)
    assert np.max(np.abs(s)) < 1e-12 * np.max(np.abs(out["dK"])) * 44


def test_rejects_invalid(orc):
    q, k, v, do = inputs(1, 32, 64, 1, 1, 32, 32)
    with pytest.raises((ValueError, AssertionError)):
        orc.attention_from_inputs(q, k, v, do, 0.2, causal=True)        # causal needs equal lengths
    q2, k2, v2, do2 = inputs(1, 64, 64, 1, 1, 32, 32)
    with pytest.raises(ValueError):
        orc.attention_from_inputs(q2, k2, v2, do2, 0.2, causal=False, row_lo=32)
