"""The protected-dP backward (App. B.6.3, correction variants; App. C.4.2):
dP = dO V^T from BF16 operands with FP32 accumulation, every other product in
FP8, the stale correction.  Against the oracle's protected-dP variant on the
same seeded inputs: the stale correction, and dQ, dK, dV given the oracle's
correction (as in the other stale-mode cases: the correction reads the BF16
O), within the parity bounds; dV, which does not involve dP, bit for bit
that of the FP8-dP backward; the instrumented kernel's gradients bit for bit
the plain one's; a padded batch of sequences of their own lengths per
sequence against the oracle."""
import numpy as np
import pytest
import torch

import oracle as orc
import paper_2609_37852_amd as pk
from paper_2609_37852_amd import synth
from _helpers import REL_TOL, block_errors, check_blocks, np64, rel_err, say, to_dev

pytestmark = pytest.mark.gpu

CASES = [
    ("gqa_d128_8k", dict(B=1, N=320, Hq=4, Hkv=2)),
    ("tiny_mha_128", dict(B=2, N=96, Nk=160, causal=False)),
    ("mla_d192_4k", dict(B=1, N=128, Hq=2, Hkv=2)),
    ("gqa_d128_8k", dict(B=1, N=256, Hq=4, Hkv=1, causal=False, Nk=192)),
]


def _problem(w, flags=pk.FLAG_PROTECTED_DP, **kw):
    return pk.Problem(w.B, w.N, w.Hq, w.Hkv, w.Dqk, w.Dv, float(np.float32(w.tau)), causal=int(w.causal),
                      seqlen_kv=w.Nk, flags=flags, **kw)


def _hilo(delta):
    hi = delta.astype(np.float32)
    lo = (delta - hi.astype(np.float64)).astype(np.float32)
    return torch.from_numpy(np.stack([hi, lo], axis=-1)).cuda()


@pytest.mark.parametrize("name,kw", CASES, ids=[f"{n}-{'-'.join(f'{k}{v}' for k, v in kw.items())}" for n, kw in CASES])
def test_protected_dp_parity(name, kw):
    w = synth.with_shape(synth.WORKLOADS[name], **kw)
    say(f"protected dP {w}")
    d = synth.generate(w, seed=21)
    q, k, v, do = (to_dev(d[n], w.dtype) for n in ("q", "k", "v", "do"))
    mq, mk, mv, mdo = (pk.attn_fp8_quantize(t) for t in (q, k, v, do))
    p = _problem(w)
    o, lse = pk.attn_fp8_fwd(p, mq, mk, mv)
    ref, _ = orc.attention_from_inputs(d["q"], d["k"], d["v"], d["do"], float(np.float32(w.tau)),
                                       delta_mode=orc.DELTA_STALE_ROWSUM, causal=w.causal, protected_dp=True)
    # the stale correction itself (GPU O against the oracle's O)
    delta = pk.attn_fp8_delta(p, pk.DELTA_STALE_ROWSUM, None, None, None, None, None, do, o)
    din = _hilo(ref["delta"])
    plain = pk.attn_fp8_bwd_protected_dp(p, mq, mk, mdo, lse, do, v, o, delta_in=din, grad_dtype=torch.float32)
    stats = pk.attn_fp8_bwd_protected_dp(p, mq, mk, mdo, lse, do, v, o, delta_in=din, grad_dtype=torch.float32,
                                         rowstats=True)
    # the same backward with FP8 dP
    f8 = pk.attn_fp8_bwd(_problem(w, flags=0), pk.DELTA_STALE_ROWSUM, mq, mk, mv, mdo, lse, do, o, delta_in=din,
                         grad_dtype=torch.float32)
    # the call's own stale correction (no delta_in) gives the same gradients
    # as passing that correction in
    own = pk.attn_fp8_bwd_protected_dp(p, mq, mk, mdo, lse, do, v, o, grad_dtype=torch.float32)
    via = pk.attn_fp8_bwd_protected_dp(p, mq, mk, mdo, lse, do, v, o, delta_in=delta, grad_dtype=torch.float32)
    torch.cuda.synchronize()
    for a, b in zip(plain[:3], stats[:3]):
        assert torch.equal(a, b), "instrumented backward differs from the plain one"
    for a, b in zip(own[:3], via[:3]):
        assert torch.equal(a, b)
    assert torch.equal(plain[2], f8[2]), "dV depends on dP"
    assert not torch.equal(plain[0], f8[0])
    g = dict(dQ=np64(plain[0]), dK=np64(plain[1]), dV=np64(plain[2]))
    errs = {n: rel_err(g[n], ref[n]) for n in g}
    blk = {n: block_errors(g[n], ref[n]) for n in g}
    dl = np64(delta)
    errs["delta"] = rel_err(dl[..., 0] + dl[..., 1], ref["delta"])
    # the FP8-dP backward against the same oracle variant (its dP operands
    # differ): a larger dQ error
    errs["dQ_fp8dp"] = rel_err(np64(f8[0]), ref["dQ"])
    say("  errors", {n: f"{e:.2e}" for n, e in errs.items()})
    for n in ("dQ", "dK", "dV"):
        assert errs[n] <= REL_TOL, (n, errs[n])
    check_blocks(blk)
    assert errs["delta"] < 1e-2
    assert errs["dQ"] < errs["dQ_fp8dp"]


def test_protected_dp_varlen():
    """Sequences of their own lengths (NaN padding) under protected dP: per
    sequence against the oracle's variant run on that sequence alone."""
    w = synth.with_shape(synth.WORKLOADS["gqa_d128_8k"], B=3, N=192, Hq=4, Hkv=2)
    lq = [192, 64, 0]
    d = synth.generate(w, seed=23)
    pad = {}
    for n in ("q", "k", "v", "do"):
        x = np.array(d[n], dtype=np.float32, copy=True)
        for b, L in enumerate(lq):
            x[b, L:] = np.nan
        pad[n] = to_dev(x, w.dtype)
    mq, mk, mv, mdo = (pk.attn_fp8_quantize(pad[n]) for n in ("q", "k", "v", "do"))
    p = _problem(w, seqlens_q=torch.tensor(lq, dtype=torch.int32, device="cuda"))
    o, lse = pk.attn_fp8_fwd(p, mq, mk, mv)
    refs, din = {}, np.zeros((w.B, w.Hq, w.N))
    for b, L in enumerate(lq):
        if L == 0:
            continue
        ws = synth.with_shape(w, B=1, N=L)
        refs[b], _ = orc.attention_from_inputs(*(d[n][b:b + 1, :L] for n in ("q", "k", "v", "do")),
                                               float(np.float32(w.tau)), delta_mode=orc.DELTA_STALE_ROWSUM,
                                               protected_dp=True)
        din[b, :, :L] = refs[b]["delta"][0]
    out = tuple(torch.full(s, 7.0, dtype=torch.float32, device="cuda")
                for s in ((w.B, w.N, w.Hq, w.Dqk), (w.B, w.N, w.Hkv, w.Dqk), (w.B, w.N, w.Hkv, w.Dv)))
    dq, dk, dv, _ = pk.attn_fp8_bwd_protected_dp(p, mq, mk, mdo, lse, pad["do"], pad["v"], o, delta_in=_hilo(din),
                                                 grad_dtype=torch.float32, out=out)
    torch.cuda.synchronize()
    g = dict(dQ=np64(dq), dK=np64(dk), dV=np64(dv))
    for b, L in enumerate(lq):
        for n in g:
            assert np.all(g[n][b, L:] == 7.0), (b, n)
        if L == 0:
            continue
        errs = {n: rel_err(g[n][b:b + 1, :L], refs[b][n]) for n in g}
        say(f"  seq {b} ({L})", {n: f"{e:.2e}" for n, e in errs.items()})
        for n in g:
            assert errs[n] <= REL_TOL, (b, n, errs[n])
