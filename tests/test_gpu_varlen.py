"""Padded batches of sequences of their own lengths (seqlens_q / seqlens_kv):
every batch entry is its own attention problem over its first Lq_b queries
and Lk_b keys.  The padding of Q, K, V and dO holds NaN, so any read of it
would show in the results.  Per sequence, against the oracle run on that
sequence alone: O, LSE, the correction and the gradients within the parity
bounds, the zero-row-sum invariant on the GPU's own pre-cast dS (reading
R12); O, LSE, the correction and dQ also bit for bit equal to the kernels
run on the sequence alone (the query-major passes visit keys in the same
order either way).  Rows past a sequence keep what the output buffers held;
keys of a sequence without queries get zero gradients; a sequence with
queries and no keys is empty."""
import numpy as np
import pytest
import torch

import oracle as orc
import paper_2609_37852_amd as pk
from paper_2609_37852_amd import synth
from _helpers import REL_TOL, block_errors, check_blocks, invariant_report, rel_err, run_oracle, say, to_dev

pytestmark = pytest.mark.gpu

SENTINEL = 7.0
CASES = [
    # causal: a full sequence, ragged query tiles (96, 160 = 5 blocks of 32), an empty one
    ("gqa_d128_8k", dict(B=4, N=256, Hq=4, Hkv=2), [256, 96, 0, 160], None),
    ("gqa_d256_8k_qknorm", dict(B=2, N=160, Hq=2, Hkv=1), [96, 160], None),
    ("tiny_mha_128", dict(B=3, N=128), [32, 128, 64], None),
    # no mask: keys above / below the query length, keys without queries (b = 2)
    ("tiny_mha_128", dict(B=3, N=192, Nk=256, causal=False), [192, 32, 0], [96, 256, 64]),
    # queries without keys (b = 1): an empty sequence
    ("mla_d192_4k", dict(B=2, N=128, Nk=192, Hq=2, Hkv=2, causal=False), [64, 128], [192, 0]),
]


def _ids():
    return [f"{n}-{'-'.join(f'{k}{v}' for k, v in kw.items())}-q{'_'.join(map(str, lq))}" for n, kw, lq, _ in CASES]


def _eff(lq, lk, causal):
    """Per-sequence (queries, keys) as the kernels take them."""
    lk = list(lq) if causal else list(lk)
    return [(q if k > 0 else 0, k) for q, k in zip(lq, lk)]


def _padded(x, lens):
    y = np.array(x, dtype=np.float32, copy=True)
    for b, n in enumerate(lens):
        y[b, n:] = np.nan
    return y


def _full(shape, dtype):
    return torch.full(shape, SENTINEL, dtype=dtype, device="cuda")


def _run(w, d, lq, lk, mode=pk.DELTA_MATCHING, delta_in=None, flags=0):
    """The path on the padded batch; outputs pre-filled with SENTINEL."""
    B, N, Nk = w.B, w.N, w.nk
    q, do = (to_dev(_padded(d[n], lq), w.dtype) for n in ("q", "do"))
    k, v = (to_dev(_padded(d[n], lk if not w.causal else lq), w.dtype) for n in ("k", "v"))
    mq, mk, mv, mdo = (pk.attn_fp8_quantize(t) for t in (q, k, v, do))
    p = pk.Problem(B, N, w.Hq, w.Hkv, w.Dqk, w.Dv, float(np.float32(w.tau)), causal=int(w.causal), seqlen_kv=w.Nk,
                   seqlens_q=torch.tensor(lq, dtype=torch.int32, device="cuda"),
                   seqlens_kv=None if w.causal else torch.tensor(lk, dtype=torch.int32, device="cuda"), flags=flags)
    o, lse = pk.attn_fp8_fwd(p, mq, mk, mv, o=_full((B, N, w.Hq, w.Dv), torch.bfloat16),
                             lse=_full((B, w.Hq, N), torch.float32))
    delta = pk.attn_fp8_delta(p, mode, mq, mk, mv, mdo, lse, do, o, delta=_full((B, w.Hq, N, 2), torch.float32))
    res = {}
    for rs in (False, True):
        out = (_full((B, N, w.Hq, w.Dqk), torch.float32), _full((B, Nk, w.Hkv, w.Dqk), torch.float32),
               _full((B, Nk, w.Hkv, w.Dv), torch.float32))
        res[rs] = pk.attn_fp8_bwd(p, mode, mq, mk, mv, mdo, lse, do, o, delta_in=delta_in, grad_dtype=torch.float32,
                                  rowstats=rs, out=out)
    torch.cuda.synchronize()
    for a, b in zip(res[False][:3], res[True][:3]):
        assert torch.equal(a.view(torch.int32), b.view(torch.int32)), "instrumented backward differs from the plain"
    f = lambda t: t.float().cpu().numpy().astype(np.float64)
    dq, dk, dv, rs = res[False][0], res[False][1], res[False][2], res[True][3]
    return dict(O=f(o), LSE=f(lse), delta=f(delta), dQ=f(dq), dK=f(dk), dV=f(dv), rowstats=rs.cpu().numpy())


def _alone(w, d, b, nq, nk, flags=0, mode=pk.DELTA_MATCHING):
    """The same kernels on sequence b alone (B = 1, its own lengths)."""
    w1 = synth.with_shape(w, B=1, N=nq, Nk=0 if w.causal else nk)
    q, do = (to_dev(d[n][b:b + 1, :nq], w.dtype) for n in ("q", "do"))
    k, v = (to_dev(d[n][b:b + 1, :nk], w.dtype) for n in ("k", "v"))
    mq, mk, mv, mdo = (pk.attn_fp8_quantize(t) for t in (q, k, v, do))
    p = pk.Problem(1, nq, w.Hq, w.Hkv, w.Dqk, w.Dv, float(np.float32(w.tau)), causal=int(w.causal), seqlen_kv=w1.Nk,
                   flags=flags)
    o, lse = pk.attn_fp8_fwd(p, mq, mk, mv)
    delta = pk.attn_fp8_delta(p, mode, mq, mk, mv, mdo, lse, do, o)
    dq, _, _, _ = pk.attn_fp8_bwd(p, mode, mq, mk, mv, mdo, lse, do, o, grad_dtype=torch.float32)
    torch.cuda.synchronize()
    f = lambda t: t.float().cpu().numpy().astype(np.float64)
    return dict(O=f(o), LSE=f(lse), delta=f(delta), dQ=f(dq))


@pytest.mark.parametrize("name,kw,lq,lk", CASES, ids=_ids())
def test_varlen_parity(name, kw, lq, lk):
    _check(name, kw, lq, lk, 0)


def test_varlen_isolate3():
    """Three isolated score channels (ATTN_FP8_FLAG_ISOLATE3) on a padded
    batch: the channels are chosen per (sequence, KV head) from maxima that
    the NaN padding does not reach, so every sequence meets the same checks
    as in the default mode, against the oracle and against the sequence run
    alone with the same flag."""
    name, kw, lq, lk = CASES[0]
    _check(name, kw, lq, lk, pk.FLAG_ISOLATE3)


@pytest.mark.parametrize("variant", ["pbwd_block_scaled", "compensated"])
@pytest.mark.parametrize("case", [0, 3], ids=["causal", "unmasked"])
def test_varlen_numerics_variants(variant, case):
    """The block-scaled backward probability operand (against the oracle's
    variant) and the compensated correction on padded batches, causal and
    without the mask: the same per-sequence checks."""
    name, kw, lq, lk = CASES[case]
    if variant == "pbwd_block_scaled":
        _check(name, kw, lq, lk, pk.FLAG_PBWD_BLOCK_SCALED, oracle_flags=orc.MX_PBWD)
    else:
        _check(name, kw, lq, lk, 0, mode=pk.DELTA_MATCHING_COMPENSATED)


def _check(name, kw, lq, lk, flags, mode=pk.DELTA_MATCHING, oracle_flags=0):
    w = synth.with_shape(synth.WORKLOADS[name], **kw)
    say(f"varlen parity {w} lens_q={lq} lens_kv={lk} flags={flags} mode={mode}")
    d = synth.generate(w, seed=11)
    g = _run(w, d, lq, lk, mode=mode, flags=flags)
    for b, (nq, nk) in enumerate(_eff(lq, lk, w.causal)):
        # padding rows untouched
        assert np.all(g["O"][b, nq:] == SENTINEL) and np.all(g["LSE"][b, :, nq:] == SENTINEL), b
        assert np.all(g["delta"][b, :, nq:] == SENTINEL) and np.all(g["dQ"][b, nq:] == SENTINEL), b
        assert np.all(g["dK"][b, nk:] == SENTINEL) and np.all(g["dV"][b, nk:] == SENTINEL), b
        if nq == 0:
            # keys without queries: zero gradients
            assert np.all(g["dK"][b, :nk] == 0.0) and np.all(g["dV"][b, :nk] == 0.0), b
            continue
        ws = synth.with_shape(w, B=1, N=nq, Nk=0 if w.causal else nk)
        ds = {n: d[n][b:b + 1, :(nq if n in ("q", "do") else nk)] for n in ("q", "k", "v", "do")}
        o = run_oracle(ws, ds, flags=oracle_flags) if oracle_flags else run_oracle(ws, ds)
        gs = dict(O=g["O"][b:b + 1, :nq], dQ=g["dQ"][b:b + 1, :nq], dK=g["dK"][b:b + 1, :nk],
                  dV=g["dV"][b:b + 1, :nk])
        errs = {n: rel_err(gs[n], o[n]) for n in gs}
        blk = {n: block_errors(gs[n], o[n]) for n in gs}
        errs["LSE"] = float(np.max(np.abs(g["LSE"][b:b + 1, :, :nq] - o["LSE"])))
        dl = g["delta"][b:b + 1, :, :nq]
        errs["delta"] = rel_err(dl[..., 0] + dl[..., 1], o["delta"])
        rep = invariant_report(g["rowstats"][b:b + 1, :, :nq], min_row=1 if w.causal else 0)
        say(f"  seq {b} ({nq} x {nk})", {n: f"{e:.2e}" for n, e in errs.items()}, "invariant", rep)
        for n in ("O", "dQ", "dK", "dV"):
            assert errs[n] <= REL_TOL, (b, n, errs[n])
        check_blocks(blk)
        assert errs["LSE"] < 1e-3 and errs["delta"] < 1e-3, (b, errs)
        assert rep["violations"] == 0, (b, rep)
        # the query-major results equal those of the sequence run alone
        a = _alone(w, d, b, nq, nk, flags, mode)
        assert np.array_equal(g["O"][b:b + 1, :nq], a["O"]), b
        assert np.array_equal(g["LSE"][b:b + 1, :, :nq], a["LSE"]), b
        assert np.array_equal(g["delta"][b:b + 1, :, :nq], a["delta"]), b
        assert np.array_equal(g["dQ"][b:b + 1, :nq], a["dQ"]), b


def test_varlen_saved_output_correction():
    """The saved-output corrections skip the padding rows as well: the stale
    correction on the padded batch equals the same pass on each sequence's
    own rows of the same O and dO, and leaves the padding rows as they were."""
    w = synth.with_shape(synth.WORKLOADS["gqa_d128_8k"], B=3, N=192, Hq=4, Hkv=2, causal=False, Nk=128)
    lq, lk = [192, 64, 96], [128, 0, 32]
    d = synth.generate(w, seed=13)
    q, do = (to_dev(_padded(d[n], lq), w.dtype) for n in ("q", "do"))
    k, v = (to_dev(_padded(d[n], lk), w.dtype) for n in ("k", "v"))
    mq, mk, mv, mdo = (pk.attn_fp8_quantize(t) for t in (q, k, v, do))
    p = pk.Problem(w.B, w.N, w.Hq, w.Hkv, w.Dqk, w.Dv, float(np.float32(w.tau)), causal=0, seqlen_kv=w.Nk,
                   seqlens_q=torch.tensor(lq, dtype=torch.int32, device="cuda"),
                   seqlens_kv=torch.tensor(lk, dtype=torch.int32, device="cuda"))
    o, lse = pk.attn_fp8_fwd(p, mq, mk, mv, o=_full((w.B, w.N, w.Hq, w.Dv), torch.bfloat16))
    for mode in (pk.DELTA_STALE_ROWSUM, pk.DELTA_CONSISTENT_DO):
        delta = pk.attn_fp8_delta(p, mode, mq, mk, mv, mdo, lse, do, o,
                                  delta=_full((w.B, w.Hq, w.N, 2), torch.float32))
        torch.cuda.synchronize()
        got = delta.cpu().numpy()
        for b, (nq, nk) in enumerate(_eff(lq, lk, False)):
            assert np.all(got[b, :, nq:] == SENTINEL), (mode, b)
            if nq == 0:
                continue
            p1 = pk.Problem(1, nq, w.Hq, w.Hkv, w.Dqk, w.Dv, float(np.float32(w.tau)), causal=0, seqlen_kv=nk)
            m1 = pk.attn_fp8_quantize(do[b:b + 1, :nq].contiguous())
            ref = pk.attn_fp8_delta(p1, mode, None, None, None, m1, None, do[b:b + 1, :nq].contiguous(),
                                    o[b:b + 1, :nq].contiguous())
            torch.cuda.synchronize()
            assert np.array_equal(got[b:b + 1, :, :nq], ref.cpu().numpy()), (mode, b)
