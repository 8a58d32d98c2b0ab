"""The workspace-free backward (attn_fp8_bwd_noalloc): through the C ABI,
two calls in a row on one device, the second with a smaller problem, each
against attn_fp8_bwd with a caller workspace (bitwise: the same kernels) and,
with the matched correction, against the oracle (relative Frobenius error
<= 2e-2); padded batches without the mask (sequences of their own lengths)
bitwise equal as well; a problem whose scratch need exceeds the library's
scratch is rejected before any launch."""
import numpy as np
import pytest
import torch

import paper_2609_37852_amd as pk
from paper_2609_37852_amd import synth
from _helpers import REL_TOL, np64, problem, rel_err, run_oracle, say, to_dev

pytestmark = pytest.mark.gpu


def _inputs(w, seed):
    d = synth.generate(w, seed=seed)
    q, k, v, do = (to_dev(d[n], w.dtype) for n in ("q", "k", "v", "do"))
    mq, mk, mv, mdo = (pk.attn_fp8_quantize(t) for t in (q, k, v, do))
    o, lse = pk.attn_fp8_fwd(problem(w), mq, mk, mv)
    return d, (mq, mk, mv, mdo), lse, do, o


@pytest.mark.parametrize("mode", [pk.DELTA_MATCHING, pk.DELTA_STALE_ROWSUM])
def test_noalloc_matches_workspace_backward(mode):
    shapes = [synth.with_shape(synth.WORKLOADS["gqa_d128_8k"], B=1, N=1024, Hq=4, Hkv=2),
              synth.with_shape(synth.WORKLOADS["gqa_d128_8k"], B=1, N=352, Hq=2, Hkv=1)]
    for i, w in enumerate(shapes):
        p = problem(w)
        need = pk.attn_fp8_bwd_workspace_size(p)
        say(f"call {i}: {w.B}x{w.N} Hq {w.Hq} Hkv {w.Hkv}, scratch need {need} of {pk.binding.NOALLOC_SCRATCH_BYTES}")
        d, (mq, mk, mv, mdo), lse, do, o = _inputs(w, seed=10 + i)
        # the correction is computed inside the call (its buffer is in the scratch too)
        na = pk.attn_fp8_bwd_noalloc(p, mode, mq, mk, mv, mdo, lse, do, o, grad_dtype=torch.float32)
        ws = pk.attn_fp8_bwd(p, mode, mq, mk, mv, mdo, lse, do, o, grad_dtype=torch.float32)
        torch.cuda.synchronize()
        for name, a, b in zip(("dQ", "dK", "dV"), na[:3], ws[:3]):
            assert torch.equal(a.view(torch.int32), b.view(torch.int32)), (i, name)
        if mode != pk.DELTA_MATCHING:
            continue   # the stale correction reads the bf16-rounded O: graded with the oracle's delta elsewhere
        ref = run_oracle(w, d, mode=mode)
        errs = {n: rel_err(np64(t), ref[n]) for n, t in zip(("dQ", "dK", "dV"), na[:3])}
        say("  vs oracle", {k: f"{v:.2e}" for k, v in errs.items()})
        for n, e in errs.items():
            assert e <= REL_TOL, (i, n, e)


def test_noalloc_varlen_unmasked():
    """Padded batches without the mask, a key length of their own and
    sequences of their own lengths (one without keys): two calls in a row,
    the second smaller, bitwise equal to the workspace backward on every
    element (padding rows keep the output buffers' contents in both)."""
    cases = [(synth.with_shape(synth.WORKLOADS["gqa_d128_8k"], B=3, N=256, Nk=320, Hq=4, Hkv=2, causal=False),
              [256, 96, 160], [320, 0, 192]),
             (synth.with_shape(synth.WORKLOADS["tiny_mha_128"], B=2, N=96, Nk=64, causal=False), [64, 96], [64, 32])]
    for i, (w, lq, lk) in enumerate(cases):
        d = synth.generate(w, seed=20 + i)
        q, k, v, do = (to_dev(d[n], w.dtype) for n in ("q", "k", "v", "do"))
        mq, mk, mv, mdo = (pk.attn_fp8_quantize(t) for t in (q, k, v, do))
        p = pk.Problem(w.B, w.N, w.Hq, w.Hkv, w.Dqk, w.Dv, float(np.float32(w.tau)), causal=0, seqlen_kv=w.Nk,
                       seqlens_q=torch.tensor(lq, dtype=torch.int32, device="cuda"),
                       seqlens_kv=torch.tensor(lk, dtype=torch.int32, device="cuda"))
        say(f"call {i}: {w} lens_q {lq} lens_kv {lk}, scratch need {pk.attn_fp8_bwd_workspace_size(p)}")
        o, lse = pk.attn_fp8_fwd(p, mq, mk, mv)

        def outs():
            return tuple(torch.full(sh, 7.0, dtype=torch.float32, device="cuda")
                         for sh in ((w.B, w.N, w.Hq, w.Dqk), (w.B, w.nk, w.Hkv, w.Dqk), (w.B, w.nk, w.Hkv, w.Dv)))
        na = pk.attn_fp8_bwd_noalloc(p, pk.DELTA_MATCHING, mq, mk, mv, mdo, lse, do, o, grad_dtype=torch.float32,
                                     out=outs())
        ws = pk.attn_fp8_bwd(p, pk.DELTA_MATCHING, mq, mk, mv, mdo, lse, do, o, grad_dtype=torch.float32, out=outs())
        torch.cuda.synchronize()
        for name, a, b in zip(("dQ", "dK", "dV"), na[:3], ws[:3]):
            assert torch.equal(a.view(torch.int32), b.view(torch.int32)), (i, name)


def test_noalloc_rejects_problems_beyond_its_scratch():
    w = synth.with_shape(synth.WORKLOADS["gqa_d128_8k"], B=1, N=8192, Hq=4, Hkv=1)
    p = problem(w)
    assert pk.attn_fp8_bwd_workspace_size(p) > pk.binding.NOALLOC_SCRATCH_BYTES
    mx = pk.MX.empty(1, 32, 1, 128, "cuda")           # never read: the call fails before any launch
    lse = torch.empty(16, device="cuda")
    with pytest.raises(pk.AttnFp8Error) as ei:
        pk.attn_fp8_bwd_noalloc(p, pk.DELTA_MATCHING, mx, mx, mx, mx, lse, grad_dtype=torch.float32,
                                out=(torch.empty(16, 1, 1, 128, device="cuda"),) * 3)
    assert ei.value.code == -2 and "scratch" in str(ei.value)
