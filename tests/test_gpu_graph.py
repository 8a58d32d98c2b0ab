"""The hot path captured once in a HIP graph and replayed: quantize, forward,
matched correction and backward enqueue kernels only (buffer clears are fill
kernels, not memset nodes), so every replay must reproduce the eager results
bit for bit.  Replays alternate with eager work on other inputs, and each
replay is checked (a replay that read stale state, or a captured node that
misbehaves after the first replay, would show).  Sequence lengths are read
from device memory when the kernels run, so one captured graph serves
every set of lengths written into its buffer."""
import numpy as np
import pytest
import torch

import paper_2609_37852_amd as pk
from paper_2609_37852_amd import synth
from _helpers import say, to_dev

pytestmark = pytest.mark.gpu


def _path(p, q, k, v, do, ws):
    mq, mk, mv, mdo = (pk.attn_fp8_quantize(t) for t in (q, k, v, do))
    o, lse = pk.attn_fp8_fwd(p, mq, mk, mv)
    delta = pk.attn_fp8_delta(p, pk.DELTA_MATCHING, mq, mk, mv, mdo, lse, do, o)
    dq, dk, dv, _ = pk.attn_fp8_bwd(p, pk.DELTA_MATCHING, mq, mk, mv, mdo, lse, do, o, delta_in=delta, workspace=ws)
    return o, lse, delta, dq, dk, dv


def _bits(ts):
    return [t.view(torch.int16 if t.dtype == torch.bfloat16 else torch.int32).clone() for t in ts]


@pytest.mark.parametrize("name,kw", [("gqa_d128_8k", dict(B=1, N=512, Hq=4, Hkv=2)),
                                     ("tiny_mha_128", dict(B=2, N=160, causal=False, Nk=96))])
def test_graph_replay_matches_eager(name, kw):
    w = synth.with_shape(synth.WORKLOADS[name], **kw)
    say(f"graph replay {w}")
    d = synth.generate(w, seed=31)
    q, k, v, do = (to_dev(d[n], w.dtype) for n in ("q", "k", "v", "do"))
    p = pk.Problem(w.B, w.N, w.Hq, w.Hkv, w.Dqk, w.Dv, float(np.float32(w.tau)), causal=int(w.causal),
                   seqlen_kv=w.Nk)
    ws = torch.empty(pk.attn_fp8_bwd_workspace_size(p), dtype=torch.uint8, device="cuda")
    eager = _bits(_path(p, q, k, v, do, ws))
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        outs = _path(p, q, k, v, do, ws)
    d2 = synth.generate(w, seed=32)
    other = [to_dev(d2[n], w.dtype) for n in ("q", "k", "v", "do")]
    for rep in range(4):
        g.replay()
        torch.cuda.synchronize()
        got = _bits(outs)
        for name_, a, b in zip(("O", "LSE", "delta", "dQ", "dK", "dV"), got, eager):
            assert torch.equal(a, b), f"replay {rep}: {name_} differs from the eager run"
        # eager work in between, on other inputs and the same workspace
        _path(p, *other, ws)
        torch.cuda.synchronize()
    say("  4 replays bitwise equal to the eager run")


def test_graph_replay_with_new_lengths():
    """Sequences of their own lengths read from device memory at run time: a
    graph captured with one set of lengths replays with lengths written into
    the same buffer afterwards, and each replay equals the eager run with
    those lengths on every row inside the sequences."""
    w = synth.with_shape(synth.WORKLOADS["gqa_d128_8k"], B=3, N=256, Hq=4, Hkv=2)
    d = synth.generate(w, seed=33)
    q, k, v, do = (to_dev(d[n], w.dtype) for n in ("q", "k", "v", "do"))
    lens = torch.tensor([256, 96, 160], dtype=torch.int32, device="cuda")
    p = pk.Problem(w.B, w.N, w.Hq, w.Hkv, w.Dqk, w.Dv, float(np.float32(w.tau)), causal=1, seqlens_q=lens)
    ws = torch.empty(pk.attn_fp8_bwd_workspace_size(p), dtype=torch.uint8, device="cuda")
    _path(p, q, k, v, do, ws)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        outs = _path(p, q, k, v, do, ws)
    for new in ([64, 256, 0], [160, 32, 224], [256, 96, 160]):
        lens.copy_(torch.tensor(new, dtype=torch.int32))
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        got = [t.clone() for t in outs]
        ref = _path(p, q, k, v, do, torch.empty_like(ws))
        torch.cuda.synchronize()
        for name, a, r in zip(("O", "LSE", "delta", "dQ", "dK", "dV"), got, ref):
            for b, L in enumerate(new):
                if name in ("LSE", "delta"):
                    sa, sr = a[b, :, :L], r[b, :, :L]
                else:
                    sa, sr = a[b, :L], r[b, :L]
                assert torch.equal(sa, sr), (new, name, b)
    say("  replays with three sets of lengths equal the eager runs")
