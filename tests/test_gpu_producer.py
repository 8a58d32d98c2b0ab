"""The input producer (App. B.6.1; readings R13, R16, R17) on the GPU: the
fused QK normalization and rotary embedding (normalized and rotated values
rounded to BF16), FP32 query prescale and per-(channel, KV head) key
centering before quantization.  Codes, scales and the key mean are bit-exact
with the oracle's producer and quantizer; the whole path on the transformed
operands (queries prescaled by tau, softmax scale 1, keys centred;
straight-through key gradient) agrees with the oracle within the parity
bounds and keeps the invariant."""
import math

import numpy as np
import pytest
import torch

import oracle as orc
import paper_2609_37852_amd as pk
from paper_2609_37852_amd import synth
from _helpers import REL_TOL, block_errors, bwd_plain_and_stats, check_blocks, invariant_report, np64, rel_err, say

pytestmark = pytest.mark.gpu


def _keys(B, N, H, D, seed, dtype):
    rng = np.random.default_rng(seed)
    # a per-channel bias, as trained keys carry, so that the mean matters
    x = rng.standard_normal((B, N, H, D)).astype(np.float32) + rng.uniform(-2, 2, (1, 1, H, D)).astype(np.float32)
    return synth.round_bf16(x) if dtype == "bf16" else x


@pytest.mark.parametrize("D", [64, 128, 192, 256])
@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("prescale,center", [(1 / math.sqrt(128), False), (1.0, True), (0.3, True)])
def test_producer_codes_bit_exact(D, dtype, prescale, center):
    B, N, H = 2, 96, 3
    x = _keys(B, N, H, D, seed=D, dtype=dtype)
    # a strided view: every other head of a wider tensor
    wide = np.zeros((B, N, 2 * H, D), np.float32)
    wide[:, :, ::2] = x
    t = torch.from_numpy(wide).cuda()
    t = (t.to(torch.bfloat16) if dtype == "bf16" else t)[:, :, ::2]
    g, mean = pk.attn_fp8_quantize_producer(t, prescale, center)
    torch.cuda.synchronize()
    y, m = orc.producer(x, prescale, center)
    ref = orc.quantize(y)
    for f in ("code_row", "scale_row", "code_col", "scale_col"):
        assert np.array_equal(getattr(g, f).cpu().numpy(), ref[f]), f
    if center:
        assert np.array_equal(mean.cpu().numpy().astype(np.float64), m)
    # channel maxima of the transformed values
    assert np.array_equal(g.channel_amax.cpu().numpy(), np.abs(y).max(axis=1).astype(np.float32))


def test_producer_path_matches_oracle():
    """Queries prescaled by tau (softmax scale 1), keys centred, outlier
    recipe (C2) at a reduced size: forward, matched correction and backward
    against the oracle run on the oracle producer's operands."""
    w = synth.with_shape(synth.WORKLOADS["gqa_d128_8k"], B=1, N=384, Hq=4, Hkv=2)
    d = synth.generate(w, seed=4)
    tau = float(np.float32(w.tau))
    k = (d["k"] + np.float32(0.7)).astype(np.float32)           # keys with a common offset
    k = synth.round_bf16(k)
    qt, kt, vt, dot = (torch.from_numpy(a).to(torch.bfloat16).cuda() for a in (d["q"], k, d["v"], d["do"]))
    mq, _ = pk.attn_fp8_quantize_producer(qt, tau, False)
    mk, kmean = pk.attn_fp8_quantize_producer(kt, 1.0, True)
    mv, mdo = pk.attn_fp8_quantize(vt), pk.attn_fp8_quantize(dot)
    p = pk.Problem(w.B, w.N, w.Hq, w.Hkv, w.Dqk, w.Dv, 1.0)
    o, lse = pk.attn_fp8_fwd(p, mq, mk, mv)
    dq, dk, dv, rs = bwd_plain_and_stats(p, pk.DELTA_MATCHING, mq, mk, mv, mdo, lse)
    torch.cuda.synchronize()
    qy, _ = orc.producer(d["q"], tau, False)
    ky, km = orc.producer(k, 1.0, True)
    assert np.array_equal(kmean.cpu().numpy().astype(np.float64), km)
    ref, _ = orc.attention_from_inputs(qy, ky, d["v"], d["do"], 1.0, want_rowstats=True)
    g = dict(O=np64(o), dQ=np64(dq), dK=np64(dk), dV=np64(dv))
    errs = {n: rel_err(g[n], ref[n]) for n in g}
    blk = {n: block_errors(g[n], ref[n]) for n in g}
    errs["LSE"] = float(np.max(np.abs(np64(lse) - ref["LSE"])))
    rep = invariant_report(rs.cpu().numpy())
    say("  errors", {n: f"{e:.2e}" for n, e in errs.items()}, "invariant", rep)
    for n in ("O", "dQ", "dK", "dV"):
        assert errs[n] <= REL_TOL, (n, errs[n])
    check_blocks(blk)
    assert errs["LSE"] < 1e-3 and rep["violations"] == 0


@pytest.mark.parametrize("D,lo,R", [(128, 0, 32), (192, 128, 64), (64, 0, 64), (256, 64, 128)])
@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("prescale,center", [(1 / math.sqrt(128), False), (1.0, True)])
def test_rope_producer_codes_bit_exact(D, lo, R, dtype, prescale, center):
    """The fused rotary producer (reading R16): codes, scales, channel maxima
    and the key mean bit-exact with the oracle's rotary producer and
    quantizer, on a strided input."""
    B, N, H = 2, 96, 3
    x = _keys(B, N, H, D, seed=D + R, dtype=dtype)
    tab = synth.rope_table(N, R, 1e4, pos0=7)
    wide = np.zeros((B, N, 2 * H, D), np.float32)
    wide[:, :, ::2] = x
    t = torch.from_numpy(wide).cuda()
    t = (t.to(torch.bfloat16) if dtype == "bf16" else t)[:, :, ::2]
    g, mean = pk.attn_fp8_quantize_producer(t, prescale, center, rope=torch.from_numpy(tab).cuda(), rope_lo=lo)
    torch.cuda.synchronize()
    y, m = orc.producer_rope(x, tab, lo, R, prescale, center)
    ref = orc.quantize(y)
    for f in ("code_row", "scale_row", "code_col", "scale_col"):
        assert np.array_equal(getattr(g, f).cpu().numpy(), ref[f]), f
    if center:
        assert np.array_equal(mean.cpu().numpy().astype(np.float64), m)
    assert np.array_equal(g.channel_amax.cpu().numpy(), np.abs(y).max(axis=1).astype(np.float32))


def test_rope_producer_path_matches_oracle():
    """MLA-shaped heads (dqk 192, dv 128) with the rotary part on channels
    128..191 applied by the fused producer: queries rotated and prescaled by
    tau (softmax scale 1), keys rotated and centred; the whole path against
    the oracle run on the oracle producer's operands."""
    w = synth.with_shape(synth.WORKLOADS["mla_d192_4k"], B=1, N=256, Hq=2, Hkv=2, transform="none")
    d = synth.generate(w, seed=8)
    tau = float(np.float32(w.tau))
    tab = synth.rope_table(w.N, 64, 1e4)
    qt, kt, vt, dot = (torch.from_numpy(a).to(torch.bfloat16).cuda() for a in (d["q"], d["k"], d["v"], d["do"]))
    tt = torch.from_numpy(tab).cuda()
    mq, _ = pk.attn_fp8_quantize_producer(qt, tau, False, rope=tt, rope_lo=128)
    mk, _ = pk.attn_fp8_quantize_producer(kt, 1.0, True, rope=tt, rope_lo=128)
    mv, mdo = pk.attn_fp8_quantize(vt), pk.attn_fp8_quantize(dot)
    p = pk.Problem(w.B, w.N, w.Hq, w.Hkv, w.Dqk, w.Dv, 1.0)
    o, lse = pk.attn_fp8_fwd(p, mq, mk, mv)
    dq, dk, dv, rs = bwd_plain_and_stats(p, pk.DELTA_MATCHING, mq, mk, mv, mdo, lse)
    torch.cuda.synchronize()
    qy, _ = orc.producer_rope(d["q"], tab, 128, 64, tau, False)
    ky, _ = orc.producer_rope(d["k"], tab, 128, 64, 1.0, True)
    ref, _ = orc.attention_from_inputs(qy, ky, d["v"], d["do"], 1.0, want_rowstats=True)
    g = dict(O=np64(o), dQ=np64(dq), dK=np64(dk), dV=np64(dv))
    errs = {n: rel_err(g[n], ref[n]) for n in g}
    blk = {n: block_errors(g[n], ref[n]) for n in g}
    rep = invariant_report(rs.cpu().numpy())
    say("  errors", {n: f"{e:.2e}" for n, e in errs.items()}, "invariant", rep)
    for n in ("O", "dQ", "dK", "dV"):
        assert errs[n] <= REL_TOL, (n, errs[n])
    check_blocks(blk)
    assert rep["violations"] == 0


@pytest.mark.parametrize("D,lo,R", [(64, 0, 0), (128, 0, 32), (192, 128, 64), (256, 64, 128)])
@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("prescale,center", [(1.0, False), (1 / math.sqrt(128), False), (1.0, True)])
def test_qknorm_producer_codes_bit_exact(D, lo, R, dtype, prescale, center):
    """The fused QK normalization (reading R17) before the rotary embedding,
    prescale and centring: codes, scales, channel maxima and the key mean
    bit-exact with the oracle's producer, on a strided input whose rows span
    several orders of magnitude (the row scale must not depend on it)."""
    B, N, H = 2, 96, 3
    x = _keys(B, N, H, D, seed=D + R + 1, dtype=dtype)
    mag = np.exp2(np.random.default_rng(D).integers(-6, 7, (B, N, H, 1))).astype(np.float32)
    x = (x * mag).astype(np.float32)
    gain = (1.0 + 0.25 * np.random.default_rng(R).standard_normal(D)).astype(np.float32)
    tab = synth.rope_table(N, R, 1e4, pos0=3) if R else None
    wide = np.zeros((B, N, 2 * H, D), np.float32)
    wide[:, :, ::2] = x
    t = torch.from_numpy(wide).cuda()
    t = (t.to(torch.bfloat16) if dtype == "bf16" else t)[:, :, ::2]
    g, mean = pk.attn_fp8_quantize_producer(t, prescale, center, rope=torch.from_numpy(tab).cuda() if R else None,
                                            rope_lo=lo, rms_gain=torch.from_numpy(gain).cuda(), rms_eps=1e-6)
    torch.cuda.synchronize()
    y, m = orc.producer_ext(x, gain=gain, eps=1e-6, rope=tab, lo=lo, R=R, prescale=prescale, center=center)
    ref = orc.quantize(y)
    for f in ("code_row", "scale_row", "code_col", "scale_col"):
        assert np.array_equal(getattr(g, f).cpu().numpy(), ref[f]), f
    if center:
        assert np.array_equal(mean.cpu().numpy().astype(np.float64), m)
    assert np.array_equal(g.channel_amax.cpu().numpy(), np.abs(y).max(axis=1).astype(np.float32))


def test_qknorm_producer_path_matches_oracle():
    """QK-normalized (gain per channel), rotated queries and keys at d 128:
    queries prescaled by tau (softmax scale 1), keys centred; the whole path
    against the oracle run on the oracle producer's operands."""
    w = synth.with_shape(synth.WORKLOADS["gqa_d128_8k"], B=1, N=384, Hq=4, Hkv=2, transform="none")
    d = synth.generate(w, seed=12)
    tau = float(np.float32(w.tau))
    tab = synth.rope_table(w.N, 64, 1e4)
    rng = np.random.default_rng(5)
    gq = (1.0 + 0.3 * rng.standard_normal(w.Dqk)).astype(np.float32)
    gk = (1.0 + 0.3 * rng.standard_normal(w.Dqk)).astype(np.float32)
    qt, kt, vt, dot = (torch.from_numpy(a).to(torch.bfloat16).cuda() for a in (d["q"], d["k"], d["v"], d["do"]))
    tt = torch.from_numpy(tab).cuda()
    mq, _ = pk.attn_fp8_quantize_producer(qt, tau, False, rope=tt, rope_lo=0, rms_gain=torch.from_numpy(gq).cuda())
    mk, _ = pk.attn_fp8_quantize_producer(kt, 1.0, True, rope=tt, rope_lo=0, rms_gain=torch.from_numpy(gk).cuda())
    mv, mdo = pk.attn_fp8_quantize(vt), pk.attn_fp8_quantize(dot)
    p = pk.Problem(w.B, w.N, w.Hq, w.Hkv, w.Dqk, w.Dv, 1.0)
    o, lse = pk.attn_fp8_fwd(p, mq, mk, mv)
    dq, dk, dv, rs = bwd_plain_and_stats(p, pk.DELTA_MATCHING, mq, mk, mv, mdo, lse)
    torch.cuda.synchronize()
    qy, _ = orc.producer_ext(d["q"], gain=gq, rope=tab, lo=0, R=64, prescale=tau)
    ky, _ = orc.producer_ext(d["k"], gain=gk, rope=tab, lo=0, R=64, center=True)
    ref, _ = orc.attention_from_inputs(qy, ky, d["v"], d["do"], 1.0, want_rowstats=True)
    g = dict(O=np64(o), dQ=np64(dq), dK=np64(dk), dV=np64(dv))
    errs = {n: rel_err(g[n], ref[n]) for n in g}
    blk = {n: block_errors(g[n], ref[n]) for n in g}
    rep = invariant_report(rs.cpu().numpy())
    say("  errors", {n: f"{e:.2e}" for n, e in errs.items()}, "invariant", rep)
    for n in ("O", "dQ", "dK", "dV"):
        assert errs[n] <= REL_TOL, (n, errs[n])
    check_blocks(blk)
    assert rep["violations"] == 0


@pytest.mark.parametrize("D,lo,R", [(128, 0, 0), (192, 128, 64)])
def test_producer_varlen_mean(D, lo, R):
    """A padded batch (NaN in every padding row) with per-sequence lengths
    for the key mean: each sequence's codes, scales, channel maxima and mean
    bit for bit those of the oracle producer run on that sequence's rows
    alone (QK normalization, rotary embedding where given, prescale and
    centering); a sequence without tokens gets a zero mean."""
    B, N, H = 3, 160, 2
    lens = [160, 64, 0]
    x = _keys(B, N, H, D, seed=7, dtype="bf16")
    for b, L in enumerate(lens):
        x[b, L:] = np.nan
    rng = np.random.default_rng(8)
    gain = rng.uniform(0.5, 2.0, D).astype(np.float32)
    rope = synth.rope_table(N, R, 10000.0) if R else None
    g, mean = pk.attn_fp8_quantize_producer(
        torch.from_numpy(x).cuda().to(torch.bfloat16), 0.3, True, rms_gain=torch.from_numpy(gain).cuda(),
        rope=torch.from_numpy(rope).cuda() if R else None, rope_lo=lo,
        seqlens=torch.tensor(lens, dtype=torch.int32, device="cuda"))
    torch.cuda.synchronize()
    got = {f: getattr(g, f).cpu().numpy() for f in ("code_row", "scale_row", "code_col", "scale_col")}
    amax, mean = g.channel_amax.cpu().numpy(), mean.cpu().numpy().astype(np.float64)
    for b, L in enumerate(lens):
        if L == 0:
            assert np.all(mean[b] == 0.0)
            continue
        y, m = orc.producer_ext(x[b:b + 1, :L], gain=gain, eps=1e-6, rope=rope[:L] if R else None, lo=lo, R=R,
                                prescale=0.3, center=True)
        ref = orc.quantize(y)
        assert np.array_equal(mean[b:b + 1], m), b
        assert np.array_equal(got["code_row"][b:b + 1, :, :L], ref["code_row"]), b
        assert np.array_equal(got["scale_row"][b:b + 1, :, :L], ref["scale_row"]), b
        assert np.array_equal(got["code_col"][b:b + 1, :, :, :L], ref["code_col"]), b
        assert np.array_equal(got["scale_col"][b:b + 1, :, :, :L // 32], ref["scale_col"]), b
        assert np.array_equal(amax[b:b + 1], np.abs(y).max(axis=1).astype(np.float32)), b
