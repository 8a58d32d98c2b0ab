"""GPU forward, correction and backward against the same-quantization oracle
(relative Frobenius error <= 2e-2 per tensor and for the median 32-row
block, <= 2^-3 for every block: one E4M3 step of a dominant element), the
zero-row-sum invariant on the GPU's own pre-cast dS, and the structural
identities of App. C.1 / App. C.4.1.  Every backward case runs the plain
kernel (the one the benchmark times) against the oracle and the
instrumented kernel, which must return bitwise the same gradients."""
import numpy as np
import pytest
import torch

import oracle as orc
import paper_2609_37852_amd as pk
from paper_2609_37852_amd import synth
from _helpers import (REL_TOL, block_errors, check_blocks, check_row_stat_fields, invariant_report, rel_err, run_gpu,
                      run_oracle, say)

pytestmark = pytest.mark.gpu

CASES = [
    # name, workload overrides (several tiles, ragged tails vs the 64/128 tiles)
    ("tiny_mha_128", {}),
    ("tiny_mha_128", dict(N=96, B=2)),
    ("gqa_d128_8k", dict(B=1, N=320, Hq=4, Hkv=1)),
    ("gqa_d256_8k_qknorm", dict(B=1, N=160, Hq=2, Hkv=1)),
    ("mla_d192_4k", dict(B=1, N=192, Hq=2, Hkv=2)),
    ("gqa_d128_64k_nope", dict(B=1, N=256, Hq=4, Hkv=2)),
]

# Share of rows the invariant must grade (reading R12).  With the x20
# outlier channel in Q and K the score of that channel alone has a standard
# deviation near 35 (400 tau), so most rows are near one-hot: their dS is
# below FP32 resolution of their largest P dP and they fall under the cond
# filter by construction (about 60 % of rows at N = 320).  Elsewhere at least
# half the rows are graded.
MIN_GRADED = {"outlier": 0.25}


def _workload(name, kw):
    w = synth.WORKLOADS[name]
    return synth.with_shape(w, **kw) if kw else w


def _compare(g, o, kinds=("O", "dQ", "dK", "dV")):
    errs = {k: rel_err(g[k], o[k]) for k in kinds}
    blk = {k: block_errors(g[k], o[k]) for k in kinds}
    return errs, blk


@pytest.mark.parametrize("name,kw", CASES, ids=[f"{n}-{'-'.join(f'{k}{v}' for k, v in kw.items()) or 'full'}"
                                                 for n, kw in CASES])
@pytest.mark.parametrize("mode", [pk.DELTA_MATCHING, pk.DELTA_STALE_ROWSUM, pk.DELTA_CONSISTENT_DO],
                         ids=["matching", "stale", "consistent"])
def test_parity(name, kw, mode):
    w = _workload(name, kw)
    say(f"parity {w} mode={mode}")
    d = synth.generate(w, seed=1)
    g = run_gpu(w, d, mode=mode)
    o = run_oracle(w, d, mode=mode)
    # input codes are bit-exact (same quantizer)
    for n in ("Q", "K", "V", "dO"):
        for f in ("code_row", "scale_row", "code_col", "scale_col"):
            assert np.array_equal(g["mx"][n][f], o["quant"][n][f]), (n, f)
    errs_own = None
    if mode != pk.DELTA_MATCHING:
        # The saved-output corrections read the bf16-rounded O.  The GPU's and
        # the oracle's O can round to neighbouring bf16 values (FP32 vs FP64
        # before the rounding), which moves delta by ~1e-3 relative, and on
        # near-one-hot rows dP - delta is only a few percent of delta, so the
        # end-to-end gradients differ by several percent there (reported).
        # The correction is graded by itself below; the backward is graded
        # given the oracle's own correction, injected as an FP32 (hi, lo) pair.
        errs_own = {k: rel_err(g[k], o[k]) for k in ("dQ", "dK")}
        hi = o["delta"].astype(np.float32)
        lo = (o["delta"] - hi.astype(np.float64)).astype(np.float32)
        inj = torch.from_numpy(np.stack([hi, lo], axis=-1)).cuda()
        gi = run_gpu(w, d, mode=mode, delta_in=inj)
        for k in ("dQ", "dK", "dV"):
            gi[k + "_own"] = g[k]
        gi["delta"], gi["rowstats"] = g["delta"], g["rowstats"]
        g = gi
    errs, blk = _compare(g, o)
    errs["LSE"] = float(np.max(np.abs(g["LSE"] - o["LSE"])))
    errs["delta"] = rel_err(g["delta"][..., 0] + g["delta"][..., 1], o["delta"])
    say("  errors", {k: f"{v:.2e}" for k, v in errs.items()})
    if errs_own is not None:
        say("  end to end, with the GPU's own correction", {k: f"{v:.2e}" for k, v in errs_own.items()})
    say("  32-row blocks (worst, at, median)", {k: (f"{v[0]:.2e}", v[1], f"{v[2]:.1e}") for k, v in blk.items()})
    for k in ("O", "dQ", "dK", "dV"):
        assert errs[k] <= REL_TOL, (k, errs[k])
    check_blocks(blk)
    assert errs["LSE"] < 1e-3
    # the saved-output corrections read the bf16-rounded O, whose rounding flips move them
    assert errs["delta"] < (1e-3 if mode == pk.DELTA_MATCHING else 1e-2)
    fields = check_row_stat_fields(g["rowstats"], o["rowstats"])
    say("  row-stat fields vs oracle (median rel. diff)", fields)
    assert fields["max_pdp"] < 1e-3 and fields["sum_pcast"] < 1e-3, fields
    if mode == pk.DELTA_MATCHING:
        rep = invariant_report(g["rowstats"])
        say("  invariant", rep)
        assert rep["violations"] == 0, rep
        need = MIN_GRADED.get(w.transform, 0.5)
        assert rep["share"] >= need, (rep["share"], need)


def test_injected_lse_reaches_the_probability_clamp():
    """Reading R6: the backward clamps the recomputed P at 1.  With an LSE
    0.5 below the forward's, P reaches e^0.5 before the clamp; the GPU and
    the oracle (given the same shift of its own LSE) clamp alike, so the
    correction, gradients and sum_j P'_ij still agree."""
    w = _workload("tiny_mha_128", dict(N=160))
    d = synth.generate(w, seed=9)
    g = run_gpu(w, d, lse_shift=-0.5)
    base = run_oracle(w, d)
    o = run_oracle(w, d, lse_in=base["LSE"] - 0.5)
    errs, blk = _compare(g, o, ("dQ", "dK", "dV"))
    errs["delta"] = rel_err(g["delta"][..., 0] + g["delta"][..., 1], o["delta"])
    fields = check_row_stat_fields(g["rowstats"], o["rowstats"])
    say("  errors", errs, "fields", fields)
    # the shift inflates every row's probabilities by e^0.5 (sum_j P'_ij
    # above 1); rows with a dominant key (row 0 at least) reach the clamp
    sp = o["rowstats"][..., orc.ST_SUM_PCAST]
    assert np.max(sp) > 1.0
    for k in ("dQ", "dK", "dV"):
        assert errs[k] <= REL_TOL, (k, errs[k])
    check_blocks(blk)
    assert errs["delta"] < 1e-3 and fields["sum_pcast"] < 1e-3


@pytest.mark.xfail(strict=True, reason="one isolated score channel: with three x20 channels the other two stay in "
                                       "the MFMA's grouped accumulation (measured O 2.1e-2, LSE 6.1e-2)")
def test_three_outlier_channels():
    """Robustness of the isolated score channel: three x20 channels in Q and K
    (the kernels take one channel out of the MFMA; the other two stay in its
    grouped accumulation).  ATTN_FP8_FLAG_ISOLATE3 (next test) covers it."""
    _three_outliers(0)


def _three_outliers(flags):
    w = _workload("gqa_d128_8k", dict(B=1, N=320, Hq=4, Hkv=1, transform="outlier3"))
    d = synth.generate(w, seed=1)
    g = run_gpu(w, d, flags=flags)
    o = run_oracle(w, d)
    errs, blk = _compare(g, o)
    errs["LSE"] = float(np.max(np.abs(g["LSE"] - o["LSE"])))
    say("  errors", {k: f"{v:.2e}" for k, v in errs.items()})
    say("  32-row blocks (worst, at, median)", {k: (f"{v[0]:.2e}", v[1], f"{v[2]:.1e}") for k, v in blk.items()})
    rep = invariant_report(g["rowstats"])
    say("  invariant", rep)
    for k in ("O", "dQ", "dK", "dV"):
        assert errs[k] <= REL_TOL, (k, errs[k])
    check_blocks(blk)
    assert rep["violations"] == 0


def test_three_outlier_channels_isolated():
    """The same three x20 channels with ATTN_FP8_FLAG_ISOLATE3: all three are
    taken out of the MFMA and their products added exactly."""
    _three_outliers(pk.FLAG_ISOLATE3)


@pytest.mark.parametrize("name,kw", [("gqa_d128_8k", dict(B=1, N=256, Hq=4, Hkv=2)),
                                     ("gqa_d256_8k_qknorm", dict(B=1, N=160, Hq=2, Hkv=1)),
                                     ("mla_d192_4k", dict(B=1, N=128, Hq=2, Hkv=2, causal=False, Nk=192)),
                                     ("tiny_mha_128", dict(B=2, N=96))])
def test_isolate3_parity(name, kw):
    """Three isolated channels on the other recipes and head dims (one or no
    outlier channel): parity and the invariant as in the default mode."""
    w = _workload(name, kw)
    d = synth.generate(w, seed=2)
    g = run_gpu(w, d, flags=pk.FLAG_ISOLATE3)
    o = run_oracle(w, d)
    errs, blk = _compare(g, o)
    errs["LSE"] = float(np.max(np.abs(g["LSE"] - o["LSE"])))
    say("  errors", {k: f"{v:.2e}" for k, v in errs.items()})
    rep = invariant_report(g["rowstats"], min_row=1 if w.causal else 0)
    say("  invariant", rep)
    for k in ("O", "dQ", "dK", "dV"):
        assert errs[k] <= REL_TOL, (k, errs[k])
    check_blocks(blk)
    assert errs["LSE"] < 1e-3 and rep["violations"] == 0


def test_key_block_order_with_partial_cohort():
    """The backward grid visits the key blocks in cohorts of pairs sized by
    the number of workgroups of one KV head that run at once (compute units
    / (B Hkv)); with 64 KV heads that is 4 on a 256-CU GPU, so 10 key blocks
    (5 pairs) make one full cohort and a partial one.  Every key block of a
    head must be visited exactly once: two of the 64 heads are checked
    against the oracle (each head's key blocks use the same grid order)."""
    w = _workload("tiny_mha_128", dict(B=1, N=1280, Hq=64, Hkv=64))
    d = synth.generate(w, seed=3)
    g = run_gpu(w, d, rowstats=False)
    heads = [0, 63]
    ds = {n: np.ascontiguousarray(d[n][:, :, heads]) for n in ("q", "k", "v", "do")}
    o = run_oracle(synth.with_shape(w, Hq=2, Hkv=2), ds)
    errs = {k: rel_err(g[k][:, :, heads], o[k]) for k in ("O", "dQ", "dK", "dV")}
    say("  errors", {k: f"{v:.2e}" for k, v in errs.items()})
    for k, e in errs.items():
        assert e <= REL_TOL, (k, e)


def test_isolated_channel_on_outlier_workload():
    """The outlier-channel workload: with the isolated score channel the
    output errors fall far below the bound; without it the MFMA's grouped
    accumulation costs an order of magnitude (reported, not asserted)."""
    w = _workload("gqa_d128_8k", dict(B=1, N=512, Hq=4, Hkv=1))
    d = synth.generate(w, seed=2)
    o = run_oracle(w, d)
    res = {}
    for iso in (True, False):
        g = run_gpu(w, d, isolate=iso, rowstats=False)
        res[iso] = {k: rel_err(g[k], o[k]) for k in ("O", "dQ", "dK", "dV")}
        res[iso]["LSE"] = float(np.max(np.abs(g["LSE"] - o["LSE"])))
    say("  isolated", res[True], "\n  plain   ", res[False])
    for k in ("O", "dQ", "dK", "dV"):
        assert res[True][k] <= REL_TOL / 4, (k, res[True][k])
    assert res[True]["LSE"] < 1e-3


def test_delta_mode_changes_only_dq_dk():
    """App. C.4.1: changing only the correction leaves O and dV bitwise
    unchanged and changes dQ and dK."""
    w = _workload("gqa_d128_8k", dict(B=1, N=256, Hq=2, Hkv=1))
    d = synth.generate(w, seed=3)
    a = run_gpu(w, d, mode=pk.DELTA_MATCHING)
    b = run_gpu(w, d, mode=pk.DELTA_STALE_ROWSUM)
    assert np.array_equal(a["O"], b["O"]) and np.array_equal(a["dV"], b["dV"])
    assert not np.array_equal(a["dQ"], b["dQ"]) and not np.array_equal(a["dK"], b["dK"])


def test_stale_residual_is_large_and_matching_small():
    """Pre-cast row sums: the stale correction leaves the largest residual,
    consistent dO (no gradient-quantization term, Sec. 3.4) a smaller but
    still large one, the matched correction almost none."""
    w = _workload("tiny_mha_128", {})
    d = synth.generate(w, seed=0)
    res = {}
    for mode in (pk.DELTA_MATCHING, pk.DELTA_STALE_ROWSUM, pk.DELTA_CONSISTENT_DO):
        g = run_gpu(w, d, mode=mode)
        rs = g["rowstats"]
        live = rs[..., 1] > 0
        res[mode] = np.median(np.abs(rs[..., 0][live]) / rs[..., 1][live])
    say("  median r_pre", res)
    assert res[pk.DELTA_STALE_ROWSUM] > 1e-4
    assert res[pk.DELTA_STALE_ROWSUM] > 100 * res[pk.DELTA_MATCHING]
    assert 100 * res[pk.DELTA_MATCHING] < res[pk.DELTA_CONSISTENT_DO] < res[pk.DELTA_STALE_ROWSUM]


def test_delta_injection_affine():
    """App. C.1 correction-pass consistency: backward row sums with injected
    corrections 0 and 1 give delta* = R(0) / (R(0) - R(1)) matching the pass
    (on the rows graded for the invariant: cond >= 2^-5)."""
    w = _workload("tiny_mha_128", dict(N=192, Hq=2, Hkv=1))
    d = synth.generate(w, seed=4)
    base = run_gpu(w, d)
    z = torch.zeros((w.B, w.Hq, w.N, 2), dtype=torch.float32, device="cuda")
    r0 = run_gpu(w, d, delta_in=z)
    one = z.clone()
    one[..., 0] = 1.0
    r1 = run_gpu(w, d, delta_in=one)
    R0, R1 = r0["rowstats"][..., 0], r1["rowstats"][..., 0]
    SP = R0 - R1                                    # = sum_j P_ij of the backward's own P
    st = base["rowstats"]
    cond = st[..., pk.RS_MAXABS_DS] / np.maximum(st[..., pk.RS_MAX_PDP], 1e-300)
    ok = (np.abs(SP) > 0.5) & (cond >= 2.0 ** -5)
    dstar = R0[ok] / SP[ok]
    dl = (base["delta"][..., 0] + base["delta"][..., 1])[ok]
    e = np.abs(dstar - dl) * np.abs(SP[ok]) / np.maximum(st[..., 1][ok], 1e-30)
    say("  rows", int(ok.sum()), "median e", float(np.median(e)), "max", float(e.max()))
    assert ok.sum() > 0.5 * ok.size
    assert np.median(e) < 1e-6 and e.max() < 1e-4


def test_determinism():
    w = _workload("gqa_d128_8k", dict(B=1, N=256, Hq=4, Hkv=2))
    d = synth.generate(w, seed=5)
    a = run_gpu(w, d, rowstats=False)
    b = run_gpu(w, d, rowstats=False)
    # every output is written once, in a fixed order (no atomics)
    for k in ("O", "LSE", "delta", "dQ", "dK", "dV"):
        assert np.array_equal(a[k], b[k]), k


def test_bf16_gradients_and_empty():
    w = _workload("tiny_mha_128", dict(N=64))
    d = synth.generate(w, seed=6)
    g = run_gpu(w, d, grad_dtype=torch.bfloat16)
    o = run_oracle(w, d, grad_round=orc.ROUND_BF16)
    for k in ("dQ", "dK", "dV"):
        assert rel_err(g[k], o[k]) <= REL_TOL
    p = pk.Problem(1, 0, 2, 2, 64, 64, 0.125)
    mx = pk.MX.empty(1, 0, 2, 64, "cuda")
    o_, lse = pk.attn_fp8_fwd(p, mx, mx, mx)
    assert o_.numel() == 0 and lse.numel() == 0
