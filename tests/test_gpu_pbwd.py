"""The block-scaled backward probability operand (ATTN_FP8_FLAG_PBWD_BLOCK_
SCALED, reading R15) on the GPU: dV and the row sums of P' against the oracle
with the same variant, everything else bitwise equal to the fixed-scale
kernel (P' only feeds dV); on rows whose small probabilities fall below the
fixed scale's normal range, and on the flat rows of the 64K workload, dV is
closer to dV from uncast probabilities."""
import numpy as np
import pytest
import torch

import oracle as orc
import paper_2609_37852_amd as pk
from paper_2609_37852_amd import synth
from _helpers import REL_TOL, block_errors, check_blocks, np64, rel_err, run_gpu, run_oracle, say, to_dev

pytestmark = pytest.mark.gpu
BLK = pk.FLAG_PBWD_BLOCK_SCALED

CASES = [
    ("tiny_mha_128", dict(N=96, B=2)),
    ("gqa_d128_8k", dict(B=1, N=320, Hq=4, Hkv=1)),
    ("gqa_d256_8k_qknorm", dict(B=1, N=160, Hq=2, Hkv=1)),
    ("mla_d192_4k", dict(B=1, N=192, Hq=2, Hkv=2)),
    ("gqa_d128_64k_nope", dict(B=1, N=256, Nk=352, Hq=4, Hkv=2, causal=False)),
]


@pytest.mark.parametrize("name,kw", CASES, ids=[f"{n}-{'-'.join(f'{k}{v}' for k, v in kw.items())}" for n, kw in CASES])
def test_block_scaled_pbwd_parity(name, kw):
    w = synth.with_shape(synth.WORKLOADS[name], **kw)
    say(f"block-scaled P' {w}")
    d = synth.generate(w, seed=2)
    g = run_gpu(w, d, flags=BLK)
    f = run_gpu(w, d)
    o = run_oracle(w, d, flags=orc.MX_PBWD)
    for k in ("O", "LSE", "delta", "dQ", "dK"):
        assert np.array_equal(g[k], f[k]), k
    err = rel_err(g["dV"], o["dV"])
    blk = block_errors(g["dV"], o["dV"])
    sp_g, sp_o = g["rowstats"][..., pk.RS_SUM_PCAST], o["rowstats"][..., orc.ST_SUM_PCAST]
    live = sp_o > 0
    sp = float(np.median(np.abs(sp_g[live] - sp_o[live]) / sp_o[live]))
    say(f"  dV {err:.2e} blocks {blk[0]:.2e} / {blk[2]:.1e}; sum P' median rel. diff {sp:.1e}; "
        f"fixed-scale dV vs the variant's oracle {rel_err(f['dV'], o['dV']):.2e}")
    assert err <= REL_TOL
    check_blocks({"dV": blk})
    assert sp < 1e-3


def _dominant_key_inputs(N, D):
    rng = np.random.default_rng(11)
    q = np.zeros((1, N, 1, D), np.float32)
    k = np.zeros((1, N, 1, D), np.float32)
    q[..., 0] = 9.5
    k[:, 0, :, 0] = 9.5          # every query's score for key 0 is 11.3 above the rest
    v = rng.standard_normal((1, N, 1, D)).astype(np.float32)
    do = rng.standard_normal((1, N, 1, D)).astype(np.float32)
    return dict(q=q, k=k, v=v, do=do)


def test_small_probabilities_keep_their_bits():
    """P ~ 1e-5 on every key but the dominant one: with the fixed scale 2^-8
    those codes vanish (dV of those keys is lost), with the block scale they
    keep three mantissa bits (as the oracle pins)."""
    w = synth.with_shape(synth.WORKLOADS["tiny_mha_128"], N=256, Hq=1, Hkv=1)
    d = _dominant_key_inputs(w.N, w.Dqk)
    g = run_gpu(w, d, flags=BLK)
    f = run_gpu(w, d)
    ex = run_oracle(w, d, flags=orc.EXACT_PBWD)
    mxo = run_oracle(w, d, flags=orc.MX_PBWD)
    ref = ex["dV"][:, 32:]
    e_blk, e_fix = rel_err(g["dV"][:, 32:], ref), rel_err(f["dV"][:, 32:], ref)
    say(f"  dV of the keys past the dominant block vs uncast P: block-scaled {e_blk:.3e}, fixed {e_fix:.3e}; "
        f"vs the variant's oracle {rel_err(g['dV'], mxo['dV']):.2e}")
    assert e_blk < 0.05 and e_fix > 0.5
    assert rel_err(g["dV"], mxo["dV"]) <= REL_TOL


@pytest.mark.slow
def test_long_flat_rows():
    """The 64K workload's last 512 keys: their dV sums the last 512 queries,
    whose rows spread over 65 536 keys.  Against dV from uncast probabilities
    (oracle on the causal suffix) the block-scaled operand is closer than the
    fixed one; against the variant's own oracle it meets the parity bound.
    The gain is small here (measured 3.67e-2 against 3.72e-2): with the
    temperature recipe most of the P mass reaching these keys lies above
    2^-14, where both casts keep three mantissa bits."""
    w = synth.WORKLOADS["gqa_d128_64k_nope"]
    d = synth.generate(w, seed=0)
    G, T = w.Hq // w.Hkv, 512
    sl = dict(q=d["q"][:, :, :G], k=d["k"][:, :, :1], v=d["v"][:, :, :1], do=d["do"][:, :, :G])
    ws = synth.with_shape(w, Hq=G, Hkv=1)
    g = run_gpu(ws, sl, flags=BLK, rowstats=False)
    f = run_gpu(ws, sl, rowstats=False)
    ex, _ = orc.attention_from_inputs(sl["q"], sl["k"], sl["v"], sl["do"], float(np.float32(w.tau)),
                                      flags=orc.EXACT_PBWD, row_lo=w.N - T)
    mx, _ = orc.attention_from_inputs(sl["q"], sl["k"], sl["v"], sl["do"], float(np.float32(w.tau)),
                                      flags=orc.MX_PBWD, row_lo=w.N - T)
    ref = ex["dV"][:, -T:]
    e_blk, e_fix = rel_err(g["dV"][:, -T:], ref), rel_err(f["dV"][:, -T:], ref)
    e_own = rel_err(g["dV"][:, -T:], mx["dV"][:, -T:])
    say(f"  last {T} keys, dV vs uncast P: block-scaled {e_blk:.3e}, fixed {e_fix:.3e}; vs the variant's oracle "
        f"{e_own:.2e}")
    assert e_blk < e_fix and e_own <= REL_TOL
