"""The code against the values the paper fixes (tests/golden/paper_values.json,
each entry citing its passage)."""
import json
import os

import numpy as np

import oracle as orc
from paper_2609_37852_amd import diagnostics, synth

GOLD = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "paper_values.json")))


def test_e4m3_saturation():
    m = GOLD["e4m3_saturation"]["value"]
    codes = orc.e4m3_round(np.array([m, 1e6, -1e6, m * 1.03]))
    vals = orc.e4m3_value(codes)
    assert np.array_equal(vals, [m, m, -m, m])


def test_mx_block_size():
    blk = GOLD["mx_block"]["value"]
    x = np.random.default_rng(0).normal(size=(1, 64, 1, 64))
    q = orc.quantize(x)
    assert q["scale_row"].shape[-1] * blk == x.shape[-1]
    assert q["scale_col"].shape[-1] * blk == x.shape[1]


def test_credited_flops_follow_the_paper():
    g = GOLD["credited_flops"]
    sh = GOLD["paper_timing_shape"]
    w = synth.with_shape(synth.WORKLOADS["gqa_d128_8k"], B=sh["batch"], N=sh["seqlen"], Hq=sh["heads_q"],
                         Hkv=sh["heads_kv"], Dqk=sh["head_dim"], Dv=sh["head_dim"])
    fwd, bwd = w.credited_flops()
    n = sh["batch"] * sh["heads_q"] * sh["seqlen"] ** 2 * sh["head_dim"]
    assert fwd == g["fwd_per_BHqN2d"] * n and bwd == g["bwd_per_BHqN2d"] * n


def test_diagnostic_row_set():
    assert diagnostics.MIN_ROW == GOLD["diagnostic_min_row"]["value"]


def test_credited_split_reproduces_the_printed_combined_rate():
    # The combined column is total credited work over total time, so with the
    # forward/backward split the code credits, the three printed rates must
    # agree to the table's rounding (one decimal).
    for r in GOLD["kernel_throughput_table"]["rows"]:
        w = synth.with_shape(synth.WORKLOADS["gqa_d128_8k"], B=2, N=8192, Hq=r["heads_q"],
                             Hkv=r["heads_kv"], Dqk=r["head_dim"], Dv=r["head_dim"])
        fwd, bwd = w.credited_flops()
        combined = (fwd + bwd) / (fwd / r["fwd"] + bwd / r["bwd"])
        assert abs(combined - r["fwd_bwd"]) <= 0.1, (r, combined)
