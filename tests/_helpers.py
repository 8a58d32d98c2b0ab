"""Shared helpers of the GPU parity tests: run the HIP path through the C ABI
and the oracle on the same seeded inputs, and compare."""
from __future__ import annotations

import sys

import numpy as np
import torch

import oracle as orc
import paper_2609_37852_amd as pk
from paper_2609_37852_amd import synth

REL_TOL = 2e-2          # relative Frobenius error bound for O, dQ, dK, dV (whole tensor)
# Per (head, 32-row block): the median block error within REL_TOL, and no
# block above 2^-3.  FP8 codes may legitimately differ where the GPU's FP32
# value and the oracle's FP64 value straddle a rounding boundary; one such
# flip moves its element by one E4M3 step, up to 2^-3 of the element, and a
# block dominated by one row (a near-one-hot row's single large dS' or P)
# moves with it.  A block with a larger error is more than a rounding flip.
BLOCK_TOL = 2.0 ** -3
INV_TOL = 1e-5          # |sum_j dS_ij| <= INV_TOL * max_j |dS_ij| on graded rows
COND_MIN = 2.0 ** -5    # grade rows with max|dS| / max P|dP| >= 2^-5


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def to_dev(x: np.ndarray, dtype: str) -> torch.Tensor:
    t = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32))
    return (t.to(torch.bfloat16) if dtype == "bf16" else t).cuda()


def np64(t: torch.Tensor) -> np.ndarray:
    return t.detach().float().cpu().numpy().astype(np.float64)


def problem(w: synth.Workload) -> pk.Problem:
    return pk.Problem(w.B, w.N, w.Hq, w.Hkv, w.Dqk, w.Dv, float(np.float32(w.tau)), causal=int(w.causal),
                      seqlen_kv=w.Nk)


def bwd_plain_and_stats(p, mode, mq, mk, mv, mdo, lse, do=None, o=None, delta_in=None, grad_dtype=torch.float32):
    """The backward twice: the plain kernel (what a caller without row
    statistics gets, and what the benchmark times) and the instrumented one.
    Returns the plain run's gradients and the instrumented run's statistics,
    after checking that the two runs' gradients are bitwise equal."""
    plain = pk.attn_fp8_bwd(p, mode, mq, mk, mv, mdo, lse, do, o, delta_in=delta_in, grad_dtype=grad_dtype,
                            rowstats=False)
    stats = pk.attn_fp8_bwd(p, mode, mq, mk, mv, mdo, lse, do, o, delta_in=delta_in, grad_dtype=grad_dtype,
                            rowstats=True)
    torch.cuda.synchronize()
    for name, a, b in zip(("dQ", "dK", "dV"), plain[:3], stats[:3]):
        assert torch.equal(a.view(torch.int16 if a.dtype == torch.bfloat16 else torch.int32),
                           b.view(torch.int16 if b.dtype == torch.bfloat16 else torch.int32)), \
            f"{name}: the instrumented backward differs from the plain one"
    return plain[0], plain[1], plain[2], stats[3]


def run_gpu(w, d, mode=pk.DELTA_MATCHING, grad_dtype=torch.float32, o_dtype=torch.bfloat16, rowstats=True,
            delta_in=None, isolate=True, lse_shift=0.0, flags=0):
    """Quantize, forward, correction and backward on the GPU.  The gradients
    are those of the plain backward kernel; with rowstats the instrumented
    kernel runs as well (bitwise-equal gradients are asserted) and supplies
    the row statistics.  isolate=False drops the per-channel maxima (no
    isolated score channel); lse_shift is added to the LSE the correction
    and the backward read; flags are the problem's numerics options."""
    q, k, v, do = (to_dev(d[n], w.dtype) for n in ("q", "k", "v", "do"))
    mq, mk, mv, mdo = (pk.attn_fp8_quantize(t, amax=isolate) for t in (q, k, v, do))
    p = problem(w)
    p.flags = flags
    o, lse = pk.attn_fp8_fwd(p, mq, mk, mv, o_dtype=o_dtype)
    lse_b = lse + lse_shift if lse_shift else lse
    delta = pk.attn_fp8_delta(p, mode, mq, mk, mv, mdo, lse_b, do, o)
    if rowstats:
        dq, dk, dv, rs = bwd_plain_and_stats(p, mode, mq, mk, mv, mdo, lse_b, do, o, delta_in=delta_in,
                                             grad_dtype=grad_dtype)
    else:
        dq, dk, dv, rs = pk.attn_fp8_bwd(p, mode, mq, mk, mv, mdo, lse_b, do, o, delta_in=delta_in,
                                         grad_dtype=grad_dtype)
    torch.cuda.synchronize()
    out = dict(O=np64(o), LSE=np64(lse), delta=np64(delta), dQ=np64(dq), dK=np64(dk), dV=np64(dv),
               rowstats=rs.cpu().numpy() if rs is not None else None)
    out["mx"] = {n: {f: getattr(m, f).cpu().numpy() for f in ("code_row", "scale_row", "code_col", "scale_col")}
                 for n, m in (("Q", mq), ("K", mk), ("V", mv), ("dO", mdo))}
    return out


def run_oracle(w, d, mode=orc.DELTA_MATCHING, o_round=orc.ROUND_BF16, **kw):
    out, quant = orc.attention_from_inputs(d["q"], d["k"], d["v"], d["do"], float(np.float32(w.tau)),
                                           delta_mode=mode, o_round=o_round, want_rowstats=True,
                                           causal=w.causal, **kw)
    out["quant"] = quant
    return out


def rel_err(a, b):
    nb = np.linalg.norm(b)
    return float(np.linalg.norm(a - b) / nb) if nb > 0 else float(np.linalg.norm(a))


def block_errors(g, r):
    """Relative Frobenius error of every (batch, head, 32-row block) of a
    [B, N, H, D] output (rows: queries for O and dQ, keys for dK and dV).
    A block's error is taken against max(its own norm, a quarter of the RMS
    block norm of its head).  Blocks far below their head's typical norm are
    made of rows whose output is a cancellation: near-one-hot rows (the rows
    reading R12 excludes), where dS_ij = P_ij (dP_ij - delta_i) is far below
    the FP32 resolution of P_ij dP_ij, and the last key blocks, which see
    only the diagonal queries; there a relative error measures that
    cancellation, not the kernel.  Returns the worst block error, its
    (b, h, block) and the median block error."""
    B, N, H, D = r.shape
    nb = N // 32
    e = (g - r).reshape(B, nb, 32, H, D)
    rr = r.reshape(B, nb, 32, H, D)
    en = np.sqrt((e ** 2).sum(axis=(2, 4)))               # [B, nb, H]
    rn = np.sqrt((rr ** 2).sum(axis=(2, 4)))
    floor = np.sqrt(np.mean(rn ** 2, axis=1, keepdims=True)) / 4
    ratio = en / np.maximum(np.maximum(rn, floor), 1e-300)
    idx = np.unravel_index(int(np.argmax(ratio)), ratio.shape)
    return float(ratio.max()), (int(idx[0]), int(idx[2]), int(idx[1])), float(np.median(ratio))


def check_blocks(blk):
    """blk: {name: block_errors(...)}; asserts the per-block bounds."""
    for k, (worst, at, med) in blk.items():
        assert worst <= BLOCK_TOL, (k, worst, at)
        assert med <= REL_TOL, (k, med)


def invariant_report(gpu_rs, min_row=1):
    """Row-sum invariant on the GPU's own pre-cast dS (reading R12).  Graded
    rows: at least two visible keys (i >= min_row) and cond = max|dS| /
    max P|dP| >= 2^-5, both maxima from the GPU's own row statistics."""
    s = gpu_rs[..., pk.RS_SUM_DS]
    mx = gpu_rs[..., pk.RS_MAXABS_DS]
    mpdp = gpu_rs[..., pk.RS_MAX_PDP]
    N = s.shape[-1]
    rows = np.broadcast_to(np.arange(N), s.shape)
    cond = np.where(mpdp > 0, mx / np.maximum(mpdp, 1e-300), 0.0)
    graded = (rows >= max(min_row, 1)) & (cond >= COND_MIN) & (mx > 0)
    ratio = np.abs(s) / np.maximum(mx, 1e-300)
    worst_idx = None
    if graded.any():
        masked = np.where(graded, ratio, -1.0)
        worst_idx = tuple(int(x) for x in np.unravel_index(int(np.argmax(masked)), masked.shape))
    n_rows = int((rows >= max(min_row, 1)).sum())
    return dict(graded=int(graded.sum()), rows=n_rows, share=float(graded.sum()) / max(n_rows, 1),
                worst=float(ratio[graded].max()) if graded.any() else 0.0, worst_at=worst_idx,
                median=float(np.median(ratio[graded])) if graded.any() else 0.0,
                violations=int((ratio[graded] > INV_TOL).sum()))


def check_row_stat_fields(gpu_rs, orc_rs):
    """The GPU's own conditioning statistics against the oracle's: max P|dP|
    and max|dS| (FP32 vs FP64 of the same products), and sum P' (same codes
    except at rounding boundaries).  Returns the median relative differences
    over rows with a nonzero oracle value."""
    out = {}
    for name, gi, oi in (("max_pdp", pk.RS_MAX_PDP, orc.ST_MAX_PDP), ("max_ds", pk.RS_MAXABS_DS, orc.ST_MAXABS_DS),
                         ("sum_pcast", pk.RS_SUM_PCAST, orc.ST_SUM_PCAST)):
        g, o = gpu_rs[..., gi], orc_rs[..., oi]
        live = o > 0
        out[name] = float(np.median(np.abs(g[live] - o[live]) / o[live])) if live.any() else 0.0
    return out
