"""Shared helpers of the GPU parity tests: run the HIP path through the C ABI
and the oracle on the same seeded inputs, and compare."""
from __future__ import annotations

import sys

import numpy as np
import torch

import oracle as orc
import paper_2609_37852_amd as pk
from paper_2609_37852_amd import synth

REL_TOL = 2e-2          # relative Frobenius error bound for O, dQ, dK, dV
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
    return pk.Problem(w.B, w.N, w.Hq, w.Hkv, w.Dqk, w.Dv, float(np.float32(w.tau)))


def run_gpu(w, d, mode=pk.DELTA_MATCHING, grad_dtype=torch.float32, o_dtype=torch.bfloat16, rowstats=True,
            delta_in=None, isolate=True):
    """Quantize, forward, correction and backward on the GPU.  isolate=False
    drops the per-channel maxima (no isolated score channel)."""
    q, k, v, do = (to_dev(d[n], w.dtype) for n in ("q", "k", "v", "do"))
    mq, mk, mv, mdo = (pk.attn_fp8_quantize(t, amax=isolate) for t in (q, k, v, do))
    p = problem(w)
    o, lse = pk.attn_fp8_fwd(p, mq, mk, mv, o_dtype=o_dtype)
    delta = pk.attn_fp8_delta(p, mode, mq, mk, mv, mdo, lse, do, o)
    dq, dk, dv, rs = pk.attn_fp8_bwd(p, mode, mq, mk, mv, mdo, lse, do, o, delta_in=delta_in,
                                     grad_dtype=grad_dtype, rowstats=rowstats)
    torch.cuda.synchronize()
    out = dict(O=np64(o), LSE=np64(lse), delta=np64(delta), dQ=np64(dq), dK=np64(dk), dV=np64(dv),
               rowstats=rs.cpu().numpy() if rs is not None else None)
    out["mx"] = {n: {f: getattr(m, f).cpu().numpy() for f in ("code_row", "scale_row", "code_col", "scale_col")}
                 for n, m in (("Q", mq), ("K", mk), ("V", mv), ("dO", mdo))}
    return out


def run_oracle(w, d, mode=orc.DELTA_MATCHING, o_round=orc.ROUND_BF16, **kw):
    out, quant = orc.attention_from_inputs(d["q"], d["k"], d["v"], d["do"], float(np.float32(w.tau)),
                                           delta_mode=mode, o_round=o_round, want_rowstats=True, **kw)
    out["quant"] = quant
    return out


def rel_err(a, b):
    nb = np.linalg.norm(b)
    return float(np.linalg.norm(a - b) / nb) if nb > 0 else float(np.linalg.norm(a))


def invariant_report(gpu_rs, orc_rs):
    """Row-sum invariant on the GPU's own pre-cast dS.  Graded rows: at least
    two visible keys and cond = max|dS| / max P|dP| >= 2^-5."""
    s = gpu_rs[..., 0]
    mx = gpu_rs[..., 3]
    mpdp = orc_rs[..., orc.ST_MAX_PDP]
    N = s.shape[-1]
    rows = np.broadcast_to(np.arange(N), s.shape)
    cond = np.where(mpdp > 0, mx / np.maximum(mpdp, 1e-300), 0.0)
    graded = (rows >= 1) & (cond >= COND_MIN) & (mx > 0)
    ratio = np.abs(s) / np.maximum(mx, 1e-300)
    return dict(graded=int(graded.sum()), excluded=int((~graded).sum()),
                worst=float(ratio[graded].max()) if graded.any() else 0.0,
                median=float(np.median(ratio[graded])) if graded.any() else 0.0,
                violations=int((ratio[graded] > INV_TOL).sum()))
