"""Row-sum and key-gradient diagnostics of the backward (App. C.1, on synthetic
data), from the per-row statistics the backward records with `rowstats`:
[B, Hq, N, 7] FP64 = (sum_j dS_ij, sum_j |dS_ij|, sum_j dS'_ij, max_j |dS_ij|,
sum_j |dS'_ij|, max_j P_ij |dP_ij|, sum_j P'_ij) with dS the FP32 score
gradient before the FP8 cast and dS', P' the decoded casts.

  r_pre_i  = |sum_j dS_ij| / l_i,   r_post_i = |sum_j dS'_ij| / l_i,
  r_post,own_i = |sum_j dS'_ij| / l'_i,  l'_i = sum_j |dS'_ij| (rows with l'_i > 0),
  kappa_i  = (sum_j dS'_ij - sum_j dS_ij) / l_i,     l_i = sum_j |dS_ij|,
  c_K      = || sum_j dK_j ||_2 / (sum_j ||dK_j||_2^2)^(1/2)   per (batch, KV head),
  e_i      = |delta_i - delta*_i| |S^P_i| / l_i,  with S^PdP_i = R_i(0),
             S^P_i = R_i(0) - R_i(1), delta*_i = S^PdP_i / S^P_i, R_i(c) the
             pre-cast row sum of a backward run with the correction injected as c.

Rows: query positions i >= 64 whose l_i is nonzero under every correction
compared (the common row set).
The numpy functions here run anywhere; run() drives the library on a GPU.
"""
import numpy as np

MIN_ROW = 64
MODES = ("stale_rowsum", "consistent_do", "matching")


def common_rows(stats_by_mode, min_row=MIN_ROW):
    """Boolean [B, Hq, N] mask of the common row set."""
    first = next(iter(stats_by_mode.values()))
    n = first.shape[2]
    keep = np.broadcast_to(np.arange(n) >= min_row, first.shape[:3]).copy()
    for st in stats_by_mode.values():
        keep &= st[..., 1] > 0
    return keep


def row_residuals(stats_by_mode, min_row=MIN_ROW):
    """Per correction: median r_pre and r_post, and mean kappa, over the
    common row set (rows whose cast gradient vanishes count with r_post 0);
    median r_post,own over those of its rows whose cast gradient does not
    vanish."""
    keep = common_rows(stats_by_mode, min_row)
    out = {}
    for name, st in stats_by_mode.items():
        s, ell, cast = st[..., 0][keep], st[..., 1][keep], st[..., 2][keep]
        out[name] = dict(r_pre_median=float(np.median(np.abs(s) / ell)),
                         r_post_median=float(np.median(np.abs(cast) / ell)),
                         kappa_mean=float(np.mean((cast - s) / ell)))
        if st.shape[-1] > 4:
            own = st[..., 4][keep]
            nz = own > 0
            out[name]["r_post_own_median"] = float(np.median(np.abs(cast[nz]) / own[nz])) if nz.any() else 0.0
    out["rows"] = int(keep.sum())
    return out


def key_common_mode(dk):
    """c_K of each (batch, KV head) from dK [B, N, Hkv, D] (any float dtype)."""
    g = np.asarray(dk, dtype=np.float64)
    num = np.linalg.norm(g.sum(axis=1), axis=-1)                  # [B, Hkv]
    den = np.sqrt((g * g).sum(axis=(1, 3)))                        # [B, Hkv]
    return np.where(den > 0, num / np.where(den > 0, den, 1.0), 0.0)


def correction_discrepancy(delta, r0, r1, ell, min_row=MIN_ROW):
    """Median e_i over rows i >= min_row with l_i > 0 and S^P_i != 0.
    delta: [..., N] correction used; r0, r1: pre-cast row sums with 0 and 1
    injected; ell: l_i of the run with delta."""
    sp = r0 - r1
    n = delta.shape[-1]
    keep = (np.broadcast_to(np.arange(n) >= min_row, delta.shape)) & (ell > 0) & (sp != 0)
    dstar = r0[keep] / sp[keep]
    e = np.abs(delta[keep] - dstar) * np.abs(sp[keep]) / ell[keep]
    return float(np.median(e)), int(keep.sum())


def run(p, mq, mk, mv, mdo, lse, dout_raw, o):
    """All diagnostics for one problem whose forward (o, lse) has been run:
    three backward runs with row statistics, one per correction, and two more
    with 0 and 1 injected for e_i.  Returns a JSON-ready dict."""
    import torch
    from . import binding as pk

    modes = dict(stale_rowsum=pk.DELTA_STALE_ROWSUM, consistent_do=pk.DELTA_CONSISTENT_DO,
                 matching=pk.DELTA_MATCHING)
    stats, ck, deltas = {}, {}, {}
    for name, mode in modes.items():
        delta = pk.attn_fp8_delta(p, mode, mq, mk, mv, mdo, lse, dout_raw, o)
        _, dk, _, rs = pk.attn_fp8_bwd(p, mode, mq, mk, mv, mdo, lse, dout_raw, o, delta_in=delta,
                                       grad_dtype=torch.float32, rowstats=True)
        torch.cuda.synchronize()
        stats[name] = rs.cpu().numpy()
        ck[name] = float(np.median(key_common_mode(dk.cpu().numpy())))
        deltas[name] = delta
    out = row_residuals(stats)
    for name in modes:
        out[name]["c_K_median"] = ck[name]
    dm = deltas["matching"]
    zero = torch.zeros_like(dm)
    one = torch.zeros_like(dm)
    one[..., 0] = 1.0
    rsum = []
    for inj in (zero, one):
        _, _, _, rs = pk.attn_fp8_bwd(p, pk.DELTA_MATCHING, mq, mk, mv, mdo, lse, delta_in=inj,
                                      grad_dtype=torch.float32, rowstats=True)
        torch.cuda.synchronize()
        rsum.append(rs[..., 0].cpu().numpy())
    d = dm.cpu().numpy().astype(np.float64)
    e, n = correction_discrepancy(d[..., 0] + d[..., 1], rsum[0], rsum[1], stats["matching"][..., 1])
    out["matching"]["e_median"] = e
    out["e_rows"] = n
    return out
