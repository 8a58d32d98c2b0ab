"""The diagnostic formulas (App. C.1) on arrays with known answers (CPU)."""
import numpy as np

from paper_2609_37852_amd import diagnostics as dg


def _stats(B=1, H=2, N=128, seed=0):
    rng = np.random.default_rng(seed)
    ell = rng.uniform(1.0, 2.0, (B, H, N))
    st = np.zeros((B, H, N, 5))
    st[..., 1] = ell
    return st, ell


def test_common_rows_excludes_early_and_empty_rows():
    a, _ = _stats()
    b, _ = _stats(seed=1)
    b[0, 1, 100, 1] = 0.0                      # l_i = 0 under one correction only
    keep = dg.common_rows({"x": a, "y": b})
    assert not keep[..., :64].any()
    assert not keep[0, 1, 100]
    assert keep.sum() == 2 * 64 - 1


def test_row_residuals_known_values():
    st, ell = _stats()
    st[..., 0] = 0.25 * ell * np.where(np.arange(128) % 2 == 0, 1.0, -1.0)   # |sum dS| = l / 4
    st[..., 2] = st[..., 0] + 0.125 * ell                                     # cast adds l / 8
    r = dg.row_residuals({"m": st})
    assert r["rows"] == 2 * 64
    assert np.isclose(r["m"]["r_pre_median"], 0.25)
    assert np.isclose(r["m"]["kappa_mean"], 0.125)
    # r_post: |+-l/4 + l/8| / l is 3/8 or 1/8 in equal numbers; the median of the 128 values
    assert np.isclose(r["m"]["r_post_median"], 0.25)
    # own denominator: with sum |dS'| = l / 2 the same rows give 3/4 and 1/4; rows with a
    # vanishing cast (sum |dS'| = 0) are left out of it only
    st[..., 4] = 0.5 * ell
    st[0, 0, 64:80, 4] = 0.0
    r = dg.row_residuals({"m": st})
    assert np.isclose(r["m"]["r_post_own_median"], 0.5)
    assert np.isclose(r["m"]["r_post_median"], 0.25)


def test_key_common_mode_extremes():
    rng = np.random.default_rng(2)
    u = rng.normal(size=(1, 1, 1, 16))
    N = 36
    same = np.broadcast_to(u, (1, N, 1, 16))
    assert np.isclose(dg.key_common_mode(same)[0, 0], np.sqrt(N))        # all keys alike: sqrt(N)
    alt = same * np.where(np.arange(N) % 2 == 0, 1.0, -1.0)[None, :, None, None]
    assert np.isclose(dg.key_common_mode(alt)[0, 0], 0.0)                # pairwise cancelling: 0
    assert dg.key_common_mode(np.zeros((1, 4, 1, 8)))[0, 0] == 0.0


def test_correction_discrepancy_recovers_known_offset():
    rng = np.random.default_rng(3)
    n = 200
    sp = rng.uniform(0.5, 1.5, n)               # S^P
    dstar = rng.normal(size=n)                  # S^PdP / S^P
    r0 = dstar * sp
    r1 = r0 - sp                                # R(1) = S^PdP - S^P
    ell = rng.uniform(1.0, 3.0, n)
    off = 1e-3
    e, rows = dg.correction_discrepancy(dstar + off, r0, r1, ell)
    assert rows == n - 64
    ref = np.median(off * sp[64:] / ell[64:])
    assert np.isclose(e, ref, rtol=1e-9)
