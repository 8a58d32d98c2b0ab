"""Reference oracle for block-scaled FP8 attention with Delta-Matching.

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
CPU-baseline leg of ``bench.py`` import this package; the product path
(``paper_2609_37852_amd``) never imports, loads or calls it, and this package
never imports the product.

A thin ctypes layer over ``attn_oracle.c`` (plain FP64 C).  The arithmetic and
the readings of the paper it implements are documented in that file.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

from . import build as _build

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB = None

_dp = ctypes.POINTER(ctypes.c_double)
_u8p = ctypes.POINTER(ctypes.c_uint8)
_i32p = ctypes.POINTER(ctypes.c_int32)

EXACT_PFWD, EXACT_PBWD, EXACT_DS, MX_PBWD = 1, 2, 4, 8
EXACT_ALL = EXACT_PFWD | EXACT_PBWD | EXACT_DS
DELTA_MATCHING, DELTA_STALE_ROWSUM, DELTA_CONSISTENT_DO = 0, 1, 2
ROUND_NONE, ROUND_F32, ROUND_BF16 = 0, 1, 2
ST_SUM_DS, ST_SUMABS_DS, ST_MAXABS_DS, ST_MAX_PDP, ST_SUM_DSCAST, ST_SUMABS_DSCAST, ST_SUM_P, \
    ST_SUM_PDP, ST_SUM_PCAST, ST_SUM_P_ABSTERMS, NSTAT = range(11)


class _Problem(ctypes.Structure):
    _fields_ = [("B", ctypes.c_int64), ("N", ctypes.c_int64), ("Hq", ctypes.c_int64),
                ("Hkv", ctypes.c_int64), ("Dqk", ctypes.c_int64), ("Dv", ctypes.c_int64),
                ("tau", ctypes.c_double), ("Nk", ctypes.c_int64), ("causal", ctypes.c_int32)]


def lib():
    """Load liborc.so, compiling it first only if it is not built yet."""
    global _LIB
    if _LIB is None:
        path = os.path.join(_HERE, "liborc.so")
        if not os.path.exists(path):
            _build.build()
        L = ctypes.CDLL(path)
        L.orc_e4m3_value.restype = ctypes.c_double
        L.orc_e4m3_value.argtypes = [ctypes.c_uint8]
        L.orc_e4m3_round.restype = ctypes.c_uint8
        L.orc_e4m3_round.argtypes = [ctypes.c_double]
        L.orc_pow2_exponent.restype = ctypes.c_int
        L.orc_pow2_exponent.argtypes = [ctypes.c_double]
        L.orc_bf16_round.restype = ctypes.c_double
        L.orc_bf16_round.argtypes = [ctypes.c_double]
        L.orc_e4m3_round_array.argtypes = [_dp, ctypes.c_int64, _u8p]
        L.orc_e4m3_value_array.argtypes = [_u8p, ctypes.c_int64, _dp]
        L.orc_pow2_exponent_array.argtypes = [_dp, ctypes.c_int64, _i32p]
        L.orc_bf16_round_array.argtypes = [_dp, ctypes.c_int64, _dp]
        L.orc_quantize.restype = ctypes.c_int64
        L.orc_quantize.argtypes = [_dp] + [ctypes.c_int64] * 4 + [_u8p] * 4
        L.orc_dequantize.argtypes = [_u8p] * 4 + [ctypes.c_int64] * 4 + [_dp, _dp]
        L.orc_producer.argtypes = [_dp] + [ctypes.c_int64] * 4 + [ctypes.c_double, ctypes.c_int, _dp, _dp]
        L.orc_producer_rope.argtypes = ([_dp] + [ctypes.c_int64] * 4 + [_dp, ctypes.c_int64, ctypes.c_int64,
                                        ctypes.c_double, ctypes.c_int, _dp, _dp])
        L.orc_producer_ext.argtypes = ([_dp] + [ctypes.c_int64] * 4 + [_dp, ctypes.c_double, _dp, ctypes.c_int64,
                                       ctypes.c_int64, ctypes.c_double, ctypes.c_int, _dp, _dp])
        L.orc_attention.restype = ctypes.c_int
        L.orc_attention.argtypes = ([ctypes.POINTER(_Problem)] + [ctypes.c_int] * 4 + [_dp] * 23
                                    + [ctypes.c_int64, ctypes.c_int])
        _LIB = L
    return _LIB


def _f64(a):
    return np.ascontiguousarray(a, dtype=np.float64)


def _ptr(a, t=_dp):
    if a is None:
        return None
    return a.ctypes.data_as(t)


# ---------------------------------------------------------------- codec
def e4m3_round(y) -> np.ndarray:
    """C8: E4M3FN round-to-nearest-even with saturation at +-448 (uint8 codes)."""
    y = _f64(y)
    out = np.empty(y.shape, np.uint8)
    lib().orc_e4m3_round_array(_ptr(y), y.size, _ptr(out, _u8p))
    return out


def e4m3_value(c) -> np.ndarray:
    c = np.ascontiguousarray(c, dtype=np.uint8)
    out = np.empty(c.shape, np.float64)
    lib().orc_e4m3_value_array(_ptr(c, _u8p), c.size, _ptr(out))
    return out


def pow2_exponent(a) -> np.ndarray:
    a = _f64(a)
    out = np.empty(a.shape, np.int32)
    lib().orc_pow2_exponent_array(_ptr(a), a.size, _ptr(out, _i32p))
    return out


def bf16_round(x) -> np.ndarray:
    x = _f64(x)
    out = np.empty(x.shape, np.float64)
    lib().orc_bf16_round_array(_ptr(x), x.size, _ptr(out))
    return out


def quantize(x):
    """x: [B, N, H, D] (exact values, any float dtype).  Returns dict with
    code_row [B,H,N,D], scale_row [B,H,N,D/32], code_col [B,H,D,N],
    scale_col [B,H,D,N/32] (uint8) and 'nonfinite'."""
    x = _f64(x)
    B, N, H, D = x.shape
    assert D % 32 == 0 and N % 32 == 0, "blocks of 32 along both D and N"
    out = dict(code_row=np.empty((B, H, N, D), np.uint8), scale_row=np.empty((B, H, N, D // 32), np.uint8),
               code_col=np.empty((B, H, D, N), np.uint8), scale_col=np.empty((B, H, D, N // 32), np.uint8))
    nf = lib().orc_quantize(_ptr(x), B, N, H, D, *[_ptr(out[k], _u8p) for k in
                                                    ("code_row", "scale_row", "code_col", "scale_col")])
    out["nonfinite"] = int(nf)
    return out


def producer(x, prescale=1.0, center=False):
    """Input producer (App. B.6.1, reading R13): x [B, N, H, D] (exact
    values) -> (y, mean): y = fl32(fl32(x * prescale) - mean), mean [B, H, D]
    the FP32 mean over tokens (zero unless center).  prescale is taken as
    the FP32 value it rounds to."""
    x = _f64(x)
    B, N, H, D = x.shape
    assert N % 32 == 0
    y = np.empty_like(x)
    mean = np.empty((B, H, D))
    lib().orc_producer(_ptr(x), B, N, H, D, float(np.float32(prescale)), int(bool(center)), _ptr(y), _ptr(mean))
    return y, mean


def producer_ext(x, gain=None, eps=1e-6, rope=None, lo=0, R=0, prescale=1.0, center=False):
    """The full producer (readings R17, R16, R13): QK normalization with
    gain [D] (FP32 values) and eps (taken as its FP32 value), the rotary
    embedding with rope [N, R/2, 2], prescale, centring.  Returns (y, mean)."""
    x = _f64(x)
    B, N, H, D = x.shape
    assert N % 32 == 0
    if gain is not None:
        gain = _f64(gain)
        assert gain.shape == (D,)
    if rope is not None:
        rope = _f64(rope)
        assert rope.shape == (N, R // 2, 2) and lo + R <= D
    y = np.empty_like(x)
    mean = np.empty((B, H, D))
    lib().orc_producer_ext(_ptr(x), B, N, H, D, _ptr(gain), float(np.float32(eps)), _ptr(rope), int(lo),
                           int(R if rope is not None else 0), float(np.float32(prescale)), int(bool(center)),
                           _ptr(y), _ptr(mean))
    return y, mean


def producer_rope(x, rope, lo, R, prescale=1.0, center=False):
    """Producer with the fused rotary embedding (App. B.6.1, reading R16):
    rope [N, R/2, 2] (cosine, sine per token and pair, FP32 values); channels
    lo .. lo + R - 1 rotated in pairs (lo + c, lo + c + R/2) and rounded to
    BF16, then producer().  Returns (y, mean)."""
    x = _f64(x)
    B, N, H, D = x.shape
    assert N % 32 == 0 and R % 2 == 0 and 0 <= lo and lo + R <= D
    rope = _f64(rope)
    assert rope.shape == (N, R // 2, 2)
    y = np.empty_like(x)
    mean = np.empty((B, H, D))
    lib().orc_producer_rope(_ptr(x), B, N, H, D, _ptr(rope), int(lo), int(R), float(np.float32(prescale)),
                            int(bool(center)), _ptr(y), _ptr(mean))
    return y, mean


def dequantize(q, B, N, H, D):
    """Decode both MX copies of one operand into [B,H,N,D] float64 arrays."""
    xr = np.empty((B, H, N, D), np.float64)
    xc = np.empty((B, H, N, D), np.float64)
    arrs = [np.ascontiguousarray(q[k], dtype=np.uint8) for k in ("code_row", "scale_row", "code_col", "scale_col")]
    lib().orc_dequantize(*[_ptr(a, _u8p) for a in arrs], B, N, H, D, _ptr(xr), _ptr(xc))
    return xr, xc


# ---------------------------------------------------------------- attention
def attention(B, N, Hq, Hkv, Dqk, Dv, tau, ops, dO_raw=None, *, flags=0, delta_mode=DELTA_MATCHING,
              o_round=ROUND_BF16, grad_round=ROUND_NONE, delta_in=None, lse_in=None, want_rowstats=False,
              want_phat=False, want_ds=False, row_lo=0, nthreads=0, causal=True, Nk=None):
    """Forward + correction + backward on dequantized operands.

    ops: dict with Qr, Kr, Vr, dOr, Qc, Kc, Vc, dOc, each [B,H,L,D] float64
    (H = Hq, L = N for Q/dO; H = Hkv, L = Nk for K/V).  dO_raw: [B,N,Hq,Dv]
    (needed for the stale correction).  causal: top-left mask (Nk must equal
    N); without it every query sees all Nk keys (Nk defaults to N).
    row_lo: compute only query rows and keys >= row_lo (the causal suffix;
    other entries stay zero).  Returns a dict of float64 arrays."""
    L = lib()
    Nk = N if Nk is None else int(Nk)
    pr = _Problem(B, N, Hq, Hkv, Dqk, Dv, float(tau), Nk, int(bool(causal)))
    names = ("Qr", "Kr", "Vr", "dOr", "Qc", "Kc", "Vc", "dOc")
    shapes = dict(Qr=(B, Hq, N, Dqk), Kr=(B, Hkv, Nk, Dqk), Vr=(B, Hkv, Nk, Dv), dOr=(B, Hq, N, Dv),
                  Qc=(B, Hq, N, Dqk), Kc=(B, Hkv, Nk, Dqk), Vc=(B, Hkv, Nk, Dv), dOc=(B, Hq, N, Dv))
    arrs = {}
    for k in names:
        a = _f64(ops[k])
        assert a.shape == shapes[k], (k, a.shape, shapes[k])
        arrs[k] = a
    if dO_raw is None:
        dO_raw = np.zeros((B, N, Hq, Dv))
    dO_raw = _f64(dO_raw)
    assert dO_raw.shape == (B, N, Hq, Dv)
    if delta_in is not None:
        delta_in = _f64(delta_in)
        assert delta_in.shape == (B, Hq, N)
    if lse_in is not None:
        lse_in = _f64(lse_in)
        assert lse_in.shape == (B, Hq, N)
    out = dict(O=np.zeros((B, N, Hq, Dv)), O_unrounded=np.zeros((B, N, Hq, Dv)), LSE=np.zeros((B, Hq, N)),
               delta=np.zeros((B, Hq, N)), dQ=np.zeros((B, N, Hq, Dqk)), dK=np.zeros((B, Nk, Hkv, Dqk)),
               dV=np.zeros((B, Nk, Hkv, Dv)))
    out["rowstats"] = np.zeros((B, Hq, N, NSTAT)) if want_rowstats else None
    out["phat"] = np.zeros((B, Hq, N, Nk)) if want_phat else None
    out["dsraw"] = np.zeros((B, Hq, N, Nk)) if want_ds else None
    out["dshat"] = np.zeros((B, Hq, N, Nk)) if want_ds else None
    out["pbhat"] = np.zeros((B, Hq, N, Nk)) if want_ds else None
    rc = L.orc_attention(ctypes.byref(pr), flags, delta_mode, o_round, grad_round,
                         *[_ptr(arrs[k]) for k in names], _ptr(dO_raw), _ptr(delta_in), _ptr(lse_in),
                         _ptr(out["O"]), _ptr(out["O_unrounded"]), _ptr(out["LSE"]), _ptr(out["delta"]),
                         _ptr(out["dQ"]), _ptr(out["dK"]), _ptr(out["dV"]), _ptr(out["rowstats"]),
                         _ptr(out["phat"]), _ptr(out["dsraw"]), _ptr(out["dshat"]), _ptr(out["pbhat"]), int(row_lo),
                         int(nthreads))
    if rc != 0:
        raise ValueError(f"orc_attention failed ({rc})")
    return out


def attention_from_inputs(q, k, v, do, tau, *, flags=0, delta_mode=DELTA_MATCHING, o_round=ROUND_BF16,
                          grad_round=ROUND_NONE, exact_inputs=False, protected_dp=False, **kw):
    """Convenience: raw inputs q,do [B,N,Hq,D], k,v [B,Nk,Hkv,D] (exact
    values) -> quantize each (or, with exact_inputs, use the raw values for
    both copies) -> attention().  Returns (outputs, quantized dict).

    protected_dp: the protected-dP variant (App. B.6.3, correction variants;
    App. C.4.2): dP = dO V^T from dO and V rounded to BF16 instead of their
    FP8 row copies (products exact, sums in FP64 here); the row copies of dO
    and V are the operands of dP only, so every other product keeps its FP8
    operands.  The paper pairs it with the stale correction."""
    q, k, v, do = (_f64(t) for t in (q, k, v, do))
    B, N, Hq, Dqk = q.shape
    Nk, Hkv, Dv = k.shape[1], k.shape[2], v.shape[3]
    quant = {}
    ops = {}
    for name, t in (("Q", q), ("K", k), ("V", v), ("dO", do)):
        Bt, Nt, Ht, Dt = t.shape
        if exact_inputs:
            xr = np.ascontiguousarray(t.transpose(0, 2, 1, 3))
            ops[name + "r"], ops[name + "c"] = xr, xr
        else:
            qd = quantize(t)
            quant[name] = qd
            ops[name + "r"], ops[name + "c"] = dequantize(qd, Bt, Nt, Ht, Dt)
    if protected_dp:
        ops["dOr"] = np.ascontiguousarray(bf16_round(do).transpose(0, 2, 1, 3))
        ops["Vr"] = np.ascontiguousarray(bf16_round(v).transpose(0, 2, 1, 3))
    out = attention(B, N, Hq, Hkv, Dqk, Dv, tau, ops, do, flags=flags, delta_mode=delta_mode,
                    o_round=o_round, grad_round=grad_round, Nk=Nk, **kw)
    return out, quant
