"""ctypes binding of libattn_fp8.so (include/attn_fp8.h).

Argument marshalling only: torch supplies device memory and the current HIP
stream; every step of the computation runs in the library's kernels.  There
is no fallback: if the library is not built, or a call fails, an exception is
raised.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass

import torch

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libattn_fp8.so")

DTYPE_F32, DTYPE_BF16 = 0, 1
DELTA_MATCHING, DELTA_STALE_ROWSUM, DELTA_CONSISTENT_DO, DELTA_MATCHING_COMPENSATED = 0, 1, 2, 3
FLAG_PBWD_BLOCK_SCALED, FLAG_PROTECTED_DP, FLAG_ISOLATE3 = 1, 2, 4
QUANT_ROW, QUANT_COL, QUANT_BOTH = 1, 2, 3
# fields of the backward's per-row statistics [B, Hq, N, ROWSTATS] (FP64)
RS_SUM_DS, RS_SUMABS_DS, RS_SUM_DSCAST, RS_MAXABS_DS, RS_SUMABS_DSCAST, RS_MAX_PDP, RS_SUM_PCAST = range(7)
ROWSTATS = 7
STATUS = {0: "OK", -1: "EINVAL", -2: "EUNSUPPORTED", -3: "EALIGN", -4: "EWORKSPACE", -5: "EHIP"}
EXPORTS = ("attn_fp8_quantize", "attn_fp8_fwd", "attn_fp8_delta", "attn_fp8_bwd_workspace_size",
           "attn_fp8_bwd", "attn_fp8_bwd_noalloc", "attn_fp8_quantize_producer",
           "attn_fp8_producer_workspace_size", "attn_fp8_bwd_protected_dp", "attn_fp8_last_error")
NOALLOC_SCRATCH_BYTES = 64 << 20   # ATTN_FP8_NOALLOC_SCRATCH_BYTES


class AttnFp8Error(RuntimeError):
    def __init__(self, fn, code, msg):
        super().__init__(f"{fn} failed: {STATUS.get(code, code)}: {msg}")
        self.code = code


class _Problem(ctypes.Structure):
    _fields_ = [("batch", ctypes.c_int64), ("seqlen", ctypes.c_int64), ("heads_q", ctypes.c_int64),
                ("heads_kv", ctypes.c_int64), ("dim_qk", ctypes.c_int64), ("dim_v", ctypes.c_int64),
                ("causal", ctypes.c_int32), ("softmax_scale", ctypes.c_float), ("seqlen_kv", ctypes.c_int64),
                ("flags", ctypes.c_int32), ("seqlens_q", ctypes.c_void_p), ("seqlens_kv", ctypes.c_void_p),
                ("cast_dump", ctypes.c_void_p)]


class _Producer(ctypes.Structure):
    _fields_ = [("prescale", ctypes.c_float), ("center", ctypes.c_int32), ("channel_mean", ctypes.c_void_p),
                ("rms_gain", ctypes.c_void_p), ("rms_eps", ctypes.c_float), ("rope_cs", ctypes.c_void_p),
                ("rope_lo", ctypes.c_int64), ("rope_dim", ctypes.c_int64), ("seqlens", ctypes.c_void_p)]


class _MX(ctypes.Structure):
    _fields_ = [("code_row", ctypes.c_void_p), ("scale_row", ctypes.c_void_p),
                ("code_col", ctypes.c_void_p), ("scale_col", ctypes.c_void_p),
                ("channel_amax", ctypes.c_void_p)]


_I64x3 = ctypes.c_int64 * 3
_LIB = None


def lib():
    """Load the library (built by paper_2609_37852_amd.build / __graft_entry__.build)."""
    global _LIB
    if _LIB is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is not built; run `python -m paper_2609_37852_amd.build`")
        L = ctypes.CDLL(LIB_PATH)
        vp, i64, i32, sz = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int, ctypes.c_size_t
        P = ctypes.POINTER
        L.attn_fp8_quantize.argtypes = [vp, i32, i64, i64, i64, i64, P(ctypes.c_int64), P(_MX), i32, vp, vp]
        L.attn_fp8_quantize_producer.argtypes = [vp, i32, i64, i64, i64, i64, P(ctypes.c_int64), P(_Producer), vp, sz,
                                                 P(_MX), i32, vp, vp]
        L.attn_fp8_producer_workspace_size.argtypes = [i64, i64, i64, i64, P(_Producer), P(sz)]
        L.attn_fp8_fwd.argtypes = [P(_Problem), P(_MX), P(_MX), P(_MX), vp, i32, P(ctypes.c_int64), vp, vp]
        L.attn_fp8_delta.argtypes = [P(_Problem), i32, P(_MX), P(_MX), P(_MX), P(_MX), vp, vp, i32,
                                     P(ctypes.c_int64), vp, i32, P(ctypes.c_int64), vp, vp]
        L.attn_fp8_bwd_workspace_size.argtypes = [P(_Problem), P(sz)]
        L.attn_fp8_bwd.argtypes = [P(_Problem), i32, P(_MX), P(_MX), P(_MX), P(_MX), vp, vp, i32,
                                   P(ctypes.c_int64), vp, i32, P(ctypes.c_int64), vp, vp, vp, vp, i32,
                                   P(ctypes.c_int64), P(ctypes.c_int64), P(ctypes.c_int64), vp, sz, vp, vp, vp]
        L.attn_fp8_bwd_noalloc.argtypes = [P(_Problem), i32, P(_MX), P(_MX), P(_MX), P(_MX), vp, vp, i32,
                                           P(ctypes.c_int64), vp, i32, P(ctypes.c_int64), vp, vp, vp, vp, i32,
                                           P(ctypes.c_int64), P(ctypes.c_int64), P(ctypes.c_int64), vp, vp, vp]
        L.attn_fp8_bwd_protected_dp.argtypes = [P(_Problem), P(_MX), P(_MX), P(_MX), vp, vp, i32, P(ctypes.c_int64),
                                                vp, i32, P(ctypes.c_int64), vp, i32, P(ctypes.c_int64), vp, vp, vp,
                                                vp, i32, P(ctypes.c_int64), P(ctypes.c_int64), P(ctypes.c_int64), vp,
                                                sz, vp, vp]
        L.attn_fp8_last_error.restype = ctypes.c_char_p
        for name in EXPORTS[:-1]:
            getattr(L, name).restype = ctypes.c_int
        _LIB = L
    return _LIB


def last_error() -> str:
    return lib().attn_fp8_last_error().decode()


def _check(fn, rc):
    if rc != 0:
        raise AttnFp8Error(fn, rc, last_error())


def _stream(device=None):
    return ctypes.c_void_p(torch.cuda.current_stream(device).cuda_stream)


def _ptr(t):
    return ctypes.c_void_p(t.data_ptr()) if t is not None else ctypes.c_void_p(0)


def _dtype_code(dt):
    if dt == torch.bfloat16:
        return DTYPE_BF16
    if dt == torch.float32:
        return DTYPE_F32
    raise ValueError(f"unsupported dtype {dt}")


def _strides_bnh(t):
    assert t.dim() == 4 and t.stride(3) == 1, "expected [B, N, H, D] with contiguous channels"
    return _I64x3(t.stride(0), t.stride(1), t.stride(2))


@dataclass
class Problem:
    batch: int
    seqlen: int
    heads_q: int
    heads_kv: int
    dim_qk: int
    dim_v: int
    softmax_scale: float
    causal: int = 1
    seqlen_kv: int = 0          # key / value length; 0 stands for seqlen
    flags: int = 0              # FLAG_* numerics options
    # per-sequence lengths of a padded batch: device int32 [batch] tensors
    # (seqlens_kv without the mask only), or None for the full lengths
    seqlens_q: torch.Tensor | None = None
    seqlens_kv: torch.Tensor | None = None
    # instrumented backward only: a device uint8 tensor of cast_dump_bytes()
    # that receives the pre-cast P, dS and their codes (or None)
    cast_dump: torch.Tensor | None = None

    @property
    def nk(self) -> int:
        return self.seqlen_kv if self.seqlen_kv else self.seqlen

    def c(self):
        for t in (self.seqlens_q, self.seqlens_kv):
            assert t is None or (t.dtype == torch.int32 and t.is_contiguous() and t.numel() == self.batch), \
                "seqlens: contiguous int32 [batch] tensors"
        return _Problem(self.batch, self.seqlen, self.heads_q, self.heads_kv, self.dim_qk, self.dim_v,
                        self.causal, self.softmax_scale, self.seqlen_kv, self.flags,
                        _ptr(self.seqlens_q).value, _ptr(self.seqlens_kv).value, _ptr(self.cast_dump).value)

    def cast_dump_bytes(self) -> int:
        s = self.batch * self.heads_q * self.seqlen * self.nk
        return 10 * s + 2 * self.batch * self.heads_q * (self.seqlen // 32) * (self.nk // 32)

    def cast_dump_views(self):
        """(P, dS, Pc, dSc, eS, eP) views of cast_dump, each [B, Hq, N, Nk] or
        [B, Hq, N/32, Nk/32]."""
        B, H, N, Nk = self.batch, self.heads_q, self.seqlen, self.nk
        s, nb = B * H * N * Nk, B * H * (N // 32) * (Nk // 32)
        d = self.cast_dump
        return (d[:4 * s].view(torch.float32).view(B, H, N, Nk), d[4 * s:8 * s].view(torch.float32).view(B, H, N, Nk),
                d[8 * s:9 * s].view(B, H, N, Nk), d[9 * s:10 * s].view(B, H, N, Nk),
                d[10 * s:10 * s + nb].view(B, H, N // 32, Nk // 32),
                d[10 * s + nb:10 * s + 2 * nb].view(B, H, N // 32, Nk // 32))


@dataclass
class MX:
    """MX copies of one operand X[B, N, H, D] (device uint8 tensors) and its
    optional per-channel maxima [B, H, D] (float32)."""
    code_row: torch.Tensor | None
    scale_row: torch.Tensor | None
    code_col: torch.Tensor | None
    scale_col: torch.Tensor | None
    channel_amax: torch.Tensor | None = None

    def c(self):
        return _MX(*(t.data_ptr() if t is not None else None
                     for t in (self.code_row, self.scale_row, self.code_col, self.scale_col, self.channel_amax)))

    @staticmethod
    def empty(B, N, H, D, device, which=QUANT_BOTH, amax=True):
        u8 = dict(dtype=torch.uint8, device=device)
        row = which & QUANT_ROW
        col = which & QUANT_COL
        return MX(torch.empty((B, H, N, D), **u8) if row else None,
                  torch.empty((B, H, N, D // 32), **u8) if row else None,
                  torch.empty((B, H, D, N), **u8) if col else None,
                  torch.empty((B, H, D, N // 32), **u8) if col else None,
                  torch.empty((B, H, D), dtype=torch.float32, device=device) if (amax and col) else None)


def attn_fp8_quantize(x: torch.Tensor, which: int = QUANT_BOTH, nonfinite: torch.Tensor | None = None,
                      amax: bool = True) -> MX:
    """x: [B, N, H, D] bf16/f32 on the GPU -> MX copies (App. B.6.1), plus the
    per-channel maxima that enable the isolated score channel (amax=True)."""
    B, N, H, D = x.shape
    out = MX.empty(B, N, H, D, x.device, which, amax=amax)
    m = out.c()
    _check("attn_fp8_quantize",
           lib().attn_fp8_quantize(_ptr(x), _dtype_code(x.dtype), B, N, H, D, _strides_bnh(x), ctypes.byref(m),
                                   which, _ptr(nonfinite), _stream(x.device)))
    return out


def attn_fp8_quantize_producer(x: torch.Tensor, prescale: float = 1.0, center: bool = False,
                               which: int = QUANT_BOTH, nonfinite: torch.Tensor | None = None, amax: bool = True,
                               rope: torch.Tensor | None = None, rope_lo: int = 0,
                               rms_gain: torch.Tensor | None = None, rms_eps: float = 1e-6,
                               seqlens: torch.Tensor | None = None):
    """The input producer (App. B.6.1) then the quantizer: x [B, N, H, D] ->
    (MX copies of fl32(fl32(r prescale) - mean), mean [B, H, D] or None).  r
    is x, RMS-normalized with the gain rms_gain [D] (float32 on the device)
    when given, with channels rope_lo .. rope_lo + R - 1 then rotated by the
    table rope [N, R/2, 2] (float32 cos, sin on the device); normalized and
    rotated values are rounded to bf16.  seqlens (int32 [B] on the device):
    each batch entry's sequence length for the key mean."""
    B, N, H, D = x.shape
    rope_dim = 0
    if rope is not None:
        assert rope.dtype == torch.float32 and rope.dim() == 3 and rope.shape[0] == N and rope.shape[2] == 2
        rope = rope.contiguous()
        rope_dim = 2 * rope.shape[1]
    if rms_gain is not None:
        assert rms_gain.dtype == torch.float32 and rms_gain.shape == (D,)
        rms_gain = rms_gain.contiguous()
    out = MX.empty(B, N, H, D, x.device, which, amax=amax)
    mean = torch.empty((B, H, D), dtype=torch.float32, device=x.device) if center else None
    if seqlens is not None:
        assert seqlens.dtype == torch.int32 and seqlens.shape == (B,)
    opt = _Producer(float(prescale), int(bool(center)), _ptr(mean).value, _ptr(rms_gain).value, float(rms_eps),
                    _ptr(rope).value, int(rope_lo), int(rope_dim), _ptr(seqlens).value)
    need = ctypes.c_size_t(0)
    _check("attn_fp8_producer_workspace_size",
           lib().attn_fp8_producer_workspace_size(B, N, H, D, ctypes.byref(opt), ctypes.byref(need)))
    ws = torch.empty(need.value, dtype=torch.uint8, device=x.device) if need.value else None
    m = out.c()
    _check("attn_fp8_quantize_producer",
           lib().attn_fp8_quantize_producer(_ptr(x), _dtype_code(x.dtype), B, N, H, D, _strides_bnh(x),
                                            ctypes.byref(opt), _ptr(ws), need.value, ctypes.byref(m), which,
                                            _ptr(nonfinite), _stream(x.device)))
    return out, mean


def attn_fp8_fwd(p: Problem, q: MX, k: MX, v: MX, o_dtype=torch.bfloat16, o: torch.Tensor | None = None,
                 lse: torch.Tensor | None = None):
    dev = q.code_row.device
    if o is None:
        o = torch.empty((p.batch, p.seqlen, p.heads_q, p.dim_v), dtype=o_dtype, device=dev)
    if lse is None:
        lse = torch.empty((p.batch, p.heads_q, p.seqlen), dtype=torch.float32, device=dev)
    pc, qc, kc, vc = p.c(), q.c(), k.c(), v.c()
    _check("attn_fp8_fwd", lib().attn_fp8_fwd(ctypes.byref(pc), ctypes.byref(qc), ctypes.byref(kc), ctypes.byref(vc),
                                              _ptr(o), _dtype_code(o.dtype), _strides_bnh(o), _ptr(lse),
                                              _stream(dev)))
    return o, lse


def _opt_mx(m):
    return ctypes.byref(m.c()) if m is not None else None


def attn_fp8_delta(p: Problem, mode: int, q: MX | None = None, k: MX | None = None, v: MX | None = None,
                   dout: MX | None = None, lse=None, dout_raw=None, o=None, delta: torch.Tensor | None = None):
    dev = (q.code_row if q is not None else dout_raw).device
    if delta is None:
        delta = torch.empty((p.batch, p.heads_q, p.seqlen, 2), dtype=torch.float32, device=dev)
    pc = p.c()
    mxs = [m.c() if m is not None else None for m in (q, k, v, dout)]
    refs = [ctypes.byref(m) if m is not None else None for m in mxs]
    ds = _strides_bnh(dout_raw) if dout_raw is not None else None
    os_ = _strides_bnh(o) if o is not None else None
    _check("attn_fp8_delta", lib().attn_fp8_delta(
        ctypes.byref(pc), mode, *refs, _ptr(lse), _ptr(dout_raw),
        _dtype_code(dout_raw.dtype) if dout_raw is not None else 0, ds, _ptr(o),
        _dtype_code(o.dtype) if o is not None else 0, os_, _ptr(delta), _stream(dev)))
    return delta


def attn_fp8_bwd_workspace_size(p: Problem) -> int:
    n = ctypes.c_size_t(0)
    pc = p.c()
    _check("attn_fp8_bwd_workspace_size", lib().attn_fp8_bwd_workspace_size(ctypes.byref(pc), ctypes.byref(n)))
    return n.value


def attn_fp8_bwd(p: Problem, mode: int, q: MX, k: MX, v: MX, dout: MX, lse, dout_raw=None, o=None,
                 delta_in=None, grad_dtype=torch.bfloat16, rowstats: bool = False, workspace=None, out=None,
                 main_events=None):
    """Returns (dq, dk, dv, rowstats or None).  main_events: optional pair of
    raw hipEvent_t handles recorded around the main backward kernel."""
    dev = q.code_row.device
    if out is None:
        dq = torch.empty((p.batch, p.seqlen, p.heads_q, p.dim_qk), dtype=grad_dtype, device=dev)
        dk = torch.empty((p.batch, p.nk, p.heads_kv, p.dim_qk), dtype=grad_dtype, device=dev)
        dv = torch.empty((p.batch, p.nk, p.heads_kv, p.dim_v), dtype=grad_dtype, device=dev)
    else:
        dq, dk, dv = out
    ws_bytes = attn_fp8_bwd_workspace_size(p)
    if workspace is None:
        workspace = torch.empty(max(ws_bytes, 256), dtype=torch.uint8, device=dev)
    rs = torch.zeros((p.batch, p.heads_q, p.seqlen, ROWSTATS), dtype=torch.float64, device=dev) if rowstats else None
    pc = p.c()
    mxs = [m.c() for m in (q, k, v, dout)]
    ds = _strides_bnh(dout_raw) if dout_raw is not None else None
    os_ = _strides_bnh(o) if o is not None else None
    _check("attn_fp8_bwd", lib().attn_fp8_bwd(
        ctypes.byref(pc), mode, *[ctypes.byref(m) for m in mxs], _ptr(lse), _ptr(dout_raw),
        _dtype_code(dout_raw.dtype) if dout_raw is not None else 0, ds, _ptr(o),
        _dtype_code(o.dtype) if o is not None else 0, os_, _ptr(delta_in), _ptr(dq), _ptr(dk), _ptr(dv),
        _dtype_code(dq.dtype), _strides_bnh(dq), _strides_bnh(dk), _strides_bnh(dv), _ptr(workspace),
        workspace.numel() * workspace.element_size(), _ptr(rs),
        (ctypes.c_void_p * 2)(*main_events) if main_events is not None else None, _stream(dev)))
    return dq, dk, dv, rs


def attn_fp8_bwd_protected_dp(p: Problem, q: MX, k: MX, dout: MX, lse, dout_raw, v_raw, o=None, delta_in=None,
                              grad_dtype=torch.bfloat16, rowstats: bool = False, workspace=None, out=None):
    """The protected-dP backward (dP from the BF16 dout_raw and v_raw, the
    stale correction from dout_raw and o, or delta_in); p.flags must hold
    FLAG_PROTECTED_DP.  Returns (dq, dk, dv, rowstats or None)."""
    dev = q.code_row.device
    if out is None:
        dq = torch.empty((p.batch, p.seqlen, p.heads_q, p.dim_qk), dtype=grad_dtype, device=dev)
        dk = torch.empty((p.batch, p.nk, p.heads_kv, p.dim_qk), dtype=grad_dtype, device=dev)
        dv = torch.empty((p.batch, p.nk, p.heads_kv, p.dim_v), dtype=grad_dtype, device=dev)
    else:
        dq, dk, dv = out
    ws_bytes = attn_fp8_bwd_workspace_size(p)
    if workspace is None:
        workspace = torch.empty(max(ws_bytes, 256), dtype=torch.uint8, device=dev)
    rs = torch.zeros((p.batch, p.heads_q, p.seqlen, ROWSTATS), dtype=torch.float64, device=dev) if rowstats else None
    pc = p.c()
    mxs = [m.c() for m in (q, k, dout)]
    os_ = _strides_bnh(o) if o is not None else None
    _check("attn_fp8_bwd_protected_dp", lib().attn_fp8_bwd_protected_dp(
        ctypes.byref(pc), *[ctypes.byref(m) for m in mxs], _ptr(lse), _ptr(dout_raw), _dtype_code(dout_raw.dtype),
        _strides_bnh(dout_raw), _ptr(v_raw), _dtype_code(v_raw.dtype), _strides_bnh(v_raw), _ptr(o),
        _dtype_code(o.dtype) if o is not None else 0, os_, _ptr(delta_in), _ptr(dq), _ptr(dk), _ptr(dv),
        _dtype_code(dq.dtype), _strides_bnh(dq), _strides_bnh(dk), _strides_bnh(dv), _ptr(workspace),
        workspace.numel() * workspace.element_size(), _ptr(rs), _stream(dev)))
    return dq, dk, dv, rs


def attn_fp8_bwd_noalloc(p: Problem, mode: int, q: MX, k: MX, v: MX, dout: MX, lse, dout_raw=None, o=None,
                         delta_in=None, grad_dtype=torch.bfloat16, rowstats: bool = False, out=None):
    """attn_fp8_bwd on the library's own scratch (no workspace argument; the
    library allocates nothing for it).  Returns (dq, dk, dv, rowstats or None);
    the output tensors are allocated here unless given in `out`."""
    dev = q.code_row.device
    if out is None:
        dq = torch.empty((p.batch, p.seqlen, p.heads_q, p.dim_qk), dtype=grad_dtype, device=dev)
        dk = torch.empty((p.batch, p.nk, p.heads_kv, p.dim_qk), dtype=grad_dtype, device=dev)
        dv = torch.empty((p.batch, p.nk, p.heads_kv, p.dim_v), dtype=grad_dtype, device=dev)
    else:
        dq, dk, dv = out
    rs = torch.zeros((p.batch, p.heads_q, p.seqlen, ROWSTATS), dtype=torch.float64, device=dev) if rowstats else None
    pc = p.c()
    mxs = [m.c() for m in (q, k, v, dout)]
    ds = _strides_bnh(dout_raw) if dout_raw is not None else None
    os_ = _strides_bnh(o) if o is not None else None
    _check("attn_fp8_bwd_noalloc", lib().attn_fp8_bwd_noalloc(
        ctypes.byref(pc), mode, *[ctypes.byref(m) for m in mxs], _ptr(lse), _ptr(dout_raw),
        _dtype_code(dout_raw.dtype) if dout_raw is not None else 0, ds, _ptr(o),
        _dtype_code(o.dtype) if o is not None else 0, os_, _ptr(delta_in), _ptr(dq), _ptr(dk), _ptr(dv),
        _dtype_code(dq.dtype), _strides_bnh(dq), _strides_bnh(dk), _strides_bnh(dv), _ptr(rs), None,
        _stream(dev)))
    return dq, dk, dv, rs
