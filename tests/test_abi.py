"""CPU checks of the C ABI: the library loads, exports every function that
include/attn_fp8.h declares, and rejects invalid arguments on the host
without launching anything (these calls never reach the GPU)."""
import ctypes
import os
import re

import pytest

import paper_2609_37852_amd as pk
from paper_2609_37852_amd import binding as bd

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared():
    txt = open(os.path.join(ROOT, "include", "attn_fp8.h")).read()
    return sorted(set(re.findall(r"^(?:int|const char\*|size_t)\s+(attn_fp8_\w+)\(", txt, re.M)))


def test_exports_every_declared_symbol():
    L = pk.lib()
    names = _declared()
    assert set(names) == set(bd.EXPORTS), names
    for n in names:
        assert hasattr(L, n)


def _prob(**kw):
    d = dict(batch=1, seqlen=128, heads_q=2, heads_kv=2, dim_qk=128, dim_v=128, softmax_scale=0.088)
    d.update(kw)
    return pk.Problem(**d)


def _fake_mx(addr=4096):
    return bd._MX(addr, addr, addr, addr, None)


@pytest.mark.parametrize("kw,code", [
    (dict(dim_qk=96, dim_v=96), -2), (dict(dim_qk=128, dim_v=64), -2), (dict(seqlen=100), -2),
    (dict(heads_q=3, heads_kv=2), -2), (dict(causal=2), -1), (dict(softmax_scale=float("nan")), -1),
    # the causal mask needs equal lengths; key lengths in blocks of 32; no keys without queries
    (dict(seqlen_kv=256), -2), (dict(causal=0, seqlen_kv=100), -2), (dict(causal=0, seqlen_kv=-32), -1),
    (dict(causal=0, seqlen=0, seqlen_kv=64), -2), (dict(causal=0, seqlen_kv=(1 << 30) + 32), -2),
    (dict(causal=0, batch=512, heads_q=64, heads_kv=64, seqlen=32, seqlen_kv=1 << 15), -2),
    (dict(seqlen=-32), -1), (dict(heads_kv=0), -1),
    # one launch dimension holds fewer than 2^32 work-items: B Hq N < 2^31, B Hkv N < 2^30
    (dict(batch=1024, heads_q=64, heads_kv=64, seqlen=1 << 15), -2),
    (dict(batch=512, heads_q=64, heads_kv=64, seqlen=1 << 15), -2),
    # one GQA group's operands within 32-bit buffer offsets: (Hq / Hkv) N D < 2^32
    (dict(heads_q=64, heads_kv=1, seqlen=1 << 20), -2)])
def test_fwd_rejects_bad_problem(kw, code):
    L = pk.lib()
    p = _prob(**kw).c()
    m = _fake_mx()
    st = bd._I64x3(128 * 2 * 128, 2 * 128, 128)
    rc = L.attn_fp8_fwd(ctypes.byref(p), ctypes.byref(m), ctypes.byref(m), ctypes.byref(m), ctypes.c_void_p(4096),
                        1, st, ctypes.c_void_p(4096), None)
    assert rc == code, pk.last_error()
    assert pk.last_error()


def test_null_alignment_and_workspace_errors():
    L = pk.lib()
    p = _prob().c()
    m = _fake_mx()
    st = bd._I64x3(128 * 2 * 128, 2 * 128, 128)
    # NULL output
    assert L.attn_fp8_fwd(ctypes.byref(p), ctypes.byref(m), ctypes.byref(m), ctypes.byref(m), None, 1, st,
                          ctypes.c_void_p(4096), None) == -1
    # misaligned operand
    bad = _fake_mx(4097)
    assert L.attn_fp8_fwd(ctypes.byref(p), ctypes.byref(bad), ctypes.byref(m), ctypes.byref(m),
                          ctypes.c_void_p(4096), 1, st, ctypes.c_void_p(4096), None) == -3
    # stride not a multiple of 16 bytes
    st_bad = bd._I64x3(128 * 2 * 128, 2 * 128 + 1, 128)
    assert L.attn_fp8_fwd(ctypes.byref(p), ctypes.byref(m), ctypes.byref(m), ctypes.byref(m),
                          ctypes.c_void_p(4096), 1, st_bad, ctypes.c_void_p(4096), None) == -3
    # bad dtype, bad delta mode
    assert L.attn_fp8_fwd(ctypes.byref(p), ctypes.byref(m), ctypes.byref(m), ctypes.byref(m),
                          ctypes.c_void_p(4096), 7, st, ctypes.c_void_p(4096), None) == -1
    assert L.attn_fp8_delta(ctypes.byref(p), 5, ctypes.byref(m), ctypes.byref(m), ctypes.byref(m),
                            ctypes.byref(m), ctypes.c_void_p(4096), None, 1, None, None, 1, None,
                            ctypes.c_void_p(4096), None) == -1
    # workspace too small / misaligned
    n = ctypes.c_size_t(0)
    assert L.attn_fp8_bwd_workspace_size(ctypes.byref(p), ctypes.byref(n)) == 0
    # stored dQ operand units (2 KB) and exponents (2 B, padded to 256) for 4 query blocks per head
    # (1 + 1 + 2 + 2 units), delta, per-query records, per-tile Q/dO col scales, per-tile K col scales
    assert n.value == (2 * 6 * 2048 + 256 + 2 * 128 * 2 * 4 + 2 * 128 * 4 * 4 + 2 * 2 * 2 * (128 + 128)
                       + 256 * ((p.heads_kv * 2 * 2 * 128 + 255) // 256))
    args = [ctypes.byref(p), 0] + [ctypes.byref(m)] * 4 + [ctypes.c_void_p(4096), None, 1, None, None, 1, None,
                                                           None] + [ctypes.c_void_p(4096)] * 3 + [1, st, st, st]
    assert L.attn_fp8_bwd(*args, ctypes.c_void_p(4096), ctypes.c_size_t(n.value - 1), None, None, None) == -4
    assert L.attn_fp8_bwd(*args, ctypes.c_void_p(4096 + 16), ctypes.c_size_t(n.value), None, None, None) == -4
    # the cast dump needs the row statistics and 16-byte alignment
    p.cast_dump = 4096
    assert L.attn_fp8_bwd(*args, ctypes.c_void_p(4096), ctypes.c_size_t(n.value), None, None, None) == -1
    assert "rowstats" in pk.last_error()
    p.cast_dump = 4096 + 4
    assert L.attn_fp8_bwd(*args, ctypes.c_void_p(4096), ctypes.c_size_t(n.value), ctypes.c_void_p(4096),
                          None, None) == -3
    p.cast_dump = None


def test_quantize_rejects_bad_args():
    L = pk.lib()
    m = _fake_mx()
    st = bd._I64x3(64 * 64, 64, 64)
    q = lambda *a: L.attn_fp8_quantize(*a)
    assert q(ctypes.c_void_p(4096), 1, 1, 64, 1, 96, st, ctypes.byref(m), 3, None, None) == -2   # D
    assert q(ctypes.c_void_p(4096), 1, 1, 40, 1, 64, st, ctypes.byref(m), 3, None, None) == -2   # N % 32
    assert q(ctypes.c_void_p(4096), 3, 1, 64, 1, 64, st, ctypes.byref(m), 3, None, None) == -1   # dtype
    assert q(ctypes.c_void_p(4096), 1, 1, 64, 1, 64, st, ctypes.byref(m), 0, None, None) == -1   # which
    assert q(None, 1, 1, 64, 1, 64, st, ctypes.byref(m), 3, None, None) == -1
    st_bad = bd._I64x3(64 * 64, 63, 64)
    assert q(ctypes.c_void_p(4096), 1, 1, 64, 1, 64, st_bad, ctypes.byref(m), 3, None, None) == -3
    # empty problems are valid and launch nothing
    assert q(ctypes.c_void_p(4096), 1, 0, 64, 1, 64, st, ctypes.byref(m), 3, None, None) == 0
    assert q(ctypes.c_void_p(4096), 1, 1, 0, 1, 64, st, ctypes.byref(m), 3, None, None) == 0


def test_empty_problem_is_a_noop():
    L = pk.lib()
    p = _prob(seqlen=0).c()
    m = _fake_mx()
    st = bd._I64x3(0, 256, 128)
    assert L.attn_fp8_fwd(ctypes.byref(p), ctypes.byref(m), ctypes.byref(m), ctypes.byref(m), ctypes.c_void_p(4096),
                          1, st, ctypes.c_void_p(4096), None) == 0


def test_package_exports_binding_names():
    """Every public name of the binding that the tests and the benchmark use
    is re-exported by the package."""
    for name in pk.__all__:
        assert hasattr(pk, name), name
    for name in ("ROWSTATS", "RS_SUM_DS", "RS_SUMABS_DS", "RS_SUM_DSCAST", "RS_MAXABS_DS", "RS_SUMABS_DSCAST",
                 "RS_MAX_PDP", "RS_SUM_PCAST"):
        assert getattr(pk, name) == getattr(bd, name)
    assert pk.ROWSTATS == 7 and sorted(getattr(bd, n) for n in dir(bd) if n.startswith("RS_")) == list(range(7))


def test_noalloc_rejects_oversized_problem_on_the_host():
    """attn_fp8_bwd_noalloc checks the scratch need before touching the
    device: an oversized problem fails with EUNSUPPORTED and a message."""
    L = pk.lib()
    p = _prob(batch=4, seqlen=8192, heads_q=16, heads_kv=4).c()
    m = _fake_mx()
    st = bd._I64x3(128 * 2 * 128, 2 * 128, 128)
    rc = L.attn_fp8_bwd_noalloc(ctypes.byref(p), 0, *[ctypes.byref(m)] * 4, ctypes.c_void_p(4096), None, 1, None,
                                None, 1, None, None, *[ctypes.c_void_p(4096)] * 3, 1, st, st, st, None, None, None)
    assert rc == -2 and "scratch" in pk.last_error()


def _opt(**kw):
    d = dict(prescale=1.0, center=0, channel_mean=None, rms_gain=None, rms_eps=1e-6, rope_cs=None, rope_lo=0,
             rope_dim=0, seqlens=None)
    d.update(kw)
    return bd._Producer(**d)


def test_producer_rejects_bad_arguments():
    L = pk.lib()
    m = _fake_mx()
    st = bd._I64x3(64 * 64, 64, 64)
    args = (ctypes.c_void_p(4096), 1, 1, 64, 1, 64, st)
    vp = ctypes.c_void_p(4096).value
    ws = (ctypes.c_void_p(4096), 1 << 20)

    def call(opt, w=ws):
        return L.attn_fp8_quantize_producer(*args, ctypes.byref(opt) if opt is not None else None, *w,
                                            ctypes.byref(m), 3, None, None)
    # (only rejected calls: the pointers here are placeholders)
    assert call(None) == -1
    assert call(_opt(prescale=float("nan"))) == -1
    assert call(_opt(prescale=0.0)) == -1
    assert call(_opt(center=2, channel_mean=vp)) == -1
    # centering needs the mean output, and a workspace for its partial sums
    assert call(_opt(center=1)) == -1
    assert call(_opt(center=1, channel_mean=vp), (None, 0)) == -4
    assert call(_opt(center=1, channel_mean=vp), (ctypes.c_void_p(4096), 255)) == -4
    assert call(_opt(center=1, channel_mean=vp), (ctypes.c_void_p(4096 + 16), 1 << 20)) == -4
    # the norm: finite non-negative eps, aligned gain, a workspace for the row scales
    assert call(_opt(rms_gain=vp, rms_eps=-1.0)) == -1
    assert call(_opt(rms_gain=vp, rms_eps=float("inf"))) == -1
    assert call(_opt(rms_gain=4100)) == -3
    assert call(_opt(rms_gain=vp), (None, 0)) == -4
    # rotary channels: 32-aligned, inside D, with a table
    for lo, R, code in ((0, 48, -2), (16, 32, -2), (32, 64, -2), (-32, 32, -1)):
        rc = call(_opt(rope_cs=vp, rope_lo=lo, rope_dim=R))
        assert rc == code, (lo, R, rc, pk.last_error())
    assert call(_opt(rope_dim=32)) == -1
    # the key mean's sequence lengths: int32 alignment
    assert call(_opt(center=1, channel_mean=vp, seqlens=4098)) == -3


def test_producer_workspace_size():
    """Partial sums FP64 [B, H, D, N/32] when centering, then the norm's row
    scales FP32 [B, N, H], each rounded up to 256 bytes; nothing otherwise."""
    L = pk.lib()
    vp = ctypes.c_void_p(4096).value
    n = ctypes.c_size_t(7)

    def size(B, N, H, D, opt):
        rc = L.attn_fp8_producer_workspace_size(B, N, H, D, ctypes.byref(opt), ctypes.byref(n))
        return rc, n.value
    r256 = lambda b: (b + 255) // 256 * 256
    assert size(2, 96, 3, 128, _opt()) == (0, 0)
    assert size(2, 96, 3, 128, _opt(prescale=0.3, rope_cs=vp, rope_dim=64)) == (0, 0)
    assert size(2, 96, 3, 128, _opt(center=1, channel_mean=vp)) == (0, r256(2 * 3 * 128 * 3 * 8))
    assert size(2, 96, 3, 128, _opt(rms_gain=vp)) == (0, r256(2 * 96 * 3 * 4))
    assert size(4, 8192, 4, 128, _opt(center=1, channel_mean=vp, rms_gain=vp)) == \
        (0, 4 * 4 * 128 * 256 * 8 + r256(4 * 8192 * 4 * 4))
    assert size(1, 100, 1, 128, _opt())[0] == -2
    assert size(1, 96, 1, 96, _opt())[0] == -2
    assert size(1, 96, 1, 128, _opt(prescale=0.0))[0] == -1
    assert L.attn_fp8_producer_workspace_size(1, 96, 1, 128, None, ctypes.byref(n)) == -1
    assert L.attn_fp8_producer_workspace_size(1, 96, 1, 128, ctypes.byref(_opt()), None) == -1


def test_workspace_size_without_mask():
    """Stored dQ operand units: causal problems keep the ones up to the
    diagonal, sum over 32-query blocks q of floor(q/2) + 1; without the mask
    every block has ceil(Nk / 64).  The K col scales per 64-key step follow
    the key length."""
    L = pk.lib()
    r256 = lambda x: (x + 255) // 256 * 256

    def ws(**kw):
        p = _prob(**kw).c()
        out = ctypes.c_size_t(0)
        assert L.attn_fp8_bwd_workspace_size(ctypes.byref(p), ctypes.byref(out)) == 0, pk.last_error()
        return out.value

    def expect(B, N, Nk, Hq, Hkv, D, units):
        nt = (N + 63) // 64
        return (r256(B * Hq * units * 2048) + r256(B * Hq * units * 2) + r256(B * Hq * N * 8) +
                r256(B * Hq * nt * 1024) + r256(B * Hq * nt * 4 * D) + r256(B * Hkv * ((Nk + 63) // 64) * 2 * D))
    causal_units = sum(q // 2 + 1 for q in range(128 // 32))
    assert ws() == expect(1, 128, 128, 2, 2, 128, causal_units)
    assert ws(causal=0) == expect(1, 128, 128, 2, 2, 128, 4 * 2)
    assert ws(causal=0, seqlen_kv=320) == expect(1, 128, 320, 2, 2, 128, 4 * 5)
    assert ws(causal=0, seqlen=352, seqlen_kv=96) == expect(1, 352, 96, 2, 2, 128, 11 * 2)


def test_unknown_delta_mode_rejected():
    """Modes 0..3 (matched, stale, consistent dO, compensated matched); others
    are rejected by the correction and by the backward, even with delta_in."""
    L = pk.lib()
    p = _prob().c()
    m = _fake_mx()
    st = bd._I64x3(128 * 2 * 128, 2 * 128, 128)
    vp = ctypes.c_void_p(4096)
    for mode in (-1, 4):
        rc = L.attn_fp8_delta(ctypes.byref(p), mode, ctypes.byref(m), ctypes.byref(m), ctypes.byref(m),
                              ctypes.byref(m), vp, vp, 1, st, vp, 1, st, vp, None)
        assert rc == -1 and "delta_mode" in pk.last_error()
        rc = L.attn_fp8_bwd(ctypes.byref(p), mode, ctypes.byref(m), ctypes.byref(m), ctypes.byref(m),
                            ctypes.byref(m), vp, vp, 1, st, vp, 1, st, vp, vp, vp, vp, 1, st, st, st,
                            ctypes.c_void_p(1 << 20), 1 << 30, None, None, None)
        assert rc == -1 and "delta_mode" in pk.last_error()
    assert pk.DELTA_MATCHING_COMPENSATED == 3


def test_seqlens_checks():
    """Per-sequence lengths: no key lengths under the mask (the key length is
    the query length there), 4-byte aligned arrays."""
    L = pk.lib()
    m = _fake_mx()
    st = bd._I64x3(128 * 2 * 128, 2 * 128, 128)

    def fwd(**kw):
        p = _prob(**{k: v for k, v in kw.items() if not k.startswith("seqlens")}).c()
        p.seqlens_q = kw.get("seqlens_q")
        p.seqlens_kv = kw.get("seqlens_kv")
        return L.attn_fp8_fwd(ctypes.byref(p), ctypes.byref(m), ctypes.byref(m), ctypes.byref(m),
                              ctypes.c_void_p(4096), 1, st, ctypes.c_void_p(4096), None)
    assert fwd(seqlens_kv=4096) == -1
    assert fwd(seqlens_q=4096, seqlens_kv=4096) == -1
    assert fwd(seqlens_q=4098) == -3
    assert fwd(causal=0, seqlens_kv=4094) == -3
    n = ctypes.c_size_t(0)
    p = _prob(causal=0).c()
    p.seqlens_q = 4096
    p.seqlens_kv = 8192
    # the workspace follows the layouts, not the lengths
    assert L.attn_fp8_bwd_workspace_size(ctypes.byref(p), ctypes.byref(n)) == 0
    ref = ctypes.c_size_t(0)
    assert L.attn_fp8_bwd_workspace_size(ctypes.byref(_prob(causal=0).c()), ctypes.byref(ref)) == 0
    assert n.value == ref.value > 0


def test_isolate3_combinations():
    """Three isolated channels combine with none of the other numerics
    variants, nor with the compensated correction."""
    L = pk.lib()
    m = _fake_mx()
    st = bd._I64x3(128 * 2 * 128, 2 * 128, 128)

    def fwd(flags):
        p = _prob(flags=flags).c()
        return L.attn_fp8_fwd(ctypes.byref(p), ctypes.byref(m), ctypes.byref(m), ctypes.byref(m),
                              ctypes.c_void_p(4096), 1, st, ctypes.c_void_p(4096), None)
    assert fwd(pk.FLAG_ISOLATE3 | pk.FLAG_PBWD_BLOCK_SCALED) == -2
    assert fwd(pk.FLAG_ISOLATE3 | pk.FLAG_PROTECTED_DP) == -2
    assert fwd(8) == -1
    p = _prob(flags=pk.FLAG_ISOLATE3).c()
    # (every call here fails a later check too, so none could launch: no LSE
    # for the correction, a one-byte workspace for the backward)
    rc = L.attn_fp8_delta(ctypes.byref(p), pk.DELTA_MATCHING_COMPENSATED, *[ctypes.byref(m)] * 4,
                          None, None, 1, None, None, 1, None, ctypes.c_void_p(4096), None)
    assert rc == -2 and "isolated" in pk.last_error()
    rc = L.attn_fp8_bwd(ctypes.byref(p), pk.DELTA_MATCHING_COMPENSATED, *[ctypes.byref(m)] * 4,
                        ctypes.c_void_p(4096), None, 1, None, None, 1, None, ctypes.c_void_p(4096),
                        *[ctypes.c_void_p(4096)] * 3, 1, st, st, st, ctypes.c_void_p(4096), 1, None, None,
                        None)
    assert rc == -2 and "isolated" in pk.last_error()
