#!/usr/bin/env python3
"""Benchmark of the FP8 attention hot path on one MI355X.

One step = the whole hot path over one batch of the causal GQA d=128 8K
workload (B=4, 16 query heads sharing 4 KV heads, N=8192, bf16 inputs with one
outlier channel x20): quantize Q, K, V, dO (both MX copies) -> forward ->
matched correction -> backward (dQ, dK, dV).  Inputs are resident in HBM
before the timed region.

Throughput uses the paper's accounting (App. C.2): credited FLOPs are
B*Hq*N^2*(dqk+dv) for the forward and B*Hq*N^2*(3 dqk + 2 dv) for the
backward; the correction pass and the quantizer earn no credit.

Prints one JSON line.  Besides the contract's fields (value = credited
TFLOP/s of the timed steps), it carries per-kernel times, the HBM rates of
the quantizer and the saved-output corrections, the main backward kernel's
roofline, the paper's own timing protocol (App. C.2: clock warm-up, five
interleaved rounds of the median of 20 timings after 5 warm-up calls, mean
and standard error, pre-quantized inputs) for the matched and the stale
backward, a whole step with the stale correction, the cost of the
compensated matched correction, the protected-dP variant, the block-scaled backward probability
operand, a padded batch of sequences of their own lengths, the input producer, the same workload
without the causal mask, the d = 256 workload, and the oracle's CPU rate.
`--gpus N` with N > 1 exits: this benchmark measures a single GPU.
"""
from __future__ import annotations

import argparse
import ctypes
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_FP8_TFLOPS = 5000.0      # MI355X dense FP8 MFMA
PEAK_HBM_GBS = 8000.0

# Measured HBM bytes of the main backward kernel (rocprofv3 FETCH_SIZE and
# WRITE_SIZE, calibrated with a plain copy kernel), valid only for the kernel
# sources it was taken on.
TRAFFIC_SUMMARY = os.path.join(ROOT, "profiles", "bwd_kernel_gqa_d128_8k_traffic.md")
BWD_SOURCES = ("bwd_main.hpp", "bwd_main_causal_v0.hip", "dma.hpp", "common.hpp", "tiles.hpp", "kernels.hpp")


def bwd_sources_sha256():
    import hashlib
    h = hashlib.sha256()
    for f in BWD_SOURCES:
        with open(os.path.join(ROOT, "paper_2609_37852_amd", "csrc", f), "rb") as fh:
            h.update(f.encode() + b"\0" + fh.read())
    return h.hexdigest()


def read_traffic(path):
    """bytes_per_launch from a traffic summary, or None if it is absent or was
    measured on other kernel sources."""
    if not path or not os.path.exists(path):
        return None
    fields = {}
    for line in open(path):
        if line.startswith("- ") and ":" in line:
            k, v = line[2:].split(":", 1)
            fields[k.strip()] = v.strip().strip("`")
    if fields.get("kernel_sources_sha256") != bwd_sources_sha256():
        return None
    return int(fields["bytes_per_launch"])


def write_traffic_summary(fetch_csv, write_csv, out, calib_mib):
    """Calibrated HBM bytes per launch of bwd_kernel<128,128> from two
    rocprofv3 --pmc runs (FETCH_SIZE, WRITE_SIZE in KiB per dispatch) of
    `bench.py --copy-calibration MIB`, whose negate kernel reads and writes
    MIB MiB each."""
    import csv

    def per_kernel(path, counter):
        vals = {"bwd": [], "copy": []}
        for r in csv.DictReader(open(path)):
            if r["Counter_Name"] != counter:
                continue
            name = r["Kernel_Name"]
            if "bwd_kernel<128, 128, false, true, 0>" in name:
                vals["bwd"].append(float(r["Counter_Value"]))
            elif "neg" in name:
                vals["copy"].append(float(r["Counter_Value"]))
        if not vals["bwd"] or not vals["copy"]:
            raise RuntimeError(f"{path}: no {counter} rows for the backward or the calibration kernel")
        return float(np.mean(vals["bwd"])), float(np.mean(vals["copy"]))

    calib = calib_mib << 20
    fb, fc = per_kernel(fetch_csv, "FETCH_SIZE")
    wb, wc = per_kernel(write_csv, "WRITE_SIZE")
    f_scale, w_scale = calib / (fc * 1024), calib / (wc * 1024)
    fetch, write = fb * 1024 * f_scale, wb * 1024 * w_scale
    total = int(round(fetch + write))
    # the profiler's output directories are those of the CSVs given here
    fdir_f, fdir_w = os.path.relpath(os.path.dirname(fetch_csv), ROOT), os.path.relpath(os.path.dirname(write_csv), ROOT)
    text = f"""# HBM traffic: bwd_kernel<128,128> on gqa_d128_8k (B=4, N=8192, Hq=16, Hkv=4, d=128, causal)

Commands (MI355X, ROCm 7.2, repository root; `cd /tmp && export TMPDIR=/tmp` first):

```
rocprofv3 --kernel-include-regex "bwd_kernel|neg" --pmc FETCH_SIZE -d {fdir_f} -o run --output-format csv -- python -u bench.py --steps 2 --warmup 1 --no-cpu-baseline --no-protocol --copy-calibration {calib_mib}
rocprofv3 --kernel-include-regex "bwd_kernel|neg" --pmc WRITE_SIZE -d {fdir_w} -o run --output-format csv -- python -u bench.py --steps 2 --warmup 1 --no-cpu-baseline --no-protocol --copy-calibration {calib_mib}
python bench.py --traffic-summary {os.path.relpath(fetch_csv, ROOT)} {os.path.relpath(write_csv, ROOT)} --copy-calibration {calib_mib}
```

The calibration kernel is a float32 negate over {calib} bytes (it reads and writes
{calib} bytes once each).

| counter | bwd_kernel (KiB / dispatch) | calibration (KiB) | scale | bwd bytes / launch |
|---|---:|---:|---:|---:|
| FETCH_SIZE | {fb:.0f} | {fc:.0f} | {f_scale:.4f} | {fetch:.4e} |
| WRITE_SIZE | {wb:.0f} | {wc:.0f} | {w_scale:.4f} | {write:.4e} |

Algorithmic bytes per launch, for comparison: written, the dS' units for the dQ pass
(one byte per causal score, B Hq N^2 / 2 = 2.15e9), their exponents (2 bytes per unit,
2.1e6) and dK, dV (bf16, 6.7e7); read once, the row and col codes of Q and dO (B Hq N 2
(dqk + dv) = 2.7e8), the K and V row codes (3.4e7), scales and per-query records (about
3e7): 2.22e9 written and 3.3e8 read.  Measured / algorithmic: reads {fetch / 3.3e8:.2f}x (query
tiles fetched again after leaving the L2), writes {write / 2.22e9:.2f}x.

Machine-read by bench.py (roofline.traffic; null when the kernel sources differ):

- bytes_per_launch: {total}
- kernel_sources_sha256: `{bwd_sources_sha256()}`
"""
    with open(out, "w") as fh:
        fh.write(text)
    print(text)


class HipEvents:
    """Raw HIP events (timing enabled) via the runtime's C API."""

    def __init__(self):
        self.hip = ctypes.CDLL("libamdhip64.so")
        self.hip.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p, ctypes.c_void_p]

    def create(self, n):
        evs = []
        for _ in range(n):
            e = ctypes.c_void_p()
            rc = self.hip.hipEventCreate(ctypes.byref(e))
            if rc != 0:
                raise RuntimeError(f"hipEventCreate failed ({rc})")
            evs.append(e)
        return evs

    def record(self, e, stream):
        rc = self.hip.hipEventRecord(e, ctypes.c_void_p(stream))
        if rc != 0:
            raise RuntimeError(f"hipEventRecord failed ({rc})")

    def ms(self, a, b):
        out = ctypes.c_float()
        rc = self.hip.hipEventElapsedTime(ctypes.byref(out), a, b)
        if rc != 0:
            raise RuntimeError(f"hipEventElapsedTime failed ({rc})")
        return float(out.value)


class Runner:
    """One workload resident on the GPU: inputs, MX copies, outputs and the
    backward workspace allocated once; step() runs the whole hot path
    (quantize Q, K, V, dO -> forward -> correction -> backward) on the
    current stream."""

    def __init__(self, w, ev):
        import torch
        import paper_2609_37852_amd as pk
        from paper_2609_37852_amd import synth
        self.pk, self.torch, self.w, self.ev = pk, torch, w, ev
        d = synth.generate(w, seed=0)
        dev = torch.device("cuda:0")
        tdt = torch.bfloat16 if w.dtype == "bf16" else torch.float32
        self.q, self.k, self.v, self.do = (torch.from_numpy(d[n]).to(tdt).to(dev) for n in ("q", "k", "v", "do"))
        del d
        self.p = pk.Problem(w.B, w.N, w.Hq, w.Hkv, w.Dqk, w.Dv, float(np.float32(w.tau)), causal=int(w.causal),
                            seqlen_kv=w.Nk)
        # channel maxima only where a kernel reads them: Q and K (the isolated score channel)
        self.mq, self.mk, self.mv, self.mdo = (pk.MX.empty(*t.shape, dev, amax=a) for t, a in
                                               ((self.q, True), (self.k, True), (self.v, False), (self.do, False)))
        self.o = torch.empty((w.B, w.N, w.Hq, w.Dv), dtype=torch.bfloat16, device=dev)
        self.lse = torch.empty((w.B, w.Hq, w.N), dtype=torch.float32, device=dev)
        self.delta = torch.empty((w.B, w.Hq, w.N, 2), dtype=torch.float32, device=dev)
        self.grads = (torch.empty((w.B, w.N, w.Hq, w.Dqk), dtype=torch.bfloat16, device=dev),
                      torch.empty((w.B, w.nk, w.Hkv, w.Dqk), dtype=torch.bfloat16, device=dev),
                      torch.empty((w.B, w.nk, w.Hkv, w.Dv), dtype=torch.bfloat16, device=dev))
        self.ws = torch.empty(pk.attn_fp8_bwd_workspace_size(self.p), dtype=torch.uint8, device=dev)
        self.L = pk.lib()
        self.stream = torch.cuda.current_stream(dev).cuda_stream

    def quantize(self):
        for x, m in ((self.q, self.mq), (self.k, self.mk), (self.v, self.mv), (self.do, self.mdo)):
            mc = m.c()
            st = (ctypes.c_int64 * 3)(x.stride(0), x.stride(1), x.stride(2))
            rc = self.L.attn_fp8_quantize(ctypes.c_void_p(x.data_ptr()), 1 if x.dtype == self.torch.bfloat16 else 0,
                                          *x.shape, st, ctypes.byref(mc), 3, None, ctypes.c_void_p(self.stream))
            if rc != 0:
                raise RuntimeError(self.pk.last_error())

    def fwd(self):
        self.pk.attn_fp8_fwd(self.p, self.mq, self.mk, self.mv, o=self.o, lse=self.lse)

    def correction(self, mode):
        self.pk.attn_fp8_delta(self.p, mode, self.mq, self.mk, self.mv, self.mdo, self.lse, self.do, self.o,
                               delta=self.delta)

    def bwd(self, mode, main_events=None):
        self.pk.attn_fp8_bwd(self.p, mode, self.mq, self.mk, self.mv, self.mdo, self.lse, self.do, self.o,
                             delta_in=self.delta, workspace=self.ws, out=self.grads, main_events=main_events)

    def step(self, marks=None, mode=None):
        """marks: 7 events recorded around quantize / fwd / correction / the
        backward call, and (4, 5) around the main backward kernel."""
        mode = self.pk.DELTA_MATCHING if mode is None else mode
        rec = (lambda i: self.ev.record(marks[i], self.stream)) if marks else (lambda i: None)
        rec(0)
        self.quantize()
        rec(1)
        self.fwd()
        rec(2)
        self.correction(mode)
        rec(3)
        self.bwd(mode, main_events=(marks[4].value, marks[5].value) if marks else None)
        rec(6)

    def correction_ms(self, mode, n=3):
        """Correction pass of the given mode, timed within n whole steps."""
        ms_ = [self.ev.create(7) for _ in range(n)]
        for m in ms_:
            self.step(m, mode=mode)
        self.torch.cuda.synchronize()
        return float(np.mean([self.ev.ms(m[2], m[3]) for m in ms_]))

    def breakdown(self, mode, n=10):
        """Mean times of the correction pass, the main backward kernel and
        the whole step over n steps in the given mode (after 3 warm-ups)."""
        for _ in range(3):
            self.step(mode=mode)
        ms_ = [self.ev.create(7) for _ in range(n)]
        for m in ms_:
            self.step(m, mode=mode)
        self.torch.cuda.synchronize()
        avg = lambda a, b: float(np.mean([self.ev.ms(m[a], m[b]) for m in ms_]))
        return {"delta_ms": round(avg(2, 3), 4), "bwd_main_ms": round(avg(4, 5), 4), "step_ms": round(avg(0, 6), 4)}

    def timed(self, fn, warm=5, reps=20):
        """Median of `reps` event timings of fn() after `warm` calls."""
        for _ in range(warm):
            fn()
        evs = [self.ev.create(2) for _ in range(reps)]
        for a, b in evs:
            self.ev.record(a, self.stream)
            fn()
            self.ev.record(b, self.stream)
        self.torch.cuda.synchronize()
        return float(np.median([self.ev.ms(a, b) for a, b in evs]))

    def full_step(self, mode):
        """Whole step (quantize + fwd + correction + bwd) in the given mode:
        median of 20 timings after 5 warm-up steps."""
        ms = self.timed(lambda: self.step(mode=mode))
        f, b = self.w.credited_flops()
        return {"ms": round(ms, 4), "tflops": round((f + b) / (ms * 1e-3) / 1e12, 2),
                "pct_of_fp8_peak": round(100 * (f + b) / (ms * 1e-3) / 1e12 / PEAK_FP8_TFLOPS, 2)}

    def protocol(self, clock_warmup_s, rounds=5):
        """The paper's timing protocol (App. C.2, Timing and accounting): a
        clock warm-up of back-to-back steps, then `rounds` interleaved rounds;
        in each, the forward, forward + matched backward and forward + stale
        backward are each the median of 20 timings after 5 warm-up calls, with
        pre-quantized inputs.  Backward = (forward + backward) - forward.
        Reported as mean and standard error over the rounds."""
        pk = self.pk
        self.quantize()
        t_end = time.perf_counter() + clock_warmup_s
        while time.perf_counter() < t_end:
            self.step()
            self.torch.cuda.synchronize()
        res = {"fwd": [], "fwd_bwd_matched": [], "fwd_bwd_stale": []}
        for _ in range(rounds):
            res["fwd"].append(self.timed(self.fwd))
            for key, mode in (("fwd_bwd_matched", pk.DELTA_MATCHING), ("fwd_bwd_stale", pk.DELTA_STALE_ROWSUM)):
                res[key].append(self.timed(lambda m=mode: (self.fwd(), self.correction(m), self.bwd(m))))
        f, b = self.w.credited_flops()
        fwd = np.array(res["fwd"])
        out = {"rounds": rounds, "timings_per_round": 20, "warmup_calls": 5, "clock_warmup_s": clock_warmup_s}

        def ms_tflops(name, t_ms, flops):
            t_ms = np.asarray(t_ms)
            tf = flops / (t_ms * 1e-3) / 1e12
            se = lambda x: float(np.std(x, ddof=1) / np.sqrt(len(x))) if len(x) > 1 else 0.0
            out[name] = {"ms_mean": round(float(t_ms.mean()), 4), "ms_se": round(se(t_ms), 4),
                         "tflops_mean": round(float(tf.mean()), 2), "tflops_se": round(se(tf), 2)}
        ms_tflops("fwd", fwd, f)
        for mode in ("matched", "stale"):
            fb = np.array(res[f"fwd_bwd_{mode}"])
            ms_tflops(f"bwd_{mode}", fb - fwd, b)
            ms_tflops(f"fwd_bwd_{mode}", fb, f + b)
        ratio = (np.array(res["fwd_bwd_matched"]) - fwd) / (np.array(res["fwd_bwd_stale"]) - fwd) - 1
        out["matched_over_stale_bwd"] = {"mean": round(float(ratio.mean()), 4),
                                         "se": round(float(np.std(ratio, ddof=1) / np.sqrt(rounds)), 4)}
        out["pct_of_fp8_peak_matched"] = round(100 * out["fwd_bwd_matched"]["tflops_mean"] / PEAK_FP8_TFLOPS, 2)
        return out


def protected_dp_line(run):
    """The protected-dP variant (dP from BF16 operands, App. C.4.2) against
    the FP8-dP backward, both with the stale correction: forward +
    correction + backward, each the median of 20 timings after 5 warm-ups,
    pre-quantized inputs."""
    import dataclasses
    import torch
    pk = run.pk
    pp = dataclasses.replace(run.p, flags=pk.FLAG_PROTECTED_DP)
    wsp = torch.empty(pk.attn_fp8_bwd_workspace_size(pp), dtype=torch.uint8, device="cuda:0")
    stale = pk.DELTA_STALE_ROWSUM

    def protected():
        run.fwd()
        run.correction(stale)
        pk.attn_fp8_bwd_protected_dp(pp, run.mq, run.mk, run.mdo, run.lse, run.do, run.v, run.o,
                                     delta_in=run.delta, workspace=wsp, out=run.grads)
    run.quantize()
    t_fwd = run.timed(run.fwd)
    t_prot = run.timed(protected)
    t_stale = run.timed(lambda: (run.fwd(), run.correction(stale), run.bwd(stale)))
    f, b = run.w.credited_flops()
    del wsp
    return {"fwd_bwd_ms": round(t_prot, 4), "bwd_ms": round(t_prot - t_fwd, 4),
            "bwd_tflops": round(b / ((t_prot - t_fwd) * 1e-3) / 1e12, 2),
            "fwd_bwd_stale_fp8dp_ms": round(t_stale, 4),
            "bwd_over_fp8dp_bwd": round((t_prot - t_fwd) / (t_stale - t_fwd) - 1, 4)}


def variants_line(run):
    """The f3/f4 options on the same workload, each the median of 20 timings
    after 5 warm-ups: the block-scaled backward probability operand (matched
    backward call against the default one), three isolated score channels
    (forward + matched correction + backward), a padded batch of sequences of
    their own lengths (forward + matched correction + backward, credited
    with each sequence's own causal FLOPs), and the input producer (query:
    QK normalization, rotary embedding on 64 channels, prescale by tau; key:
    the same with centring instead of the prescale) against the plain
    quantizer."""
    import dataclasses
    import torch
    pk, w = run.pk, run.w
    from paper_2609_37852_amd import synth
    out = {}
    mode = pk.DELTA_MATCHING
    run.quantize()
    run.fwd()
    run.correction(mode)
    pm = dataclasses.replace(run.p, flags=pk.FLAG_PBWD_BLOCK_SCALED)
    t_def = run.timed(lambda: run.bwd(mode))
    t_pmx = run.timed(lambda: pk.attn_fp8_bwd(pm, mode, run.mq, run.mk, run.mv, run.mdo, run.lse, run.do, run.o,
                                              delta_in=run.delta, workspace=run.ws, out=run.grads))
    out["pbwd_block_scaled"] = {"bwd_call_ms": round(t_pmx, 4), "default_bwd_call_ms": round(t_def, 4),
                                "over_default": round(t_pmx / t_def - 1, 4)}
    # three isolated score channels (forward + matched correction + backward)
    pi = dataclasses.replace(run.p, flags=pk.FLAG_ISOLATE3)

    def iso3_step():
        pk.attn_fp8_fwd(pi, run.mq, run.mk, run.mv, o=run.o, lse=run.lse)
        pk.attn_fp8_delta(pi, mode, run.mq, run.mk, run.mv, run.mdo, run.lse, run.do, run.o, delta=run.delta)
        pk.attn_fp8_bwd(pi, mode, run.mq, run.mk, run.mv, run.mdo, run.lse, run.do, run.o, delta_in=run.delta,
                        workspace=run.ws, out=run.grads)
    t_iso = run.timed(iso3_step)
    t_one = run.timed(lambda: (run.fwd(), run.correction(mode), run.bwd(mode)))
    out["isolate3"] = {"fwd_bwd_ms": round(t_iso, 4), "one_channel_fwd_bwd_ms": round(t_one, 4),
                       "over_one_channel": round(t_iso / t_one - 1, 4)}
    # sequences of their own lengths in the padded layout
    lens = [w.N - (w.N // 4) * (b % 4) for b in range(w.B)]
    pv = dataclasses.replace(run.p, seqlens_q=torch.tensor(lens, dtype=torch.int32, device="cuda:0"))

    def varlen_step():
        pk.attn_fp8_fwd(pv, run.mq, run.mk, run.mv, o=run.o, lse=run.lse)
        pk.attn_fp8_delta(pv, mode, run.mq, run.mk, run.mv, run.mdo, run.lse, run.do, run.o, delta=run.delta)
        pk.attn_fp8_bwd(pv, mode, run.mq, run.mk, run.mv, run.mdo, run.lse, run.do, run.o, delta_in=run.delta,
                        workspace=run.ws, out=run.grads)
    t_var = run.timed(varlen_step)
    t_full = run.timed(lambda: (run.fwd(), run.correction(mode), run.bwd(mode)))
    fl = sum(sum(synth.with_shape(w, B=1, N=L).credited_flops()) for L in lens)
    ff = sum(w.credited_flops())
    out["varlen"] = {"seqlens": lens, "fwd_bwd_ms": round(t_var, 4),
                     "tflops": round(fl / (t_var * 1e-3) / 1e12, 2),
                     "full_length_fwd_bwd_ms": round(t_full, 4),
                     "full_length_tflops": round(ff / (t_full * 1e-3) / 1e12, 2)}
    # the input producer
    R = 64
    tab = torch.from_numpy(synth.rope_table(w.N, R, 1e4)).cuda()
    g = torch.ones(w.Dqk, dtype=torch.float32, device="cuda:0")
    t_q = run.timed(lambda: pk.attn_fp8_quantize(run.q))
    t_k = run.timed(lambda: pk.attn_fp8_quantize(run.k))
    t_pq = run.timed(lambda: pk.attn_fp8_quantize_producer(run.q, float(np.float32(w.tau)), False, rope=tab,
                                                           rms_gain=g))
    t_pk = run.timed(lambda: pk.attn_fp8_quantize_producer(run.k, 1.0, True, rope=tab, rms_gain=g))
    bq, bk = 4.0625 * run.q.numel(), 4.0625 * run.k.numel()
    out["producer"] = {"q_ms": round(t_pq, 4), "q_plain_quantize_ms": round(t_q, 4),
                       "k_ms": round(t_pk, 4), "k_plain_quantize_ms": round(t_k, 4),
                       "q_gbs_algorithmic": round(bq / (t_pq * 1e-3) / 1e9, 1),
                       "k_gbs_algorithmic": round(bk / (t_pk * 1e-3) / 1e9, 1)}
    return out


def cpu_baseline(w, d, threads, kv_heads=2):
    """The oracle (FP64 C, OpenMP) timed on the host cores on the first
    `kv_heads` KV groups of batch 0 at the full sequence length."""
    import oracle as orc
    from paper_2609_37852_amd import synth
    hk = min(kv_heads, w.Hkv)
    hq = hk * (w.Hq // w.Hkv)
    sl = dict(q=d["q"][:1, :, :hq], k=d["k"][:1, :, :hk], v=d["v"][:1, :, :hk], do=d["do"][:1, :, :hq])
    ws = synth.with_shape(w, B=1, Hq=hq, Hkv=hk)
    t = time.perf_counter()
    orc.attention_from_inputs(sl["q"], sl["k"], sl["v"], sl["do"], float(np.float32(w.tau)), nthreads=threads)
    dt = time.perf_counter() - t
    f, b = ws.credited_flops()
    fw, bw = w.credited_flops()
    model = "unknown"
    try:
        for ln in open("/proc/cpuinfo"):
            if ln.startswith("model name"):
                model = ln.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    return dict(value=round((f + b) / dt / 1e12, 6), unit="TFLOP/s", cores=threads, kind="oracle",
                cpu_model=model, host_threads=os.cpu_count(),
                sample=f"batch 0, query heads 0..{hq - 1} (KV heads 0..{hk - 1}), N={w.N}: quantize + fwd + "
                       f"matched delta + bwd in FP64, {dt:.1f} s, credited {(f + b) / 1e9:.1f} GFLOP",
                extrapolated_full_workload_s=round(dt * (fw + bw) / (f + b), 1),
                extrapolation="linear in credited FLOP from the sample to the whole workload (not measured)")


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="gqa_d128_8k")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-protocol", action="store_true",
                    help="skip the paper's timing protocol, the stale-mode step and the d = 256 line")
    ap.add_argument("--clock-warmup", type=float, default=3.0,
                    help="seconds of back-to-back steps before the paper's protocol (clock warm-up)")
    ap.add_argument("--diagnostics", action="store_true",
                    help="also report the row-sum and key-gradient diagnostics of the three corrections "
                         "(untimed; five extra backward runs)")
    ap.add_argument("--traffic", default=TRAFFIC_SUMMARY,
                    help="summary with the measured HBM bytes of the bwd kernel (used while its sources match)")
    ap.add_argument("--traffic-summary", nargs=2, metavar=("FETCH_CSV", "WRITE_CSV"),
                    help="write the traffic summary from two rocprofv3 --pmc counter CSVs and exit")
    ap.add_argument("--more-configs", action="store_true",
                    help="also time the MLA d = 192/128 4K and the 64K long-context workloads (whole step, "
                         "matched and stale, and the matched per-kernel split; their inputs take about a "
                         "minute to generate on the host)")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                    help="after the timed steps, copy MIB MiB device-to-device once (a plain copy kernel whose "
                         "FETCH_SIZE / WRITE_SIZE calibrate the HBM counters)")
    args = ap.parse_args()
    if args.traffic_summary:
        write_traffic_summary(*args.traffic_summary, TRAFFIC_SUMMARY, args.copy_calibration or 1024)
        return
    if args.gpus != 1:
        print(f"bench.py measures one GPU; --gpus {args.gpus} is not supported (the hot path runs on a "
              f"single MI355X; the problem shards by (batch, KV head) without communication)", file=sys.stderr)
        sys.exit(2)

    import torch
    import paper_2609_37852_amd as pk
    from paper_2609_37852_amd import synth

    ev = HipEvents()
    w = synth.WORKLOADS[args.workload]
    run = Runner(w, ev)

    for _ in range(args.warmup):
        run.step()
    torch.cuda.synchronize()

    # the contract's timed region: exactly `steps` steps between two events
    marks = [ev.create(7) for _ in range(args.steps)]
    t0, t1 = ev.create(2)
    torch.cuda.synchronize()
    ev.record(t0, run.stream)
    for i in range(args.steps):
        run.step(marks[i])
    ev.record(t1, run.stream)
    torch.cuda.synchronize()
    total_ms = ev.ms(t0, t1)
    ms_per_step = total_ms / args.steps

    def avg(a, b):
        return float(np.mean([ev.ms(m[a], m[b]) for m in marks]))

    t_quant, t_fwd, t_delta = avg(0, 1), avg(1, 2), avg(2, 3)
    t_bwd_main, t_bwd_call = avg(4, 5), avg(3, 6)
    t_delta_stale = run.correction_ms(pk.DELTA_STALE_ROWSUM)
    t_delta_consistent = run.correction_ms(pk.DELTA_CONSISTENT_DO)

    fwd_f, bwd_f = w.credited_flops()
    credited = fwd_f + bwd_f
    value = credited / (ms_per_step * 1e-3) / 1e12
    paper_ms = t_fwd + t_delta + t_bwd_call
    # the main backward kernel computes S, dP, dV and dK over the causal half
    # (dQ is the separate dq pass): B*Hq*N^2*2*(dqk + dv) algorithmic FLOPs
    main_f = w.B * w.Hq * w.N * w.N * 2 * (w.Dqk + w.Dv)
    achieved = main_f / (t_bwd_main * 1e-3) / 1e12
    traffic = read_traffic(args.traffic)
    n_in = sum(t.numel() for t in (run.q, run.k, run.v, run.do))
    quant_bytes = 4.0625 * n_in                     # bf16 in, two fp8 copies + scales out
    rows = w.B * w.N * w.Hq
    stale_bytes = 4.0 * rows * w.Dv + 8.0 * rows    # bf16 dO and O in, (hi, lo) out
    consistent_bytes = (1 + 1 / 32 + 2) * rows * w.Dv + 8.0 * rows
    # the matched correction reads the Q and dO row copies, the K and V row
    # copies (codes and scales) and the LSE, and writes (hi, lo) per row
    kv_rows = w.B * w.nk * w.Hkv
    delta_bytes = (rows * (1 + 1 / 32) * (w.Dqk + w.Dv) + kv_rows * (1 + 1 / 32) * (w.Dqk + w.Dv)
                   + 4.0 * rows + 8.0 * rows)
    # after the main kernel: the dQ pass reads the one-byte dS' units (one per
    # causal score) and the K col copy, and writes dQ (bf16); the preparation
    # kernel's few MB are in the same interval
    dq_bytes = rows * w.N / 2 + kv_rows * (1 + 1 / 32) * w.Dqk + 2.0 * rows * w.Dqk

    line = {
        "metric": "FP8 attention fwd+bwd TFLOP/s and % of FP8 MFMA peak (causal GQA d128, 8K)",
        "value": round(value, 2),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "fp8_e4m3",
        "data": "synthetic",
        "config": {"workload": w.name, "batch": w.B, "seqlen": w.N, "heads_q": w.Hq, "heads_kv": w.Hkv,
                   "dim_qk": w.Dqk, "dim_v": w.Dv, "causal": True, "delta_mode": "matching",
                   "inputs": "bf16, one outlier channel x20 in Q and K", "step": "quantize+fwd+delta+bwd"},
        "pct_of_fp8_peak": round(100.0 * value / PEAK_FP8_TFLOPS, 2),
        "breakdown_ms": {"quantize": round(t_quant, 4), "fwd": round(t_fwd, 4), "delta_matching": round(t_delta, 4),
                         "delta_stale_rowsum": round(t_delta_stale, 4),
                         "delta_consistent_do": round(t_delta_consistent, 4), "bwd_main_kernel": round(t_bwd_main, 4),
                         "bwd_call": round(t_bwd_call, 4)},
        "paper_accounting": {"fwd_tflops": round(fwd_f / (t_fwd * 1e-3) / 1e12, 2),
                             "bwd_tflops_incl_delta": round(bwd_f / ((t_delta + t_bwd_call) * 1e-3) / 1e12, 2),
                             "fwd_bwd_tflops_prequantized": round(credited / (paper_ms * 1e-3) / 1e12, 2),
                             "pct_of_fp8_peak_prequantized": round(100 * credited / (paper_ms * 1e-3) / 1e12 /
                                                                   PEAK_FP8_TFLOPS, 2),
                             "delta_over_bwd_main": round(t_delta / t_bwd_main, 4),
                             "delta_over_delta_plus_bwd": round(t_delta / (t_delta + t_bwd_call), 4),
                             # the paper's reading: the matched backward's added time over the stale one
                             "matched_over_stale_bwd": round((t_delta + t_bwd_call) / (t_delta_stale + t_bwd_call) - 1,
                                                             4)},
        "hbm_gbs": {"quantize": round(quant_bytes / (t_quant * 1e-3) / 1e9, 1),
                    "delta_stale_rowsum": round(stale_bytes / (t_delta_stale * 1e-3) / 1e9, 1),
                    "delta_consistent_do": round(consistent_bytes / (t_delta_consistent * 1e-3) / 1e9, 1),
                    # compute-bound (its GEMMs and exponentials), listed for completeness
                    "delta_matching": round(delta_bytes / (t_delta * 1e-3) / 1e9, 1),
                    "dq_pass_and_prep": round(dq_bytes / ((t_bwd_call - t_bwd_main) * 1e-3) / 1e9, 1),
                    "peak": PEAK_HBM_GBS},
        # the other attention kernels against the same FP8 MFMA peak: the
        # forward's credited FLOPs and the correction pass's S and dP
        # (uncredited), each over its own time
        "mfma_other": {"fwd_kernel": {"achieved": round(fwd_f / (t_fwd * 1e-3) / 1e12, 2),
                                      "frac": round(fwd_f / (t_fwd * 1e-3) / 1e12 / PEAK_FP8_TFLOPS, 4)},
                       "delta_matching_kernel": {"achieved": round(fwd_f / (t_delta * 1e-3) / 1e12, 2),
                                                 "frac": round(fwd_f / (t_delta * 1e-3) / 1e12 / PEAK_FP8_TFLOPS,
                                                               4)}},
        "roofline": {"kernel": "bwd_kernel<128,128>", "bound": "mfma", "achieved": round(achieved, 2),
                     "peak": PEAK_FP8_TFLOPS, "unit": "TFLOP/s", "frac": round(achieved / PEAK_FP8_TFLOPS, 4),
                     "traffic": traffic, "flops_per_launch": main_f, "ms_per_launch": round(t_bwd_main, 4)},
    }
    if args.diagnostics:
        from paper_2609_37852_amd import diagnostics
        line["diagnostics"] = diagnostics.run(run.p, run.mq, run.mk, run.mv, run.mdo, run.lse, run.do, run.o)
    if not args.no_protocol:
        line["paper_protocol"] = run.protocol(args.clock_warmup)
        line["stale_step"] = run.full_step(pk.DELTA_STALE_ROWSUM)
        # the opt-in compensated matched correction against the plain one
        cm, pm = run.breakdown(pk.DELTA_MATCHING_COMPENSATED), run.breakdown(pk.DELTA_MATCHING)
        line["compensated"] = {"matching": pm, "compensated": cm,
                               "step_over_matching": round(cm["step_ms"] / pm["step_ms"] - 1, 4)}
        line["protected_dp"] = protected_dp_line(run)
        line["variants"] = variants_line(run)
        if args.workload == "gqa_d128_8k":
            # the same workload without the causal mask (every query sees all
            # 8192 keys; credited FLOPs count the full N x N products)
            del run
            torch.cuda.empty_cache()
            wn = synth.with_shape(w, causal=False)
            rn = Runner(wn, ev)
            for _ in range(3):
                rn.step()
            torch.cuda.synchronize()
            line["noncausal"] = {"workload": wn.name + " without the mask",
                                 "matched_step": rn.full_step(pk.DELTA_MATCHING),
                                 "paper_protocol": rn.protocol(0.0, rounds=3)}
            del rn
            torch.cuda.empty_cache()
            # the paper's other throughput shape: d = 256 (QK-norm workload), matched and stale
            w3 = synth.WORKLOADS["gqa_d256_8k_qknorm"]
            r3 = Runner(w3, ev)
            for _ in range(3):
                r3.step()
            torch.cuda.synchronize()
            line["secondary"] = {"workload": w3.name, "matched_step": r3.full_step(pk.DELTA_MATCHING),
                                 "stale_step": r3.full_step(pk.DELTA_STALE_ROWSUM),
                                 "paper_protocol": r3.protocol(0.0)}
            run = r3
    if args.more_configs:
        # the other throughput shapes of the workload table, measured as C2 is
        del run
        torch.cuda.empty_cache()
        more = {}
        for name in ("mla_d192_4k", "gqa_d128_64k_nope"):
            wm = synth.WORKLOADS[name]
            rm = Runner(wm, ev)
            for _ in range(3):
                rm.step()
            torch.cuda.synchronize()
            more[name] = {"matched_step": rm.full_step(pk.DELTA_MATCHING),
                          "stale_step": rm.full_step(pk.DELTA_STALE_ROWSUM),
                          "matched_split": rm.breakdown(pk.DELTA_MATCHING, n=5)}
            del rm
            torch.cuda.empty_cache()
        line["more_configs"] = more
        run = None
    if args.copy_calibration > 0:
        # a plain streaming kernel of known size: n bytes read, n written
        n = args.copy_calibration << 20
        src = torch.ones(n // 4, dtype=torch.float32, device="cuda:0")
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        torch.neg(src, out=dst)
        torch.cuda.synchronize()
        line["copy_calibration_bytes"] = n
    if not args.no_cpu_baseline:
        threads = int(os.environ.get("OMP_NUM_THREADS", "0")) or os.cpu_count()
        line["cpu_baseline"] = cpu_baseline(w, synth.generate(w, seed=0), threads)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
