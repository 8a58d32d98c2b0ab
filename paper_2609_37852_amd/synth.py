"""Seeded synthetic inputs for the attention workloads.

This module holds no arithmetic of the attention method: it only draws random
tensors and applies the input-side transforms that shape them like the
workloads the paper trains on (outlier channels, QK-norm gains, partial rotary
embedding, per-row logit temperature), then rounds them to the storage dtype.
Both the GPU path's tests/benchmark and the oracle consume its outputs.

Streams: numpy Philox keyed by seed*16 + {Q:0, K:1, V:2, dO:3, aux:4}.
All tensors are returned as float32 numpy arrays holding exactly
representable values of the stated dtype, in [B, N, H, D] layout.
"""
from __future__ import annotations

import math
from dataclasses import dataclass

import numpy as np

_STREAM = {"q": 0, "k": 1, "v": 2, "do": 3, "aux": 4}


@dataclass(frozen=True)
class Workload:
    name: str
    B: int
    N: int
    Hq: int
    Hkv: int
    Dqk: int
    Dv: int
    dtype: str          # "f32" or "bf16": storage dtype of Q, K, V, dO
    transform: str      # "none", "outlier", "outlier3", "qknorm", "rope", "temperature"
    tau: float          # softmax scale
    causal: bool = True
    Nk: int = 0         # key / value length (0: N); causal problems have Nk = N

    @property
    def nk(self) -> int:
        return self.Nk if self.Nk else self.N

    @property
    def causal_pairs(self) -> int:
        return self.B * self.Hq * self.N * (self.N + 1) // 2

    def credited_flops(self):
        """Paper's accounting (App. C.2) generalized to dqk != dv:
        fwd B*Hq*N^2*(dqk+dv), bwd B*Hq*N^2*(3*dqk+2*dv) for the causal
        problem (half of the full N x N products); without the mask the full
        N x Nk products count, twice as many per query-key pair."""
        n2 = self.B * self.Hq * self.N * self.N if self.causal else 2 * self.B * self.Hq * self.N * self.nk
        return n2 * (self.Dqk + self.Dv), n2 * (3 * self.Dqk + 2 * self.Dv)


WORKLOADS = {
    "tiny_mha_128": Workload("tiny_mha_128", 1, 128, 2, 2, 64, 64, "f32", "none", 1.0 / 8.0),
    "gqa_d128_8k": Workload("gqa_d128_8k", 4, 8192, 16, 4, 128, 128, "bf16", "outlier", 1.0 / math.sqrt(128)),
    "gqa_d256_8k_qknorm": Workload("gqa_d256_8k_qknorm", 2, 8192, 8, 2, 256, 256, "bf16", "qknorm", 1.0 / 16.0),
    "mla_d192_4k": Workload("mla_d192_4k", 2, 4096, 32, 32, 192, 128, "bf16", "rope", 1.0 / math.sqrt(192)),
    "gqa_d128_64k_nope": Workload("gqa_d128_64k_nope", 1, 65536, 16, 4, 128, 128, "bf16", "temperature",
                                  1.0 / math.sqrt(128)),
}


def with_shape(w: Workload, **kw) -> Workload:
    """Same recipe at another size (used for small parity cases)."""
    d = dict(w.__dict__)
    d.update(kw)
    return Workload(**d)


def _rng(seed: int, which: str) -> np.random.Generator:
    return np.random.Generator(np.random.Philox(key=seed * 16 + _STREAM[which]))


def round_bf16(x: np.ndarray) -> np.ndarray:
    """float32 -> nearest bfloat16 (ties to even), returned as float32."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.view(np.uint32).astype(np.uint64)
    u = (u + 0x7FFF + ((u >> 16) & 1)) & 0xFFFF0000
    return u.astype(np.uint32).view(np.float32)


def bf16_bits(x: np.ndarray) -> np.ndarray:
    """Upper 16 bits of float32 values that are already bfloat16-exact."""
    return (np.ascontiguousarray(x, dtype=np.float32).view(np.uint32) >> 16).astype(np.uint16)


def generate(w: Workload, seed: int = 0):
    """Returns dict q [B,N,Hq,Dqk], k [B,Nk,Hkv,Dqk], v [B,Nk,Hkv,Dv],
    do [B,N,Hq,Dv] (float32 arrays of dtype-exact values)."""
    B, N, Nk = w.B, w.N, w.nk
    q = _rng(seed, "q").standard_normal((B, N, w.Hq, w.Dqk), dtype=np.float32)
    k = _rng(seed, "k").standard_normal((B, Nk, w.Hkv, w.Dqk), dtype=np.float32)
    v = _rng(seed, "v").standard_normal((B, Nk, w.Hkv, w.Dv), dtype=np.float32)
    do = _rng(seed, "do").standard_normal((B, N, w.Hq, w.Dv), dtype=np.float32)
    aux = _rng(seed, "aux")
    if w.transform in ("outlier", "outlier3"):
        # 1% of head_dim channels (at least one), shared by all heads, x20 in Q
        # and K; "outlier3": three such channels (a robustness recipe)
        n_out = 3 if w.transform == "outlier3" else max(1, int(round(0.01 * w.Dqk)))
        idx = aux.choice(w.Dqk, size=n_out, replace=False)
        q[..., idx] *= 20.0
        k[..., idx] *= 20.0
    elif w.transform == "qknorm":
        # RMS-normalize each (token, head) vector of Q and K (eps 1e-6, fp32),
        # then per-channel gains U(0.5, 2) shared across heads
        gq = aux.uniform(0.5, 2.0, w.Dqk).astype(np.float32)
        gk = aux.uniform(0.5, 2.0, w.Dqk).astype(np.float32)
        for t, g in ((q, gq), (k, gk)):
            rms = np.sqrt(np.mean(t.astype(np.float32) ** 2, axis=-1, keepdims=True) + np.float32(1e-6))
            t *= (g / rms).astype(np.float32)
    elif w.transform == "rope":
        # MLA-style: the last 64 of 192 query/key channels carry rotary position
        # (NeoX half-split, base 10000, position = token index); the key's rotary
        # part is one vector per (batch, token) shared by every head.
        nope = w.Dqk - 64
        k_rope = aux.standard_normal((B, Nk, 1, 64), dtype=np.float32)
        k[..., nope:] = k_rope
        inv = 10000.0 ** (-np.arange(0, 32, dtype=np.float64) * 2.0 / 64.0)
        for t in (q, k):
            ang = np.arange(t.shape[1], dtype=np.float64)[:, None] * inv[None, :]
            cos = np.cos(ang).astype(np.float32)[None, :, None, :]
            sin = np.sin(ang).astype(np.float32)[None, :, None, :]
            x1 = t[..., nope:nope + 32].copy()
            x2 = t[..., nope + 32:].copy()
            t[..., nope:nope + 32] = x1 * cos - x2 * sin
            t[..., nope + 32:] = x2 * cos + x1 * sin
    elif w.transform == "temperature":
        # per query row (b, token, head) logit temperature t ~ U(0.5, 3)
        temp = aux.uniform(0.5, 3.0, (B, N, w.Hq, 1)).astype(np.float32)
        q *= temp
    elif w.transform != "none":
        raise ValueError(w.transform)
    if w.dtype == "bf16":
        q, k, v, do = (round_bf16(t) for t in (q, k, v, do))
    return dict(q=q, k=k, v=v, do=do)


def rope_table(N: int, R: int, base: float, pos0: int = 0) -> np.ndarray:
    """Cosine and sine of the rotary angles, [N, R/2, 2] float32: token n at
    position pos0 + n, pair c at frequency base^(-2c/R) (angles in float64,
    each value rounded once to float32).  An input of the producer, like the
    tensors above."""
    pos = np.arange(pos0, pos0 + N, dtype=np.float64)[:, None]
    inv = base ** (-np.arange(R // 2, dtype=np.float64) * 2.0 / R)
    ang = pos * inv[None, :]
    return np.stack([np.cos(ang), np.sin(ang)], axis=-1).astype(np.float32)
