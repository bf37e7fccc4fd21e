"""Seeded synthetic attention inputs shaped like the paper's video-DiT workloads.

This module only draws random numbers; it holds none of the quantization or
attention arithmetic.  Both the HIP path and the CPU oracle take their inputs
from here.

The paper evaluates Wan2.2 (720p, 81 frames) and HunyuanVideo (720p, 129
frames) attention (Sec. 5.1, "Implementation Details").  Their tensors,
weights and prompts are not available, so synthetic Q/K/V with the shapes
those settings imply stand in for them:

* ``tiny_iid``            B=1 H=2  N=512    iid N(0,1) Q/K/V.
* ``outlier_channels``    B=1 H=40 N=4096   N(0,1); 4 seed-chosen channels per
                          head (shared by Q and K) scaled x20.
* ``video480p``           B=1 H=40 N=32760 (21x30x52 latent grid): Q, K
                          Student-t (df=4); K gets a per-(head, channel) mean
                          offset drawn from N(0, variance 2); V N(0,1).
* ``video720p``           B=1 H=40 N=75600 (21x45x80), distributions as
                          ``video480p``.  The headline throughput workload.
* ``joint_text_video``    B=1 H=24 N=119056 (33x45x80 video tokens + 256 text
                          tokens, the text tokens last): video tokens as
                          ``video480p``; text-token Q and K (after the offset)
                          scaled x4; V never scaled.

Cross-attention (separate query and key/value lengths, as in Wan2.2's
cross-attention modules, Sec. 5.1): ``cross720p`` has B=1 H=40, 75600 video
queries distributed as ``video480p``'s Q, and 512 keys/values standing in
for the text context (K Student-t df=4 scaled x2 with a per-(head, channel)
offset drawn from N(0, variance 2), V N(0,1)); ``cross_ragged`` is a small
case with ragged lengths.

All configs use d=128 and bf16 storage (round to nearest even from fp32
draws).  Every (tensor, head) pair has its own seed stream,
``SeedSequence(20260000 + config_index, spawn_key=(tensor, head))``, so any
head can be regenerated alone.
"""
from __future__ import annotations

import concurrent.futures as _cf
import os
from dataclasses import dataclass

import numpy as np

_Q, _K, _V, _AUX = 0, 1, 2, 3


@dataclass(frozen=True)
class Workload:
    index: int
    name: str
    B: int
    H: int
    N: int
    d: int
    kind: str
    text_tokens: int = 0
    Nkv: int = 0  # keys/values per head if different from N (cross-attention)

    @property
    def n_kv(self) -> int:
        return self.Nkv or self.N

    @property
    def flops(self) -> float:
        """Algorithmic MXFP4 MFMA work of one forward: 4 * B * H * N * Nkv * d."""
        return 4.0 * self.B * self.H * self.N * self.n_kv * self.d


WORKLOADS = [
    Workload(0, "tiny_iid", 1, 2, 512, 128, "iid"),
    Workload(1, "outlier_channels", 1, 40, 4096, 128, "outlier"),
    Workload(2, "video480p", 1, 40, 32760, 128, "video"),
    Workload(3, "video720p", 1, 40, 75600, 128, "video"),
    Workload(4, "joint_text_video", 1, 24, 119056, 128, "video", text_tokens=256),
]
CROSS_WORKLOADS = [
    Workload(10, "cross720p", 1, 40, 75600, 128, "cross", Nkv=512),
    Workload(11, "cross_ragged", 1, 4, 1000, 128, "cross", Nkv=333),
]
BY_NAME = {w.name: w for w in WORKLOADS + CROSS_WORKLOADS}


def workload(key) -> Workload:
    if isinstance(key, Workload):
        return key
    if isinstance(key, int):
        return WORKLOADS[key]
    return BY_NAME[key]


def custom(B: int, H: int, N: int, d: int = 128, kind: str = "iid", text_tokens: int = 0,
           index: int = 99) -> Workload:
    """A workload with the given shape and one of the distribution recipes."""
    return Workload(index, f"custom_{kind}_b{B}h{H}n{N}", B, H, N, d, kind, text_tokens)


def _rng(w: Workload, tensor: int, head: int) -> np.random.Generator:
    ss = np.random.SeedSequence(20260000 + w.index, spawn_key=(tensor, head))
    return np.random.Generator(np.random.PCG64(ss))


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """fp32 -> bf16 bits, round to nearest even (inputs are finite)."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    r = (u + (np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1)))) >> np.uint32(16)
    return r.astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def _student_t4(rng: np.random.Generator, shape) -> np.ndarray:
    """Student-t with 4 degrees of freedom: Z / sqrt(chi2_4 / 4), chi2_4 = 2 Gamma(2)."""
    z = rng.standard_normal(shape, dtype=np.float32)
    g = rng.standard_gamma(2.0, shape, dtype=np.float32)
    return z / np.sqrt(g * np.float32(0.5))


def _head(w: Workload, b: int, h: int):
    """fp32 Q [N, d] and K, V [Nkv, d] of one (batch, head)."""
    head = b * w.H + h
    N, d = w.N, w.d
    rq, rk, rv, ra = (_rng(w, t, head) for t in (_Q, _K, _V, _AUX))
    if w.kind == "cross":
        q = _student_t4(rq, (N, d))
        k = _student_t4(rk, (w.n_kv, d)) * np.float32(2.0)
        mu = ra.normal(0.0, np.sqrt(2.0), size=d).astype(np.float32)
        k += mu[None, :]
        v = rv.standard_normal((w.n_kv, d), dtype=np.float32)
        return q, k, v
    v = rv.standard_normal((N, d), dtype=np.float32)
    if w.kind == "iid":
        q = rq.standard_normal((N, d), dtype=np.float32)
        k = rk.standard_normal((N, d), dtype=np.float32)
    elif w.kind == "outlier":
        q = rq.standard_normal((N, d), dtype=np.float32)
        k = rk.standard_normal((N, d), dtype=np.float32)
        ch = ra.choice(d, size=4, replace=False)
        q[:, ch] *= np.float32(20.0)
        k[:, ch] *= np.float32(20.0)
    elif w.kind == "video":
        q = _student_t4(rq, (N, d))
        k = _student_t4(rk, (N, d))
        mu = ra.normal(0.0, np.sqrt(2.0), size=d).astype(np.float32)
        k += mu[None, :]
        if w.text_tokens:
            q[N - w.text_tokens:] *= np.float32(4.0)
            k[N - w.text_tokens:] *= np.float32(4.0)
    else:
        raise ValueError(f"unknown workload kind {w.kind!r}")
    return q, k, v


def generate(key, heads=None, threads: int | None = None):
    """bf16 bits (uint16) Q, K, V of shape [B, H', N, d] for the selected heads.

    ``heads`` is a list of flat (b*H + h) head indices, default all."""
    w = workload(key)
    all_heads = list(range(w.B * w.H))
    sel = all_heads if heads is None else list(heads)
    shape = (len(sel), w.N, w.d)
    kv_shape = (len(sel), w.n_kv, w.d)
    Q = np.empty(shape, dtype=np.uint16)
    K = np.empty(kv_shape, dtype=np.uint16)
    V = np.empty(kv_shape, dtype=np.uint16)

    def one(i):
        b, h = divmod(sel[i], w.H)
        q, k, v = _head(w, b, h)
        Q[i] = f32_to_bf16_bits(q)
        K[i] = f32_to_bf16_bits(k)
        V[i] = f32_to_bf16_bits(v)

    nt = threads or min(16, os.cpu_count() or 1)
    if len(sel) <= 1 or nt <= 1:
        for i in range(len(sel)):
            one(i)
    else:
        with _cf.ThreadPoolExecutor(nt) as ex:
            list(ex.map(one, range(len(sel))))
    if heads is None:
        return (Q.reshape(w.B, w.H, w.N, w.d), K.reshape(w.B, w.H, w.n_kv, w.d),
                V.reshape(w.B, w.H, w.n_kv, w.d))
    return Q, K, V
