"""Helpers shared by the GPU parity tests: cached workloads, row sampling,
oracle evaluation on the GPU's own codes, error metrics."""
from __future__ import annotations

import functools
import sys

import numpy as np

import oracle
from paper_2607_24377_amd import inputs

# Attention output against the oracle fed identical quantized operands.
REL_L2_TOL = 2e-3
MAX_ABS_TOL = 1e-2


# A bf16 output element whose oracle (fp64) value lies within this relative
# distance of the midpoint between two neighbouring bf16 values has two valid
# roundings: the kernel takes that decision on an fp32 accumulation, the
# oracle on fp64, so either neighbour is a correct result there.  The window
# is 1/16 of bf16's half-ulp (2^-9 relative) and four times the largest
# distance seen on the full-size workloads (2.5e-5).
BF16_TIE_WINDOW = 2.0 ** -14


def bf16_ties(got, ref, ref64):
    """Boolean mask of elements where got and ref (bf16 values as fp64) are
    the two bf16 neighbours of ref64 and ref64 lies within BF16_TIE_WINDOW
    (relative) of their midpoint."""
    got, ref, ref64 = (np.asarray(x, np.float64) for x in (got, ref, ref64))
    lo, hi = np.minimum(got, ref), np.maximum(got, ref)
    mid = 0.5 * (lo + hi)
    neighbours = (got != ref) & (lo <= ref64) & (ref64 <= hi)
    # lo and hi adjacent: no bf16 value strictly between them (bf16 = top 16
    # bits of fp32, so adjacent values differ by one in those bits)
    b = lambda x: (x.astype(np.float32).view(np.uint32) >> 16).astype(np.int64)
    adjacent = np.abs(b(got) - b(ref)) == 1
    return neighbours & adjacent & (np.abs(ref64 - mid) <= BF16_TIE_WINDOW * np.abs(ref64))


def log(*a):
    print(*a, flush=True)
    sys.stdout.flush()


@functools.lru_cache(maxsize=5)
def workload_bits(key):
    """bf16 bits of Q, K, V [B, H, N, d] for a workload (cached)."""
    w = inputs.workload(key)
    log(f"[gen] {w.name} B={w.B} H={w.H} N={w.N}")
    return inputs.generate(w)


def rel_l2(a, b) -> float:
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    return float(np.sqrt(np.sum((a - b) ** 2) / max(np.sum(b ** 2), 1e-300)))


def max_abs(a, b) -> float:
    return float(np.max(np.abs(np.asarray(a, np.float64) - np.asarray(b, np.float64))))


def sample_rows(N: int, n_random: int, seed: int, text_tokens: int = 0, tile: int = 128):
    """Stratified query rows: the first tile's first rows, the last rows of the
    sequence (the ragged query tile), the text rows if any, and random rows."""
    rng = np.random.default_rng(seed)
    rows = set(range(min(8, N)))
    rows |= set(range(max(0, N - 8), N))
    last_tile = (N - 1) // tile * tile
    rows |= set(range(last_tile, min(N, last_tile + 4)))
    if text_tokens:
        rows |= set(range(N - text_tokens, N, max(1, text_tokens // 16)))
    if n_random:
        rows |= set(rng.choice(N, size=min(N, n_random), replace=False).tolist())
    return np.array(sorted(rows), dtype=np.int64)


def oracle_rows(codes: dict, head: int, N: int, rows, mode: str, block_c: int, diag=False):
    """Oracle O (fp64 and bf16-rounded) of `rows` of flat head `head`, from
    codes/scales arrays shaped [BH, ...]."""
    res = oracle.mx_attention_head_rows(codes["qc"][head], codes["qs"][head], codes["kc"][head],
                                        codes["ks"][head], codes["vc"][head], codes["vs"][head],
                                        N, rows, mode, block_c, diag=diag)
    out, dg = res if diag else (res, None)
    rounded = oracle.bf16_to_f64(oracle.round_bf16(out))
    return (rounded, out, dg) if diag else (rounded, out)


def flat(a: np.ndarray) -> np.ndarray:
    """[B, H, ...] -> [B*H, ...]."""
    return a.reshape((-1,) + a.shape[2:])


# Full-size parity sample: at least this many query rows per workload, spread
# evenly over every (batch, head).
FULL_SAMPLE_ROWS = 2048


def stratified_rows(N: int, head: int, n_heads: int, per_head: int, seed: int, text_tokens: int = 0,
                    tile: int = 128):
    """Query rows of one head for the full-size parity sample: rows of the
    first query tile (0, 1, 63, 127), of the ragged last query tile (its first
    two rows and the last two of the sequence), this head's share of the text
    rows (every n_heads-th one, so that the heads together cover each text row
    exactly once), and random rows up to per_head."""
    rng = np.random.default_rng(seed)
    rows = {r for r in (0, 1, 63, 127) if r < N}
    last = (N - 1) // tile * tile
    rows |= {r for r in (last, last + 1, N - 2, N - 1) if 0 <= r < N}
    if text_tokens:
        rows |= set(range(N - text_tokens + head % n_heads, N, n_heads))
    while len(rows) < min(per_head, N):
        rows.add(int(rng.integers(N)))
    return np.array(sorted(rows), dtype=np.int64)


def gpu_codes(mx, qt, kt, vt, mode):
    """The GPU quantizer's codes and scales of Q, K, V as host arrays [BH, ...]."""
    qc, qs = mx.quantize(qt, mx.AXIS_HEAD_DIM, mode)
    kc, ks = mx.quantize(kt, mx.AXIS_HEAD_DIM, mode)
    vc, vs = mx.quantize(vt, mx.AXIS_TOKENS, mode)
    return {n: flat(t.cpu().numpy()) for n, t in dict(qc=qc, qs=qs, kc=kc, ks=ks, vc=vc, vs=vs).items()}


@functools.lru_cache(maxsize=8)
def full_size_rows(cfg: int):
    """{head: rows} of the full-size sample of workload `cfg` (mode-independent)."""
    w = inputs.workload(cfg)
    BH = w.B * w.H
    per_head = -(-FULL_SAMPLE_ROWS // BH)
    return {h: stratified_rows(w.N, h, BH, per_head, 5000 * cfg + h, w.text_tokens) for h in range(BH)}


@functools.lru_cache(maxsize=8)
def exact_reference(cfg: int):
    """Exact fp64 attention (no quantization) of the full-size sample's rows,
    in the same order as full_size_sample's arrays."""
    w = inputs.workload(cfg)
    q, k, v = (flat(x) for x in workload_bits(cfg))
    out = []
    for h, rows in full_size_rows(cfg).items():
        out.append(oracle.attention_exact_rows(oracle.bf16_to_f64(q[h][rows]), oracle.bf16_to_f64(k[h]),
                                               oracle.bf16_to_f64(v[h])))
    return np.concatenate(out)


@functools.lru_cache(maxsize=32)
def full_size_sample(cfg: int, mode: str):
    """The forward of workload `cfg` on the GPU (the launch the benchmark
    times) and the oracle, fed the GPU's own codes, on >= FULL_SAMPLE_ROWS
    stratified rows covering every head.  Cached so that the parity test
    and the error report share one sample.

    Returns dict(rows={head: rows}, got, ref, ref64 [R, d] in head order,
    diag [R, 8] (oracle diagnostics), head_of [R])."""
    import torch

    from paper_2607_24377_amd import mxattn as mx

    w = inputs.workload(cfg)
    q, k, v = workload_bits(cfg)
    qt, kt, vt = (mx.bf16_from_bits(x) for x in (q, k, v))
    out = mx.forward(qt, kt, vt, mode)
    torch.cuda.synchronize()
    got_all = flat(mx.bits_from_bf16(out))
    del out
    codes = gpu_codes(mx, qt, kt, vt, mode)
    del qt, kt, vt
    torch.cuda.empty_cache()
    BH = w.B * w.H
    rows = full_size_rows(cfg)
    got, ref, ref64, diag, head_of = [], [], [], [], []
    for h in range(BH):
        r, r64, dg = oracle_rows(codes, h, w.N, rows[h], mode, mx.kv_tile(), diag=True)
        got.append(oracle.bf16_to_f64(got_all[h][rows[h]]))
        ref.append(r)
        ref64.append(r64)
        diag.append(dg)
        head_of.append(np.full(rows[h].size, h))
    return dict(rows=rows, got=np.concatenate(got), ref=np.concatenate(ref), ref64=np.concatenate(ref64),
                diag=np.concatenate(diag), head_of=np.concatenate(head_of))
