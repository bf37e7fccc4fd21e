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
