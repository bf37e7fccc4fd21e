#!/usr/bin/env python3
"""Throughput of the MXFP4 attention forward (quantize Q/K/V + fused kernel)
on one MI355X, on synthetic video-DiT-shaped inputs.

    python bench.py [--steps K] [--warmup W] [--workload video720p] [--mode uos_pnq]

Prints one JSON line.  ``value`` is 4*B*H*N^2*d / t in TFLOP/s for the whole
forward (the three quantize launches and the fused attention kernel), inputs
already resident in HBM.  ``roofline`` rates the fused attention kernel alone
against the dense MXFP4 matrix-core peak; ``cpu_baseline`` times the CPU
oracle on a bounded sample of the same workload on this host's cores.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "MXFP4 attn fwd TFLOPS (4·B·H·N²·d/t) & % of MXFP4 MFMA peak, N=75600"
PEAK_FP4_TFLOPS = 10100.0  # MI355X dense MXFP4 matrix-core peak, 10.1 PFLOP/s
PEAK_BF16_TFLOPS = 2500.0  # MI355X dense bf16 matrix-core peak, 2.5 PFLOP/s
PROFILES = os.path.join(ROOT, "profiles")
KERNEL_SOURCE = os.path.join(ROOT, "paper_2607_24377_amd", "csrc", "attention.hip")


def log(msg: str):
    print(msg, file=sys.stderr, flush=True)


def time_steps(fn, steps: int, warmup: int, torch):
    """Per-step times (ms) of `steps` calls after `warmup` untimed calls: the
    timed calls are bracketed by device synchronizations and each is timed
    between HIP events recorded on the current stream (the stream the
    library launches on)."""
    for _ in range(warmup):
        fn()
    torch.cuda.synchronize()
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(steps + 1)]
    ev[0].record()
    for i in range(steps):
        fn()
        ev[i + 1].record()
    torch.cuda.synchronize()
    return [ev[i].elapsed_time(ev[i + 1]) for i in range(steps)]


def median(xs):
    xs = sorted(xs)
    n = len(xs)
    return xs[n // 2] if n % 2 else 0.5 * (xs[n // 2 - 1] + xs[n // 2])


def time_ms(fn, steps: int, warmup: int, torch) -> float:
    """Median ms per call (see time_steps)."""
    return median(time_steps(fn, steps, warmup, torch))


def measured_traffic(workload: str, mode: str):
    """HBM bytes per launch of the attention kernel from the committed PMC
    counter summary of this workload and mode, if it was taken on the current
    kernel source."""
    try:
        with open(os.path.join(PROFILES, f"attention_{workload}_hbm_traffic.json")) as f:
            rec = json.load(f)
        with open(KERNEL_SOURCE, "rb") as f:
            sha = hashlib.sha256(f.read()).hexdigest()
        if (rec.get("kernel_source_sha256") != sha or rec.get("workload_name") != workload
                or rec.get("mode") != mode):
            return None
        return float(rec["hbm_bytes_per_launch"])
    except (OSError, ValueError, KeyError):
        return None


def cpu_baseline(w, mode: str, rows_req: int, q_bits, k_bits, v_bits, block_c: int):
    """Time the CPU oracle on sampled query rows of head 0 (its own quantization
    of that head, then the tiled recurrence over all N keys)."""
    import numpy as np

    import oracle

    qh, kh, vh = (x.reshape((-1,) + x.shape[2:])[0:1][None] for x in (q_bits, k_bits, v_bits))
    codes = oracle.quantize_qkv(qh, kh, vh, mode)

    def run(rows):
        return oracle.mx_attention_head_rows(codes["qc"][0, 0], codes["qs"][0, 0], codes["kc"][0, 0],
                                             codes["ks"][0, 0], codes["vc"][0, 0], codes["vs"][0, 0],
                                             w.n_kv, rows, mode, block_c)

    nthreads = oracle.threads(0)
    rng = np.random.default_rng(1)
    order = rng.permutation(w.N)
    if rows_req > 0:  # fixed sample
        rows = np.sort(order[:rows_req])
        t0 = time.perf_counter()
        run(rows)
        dt = time.perf_counter() - t0
        done = rows.size
    else:  # batches of random rows until ~12 s of CPU work
        done, dt, batch = 0, 0.0, 4 * nthreads
        while dt < 12.0 and done < w.N:
            rows = np.sort(order[done:done + batch])
            t0 = time.perf_counter()
            run(rows)
            dt += time.perf_counter() - t0
            done += rows.size
            batch = min(8 * batch, 16384)
    rows = np.arange(done)
    flops = 4.0 * w.n_kv * w.d * rows.size
    # the whole-tensor quantizer oracle: Q and K blocked along d, V along the
    # keys, every element, with the mode's scale rule (and rotation)
    rule = oracle.MODES[mode][0]
    rot = mode in oracle.ROTATED
    t0 = time.perf_counter()
    oracle.quantize_rows(q_bits, rule, rotate=rot)
    oracle.quantize_rows(k_bits, rule, rotate=rot)
    oracle.quantize_keys(v_bits, rule)
    qdt = time.perf_counter() - t0
    elems = q_bits.size + k_bits.size + v_bits.size
    return {"value": flops / dt / 1e12, "unit": "TFLOP/s", "cores": nthreads, "kind": "oracle",
            "sample": f"{done} random query rows of head 0 of {w.name} ({mode}), all "
                      f"{w.n_kv} keys, fp64 tiled recurrence incl. dequantization; "
                      f"{dt:.1f} s wall",
            "projected_forward_s": dt * (w.B * w.H * w.N) / done,
            "quantizer": {"elements": elems, "seconds": qdt, "Melem_per_s": elems / qdt / 1e6,
                          "GBps_equivalent": elems * 2.53125 / qdt / 1e9,
                          "sample": f"every element of Q, K and V of {w.name}"}}


def stratified_rows(N: int, n_heads: int, per_head: int, seed: int, text_tokens: int = 0, tile: int = 128):
    """{head: query rows} of a bounded oracle sample: rows of the first query
    tile, of the ragged last query tile and the sequence's end, each head's
    share of the text rows, and random rows, per_head rows per head."""
    import numpy as np

    out = {}
    last = (N - 1) // tile * tile
    for h in range(n_heads):
        rng = np.random.default_rng(seed + h)
        rows = {r for r in (0, 1, 63, 127, last, last + 1, N - 2, N - 1) if 0 <= r < N}
        if text_tokens:
            rows |= set(range(N - text_tokens + h, N, n_heads))
        while len(rows) < min(per_head, N):
            rows.add(int(rng.integers(N)))
        out[h] = np.array(sorted(rows), dtype=np.int64)
    return out


def cpu_table(modes, sample_rows: int, steps: int, warmup: int):
    """The CPU oracle per configuration, beside the GPU forward of the same
    configuration and mode: the quantizer oracle over every element of Q, K
    and V, and the attention oracle on every row of the two small workloads
    and on about `sample_rows` rows spread over every head of the long ones,
    projected to the whole problem.  One JSON line per (workload, mode)."""
    import numpy as np
    import torch

    import oracle
    from paper_2607_24377_amd import inputs, mxattn

    dev = torch.device("cuda:0")
    nthreads = oracle.threads(0)
    for w in inputs.WORKLOADS:
        log(f"[cpu-table] generating {w.name}")
        q_bits, k_bits, v_bits = inputs.generate(w)
        q, k, v = (mxattn.bf16_from_bits(x, dev) for x in (q_bits, k_bits, v_bits))
        out = torch.empty_like(q)
        bh = w.B * w.H
        if w.flops < 1e12:  # every row
            sample = {h: np.arange(w.N, dtype=np.int64) for h in range(bh)}
        else:
            sample = stratified_rows(w.N, bh, -(-sample_rows // bh), 7, w.text_tokens)
        nrows = sum(r.size for r in sample.values())
        for mode in modes:
            log(f"[cpu-table] {w.name} {mode}: GPU forward")
            short = w.flops < 1e13
            gpu_ms = time_ms(lambda: mxattn.forward(q, k, v, mode, out=out), max(steps, 100 if short else steps),
                             max(warmup, 20 if short else warmup), torch)
            log(f"[cpu-table] {w.name} {mode}: oracle quantizer, every element")
            rule = oracle.MODES[mode][0]
            rot = mode in oracle.ROTATED
            t0 = time.perf_counter()
            qc, qs = oracle.quantize_rows(q_bits, rule, rotate=rot)
            kc, ks = oracle.quantize_rows(k_bits, rule, rotate=rot)
            vc, vs = oracle.quantize_keys(v_bits, rule)
            qdt = time.perf_counter() - t0
            flat = lambda a: a.reshape((-1,) + a.shape[2:])
            qc, qs, kc, ks, vc, vs = (flat(a) for a in (qc, qs, kc, ks, vc, vs))
            log(f"[cpu-table] {w.name} {mode}: oracle attention, {nrows} rows over {bh} heads")
            # per head: dequantize K^, V^ (a cost per head, not per row), then
            # the tiled recurrence for the sampled rows (a cost per row)
            p_rule, pnq = oracle.MODES[mode]
            ddt = adt = 0.0
            for h, rows in sample.items():
                t0 = time.perf_counter()
                qh = oracle.dequant_rows(np.ascontiguousarray(qc[h][rows]), np.ascontiguousarray(qs[h][rows]))
                kh = oracle.dequant_rows(kc[h], ks[h])
                vh = oracle.dequant_keys(vc[h], vs[h], w.n_kv)
                t1 = time.perf_counter()
                oracle.attention_rows(qh, kh, vh, p_rule, pnq, 0, mxattn.kv_tile())
                ddt += t1 - t0
                adt += time.perf_counter() - t1
            elems = q_bits.size + k_bits.size + v_bits.size
            proj = ddt + adt * (bh * w.N) / nrows
            print(json.dumps({
                "workload": w.name, "B": w.B, "H": w.H, "N": w.N, "mode": mode, "cores": nthreads,
                "gpu_forward_ms": gpu_ms,
                "oracle_quantizer": {"elements": elems, "seconds": qdt, "Melem_per_s": elems / qdt / 1e6,
                                     "GBps_equivalent": elems * 2.53125 / qdt / 1e9},
                "oracle_attention": {"rows": nrows, "all_rows": nrows == bh * w.N, "seconds": adt,
                                     "dequantize_seconds": ddt,
                                     "rows_per_s": nrows / adt,
                                     "score_elements_per_s": nrows * w.n_kv / adt,
                                     "TFLOPs": 4.0 * w.n_kv * w.d * nrows / adt / 1e12,
                                     "projected_full_s": proj},
                "oracle_over_gpu": proj * 1e3 / gpu_ms,
            }), flush=True)
        del q, k, v, out
        torch.cuda.empty_cache()


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=None, help="timed steps (default 10; 200 for short workloads)")
    ap.add_argument("--warmup", type=int, default=None, help="untimed steps (default 3; 50 for short workloads)")
    ap.add_argument("--workload", default="video720p")
    ap.add_argument("--mode", default="uos_pnq", choices=["ocp_vanilla", "uos", "uos_pnq", "uos_pnq_rot"])
    ap.add_argument("--cpu-rows", type=int, default=0, help="oracle sample rows (0: ~15 s)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-overhead", action="store_true")
    ap.add_argument("--no-next", action="store_true",
                    help="skip the boundary-sweep and row-sum diagnostic timings")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="also run one plain 1 GiB device copy (reference for HBM byte counters)")
    ap.add_argument("--cpu-table", action="store_true",
                    help="instead of the bench line: the CPU oracle per workload and mode beside the GPU "
                         "forward (one JSON line each)")
    ap.add_argument("--cpu-table-rows", type=int, default=2048)
    args = ap.parse_args()

    if args.gpus != 1:
        print(f"bench.py: this build runs on one GPU only (asked for --gpus {args.gpus}); "
              "the path shards over heads without communication, see the design notes.",
              file=sys.stderr)
        sys.exit(2)

    import torch

    from paper_2607_24377_amd import inputs, mxattn

    if not torch.cuda.is_available():
        print("bench.py: no GPU visible", file=sys.stderr)
        sys.exit(1)
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    if args.cpu_table:
        mxattn.lib()
        cpu_table(["ocp_vanilla", "uos", "uos_pnq"], args.cpu_table_rows, args.steps or 10, args.warmup or 3)
        return
    w = inputs.workload(args.workload)
    log(f"[bench] generating {w.name} B={w.B} H={w.H} N={w.N} d={w.d}")
    q_bits, k_bits, v_bits = inputs.generate(w)
    q, k, v = (mxattn.bf16_from_bits(x, dev) for x in (q_bits, k_bits, v_bits))
    out = torch.empty_like(q)
    mxattn.lib()

    cross = w.n_kv != w.N
    # a workload of under 10 TFLOP a step gets enough steps for the timed
    # region to last ~0.1 s: a burst of a few ms runs well below the steady
    # rate (0.60 against 0.47 ms per cross720p forward)
    short = w.flops < 1e13
    if args.steps is None:
        args.steps = 200 if short else 10
    if args.warmup is None:
        args.warmup = 50 if short else 3

    def fwd(mode):
        if cross:
            return lambda: mxattn.cross_forward(q, k, v, mode, out=out)
        return lambda: mxattn.forward(q, k, v, mode, out=out)

    log(f"[bench] timing forward {args.mode}: warmup {args.warmup}, steps {args.steps}")
    step_ms = time_steps(fwd(args.mode), args.steps, args.warmup, torch)
    ms = median(step_ms)
    value = w.flops / (ms * 1e-3) / 1e12

    # the fused attention kernel alone (dominant kernel) on pre-quantized operands
    qc, qs = mxattn.quantize(q, mxattn.AXIS_HEAD_DIM, args.mode)
    kc, ks = mxattn.quantize(k, mxattn.AXIS_HEAD_DIM, args.mode)
    vc, vs = mxattn.quantize(v, mxattn.AXIS_TOKENS, args.mode)
    log("[bench] timing the attention kernel alone")
    attn_ms = time_ms(lambda: mxattn.cross_attend(qc, qs, kc, ks, vc, vs, w.N, w.n_kv, args.mode, out=out),
                      args.steps, 1, torch)
    quant_ms = time_ms(lambda: mxattn.quantize(v, mxattn.AXIS_TOKENS, args.mode, codes=vc, scales=vs),
                       args.steps, 1, torch)
    quant_q_ms = time_ms(lambda: mxattn.quantize(q, mxattn.AXIS_HEAD_DIM, args.mode, codes=qc, scales=qs),
                         args.steps, 1, torch)
    achieved = w.flops / (attn_ms * 1e-3) / 1e12
    elems = w.B * w.H * w.N * w.d
    extra = {
        "timing": "median of per-step HIP-event times",
        "ms_per_step_mean": sum(step_ms) / len(step_ms),
        "ms_per_step_min": min(step_ms),
        "ms_per_step_max": max(step_ms),
        "pct_of_mxfp4_peak": 100.0 * value / PEAK_FP4_TFLOPS,
        "attention_kernel_ms": attn_ms,
        "quantize_headdim_ms": quant_q_ms,
        "quantize_tokens_ms": quant_ms,
        "quantize_headdim_GBps": elems * 2.53125 / (quant_q_ms * 1e-3) / 1e9,
        "quantize_tokens_GBps": w.B * w.H * w.n_kv * w.d * 2.53125 / (quant_ms * 1e-3) / 1e9,
    }
    if not args.no_next:
        # the boundary family and the 41-point MSE sweep of Table cx_distribution
        sweep = [round(6.0 + 0.05 * i, 2) for i in range(41)]
        sse = torch.empty((w.B * w.H, len(sweep)), dtype=torch.float64, device=dev)
        log("[bench] timing the boundary quantizer and the MSE sweep")
        qq_ms = time_ms(lambda: mxattn.quantize_qmax(q, mxattn.AXIS_HEAD_DIM, 7.0, codes=qc, scales=qs),
                        args.steps, 1, torch)
        sq_ms = time_ms(lambda: mxattn.qmax_sse(q, mxattn.AXIS_HEAD_DIM, sweep, out=sse), args.steps, 1, torch)
        sv_ms = time_ms(lambda: mxattn.qmax_sse(v, mxattn.AXIS_TOKENS, sweep, out=sse), args.steps, 1, torch)
        extra["boundary_sweep"] = {
            "boundaries": len(sweep),
            "quantize_qmax_headdim_ms": qq_ms,
            "sse_headdim_ms": sq_ms,
            "sse_tokens_ms": sv_ms,
            "sse_headdim_GBps": elems * 2.0 / (sq_ms * 1e-3) / 1e9,
            "sse_tokens_GBps": w.B * w.H * w.n_kv * w.d * 2.0 / (sv_ms * 1e-3) / 1e9,
        }
        del sse
        # row-sum diagnostics (Fig. pnq_rowsum): the fused whole-tensor pass
        # and, on a materialized 128-row tile of P, the standalone quantizer
        log("[bench] timing the row-sum diagnostics")
        stats = torch.empty((w.B, w.H, w.N, 8), dtype=torch.float64, device=dev)
        fused_ms = time_ms(lambda: mxattn.attention_rowsum_diag(q, k, args.mode, out=stats),
                           max(1, args.steps // 5), 1, torch)
        rows = min(128, w.N)
        P = mxattn.softmax_rows(q, k, 0, rows)
        tile_stats = torch.empty((w.B * w.H * rows, 8), dtype=torch.float64, device=dev)
        soft_ms = time_ms(lambda: mxattn.softmax_rows(q, k, 0, rows, out=P), args.steps, 1, torch)
        diag_ms = time_ms(lambda: mxattn.rowsum_diag(P, w.n_kv, args.mode, out=tile_stats), args.steps, 1, torch)
        score_flops = 2 * 2.0 * w.B * w.H * w.N * w.n_kv * w.d  # two passes of Q K^T
        extra["rowsum_diag"] = {
            "fused_ms": fused_ms,
            "fused_score_TFLOPs": score_flops / (fused_ms * 1e-3) / 1e12,
            "fused_frac_of_bf16_peak": score_flops / (fused_ms * 1e-3) / 1e12 / PEAK_BF16_TFLOPS,
            "tile_rows": rows,
            "softmax_rows_tile_ms": soft_ms,
            "diag_tile_ms": diag_ms,
            "diag_tile_GBps": P.numel() * 4 / (diag_ms * 1e-3) / 1e9,
        }
        del stats, P, tile_stats
    if not args.no_overhead:
        other = "ocp_vanilla" if args.mode != "ocp_vanilla" else "uos_pnq"
        log(f"[bench] timing forward {other} for the overhead comparison")
        ms_other = time_ms(fwd(other), args.steps, 1, torch)
        ms_again = time_ms(fwd(args.mode), args.steps, 1, torch)
        extra[f"{other}_ms_per_step"] = ms_other
        extra[f"{args.mode}_ms_per_step_repeat"] = ms_again
        extra[f"overhead_{args.mode}_vs_{other}"] = min(ms, ms_again) / ms_other - 1.0
    del qc, qs, kc, ks, vc, vs
    if args.copy_calibration:
        # an elementwise kernel that reads 1 GiB and writes 1 GiB
        src = torch.zeros(1 << 28, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        torch.neg(src, out=dst)
        torch.cuda.synchronize()
        del src, dst

    result = {
        "metric": METRIC,
        "value": value,
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "mxfp4",
        "data": "synthetic",
        "config": {"workload": w.name, "B": w.B, "H": w.H, "N": w.N, "Nkv": w.n_kv, "d": w.d, "mode": args.mode,
                   "kv_tile": mxattn.kv_tile(), "query_tile": mxattn.query_tile()},
        "roofline": {"bound": "mfma", "achieved": achieved, "peak": PEAK_FP4_TFLOPS,
                     "unit": "TFLOP/s", "frac": achieved / PEAK_FP4_TFLOPS,
                     "traffic": measured_traffic(w.name, args.mode)},
    }
    result.update(extra)
    if not args.no_cpu_baseline:
        log("[bench] timing the CPU oracle baseline")
        result["cpu_baseline"] = cpu_baseline(w, args.mode, args.cpu_rows, q_bits, k_bits, v_bits,
                                              mxattn.kv_tile())
    else:
        result["cpu_baseline"] = None
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
