#!/usr/bin/env python3
"""Per-(workload, mode) measurements of the MXFP4 attention forward on one
MI355X: one JSON line per row.

    python bench_table.py [--steps 10] [--workloads outlier_channels,video480p,video720p,joint_text_video]

For each workload (inputs generated once) and each mode: the whole forward
(quantizers + fused kernel) and the fused attention kernel alone on quantized
operands, each the median of --steps HIP-event-timed calls after warm-up, as
TFLOP/s and fraction of the dense MXFP4 peak; the two standalone quantizers
in GB/s of algorithmic traffic (2.53125 B per element).  Under rocprofv3 the
launches of one row are told apart by their grid (one per workload) and the
mode in the kernel's name.
"""
from __future__ import annotations

import argparse
import json
import os
import sys

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

from bench import PEAK_FP4_TFLOPS, log, time_ms  # noqa: E402

DEFAULT = "outlier_channels,video480p,video720p,joint_text_video"
MODES = ["ocp_vanilla", "uos", "uos_pnq"]


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workloads", default=DEFAULT)
    ap.add_argument("--modes", default=",".join(MODES))
    args = ap.parse_args()

    import torch

    from paper_2607_24377_amd import inputs, mxattn

    if not torch.cuda.is_available():
        print("bench_table.py: no GPU visible", file=sys.stderr)
        sys.exit(1)
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    mxattn.lib()
    for name in args.workloads.split(","):
        w = inputs.workload(name)
        log(f"[table] generating {w.name}")
        q, k, v = (mxattn.bf16_from_bits(x, dev) for x in inputs.generate(w))
        out = torch.empty_like(q)
        short = w.flops < 1e13
        steps = max(args.steps, 100 if short else args.steps)
        warm = max(args.warmup, 20 if short else args.warmup)
        for mode in args.modes.split(","):
            log(f"[table] {w.name} {mode}")
            fwd_ms = time_ms(lambda: mxattn.forward(q, k, v, mode, out=out), steps, warm, torch)
            qc, qs = mxattn.quantize(q, mxattn.AXIS_HEAD_DIM, mode)
            kc, ks = mxattn.quantize(k, mxattn.AXIS_HEAD_DIM, mode)
            vc, vs = mxattn.quantize(v, mxattn.AXIS_TOKENS, mode)
            attn_ms = time_ms(lambda: mxattn.attend(qc, qs, kc, ks, vc, vs, w.N, mode, out=out), steps, 1, torch)
            qd_ms = time_ms(lambda: mxattn.quantize(k, mxattn.AXIS_HEAD_DIM, mode, codes=kc, scales=ks), steps, 1,
                            torch)
            qt_ms = time_ms(lambda: mxattn.quantize(v, mxattn.AXIS_TOKENS, mode, codes=vc, scales=vs), steps, 1,
                            torch)
            elems = w.B * w.H * w.N * w.d
            row = {
                "workload": w.name, "B": w.B, "H": w.H, "N": w.N, "mode": mode, "steps": steps,
                "forward_ms": fwd_ms, "forward_TFLOPs": w.flops / fwd_ms / 1e9,
                "forward_frac_of_peak": w.flops / fwd_ms / 1e9 / PEAK_FP4_TFLOPS,
                "attention_ms": attn_ms, "attention_TFLOPs": w.flops / attn_ms / 1e9,
                "attention_frac_of_peak": w.flops / attn_ms / 1e9 / PEAK_FP4_TFLOPS,
                "quantize_headdim_GBps": elems * 2.53125 / qd_ms / 1e6,
                "quantize_tokens_GBps": elems * 2.53125 / qt_ms / 1e6,
                "grid_workgroups": w.B * w.H * ((w.N + 127) // 128),
            }
            print(json.dumps(row), flush=True)
            del qc, qs, kc, ks, vc, vs
        del q, k, v, out
        torch.cuda.empty_cache()


if __name__ == "__main__":
    main()
