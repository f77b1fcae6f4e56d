"""Write csrc/model_calibration.h, the block-step times of the DAG model that
DASH_SCHED_AUTO simulates, from a measured sweep.

Input: the JSON lines of measure_model_grid.py on MI355X (one line per shape:
B, H, N, d, mask and whole-call TFLOP/s per schedule), stored next to this
script as model_grid.jsonl.  For every ordered schedule of every line,
the call's measured time is divided by the makespan the model gives that
shape with a unit block step (compute share kModelComputeShare, the rest
reduction), simulated exactly as the library does for DASH_SCHED_AUTO (256
resident workgroups, the library's ticket order, and for many heads the
extrapolation from ceil(3 * 256 / chains) and twice that many heads).  At a sweep shape the model then reproduces the measured time of
every schedule, and AUTO picks the measured fastest; elsewhere the step time
is interpolated in N and in the number of heads, and the DAG decides.

    python -m paper_2601_21824_amd.calibrate_model > paper_2601_21824_amd/csrc/model_calibration.h

(B*H heads per line; the step time depends on both N and the number of heads,
through the caches more than through the DAG.)

(libdash.so must be built; the table does not enter the model itself, so
rebuilding after writing it changes nothing here.)
"""
from __future__ import annotations

import json
import math
import os
import sys

from . import binding as b

HERE = os.path.dirname(os.path.abspath(__file__))
WORKERS = 256        # resident workgroups of the d = 64 / 128 / 256 kernels on MI355X (one per CU)
COMPUTE_SHARE = 0.02  # c / (c + r) per block step (the wait lags a whole step)
ORDERED = {"naive": b.DASH_SCHED_NAIVE, "descending": b.DASH_SCHED_DESCENDING,
           "shift": b.DASH_SCHED_SHIFT, "symshift": b.DASH_SCHED_SYMSHIFT}


def rows(path):
    with open(path) as f:
        for line in f:
            if line.strip():
                yield json.loads(line)


def main(path=os.path.join(HERE, "model_grid.jsonl")):
    out = []
    for r in rows(path):
        B, H, N, d, causal = r["B"], r["H"], r["N"], r["d"], r["mask"] == "causal"
        flops = 4.0 * B * H * N * N * d * 2.5 / (2 if causal else 1)
        for name, sched in ORDERED.items():
            if name not in r:
                continue
            chains = b.dash_schedule_table(sched, N, d, causal, heads=B * H)["chains"]
            cap = max(1, -(-3 * WORKERS // chains))
            unit = b.dash_model_makespan(sched, B, H, N, d, causal, WORKERS, COMPUTE_SHARE, 1.0 - COMPUTE_SHARE,
                                         max_heads=cap)
            us = flops / (r[name] * 1e12) * 1e6
            out.append((d, int(causal), sched, N, B * H, us / unit, name, r[name]))
    out.sort()
    print("// model_calibration.h -- block-step times of the DAG model behind DASH_SCHED_AUTO,")
    print("// measured on MI355X.  Written by calibrate_model.py from model_grid.jsonl")
    print("// (python -m paper_2601_21824_amd.calibrate_model); do not edit by hand.")
    print("#pragma once")
    print()
    print("namespace dash {")
    print()
    print("struct StepCost {")
    print("  int d, causal, sched, n, heads;")
    print("  double us;  // time of one 64-row block step, microseconds")
    print("};")
    print()
    print(f"constexpr double kModelComputeShare = {COMPUTE_SHARE};")
    print("constexpr StepCost kStepCosts[] = {")
    for d, c, s, n, bh, us, name, tf in out:
        print(f"    {{{d}, {c}, {s}, {n}, {bh}, {us:.6f}}},  // {name}: {tf} TFLOP/s")
    print("};")
    print()
    print("}  // namespace dash")
    return 0


if __name__ == "__main__":
    sys.exit(main(*sys.argv[1:]))
