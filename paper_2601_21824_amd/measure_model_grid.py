"""Measure the ordered schedules over a grid of shapes on the GPU: the data
behind the block-step times of the DAG model that picks DASH_SCHED_AUTO.

For d in (64, 128, 256), both masks, N from 512 to 16384 (d = 256: 4096 to
32768) and B*H of 1, 2, 4, 16, 32, 64, 128, 256, 512 and 1024 heads (at most
2^21 tokens and 6e13 FLOPs per call), every
candidate deterministic schedule is timed as bench.py times a backward call
(whole call, wall clock over back-to-back calls after 3 checked warm-up
calls, >= 20 ms of work per timing), twice in opposite orders; the better of
the two is kept.  One JSON line per shape on stdout, in the format of
``bench.py --sweep``:

    python -m paper_2601_21824_amd.measure_model_grid > paper_2601_21824_amd/model_grid.jsonl

(Head dims as arguments measure only those, e.g. ``... measure_model_grid 64``;
``--heads 32,128`` only those head counts, ``--mask causal`` only that mask.)
"""
from __future__ import annotations

import json
import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


HEADS = (1, 2, 4, 16, 32, 64, 128, 256, 512, 1024)


def shapes(dims=(64, 128, 256), heads=HEADS, masks=(False, True)):
    for d in dims:
        lengths = (4096, 8192, 16384, 32768) if d == 256 else (512, 1024, 2048, 4096, 8192, 16384)
        for causal in masks:
            for n in lengths:
                for bh in heads:
                    flops = 4.0 * bh * n * n * d * 2.5 / (2 if causal else 1)
                    if bh * n <= (1 << 21) and flops <= 6e13:
                        yield d, causal, n, bh


def main(*dims):
    sys.path.insert(0, ROOT)
    import torch

    import bench
    from paper_2601_21824_amd import binding as dash
    from paper_2601_21824_amd.synth import make_inputs

    heads = HEADS
    if "--heads" in dims:
        i = dims.index("--heads")
        heads = tuple(int(x) for x in dims[i + 1].split(","))
        dims = dims[:i] + dims[i + 2:]
    masks = (False, True)
    if "--mask" in dims:
        i = dims.index("--mask")
        masks = (dims[i + 1] == "causal",)
        dims = dims[:i] + dims[i + 2:]
    ev = bench.HipEvents()
    for d, causal, N, bh in shapes(tuple(int(x) for x in dims) or (64, 128, 256), heads, masks):
        q, k, v, do = make_inputs(1, bh, N, d, seed=N + d + bh, sigma=0.5 if d == 256 else 1.0)
        qg, kg, vg, dog = (t.cuda() for t in (q, k, v, do))
        og, lseg = dash.attn_fwd(qg, kg, vg, causal)
        dq, dk, dv = torch.empty_like(qg), torch.empty_like(kg), torch.empty_like(vg)
        ws = dash.new_workspace(1, bh, N, d, "shift")
        tensors = (qg, kg, vg, og, dog, lseg, dq, dk, dv, ws)
        flops = 4.0 * bh * N * N * d * 2.5 / (2 if causal else 1)
        scheds = ["descending", "symshift", "naive"] if causal else ["shift", "descending", "naive"]
        steps = max(5, min(200, int(20e-3 / (flops / 4e14))))
        best = {}
        for order in (scheds, scheds[::-1]):
            for s in order:
                ms, _ = bench.time_schedule(dash, tensors, causal, s, steps, 3, ev)
                best[s] = max(best.get(s, 0.0), flops / (ms * 1e-3) / 1e12)
        row = {"B": 1, "H": bh, "N": N, "d": d, "mask": "causal" if causal else "full"}
        row.update({s: round(best[s], 1) for s in scheds})
        print(json.dumps(row), flush=True)
        del tensors, qg, kg, vg, dog, og, lseg, dq, dk, dv, ws
        torch.cuda.empty_cache()
    return 0


if __name__ == "__main__":
    sys.exit(main(*sys.argv[1:]))
