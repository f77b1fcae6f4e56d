"""Benchmark: deterministic attention backward on one MI355X.

One step = one full backward call (D = rowsum(dO o O) preprocessing + the main
kernel with the ordered dQ reduction) over the whole batch of the workload
B=2, H=16, N=8192, d=128, full mask (16384 tokens, hidden 2048), inputs bf16
~N(0,1), already resident in HBM.  Reports, as one JSON line:

  value        backward TFLOPS of the deterministic Shift schedule
               (FLOPs = 4*B*H*N^2*d*2.5, the five-GEMM count)
  pct_of_atomic that throughput as a percentage of the atomic-add variant's
  roofline     the main kernel's algorithmic MFMA FLOPs per launch divided by
               its mean duration (HIP events recorded by the library on the
               launch stream around that kernel), against the bf16 dense peak;
               with the per-call median and minimum of that duration
  spinup       the untimed calls run first so that the device is at its
               steady clock before the first schedule's warm-up
  cpu_baseline the fp64 oracle timed on the host on one full head of the
               same workload, scaled to the same FLOP count
"""
from __future__ import annotations

import argparse
import ctypes
import json
import os
import statistics
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0  # MI355X dense bf16 MFMA


class HipEvents:
    """hipEvent_t pairs via the HIP runtime (for events on the library stream)."""

    def __init__(self):
        self.hip = ctypes.CDLL("libamdhip64.so")
        self.hip.hipEventCreate.argtypes = [ctypes.POINTER(ctypes.c_void_p)]
        self.hip.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p,
                                                 ctypes.c_void_p]
        self.hip.hipEventDestroy.argtypes = [ctypes.c_void_p]

    def create(self):
        e = ctypes.c_void_p()
        assert self.hip.hipEventCreate(ctypes.byref(e)) == 0
        return e

    def elapsed_ms(self, a, b):
        ms = ctypes.c_float()
        assert self.hip.hipEventElapsedTime(ctypes.byref(ms), a, b) == 0
        return ms.value

    def destroy(self, e):
        self.hip.hipEventDestroy(e)


def time_schedule(dash, tensors, causal, sched, steps, warmup, ev, samples=None):
    """Mean wall-clock ms per call over `steps` back-to-back calls, and the mean
    main-kernel ms from HIP events around each call's main kernel (appended
    per call to `samples` when given)."""
    import torch
    q, k, v, o, do, lse, dq, dk, dv, ws = tensors
    for _ in range(warmup):  # each warm-up call is checked (the check synchronizes)
        dash.dash_attn_bwd(q, k, v, o, do, lse, dq, dk, dv, causal, sched, workspace=ws)
        if dash.dash_bwd_check(ws) != dash.DASH_OK:
            raise RuntimeError(f"{sched}: ordering wait timed out (warm-up)")
    pairs = [(ev.create(), ev.create()) for _ in range(steps)]
    opts = [dash.dash_bwd_options_t(0, 0, None, None, None, a.value, b.value) for a, b in pairs]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(steps):
        dash.dash_attn_bwd(q, k, v, o, do, lse, dq, dk, dv, causal, sched, workspace=ws, options=opts[i])
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    if dash.dash_bwd_check(ws) != dash.DASH_OK:
        raise RuntimeError(f"{sched}: ordering wait timed out")
    main_ms = [ev.elapsed_ms(a, b) for a, b in pairs]
    if samples is not None:
        samples.extend(main_ms)
    for a, b in pairs:
        ev.destroy(a)
        ev.destroy(b)
    return wall * 1e3 / steps, sum(main_ms) / len(main_ms)


def spin_up(dash, tensors, causal, sched, ms_target):
    """Untimed backward calls until the device has run them for ms_target ms.
    A device that has been idle starts below its steady clock: without this
    the first schedule timed pays for the ramp (a 2 ms call measured 5-7%
    slower after a 3-call warm-up than after a 10-call one).  Returns the
    number of calls made."""
    import torch
    q, k, v, o, do, lse, dq, dk, dv, ws = tensors
    calls, t0 = 0, time.perf_counter()
    while (time.perf_counter() - t0) * 1e3 < ms_target:
        dash.dash_attn_bwd(q, k, v, o, do, lse, dq, dk, dv, causal, sched, workspace=ws)
        torch.cuda.synchronize()
        calls += 1
    return calls


def ordering_wait(dash, tensors, causal, sched, B, H, N, d):
    """One instrumented (untimed) call: the share of the main kernel's
    wave-time spent waiting for a dQ turn, and the share of wave-steps whose
    turn was not yet visible one step ahead (those waited)."""
    import torch
    q, k, v, o, do, lse, dq, dk, dv, ws = tensors
    stats = torch.zeros(3, dtype=torch.int64, device=q.device)
    opts = dash.dash_bwd_options_t(0, 0, None, None, None, None, None, 0, 0, 0, stats.data_ptr())
    dash.dash_attn_bwd(q, k, v, o, do, lse, dq, dk, dv, causal, sched, workspace=ws, options=opts)
    if dash.dash_bwd_check(ws) != dash.DASH_OK:
        raise RuntimeError(f"{sched}: ordering wait timed out (instrumented call)")
    late, wait_ticks, wave_ticks = (int(x) for x in stats.cpu())
    tab = dash.dash_schedule_table(sched, N, d, causal, heads=B * H)
    wave_steps = 4 * B * H * int(tab["chain_len"].sum()) * (tab["br"] // 64)  # 64-row steps, 4 waves
    return {"stall_frac": round(wait_ticks / wave_ticks, 4) if wave_ticks > 0 else None,
            "late_wave_steps": late, "wave_steps": wave_steps,
            "late_frac": round(late / wave_steps, 4) if wave_steps else None}


def measured_traffic():
    """HBM bytes per launch of the main kernel from the committed rocprofv3
    FETCH_SIZE / WRITE_SIZE summary, or None if the kernel source changed since
    the counters were taken."""
    import hashlib
    summary = os.path.join(ROOT, "profiles", "bwd_main_b2h16n8192d128_full.md")
    try:
        text = open(summary).read()
        fields = dict(line.split(": ", 1) for line in text.splitlines() if ": " in line and not line.startswith(" "))
        src = os.path.join(ROOT, fields["source_file"].strip())
        sha = hashlib.sha256(open(src, "rb").read()).hexdigest()[:16]
    except (OSError, KeyError):
        return None
    if fields.get("source_sha256_prefix", "").strip() != sha:
        return None
    return float(fields["traffic_bytes_per_launch"])


def cpu_baseline(q, k, v, do, causal, flops_per_head):
    """The oracle, as it is, on whole heads of the workload taken in order until
    at least 10 s of CPU work (at most 6 heads)."""
    import oracle
    threads = int(os.environ.get("OMP_NUM_THREADS", "0")) or len(os.sched_getaffinity(0))
    os.environ.setdefault("OMP_NUM_THREADS", str(threads))
    B, H = q.shape[0], q.shape[1]
    heads, t0 = 0, time.perf_counter()
    while heads < min(6, B * H):
        b, h = divmod(heads, H)
        oracle.attn_bwd(q[b, h], k[b, h], v[b, h], do[b, h], causal)
        heads += 1
        if time.perf_counter() - t0 >= 10.0:
            break
    dt = time.perf_counter() - t0
    model = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            model = next((ln.split(":", 1)[1].strip() for ln in f if ln.startswith("model name")), model)
    except OSError:
        pass
    return {"value": heads * flops_per_head / dt / 1e12, "unit": "TFLOPS", "cores": threads, "kind": "oracle",
            "cpu_model": model,
            "sample": f"{heads} full head(s) of the workload in order from (b=0,h=0), fp64 forward recompute "
                      f"+ dQ/dK/dV, {dt:.1f} s; FLOPs counted as 4*N^2*d*2.5 per head (halved for causal)"}


def sweep(dash, make_inputs, args):
    import torch
    ev = HipEvents()
    ns = (512, 1024, 2048, 4096, 8192, 16384)
    cases = [(16384 // n, 16, n, 128, False) for n in ns]
    cases += [(16384 // n, 32, n, 128, True) for n in ns]
    cases += [(16384 // n, 32, n, 64, False) for n in ns]  # head dim 64, hidden 2048
    cases += [(16384 // n, 32, n, 64, True) for n in ns]
    cases += [(4, 16, 1024, 64, True)]
    cases += [(1, 8, 32768, 256, False), (1, 8, 32768, 256, True)]  # long sequence, head dim 256
    for B, H, N, d, causal in cases:
        flops = 4.0 * B * H * N * N * d * 2.5 / (2 if causal else 1)
        q, k, v, do = make_inputs(B, H, N, d, seed=N + d, sigma=0.5 if d == 256 else 1.0)
        qg, kg, vg, dog = (t.cuda() for t in (q, k, v, do))
        og, lseg = dash.attn_fwd(qg, kg, vg, causal)
        dq, dk, dv = torch.empty_like(qg), torch.empty_like(kg), torch.empty_like(vg)
        scheds = ("descending", "symshift", "naive", "atomic") if causal else ("shift", "descending", "naive", "atomic")
        if d <= 128:  # the comparison designs are built for d = 64, 128
            scheds += ("split", "partials")
        ws = dash.new_workspace(B, H, N, d, "partials" if "partials" in scheds else "shift")
        tensors = (qg, kg, vg, og, dog, lseg, dq, dk, dv, ws)
        row = {"B": B, "H": H, "N": N, "d": d, "mask": "causal" if causal else "full"}
        if (B, H, N, d, causal) == cases[0]:
            spin_up(dash, tensors, causal, scheds[0], args.spinup_ms)
        # every schedule timed twice, in opposite orders, the faster kept: a
        # rare stall of the host or the device costs one timing, not the row
        for order in (scheds, scheds[::-1]):
            for sched in order:
                ms, main_ms = time_schedule(dash, tensors, causal, sched, args.steps, args.warmup, ev)
                row[sched] = max(row.get(sched, 0.0), round(flops / (ms * 1e-3) / 1e12, 1))
        det = max(row[s] for s in scheds if s not in ("atomic", "split", "partials"))
        row["best_det_pct_of_atomic"] = round(100 * det / row["atomic"], 1)
        print(json.dumps(row), flush=True)
        del tensors, qg, kg, vg, dog, og, lseg, dq, dk, dv, ws
        torch.cuda.empty_cache()


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--spinup-ms", type=float, default=200.0,
                    help="before the first schedule's warm-up, untimed calls for this long (device clock ramp)")
    ap.add_argument("--schedule", default="shift")
    ap.add_argument("--no-cpu", action="store_true", help="skip the oracle CPU baseline")
    ap.add_argument("--N", type=int, default=8192)
    ap.add_argument("--causal", action="store_true")
    ap.add_argument("--d", type=int, default=128,
                    help="head dim; 256 selects the long-sequence workload B=1 H=8 (inputs ~N(0, 0.5^2))")
    ap.add_argument("--schedules", default="",
                    help="comma list of schedules to time (default: the schedule, atomic, naive)")
    ap.add_argument("--sweep", action="store_true",
                    help="time every schedule over the 16k-token sweeps (d=128: full H=16, causal H=32; "
                         "d=64: H=32, both masks), the B=4 H=16 N=1024 d=64 causal case and B=1 H=8 "
                         "N=32768 d=256 (both masks), twice in opposite orders (the faster kept); "
                         "one JSON line per case")
    ap.add_argument("--copy-bytes", type=int, default=0,
                    help="only run 5 plain device copies of this many bytes (counter calibration)")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py measures one GPU: the backward shards over heads with no communication, "
              "so a run on N GPUs is N independent single-GPU runs; use --gpus 1", file=sys.stderr)
        sys.exit(2)

    import torch

    if args.copy_bytes:
        src = torch.empty(args.copy_bytes, dtype=torch.uint8, device="cuda").fill_(1)
        dst = torch.empty_like(src)
        for _ in range(5):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_bytes": args.copy_bytes, "copies": 5}))
        return

    from paper_2601_21824_amd import binding as dash
    from paper_2601_21824_amd.synth import make_inputs

    dash.load()
    if args.sweep:
        sweep(dash, make_inputs, args)
        return
    N, d, causal = args.N, args.d, args.causal
    if d == 256:
        B, H, sigma = 1, 8, 0.5
    else:
        B, H, sigma = max(1, 16384 // N), (32 if causal else 16), 1.0
    flops = 4.0 * B * H * N * N * d * 2.5 / (2 if causal else 1)
    q, k, v, do = make_inputs(B, H, N, d, seed=1234, sigma=sigma)
    qg, kg, vg, dog = (t.cuda() for t in (q, k, v, do))
    og, lseg = dash.attn_fwd(qg, kg, vg, causal)
    dq, dk, dv = torch.empty_like(qg), torch.empty_like(kg), torch.empty_like(vg)
    det = args.schedule
    scheds = [x for x in args.schedules.split(",") if x] or [det, "atomic", "naive"]
    ws = dash.new_workspace(B, H, N, d, "partials" if "partials" in scheds else det)
    torch.cuda.synchronize()
    tensors = (qg, kg, vg, og, dog, lseg, dq, dk, dv, ws)
    ev = HipEvents()

    results = {}
    per_call = {}
    spin_calls = spin_up(dash, tensors, causal, scheds[0], args.spinup_ms)
    for sched in dict.fromkeys(scheds):
        per_call[sched] = []
        ms, main_ms = time_schedule(dash, tensors, causal, sched, args.steps, args.warmup, ev, per_call[sched])
        results[sched] = (ms, main_ms, flops / (ms * 1e-3) / 1e12)
        print(f"[bench] {sched}: {ms:.3f} ms/step, main kernel {main_ms:.3f} ms, "
              f"{results[sched][2]:.1f} TFLOPS", file=sys.stderr, flush=True)

    if det not in results or "atomic" not in results:
        print(json.dumps({s: {"ms_per_step": r[0], "main_kernel_ms": r[1], "tflops": r[2]}
                          for s, r in results.items()}), flush=True)
        return
    ms, main_ms, tflops = results[det]
    main_tflops = flops / (main_ms * 1e-3) / 1e12
    placement = "global" if det == "atomic" else \
        ("XCD-local" if dash.dash_bwd_placement(B, H, N, d, causal, det) == dash.DASH_PLACEMENT_XCD else "global")
    bc = dash.dash_schedule_table(det, N, d, causal, heads=B * H)["bc"]
    kname = "bwd_main256_kernel" if d == 256 else ("bwd_main64w_kernel" if bc == 256 else "bwd_main_kernel")
    out = {
        "metric": "deterministic attn-bwd TFLOPS (bf16, d=128, N=8192) + % of atomic variant",
        "value": round(tflops, 2),
        "unit": "TFLOPS",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "spinup": {"ms": args.spinup_ms, "calls": spin_calls, "schedule": scheds[0]},
        "ms_per_step": round(ms, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": f"attention backward B={B} H={H} N={N} d={d} "
                               f"{'causal' if causal else 'full'} mask, {det} schedule",
                   "B": B, "H": H, "N": N, "d": d, "mask": "causal" if causal else "full",
                   "schedule": det, "global_batch": B, "seq_len": N},
        "pct_of_atomic": round(100.0 * tflops / results["atomic"][2], 2),
        "atomic_tflops": round(results["atomic"][2], 2),
        "naive_tflops": round(results["naive"][2], 2) if "naive" in results else None,
        "roofline": {"bound": "mfma", "kernel": f"{kname}<{d}, "
                               f"{'causal' if causal else 'full'} mask, {'atomic' if det == 'atomic' else 'ordered'}>"
                               f", placement {placement}",
                     "achieved": round(main_tflops, 2), "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                     "frac": round(main_tflops / PEAK_BF16_TFLOPS, 4),
                     "traffic": measured_traffic() if (N, d, causal, det) == (8192, 128, False, "shift") else None,
                     "main_kernel_ms": round(main_ms, 4),
                     "main_kernel_ms_median": round(statistics.median(per_call[det]), 4),
                     "main_kernel_ms_min": round(min(per_call[det]), 4)},
    }
    # the measured MFMA peak of this device beside the published one
    measured = dash.dash_mfma_peak()
    out["roofline"]["measured_peak"] = round(measured, 1)
    out["roofline"]["frac_of_measured"] = round(main_tflops / measured, 4) if measured > 0 else None
    # the ordering wait, measured in an extra instrumented call per ordered schedule
    out["ordering_wait"] = {s_: ordering_wait(dash, tensors, causal, s_, B, H, N, d)
                            for s_ in results if s_ not in ("atomic", "split", "partials")}
    if not args.no_cpu:
        out["cpu_baseline"] = cpu_baseline(q, k, v, do, causal, flops / (B * H))
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
