"""The library's DAG model (Section 3.1) and the DASH_SCHED_AUTO choice it drives.

* dash_model_makespan -- the library's own simulation of the DAG over the
  kernels' block steps -- equals the oracle's list-scheduling simulator
  (oracle/schedule.py) on the same schedules, expanded to 64-row blocks, for
  every ordered schedule, both masks and ticket orders, several worker counts
  and costs, including the cases where a Shift group cannot run at once.
* At every measured shape of the calibration grid the model reproduces the
  measured call time of each schedule, so AUTO picks the measured fastest.
No GPU needed: the model is host code.
"""
import itertools
import json
import os

import pytest

from oracle import schedule as sc
from oracle.schedule import Schedule
from paper_2601_21824_amd import binding as b

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
GRID = os.path.join(ROOT, "paper_2601_21824_amd", "model_grid.jsonl")
NAMES = {b.DASH_SCHED_NAIVE: "naive", b.DASH_SCHED_DESCENDING: "descending", b.DASH_SCHED_SHIFT: "shift",
         b.DASH_SCHED_SYMSHIFT: "symshift"}


def oracle_blocks(kind, n, causal, bc=128):
    """The oracle's schedule of one head at the kernels' step granularity: a
    causal scheduling tile of bc rows is two 64-row blocks with its rank order."""
    t_c = -(-n // bc)
    if causal:
        if kind == sc.SYMSHIFT:
            t_c += t_c & 1
        s = sc.build(kind, t_c, t_c, True, bc, bc)
        chains = [[(j, i2) for (j, i) in ch for i2 in (2 * i, 2 * i + 1)] for ch in s.chains]
        order = {}
        for i, js in s.order.items():
            order[2 * i] = list(js)
            order[2 * i + 1] = list(js)
        return Schedule(chains, order)
    return sc.build(kind, 2 * t_c, t_c, False, 64, bc)


CASES = [(k, c, n, h, w, cm, cost)
         for (k, c) in ((sc.NAIVE, False), (sc.DESCENDING, False), (sc.SHIFT, False),
                        (sc.NAIVE, True), (sc.DESCENDING, True), (sc.SYMSHIFT, True))
         for n, h, w, cm, cost in itertools.product((512, 1024), (1, 3), (4, 16, 64), (False, True),
                                                    ((1.0, 2.5), (0.3, 1.0)))
         if not (k in (sc.SHIFT, sc.SYMSHIFT) and cm)]


@pytest.mark.parametrize("kind,causal,n,heads,workers,chain_major,cost", CASES)
def test_model_equals_oracle_simulator(kind, causal, n, heads, workers, chain_major, cost):
    c, r = cost
    s = oracle_blocks(kind, n, causal)
    try:
        want = sc.simulate([s] * heads, workers, c, r, chain_major=chain_major)
    except sc.Deadlock:
        want = None
    tickets = b.DASH_TICKETS_CHAIN_MAJOR if chain_major else b.DASH_TICKETS_HEAD_MAJOR
    if want is None:
        with pytest.raises(b.DashError) as e:
            b.dash_model_makespan(kind, 1, heads, n, 128, causal, workers, c, r, ticket_order=tickets)
        assert e.value.code == b.DASH_ERR_UNSUPPORTED
    else:
        got = b.dash_model_makespan(kind, 1, heads, n, 128, causal, workers, c, r, ticket_order=tickets)
        assert got == pytest.approx(want, rel=1e-12, abs=1e-9)


def test_model_ragged_length():
    """Steps past N are left out, as the kernels skip them.  A full-mask head of
    130 rows at d = 128 has KV tiles 0 and 1 and blocks 0..2 (block 3 starts
    past N); naive runs both chains over blocks 0, 1, 2, and tile 1 reduces each
    block right after tile 0: one step behind, 4 steps in all."""
    one = b.dash_model_makespan("naive", 1, 1, 130, 128, False, 64, 0.0, 1.0, ticket_order=b.DASH_TICKETS_HEAD_MAJOR)
    assert one == pytest.approx(4.0)
    # the same head at 192 rows still has 3 blocks; at 193 a fourth appears
    assert b.dash_model_makespan("naive", 1, 1, 192, 128, False, 64, 0.0, 1.0) == pytest.approx(4.0)
    assert b.dash_model_makespan("naive", 1, 1, 193, 128, False, 64, 0.0, 1.0) == pytest.approx(5.0)
    # at d = 64 one head keeps 128-row tiles (4 steps); a call of 256 heads
    # takes 256-row tiles, one chain of 3 steps per head, all at once
    assert b.dash_model_makespan("naive", 1, 1, 130, 64, False, 64, 0.0, 1.0) == pytest.approx(4.0)
    assert b.dash_model_makespan("naive", 1, 256, 130, 64, False, 256, 0.0, 1.0) == pytest.approx(3.0)


EXTRAP = [(s, c, d, n, h) for s, c in (("shift", False), ("naive", False), ("descending", False), ("naive", True),
                                       ("descending", True), ("symshift", True))
          for d, n, h in ((64, 6144, 128), (64, 12288, 128), (128, 2048, 512), (128, 3072, 200), (256, 8192, 40))]


@pytest.mark.parametrize("sched,causal,d,n,heads", EXTRAP)
def test_model_extrapolation_in_heads(sched, causal, d, n, heads):
    """With max_heads the model simulates max_heads and twice that many heads
    and extrapolates linearly in the number of heads, held at or above the
    steps' own bound.  Against the simulation of every head, at the cap AUTO
    uses (three rounds of 256 workgroups): within 5%, and exact for Shift
    where a head's chains do not divide the workgroups
    (48 or 24 chains per head), the case that scaling one simulation by
    heads / max_heads overcharged by 25-30%."""
    chains = b.dash_schedule_table(sched, n, d, causal, heads=heads)["chains"]
    cap = -(-3 * 256 // chains)
    full = b.dash_model_makespan(sched, 1, heads, n, d, causal, 256, 0.02, 0.98)
    ext = b.dash_model_makespan(sched, 1, heads, n, d, causal, 256, 0.02, 0.98, max_heads=cap)
    # up to twice the cap every head is simulated
    assert ext == pytest.approx(full, rel=5e-2 if heads > 2 * cap else 1e-12)
    if sched == "shift" and n in (6144, 12288):
        assert ext == pytest.approx(full, rel=1e-12)


def test_model_head_cap_scales():
    full = b.dash_model_makespan("shift", 1, 8, 1024, 128, False, 16, 0.1, 0.9)
    capped = b.dash_model_makespan("shift", 1, 8, 1024, 128, False, 16, 0.1, 0.9, max_heads=2)
    assert capped == pytest.approx(full)  # whole rounds of 2 heads on 16 workgroups
    assert b.dash_model_makespan("shift", 1, 1, 1024, 128, False, 16, 0.0, 1.0) == pytest.approx(16.0)


def grid_rows():
    with open(GRID) as f:
        return [json.loads(x) for x in f if x.strip()]


def test_grid_covers_both_masks_and_head_dims():
    rows = grid_rows()
    assert {(r["d"], r["mask"]) for r in rows} == {(d, m) for d in (64, 128, 256) for m in ("full", "causal")}
    assert all(r["B"] * r["H"] >= 1 for r in rows)


@pytest.mark.parametrize("row", grid_rows(), ids=lambda r: f"d{r['d']}{r['mask'][0]}H{r['H']}N{r['N']}")
def test_auto_reproduces_measured_grid(row):
    """At a calibrated shape the model's prediction is the measured time of
    every schedule, so AUTO takes the measured fastest (ties: any of them)."""
    causal = row["mask"] == "causal"
    B, H, N, d = row["B"], row["H"], row["N"], row["d"]
    flops = 4.0 * B * H * N * N * d * 2.5 / (2 if causal else 1)
    sched, ms = b.dash_auto_schedule(B, H, N, d, causal, 256)
    cands = [s for s in ("shift", "symshift", "descending", "naive") if s in row]
    best = max(row[s] for s in cands)
    assert NAMES[sched] in cands
    assert row[NAMES[sched]] >= best * (1 - 1e-9)
    assert flops / (ms * 1e-3) / 1e12 == pytest.approx(best, rel=1e-3)


def test_auto_leaves_out_what_cannot_run():
    # 300 KV tiles per head: a Shift group of 256 chains needs 256 resident
    # workgroups; with 128 only naive or Descending can run
    s, _ = b.dash_auto_schedule(1, 1, 300 * 128, 128, False, 128)
    assert s in (b.DASH_SCHED_NAIVE, b.DASH_SCHED_DESCENDING)
    # an empty problem takes the mask's default
    assert b.dash_auto_schedule(0, 4, 1024, 128, True, 256) == (b.DASH_SCHED_DESCENDING, -1.0)
    assert b.dash_auto_schedule(1, 4, 0, 128, False, 256) == (b.DASH_SCHED_SHIFT, -1.0)


def test_model_argument_checks():
    for bad in (dict(workers=0), dict(c=-1.0), dict(r=float("nan"))):
        args = dict(workers=16, c=1.0, r=1.0)
        args.update(bad)
        with pytest.raises(b.DashError) as e:
            b.dash_model_makespan("naive", 1, 1, 512, 128, False, args["workers"], args["c"], args["r"])
        assert e.value.code == b.DASH_ERR_INVALID_ARG
    with pytest.raises(b.DashError):
        b.dash_model_makespan("atomic", 1, 1, 512, 128, False, 16, 1.0, 1.0)
    with pytest.raises(b.DashError):
        b.dash_model_makespan("symshift", 1, 1, 512, 128, False, 16, 1.0, 1.0)
    with pytest.raises(b.DashError):
        b.dash_auto_schedule(1, 1, 512, 96, False, 256)


def test_auto_cache_starts_over_with_the_same_answers():
    """The per-process cache of AUTO picks holds up to 4096 shapes; past that
    it is cleared, and a shape simulated again gets the same pick."""
    shapes = [(2, 16, 8192, 128, False), (2, 32, 8192, 128, True), (1, 8, 4096, 256, False)]
    first = [b.dash_auto_schedule(*s, 256) for s in shapes]
    for n in range(1, 4200):
        b.dash_auto_schedule(1, 1, n, 64, n % 2 == 1, 256)
    assert [b.dash_auto_schedule(*s, 256) for s in shapes] == first
