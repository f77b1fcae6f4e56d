"""GPU tests of the ordered reduction itself: bitwise run-to-run determinism,
the ordering witness against the oracle's accumulation order, an exact replay
of the fp32 summation from the exported partials, NAIVE == DESCENDING on dQ,
and the wait watchdog (forced from the host)."""
import numpy as np
import pytest
import torch

import oracle
from oracle import schedule as osched
from gpu_util import inputs, run_bwd, run_fwd
from paper_2601_21824_amd import binding as dash

pytestmark = pytest.mark.gpu

DET_CASES = [  # (B, H, N, d, causal, schedule[, placement])
    (4, 16, 1024, 64, True, "naive"),
    (4, 16, 1024, 64, True, "descending"),
    (4, 16, 1024, 64, True, "symshift"),
    (1, 1, 256, 64, False, "shift"),
    (2, 4, 2048, 128, False, "shift"),
    (2, 4, 2048, 128, False, "naive"),
    (2, 4, 2048, 128, True, "descending"),
    (2, 4, 2048, 128, True, "symshift"),
    (1, 2, 1024, 256, False, "shift"),
    (1, 2, 1024, 256, True, "symshift"),
    (2, 4, 2048, 128, True, "split"),
    (2, 4, 2048, 128, False, "partials"),
    # XCD-local placement: several workgroups of one head on each XCD read
    # the accumulator slots that the others wrote just before
    (4, 16, 1024, 64, True, "descending", 2),
    (4, 16, 1024, 64, True, "naive", 2),
    (2, 8, 2048, 128, False, "shift", 2),
    (2, 8, 1024, 256, True, "naive", 2),
    # the full-size workloads: the benchmark's Shift (16384 tokens, 16 heads
    # of 128, full mask) and the causal schedules at N = 8192 (32 heads of 128)
    (2, 16, 8192, 128, False, "shift"),
    (2, 32, 8192, 128, True, "descending"),
    (2, 32, 8192, 128, True, "symshift"),
    # the long-sequence workload (8 heads of 32768 rows at d = 256): Symmetric
    # Shift's 256 chains per head change KV tiles half way, releasing the
    # block before the switch at the end of the tile
    (1, 8, 32768, 256, True, "symshift"),
    # d = 64 with 256-row KV tiles
    (1, 128, 400, 64, False, "shift"),
    (1, 128, 2100, 64, True, "descending"),
    (1, 128, 2100, 64, True, "symshift"),
    (2, 64, 1030, 64, True, "descending"),
    (2, 32, 8192, 64, False, "shift"),
]


@pytest.mark.parametrize("case", DET_CASES, ids=[f"N{c[2]}d{c[3]}{'c' if c[4] else 'f'}-{c[5]}{'-xcd' if c[6:] == (2,) else ''}"
                                                 for c in DET_CASES])
def test_bitwise_identical_over_100_runs(case):
    B, H, N, d, causal, sched = case[:6]
    opts = dash.dash_bwd_options_t(0, 0, None, None, None, None, None, 0, 0, case[6]) if len(case) > 6 else None
    print(f"\n[determinism] {case}", flush=True)
    _, _, _, _, (qg, kg, vg, dog) = inputs(B, H, N, d, seed=77)
    og, lseg = run_fwd(qg, kg, vg, causal)
    ws = dash.new_workspace(B, H, N, d, sched)
    first = run_bwd(qg, kg, vg, og, dog, lseg, causal, sched, workspace=ws, options=opts)
    outs = [torch.empty_like(t) for t in first]
    for r in range(99):
        dash.dash_attn_bwd(qg, kg, vg, og, dog, lseg, *outs, causal, sched, workspace=ws, options=opts)
        torch.cuda.synchronize()
        for a, b in zip(first, outs):
            assert torch.equal(a.view(torch.int16), b.view(torch.int16)), f"run {r + 2} differs"
    assert dash.dash_bwd_check(ws) == dash.DASH_OK


SERIAL_CASES = [
    (1, 8, 32768, 256, False, "naive"),
    (1, 8, 32768, 256, False, "descending"),
    (1, 8, 32768, 256, True, "naive"),
    (1, 8, 32768, 256, True, "descending"),
    (1, 16, 16384, 128, True, "naive"),
]


@pytest.mark.parametrize("case", SERIAL_CASES, ids=[f"N{c[2]}d{c[3]}{'c' if c[4] else 'f'}-{c[5]}" for c in SERIAL_CASES])
def test_serialized_schedules_never_miss_a_turn(case):
    """Naive and Descending wait at almost every step, with more chains than
    resident workgroups at these lengths.  All waves of a workgroup share the
    contributor's rank and each bumps the counter after its own slice, so a
    wave that polls after a sibling's bump must still take its turn: every call
    completes without a wait timeout and gives the same bits."""
    B, H, N, d, causal, sched = case
    print(f"\n[serialized] {case}", flush=True)
    _, _, _, _, (qg, kg, vg, dog) = inputs(B, H, N, d, seed=5, sigma=0.5)
    og, lseg = run_fwd(qg, kg, vg, causal)
    ws = dash.new_workspace(B, H, N, d, sched)
    opts = dash.dash_bwd_options_t(1 << 20, 0, None, None, None, None, None, 0)
    first = run_bwd(qg, kg, vg, og, dog, lseg, causal, sched, workspace=ws, options=opts)
    assert dash.dash_bwd_check(ws) == dash.DASH_OK
    outs = [torch.empty_like(t) for t in first]
    for r in range(7):
        dash.dash_attn_bwd(qg, kg, vg, og, dog, lseg, *outs, causal, sched, workspace=ws, options=opts)
        assert dash.dash_bwd_check(ws) == dash.DASH_OK, f"call {r + 2} timed out"
        for a, b in zip(first, outs):
            assert torch.equal(a.view(torch.int16), b.view(torch.int16)), f"call {r + 2} differs"


def test_symmetric_shift_releases_before_its_tile_switch():
    """A Symmetric Shift chain changes KV tiles once, after the upper-left
    triangle.  The block it finishes just before the switch is released at
    once, not after the switch's dK/dV stores and K/V loads: held back, that
    release made every later contributor of a Q tile in the triangle wait for
    its predecessor's switch in turn, and the waits grew along the line
    (9.6% of the wave time at B=2 H=32 N=8192 d=128; 0.6% since).  Checked
    through the instrumented kernel's ordering-wait share, with a margin."""
    B, H, N, d = 2, 32, 8192, 128
    print(f"\n[symshift waits] B={B} H={H} N={N} d={d}", flush=True)
    _, _, _, _, (qg, kg, vg, dog) = inputs(B, H, N, d, seed=9)
    og, lseg = run_fwd(qg, kg, vg, True)
    ws = dash.new_workspace(B, H, N, d, "symshift")
    for _ in range(5):  # device clock up
        run_bwd(qg, kg, vg, og, dog, lseg, True, "symshift", workspace=ws)
    stats = torch.zeros(3, dtype=torch.int64, device="cuda")
    opts = dash.dash_bwd_options_t(0, 0, None, None, None, None, None, 0, 0, 0, stats.data_ptr())
    run_bwd(qg, kg, vg, og, dog, lseg, True, "symshift", workspace=ws, options=opts)
    assert dash.dash_bwd_check(ws) == dash.DASH_OK
    late, wait_ticks, wave_ticks = (int(x) for x in stats.cpu())
    assert wave_ticks > 0
    share = wait_ticks / wave_ticks
    print(f"[symshift waits] wait share {share:.4f}, late wave-steps {late}", flush=True)
    assert share < 0.04, f"Symmetric Shift waits {share:.1%} of its wave time"


@pytest.mark.parametrize("N,d", [(1024, 64), (2048, 128)])
def test_naive_and_descending_give_identical_dq(N, d):
    """Both sum every dQ tile in ascending KV order from identical partials."""
    B, H = 2, 4
    _, _, _, _, (qg, kg, vg, dog) = inputs(B, H, N, d, seed=9)
    og, lseg = run_fwd(qg, kg, vg, True)
    dq1, _, _ = run_bwd(qg, kg, vg, og, dog, lseg, True, "naive")
    dq2, _, _ = run_bwd(qg, kg, vg, og, dog, lseg, True, "descending")
    assert torch.equal(dq1.view(torch.int16), dq2.view(torch.int16))


@pytest.mark.parametrize("N,d,causal", [(1024, 64, True), (333, 64, False), (2048, 128, False), (1000, 128, True)])
def test_partials_variant_equals_naive_bitwise(N, d, causal):
    """The materialized-partials comparison variant sums the same partials in
    the same (ascending KV) order as NAIVE's counters: identical dQ, and dK,
    dV identical too (same chains)."""
    B, H = 2, 3
    _, _, _, _, (qg, kg, vg, dog) = inputs(B, H, N, d, seed=19)
    og, lseg = run_fwd(qg, kg, vg, causal)
    ref = run_bwd(qg, kg, vg, og, dog, lseg, causal, "naive")
    got = run_bwd(qg, kg, vg, og, dog, lseg, causal, "partials")
    for a_, b_ in zip(ref, got):
        assert torch.equal(a_.view(torch.int16), b_.view(torch.int16))


GL, XL = 1, 2  # DASH_PLACEMENT_GLOBAL, DASH_PLACEMENT_XCD
PROTO_CASES = [
    (1, 2, 512, 128, False, "shift", GL),
    (1, 2, 512, 128, False, "naive", GL),
    (1, 2, 576, 64, True, "symshift", GL),
    (1, 2, 512, 128, True, "symshift", GL),
    (1, 2, 512, 128, True, "descending", GL),
    (2, 1, 300, 64, True, "symshift", GL),
    (2, 1, 300, 128, False, "shift", GL),
    (1, 2, 512, 256, False, "shift", GL),
    (1, 2, 512, 256, True, "symshift", GL),
    (1, 1, 333, 256, True, "descending", GL),
    # d = 64 with 256-row KV tiles (enough of them over the call's heads)
    (1, 128, 400, 64, False, "shift", GL),
    (1, 128, 2048, 64, True, "symshift", GL),
    # every chain of a head on one XCD; at 33 KV tiles
    # Shift runs as two groups, 32 chains then 1
    (1, 2, 4224, 128, False, "shift", XL),
    (3, 3, 700, 64, False, "shift", XL),
    (1, 2, 576, 64, True, "symshift", XL),
    (2, 5, 512, 128, True, "descending", XL),
    (2, 1, 300, 128, False, "naive", XL),
]


@pytest.mark.parametrize("case", PROTO_CASES,
                         ids=[f"N{c[2]}d{c[3]}{'c' if c[4] else 'f'}-{c[5]}-{'xcd' if c[6] == XL else 'global'}"
                              for c in PROTO_CASES])
def test_witness_and_partial_sum_replay(case):
    """The order the workgroups actually added their partials in equals the
    oracle's order, and summing the exported partials in that order in fp32
    reproduces the accumulator bit for bit (and dQ = bf16(scale * acc))."""
    B, H, N, d, causal, sched, placement = case
    print(f"\n[protocol] {case}", flush=True)
    _, _, _, _, (qg, kg, vg, dog) = inputs(B, H, N, d, seed=21)
    og, lseg = run_fwd(qg, kg, vg, causal)
    nblk = (N + 63) // 64
    tab = dash.dash_schedule_table(sched, N, d, causal, placement, heads=B * H)
    tc = (N + tab["bc"] - 1) // tab["bc"]  # KV tiles (before Symmetric Shift's padding)
    witness = torch.full((B * H, nblk, tc), -1, dtype=torch.int32, device="cuda")
    partials = torch.full((B * H, tc, N, d), float("nan"), dtype=torch.float32, device="cuda")
    acc = torch.full((B * H, N, d), float("nan"), dtype=torch.float32, device="cuda")
    opts = dash.dash_bwd_options_t(0, 0, witness.data_ptr(), partials.data_ptr(), acc.data_ptr(), None, None,
                                   0, 0, placement)
    dq, dk, dv = run_bwd(qg, kg, vg, og, dog, lseg, causal, sched, options=opts)
    kind = {"shift": osched.SHIFT, "naive": osched.NAIVE, "descending": osched.DESCENDING,
            "symshift": osched.SYMSHIFT}[sched]
    ref = osched.build(kind, tab["t_r"], tab["t_c"], causal, tab["br"], tab["bc"],
                       group=tab["group"] if kind == osched.SHIFT else None)
    nsub = tab["br"] // 64
    W = witness.cpu().numpy()
    P = partials.cpu().numpy()
    A = acc.cpu().numpy()
    scale = np.float32(1.0 / np.sqrt(d))
    for bh in range(B * H):
        for pb in range(nblk):
            order = [j for j in ref.order[pb // nsub] if j < tc]
            assert W[bh, pb, :len(order)].tolist() == order, (bh, pb)
            assert (W[bh, pb, len(order):] == -1).all()
            rows = slice(pb * 64, min(N, pb * 64 + 64))
            want = oracle.ordered_sum_f32([P[bh, j, rows] for j in order])
            assert np.array_equal(want.view(np.int32), A[bh, rows].view(np.int32)), (bh, pb)
    want_dq = torch.from_numpy(A * scale).to(torch.bfloat16)
    assert torch.equal(want_dq.view(torch.int16), dq.cpu().reshape(B * H, N, d).view(torch.int16))


GRID_CASES = [
    (2, 4, 2048, 128, False, "shift"),
    (2, 4, 2048, 128, False, "naive"),
    (2, 4, 2048, 128, True, "symshift"),
    (2, 4, 2048, 128, True, "descending"),
    (2, 8, 1024, 64, True, "symshift"),
]


@pytest.mark.parametrize("case", GRID_CASES, ids=[f"N{c[2]}d{c[3]}{'c' if c[4] else 'f'}-{c[5]}" for c in GRID_CASES])
def test_grid_size_does_not_change_bits(case):
    """The summation order is a function of the schedule, shape and placement
    only: the persistent grid's size (from the chains that must run at once --
    per XCD under XCD-local placement -- up to the GPU's resident count)
    leaves every output bit unchanged; below that the call is rejected."""
    B, H, N, d, causal, sched = case
    print(f"\n[grid] {case}", flush=True)
    _, _, _, _, (qg, kg, vg, dog) = inputs(B, H, N, d, seed=31)
    og, lseg = run_fwd(qg, kg, vg, causal)
    ws = dash.new_workspace(B, H, N, d)
    for place, queues in ((GL, 1), (XL, 8)):  # MI355X: 8 XCDs, one queue each
        tab = dash.dash_schedule_table(sched, N, d, causal, place, heads=B * H)
        together = (tab["group"] if sched in ("shift", "symshift") else 1) * queues
        opts = lambda cap: dash.dash_bwd_options_t(0, 0, None, None, None, None, None, cap, 0, place)
        ref = run_bwd(qg, kg, vg, og, dog, lseg, causal, sched, workspace=ws, options=opts(0))
        for cap in (max(together, 2), together + 3, 2 * together + 1):
            got = run_bwd(qg, kg, vg, og, dog, lseg, causal, sched, options=opts(cap), workspace=ws)
            assert dash.dash_bwd_check(ws) == dash.DASH_OK
            for a, b in zip(ref, got):
                assert torch.equal(a.view(torch.int16), b.view(torch.int16)), f"placement {place} grid {cap} differs"
        if together > 1:
            with pytest.raises(dash.DashError) as e:
                run_bwd(qg, kg, vg, og, dog, lseg, causal, sched, workspace=ws, options=opts(together - 1))
            assert e.value.code == dash.DASH_ERR_INVALID_ARG


TICKET_CASES = [
    (2, 4, 2048, 128, True, "naive"),
    (2, 4, 2048, 128, True, "descending"),
    (2, 4, 2048, 128, False, "naive"),
    (1, 4, 4096, 256, True, "descending"),
    (1, 4, 4096, 256, True, "naive"),
    (4, 8, 1024, 64, True, "descending"),
    (2, 4, 2048, 128, True, "split"),
    (2, 4, 2048, 128, True, "partials"),
]


@pytest.mark.parametrize("case", TICKET_CASES, ids=[f"N{c[2]}d{c[3]}{'c' if c[4] else 'f'}-{c[5]}" for c in TICKET_CASES])
def test_ticket_order_does_not_change_bits(case):
    """Head-major and chain-major work tickets (with the GPU's resident grid
    and with three workgroups) give the same bits as the default order; Shift
    and Symmetric Shift refuse chain-major tickets."""
    B, H, N, d, causal, sched = case
    print(f"\n[tickets] {case}", flush=True)
    _, _, _, _, (qg, kg, vg, dog) = inputs(B, H, N, d, seed=19)
    og, lseg = run_fwd(qg, kg, vg, causal)
    ws = dash.new_workspace(B, H, N, d, sched)
    ref = run_bwd(qg, kg, vg, og, dog, lseg, causal, sched, workspace=ws)
    for order in (dash.DASH_TICKETS_HEAD_MAJOR, dash.DASH_TICKETS_CHAIN_MAJOR):
        for cap in (0, 3):
            opts = dash.dash_bwd_options_t(0, 0, None, None, None, None, None, cap, order)
            got = run_bwd(qg, kg, vg, og, dog, lseg, causal, sched, options=opts, workspace=ws)
            assert dash.dash_bwd_check(ws) == dash.DASH_OK
            for a, b in zip(ref, got):
                assert torch.equal(a.view(torch.int16), b.view(torch.int16)), f"order {order} grid {cap} differs"
    for s in ("shift", "symshift") if causal else ("shift",):
        with pytest.raises(dash.DashError) as e:
            run_bwd(qg, kg, vg, og, dog, lseg, causal, s, workspace=dash.new_workspace(B, H, N, d, s),
                    options=dash.dash_bwd_options_t(0, 0, None, None, None, None, None, 0,
                                                    dash.DASH_TICKETS_CHAIN_MAJOR))
        assert e.value.code == dash.DASH_ERR_INVALID_ARG


PLACE_CASES = [
    (2, 8, 2048, 128, False, "naive"),
    (2, 8, 2048, 128, True, "descending"),
    (2, 8, 4096, 128, False, "shift"),
    (2, 8, 2048, 128, True, "symshift"),
    (4, 4, 1024, 64, True, "symshift"),
    (1, 8, 8192, 64, True, "descending"),
    (2, 4, 6144, 128, False, "shift"),
    (1, 8, 4096, 256, False, "shift"),
    (1, 8, 2048, 256, True, "descending"),
    (2, 4, 2048, 256, True, "symshift"),
    # d = 64 with 256-row KV tiles (64 heads x 8 tiles)
    (2, 32, 2048, 64, False, "shift"),
    (2, 32, 2048, 64, False, "naive"),
    (1, 128, 2048, 64, True, "descending"),
    # causal d = 64 at N = 1024 with 256-row tiles (128 heads x 4 tiles)
    (1, 128, 1024, 64, True, "symshift"),
    (1, 128, 1024, 64, True, "naive"),
]


@pytest.mark.parametrize("case", PLACE_CASES, ids=[f"B{c[0]}H{c[1]}N{c[2]}d{c[3]}{'c' if c[4] else 'f'}-{c[5]}"
                                                    for c in PLACE_CASES])
def test_placement(case):
    """XCD-local placement (each head's chains on one XCD, from that XCD's
    ticket queue) against one global queue: bitwise the same result wherever
    the schedule's order does not depend on the placement (all but Shift with
    more than 32 KV tiles, whose groups shrink to 32 chains); there the
    witnessed order is the oracle's with groups of 32, and the result is
    deterministic.  AUTO is the global queue, also under a workgroup cap."""
    B, H, N, d, causal, sched = case
    print(f"\n[placement] {case}", flush=True)
    _, _, _, _, (qg, kg, vg, dog) = inputs(B, H, N, d, seed=23)
    og, lseg = run_fwd(qg, kg, vg, causal)
    ws = dash.new_workspace(B, H, N, d, sched)
    assert dash.dash_bwd_placement(B, H, N, d, causal, sched) == GL
    place = lambda p, cap=0: dash.dash_bwd_options_t(0, 0, None, None, None, None, None, cap, 0, p)
    auto = run_bwd(qg, kg, vg, og, dog, lseg, causal, sched, workspace=ws)
    assert dash.dash_bwd_check(ws) == dash.DASH_OK
    xcd = run_bwd(qg, kg, vg, og, dog, lseg, causal, sched, workspace=ws, options=place(XL))
    glob = run_bwd(qg, kg, vg, og, dog, lseg, causal, sched, workspace=ws, options=place(GL))
    assert dash.dash_bwd_check(ws) == dash.DASH_OK
    for a_, b_ in zip(auto, glob):
        assert torch.equal(a_.view(torch.int16), b_.view(torch.int16))
    tab_x = dash.dash_schedule_table(sched, N, d, causal, XL, heads=B * H)
    tab_g = dash.dash_schedule_table(sched, N, d, causal, GL, heads=B * H)
    if np.array_equal(tab_x["rank"], tab_g["rank"]):
        for a_, b_ in zip(xcd, glob):
            assert torch.equal(a_.view(torch.int16), b_.view(torch.int16))
        # a cap of 3 workgroups: the global queue, same bits
        small = run_bwd(qg, kg, vg, og, dog, lseg, causal, sched, workspace=ws, options=place(0, 3)) \
            if sched in ("naive", "descending") else None
        if small is not None:
            for a_, b_ in zip(xcd, small):
                assert torch.equal(a_.view(torch.int16), b_.view(torch.int16))
    else:
        nblk = (N + 63) // 64
        witness = torch.full((B * H, nblk, tab_x["t_c"]), -1, dtype=torch.int32, device="cuda")
        opts = dash.dash_bwd_options_t(0, 0, witness.data_ptr(), None, None, None, None, 0, 0, XL)
        again = run_bwd(qg, kg, vg, og, dog, lseg, causal, sched, workspace=ws, options=opts)
        for a_, b_ in zip(xcd, again):
            assert torch.equal(a_.view(torch.int16), b_.view(torch.int16))
        order = osched.build(osched.SHIFT, tab_x["t_r"], tab_x["t_c"], causal, tab_x["br"], tab_x["bc"],
                             group=tab_x["group"]).order
        W = witness.cpu().numpy()
        for bh in range(B * H):
            for pb in range(nblk):
                assert W[bh, pb].tolist() == order[pb], (bh, pb)
        # the groups are part of the order: a cap too small for them is rejected
        with pytest.raises(dash.DashError) as e:
            run_bwd(qg, kg, vg, og, dog, lseg, causal, sched, workspace=ws, options=place(0, 3))
        assert e.value.code == dash.DASH_ERR_INVALID_ARG


AUTO_CASES = [  # shapes at which the model picks each of the four schedules on MI355X
    (1, 32, 512, 128, False),
    (1, 2, 8192, 128, False),
    (1, 8, 2048, 128, True),
    (1, 128, 4096, 128, True),
    (1, 16, 1024, 64, True),
    (2, 3, 200, 64, True),
]


@pytest.mark.parametrize("case", AUTO_CASES, ids=[f"B{c[0]}H{c[1]}N{c[2]}d{c[3]}{'c' if c[4] else 'f'}"
                                                  for c in AUTO_CASES])
def test_auto_runs_the_model_choice(case):
    """DASH_SCHED_AUTO runs the schedule dash_auto_schedule reports for the
    device (the DAG model's pick): the same bits as that schedule called by
    name, twice; the pick is one of the mask's deterministic schedules."""
    B, H, N, d, causal = case
    pick, ms = dash.dash_auto_schedule(B, H, N, d, causal)
    allowed = (dash.DASH_SCHED_DESCENDING, dash.DASH_SCHED_NAIVE, dash.DASH_SCHED_SYMSHIFT) if causal else \
        (dash.DASH_SCHED_SHIFT, dash.DASH_SCHED_NAIVE, dash.DASH_SCHED_DESCENDING)
    assert pick in allowed and ms > 0
    print(f"\n[auto] {case} -> {pick} ({ms:.3f} ms predicted)", flush=True)
    _, _, _, _, (qg, kg, vg, dog) = inputs(B, H, N, d, seed=31)
    og, lseg = run_fwd(qg, kg, vg, causal)
    ws = dash.new_workspace(B, H, N, d, "auto")
    ref = run_bwd(qg, kg, vg, og, dog, lseg, causal, pick, workspace=ws)
    for _ in range(2):
        got = run_bwd(qg, kg, vg, og, dog, lseg, causal, "auto", workspace=ws)
        assert dash.dash_bwd_check(ws) == dash.DASH_OK
        for a_, b_ in zip(got, ref):
            assert torch.equal(a_.view(torch.int16), b_.view(torch.int16))


@pytest.mark.parametrize("d", [256])
def test_shift_groups_order_and_minimal_grid(d):
    """N = 32768 gives 512 KV tiles per head at d = 256 (64-row KV tiles), so
    full-mask Shift runs as two groups of 256 chains: the order the workgroups
    added their partials in equals the oracle's group-major order, and a grid
    of exactly one group (256 workgroups) gives the same bits as the default
    grid.  (With 128-row KV tiles, d = 64 and 128 stay within one group up to
    N = 32768.)"""
    B, H, N, causal = 1, 1, 32768, False
    print(f"\n[groups] N={N} d={d}", flush=True)
    _, _, _, _, (qg, kg, vg, dog) = inputs(B, H, N, d, seed=41, sigma=0.5)
    og, lseg = run_fwd(qg, kg, vg, causal)
    tab = dash.dash_schedule_table("shift", N, d, causal, heads=B * H)
    assert tab["t_c"] == 512 and tab["group"] == 256
    nblk = (N + 63) // 64
    witness = torch.full((B * H, nblk, tab["t_c"]), -1, dtype=torch.int32, device="cuda")
    ws = dash.new_workspace(B, H, N, d)
    opts = dash.dash_bwd_options_t(0, 0, witness.data_ptr(), None, None, None, None, 0)
    ref = run_bwd(qg, kg, vg, og, dog, lseg, causal, "shift", options=opts, workspace=ws)
    assert dash.dash_bwd_check(ws) == dash.DASH_OK
    order = osched.build(osched.SHIFT, tab["t_r"], tab["t_c"], causal, tab["br"], tab["bc"], group=256).order
    W = witness.cpu().numpy()
    nsub = tab["br"] // 64
    for pb in range(nblk):
        assert W[0, pb].tolist() == order[pb // nsub], pb
    got = run_bwd(qg, kg, vg, og, dog, lseg, causal, "shift", workspace=ws,
                  options=dash.dash_bwd_options_t(0, 0, None, None, None, None, None, 256))
    assert dash.dash_bwd_check(ws) == dash.DASH_OK
    for a_, b_ in zip(ref, got):
        assert torch.equal(a_.view(torch.int16), b_.view(torch.int16))


def test_watchdog_reports_timeout_and_library_recovers():
    """Counters poisoned from the host: every first wait times out after a few
    polls, the kernels still exit, the call reports DASH_ERR_TIMEOUT, and the
    next ordinary call is correct."""
    B, H, N, d, causal = 1, 2, 512, 64, False
    q, k, v, do, (qg, kg, vg, dog) = inputs(B, H, N, d, seed=3)
    og, lseg = run_fwd(qg, kg, vg, causal)
    ws = dash.new_workspace(B, H, N, d)
    opts = dash.dash_bwd_options_t(64, dash.DASH_FLAG_POISON_COUNTERS, None, None, None, None, None)
    dq, dk, dv = (torch.empty_like(t) for t in (qg, kg, vg))
    dash.dash_attn_bwd(qg, kg, vg, og, dog, lseg, dq, dk, dv, causal, "shift", workspace=ws, options=opts)
    assert dash.dash_bwd_check(ws) == dash.DASH_ERR_TIMEOUT
    dash.dash_attn_bwd(qg, kg, vg, og, dog, lseg, dq, dk, dv, causal, "shift", workspace=ws)
    assert dash.dash_bwd_check(ws) == dash.DASH_OK
    from gpu_util import assert_close
    rdq, rdk, rdv, _, _ = oracle.attn_bwd(q, k, v, do, causal)
    assert_close("dQ", dq, rdq)
    assert_close("dK", dk, rdk)


def test_atomic_variant_run_to_run_deviation_reported():
    """The atomic variant's run-to-run deviation is only reported (cf. Table 1):
    print the mean over runs of max |dQ_r - dQ_1|.  Every run must still match
    the oracle within the tolerance (sampled dQ, dK, dV rows of the first and
    last head), whatever order its atomic adds landed in."""
    from gpu_util import assert_close
    B, H, N, d, causal = 2, 16, 2048, 128, True
    q, k, v, do, (qg, kg, vg, dog) = inputs(B, H, N, d, seed=13)
    og, lseg = run_fwd(qg, kg, vg, causal)
    rows = np.array([0, 1, 63, 64, 1000, 2046, 2047])
    heads = ((0, 0), (B - 1, H - 1))
    refs = {bh: oracle.attn_bwd(q[bh], k[bh], v[bh], do[bh], causal, dq_rows=rows, kv_rows=rows) for bh in heads}
    ref = run_bwd(qg, kg, vg, og, dog, lseg, causal, "atomic")
    devs = []
    for r in range(10):
        out = ref if r == 0 else run_bwd(qg, kg, vg, og, dog, lseg, causal, "atomic")
        for bh in heads:
            for name, got, want in zip(("dQ", "dK", "dV"), out, refs[bh][:3]):
                assert_close(f"run {r + 1} {name} head {bh}", got[bh][rows], want[rows])
        if r:
            devs.append(float((out[0].float() - ref[0].float()).abs().max()))
    print(f"\n[atomic] mean max|dQ_r - dQ_1| over 9 runs: {np.mean(devs):.3e}", flush=True)


def test_bad_arguments_on_device():
    B, H, N, d = 1, 1, 128, 64
    _, _, _, _, (qg, kg, vg, dog) = inputs(B, H, N, d, seed=1)
    og, lseg = run_fwd(qg, kg, vg, False)
    with pytest.raises(dash.DashError) as e:
        dash.attn_bwd(qg, kg, vg, og, dog, lseg, False, "symshift")
    assert e.value.code == dash.DASH_ERR_UNSUPPORTED
    ws = torch.empty(64, dtype=torch.uint8, device="cuda")
    with pytest.raises(dash.DashError) as e:
        dash.attn_bwd(qg, kg, vg, og, dog, lseg, False, "shift", workspace=ws)
    assert e.value.code == dash.DASH_ERR_INVALID_ARG


def test_plain_form_workspace_is_cached_and_released():
    """The plain dash_attn_bwd (no workspace argument) runs on the library's
    own workspace of the current device: bitwise the result of the same
    schedule on a caller workspace, at a shape that grows the cached one, and
    again after dash_release_workspace freed it."""
    for B, H, N, d, causal, sched in ((1, 2, 512, 64, False, "shift"), (2, 4, 1500, 128, True, "descending"),
                                      (1, 2, 512, 64, False, "shift")):
        print(f"\n[plain] B={B} H={H} N={N} d={d} causal={causal} {sched}", flush=True)
        q, k, v, do, (qg, kg, vg, dog) = inputs(B, H, N, d, 77 + N)
        og, lseg = run_fwd(qg, kg, vg, causal)
        want = run_bwd(qg, kg, vg, og, dog, lseg, causal, sched, workspace=dash.new_workspace(B, H, N, d, sched))
        got = run_bwd(qg, kg, vg, og, dog, lseg, causal, sched)
        for a, b in zip(got, want):
            assert torch.equal(a, b)
        if N == 1500:
            dash.dash_release_workspace()
    dash.dash_release_workspace()


@pytest.mark.parametrize("shape", [(0, 2, 128, 64), (1, 0, 128, 128), (2, 3, 0, 256)],
                         ids=["B0", "H0", "N0"])
def test_empty_problems_are_no_ops(shape):
    """A call with no rows (B, H or N zero) returns DASH_OK in every form
    (zero-size tensors may carry null pointers) and computes nothing; given a
    workspace, it resets the workspace's error flag, so dash_bwd_check reads
    OK even on a workspace no call has used; the allocation-free form sets its
    status word to 0."""
    B, H, N, d = shape
    q = torch.empty((B, H, N, d), dtype=torch.bfloat16, device="cuda")
    o, lse = dash.attn_fwd(q, q, q, False)
    assert o.shape == q.shape and lse.shape == (B, H, N)
    for causal in (False, True):
        for sched in ("atomic", "naive", "descending", "shift", "auto") + (("partials", "split") if d <= 128 else ()):
            dash.attn_bwd(q, q, q, o, q, lse, causal, sched)
            ws = dash.new_workspace(B, H, N, d, sched)
            ws.fill_(0xA5)  # what a fresh allocation may hold: the flag reads "timed out"
            dash.attn_bwd(q, q, q, o, q, lse, causal, sched, workspace=ws)
            assert dash.dash_bwd_check(ws) == dash.DASH_OK
            status = torch.full((1,), 7, dtype=torch.int32, device="cuda")
            dash.dash_attn_bwd_noalloc(q, q, q, o, q, lse, *(torch.empty_like(q) for _ in range(3)), causal,
                                       sched, status=status)
            torch.cuda.synchronize()
            assert int(status.item()) == 0
    torch.cuda.synchronize()


_CHILD = r"""
import hashlib, sys
sys.path.insert(0, {root!r}); sys.path.insert(0, {tests!r})
import torch
from gpu_util import inputs, run_fwd, run_bwd
from paper_2601_21824_amd import binding as dash
_, _, _, _, (qg, kg, vg, dog) = inputs(2, 4, 1500, 128, 2024)
og, lseg = run_fwd(qg, kg, vg, {causal})
out = run_bwd(qg, kg, vg, og, dog, lseg, {causal}, {sched!r})
h = hashlib.sha256()
for t in (og, lseg) + tuple(out):
    h.update(t.cpu().contiguous().view(torch.uint8).numpy().tobytes())
print(h.hexdigest())
"""


@pytest.mark.parametrize("causal,sched", [(False, "naive"), (True, "descending")])
def test_bits_identical_across_processes(causal, sched):
    """The forward and backward outputs of a call hash the same in a fresh
    process as in this one: nothing in the result depends on the process
    (work tickets, allocation addresses, timing).  Schedules without a
    cooperative launch: while this process is alive, a second process's
    cooperative launch is refused on this platform (Shift and Symmetric
    Shift then fail with DASH_ERR_HIP; see dash_attn_bwd_ex)."""
    import hashlib
    import os
    import subprocess
    import sys
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    _, _, _, _, (qg, kg, vg, dog) = inputs(2, 4, 1500, 128, 2024)
    og, lseg = run_fwd(qg, kg, vg, causal)
    out = run_bwd(qg, kg, vg, og, dog, lseg, causal, sched)
    h = hashlib.sha256()
    for t in (og, lseg) + tuple(out):
        h.update(t.cpu().contiguous().view(torch.uint8).numpy().tobytes())
    code = _CHILD.format(root=root, tests=os.path.join(root, "tests"), causal=causal, sched=sched)
    p = subprocess.run([sys.executable, "-c", code], capture_output=True, text=True, timeout=240)
    assert p.returncode == 0, p.stderr[-2000:]
    assert p.stdout.strip().splitlines()[-1] == h.hexdigest()


@pytest.mark.parametrize("sched", ["naive", "descending"])
def test_concurrent_calls_on_two_streams(sched):
    """Two backward calls running at the same time on two streams, each with
    its own workspace, give the bits of the same calls run one after the
    other (the two persistent grids share the CUs; naive and Descending wait
    only on earlier tickets of their own launch)."""
    B, H, N, d = 2, 8, 2048, 128
    _, _, _, _, (qg, kg, vg, dog) = inputs(B, H, N, d, 55)
    _, _, _, _, (qg2, kg2, vg2, dog2) = inputs(B, H, N, d, 56)
    og, lseg = run_fwd(qg, kg, vg, True)
    og2, lseg2 = run_fwd(qg2, kg2, vg2, True)
    want = run_bwd(qg, kg, vg, og, dog, lseg, True, sched, workspace=dash.new_workspace(B, H, N, d, sched))
    want2 = run_bwd(qg2, kg2, vg2, og2, dog2, lseg2, True, sched, workspace=dash.new_workspace(B, H, N, d, sched))
    ws, ws2 = dash.new_workspace(B, H, N, d, sched), dash.new_workspace(B, H, N, d, sched)
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    torch.cuda.synchronize()
    with torch.cuda.stream(s1):
        got = dash.attn_bwd(qg, kg, vg, og, dog, lseg, True, sched, workspace=ws)
    with torch.cuda.stream(s2):
        got2 = dash.attn_bwd(qg2, kg2, vg2, og2, dog2, lseg2, True, sched, workspace=ws2)
    torch.cuda.synchronize()
    assert dash.dash_bwd_check(ws) == dash.DASH_OK and dash.dash_bwd_check(ws2) == dash.DASH_OK
    for a, b in zip(got + got2, want + want2):
        assert torch.equal(a, b)
