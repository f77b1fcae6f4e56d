"""Ordering-wait statistics of the main kernel (the `wait_stats` option):
an instrumented call gives the same bits as a plain one, and its counters
stay within what they count."""
import pytest
import torch

from gpu_util import inputs, run_bwd, run_fwd
from paper_2601_21824_amd import binding as dash

pytestmark = pytest.mark.gpu

STAT_CASES = [  # (B, H, N, d, causal, schedule, placement)
    (2, 4, 2048, 128, False, "shift", 0),
    (2, 4, 2048, 128, False, "naive", 0),
    (2, 4, 2048, 128, True, "descending", 0),
    (2, 4, 1024, 64, True, "symshift", 0),
    (2, 8, 2048, 128, False, "shift", 2),
    (1, 2, 1024, 256, True, "descending", 0),
    (1, 2, 1024, 256, False, "naive", 2),
]


@pytest.mark.parametrize("case", STAT_CASES, ids=[f"N{c[2]}d{c[3]}{'c' if c[4] else 'f'}-{c[5]}{'-xcd' if c[6] else ''}"
                                                  for c in STAT_CASES])
def test_wait_stats(case):
    B, H, N, d, causal, sched, place = case
    print(f"\n[wait_stats] {case}", flush=True)
    _, _, _, _, (qg, kg, vg, dog) = inputs(B, H, N, d, seed=5)
    og, lseg = run_fwd(qg, kg, vg, causal)
    ws = dash.new_workspace(B, H, N, d, sched)
    plain = run_bwd(qg, kg, vg, og, dog, lseg, causal, sched, workspace=ws,
                    options=dash.dash_bwd_options_t(0, 0, None, None, None, None, None, 0, 0, place))
    stats = torch.zeros(3, dtype=torch.int64, device="cuda")
    opts = dash.dash_bwd_options_t(0, 0, None, None, None, None, None, 0, 0, place, stats.data_ptr())
    inst = run_bwd(qg, kg, vg, og, dog, lseg, causal, sched, workspace=ws, options=opts)
    assert dash.dash_bwd_check(ws) == dash.DASH_OK
    for a, b in zip(plain, inst):
        assert torch.equal(a.view(torch.int16), b.view(torch.int16))
    late, wait_ticks, wave_ticks = (int(x) for x in stats.cpu())
    tab = dash.dash_schedule_table(sched, N, d, causal, place or dash.DASH_PLACEMENT_GLOBAL, heads=B * H)
    sub = tab["br"] // 64  # kernel steps (64-row blocks) per scheduled Q tile
    wave_steps = 4 * B * H * int(tab["chain_len"].sum()) * sub
    # a block's first contributor (rank 0) always sees its turn early: every
    # 64-row dQ block has one, and each of its 4 waves counts separately
    assert 0 <= late <= wave_steps - 4 * B * H * tab["t_r"] * sub
    assert wave_ticks > 0 and 0 <= wait_ticks <= wave_ticks

def test_wait_stats_untouched_by_the_atomic_variant():
    B, H, N, d, causal = 1, 2, 1024, 128, False
    _, _, _, _, (qg, kg, vg, dog) = inputs(B, H, N, d, seed=6)
    og, lseg = run_fwd(qg, kg, vg, causal)
    stats = torch.zeros(3, dtype=torch.int64, device="cuda")
    opts = dash.dash_bwd_options_t(0, 0, None, None, None, None, None, 0, 0, 0, stats.data_ptr())
    run_bwd(qg, kg, vg, og, dog, lseg, causal, "atomic", options=opts)
    assert stats.cpu().tolist() == [0, 0, 0]
