"""The allocation-free backward entry point (dash_attn_bwd_noalloc) against
dash_attn_bwd_ex on the same inputs: two calls in a row on the library's fixed
scratch, the second with a smaller problem, each bitwise equal to the
explicit-workspace call for the deterministic schedules (same kernels, same
summation order) and within the oracle tolerance of it for the atomic
variant; the status word is reset to 0; oversized problems are refused before
any device work."""
import ctypes

import pytest
import torch

from gpu_util import assert_close, inputs, run_fwd
from paper_2601_21824_amd import binding as dash

pytestmark = pytest.mark.gpu

# (first call, second smaller call): (B, H, N, d, causal)
PAIRS = [
    ((2, 4, 2048, 128, False), (1, 2, 1000, 64, False)),
    ((2, 4, 2048, 128, True), (1, 3, 333, 128, True)),
    ((1, 4, 4096, 256, False), (1, 1, 700, 256, False)),
    ((1, 4, 4096, 256, True), (2, 1, 200, 64, True)),
]
SCHEDS = {False: ("shift", "naive", "descending", "atomic", "partials", "split"),
          True: ("symshift", "descending", "naive", "atomic", "partials", "split")}


def ex_call(qg, kg, vg, og, dog, lseg, causal, sched):
    B, H, N, d = qg.shape
    ws = dash.new_workspace(B, H, N, d, sched)
    out = [torch.empty_like(t) for t in (qg, kg, vg)]
    dash.dash_attn_bwd(qg, kg, vg, og, dog, lseg, *out, causal, sched, workspace=ws)
    assert dash.dash_bwd_check(ws) == dash.DASH_OK
    return out


@pytest.mark.parametrize("pair", PAIRS, ids=[f"N{p[0][2]}d{p[0][3]}-N{p[1][2]}d{p[1][3]}{'c' if p[0][4] else 'f'}"
                                             for p in PAIRS])
def test_noalloc_matches_explicit_workspace(pair):
    status = torch.full((1,), 7, dtype=torch.int32, device="cuda")
    for sched in SCHEDS[pair[0][4]]:
        for (B, H, N, d, causal) in pair:
            if sched in ("partials", "split") and d > 128:
                continue
            print(f"\n[noalloc] B={B} H={H} N={N} d={d} causal={causal} schedule={sched}", flush=True)
            _, _, _, _, (qg, kg, vg, dog) = inputs(B, H, N, d, seed=N + d)
            og, lseg = run_fwd(qg, kg, vg, causal)
            ref = ex_call(qg, kg, vg, og, dog, lseg, causal, sched)
            got = [torch.full_like(t, float("nan")) for t in (qg, kg, vg)]
            status.fill_(7)
            dash.dash_attn_bwd_noalloc(qg, kg, vg, og, dog, lseg, *got, causal, sched, status=status)
            torch.cuda.synchronize()
            assert int(status.item()) == 0
            for name, a, b in zip(("dQ", "dK", "dV"), got, ref):
                if sched == "atomic":
                    assert_close(f"{sched} {name}", a, b.float().cpu().double().numpy())
                else:
                    assert torch.equal(a.view(torch.int16), b.view(torch.int16)), f"{sched} {name} differs"


def test_noalloc_refuses_problems_beyond_its_scratch():
    lib = dash.load()
    p = [ctypes.c_void_p(1 << 20)] * 9
    # B*H*N*d = 2^27 elements: a 512 MiB accumulator, beyond the 256 MiB scratch
    rc = lib.dash_attn_bwd_noalloc(*p, 1, 64, 16384, 128, 0, dash.DASH_SCHED_SHIFT, ctypes.c_float(0.0), None, None)
    assert rc == dash.DASH_ERR_UNSUPPORTED and "scratch" in dash.dash_last_error()
    # the partials variant's T_c accumulator copies count too
    need = dash.dash_bwd_workspace_size(2, 16, 8192, 128, "partials")
    assert need > (256 << 20)
    rc = lib.dash_attn_bwd_noalloc(*p, 2, 16, 8192, 128, 0, dash.DASH_SCHED_PARTIALS, ctypes.c_float(0.0), None, None)
    assert rc == dash.DASH_ERR_UNSUPPORTED
    # the benchmark workload (16384 tokens, 16 heads of 128) fits
    assert dash.dash_bwd_workspace_size(2, 16, 8192, 128, "shift") <= (256 << 20)
