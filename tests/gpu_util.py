"""Helpers shared by the GPU tests: run the HIP path, compare with the oracle."""
import numpy as np
import torch

import oracle
from paper_2601_21824_amd import binding as dash
from paper_2601_21824_amd.synth import make_inputs

# tolerance of the deterministic-backward target: relative Frobenius error and
# per-element error relative to the largest reference magnitude
REL_FROB = 5e-3
REL_MAX = 2e-2

FULL_SCHEDULES = ("atomic", "naive", "descending", "shift", "partials", "split")
CAUSAL_SCHEDULES = ("atomic", "naive", "descending", "symshift", "partials", "split")


def schedules(causal, d=128):
    s = CAUSAL_SCHEDULES if causal else FULL_SCHEDULES
    return tuple(x for x in s if x not in ("partials", "split") or d <= 128)


def errors(got, ref):
    g = got.detach().float().cpu().double().numpy() if hasattr(got, "detach") else np.asarray(got, np.float64)
    r = np.asarray(ref, np.float64)
    assert np.all(np.isfinite(g)), "non-finite values"
    nr = np.linalg.norm(r)
    rel_f = np.linalg.norm(g - r) / nr if nr > 0 else np.linalg.norm(g - r)
    mr = np.max(np.abs(r)) if r.size else 0.0
    rel_m = np.max(np.abs(g - r)) / mr if mr > 0 else (np.max(np.abs(g - r)) if r.size else 0.0)
    return float(rel_f), float(rel_m)


def assert_close(name, got, ref, rel_frob=REL_FROB, rel_max=REL_MAX):
    rf, rm = errors(got, ref)
    assert rf <= rel_frob and rm <= rel_max, f"{name}: rel_frob={rf:.3e} rel_max={rm:.3e}"
    return rf, rm


def inputs(B, H, N, d, seed, sigma=1.0):
    q, k, v, do = make_inputs(B, H, N, d, seed, sigma)
    return q, k, v, do, [t.cuda() for t in (q, k, v, do)]


def run_fwd(qg, kg, vg, causal):
    o, lse = dash.attn_fwd(qg, kg, vg, causal)
    torch.cuda.synchronize()
    return o, lse


def run_bwd(qg, kg, vg, og, dog, lseg, causal, schedule, options=None, workspace=None):
    B, H, N, d = qg.shape
    if options is not None and workspace is None:
        workspace = dash.new_workspace(B, H, N, d, schedule)
    dq, dk, dv = dash.attn_bwd(qg, kg, vg, og, dog, lseg, causal, schedule, workspace=workspace,
                               options=options)
    torch.cuda.synchronize()
    return dq, dk, dv
