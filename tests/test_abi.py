"""C-ABI checks that need no GPU: the library loads and exports every symbol
the header declares, argument errors are reported before any device work, and
the schedule the kernels follow equals the oracle's independent enumeration
(bit-exact integer tables)."""
import ctypes
import os
import re

import numpy as np
import pytest

from oracle import schedule as osched
from paper_2601_21824_amd import binding as b

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def header_functions():
    text = open(os.path.join(ROOT, "include", "dash.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(dash_[a-z_0-9]+)\s*\(", text)))


def test_library_exports_every_declared_symbol():
    lib = b.load()
    names = header_functions()
    assert set(names) == set(b.EXPORTS)
    for n in names:
        assert hasattr(lib, n), n


def call_bwd(lib, ptr, B=1, H=1, N=128, d=64, causal=0, sched=1):
    p = [ctypes.c_void_p(ptr)] * 9
    return lib.dash_attn_bwd(*p, B, H, N, d, causal, sched)


def test_argument_errors_without_device():
    lib = b.load()
    assert call_bwd(lib, 0) == b.DASH_ERR_INVALID_ARG  # null pointers
    assert call_bwd(lib, 4096, d=96) == b.DASH_ERR_INVALID_ARG
    assert call_bwd(lib, 4096, N=-1) == b.DASH_ERR_INVALID_ARG
    assert call_bwd(lib, 4096, B=1 << 14, H=1 << 6, N=1 << 10) == b.DASH_ERR_INVALID_ARG  # 2^30 rows
    assert call_bwd(lib, 4096, sched=9) == b.DASH_ERR_INVALID_ARG
    assert call_bwd(lib, 4096, sched=b.DASH_SCHED_SYMSHIFT, causal=0) == b.DASH_ERR_UNSUPPORTED
    assert "symmetric shift" in b.dash_last_error()
    # empty problems are successful no-ops, even with null pointers
    assert call_bwd(lib, 0, N=0) == b.DASH_OK
    assert call_bwd(lib, 0, B=0) == b.DASH_OK
    assert lib.dash_attn_fwd(*([ctypes.c_void_p(0)] * 5), 1, 1, 0, 64, 0) == b.DASH_OK
    assert lib.dash_attn_fwd(*([ctypes.c_void_p(0)] * 5), 1, 1, 8, 64, 0) == b.DASH_ERR_INVALID_ARG
    assert b.dash_bwd_workspace_size(1, 1, 100, 96) == 0
    assert b.dash_bwd_workspace_size(1, 1, 100, 64, 9) == 0
    assert b.dash_bwd_workspace_size(2, 16, 8192, 128) >= 2 * 16 * 8192 * 128 * 4
    # the partials comparison variant keeps one accumulator-sized buffer per KV tile
    base = b.dash_bwd_workspace_size(2, 16, 8192, 128, "naive")
    assert b.dash_bwd_workspace_size(2, 16, 8192, 128, "partials") >= base + 63 * 2 * 16 * 8192 * 128 * 4
    assert call_bwd(lib, 4096, d=256, sched=b.DASH_SCHED_PARTIALS) == b.DASH_ERR_UNSUPPORTED
    assert call_bwd(lib, 4096, d=256, sched=b.DASH_SCHED_SPLIT) == b.DASH_ERR_UNSUPPORTED
    assert call_bwd(lib, 4096, sched=8) == b.DASH_ERR_INVALID_ARG
    assert lib.dash_bwd_check(ctypes.c_void_p(0), ctypes.c_void_p(0)) == b.DASH_ERR_INVALID_ARG
    # explicit-workspace form: too small a workspace is an argument error
    opts = b.dash_bwd_options_t(0, 0, None, None, None, None, None)
    p = [ctypes.c_void_p(4096)] * 9
    rc = lib.dash_attn_bwd_ex(*p, 1, 1, 128, 64, 0, 1, ctypes.c_float(0.125), ctypes.c_void_p(4096),
                              16, ctypes.byref(opts), None)
    assert rc == b.DASH_ERR_INVALID_ARG
    # an unknown ticket order is an argument error (checked before any device call)
    opts = b.dash_bwd_options_t(0, 0, None, None, None, None, None, 0, 3)
    rc = lib.dash_attn_bwd_ex(*p, 1, 1, 128, 64, 0, 1, ctypes.c_float(0.125), ctypes.c_void_p(4096),
                              1 << 40, ctypes.byref(opts), None)
    assert rc == b.DASH_ERR_INVALID_ARG and "ticket_order" in b.dash_last_error()
    # ... and so is an unknown placement
    opts = b.dash_bwd_options_t(0, 0, None, None, None, None, None, 0, 0, 3)
    rc = lib.dash_attn_bwd_ex(*p, 1, 1, 128, 64, 0, 1, ctypes.c_float(0.125), ctypes.c_void_p(4096),
                              1 << 40, ctypes.byref(opts), None)
    assert rc == b.DASH_ERR_INVALID_ARG and "placement" in b.dash_last_error()
    assert lib.dash_schedule_table(1, 1, 128, 64, 0, 0, None, None, None, None, None) == b.DASH_ERR_INVALID_ARG
    assert lib.dash_schedule_table(1, 0, 128, 64, 0, b.DASH_PLACEMENT_GLOBAL, None, None, None, None, None) == \
        b.DASH_ERR_INVALID_ARG
    # the MFMA peak measurement checks its arguments before touching the device
    assert lib.dash_mfma_peak(0, None) == b.DASH_ERR_INVALID_ARG
    out = ctypes.c_double(0.0)
    assert lib.dash_mfma_peak(-1, ctypes.byref(out)) == b.DASH_ERR_INVALID_ARG


def test_schedule_resolution():
    assert b.dash_resolve_schedule("auto", 128, False) == b.DASH_SCHED_SHIFT
    assert b.dash_resolve_schedule("auto", 128, True) == b.DASH_SCHED_DESCENDING
    assert b.dash_resolve_schedule("auto", 64, True) == b.DASH_SCHED_DESCENDING
    assert b.dash_resolve_schedule("auto", 256, True) == b.DASH_SCHED_DESCENDING
    assert b.dash_resolve_schedule("auto", 256, False) == b.DASH_SCHED_SHIFT
    assert b.dash_resolve_schedule("shift", 64, True) == b.DASH_SCHED_SYMSHIFT
    assert b.dash_resolve_schedule("naive", 64, True) == b.DASH_SCHED_NAIVE


KINDS = {b.DASH_SCHED_NAIVE: osched.NAIVE, b.DASH_SCHED_DESCENDING: osched.DESCENDING,
         b.DASH_SCHED_SHIFT: osched.SHIFT, b.DASH_SCHED_SYMSHIFT: osched.SYMSHIFT,
         b.DASH_SCHED_ATOMIC: osched.NAIVE, b.DASH_SCHED_PARTIALS: osched.NAIVE,
         b.DASH_SCHED_SPLIT: osched.NAIVE}


@pytest.mark.parametrize("placement", [b.DASH_PLACEMENT_GLOBAL, b.DASH_PLACEMENT_XCD])
@pytest.mark.parametrize("d", [64, 128, 256])
@pytest.mark.parametrize("N", [64, 200, 256, 1000, 1024, 4096, 4224, 8192, 16384, 32768])
@pytest.mark.parametrize("causal", [False, True])
@pytest.mark.parametrize("sched", [0, 1, 2, 3, 4, 6, 7])
@pytest.mark.parametrize("heads", [1, 64])
def test_schedule_table_matches_oracle(heads, sched, causal, N, d, placement):
    if sched == b.DASH_SCHED_SYMSHIFT and not causal:
        pytest.skip("symshift is causal-only")
    if heads > 1 and d != 64:
        pytest.skip("the head count decides the tile size at d = 64 only")
    tab = b.dash_schedule_table(sched, N, d, causal, placement, heads=heads)
    concrete = b.dash_resolve_schedule(sched, d, causal)
    kind = KINDS[concrete]
    t_r, t_c, br, bc, grp = tab["t_r"], tab["t_c"], tab["br"], tab["bc"], tab["group"]
    # tile sizes: KV tiles of 128 rows at d = 128, 64 at d = 256, and at d = 64
    # 256 rows when the call has enough of them (full: 256 over all heads;
    # causal: 512 and N >= 1024), else 128; Q tiles of 64 rows (full) or
    # KV-tile rows (causal); Shift groups of at most 256 chains, 32 when every
    # chain of a head runs on one XCD
    wide = heads * -(-N // 256)
    bc64 = 256 if ((N >= 1024 and wide >= 512) if causal else wide >= 256) else 128
    assert bc == {64: bc64, 128: 128, 256: 64}[d]
    assert br == (bc if causal else 64) and t_r * br == t_c * bc
    most = 32 if placement == b.DASH_PLACEMENT_XCD else 256
    assert grp == (min(t_c, most) if kind == osched.SHIFT else tab["chains"])
    ref = osched.build(kind, t_r, t_c, causal, br, bc, group=grp if kind == osched.SHIFT else None)
    assert tab["chains"] == len(ref.chains)
    for w, ch in enumerate(ref.chains):
        n = tab["chain_len"][w]
        assert n == len(ch)
        got = list(zip(tab["task_kv"][w][:n].tolist(), tab["task_q"][w][:n].tolist()))
        assert got == ch, (w, got, ch)
    want = np.full((t_r, t_c), -1)
    for i, js in ref.order.items():
        for r, j in enumerate(js):
            want[i, j] = r
    np.testing.assert_array_equal(tab["rank"], want)
    if kind in (osched.SHIFT, osched.SYMSHIFT):
        props = osched.check(ref, t_r, t_c, causal, br, bc, group=grp if kind == osched.SHIFT else None)
        assert props["coverage"] and props["conflict_free"] and props["monotone"]


def test_missing_library_raises_instead_of_falling_back():
    """With no built library every entry point raises, and CPU tensors are
    refused rather than computed on: there is no CPU fallback."""
    import subprocess
    import sys
    code = (
        "import sys, torch\n"
        f"sys.path.insert(0, {ROOT!r})\n"
        "from paper_2601_21824_amd import binding as b\n"
        "b.LIB_PATH = '/nonexistent/libdash.so'\n"
        "for call in (b.load, lambda: b.dash_resolve_schedule('auto', 128, False),\n"
        "             lambda: b.dash_bwd_workspace_size(1, 1, 64, 64)):\n"
        "    try:\n"
        "        call()\n"
        "        sys.exit(1)\n"
        "    except b.DashError as e:\n"
        "        assert 'is not built' in str(e), e\n"
        "q = torch.zeros(1, 1, 64, 64, dtype=torch.bfloat16)\n"
        "try:\n"
        "    b.attn_bwd(q, q, q, q, q, torch.zeros(1, 1, 64), False, 'shift')\n"
        "    sys.exit(1)\n"
        "except b.DashError as e:\n"
        "    assert 'device tensors' in str(e), e\n"
        "print('ok')\n")
    r = subprocess.run([sys.executable, "-c", code], capture_output=True, text=True, timeout=300)
    assert r.returncode == 0 and "ok" in r.stdout, r.stdout + r.stderr


@pytest.mark.parametrize("N,d", [(8000, 128), (8192, 128), (1000, 64), (32704, 256), (32768, 256), (333, 256)])
@pytest.mark.parametrize("sized_for", ["shift", "auto", "naive", "descending", "atomic", "split"])
def test_workspace_size_serves_every_schedule_and_mask(N, d, sized_for):
    """A workspace of dash_bwd_workspace_size(..., s) bytes passes the size
    check of dash_attn_bwd_ex for every schedule but PARTIALS under both masks
    -- including causal SHIFT, which runs as Symmetric Shift with T_c padded to
    even (odd T_c at N = 8000, d = 128 and N = 32704, d = 256).  The call is
    stopped right after the size check by an invalid option, so no device is
    touched; one byte less is reported as a workspace error."""
    lib = b.load()
    B, H = 2, 3
    ws = b.dash_bwd_workspace_size(B, H, N, d, sized_for)
    assert ws > 0
    p = [ctypes.c_void_p(1 << 20)] * 9
    bad_opts = b.dash_bwd_options_t(-1)  # spin_limit < 0: checked right after the workspace
    for causal in (0, 1):
        for sched in ("atomic", "naive", "descending", "shift", "symshift", "auto", "split"):
            if sched == "symshift" and not causal:
                continue
            if sched == "split" and d > 128:
                continue
            args = (*p, B, H, N, d, causal, b.SCHEDULES[sched], ctypes.c_float(0.125), ctypes.c_void_p(1 << 20))
            rc = lib.dash_attn_bwd_ex(*args, ws, ctypes.byref(bad_opts), None)
            assert rc == b.DASH_ERR_INVALID_ARG and "spin_limit" in b.dash_last_error(), (sched, causal)
            need = b.dash_bwd_workspace_size(B, H, N, d, sched)
            rc = lib.dash_attn_bwd_ex(*args[:-1], ctypes.c_void_p(1 << 20), need - 1, ctypes.byref(bad_opts), None)
            assert rc == b.DASH_ERR_INVALID_ARG and "workspace" in b.dash_last_error(), (sched, causal)
