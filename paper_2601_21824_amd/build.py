"""Build libdash.so (the HIP kernels + C ABI) in-tree for gfx950 with hipcc."""
from __future__ import annotations

import os
import subprocess
import sys
import tempfile
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(HERE, "libdash.so")
SOURCES = ["attn_fwd.hip", "attn_bwd.hip", "attn_bwd_d64.hip", "attn_bwd64w.hip", "attn_bwd256.hip", "attn_dq.hip", "mfma_peak.hip",
           "dash_api.hip"]
HEADERS = ["common.h", "kernels.h", "schedule.h", "bwd_common.h", "bwd_main.h", "lds_layout.h", "dag_model.h", "model_calibration.h"]

HIPCC_FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC",
    # no packed-fp32 (v_pk_*_f32) instructions: some of their forms have given
    # silently wrong results on this hardware
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wno-unused-command-line-argument",
]
# per-source flags: the d = 64 kernels (128- and 256-row tiles) run faster
# with their MFMA results in VGPRs (S and dP feed the softmax without AGPR
# reads), and the d = 256 kernel compiles that way without the VGPR spills
# (and scratch) it has otherwise; the d = 128 kernel, with less room in its
# VGPRs, runs slower that way
_VGPR_MFMA = ["-mllvm", "-amdgpu-mfma-vgpr-form"]
SOURCE_FLAGS = {"attn_bwd_d64.hip": _VGPR_MFMA, "attn_bwd64w.hip": _VGPR_MFMA, "attn_bwd256.hip": _VGPR_MFMA}


def hipcc() -> str:
    for cand in ("/opt/rocm/bin/hipcc", "hipcc"):
        if os.path.sep not in cand or os.path.exists(cand):
            return cand
    return "hipcc"


def _run(cmd, verbose):
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        sys.stderr.write(res.stdout + res.stderr)
        raise RuntimeError("hipcc failed building libdash.so")


def build(verbose: bool = False, extra=()) -> str:
    """Compile every source and link libdash.so (always recompiles)."""
    with tempfile.TemporaryDirectory(prefix="libdash") as tmpdir:
        objs = [os.path.join(tmpdir, s + ".o") for s in SOURCES]
        cmds = [[hipcc(), *HIPCC_FLAGS, *SOURCE_FLAGS.get(s, []), *extra, "-I", INCLUDE, "-I", CSRC, "-c",
                 os.path.join(CSRC, s), "-o", o] for s, o in zip(SOURCES, objs)]
        with ThreadPoolExecutor(max_workers=min(len(cmds), os.cpu_count() or 1)) as pool:
            for f in [pool.submit(_run, c, verbose) for c in cmds]:
                f.result()
        tmp = LIB + ".tmp%d" % os.getpid()
        _run([hipcc(), "--offload-arch=gfx950", "-shared", "-fPIC", *objs, "-o", tmp], verbose)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
