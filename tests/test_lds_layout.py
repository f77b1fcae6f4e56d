"""Host check of the backward kernels' LDS layouts: every access pattern of
the d = 64 / 128 / 256 kernels is bank-conflict free under gfx950's measured
bank model (64 banks of 4 bytes; 16-byte accesses served 16 lanes at a time,
8-byte accesses 32 at a time).  The model itself is pinned by the conflict
counts a one-wave hardware probe measured for fixed address patterns."""
import os
import subprocess

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_lds_layouts_are_bank_conflict_free(tmp_path):
    exe = tmp_path / "lds_layout_check"
    subprocess.run(["g++", "-std=c++17", "-O1", "-I", os.path.join(ROOT, "paper_2601_21824_amd", "csrc"),
                    os.path.join(ROOT, "tests", "lds_layout_check.cpp"), "-o", str(exe)], check=True)
    res = subprocess.run([str(exe)], capture_output=True, text=True)
    print(res.stdout)
    assert res.returncode == 0, res.stdout
