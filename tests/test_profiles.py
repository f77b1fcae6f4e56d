"""The committed rocprofv3 summaries: every command runs committed files only
(the program after `--` is bench.py or a file in the repository; outputs go
under gpurun_out/), and each names the kernel source it measured with a
sha256 prefix of a file that exists."""
import glob
import os
import re

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
PROFILES = sorted(glob.glob(os.path.join(ROOT, "profiles", "*.md")))


def test_profiles_exist():
    assert len(PROFILES) >= 4


def test_commands_run_committed_files_only():
    for path in PROFILES:
        text = open(path).read()
        cmds = [l.strip() for l in text.splitlines() if l.strip().startswith(("rocprofv3", "timeout", "hipcc"))]
        assert cmds, path
        for c in cmds:
            if " -- " in c:
                prog = c.split(" -- ", 1)[1].split()
                assert prog[0] == "python3", (path, c)
                target = prog[1].replace("REPO/", "")
                assert os.path.isfile(os.path.join(ROOT, target)), (path, c)
            for ref in re.findall(r"REPO/([\w./-]+)", c):
                assert ref.startswith("gpurun_out/") or os.path.exists(os.path.join(ROOT, ref)), (path, ref)
            assert "_work" not in c, (path, c)


def test_sources_named_exist():
    for path in PROFILES:
        text = open(path).read()
        srcs = re.findall(r"Source of the kernel at measurement time: (\S+) sha256 prefix ([0-9a-f]{16})", text)
        assert srcs, path
        for src, _ in srcs:
            assert os.path.isfile(os.path.join(ROOT, src)), (path, src)
