"""bench.py's host-side contract, without a GPU: the multi-GPU refusal, the
committed counter summaries matching the kernel sources they describe, and
every profile summary's command running committed files only."""

import glob
import os
import re
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)


def test_more_than_one_gpu_is_refused_with_a_message():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode != 0
    assert "one GPU only" in r.stdout


def test_committed_counter_summaries_match_the_kernel_sources():
    import bench
    found = glob.glob(os.path.join(ROOT, "profiles", "*_pmc.md"))
    assert found
    for path in found:
        kernel = os.path.basename(path).split("_", 1)[0]
        text = open(path).read()
        sha = re.search(r"source_sha:\s*(\w+)", text)
        assert sha, path
        assert sha.group(1) == bench.kernel_source_sha(kernel), \
            f"{os.path.basename(path)} was taken on other {kernel} sources: retake it"
        workload = os.path.basename(path)[len(kernel) + 1:-len("_pmc.md")]
        assert bench.committed_traffic(workload, kernel) is not None, path


def test_profile_summaries_name_commands_that_run_committed_files():
    """Every summary under profiles/ gives the rocprofv3 command it came
    from, and that command runs bench.py from the repository with a workload
    bench.py defines (nothing outside the committed tree)."""
    import bench  # noqa: F401  (the workloads bench.py can run)
    from synth import WORKLOADS
    found = sorted(glob.glob(os.path.join(ROOT, "profiles", "*.md")))
    assert found
    for path in found:
        cmds = re.findall(r"^rocprofv3 .*$", open(path).read(), re.M)
        assert cmds, f"{os.path.basename(path)}: no command"
        for cmd in cmds:
            prog = cmd.split(" -- ", 1)[1].split()
            assert prog[:2] == ["python3", "$REPO/bench.py"], f"{os.path.basename(path)}: {cmd}"
            wl = prog[prog.index("--workload") + 1]
            assert wl in WORKLOADS, f"{os.path.basename(path)}: unknown workload {wl}"
            assert "_work" not in cmd, f"{os.path.basename(path)}: {cmd}"
