"""bench.py's host-side contract, without a GPU: the multi-GPU refusal and
the committed counter summaries matching the kernel sources they describe."""

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
