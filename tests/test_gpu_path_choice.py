"""The automatic choice between the resolve paths (bkmoo_resolve_path) on
MI355X shapes.  The hybrid path (K <= 8) needs at least 8 buckets, at least
10% of a bucket kept on chip, and buckets (all K rows) of at least
max(24, 6 K) MiB plus 4 MiB per microsecond of estimated solve latency L
(0.07 K us per MGDA and 0.22 K us per CAGrad iteration, 0.1 K^2 us for
PCGrad).  The refill path (K <= 10) needs at least 8 buckets and a round of
its G = clamp(round(180 MiB / bucket), 1, 32) groups' buckets of at least
64 + 2 L MiB and, with more than one group, at most 300 MiB; it runs where
the hybrid path does not, and instead
of it for K = 3 and for K <= 4 with L >= 4 us.  Everything else runs the
two passes.
Only shapes are used (no resolve runs); the cases sit away from the
thresholds."""

import pytest
import torch

pytestmark = pytest.mark.gpu

MIB = 1 << 20


@pytest.fixture(scope="module")
def rows_4x2g():
    """K=4 bf16 rows of 2^28 elements (512 MiB each)."""
    return torch.empty((4, 1 << 28), dtype=torch.bfloat16, device="cuda")


# (buckets, method, iterations, expected path name); rows of 512 MiB
CASES_4x2G = [
    (8, "mgda", 20, "refill"),       # both run (256 MiB buckets (all rows) >= 24 + 4 * 5.6, G = 1); L >= 4
    (8, "mgda", 5, "hybrid"),        # both run; L = 1.4 < 4
    (8, "mgda", 100, "refill"),      # both run (256 >= 24 + 4 * 28); L = 28
    (8, "cagrad", 20, "refill"),     # both run; L = 17.6
    (8, "cagrad", 100, "refill"),    # hybrid: 256 < 24 + 4 * 88; refill: 256 >= 64 + 2 * 88
    (8, "pcgrad", 0, "hybrid"),
    (8, "mean", 0, "hybrid"),
    (32, "mgda", 20, "refill"),      # 64 MiB: both run (G = 3, round 192); L = 5.6 >= 4
    (32, "mgda", 10, "hybrid"),      # both run; L = 2.8 < 4
    (32, "mgda", 100, "refill"),     # hybrid 64 < 136; G = 3, round 192 >= 120
    (32, "cagrad", 20, "refill"),    # hybrid 64 < 94.4; round 192 >= 99.2
    (48, "mgda", 20, "refill"),      # hybrid 42.7 MiB < 46.4; G = 4, round 171
    (48, "mean", 0, "hybrid"),
    (64, "mean", 0, "hybrid"),       # 32 MiB
    (64, "mgda", 20, "refill"),      # hybrid 32 < 46.4; G = 6, round 192
    (96, "mean", 0, "refill"),       # hybrid 21.3 MiB < 24; G = 8, round 171
    (4, "mean", 0, "two-pass"),      # fewer than 8 buckets
    (8, "mgda-exact", 0, "two-pass"),
]


@pytest.mark.parametrize("B,method,iters,want", CASES_4x2G)
def test_automatic_path(gpu_lib, rows_4x2g, B, method, iters, want):
    names = {gpu_lib.PATH_TWO_PASS: "two-pass", gpu_lib.PATH_HYBRID: "hybrid", gpu_lib.PATH_REFILL: "refill"}
    gpu_lib.set_resolve_path(0)
    got = names[gpu_lib.resolve_path(rows_4x2g, B + 1, method, iters)]
    assert got == want, f"B={B} {method}-{iters}: {got}"


# (K, buckets, method, iterations, expected path name); rows of 2^28 bf16
# elements (512 MiB).  Each case's side was measured on MI355X: at K = 8
# the two-buffer kernel loses at 4 MiB per row, wins at 8-25 MiB when the
# solve is short enough, and keeps too little on chip at 50 MiB; grouped
# buckets on the refill kernel take the smaller buckets.
CASES_MORE_TASKS = [
    (8, 128, "mean", 0, "refill"),     # hybrid: 32 MiB < 48 (6 MiB per row); G = 6, round 192
    (8, 64, "mean", 0, "hybrid"),      # 64 MiB >= 48
    (8, 64, "mgda", 20, "refill"),     # hybrid 64 < 48 + 4 * 11.2; G = 3, round 192 >= 86.4
    (8, 32, "mgda", 20, "hybrid"),     # 128 >= 92.8
    (8, 32, "pcgrad", 0, "hybrid"),    # 128 >= 48 + 4 * 6.4
    (8, 32, "cagrad", 20, "two-pass"), # hybrid 128 < 48 + 4 * 35.2; G = 1, round 128 < 64 + 2 * 35.2
    (8, 20, "cagrad", 20, "hybrid"),   # 204.8 >= 188.8
    (8, 10, "mean", 0, "refill"),      # 51 MiB per row: hybrid keeps < 10%; G = 1, round 410 (no cap)
    (6, 64, "mean", 0, "hybrid"),      # 48 MiB >= 36
    (6, 128, "mean", 0, "refill"),     # hybrid 24 MiB < 36; G = 8, round 192
    (5, 32, "mgda", 20, "hybrid"),     # 80 MiB >= 30 + 4 * 7
]


@pytest.mark.parametrize("K,B,method,iters,want", CASES_MORE_TASKS)
def test_automatic_path_more_tasks(gpu_lib, K, B, method, iters, want):
    names = {gpu_lib.PATH_TWO_PASS: "two-pass", gpu_lib.PATH_HYBRID: "hybrid", gpu_lib.PATH_REFILL: "refill"}
    g = torch.empty((K, 1 << 28), dtype=torch.bfloat16, device="cuda")
    gpu_lib.set_resolve_path(0)
    got = names[gpu_lib.resolve_path(g, B + 1, method, iters)]
    assert got == want, f"K={K} B={B} {method}-{iters}: {got}"


def test_more_than_eight_tasks(gpu_lib):
    """Nine tasks in 8 buckets of 16 MiB per row: beyond the two-buffer
    kernel, so the single-buffer one takes them (forcing the two-buffer one
    falls back to the two passes); eleven tasks only run the two passes,
    whatever is forced."""
    g = torch.empty((9, 1 << 26), dtype=torch.bfloat16, device="cuda")
    g11 = torch.empty((11, 1 << 24), dtype=torch.bfloat16, device="cuda")
    gpu_lib.set_resolve_path(0)
    assert gpu_lib.resolve_path(g, 9, "mean", 0) == gpu_lib.PATH_REFILL
    assert gpu_lib.resolve_path(g11, 9, "mean", 0) == gpu_lib.PATH_TWO_PASS
    try:
        gpu_lib.set_resolve_path(gpu_lib.PATH_HYBRID)
        assert gpu_lib.resolve_path(g, 9, "mean", 0) == gpu_lib.PATH_TWO_PASS
        gpu_lib.set_resolve_path(gpu_lib.PATH_REFILL)
        assert gpu_lib.resolve_path(g11, 9, "mean", 0) == gpu_lib.PATH_TWO_PASS
    finally:
        gpu_lib.set_resolve_path(0)


def test_hybrid_needs_a_tenth_on_chip(gpu_lib):
    """K=4 bf16, 2^30 elements in 8 buckets of 256 MiB per row: about 5% of
    each bucket fits in the two-buffer kernel, so the single-buffer one takes
    the buckets one at a time (a 1 GiB round, beyond the cache, is allowed
    with one group); with 32 buckets (64 MiB per row, ~19% kept) the
    two-buffer kernel runs."""
    g = torch.empty((4, 1 << 30), dtype=torch.bfloat16, device="cuda")
    gpu_lib.set_resolve_path(0)
    assert gpu_lib.resolve_path(g, 9, "mean", 0) == gpu_lib.PATH_REFILL
    assert gpu_lib.resolve_path(g, 33, "mean", 0) == gpu_lib.PATH_HYBRID


def test_three_tasks_take_the_refill_kernel(gpu_lib):
    """K=3 bf16 rows of 2^28 elements in 8 buckets (192 MiB each, one
    group) and 32 (48 MiB, four groups): the single-buffer kernel for every
    method, also where the two-buffer kernel could run."""
    g = torch.empty((3, 1 << 28), dtype=torch.bfloat16, device="cuda")
    gpu_lib.set_resolve_path(0)
    for B in (8, 32):
        for method, iters in (("mean", 0), ("pcgrad", 0), ("mgda", 20), ("cagrad", 20)):
            assert gpu_lib.resolve_path(g, B + 1, method, iters) == gpu_lib.PATH_REFILL, (B, method)


def test_misaligned_rows_take_the_two_passes(gpu_lib):
    base = torch.empty((4 * (1 << 26) + 8,), dtype=torch.bfloat16, device="cuda")
    rows = [base[1 + i * (1 << 26): 1 + (i + 1) * (1 << 26)] for i in range(4)]
    rows[1] = base[2 + (1 << 26): 2 + 2 * (1 << 26)]
    gpu_lib.set_resolve_path(0)
    assert gpu_lib.resolve_path(rows, 9, "mean", 0) == gpu_lib.PATH_TWO_PASS


def test_forced_hybrid_and_unknown_paths(gpu_lib, rows_4x2g):
    """Forced, the hybrid path runs wherever it can (aligned rows, K <= 8,
    iterative or not, any bucket count), and so does the refill path (K <= 10);
    a path value other than 0, 1, 3 and 4 is rejected."""
    gpu_lib.set_resolve_path(gpu_lib.PATH_HYBRID)
    try:
        for B in (4, 48, 613):
            assert gpu_lib.resolve_path(rows_4x2g, B + 1, "mgda", 20) == gpu_lib.PATH_HYBRID
        gpu_lib.set_resolve_path(gpu_lib.PATH_REFILL)
        for B in (4, 48, 613):
            assert gpu_lib.resolve_path(rows_4x2g, B + 1, "mgda", 20) == gpu_lib.PATH_REFILL
    finally:
        gpu_lib.set_resolve_path(0)
    for bad in (-1, 2, 5):
        with pytest.raises(gpu_lib.BkmooError):
            gpu_lib.set_resolve_path(bad)
