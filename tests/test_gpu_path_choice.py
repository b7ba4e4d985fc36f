"""The automatic choice between the resolve paths (bkmoo_resolve_path) on
MI355X shapes: the hybrid path needs at least 8 buckets of at least 48 MiB
(all K rows), at least 10% of each kept on chip, and a solve short enough
to hide behind the next bucket's Gram read; the resident path needs at
least 32 buckets and a short solve; everything else runs the two passes.
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


# (buckets, method, iterations, expected path name)
CASES_4x2G = [
    (8, "mgda", 20, "hybrid"),      # 64 MiB per row: the solve hides (5.6 us vs 57 us)
    (8, "mgda", 100, "hybrid"),     # 28 us
    (8, "cagrad", 20, "hybrid"),    # 17.6 us
    (8, "cagrad", 100, "two-pass"),  # 88 us: exposed
    (8, "pcgrad", 0, "hybrid"),
    (8, "mean", 0, "hybrid"),
    (32, "mgda", 20, "hybrid"),     # 16 MiB per row: 5.6 us vs 14.4 us
    (32, "mgda", 100, "two-pass"),  # 28 us
    (32, "cagrad", 20, "two-pass"),  # 17.6 us
    (48, "mgda", 20, "two-pass"),   # 10.7 MiB per row: below 48 MiB all rows
    (48, "mean", 0, "resident"),    # short solve, 48 buckets of 42.7 MiB
    (4, "mean", 0, "two-pass"),     # fewer than 8 buckets
    (8, "mgda-exact", 0, "two-pass"),
]


@pytest.mark.parametrize("B,method,iters,want", CASES_4x2G)
def test_automatic_path(gpu_lib, rows_4x2g, B, method, iters, want):
    names = {gpu_lib.PATH_TWO_PASS: "two-pass", gpu_lib.PATH_RESIDENT: "resident",
             gpu_lib.PATH_HYBRID: "hybrid"}
    gpu_lib.set_resolve_path(0)
    got = names[gpu_lib.resolve_path(rows_4x2g, B + 1, method, iters)]
    assert got == want, f"B={B} {method}-{iters}: {got}"


def test_hybrid_needs_a_tenth_on_chip(gpu_lib):
    """K=4 bf16, 2^30 elements in 8 buckets of 256 MiB per row: about 5% of
    each bucket fits on chip, so the two passes run."""
    g = torch.empty((4, 1 << 30), dtype=torch.bfloat16, device="cuda")
    gpu_lib.set_resolve_path(0)
    assert gpu_lib.resolve_path(g, 9, "mean", 0) == gpu_lib.PATH_TWO_PASS
    assert gpu_lib.resolve_path(g, 33, "mean", 0) == gpu_lib.PATH_HYBRID  # 64 MiB per row: ~19%


def test_misaligned_rows_take_the_two_passes(gpu_lib):
    base = torch.empty((4 * (1 << 26) + 8,), dtype=torch.bfloat16, device="cuda")
    rows = [base[1 + i * (1 << 26): 1 + (i + 1) * (1 << 26)] for i in range(4)]
    rows[1] = base[2 + (1 << 26): 2 + 2 * (1 << 26)]
    gpu_lib.set_resolve_path(0)
    assert gpu_lib.resolve_path(rows, 9, "mean", 0) == gpu_lib.PATH_TWO_PASS
