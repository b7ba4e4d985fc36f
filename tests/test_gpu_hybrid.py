"""The pipelined, partly resident resolve kernels (two-buffer and
single-buffer) against the oracle.  Every method and input type for K =
2..10, ragged and unaligned buckets, 1 to 41 buckets (the two-buffer kernel
alternates two buffers), full 25 MiB buckets and buckets long enough that
every kept vector holds data (their segments stream the rest), a bucket
larger than the chip holds, determinism, agreement with the two-pass path,
and the bounded waits' timeout forced from the host."""

import numpy as np
import pytest
import torch

from synth import WORKLOADS, fill_grads, small_workload
from tests.parity import full_parity, run_resolve, to_device_inputs

pytestmark = pytest.mark.gpu

BASE = WORKLOADS["llama3-8b-k4-mgda-bf16"]
# ragged, unaligned bucket starts, a 1-element and an empty bucket; the total
# keeps every row of a [K, N] tensor at the same 16-byte phase
LENS = [70_001, 1, 0, 33_333, 131_072, 7, 65_539, 40_047]


@pytest.fixture(params=["PATH_HYBRID", "PATH_REFILL"])
def coop(gpu_lib, request):
    """The library with a cooperative path forced (the two-buffer hybrid or
    the single-buffer refill kernel), and that path."""
    path = getattr(gpu_lib, request.param)
    gpu_lib.set_resolve_path(path)
    yield gpu_lib, path
    gpu_lib.set_resolve_path(0)


@pytest.fixture
def two_pass(gpu_lib):
    gpu_lib.set_resolve_path(gpu_lib.PATH_TWO_PASS)
    yield gpu_lib
    gpu_lib.set_resolve_path(0)


@pytest.mark.parametrize("method", ["mgda", "pcgrad", "cagrad", "mean"])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("K", [2, 3, 4])
def test_coop_parity(coop, method, dtype, K):
    lib, path = coop
    wl = small_workload(BASE, sum(LENS), bucket_lens=LENS, K=K, dtype=dtype, method=method,
                        seed=9000 + 10 * K + (dtype == "bf16"))
    grads, _, _ = to_device_inputs(wl)
    assert lib.resolve_path(grads, wl.B + 1, method) == path
    print(f"case path {path} {wl.name} K={K} {dtype} {method}", full_parity(lib, wl, grads=grads), flush=True)


@pytest.mark.parametrize("method", ["mgda", "pcgrad", "cagrad", "mean"])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("K,path_name", [(K, p) for K in (5, 6, 7, 8) for p in ("PATH_HYBRID", "PATH_REFILL")]
                         + [(K, "PATH_REFILL") for K in (9, 10)])
def test_coop_parity_more_tasks(gpu_lib, method, dtype, K, path_name):
    """The cooperative kernels for K = 5..10 (the two-buffer kernel up to
    K = 8: one or two kept register vectors, one LDS vector, one or two
    streamed per step; the single-buffer kernel up to K = 10)."""
    path = getattr(gpu_lib, path_name)
    gpu_lib.set_resolve_path(path)
    try:
        wl = small_workload(BASE, sum(LENS), bucket_lens=LENS, K=K, dtype=dtype, method=method,
                            seed=9100 + 10 * K + (dtype == "bf16"))
        grads, _, _ = to_device_inputs(wl)
        assert gpu_lib.resolve_path(grads, wl.B + 1, method) == path
        print(f"case {path_name} {wl.name} K={K} {dtype} {method}", full_parity(gpu_lib, wl, grads=grads),
              flush=True)
    finally:
        gpu_lib.set_resolve_path(0)


@pytest.mark.parametrize("out_dtype", [torch.float32, torch.bfloat16])
def test_coop_output_types(coop, out_dtype):
    lib, path = coop
    wl = small_workload(BASE, 200_000, bucket_lens=[99_999, 100_001], K=3, dtype="bf16", seed=77)
    grads, _, _ = to_device_inputs(wl)
    assert lib.resolve_path(grads, wl.B + 1, wl.method, wl.max_iter, out_dtype=out_dtype) == path
    print(full_parity(lib, wl, grads=grads, out_dtype=out_dtype), flush=True)


@pytest.mark.parametrize("nb", [1, 2, 3, 41])
def test_coop_bucket_counts(coop, nb):
    """Odd and even bucket counts through the two-buffer pipeline."""
    lib, path = coop
    rng = np.random.default_rng(nb)
    lens = [int(x) for x in rng.integers(1, 90_000, size=nb)]
    lens[-1] += -sum(lens) % 8  # rows of the [K, N] tensor at one 16-byte phase
    wl = small_workload(BASE, sum(lens), bucket_lens=lens, K=4, dtype="bf16", method="mgda", seed=600 + nb)
    grads, _, _ = to_device_inputs(wl)
    assert lib.resolve_path(grads, wl.B + 1, "mgda") == path
    print(f"case path {path} B={nb}", full_parity(lib, wl, grads=grads), flush=True)


def test_coop_many_small_buckets(coop):
    """1,500 ragged buckets of 1..2,000 elements (per-bucket counters and
    flags for every bucket, most segments empty)."""
    lib, path = coop
    rng = np.random.default_rng(1500)
    lens = [int(x) for x in rng.integers(1, 2_000, size=1500)]
    lens[-1] += -sum(lens) % 8
    wl = small_workload(BASE, sum(lens), bucket_lens=lens, K=4, dtype="bf16", method="cagrad", seed=1501)
    grads, _, _ = to_device_inputs(wl)
    assert lib.resolve_path(grads, wl.B + 1, "cagrad") == path
    print(f"case path {path} B=1500", full_parity(lib, wl, grads=grads), flush=True)


def test_coop_full_size_buckets(coop):
    """Three 25 MiB-per-task K=4 bf16 buckets: the hybrid kernel keeps part
    of each segment and streams the rest twice."""
    lib, path = coop
    wl = small_workload(BASE, 3 * 13_107_200, bucket_elems=13_107_200, K=4, dtype="bf16", method="mgda",
                        seed=620)
    grads, _, _ = to_device_inputs(wl)
    assert lib.resolve_path(grads, wl.B + 1, "mgda") == path
    print(f"case path {path} 3 x 25 MiB", full_parity(lib, wl, grads=grads), flush=True)


def _layout_case(gpu_lib, method, dtype, seed):
    """K=4 buckets of 19-25 MiB per row, ragged, sized so that 504 and 508
    segment slots give different segment lengths; results match the oracle
    and repeat bitwise on the forced hybrid path."""
    unit = 256 * (8 if dtype == "bf16" else 4)  # one 16-byte vector per thread
    lens = [5050 * unit + 3, 6060 * unit, 6200 * unit + 1001, 5000 * unit]
    lens[-1] += -sum(lens) % (8 if dtype == "bf16" else 4)  # rows at one 16-byte phase
    wl = small_workload(BASE, sum(lens), bucket_lens=lens, K=4, dtype=dtype, method=method, seed=seed)
    grads, offs, order = to_device_inputs(wl)
    gpu_lib.set_resolve_path(gpu_lib.PATH_HYBRID)
    try:
        assert gpu_lib.resolve_path(grads, wl.B + 1, method, 20) == gpu_lib.PATH_HYBRID
        print(f"case layout {method} {dtype}", full_parity(gpu_lib, wl, grads=grads), flush=True)
        r1 = run_resolve(gpu_lib, wl, grads, offs, order)
        r2 = run_resolve(gpu_lib, wl, grads, offs, order)
    finally:
        gpu_lib.set_resolve_path(0)
    assert np.array_equal(r1["gram"], r2["gram"]) and np.array_equal(r1["weights"], r2["weights"])
    assert torch.equal(r1["out"].view(torch.int32 if dtype == "f32" else torch.int16),
                       r2["out"].view(torch.int32 if dtype == "f32" else torch.int16))
    return wl


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_hybrid_skewed_segments(gpu_lib, dtype):
    """MGDA FW-20 at K=4 (a solve of a few microseconds): the first
    workgroup of each CU gets a longer segment, so the bytes requested
    differ from the even layout's (the mean method's) and from the layout
    that leaves the solvers' CU mates empty (MGDA FW-100)."""
    wl = _layout_case(gpu_lib, "mgda", dtype, 630 + (dtype == "f32"))
    traffic = lambda m, it: gpu_lib.resolve_traffic(4, wl.offsets(), dtype, gpu_lib.PATH_HYBRID, method=m,
                                                    max_iter=it)
    skewed, even, mates = traffic("mgda", 20), traffic("mean", 0), traffic("mgda", 100)
    assert skewed != even and skewed != mates


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_hybrid_solver_mates_hold_no_segment(gpu_lib, dtype):
    """CAGrad FW-20 at K=4 (a solve of ~18 us): the four data workgroups on
    the solvers' CUs hold no segment, the others share each bucket (504
    slots instead of 508: other segment lengths, other bytes requested than
    the even layout's); a short MGDA solve (FW-5) keeps the even layout."""
    wl = _layout_case(gpu_lib, "cagrad", dtype, 640 + (dtype == "f32"))
    traffic = lambda m, it: gpu_lib.resolve_traffic(4, wl.offsets(), dtype, gpu_lib.PATH_HYBRID, method=m,
                                                    max_iter=it)
    mates, even = traffic("cagrad", 20), traffic("mean", 0)
    assert mates != even
    assert traffic("mgda", 5) == even and traffic("pcgrad", 0) == even


# Vectors per task row and thread a segment needs so that every kept
# register and LDS vector of either kernel holds data and the rest streams
# (the single-buffer kernel always streams four; its largest kept counts
# are 24 at K = 2, 14 at K = 3, 13 at K = 4, 8 at K = 5, fewer above).
_SLOTS = {2: 30, 3: 19, 4: 18, 5: 13, 6: 11, 7: 10, 8: 9, 9: 8, 10: 8}


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("K,path_name", [(K, "PATH_HYBRID") for K in range(2, 9)]
                         + [(K, "PATH_REFILL") for K in range(2, 11)])
def test_coop_every_kept_slot(gpu_lib, K, path_name, dtype):
    """Two ragged buckets of _SLOTS[K] vectors per row, thread and data
    workgroup: every kept register and LDS vector holds data and part of
    each segment streams (the bytes requested exceed the one-read floor),
    for K = 2..10, both input types and one method per K, against the
    oracle."""
    path = getattr(gpu_lib, path_name)
    V = 8 if dtype == "bf16" else 4
    n = 508 * 256 * V * _SLOTS[K]
    method = ("mgda", "cagrad", "pcgrad", "mean")[K % 4]
    wl = small_workload(BASE, 2 * n + 8, bucket_lens=[n + 3, n + 5], K=K, dtype=dtype, method=method,
                        seed=9300 + 10 * K + (dtype == "bf16"))
    s = 2 if dtype == "bf16" else 4
    gpu_lib.set_resolve_path(path)
    try:
        grads, _, _ = to_device_inputs(wl)
        assert gpu_lib.resolve_path(grads, wl.B + 1, method, wl.max_iter) == path
        floor = (K + 1) * s * wl.N
        assert gpu_lib.resolve_traffic(K, wl.offsets(), dtype, path, method=method, max_iter=wl.max_iter) > floor
        print(f"case {path_name} K={K} {dtype} {method} N={wl.N}", full_parity(gpu_lib, wl, grads=grads),
              flush=True)
    finally:
        gpu_lib.set_resolve_path(0)


def test_coop_bucket_larger_than_chip(coop):
    """One K=2 fp32 bucket of 14.5M elements: the segments stream most of
    their data."""
    lib, path = coop
    wl = small_workload(WORKLOADS["k2-mgda-1m-f32"], 14_500_000, bucket_lens=[14_500_000], seed=5)
    grads, _, _ = to_device_inputs(wl)
    assert lib.resolve_path(grads, wl.B + 1, wl.method, wl.max_iter) == path
    print(full_parity(lib, wl, grads=grads), flush=True)


@pytest.mark.parametrize("path_name", ["PATH_HYBRID", "PATH_REFILL"])
def test_coop_deterministic_and_close_to_two_pass(gpu_lib, path_name):
    wl = small_workload(BASE, sum(LENS), bucket_lens=LENS, K=4, dtype="bf16", method="cagrad", seed=31)
    grads, offs, order = to_device_inputs(wl)
    try:
        gpu_lib.set_resolve_path(getattr(gpu_lib, path_name))
        assert gpu_lib.resolve_path(grads, wl.B + 1, wl.method, wl.max_iter) == getattr(gpu_lib, path_name)
        r1 = run_resolve(gpu_lib, wl, grads, offs, order)
        r2 = run_resolve(gpu_lib, wl, grads, offs, order)
        gpu_lib.set_resolve_path(gpu_lib.PATH_TWO_PASS)
        r3 = run_resolve(gpu_lib, wl, grads, offs, order)
    finally:
        gpu_lib.set_resolve_path(0)
    assert np.array_equal(r1["gram"], r2["gram"]) and np.array_equal(r1["weights"], r2["weights"])
    assert torch.equal(r1["out"].view(torch.int16), r2["out"].view(torch.int16))
    d = np.sqrt(np.einsum("bii->bi", r3["gram"]))
    assert np.all(np.abs(r1["gram"] - r3["gram"]) <= 1e-6 * d[:, :, None] * d[:, None, :] + 1e-300)
    np.testing.assert_allclose(r1["weights"], r3["weights"], rtol=0, atol=1e-5)


def test_coop_wait_timeout_forced_from_host(coop):
    """A one-poll wait limit makes waiting workgroups give up at once.  The
    first bucket (25 MiB per task) takes every data workgroup microseconds to
    stream, while the solver polls its arrivals right at the start, so that
    wait expires: the call completes (no hang), the error word says so, the
    first bucket's Gram, weights and update are NaN, and the binding's
    checked call raises.  A normal call on the same workspace is clean."""
    lib, path = coop
    lens = [13_107_200, 65_536, 65_536, 131_072]
    wl = small_workload(BASE, sum(lens), bucket_lens=lens, K=4, dtype="bf16", method="mgda", seed=41)
    grads, offs, _ = to_device_inputs(wl)
    assert lib.resolve_path(grads, wl.B + 1, wl.method, wl.max_iter) == path
    ws = torch.empty(lib.workspace_size(wl.K, wl.N, wl.B, "bf16"), dtype=torch.uint8, device="cuda")
    G = torch.empty((wl.B, wl.K, wl.K), dtype=torch.float64, device="cuda")
    W = torch.empty((wl.B, wl.K), dtype=torch.float32, device="cuda")
    try:
        lib.set_wait_limit(1)
        out = lib.resolve(grads, offs, "mgda", 20, gram_out=G, weights=W, workspace=ws)
        err = lib.read_device_error(ws)
        with pytest.raises(lib.BkmooError, match="bounded wait"):
            lib.resolve(grads, offs, "mgda", 20, workspace=ws, check_error=True)
    finally:
        lib.set_wait_limit(1 << 22)
    assert err & lib.DEVERR_TIMEOUT
    assert bool(torch.isnan(G[0]).all()) and bool(torch.isnan(W[0]).all())
    assert bool(torch.isnan(out[:lens[0]].float()).all())
    out2 = lib.resolve(grads, offs, "mgda", 20, workspace=ws, check_error=True)
    assert lib.read_device_error(ws) == 0
    assert not bool(torch.isnan(out2.float()).any())
