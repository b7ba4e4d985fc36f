"""The single-read (resident) resolve against the oracle: every method and
input type for K = 2..4, ragged and unaligned buckets, a bucket larger than
the chip holds (two reads), determinism, agreement with the two-pass path,
and the bounded wait's timeout forced from the host."""

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


@pytest.fixture
def resident(gpu_lib):
    gpu_lib.set_resolve_path(gpu_lib.PATH_RESIDENT)
    yield gpu_lib
    gpu_lib.set_resolve_path(0)


@pytest.fixture
def two_pass(gpu_lib):
    gpu_lib.set_resolve_path(gpu_lib.PATH_TWO_PASS)
    yield gpu_lib
    gpu_lib.set_resolve_path(0)


@pytest.mark.parametrize("method", ["mgda", "pcgrad", "cagrad", "mean"])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("K", [2, 3, 4])
def test_resident_parity(resident, method, dtype, K):
    wl = small_workload(BASE, sum(LENS), bucket_lens=LENS, K=K, dtype=dtype, method=method,
                        seed=9000 + 10 * K + (dtype == "bf16"))
    grads, _, _ = to_device_inputs(wl)
    assert resident.resolve_path(grads, wl.B + 1, method) == resident.PATH_RESIDENT
    print(f"case {wl.name} K={K} {dtype} {method}", full_parity(resident, wl, grads=grads), flush=True)


@pytest.mark.parametrize("out_dtype", [torch.float32, torch.bfloat16])
def test_resident_output_types(resident, out_dtype):
    wl = small_workload(BASE, 200_000, bucket_lens=[99_999, 100_001], K=3, dtype="bf16", seed=77)
    print(full_parity(resident, wl, out_dtype=out_dtype), flush=True)


def test_resident_bucket_larger_than_chip(resident):
    """One K=2 fp32 bucket of 14.5M elements exceeds 256 workgroups x one
    segment, so workgroups hold several segments and re-read them."""
    wl = small_workload(WORKLOADS["k2-mgda-1m-f32"], 14_500_000, bucket_lens=[14_500_000], seed=5)
    print(full_parity(resident, wl), flush=True)


def test_resident_deterministic_and_close_to_two_pass(gpu_lib):
    wl = small_workload(BASE, sum(LENS), bucket_lens=LENS, K=4, dtype="bf16", method="cagrad", seed=31)
    grads, offs, order = to_device_inputs(wl)
    try:
        gpu_lib.set_resolve_path(gpu_lib.PATH_RESIDENT)
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


def test_resident_wait_timeout_forced_from_host(resident):
    """A one-poll wait limit makes waiting workgroups give up at once: the
    call still completes (no hang) and, if any wait expired, says so."""
    wl = small_workload(BASE, sum(LENS), bucket_lens=LENS, K=4, dtype="bf16", seed=41)
    grads, offs, _ = to_device_inputs(wl)
    ws = torch.empty(resident.workspace_size(wl.K, wl.N, wl.B, "bf16"), dtype=torch.uint8, device="cuda")
    try:
        resident.set_wait_limit(1)
        resident.resolve(grads, offs, "mgda", workspace=ws)
        err = resident.read_device_error(ws)
    finally:
        resident.set_wait_limit(1 << 22)
    assert err in (0, resident.DEVERR_TIMEOUT)
    resident.resolve(grads, offs, "mgda", workspace=ws)
    assert resident.read_device_error(ws) == 0
