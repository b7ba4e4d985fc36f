"""GPU parity of the HIP path against the float64 oracle on small seeded
workloads (several chunks per bucket, ragged tails, 1-element and empty
buckets), for every method, both input types and a range of task counts."""

import numpy as np
import pytest
import torch

import oracle
from synth import WORKLOADS, fill_grads, host_rows, small_workload
from tests.parity import assert_gram, assert_out, assert_weights, full_parity, host_out, run_resolve, \
    to_device_inputs

pytestmark = pytest.mark.gpu

BASE = {
    "mgda": WORKLOADS["llama3-8b-k4-mgda-bf16"],
    "pcgrad": WORKLOADS["gpt2-124m-k4-pcgrad-f32"],
    "cagrad": WORKLOADS["llama3-8b-k8-cagrad-bf16"],
}

# ragged buckets: several chunks, 1-element and empty buckets, odd sizes
LENS = [70_001, 1, 0, 33_333, 131_072, 7, 65_536 + 3, 40_000]


@pytest.mark.parametrize("method", ["mgda", "pcgrad", "cagrad", "mean"])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("K", [2, 3, 4, 8, 10, 16])
def test_small_parity(gpu_lib, method, dtype, K):
    base = BASE.get(method, BASE["mgda"])
    wl = small_workload(base, sum(LENS), bucket_lens=LENS, K=K, dtype=dtype, method=method,
                        seed=7000 + 10 * K + (dtype == "bf16"))
    print(f"case {wl.name} K={K} {dtype} {method}", flush=True)
    errs = full_parity(gpu_lib, wl)
    print(errs, flush=True)


def test_headline_shape_small(gpu_lib):
    """The headline workload's recipe (K=4 bf16 MGDA FW-20, correlations
    U[-0.8, 0.8]) at 1/500 of its size with its own 25 MiB cut scaled down."""
    wl = small_workload(WORKLOADS["llama3-8b-k4-mgda-bf16"], 16_060_522, bucket_elems=262_144)
    print(full_parity(gpu_lib, wl), flush=True)


def test_k2_mgda_closed_form_on_gpu(gpu_lib):
    """The K=2 configuration (4 buckets of 256 Ki fp32): GPU weights equal the
    two-task closed form computed from the vectors, in every clip branch."""
    wl = WORKLOADS["k2-mgda-1m-f32"]
    import dataclasses
    wl = dataclasses.replace(wl, task_scale=(0.1, 10.0), seed=1201)
    grads, offs, order = to_device_inputs(wl)
    res = run_resolve(gpu_lib, wl, grads, offs, order)
    rows = host_rows(grads, 0, wl.N).astype(np.float64)
    o = wl.offsets()
    for b in range(wl.B):
        g1, g2 = rows[0, o[b]:o[b + 1]], rows[1, o[b]:o[b + 1]]
        den = float(np.dot(g1 - g2, g1 - g2))
        a = min(max(float(np.dot(g2 - g1, g2)) / den, 0.0), 1.0)
        assert abs(res["aux"][b, 0] - a) <= 1e-4, (b, res["aux"][b], a)
        assert abs(res["aux"][b].sum() - 1.0) <= 1e-12
    print(full_parity(gpu_lib, wl), flush=True)


@pytest.mark.parametrize("out_dtype", [torch.float32, torch.bfloat16])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_output_dtype_conversion(gpu_lib, dtype, out_dtype):
    wl = small_workload(BASE["cagrad"], 200_003, bucket_lens=[100_000, 100_003], K=5, dtype=dtype,
                        seed=42)
    print(full_parity(gpu_lib, wl, out_dtype=out_dtype), flush=True)


def test_stage_calls_equal_resolve_bitwise(gpu_lib):
    """The two-pass resolve is exactly the three stage calls."""
    gpu_lib.set_resolve_path(gpu_lib.PATH_TWO_PASS)
    wl = small_workload(BASE["cagrad"], sum(LENS), bucket_lens=LENS, seed=99)
    grads, offs, order = to_device_inputs(wl)
    res = run_resolve(gpu_lib, wl, grads, offs, order)
    G = gpu_lib.gram(grads, offs)
    W, A = gpu_lib.solve(G, wl.method, wl.max_iter, wl.cagrad_c)
    out = gpu_lib.combine(grads, offs, W)
    torch.cuda.synchronize()
    gpu_lib.set_resolve_path(0)
    assert np.array_equal(G.cpu().numpy(), res["gram"])
    assert np.array_equal(W.cpu().numpy().astype(np.float64), res["weights"])
    assert np.array_equal(A.cpu().numpy(), res["aux"])
    assert torch.equal(out.view(torch.int16), res["out"].view(torch.int16))


@pytest.mark.parametrize("grid", [1, 3, 64, 0])
def test_bitwise_deterministic_across_grids(gpu_lib, grid):
    wl = small_workload(BASE["mgda"], sum(LENS), bucket_lens=LENS, K=6, seed=5)
    grads, offs, order = to_device_inputs(wl)
    gpu_lib.set_grid_override(0)
    ref = run_resolve(gpu_lib, wl, grads, offs, order)
    try:
        gpu_lib.set_grid_override(grid)
        again = run_resolve(gpu_lib, wl, grads, offs, order)
    finally:
        gpu_lib.set_grid_override(0)
    assert np.array_equal(ref["gram"], again["gram"])
    assert np.array_equal(ref["weights"], again["weights"])
    assert torch.equal(ref["out"].view(torch.int16), again["out"].view(torch.int16))
