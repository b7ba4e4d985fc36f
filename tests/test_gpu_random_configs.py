"""Seeded random small configurations through the same parity checks as the
hand-picked tests: K = 2..10, fp32 and bf16 inputs, either output type,
every method (exact solvers included), 0..20 iterations, CAGrad radii
0..0.9, 1..47 ragged buckets with empty and one-element ones, aligned and
unaligned rows, on the automatic path and on each forced path.  The
cooperative half draws a cooperative kernel first and then only cases it
can run (K <= 8 for the two-buffer kernel, K <= 10 for the single-buffer
one, aligned rows, non-exact methods) and asserts that it ran."""

import numpy as np
import pytest
import torch

from synth import WORKLOADS, small_workload
from tests.parity import full_parity, to_device_inputs

pytestmark = pytest.mark.gpu

BASES = {"bf16": WORKLOADS["llama3-8b-k4-mgda-bf16"], "f32": WORKLOADS["gpt2-124m-k4-pcgrad-f32"]}


def _draw(case, cooperative):
    rng = np.random.default_rng(20_261_202 + 1_000 * cooperative + case)
    path = str(rng.choice(["PATH_HYBRID", "PATH_REFILL"] if cooperative
                          else ["auto", "PATH_TWO_PASS", "PATH_HYBRID", "PATH_REFILL"]))
    Ks = [2, 3, 4, 4, 6, 8] if path == "PATH_HYBRID" else [2, 3, 4, 6, 8, 9, 10] if cooperative \
        else [2, 3, 4, 5, 8, 10]
    K = int(rng.choice(Ks))
    dt = str(rng.choice(["bf16", "f32"]))
    methods = ["mgda", "pcgrad", "cagrad", "mean"] + ([] if cooperative else ["mgda-exact", "cagrad-exact"])
    method = str(rng.choice(methods))
    iters = int(rng.choice([0, 1, 5, 20]))
    c = float(rng.choice([0.0, 0.3, 0.5, 0.9]))
    B = int(rng.integers(1, 48))
    lens = [int(x) for x in rng.integers(0, 100_000, size=B)]
    if rng.random() < 0.3:
        lens[int(rng.integers(B))] = int(rng.choice([0, 1, 7]))
    align = 8 if dt == "bf16" else 4
    if (cooperative or rng.random() < 0.7) and sum(lens) % align:
        lens[-1] += -sum(lens) % align
    if sum(lens) == 0:
        lens[-1] = 16
    out_dt = None if rng.random() < 0.7 else (torch.float32 if dt == "bf16" else torch.bfloat16)
    wl = small_workload(BASES[dt], sum(lens), bucket_lens=lens, K=K, dtype=dt, method=method, max_iter=iters,
                        cagrad_c=c, seed=7_000 + 100 * cooperative + case)
    return wl, out_dt, path


@pytest.mark.parametrize("cooperative", [False, True])
@pytest.mark.parametrize("case", range(16))
def test_random_config(gpu_lib, case, cooperative):
    wl, out_dt, path = _draw(case, cooperative)
    grads, _, _ = to_device_inputs(wl)
    forced = 0 if path == "auto" else getattr(gpu_lib, path)
    gpu_lib.set_resolve_path(forced)
    try:
        took = gpu_lib.resolve_path(grads, wl.B + 1, wl.method, wl.max_iter, out_dtype=out_dt)
        if cooperative:
            assert took == forced
        print(f"case {case}: K={wl.K} {wl.dtype}->{out_dt} {wl.method} it={wl.max_iter} c={wl.cagrad_c} "
              f"B={wl.B} N={wl.N} path {took}", flush=True)
        print(full_parity(gpu_lib, wl, grads=grads, out_dtype=out_dt), flush=True)
    finally:
        gpu_lib.set_resolve_path(0)
