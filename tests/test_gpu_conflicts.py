"""GPU parity of the per-bucket conflict diagnostics (bkmoo_conflicts)
against the oracle: on the same Gram matrices (stage-isolated), and end to
end from the gradients through the GPU Gram pass."""

import numpy as np
import pytest
import torch

import oracle
from synth import WORKLOADS, host_rows, small_workload
from tests.parity import TAU, assert_conflicts, to_device_inputs

pytestmark = pytest.mark.gpu


def _grams_with_edges(k, nb, seed):
    """Gram matrices of seeded random vectors, with edge buckets: a zero
    gradient, a duplicated and a negated task, exact ties (orthonormal
    rows), an all-zero bucket and non-finite entries."""
    rng = np.random.default_rng(seed)
    out = []
    for b in range(nb):
        n = int(rng.integers(1, 60))
        x = rng.standard_normal((k, n)) * np.exp(rng.uniform(-3, 3, size=(k, 1)))
        kind = b % 8
        if kind == 1:
            x[rng.integers(k)] = 0.0
        elif kind == 2:
            x[1] = x[0]
        elif kind == 3:
            x[-1] = -x[0]
        elif kind == 4:
            x = np.eye(k, max(k, n))[:, :max(k, n)]
        elif kind == 5:
            x[:] = 0.0
        out.append(x @ x.T)
    G = np.stack(out)
    if nb > 7:
        G[6, 0, 1] = G[6, 1, 0] = np.nan
        G[7, k - 1, k - 1] = np.inf
    return G


@pytest.mark.parametrize("K", [2, 3, 4, 8, 10, 16])
def test_conflicts_stage_isolated(gpu_lib, K):
    G = _grams_with_edges(K, 300, 500 + K)
    print(f"case conflicts stage-isolated K={K} B={len(G)}", flush=True)
    got = gpu_lib.conflicts(torch.from_numpy(G).cuda())
    torch.cuda.synchronize()
    assert_conflicts([t.cpu().numpy() for t in got], oracle.conflicts(G), f"K={K}")


def test_conflicts_optional_outputs_agree(gpu_lib):
    G = torch.from_numpy(_grams_with_edges(5, 70, 9)).cuda()
    full = [t.cpu() for t in gpu_lib.conflicts(G)]
    for which in range(3):
        flags = [i == which for i in range(3)]
        part = gpu_lib.conflicts(G, *flags)
        assert all((p is None) != f for p, f in zip(part, flags))
        bits = lambda t: t.view(torch.int64) if t.dtype == torch.float64 else t   # NaN-safe, bitwise
        assert torch.equal(bits(part[which].cpu()), bits(full[which]))


def test_conflicts_many_buckets(gpu_lib):
    """Thousands of buckets (several launch blocks), as at 1 MiB buckets."""
    G = _grams_with_edges(10, 6564, 77)
    got = gpu_lib.conflicts(torch.from_numpy(G).cuda())
    torch.cuda.synchronize()
    assert_conflicts([t.cpu().numpy() for t in got], oracle.conflicts(G), "B=6564")


LENS = [70_001, 1, 0, 33_333, 131_072, 7, 65_539, 40_000]


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("K", [2, 4, 8])
def test_conflicts_end_to_end(gpu_lib, K, dtype):
    base = WORKLOADS["llama3-8b-k8-cagrad-bf16"]     # conflict buckets: one pair in [-0.9, -0.5]
    wl = small_workload(base, sum(LENS), bucket_lens=LENS, K=K, dtype=dtype, seed=910 + K)
    print(f"case conflicts e2e {wl.name} K={K} {dtype}", flush=True)
    grads, offs, _ = to_device_inputs(wl)
    G = gpu_lib.gram(grads, offs)
    got = [t.cpu().numpy() for t in gpu_lib.conflicts(G)]
    rows = host_rows(grads, 0, wl.N)
    want = oracle.conflicts(oracle.gram(oracle.decode_rows(rows), wl.offsets()))
    tau = TAU[dtype]
    assert_conflicts(got, want, wl.name, tol_cos=3 * tau, tol_sum=3 * tau, sign_margin=3 * tau)
