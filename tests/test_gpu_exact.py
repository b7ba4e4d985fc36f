"""GPU parity of the exact per-bucket solvers (methods "mgda-exact" and
"cagrad-exact", support enumeration) against the oracle's exact solvers.

Tolerances: see tests/parity.py (assert_exact_weights).
"""

import numpy as np
import pytest
import torch

import oracle
from synth import WORKLOADS, small_workload
from tests.parity import assert_exact_weights as _compare, full_parity

pytestmark = pytest.mark.gpu


def _grams(k, nb, seed):
    """Gram matrices of seeded random task vectors: correlated, per-task
    scales over two decades, a seeded conflicting pair, and singular buckets
    (a duplicated task, a zero task, two colinear tasks)."""
    rng = np.random.default_rng(seed)
    out = []
    for b in range(nb):
        n = int(rng.integers(k + 2, 80))
        c = np.eye(k)
        for i in range(k):
            for j in range(i + 1, k):
                c[i, j] = c[j, i] = rng.uniform(-0.6, 0.8)
        ev, v = np.linalg.eigh(c)
        c = (v * np.maximum(ev, 1e-2)) @ v.T
        x = np.linalg.cholesky(c) @ rng.standard_normal((k, n))
        x *= np.exp(rng.uniform(-2.3, 2.3, size=(k, 1)))
        kind = b % 6
        if kind == 1:
            x[1] = x[0]
        elif kind == 2:
            x[rng.integers(k)] = 0.0
        elif kind == 3:
            x[-1] = 2.5 * x[0]
        out.append(x @ x.T)
    return np.stack(out)


@pytest.mark.parametrize("method", ["mgda", "cagrad"])
@pytest.mark.parametrize("K", [2, 3, 4, 5, 6, 8, 10])
def test_exact_solvers_stage_isolated(gpu_lib, K, method):
    nb = 96 if K >= 8 else 240
    G = _grams(K, nb, 3000 + 10 * K + (method == "cagrad"))
    print(f"case exact {method} K={K} B={nb}", flush=True)
    W, A = gpu_lib.solve(torch.from_numpy(G).cuda(), f"{method}-exact", cagrad_c=0.5)
    torch.cuda.synchronize()
    w_ora, a_ora = oracle.solve(G, method, cagrad_c=0.5, exact=True)
    _compare(G, W.cpu().numpy().astype(np.float64), A.cpu().numpy(), w_ora, a_ora, method,
             f"{method}-exact K={K}")


@pytest.mark.parametrize("c", [0.0, 0.2, 0.9])
def test_cagrad_exact_radius_range(gpu_lib, c):
    """c = 0 (vertices only: the task with the least <g_t, g_avg>, weights
    1/K) up to a wide trust region."""
    G = _grams(5, 120, 4100)
    W, A = gpu_lib.solve(torch.from_numpy(G).cuda(), "cagrad-exact", cagrad_c=c)
    torch.cuda.synchronize()
    w_ora, a_ora = oracle.solve(G, "cagrad", cagrad_c=c, exact=True)
    _compare(G, W.cpu().numpy().astype(np.float64), A.cpu().numpy(), w_ora, a_ora, "cagrad", f"c={c}")


def test_exact_non_finite_gram_gives_nan(gpu_lib):
    G = _grams(4, 3, 11)
    G[1, 0, 2] = G[1, 2, 0] = np.nan
    for m in ("mgda-exact", "cagrad-exact"):
        W, A = gpu_lib.solve(torch.from_numpy(G).cuda(), m, cagrad_c=0.5)
        W, A = W.cpu().numpy(), A.cpu().numpy()
        assert np.all(np.isnan(W[1])) and np.all(np.isnan(A[1]))
        assert np.all(np.isfinite(W[[0, 2]]))


def test_exact_rejects_k_above_10(gpu_lib):
    G = torch.eye(11, dtype=torch.float64, device="cuda").expand(2, 11, 11).contiguous()
    with pytest.raises(gpu_lib.BkmooError, match="EUNSUPPORTED"):
        gpu_lib.solve(G, "mgda-exact")


@pytest.mark.parametrize("method", ["mgda-exact", "cagrad-exact"])
@pytest.mark.parametrize("K", [2, 4, 8])
def test_exact_end_to_end(gpu_lib, K, method):
    """Gram, exact solve and combine through bkmoo_resolve on a small
    workload with ragged buckets, against the oracle end to end."""
    lens = [70_001, 1, 0, 33_333, 131_072, 7, 65_539, 40_000]
    base = WORKLOADS["llama3-8b-k8-cagrad-bf16"]
    wl = small_workload(base, sum(lens), bucket_lens=lens, K=K, method=method, seed=6000 + K)
    print(f"case {wl.name} K={K} {method}", flush=True)
    assert gpu_lib.resolve_path(torch.empty((K, 1), dtype=torch.bfloat16, device="cuda"), len(lens) + 1,
                                method=method, max_iter=0) == gpu_lib.PATH_TWO_PASS
    print(full_parity(gpu_lib, wl), flush=True)


def test_exact_never_takes_the_cooperative_path(gpu_lib):
    gpu_lib.set_resolve_path(gpu_lib.PATH_HYBRID)
    try:
        g = torch.empty((4, 1 << 26), dtype=torch.bfloat16, device="cuda")
        for m in ("mgda-exact", "cagrad-exact"):
            assert gpu_lib.resolve_path(g, 3, method=m, max_iter=0) == gpu_lib.PATH_TWO_PASS
    finally:
        gpu_lib.set_resolve_path(0)
