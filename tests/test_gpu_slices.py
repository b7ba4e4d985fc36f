"""GPU parity of the sliced (partial-Gram) mode: every bucket cut into T
slices, per-slice Gram matrices, and their slice-order sum; the sharded
resolve emulated on one GPU; and B = 1 (global MOO, one bucket for the
whole vector)."""

import numpy as np
import pytest
import torch

import oracle
from synth import WORKLOADS, host_rows, small_workload
from tests.parity import assert_gram, assert_out, assert_weights, host_out, singular_buckets, \
    to_device_inputs

pytestmark = pytest.mark.gpu

LENS = [70_001, 1, 0, 33_333, 131_072, 7, 65_539, 40_000]


@pytest.mark.parametrize("T", [1, 2, 3, 8, 64])
def test_slice_offsets_match_oracle(gpu_lib, T):
    rng = np.random.default_rng(T)
    lens = LENS + [int(x) for x in rng.integers(0, 10_000, size=50)] + [(1 << 33) + 12345]
    offs = np.concatenate([[0], np.cumsum(lens)]).astype(np.int64)
    got = gpu_lib.slice_offsets(torch.from_numpy(offs).cuda(), T).cpu().numpy()
    assert np.array_equal(got, oracle.slice_offsets(offs, T))


@pytest.mark.parametrize("layout", [0, 1])
@pytest.mark.parametrize("T", [1, 2, 7])
def test_gram_reduce_bitwise(gpu_lib, T, layout):
    rng = np.random.default_rng(40 + T)
    parts = rng.standard_normal((T, 37, 5, 5)) * np.exp(rng.uniform(-20, 20, size=(T, 37, 1, 1)))
    x = parts if layout == gpu_lib.SLICES_RANK_MAJOR else np.ascontiguousarray(parts.transpose(1, 0, 2, 3))
    got = gpu_lib.gram_reduce(torch.from_numpy(x).cuda(), layout).cpu().numpy()
    assert np.array_equal(got, oracle.gram_reduce(parts))


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("T", [2, 8])
def test_sharded_resolve_emulated(gpu_lib, T, dtype):
    """T ranks on one GPU: rank r gathers slice r of every task's bucket into
    a contiguous buffer (the stand-in for the all-to-all), runs the Gram pass
    on it, the T partial sets are stacked (the all-gather) and reduced in rank
    order, every rank solves the same Grams, and rank r combines its slice.
    The reassembled update must match the oracle end to end."""
    wl = small_workload(WORKLOADS["llama3-8b-k4-mgda-bf16"], sum(LENS), bucket_lens=LENS, K=4,
                        dtype=dtype, seed=7100 + T)
    print(f"case sharded emulation T={T} {dtype}", flush=True)
    grads, offs, _ = to_device_inputs(wl)
    so = gpu_lib.slice_offsets(offs, T).cpu().numpy()
    B = wl.B
    idx = [np.concatenate([np.arange(so[b * T + r], so[b * T + r + 1]) for b in range(B)]).astype(np.int64)
           for r in range(T)]
    parts = []
    rank_data = []
    for r in range(T):
        sel = torch.from_numpy(idx[r]).cuda()
        xr = grads.index_select(1, sel).contiguous()
        lens_r = np.array([so[b * T + r + 1] - so[b * T + r] for b in range(B)])
        offs_r = torch.from_numpy(np.concatenate([[0], np.cumsum(lens_r)]).astype(np.int64)).cuda()
        parts.append(gpu_lib.gram(xr, offs_r))
        rank_data.append((sel, xr, offs_r))
    G = gpu_lib.gram_reduce(torch.stack(parts).contiguous())
    W, A = gpu_lib.solve(G, wl.method, wl.max_iter, wl.cagrad_c)
    out = torch.empty(wl.N, dtype=grads.dtype, device="cuda")
    for sel, xr, offs_r in rank_data:
        out.index_copy_(0, sel, gpu_lib.combine(xr, offs_r, W))
    torch.cuda.synchronize()
    rows = host_rows(grads, 0, wl.N)
    ora = oracle.resolve(rows, wl.offsets(), wl.method, max_iter=wl.max_iter)
    assert_gram(G.cpu().numpy(), ora["gram"], dtype, f"T={T}")
    w = W.cpu().numpy().astype(np.float64)
    w_iso, _ = oracle.solve(G.cpu().numpy(), wl.method, wl.max_iter)
    assert_weights(w, w_iso, "weights(iso)", f"T={T}")
    assert_weights(w, ora["weights"], "weights(e2e)", f"T={T}", skip=singular_buckets(ora["gram"]))
    assert_out(host_out(out), oracle.decode_rows(rows), wl.offsets(), w, ora["weights"], dtype,
               where=f"T={T}")
    # the partial Grams are the oracle's slice Grams
    sub = oracle.gram(oracle.decode_rows(rows), so)
    parts_ora = sub.reshape(B, T, 4, 4).transpose(1, 0, 2, 3)
    for r in range(T):
        assert_gram(parts[r].cpu().numpy(), parts_ora[r], dtype, f"rank {r} of {T}")


def test_sliced_gram_in_one_pass(gpu_lib):
    """The Gram pass over the B*T slice offsets (bucket-major) and the
    reduction give the bucket Grams."""
    wl = small_workload(WORKLOADS["llama3-8b-k8-cagrad-bf16"], sum(LENS), bucket_lens=LENS, K=6, seed=71)
    grads, offs, _ = to_device_inputs(wl)
    T = 5
    so = gpu_lib.slice_offsets(offs, T)
    sub = gpu_lib.gram(grads, so)
    G = gpu_lib.gram_reduce(sub.view(wl.B, T, 6, 6), gpu_lib.SLICES_BUCKET_MAJOR)
    rows = oracle.decode_rows(host_rows(grads, 0, wl.N))
    assert_gram(sub.cpu().numpy(), oracle.gram(rows, so.cpu().numpy()), wl.dtype, "slices")
    assert_gram(G.cpu().numpy(), oracle.gram(rows, wl.offsets()), wl.dtype, "reduced")


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_global_moo_one_bucket(gpu_lib, dtype):
    """B = 1: the whole vector is one bucket (global MOO, the 'without
    buckets' configuration), here 48 Mi elements: 1,536 (bf16) or 3,072
    (fp32) chunks, two or three finalize groups."""
    wl = small_workload(WORKLOADS["llama3-8b-k4-mgda-bf16"], 48 << 20, bucket_lens=[48 << 20], K=4,
                        dtype=dtype, seed=72)
    print(f"case global MOO {dtype}: N={wl.N}", flush=True)
    grads, offs, _ = to_device_inputs(wl)
    G = gpu_lib.gram(grads, offs).cpu().numpy()
    rows = oracle.decode_rows(host_rows(grads, 0, wl.N))
    assert_gram(G, oracle.gram(rows, wl.offsets()), dtype, "B=1")
