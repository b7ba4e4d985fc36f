"""GPU edge cases: invalid offsets, non-finite inputs, misaligned and
separately allocated rows, in-place update, one global bucket, empty input,
degenerate Gram matrices, invalid PCGrad orders and mismatched output
tensors refused by the binding."""

import numpy as np
import pytest
import torch

import oracle
from synth import WORKLOADS, fill_grads, small_workload
from tests.parity import assert_gram, assert_out, assert_weights, full_parity, host_out

pytestmark = pytest.mark.gpu

BASE = WORKLOADS["llama3-8b-k8-cagrad-bf16"]


def _host(t):
    return host_out(t)


def test_invalid_offsets_flag_error_and_touch_nothing(gpu_lib):
    K, N = 3, 10_000
    g = torch.randn((K, N), device="cuda")
    out = torch.full((N,), 7.0, device="cuda")
    ws = torch.empty(gpu_lib.workspace_size(K, N, 3, "f32"), dtype=torch.uint8, device="cuda")
    for bad in ([0, 5000, 4000, N], [0, 5000, 6000, N - 1], [1, 5000, 6000, N]):
        offs = torch.tensor(bad, dtype=torch.int64, device="cuda")
        G = torch.zeros((3, K, K), dtype=torch.float64, device="cuda")
        gpu_lib.resolve(g, offs, "mgda", out=out, gram_out=G, workspace=ws)
        assert gpu_lib.read_device_error(ws) == gpu_lib.DEVERR_OFFSETS
        assert torch.isnan(G).all()
        assert torch.all(out == 7.0)
    offs = torch.tensor([0, 5000, 6000, N], dtype=torch.int64, device="cuda")
    gpu_lib.resolve(g, offs, "mgda", out=out, workspace=ws)
    assert gpu_lib.read_device_error(ws) == 0


@pytest.mark.parametrize("method", ["mgda", "pcgrad", "cagrad", "mean"])
def test_nan_propagates_to_its_bucket_only(gpu_lib, method):
    wl = small_workload(BASE, 30_000, bucket_lens=[10_000, 10_000, 10_000], K=4, dtype="f32",
                        method=method, seed=3)
    g = fill_grads(wl, device="cuda")
    g[2, 12_345] = float("nan")
    offs = torch.from_numpy(wl.offsets()).cuda()
    W = torch.empty((3, 4), device="cuda")
    out = gpu_lib.resolve(g, offs, method, weights=W)
    torch.cuda.synchronize()
    assert torch.isnan(W[1]).all() and torch.isfinite(W[0]).all() and torch.isfinite(W[2]).all()
    assert torch.isnan(out[10_000:20_000]).all()
    assert torch.isfinite(out[:10_000]).all() and torch.isfinite(out[20_000:]).all()


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("layout", ["same_phase_shifted", "mixed_phase", "separate_buffers"])
def test_row_layouts(gpu_lib, dtype, layout):
    wl = small_workload(BASE, 90_011, bucket_lens=[30_000, 1, 60_010], K=5, dtype=dtype, seed=11)
    dense = fill_grads(wl, device="cuda")
    K, N = wl.K, wl.N
    tdt = dense.dtype
    if layout == "same_phase_shifted":
        # every row starts one element past a 16-byte boundary
        buf = torch.empty((K, N + 15), dtype=tdt, device="cuda")
        buf[:, 1:N + 1] = dense
        stride = N + 15
        flat = buf.view(-1)
        rows = [flat[i * stride + 1: i * stride + 1 + N] for i in range(K)]
    elif layout == "mixed_phase":
        buf = torch.empty(K * (N + 3), dtype=tdt, device="cuda")
        rows = []
        for i in range(K):
            s = i * (N + 3) + i % 3
            buf[s:s + N] = dense[i]
            rows.append(buf[s:s + N])
    else:
        rows = [dense[i].clone() for i in range(K)]
    offs = torch.from_numpy(wl.offsets()).cuda()
    ref = gpu_lib.resolve(dense, offs, wl.method, max_iter=wl.max_iter, cagrad_c=wl.cagrad_c)
    got = gpu_lib.resolve(rows, offs, wl.method, max_iter=wl.max_iter, cagrad_c=wl.cagrad_c)
    # the layout changes the load path, never the per-element arithmetic
    # or the reduction order of whole vectors; results agree to rounding
    torch.cuda.synchronize()
    r, g_ = oracle.decode_rows(_host(ref)), oracle.decode_rows(_host(got))
    np.testing.assert_allclose(g_, r, rtol=2e-2 if dtype == "bf16" else 1e-5, atol=1e-6)
    print(full_parity(gpu_lib, wl, grads=rows), flush=True)


@pytest.mark.parametrize("path,K", [("PATH_TWO_PASS", 4), ("PATH_HYBRID", 4), ("PATH_HYBRID", 6),
                                    ("PATH_HYBRID", 8)])
def test_in_place_update(gpu_lib, path, K):
    """The update written over one of the gradient rows equals the
    out-of-place update of the same path bitwise (every position is read
    before it is written, on each path)."""
    wl = small_workload(BASE, 350_008, bucket_lens=[20_000, 130_000, 1, 200_007], K=K, dtype="bf16", seed=4)
    g = fill_grads(wl, device="cuda")
    offs = torch.from_numpy(wl.offsets()).cuda()
    gpu_lib.set_resolve_path(getattr(gpu_lib, path))
    try:
        assert gpu_lib.resolve_path(g, wl.B + 1, wl.method, wl.max_iter) == getattr(gpu_lib, path)
        ref = gpu_lib.resolve(g.clone(), offs, wl.method, max_iter=wl.max_iter, cagrad_c=wl.cagrad_c)
        gpu_lib.resolve(g, offs, wl.method, max_iter=wl.max_iter, cagrad_c=wl.cagrad_c, out=g[2])
        torch.cuda.synchronize()
    finally:
        gpu_lib.set_resolve_path(0)
    assert torch.equal(g[2].view(torch.int16), ref.view(torch.int16))


def test_one_global_bucket(gpu_lib):
    """The trivial partition (one bucket) is the global method."""
    wl = small_workload(BASE, 123_457, bucket_lens=[123_457], K=8, seed=8)
    print(full_parity(gpu_lib, wl), flush=True)


def test_empty_input(gpu_lib):
    g = torch.empty((3, 0), device="cuda")
    offs = torch.zeros(2, dtype=torch.int64, device="cuda")
    G = torch.full((1, 3, 3), 5.0, dtype=torch.float64, device="cuda")
    W = torch.empty((1, 3), device="cuda")
    out = gpu_lib.resolve(g, offs, "cagrad", gram_out=G, weights=W)
    torch.cuda.synchronize()
    assert out.numel() == 0 and torch.all(G == 0)
    assert torch.allclose(W, torch.full((1, 3), 1 / 3, device="cuda"))


@pytest.mark.parametrize("method", ["mgda", "pcgrad", "cagrad"])
def test_degenerate_grams(gpu_lib, method):
    """Identical rows, zero rows and exactly opposite rows, per bucket."""
    K, n = 3, 4096
    g = torch.randn((K, 4 * n), device="cuda")
    g[1, :n] = g[0, :n]                      # bucket 0: duplicate tasks
    g[:, n:2 * n] = 0.0                      # bucket 1: all-zero gradients
    g[1, 2 * n:3 * n] = -2.0 * g[0, 2 * n:3 * n]   # bucket 2: opposite pair
    offs = torch.tensor([0, n, 2 * n, 3 * n, 4 * n], dtype=torch.int64, device="cuda")
    W = torch.empty((4, K), device="cuda")
    A = torch.empty((4, K), dtype=torch.float64, device="cuda")
    G = torch.empty((4, K, K), dtype=torch.float64, device="cuda")
    out = gpu_lib.resolve(g, offs, method, gram_out=G, weights=W, aux=A)
    torch.cuda.synchronize()
    x = g.cpu().numpy().astype(np.float64)
    Go = oracle.gram(x, offs.cpu().numpy())
    assert_gram(G.cpu().numpy(), Go, "f32")
    Wi, Ai = oracle.solve(G.cpu().numpy(), method)
    assert_weights(W.cpu().numpy().astype(np.float64), Wi, "weights")
    Wo, _ = oracle.solve(Go, method)
    assert_out(host_out(out), x, offs.cpu().numpy(), W.cpu().numpy().astype(np.float64), Wo, "f32")
    assert torch.all(out[n:2 * n] == 0)


def test_invalid_pcgrad_order_gives_nan_weights(gpu_lib):
    K = 4
    G = torch.eye(K, dtype=torch.float64, device="cuda").repeat(3, 1, 1)
    order = torch.tensor([[[j for j in range(K) if j != t] for t in range(K)]] * 3,
                         dtype=torch.int8, device="cuda")
    order[1, 2, 0] = 2          # task 2 listed against itself
    order[2, 0, 1] = 9          # out of range
    W, _ = gpu_lib.solve(G, "pcgrad", pcgrad_order=order)
    torch.cuda.synchronize()
    assert torch.all(W[0] == 1) and torch.isnan(W[1]).all() and torch.isnan(W[2]).all()


def test_binding_refuses_mismatched_outputs(gpu_lib):
    """Outputs and parameters on the host, or of the wrong shape or type,
    are refused before any call reaches the library; the inputs stay intact."""
    K, N, B = 3, 4096, 2
    g = torch.randn((K, N), device="cuda")
    keep = g.clone()
    offs = torch.tensor([0, 1000, N], dtype=torch.int64, device="cuda")
    bad_calls = [
        lambda: gpu_lib.resolve(g, offs, "mgda", out=torch.empty(N)),
        lambda: gpu_lib.resolve(g, offs, "mgda", out=torch.empty(N - 1, device="cuda")),
        lambda: gpu_lib.resolve(g, offs, "mgda", weights=torch.empty((B, K))),
        lambda: gpu_lib.resolve(g, offs, "mgda", gram_out=torch.empty((B, K, K), device="cuda")),
        lambda: gpu_lib.resolve(g, offs, "pcgrad", pcgrad_order=torch.zeros((B, K, K - 1), dtype=torch.int8)),
        lambda: gpu_lib.gram(g, offs, gram_out=torch.empty((B + 1, K, K), dtype=torch.float64, device="cuda")),
        lambda: gpu_lib.combine(g, offs, torch.full((B, K), 0.5)),
        lambda: gpu_lib.combine(g, offs, torch.full((B, K), 0.5, device="cuda"),
                                out=torch.empty((1, N), device="cuda")),
        lambda: gpu_lib.solve(torch.eye(K, dtype=torch.float64, device="cuda").expand(B, K, K).contiguous(),
                              "mgda", weights=torch.empty((B, K), dtype=torch.float64, device="cuda")),
    ]
    for call in bad_calls:
        with pytest.raises(ValueError):
            call()
    torch.cuda.synchronize()
    assert torch.equal(g, keep)
