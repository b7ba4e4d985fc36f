"""The no-allocation resolve (bkmoo_resolve_noalloc: the library's fixed
device scratch instead of a caller's workspace) against bkmoo_resolve on the
same inputs, through the C ABI: equal Gram matrices, weights, method
variables and update, bit for bit, for consecutive calls on the shared
scratch (each later call on a different and partly smaller input, so
leftovers of the previous call in the scratch would show), on the two
cooperative paths and on the two-pass path."""

import pytest
import torch

from synth import WORKLOADS, small_workload
from tests.parity import to_device_inputs

pytestmark = pytest.mark.gpu

BASE = WORKLOADS["llama3-8b-k4-mgda-bf16"]


def _both(lib, wl, path):
    grads, offs, order = to_device_inputs(wl)
    dev = grads.device
    K, B = wl.K, wl.B
    res = []
    lib.set_resolve_path(path)
    try:
        assert lib.resolve_path(grads, B + 1, wl.method, wl.max_iter) == path
        for noalloc in (False, True):
            G = torch.full((B, K, K), float("nan"), dtype=torch.float64, device=dev)
            W = torch.full((B, K), float("nan"), dtype=torch.float32, device=dev)
            A = torch.full((B, K), float("nan"), dtype=torch.float64, device=dev)
            out = torch.full((wl.N,), float("nan"), dtype=grads.dtype, device=dev)
            if noalloc:
                lib.resolve_noalloc(grads, offs, wl.method, out, wl.max_iter, wl.cagrad_c, order,
                                    gram_out=G, weights=W, aux=A)
            else:
                lib.resolve(grads, offs, wl.method, wl.max_iter, wl.cagrad_c, order, out=out, gram_out=G,
                            weights=W, aux=A)
            torch.cuda.synchronize()
            res.append((G, W, A, out))
    finally:
        lib.set_resolve_path(0)
    (G1, W1, A1, o1), (G2, W2, A2, o2) = res
    assert not bool(torch.isnan(G1).any()) and not bool(torch.isnan(o1.float()).any())
    assert torch.equal(G1, G2) and torch.equal(W1, W2) and torch.equal(A1, A2)
    iv = torch.int16 if o1.dtype == torch.bfloat16 else torch.int32
    assert torch.equal(o1.view(iv), o2.view(iv))


def test_noalloc_equals_resolve_on_consecutive_calls(gpu_lib):
    lib = gpu_lib
    # 1: K=4 bf16, ten ragged buckets (an empty and a one-element one), hybrid path
    lens = [300_000, 0, 250_003, 1, 180_000, 420_000, 99_999, 310_000, 200_005, 240_000]
    lens[-1] += -sum(lens) % 8
    wl1 = small_workload(BASE, sum(lens), bucket_lens=lens, K=4, dtype="bf16", method="mgda", seed=8101)
    print(f"case noalloc 1: K=4 bf16 mgda B={wl1.B} N={wl1.N} hybrid", flush=True)
    _both(lib, wl1, lib.PATH_HYBRID)
    # 2: smaller, K=3 fp32 CAGrad on the two passes
    lens = [70_001, 33_333, 5, 96_661]
    wl2 = small_workload(WORKLOADS["gpt2-124m-k4-pcgrad-f32"], sum(lens), bucket_lens=lens, K=3, dtype="f32",
                         method="cagrad", seed=8102)
    print(f"case noalloc 2: K=3 f32 cagrad B={wl2.B} N={wl2.N} two-pass", flush=True)
    _both(lib, wl2, lib.PATH_TWO_PASS)
    # 3: K=8 bf16 PCGrad with visiting orders, hybrid path, after the smaller call
    lens = [150_000, 262_144, 77_777, 300_001, 180_000]
    lens[-1] += -sum(lens) % 8
    wl3 = small_workload(BASE, sum(lens), bucket_lens=lens, K=8, dtype="bf16", method="pcgrad", seed=8103)
    print(f"case noalloc 3: K=8 bf16 pcgrad B={wl3.B} N={wl3.N} hybrid", flush=True)
    _both(lib, wl3, lib.PATH_HYBRID)
    # 4: the second case again, now after a larger call
    print("case noalloc 4: case 2 again", flush=True)
    _both(lib, wl2, lib.PATH_TWO_PASS)
    # 5: K=10 fp32 MGDA on the single-buffer path (bucket groups), then case 1
    #    on that path after it
    lens = [120_000, 64_001, 0, 200_000, 33_333, 150_000, 90_000, 111_111, 76_543, 88_888]
    lens[-1] += -sum(lens) % 4
    wl5 = small_workload(WORKLOADS["gpt2-124m-k4-pcgrad-f32"], sum(lens), bucket_lens=lens, K=10, dtype="f32",
                         method="mgda", seed=8105)
    print(f"case noalloc 5: K=10 f32 mgda B={wl5.B} N={wl5.N} refill", flush=True)
    _both(lib, wl5, lib.PATH_REFILL)
    print("case noalloc 6: case 1 on the refill path", flush=True)
    _both(lib, wl1, lib.PATH_REFILL)


def test_noalloc_needs_an_output(gpu_lib):
    """The binding allocates nothing for this entry point: no output, no call."""
    wl = small_workload(BASE, 1024, bucket_lens=[1024], K=2, dtype="bf16", seed=8104)
    grads, offs, _ = to_device_inputs(wl)
    with pytest.raises(TypeError):
        gpu_lib.resolve_noalloc(grads, offs, "mgda")
