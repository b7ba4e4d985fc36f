"""Parity at the full sizes of the five model-shaped workloads, in the launch
configuration the benchmark times (automatic grid).

At these sizes the oracle cannot redo everything, so each workload checks:
* every bucket: the oracle's solver run on the GPU's own Gram matrix
  (stage-isolated weights and method variable) and simplex feasibility;
* sampled buckets (first, last and fourteen seeded others, plus four seeded
  conflict buckets where the workload plants a strongly negative pair): the
  oracle's Gram, its end-to-end weights and the update, as in the
  small-size tests;
* 100k seeded element positions spread over all N: the update element
  against the exactly computed weighted sum of the GPU weights (bf16 output:
  the correctly rounded value; fp32 output: within K fp32 ulps of the sum
  of magnitudes);
* the exact MGDA and CAGrad solvers on the GPU's Gram (K <= 10): every
  bucket, or 48 seeded buckets when there are thousands, against the
  oracle's exact solvers;
* the sliced mode (8 slices per bucket, Gram pass over the slice offsets,
  slice-order reduction) and B = 1 (one bucket for all N, global MOO)
  against the per-bucket Grams: each Gram carries at most tau sqrt(G_ii G_jj)
  of fp32-accumulation error, so they agree within twice that;
* conflict diagnostics: every bucket against the oracle on the GPU's Gram,
  sampled buckets against the oracle's Gram, and, for the unit-scale
  normal workloads, every bucket's cosines against the correlation matrix
  the gradients were drawn with (sampling error ~1/sqrt(n_b) ~ 3e-4).
"""

import dataclasses
import gc

import numpy as np
import pytest
import torch

import oracle
from synth import WORKLOADS, fill_grads, host_rows
from tests.parity import TAU, assert_conflicts, assert_exact_weights, assert_gram, assert_out, \
    assert_weights, run_resolve, singular_buckets

pytestmark = [pytest.mark.gpu, pytest.mark.slow]


def _free():
    gc.collect()
    torch.cuda.empty_cache()


N_SAMPLED = 16      # buckets checked end to end per workload
N_CONFLICT = 4      # of which drawn with a strongly negative pair, where the workload has them


def _sampled_buckets(wl):
    """First, last and seeded others, up to N_SAMPLED; for a workload whose
    recipe plants a strongly negative pair in some buckets, N_CONFLICT of
    those as well (they define the K=8 CAGrad workload)."""
    rng = np.random.default_rng(wl.seed)
    picks = {0, wl.B - 1}
    if wl.corr.kind == "conflict":
        C = wl.correlations()
        iu = np.triu_indices(wl.K, 1)
        conflict = np.flatnonzero(C[:, iu[0], iu[1]].min(axis=1) <= 0.5 * wl.corr.c_hi)
        picks |= set(rng.choice(conflict, size=min(N_CONFLICT, len(conflict)), replace=False).tolist())
    rest = np.setdiff1d(np.arange(wl.B), sorted(picks))
    picks |= set(rng.choice(rest, size=min(max(N_SAMPLED - len(picks), 0), len(rest)),
                            replace=False).tolist())
    return sorted(picks), rng


def _check_workload(lib, wl, grads, offs, order, gram_cache=None):
    """gram_cache: bucket -> the oracle's Gram of that bucket, shared by calls
    on the same gradients (the methods of one bucket-size sweep)."""
    print(f"case {wl.name}: K={wl.K} N={wl.N} B={wl.B} {wl.dtype} {wl.method}", flush=True)
    res = run_resolve(lib, wl, grads, offs, order)
    orders_np = wl.orders() if wl.method == "pcgrad" else None
    # every bucket: stage-isolated solve and feasibility
    w_iso, a_iso = oracle.solve(res["gram"], wl.method, wl.max_iter, wl.cagrad_c, orders_np)
    assert_weights(res["weights"], w_iso, "weights(iso)", wl.name)
    assert_weights(res["aux"], a_iso, "aux(iso)", wl.name)
    assert np.all(np.isfinite(res["weights"]))
    if wl.method in ("mgda", "cagrad"):
        a = res["aux"]
        assert a.min() >= -1e-12 and np.abs(a.sum(1) - 1).max() <= 1e-9
    # sliced mode and global MOO at full size
    tau = TAU[wl.dtype]
    so = lib.slice_offsets(offs, 8)
    G8 = lib.gram_reduce(lib.gram(grads, so).view(wl.B, 8, wl.K, wl.K), lib.SLICES_BUCKET_MAJOR)
    G8 = G8.cpu().numpy()
    d = np.sqrt(np.einsum("bii->bi", np.maximum(res["gram"], 0)))
    assert np.all(np.abs(G8 - res["gram"]) <= 2 * tau * d[:, :, None] * d[:, None, :] + 1e-300), \
        f"{wl.name}: sliced Grams"
    G1 = lib.gram(grads, torch.tensor([0, wl.N], dtype=torch.int64, device=grads.device)).cpu().numpy()[0]
    Gs = res["gram"].sum(0)
    dg = np.sqrt(np.maximum(np.diag(Gs), 0))
    assert np.all(np.abs(G1 - Gs) <= 2 * tau * np.outer(dg, dg)), f"{wl.name}: global Gram"
    print("  sliced (T=8) and global (B=1) Grams agree", flush=True)
    # exact solvers on the GPU Gram
    if wl.K <= 10 and wl.method in ("mgda", "cagrad"):
        Gd = torch.from_numpy(res["gram"]).to(grads.device)
        W_ex, A_ex = lib.solve(Gd, f"{wl.method}-exact", cagrad_c=wl.cagrad_c)
        W_ex, A_ex = W_ex.cpu().numpy().astype(np.float64), A_ex.cpu().numpy()
        rs = np.random.default_rng(wl.seed + 77)
        sel = np.arange(wl.B) if wl.B <= 700 else np.sort(rs.choice(wl.B, size=48, replace=False))
        w_o, a_o = oracle.solve(res["gram"][sel], wl.method, cagrad_c=wl.cagrad_c, exact=True)
        assert_exact_weights(res["gram"][sel], W_ex[sel], A_ex[sel], w_o, a_o, wl.method,
                             f"{wl.name} {wl.method}-exact")
        print(f"  exact {wl.method}: {len(sel)} buckets match the oracle", flush=True)
    # conflict diagnostics on the GPU Gram, every bucket
    conf = [t.cpu().numpy() for t in lib.conflicts(torch.from_numpy(res["gram"]).to(grads.device))]
    assert_conflicts(conf, oracle.conflicts(res["gram"]), f"{wl.name} conflicts(iso)")
    if wl.dist == "normal" and wl.tensor_scale is None and wl.task_scale is None:
        C = wl.correlations()
        iu = np.triu_indices(wl.K, 1)
        rho = C[:, iu[0], iu[1]]
        n_b = np.maximum(np.diff(wl.offsets()), 1)[:, None]
        bound = 8 * (1 - rho ** 2) / np.sqrt(n_b) + 1e-3      # 8 sigma of a sample correlation
        err = np.abs(conf[0][:, iu[0], iu[1]] - rho)
        dev = err.max()
        assert np.all(err <= bound), f"{wl.name}: cosines {dev:.2e} away from the drawn correlations"
        clear = (np.abs(rho) > bound).all(axis=1)
        neg = (C[:, iu[0], iu[1]] < 0).sum(axis=1)
        assert np.array_equal(conf[2][clear, 2], neg[clear]), f"{wl.name}: conflict counts"
        print(f"  conflicts: {int((conf[2][:, 2] > 0).sum())} of {wl.B} buckets, max |cos - C| {dev:.1e}",
              flush=True)
    # sampled buckets end to end
    offs_np = wl.offsets()
    picks, rng = _sampled_buckets(wl)
    if gram_cache is None:
        gram_cache = {}
    for b in picks:
        lo, hi = int(offs_np[b]), int(offs_np[b + 1])
        rows = host_rows(grads, lo, hi)
        ob = np.array([0, hi - lo])
        x64 = oracle.decode_rows(rows)
        if b not in gram_cache:
            gram_cache[b] = oracle.gram(x64, ob)
        ora = {"gram": gram_cache[b]}
        ora["weights"], _ = oracle.solve(ora["gram"], wl.method, wl.max_iter, wl.cagrad_c,
                                         None if orders_np is None else orders_np[b:b + 1])
        assert_gram(res["gram"][b:b + 1], ora["gram"], wl.dtype, f"{wl.name} bucket {b}")
        tau = TAU[wl.dtype]
        assert_conflicts([c[b:b + 1] for c in conf], oracle.conflicts(ora["gram"]),
                         f"{wl.name} bucket {b} conflicts(e2e)", tol_cos=3 * tau, tol_sum=3 * tau,
                         sign_margin=3 * tau)
        skip = singular_buckets(ora["gram"]) if wl.method in ("mgda", "cagrad") else None
        assert_weights(res["weights"][b:b + 1], ora["weights"], "weights(e2e)", f"{wl.name} bucket {b}",
                       skip=skip)
        out_b = res["out"][lo:hi].cpu()
        store = out_b.view(torch.int16).numpy().view(np.uint16) if out_b.dtype == torch.bfloat16 \
            else out_b.numpy()
        assert_out(store, x64, ob, res["weights"][b:b + 1], ora["weights"], wl.dtype,
                   where=f"{wl.name} bucket {b}")
        del rows, x64, ora
    # sampled elements over all of N
    idx_np = np.sort(rng.choice(wl.N, size=100_000, replace=False)).astype(np.int64)
    idx = torch.from_numpy(idx_np).to(grads.device)
    xs = grads.index_select(1, idx)
    xs_np = host_rows(xs, 0, xs.shape[1])
    x64 = oracle.decode_rows(xs_np)
    bucket = np.searchsorted(offs_np, idx_np, side="right") - 1
    W = res["weights"][bucket]                              # [n, K]
    exact = np.einsum("nk,kn->n", W, x64)
    got_t = res["out"].index_select(0, idx).cpu()
    if wl.dtype == "bf16":
        got = got_t.view(torch.int16).numpy().view(np.uint16)
        want = oracle.f64_to_bf16_bits(exact)
        mism = np.mean(got != want)
        assert mism <= 1e-4, f"{wl.name}: {mism:.2e} of sampled bf16 outputs not correctly rounded"
    else:
        got = got_t.numpy().astype(np.float64)
        bound = wl.K * 2.0 ** -23 * np.einsum("nk,kn->n", np.abs(W), np.abs(x64)) + 1e-45
        assert np.all(np.abs(got - exact) <= bound), f"{wl.name}: fp32 output off by more than K ulps"
    del res, xs, got_t
    print(f"  ok: buckets {picks} checked end to end", flush=True)


# the path bkmoo_resolve takes for each workload (what bench.py times)
EXPECTED_PATH = {"k2-mgda-1m-f32": "PATH_TWO_PASS", "gpt2-124m-k4-pcgrad-f32": "PATH_HYBRID",
                 "llama3-8b-k4-mgda-bf16": "PATH_REFILL", "llama3-8b-k8-cagrad-bf16": "PATH_HYBRID"}


@pytest.mark.parametrize("name", list(EXPECTED_PATH))
def test_full_workload(gpu_lib, name):
    _free()
    wl = WORKLOADS[name]
    grads = fill_grads(wl, device="cuda")
    offs = torch.from_numpy(wl.offsets()).cuda()
    order = torch.from_numpy(wl.orders()).cuda() if wl.method == "pcgrad" else None
    gpu_lib.set_resolve_path(0)
    assert gpu_lib.resolve_path(grads, wl.B + 1, wl.method, wl.max_iter) == getattr(gpu_lib, EXPECTED_PATH[name])
    try:
        _check_workload(gpu_lib, wl, grads, offs, order)
    finally:
        del grads
        _free()


# the other methods on the two Llama-3-8B-shaped draws, and the path each
# takes at that shape
OTHER_METHODS = {
    "llama3-8b-k4-mgda-bf16": {"pcgrad": "PATH_HYBRID", "cagrad": "PATH_REFILL", "mean": "PATH_HYBRID"},
    "llama3-8b-k8-cagrad-bf16": {"mgda": "PATH_HYBRID", "pcgrad": "PATH_HYBRID"},
}


@pytest.mark.parametrize("name", list(OTHER_METHODS))
def test_full_llama_shapes_other_methods(gpu_lib, name):
    """The Llama-3-8B-shaped gradients (K=4 and K=8 bf16, 613 buckets of 25
    MiB) with the methods their workloads do not name, on the path the
    automatic choice gives each, through the same full-size checks."""
    _free()
    base = WORKLOADS[name]
    grads = fill_grads(base, device="cuda")
    offs = torch.from_numpy(base.offsets()).cuda()
    gpu_lib.set_resolve_path(0)
    try:
        grams = {}
        for m, path in OTHER_METHODS[name].items():
            wl = dataclasses.replace(base, name=f"{name}/{m}", method=m)
            assert gpu_lib.resolve_path(grads, wl.B + 1, m, wl.max_iter) == getattr(gpu_lib, path), m
            order = torch.from_numpy(wl.orders()).cuda() if m == "pcgrad" else None
            _check_workload(gpu_lib, wl, grads, offs, order, grams)
    finally:
        del grads
        _free()


@pytest.mark.parametrize("mib", [1, 5, 25, 100])
def test_full_qwen_k10_bucket_sweep(gpu_lib, mib):
    """K=10 fp32 heavy-tailed gradients, one draw per bucket size, all three
    methods on it."""
    _free()
    base = WORKLOADS[f"qwen-1.7b-k10-{mib}mib-mgda-f32"]
    grads = fill_grads(base, device="cuda")
    offs = torch.from_numpy(base.offsets()).cuda()
    gpu_lib.set_resolve_path(0)
    # every size takes the single-buffer cooperative kernel: 1 and 5 MiB
    # buckets in groups of 18 and 4, 25 and 100 MiB ones one at a time
    want = gpu_lib.PATH_REFILL
    for m in ("mgda", "pcgrad", "cagrad"):
        assert gpu_lib.resolve_path(grads, base.B + 1, m, 20 if m != "pcgrad" else 0) == want, (mib, m)
    try:
        grams = {}
        for m in ("mgda", "pcgrad", "cagrad"):
            wl = WORKLOADS[f"qwen-1.7b-k10-{mib}mib-{m}-f32"]
            order = torch.from_numpy(wl.orders()).cuda() if m == "pcgrad" else None
            _check_workload(gpu_lib, wl, grads, offs, order, grams)
    finally:
        del grads
        _free()
