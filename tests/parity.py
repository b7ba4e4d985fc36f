"""Shared helpers for the GPU parity tests: run the HIP path through the
binding, run the oracle on the same bytes, and compare with the tolerances
the method's specification fixes.

Tolerances (written here once, used by every parity test):

* Gram: |G_gpu - G_ora| <= tau * sqrt(G_ii G_jj) with tau = 1e-5 for fp32
  inputs and 1e-3 for bf16 inputs (fp32 accumulation); the Cauchy-Schwarz
  scale makes near-zero off-diagonals meaningful.  Empty buckets: exact 0.
* Weights and the method's variable: |dw| <= 1e-4 * max(1, |w_ora|).
  End to end, MGDA and CAGrad weights are compared only on buckets whose
  Gram matrix is non-singular (lambda_min > 1e-10 lambda_max): on a
  singular one the minimiser over the simplex is not unique (the update is),
  so those buckets are judged by their update alone.
* Update, per bucket, relative L2 <= 1e-4 where the denominator is
  ||ref_b||, or sum_i |w_i| ||g_{b,i}|| when ||ref_b|| < 1e-3 max_i ||g_{b,i}||
  (a near-stationary bucket whose update nearly cancels):
    - stage-isolated: against the oracle's combine of the GPU's own weights,
      after the same single RNE rounding to the output type;
    - end to end: ||gpu - d|| <= ||round(d) - d|| + 1e-4 ||d|| with d the
      oracle's float64 update from its own weights (the output type's own
      rounding is unavoidable and is not counted against the path).
* Conflict diagnostics: from the same Gram, cosines within 1e-15 and the
  summary within 1e-14 (fp64, only the summation order differs), counts
  exact, the argmin pair exact when the smallest cosine is unique by more
  than 1e-14 (else the GPU's pair must attain the minimum); end to end
  (GPU Gram vs exact Gram) cosines and summary within 3 tau, since a Gram
  error of tau sqrt(G_ii G_jj) moves a cosine by at most ~2 tau, and signs
  compared only on pairs with |cos| > 3 tau.
"""

from __future__ import annotations

import numpy as np
import torch

import oracle
from synth import fill_grads, host_rows

TAU = {"f32": 1e-5, "bf16": 1e-3}
W_TOL = 1e-4
OUT_TOL = 1e-4


def to_device_inputs(wl, device="cuda", grads=None):
    """Seeded grads [K, N], offsets and (PCGrad) visiting orders on the device."""
    if grads is None:
        grads = fill_grads(wl, device=device)
    offs = torch.from_numpy(wl.offsets()).to(device)
    order = torch.from_numpy(wl.orders()).to(device) if wl.method == "pcgrad" else None
    return grads, offs, order


def host_out(t: torch.Tensor) -> np.ndarray:
    t = t.cpu()
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).numpy().view(np.uint16)
    return t.numpy()


def run_resolve(lib, wl, grads, offs, order, out_dtype=None):
    K, B = wl.K, wl.B
    dev = offs.device
    G = torch.empty((B, K, K), dtype=torch.float64, device=dev)
    W = torch.empty((B, K), dtype=torch.float32, device=dev)
    A = torch.empty((B, K), dtype=torch.float64, device=dev)
    out = lib.resolve(grads, offs, wl.method, max_iter=wl.max_iter, cagrad_c=wl.cagrad_c,
                      pcgrad_order=order, out_dtype=out_dtype, gram_out=G, weights=W, aux=A)
    torch.cuda.synchronize()
    return {"gram": G.cpu().numpy(), "weights": W.cpu().numpy().astype(np.float64),
            "aux": A.cpu().numpy(), "out": out}


def assert_gram(g_gpu, g_ora, dtype, where=""):
    tau = TAU[dtype]
    d = np.sqrt(np.maximum(np.einsum("bii->bi", g_ora), 0.0))
    scale = d[:, :, None] * d[:, None, :]
    diff = np.abs(g_gpu - g_ora)
    zero = scale == 0.0
    assert np.all(diff[zero] == 0.0), f"{where}: empty-bucket Gram not exactly 0"
    if np.any(~zero):
        rel = diff[~zero] / scale[~zero]
        assert rel.max() <= tau, f"{where}: Gram rel err {rel.max():.3e} > {tau}"
    return float((diff / np.where(zero, 1.0, scale)).max())


def singular_buckets(grams: np.ndarray) -> np.ndarray:
    """Buckets whose Gram matrix has lambda_min <= 1e-10 lambda_max (or is 0)."""
    out = np.zeros(len(grams), dtype=bool)
    for b, G in enumerate(grams):
        if not np.all(np.isfinite(G)):
            continue
        ev = np.linalg.eigvalsh(G)
        out[b] = ev[-1] <= 0.0 or ev[0] <= 1e-10 * ev[-1]
    return out


def assert_weights(w_gpu, w_ora, what, where="", skip=None):
    err = np.abs(w_gpu - w_ora) / np.maximum(1.0, np.abs(w_ora))
    assert np.all(np.isfinite(w_gpu) == np.isfinite(w_ora)), f"{where}: {what} finiteness differs"
    fin = np.isfinite(w_ora)
    if skip is not None:
        fin &= ~np.asarray(skip)[:, None]
    m = float(err[fin].max()) if np.any(fin) else 0.0
    assert m <= W_TOL, f"{where}: {what} err {m:.3e} > {W_TOL} at {np.unravel_index(np.argmax(np.where(fin, err, 0)), err.shape)}"
    return m


def _bucket_den(ref_b, x_b, w_b):
    nrm = float(np.linalg.norm(ref_b))
    gn = np.linalg.norm(x_b, axis=1)
    if nrm < 1e-3 * float(gn.max(initial=0.0)):
        nrm = float(np.sum(np.abs(w_b) * gn))
    return nrm


def assert_out(out_gpu_store, x64, offs, w_gpu, w_ora, out_dtype, lo_hi=None, where=""):
    """out_gpu_store: host storage (float32 or bf16 bits) of the GPU update for
    columns [lo, hi) of x64 (float64 [K, hi-lo]); offsets relative to lo."""
    got = oracle.decode_rows(out_gpu_store)
    worst = [0.0, 0.0]
    for b in range(len(offs) - 1):
        lo, hi = int(offs[b]), int(offs[b + 1])
        if hi == lo:
            continue
        xb = x64[:, lo:hi]
        g = got[lo:hi]
        # stage-isolated: the oracle's combine of the GPU weights, same rounding
        ref = oracle.decode_rows(oracle.round_to_dtype(w_gpu[b] @ xb, out_dtype))
        den = _bucket_den(ref, xb, w_gpu[b])
        e1 = float(np.linalg.norm(g - ref)) / den if den > 0 else float(np.linalg.norm(g - ref))
        assert e1 <= OUT_TOL, f"{where}: bucket {b} stage-isolated update err {e1:.3e}"
        # end to end: against the exact update from the oracle's weights
        if w_ora is not None and np.all(np.isfinite(w_ora[b])):
            d = w_ora[b] @ xb
            rd = oracle.decode_rows(oracle.round_to_dtype(d, out_dtype))
            den2 = _bucket_den(d, xb, w_ora[b])
            allow = float(np.linalg.norm(rd - d)) + OUT_TOL * den2
            e2 = float(np.linalg.norm(g - d))
            assert e2 <= allow * (1 + 1e-12) + 1e-300, \
                f"{where}: bucket {b} end-to-end update err {e2:.3e} > {allow:.3e}"
            worst[1] = max(worst[1], (e2 - float(np.linalg.norm(rd - d))) / den2 if den2 > 0 else 0.0)
        worst[0] = max(worst[0], e1)
    return worst


def oracle_method(method):
    """The oracle's (method, exact) for a library method name."""
    if method.endswith("-exact"):
        return method[:-len("-exact")], True
    return method, False


def oracle_for(wl, rows_np, offs_np, orders_np):
    m, exact = oracle_method(wl.method)
    return oracle.resolve(rows_np, offs_np, m, max_iter=wl.max_iter, cagrad_c=wl.cagrad_c,
                          orders=orders_np, exact=exact)


def full_parity(lib, wl, grads=None, out_dtype=None):
    """Run the HIP path on `wl` (small enough for the oracle) and check
    every stage against the oracle.  Returns the worst errors seen."""
    grads, offs, order = to_device_inputs(wl, grads=grads)
    res = run_resolve(lib, wl, grads, offs, order, out_dtype=out_dtype)
    rows = host_rows(grads if isinstance(grads, torch.Tensor) else torch.stack(list(grads)), 0, wl.N)
    offs_np = wl.offsets()
    orders_np = wl.orders() if wl.method == "pcgrad" else None
    ora = oracle_for(wl, rows, offs_np, orders_np)
    odt = wl.dtype if out_dtype is None else ("f32" if out_dtype == torch.float32 else "bf16")
    e_g = assert_gram(res["gram"], ora["gram"], wl.dtype, wl.name)
    # stage-isolated solve: the oracle solver on the GPU's own Gram
    m, exact = oracle_method(wl.method)
    w_iso, a_iso = oracle.solve(res["gram"], m, wl.max_iter, wl.cagrad_c, orders_np, exact=exact)
    e_wi = assert_weights(res["weights"], w_iso, "weights(iso)", wl.name)
    assert_weights(res["aux"], a_iso, "aux(iso)", wl.name)
    # end to end: the oracle solver on the oracle Gram
    skip = singular_buckets(ora["gram"]) if m in ("mgda", "cagrad") else None
    e_we = assert_weights(res["weights"], ora["weights"], "weights(e2e)", wl.name, skip=skip)
    x64 = oracle.decode_rows(rows)
    e_o = assert_out(host_out(res["out"]), x64, offs_np, res["weights"], ora["weights"], odt,
                     where=wl.name)
    return {"gram": e_g, "w_iso": e_wi, "w_e2e": e_we, "out_iso": e_o[0], "out_e2e": e_o[1]}


def assert_conflicts(got, want, where="", tol_cos=1e-15, tol_sum=1e-14, sign_margin=None):
    """Compare (cos, summary, pairs) from the GPU with the oracle's.  With
    `sign_margin` (end to end) the pair statistics are compared only where
    the exact cosine is farther than the margin from 0 or from a tie."""
    cos_g, sum_g, pr_g = (np.asarray(t) for t in got)
    cos_o, sum_o, pr_o = (np.asarray(t) for t in want)
    nb, k, _ = cos_o.shape
    bad = ~np.isfinite(cos_o).all(axis=(1, 2))
    assert np.array_equal(bad, ~np.isfinite(cos_g).all(axis=(1, 2))), where
    assert np.all(pr_g[bad] == -1) and np.all(np.isnan(sum_g[bad])), where
    ok = ~bad
    dc = np.abs(cos_g[ok] - cos_o[ok]).max() if ok.any() else 0.0
    assert dc <= tol_cos, f"{where}: cosines differ by {dc:.3e} > {tol_cos:.1e}"
    ds = np.abs(sum_g[ok] - sum_o[ok]).max() if ok.any() else 0.0
    assert ds <= tol_sum, f"{where}: summary differs by {ds:.3e} > {tol_sum:.1e}"
    iu = np.triu_indices(k, 1)
    for b in np.nonzero(ok)[0]:
        vals = cos_o[b][iu]
        i, j = int(pr_g[b, 0]), int(pr_g[b, 1])
        assert 0 <= i < j < k, f"{where} bucket {b}: invalid pair {(i, j)}"
        assert abs(cos_o[b, i, j] - sum_o[b, 2]) <= tol_sum + 2 * tol_cos, \
            f"{where} bucket {b}: pair {(i, j)} does not attain the minimum"
        gap = np.sort(vals)[1] - vals.min() if len(vals) > 1 else np.inf
        if gap > tol_sum + 2 * tol_cos:
            assert (i, j) == (int(pr_o[b, 0]), int(pr_o[b, 1])), f"{where} bucket {b}: argmin pair"
        if sign_margin is None:
            assert pr_g[b, 2] == pr_o[b, 2], f"{where} bucket {b}: conflict count"
        else:
            clear = np.abs(vals) > sign_margin
            neg_g = (cos_g[b][iu] < 0)[clear]
            neg_o = (vals < 0)[clear]
            assert np.array_equal(neg_g, neg_o), f"{where} bucket {b}: conflict signs"
            if clear.all():
                assert pr_g[b, 2] == pr_o[b, 2], f"{where} bucket {b}: conflict count"


def assert_exact_weights(G, w_gpu, a_gpu, w_ora, a_ora, method, where):
    """Exact solvers: both sides solve the same small fp64 systems by
    different factorisations (Gaussian elimination on the GPU, least squares
    or an inverse in the oracle), so they agree to ~cond * 1e-16.  On a
    non-singular Gram the method variable (fp64 aux) must agree to
    1e-7 max(1, |a|) and the fp32 weights to 1e-6 max(1, |w|).  On a singular
    one the minimiser over the simplex need not be unique: the update
    (measured through G) must agree to 1e-6 of the gradient scale, MGDA's
    objective to 1e-9 of it, and the GPU variable must lie on the simplex."""
    sing = singular_buckets(G)
    for b in range(len(G)):
        if not sing[b]:
            da = np.abs(a_gpu[b] - a_ora[b]) / np.maximum(1.0, np.abs(a_ora[b]))
            dw = np.abs(w_gpu[b] - w_ora[b]) / np.maximum(1.0, np.abs(w_ora[b]))
            assert da.max() <= 1e-7, f"{where} bucket {b}: aux off by {da.max():.2e}"
            assert dw.max() <= 1e-6, f"{where} bucket {b}: weights off by {dw.max():.2e}"
            continue
        g = G[b]
        scale = max(float(np.max(np.diag(g))), 1e-300)
        dd = w_gpu[b] - w_ora[b]
        upd = float(dd @ g @ dd)                  # ||d_gpu - d_ora||^2
        assert upd <= (1e-6) ** 2 * scale * max(1.0, float(np.abs(w_ora[b]).sum()) ** 2), \
            f"{where} bucket {b} (singular): updates differ"
        if method == "mgda":
            qg, qo = float(a_gpu[b] @ g @ a_gpu[b]), float(a_ora[b] @ g @ a_ora[b])
            assert abs(qg - qo) <= 1e-9 * scale, f"{where} bucket {b} (singular): objective"
        assert a_gpu[b].min() >= -1e-12 and abs(a_gpu[b].sum() - 1.0) <= 1e-9
