"""Plain float64 restatement of Bucket-Level MOO (test infrastructure only).

Notation.  The paper writes T for the number of languages and K for the
number of buckets; this code writes K for the languages (tasks) and B for the
buckets.  For bucket b the local gradient set is the K rows
x_0[o_b:o_{b+1}], ..., x_{K-1}[o_b:o_{b+1}] (Section 3.2, the set G_(k)).

Everything here is float64 numpy, one bucket at a time, with no blocking,
fusion or reordering beyond what each definition states.  Inputs are float32
arrays or bfloat16 bit patterns (uint16); both convert to float64 exactly.
"""

from __future__ import annotations

import itertools
import math
from typing import Optional

import numpy as np

# ----------------------------------------------------------------------------
# storage formats
# ----------------------------------------------------------------------------


def bf16_bits_to_f64(bits: np.ndarray) -> np.ndarray:
    """bfloat16 bit patterns -> float64 (exact: bf16 is the top half of fp32)."""
    u = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
    return u.view(np.float32).astype(np.float64)


def decode_rows(rows: np.ndarray) -> np.ndarray:
    """float32 rows, or uint16 bfloat16 bit patterns, -> float64 rows."""
    rows = np.asarray(rows)
    if rows.dtype == np.uint16:
        return bf16_bits_to_f64(rows)
    if rows.dtype == np.float32:
        return rows.astype(np.float64)
    if rows.dtype == np.float64:
        return rows
    raise TypeError(f"unsupported storage dtype {rows.dtype}")


def f64_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float64 to bfloat16 once, to nearest with ties to even.

    bfloat16 keeps 8 significant bits and fp32's exponent range (normal
    exponents -126..127, subnormal quantum 2^-133).  With x = m 2^e, m in
    [0.5, 1), the bf16 quantum at x is 2^(max(e, -125) - 8); rounding x to a
    multiple of it (numpy's rint is ties-to-even) is the single correct
    rounding.  Results of magnitude >= 2^128 overflow to infinity; NaN maps
    to the canonical quiet NaN 0x7FC0.
    """
    x = np.asarray(x, dtype=np.float64)
    _, e = np.frexp(x)
    q = np.ldexp(1.0, np.maximum(e, -125) - 8)
    r = np.rint(x / q) * q
    with np.errstate(over="ignore"):
        f = r.astype(np.float32)          # exact for every finite bf16 value
    bits = (f.view(np.uint32) >> np.uint32(16)).astype(np.uint16)
    bits = np.where(np.isnan(x), np.uint16(0x7FC0), bits)
    return bits


def round_to_dtype(x: np.ndarray, dtype: str) -> np.ndarray:
    """float64 -> storage of `dtype` ("f32": float32 RNE; "bf16": bit patterns)."""
    if dtype == "f32":
        return np.asarray(x, dtype=np.float64).astype(np.float32)
    if dtype == "bf16":
        return f64_to_bf16_bits(x)
    raise ValueError(dtype)


# ----------------------------------------------------------------------------
# Gram matrices
# ----------------------------------------------------------------------------


def gram(x: np.ndarray, offsets: np.ndarray) -> np.ndarray:
    """Per-bucket Gram matrices G_b[i, j] = <x_i[o_b:o_{b+1}], x_j[o_b:o_{b+1}]>.

    The bucket-level problems only see the local gradients through these inner
    products: the MGDA objective of Eq. (shard-mgda) is
    ||sum_t a_t g_t||^2 = a^T G a, the CAGrad objective of Section 3.2 and
    PCGrad's conflict test and projection (Eq. pcgrad_proj, Algorithm 1) use
    <g_i, g_j> only.  x: [K, N] float64.  Returns [B, K, K] float64.
    """
    x = np.asarray(x, dtype=np.float64)
    offsets = np.asarray(offsets, dtype=np.int64)
    nb = len(offsets) - 1
    k = x.shape[0]
    out = np.empty((nb, k, k))
    for b in range(nb):
        xb = x[:, offsets[b]:offsets[b + 1]]
        out[b] = xb @ xb.T
    return out


def slice_offsets(offsets: np.ndarray, T: int) -> np.ndarray:
    """Cut every bucket into T contiguous slices, the pieces T ranks would
    each hold after exchanging bucket slices: slice t of bucket b is
    [o_b + floor(t n_b / T), o_b + floor((t + 1) n_b / T)), n_b = o_{b+1} - o_b.
    Returns the B*T+1 offsets of the slices, bucket-major (bucket b's
    slices 0..T-1 are consecutive)."""
    offsets = np.asarray(offsets, dtype=np.int64)
    nb = len(offsets) - 1
    out = np.empty(nb * T + 1, dtype=np.int64)
    for b in range(nb):
        n = int(offsets[b + 1] - offsets[b])
        for t in range(T):
            out[b * T + t] = int(offsets[b]) + (t * n) // T
    out[nb * T] = offsets[nb]
    return out


def gram_reduce(partials: np.ndarray) -> np.ndarray:
    """Sum per-slice partial Gram matrices partials[t, b] over the slices in
    order t = 0, 1, ..., T-1: inner products add over disjoint pieces of a
    bucket, as over the buckets of the whole vector (Eq. decomp), so the sum
    is the bucket's Gram matrix.  partials: [T, B, K, K].  Returns [B, K, K]."""
    partials = np.asarray(partials, dtype=np.float64)
    acc = partials[0].copy()
    for t in range(1, partials.shape[0]):
        acc = acc + partials[t]
    return acc


# ----------------------------------------------------------------------------
# MGDA (Eq. mgda; Eq. shard-mgda over the simplex, Appendix B)
# ----------------------------------------------------------------------------


def pair_min_norm(aa: float, ab: float, bb: float):
    """Minimise ||gamma a + (1 - gamma) b||^2 over gamma in [0, 1].

    The quadratic gamma^2 aa + 2 gamma (1-gamma) ab + (1-gamma)^2 bb has its
    stationary point at gamma = (bb - ab) / (aa - 2 ab + bb); clip to [0, 1].
    When a = b (denominator <= 0) every gamma is optimal: take gamma = 1.
    Returns (gamma, squared norm at gamma).
    """
    den = aa - 2.0 * ab + bb
    if den <= 0.0:
        gamma = 1.0
    else:
        gamma = min(max((bb - ab) / den, 0.0), 1.0)
    val = gamma * gamma * aa + 2.0 * gamma * (1.0 - gamma) * ab + (1.0 - gamma) ** 2 * bb
    return gamma, val


def mgda_fw(G: np.ndarray, max_iter: int) -> np.ndarray:
    """Frank-Wolfe on the bucket MGDA problem min_{a in simplex} a^T G a.

    The paper states the problem (Eq. mgda, Eq. shard-mgda with a >= 0 as in
    Appendix A's simplex) but not a solver; this is the min-norm Frank-Wolfe
    scheme of the MGDA literature it builds on:

    1. start on the best edge: for every pair i < j (lexicographic), solve the
       two-point problem on (g_i, g_j); keep the smallest norm, first pair on
       ties; a = gamma e_i + (1 - gamma) e_j;
    2. repeat max_iter times (no early exit): t* = argmin_t (G a)_t (lowest
       index on ties); line search between the current point v = sum a_t g_t
       (|v|^2 = a^T G a, <v, g_t*> = (G a)_t*) and g_t*; a <- gamma a +
       (1 - gamma) e_t*.

    For K = 2 step 1 is the exact minimiser.  Returns a, shape [K].
    """
    G = np.asarray(G, dtype=np.float64)
    k = G.shape[0]
    best = None
    for i in range(k):
        for j in range(i + 1, k):
            gamma, val = pair_min_norm(G[i, i], G[i, j], G[j, j])
            if best is None or val < best[0]:
                best = (val, i, j, gamma)
    _, i, j, gamma = best
    a = np.zeros(k)
    a[i] = gamma
    a[j] = 1.0 - gamma
    for _ in range(max_iter):
        ga = G @ a
        t = int(np.argmin(ga))
        gamma, _ = pair_min_norm(float(a @ ga), float(ga[t]), float(G[t, t]))
        a = gamma * a
        a[t] += 1.0 - gamma
    return a


def mgda_exact(G: np.ndarray, tol: float = 1e-12) -> np.ndarray:
    """Exact minimiser of a^T G a over the simplex (the plain definition of
    Eq. mgda), by enumerating supports S and solving the KKT system
    G_SS a_S = mu 1, 1^T a_S = 1; keep a_S >= 0 with (G a)_t >= a^T G a for
    every t (the min-norm property of Eq. local_prop, Appendix B); return the
    feasible candidate of least a^T G a.  Cost 2^K small solves (K <= 12)."""
    G = np.asarray(G, dtype=np.float64)
    k = G.shape[0]
    scale = max(float(np.max(np.diag(G))), 1e-300)
    Gn = G / scale
    best = None
    for size in range(1, k + 1):
        for S in itertools.combinations(range(k), size):
            S = list(S)
            m = np.zeros((size + 1, size + 1))
            m[:size, :size] = Gn[np.ix_(S, S)]
            m[:size, size] = 1.0
            m[size, :size] = 1.0
            rhs = np.zeros(size + 1)
            rhs[size] = 1.0
            sol, *_ = np.linalg.lstsq(m, rhs, rcond=None)
            a = np.zeros(k)
            a[S] = sol[:size]
            if a.min() < -1e-10 or abs(a.sum() - 1.0) > 1e-9:
                continue
            a = np.maximum(a, 0.0)
            a /= a.sum()
            ga = Gn @ a
            q = float(a @ ga)
            if ga.min() < q - 1e-9:
                continue
            if best is None or q < best[0] - tol:
                best = (q, a)
    if best is None:  # numerically degenerate: fall back to a long FW run
        return mgda_fw(G, 5000)
    return best[1]


# ----------------------------------------------------------------------------
# PCGrad (Eq. pcgrad_proj; Algorithm 1, the PCGrad branch)
# ----------------------------------------------------------------------------


def pcgrad(G: np.ndarray, order: Optional[np.ndarray] = None) -> np.ndarray:
    """Bucket-level PCGrad in the coefficient basis of the original gradients.

    Algorithm 1 starts from d_t = g_t for every task t, visits the other tasks
    j != t in a (random) order, and whenever <d_t, g_j> < 0 replaces d_t by
    d_t - <d_t, g_j> / ||g_j||^2 g_j (Eq. pcgrad_proj); the bucket update is
    d = sum_t d_t.  Writing d_t = sum_i C[t, i] g_i turns every step into an
    exact operation on C that needs only G: <d_t, g_j> = sum_i C[t, i] G[i, j]
    and the projection subtracts <d_t, g_j>/G[j, j] from C[t, j].  The test
    is strict (< 0), and if G[j, j] = 0 then <d_t, g_j> = 0 so nothing is
    divided.  `order[t]` lists the other tasks in visiting order (None:
    ascending).  Returns the combine weights w = sum_t C[t, :], shape [K].
    """
    G = np.asarray(G, dtype=np.float64)
    k = G.shape[0]
    C = np.eye(k)
    for t in range(k):
        visit = [j for j in range(k) if j != t] if order is None else [int(j) for j in order[t]]
        for j in visit:
            p = float(C[t] @ G[:, j])
            if p < 0.0:
                C[t, j] -= p / G[j, j]
    return C.sum(axis=0)


# ----------------------------------------------------------------------------
# CAGrad (Eq. cagrad; the bucket-level problem of Section 3.2, Appendix C)
# ----------------------------------------------------------------------------


def _cagrad_terms(G: np.ndarray, c: float):
    k = G.shape[0]
    b = G.sum(axis=1) / k                  # b_t = <g_t, g_avg>
    g0sq = max(float(G.sum()) / (k * k), 0.0)
    r = c * math.sqrt(g0sq)                # trust-region radius c ||g_avg||
    return b, r


def _cagrad_weights(G: np.ndarray, w: np.ndarray, r: float) -> np.ndarray:
    """Primal direction d = g_avg + r g_w / ||g_w|| in the basis of the g_t:
    weights 1/K + (r / ||g_w||) w_t; if r = 0 or g_w vanishes (relative to
    the largest gradient) d = g_avg, weights 1/K."""
    k = G.shape[0]
    nrm = math.sqrt(max(float(w @ G @ w), 0.0))
    scale = math.sqrt(max(float(np.max(np.diag(G))), 0.0))
    if r == 0.0 or nrm <= 1e-12 * scale or nrm == 0.0:
        return np.full(k, 1.0 / k)
    return 1.0 / k + (r / nrm) * w


def cagrad_fw(G: np.ndarray, c: float, max_iter: int):
    """Bucket CAGrad through its dual, solved by Frank-Wolfe.

    For the problem max_d min_t <g_t, d> s.t. ||d - g_avg|| <= c ||g_avg||
    (Eq. cagrad per bucket), min_t <g_t, d> = min_{w in simplex} <g_w, d>
    with g_w = sum w_t g_t, and swapping max and min (convex-concave, compact)
    leaves min_{w in simplex} F(w), F(w) = b^T w + r sqrt(w^T G w), with
    b = G 1 / K and r = c ||g_avg||; the maximiser for the optimal w is
    d = g_avg + r g_w / ||g_w||.

    Frank-Wolfe from w = 1/K, max_iter iterations, no early exit:
    grad F = b + r G w / ||g_w|| (second term 0 when ||g_w|| <= 1e-300);
    s = argmin grad F (lowest index on ties); exact line search over
    w(gamma) = (1 - gamma) w + gamma e_s, where
    F(gamma) = b^T w + beta1 gamma + r sqrt(A gamma^2 + 2 Bq gamma + Cq),
    beta1 = b_s - b^T w, A = G_ss - 2 (G w)_s + Cq, Bq = (G w)_s - Cq,
    Cq = w^T G w.  Setting F'(gamma) = 0 and squaring gives
    gamma = (-Bq +- |beta1| sqrt((A Cq - Bq^2) / D)) / A with D = r^2 A - beta1^2
    (real when A > 0 and D > 0).  Candidates: 0, 1 and those roots inside
    (0, 1); the one of least F wins, the smaller gamma on ties.

    Returns (combine weights [K], dual simplex variable w [K]).
    """
    G = np.asarray(G, dtype=np.float64)
    k = G.shape[0]
    b, r = _cagrad_terms(G, c)
    w = np.full(k, 1.0 / k)
    for _ in range(max_iter):
        gw = G @ w
        cq = float(w @ gw)
        nrm = math.sqrt(max(cq, 0.0))
        grad = b + (r * gw / nrm if nrm > 1e-300 else 0.0)
        s = int(np.argmin(grad))
        bw = float(b @ w)
        beta1 = float(b[s]) - bw
        A = float(G[s, s]) - 2.0 * float(gw[s]) + cq
        Bq = float(gw[s]) - cq
        cands = [0.0, 1.0]
        D = r * r * A - beta1 * beta1
        if A > 0.0 and D > 0.0:
            disc = (A * cq - Bq * Bq) / D
            if disc >= 0.0:
                root = abs(beta1) * math.sqrt(disc)
                for g in ((-Bq - root) / A, (-Bq + root) / A):
                    if 0.0 < g < 1.0:
                        cands.append(g)
        cands.sort()

        def f(g):
            return bw + beta1 * g + r * math.sqrt(max(A * g * g + 2.0 * Bq * g + cq, 0.0))

        vals = [f(g) for g in cands]
        gamma = cands[int(np.argmin(vals))]
        w = (1.0 - gamma) * w
        w[s] += gamma
    return _cagrad_weights(G, w, r), w


def cagrad_exact(G: np.ndarray, c: float):
    """Exact minimiser of the CAGrad dual F(w) = b^T w + r ||g_w|| over the
    simplex, by support enumeration.  On a support S the stationarity
    condition b_S + r G_SS v_S = lam 1 with v = w / ||g_w|| (so v^T G v = 1)
    gives v_S = G_SS^{-1} (lam 1 - b_S) / r, and v_S^T G_SS v_S = 1 is a
    quadratic in lam.  Candidates with v >= 0 are normalised to the simplex;
    together with every vertex they are scored by F and the least wins.
    Returns (combine weights [K], w [K])."""
    G = np.asarray(G, dtype=np.float64)
    k = G.shape[0]
    b, r = _cagrad_terms(G, c)

    def F(w):
        return float(b @ w) + r * math.sqrt(max(float(w @ G @ w), 0.0))

    cands = [np.eye(k)[i] for i in range(k)]
    if r > 0.0:
        for size in range(2, k + 1):
            for S in itertools.combinations(range(k), size):
                S = list(S)
                Gs = G[np.ix_(S, S)]
                try:
                    H = np.linalg.inv(Gs)
                except np.linalg.LinAlgError:
                    continue
                one = np.ones(size)
                bs = b[S]
                qa = float(one @ H @ one)
                qb = -2.0 * float(one @ H @ bs)
                qc = float(bs @ H @ bs) - r * r
                disc = qb * qb - 4.0 * qa * qc
                if qa <= 0.0 or disc < 0.0:
                    continue
                for lam in ((-qb - math.sqrt(disc)) / (2 * qa), (-qb + math.sqrt(disc)) / (2 * qa)):
                    v = H @ (lam * one - bs) / r
                    if v.min() < -1e-12 or v.sum() <= 0.0:
                        continue
                    w = np.zeros(k)
                    w[S] = np.maximum(v, 0.0)
                    w /= w.sum()
                    cands.append(w)
    vals = [F(w) for w in cands]
    w = cands[int(np.argmin(vals))]
    return _cagrad_weights(G, w, r), w


# ----------------------------------------------------------------------------
# Conflict diagnostics (the conflicting-gradients definition of Section 2.1
# and its appendix restatement; the statistics of Figure 1)
# ----------------------------------------------------------------------------


def conflicts(grams: np.ndarray):
    """Per-bucket gradient-conflict statistics from the Gram matrices.

    Two task gradients conflict when their inner product is negative
    (equivalently, their cosine similarity is negative).  Figure 1 tracks the
    mean and standard deviation of the pairwise cosine similarities over all
    task pairs, and counts a conflict at a step when at least one pair has a
    negative cosine.  Per bucket b, over the pairs i < j in lexicographic
    order:

      cos[b, i, j] = G_ij / sqrt(G_ii G_jj), clipped to [-1, 1]; 0 when either
                     gradient is zero (no direction, so no conflict); the
                     diagonal is 1 for a nonzero gradient and 0 otherwise
      summary[b]   = (mean, population standard deviation, minimum) of the
                     K(K-1)/2 pairwise cosines
      pairs[b]     = (i, j) of the smallest cosine (first pair on ties) and the
                     number of pairs with G_ij < 0; a count > 0 is Figure 1's
                     per-step conflict event

    A bucket whose Gram holds a NaN or infinity gets NaN cosines and summary
    and pairs (-1, -1, -1).  Returns (cos [B, K, K], summary [B, 3] float64,
    pairs [B, 3] int64).
    """
    grams = np.asarray(grams, dtype=np.float64)
    nb, k, _ = grams.shape
    cos = np.zeros((nb, k, k))
    summary = np.empty((nb, 3))
    pairs = np.empty((nb, 3), dtype=np.int64)
    for b in range(nb):
        G = grams[b]
        if not np.all(np.isfinite(G)):
            cos[b] = np.nan
            summary[b] = np.nan
            pairs[b] = -1
            continue
        vals = []
        count = 0
        best = None
        for i in range(k):
            cos[b, i, i] = 1.0 if G[i, i] > 0.0 else 0.0
            for j in range(i + 1, k):
                if G[i, i] > 0.0 and G[j, j] > 0.0:
                    c = G[i, j] / math.sqrt(G[i, i] * G[j, j])
                    c = min(max(c, -1.0), 1.0)
                else:
                    c = 0.0
                cos[b, i, j] = cos[b, j, i] = c
                vals.append(c)
                if G[i, j] < 0.0:
                    count += 1
                if best is None or c < best[0]:
                    best = (c, i, j)
        v = np.array(vals)
        summary[b] = (v.mean(), v.std(), best[0])
        pairs[b] = (best[1], best[2], count)
    return cos, summary, pairs


# ----------------------------------------------------------------------------
# per-bucket solve, combine and the whole resolve step (Algorithm 1)
# ----------------------------------------------------------------------------


def solve(grams: np.ndarray, method: str, max_iter: int = 20, cagrad_c: float = 0.5,
          orders: Optional[np.ndarray] = None, exact: bool = False):
    """Per-bucket combine weights and auxiliary variables.

    method: "mgda" (weights = aux = simplex a, d = sum a_t g_t, Algorithm 1's
    MGDA branch), "pcgrad" (weights = column sums of C, aux = weights),
    "cagrad" (weights = 1/K + r w / ||g_w||, aux = dual w), "mean" (the
    averaged gradient of Section 2.1, weights = aux = 1/K).
    The paper says nothing about non-finite gradients; the reading here is
    that a bucket whose Gram matrix holds a NaN or infinity gets NaN weights
    (and so a NaN update) rather than a silently filtered one.
    Returns (weights [B, K], aux [B, K]) float64.
    """
    grams = np.asarray(grams, dtype=np.float64)
    nb, k, _ = grams.shape
    W = np.empty((nb, k))
    A = np.empty((nb, k))
    for i in range(nb):
        G = grams[i]
        if not np.all(np.isfinite(G)):
            W[i] = np.nan
            A[i] = np.nan
            continue
        if method == "mgda":
            a = mgda_exact(G) if exact else mgda_fw(G, max_iter)
            W[i] = a
            A[i] = a
        elif method == "pcgrad":
            W[i] = pcgrad(G, None if orders is None else orders[i])
            A[i] = W[i]
        elif method == "cagrad":
            W[i], A[i] = cagrad_exact(G, cagrad_c) if exact else cagrad_fw(G, cagrad_c, max_iter)
        elif method == "mean":
            W[i] = 1.0 / k
            A[i] = W[i]
        else:
            raise ValueError(method)
    return W, A


def combine(x: np.ndarray, offsets: np.ndarray, W: np.ndarray) -> np.ndarray:
    """d[o_b:o_{b+1}] = sum_i W[b, i] x_i[o_b:o_{b+1}] in float64: the bucket
    updates of Algorithm 1, concatenated into d = [d_(1), ..., d_(B)]."""
    x = np.asarray(x, dtype=np.float64)
    offsets = np.asarray(offsets, dtype=np.int64)
    W = np.asarray(W, dtype=np.float64)
    out = np.empty(x.shape[1])
    for b in range(len(offsets) - 1):
        lo, hi = offsets[b], offsets[b + 1]
        out[lo:hi] = W[b] @ x[:, lo:hi]
    return out


def resolve(rows: np.ndarray, offsets: np.ndarray, method: str, max_iter: int = 20,
            cagrad_c: float = 0.5, orders: Optional[np.ndarray] = None,
            out_dtype: Optional[str] = None, exact: bool = False) -> dict:
    """The bucket-level resolve step end to end: Gram, per-bucket solve and
    combine, with the update rounded once to the output dtype (default: the
    input's storage dtype).  rows: [K, N] float32 or bf16 bit patterns."""
    rows = np.asarray(rows)
    if out_dtype is None:
        out_dtype = "bf16" if rows.dtype == np.uint16 else "f32"
    x = decode_rows(rows)
    G = gram(x, offsets)
    W, A = solve(G, method, max_iter, cagrad_c, orders, exact)
    d = combine(x, offsets, W)
    return {"gram": G, "weights": W, "aux": A, "out_f64": d, "out": round_to_dtype(d, out_dtype)}
