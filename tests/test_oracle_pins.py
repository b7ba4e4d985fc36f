"""Pins for the float64 oracle: closed forms, brute force, invariants and
library routines that fix what each oracle function must return.

None of these compares the oracle with itself or retypes its formulas: the
expected values come from vector-space computations on the gradients
themselves (not their Gram matrices), from exhaustive search, from
hand-derived examples, or from numpy/torch/math routines.
"""

import itertools
import json
import math
import os

import numpy as np
import pytest

import oracle

GOLD = os.path.join(os.path.dirname(__file__), "golden", "hand_examples.json")


def rand_grads(rng, k, n, corr=None, scales=None):
    z = rng.standard_normal((k, n))
    if corr is not None:
        z = np.linalg.cholesky(corr) @ z
    if scales is not None:
        z = z * np.asarray(scales)[:, None]
    return z.astype(np.float32).astype(np.float64)


def rand_corr(rng, k, lo, hi):
    c = np.eye(k)
    for i in range(k):
        for j in range(i + 1, k):
            c[i, j] = c[j, i] = rng.uniform(lo, hi)
    ev, v = np.linalg.eigh(c)
    if ev.min() < 1e-2:
        c = (v * np.maximum(ev, 1e-2)) @ v.T
        s = 1 / np.sqrt(np.diag(c))
        c = c * s[:, None] * s[None, :]
    return c


# ----------------------------------------------------------------------------
# storage formats
# ----------------------------------------------------------------------------


def test_bf16_decode_known_patterns():
    bits = np.array([0x3F80, 0xC000, 0x0001, 0x7F7F, 0x0080, 0x8000, 0x7F80], dtype=np.uint16)
    want = [1.0, -2.0, 2.0 ** -133, (2 - 2 ** -7) * 2.0 ** 127, 2.0 ** -126, -0.0, math.inf]
    got = oracle.bf16_bits_to_f64(bits)
    assert list(got) == want
    assert math.copysign(1.0, got[5]) == -1.0


def test_bf16_rounding_matches_torch_rne_on_fp32_values():
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(0)
    f = np.concatenate([
        rng.standard_normal(20000).astype(np.float32) * np.float32(3.0),
        (rng.standard_normal(2000) * 1e-39).astype(np.float32),      # fp32/bf16 subnormals
        np.array([3.3895314e38, 3.4e38, -3.4e38, 1e-45, 0.0, -0.0], dtype=np.float32),
    ])
    # exact ties: bf16 value + half an ulp, both parities of the kept bit
    base = (rng.integers(0, 0x7F00, 4000).astype(np.uint32) << 16)
    ties = (base | 0x8000).view(np.float32)
    f = np.concatenate([f, ties, -ties])
    want = torch.from_numpy(f).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    got = oracle.f64_to_bf16_bits(f.astype(np.float64))
    assert np.array_equal(got, want)


def test_bf16_rounding_is_single_rounding_from_f64():
    # 1 + 2^-8 is the exact midpoint between bf16 neighbours 1 and 1 + 2^-7:
    # ties-to-even gives 1.  A hair above it must round up; going through
    # fp32 first would erase the hair (1 + 2^-8 + 2^-40 -> fp32 1 + 2^-8)
    # and then round to even, i.e. down.
    assert oracle.f64_to_bf16_bits(np.array([1 + 2.0 ** -8]))[0] == 0x3F80
    assert oracle.f64_to_bf16_bits(np.array([1 + 2.0 ** -8 + 2.0 ** -40]))[0] == 0x3F81
    assert oracle.f64_to_bf16_bits(np.array([1 + 3 * 2.0 ** -8]))[0] == 0x3F82   # tie -> even up
    assert oracle.f64_to_bf16_bits(np.array([-(1 + 2.0 ** -8 + 2.0 ** -40)]))[0] == 0xBF81
    assert oracle.f64_to_bf16_bits(np.array([3.4e38]))[0] == 0x7F80               # overflow
    assert oracle.f64_to_bf16_bits(np.array([np.nan]))[0] == 0x7FC0
    assert oracle.f64_to_bf16_bits(np.array([2.0 ** -134 + 2.0 ** -160]))[0] == 0x0001


# ----------------------------------------------------------------------------
# Gram
# ----------------------------------------------------------------------------


def test_gram_matches_fsum_on_ragged_buckets():
    rng = np.random.default_rng(1)
    k = 5
    lens = [1, 7, 64, 3, 130, 2]
    x = rand_grads(rng, k, sum(lens))
    offs = np.concatenate([[0], np.cumsum(lens)])
    G = oracle.gram(x, offs)
    assert G.shape == (len(lens), k, k)
    for b in range(len(lens)):
        for i in range(k):
            for j in range(k):
                ref = math.fsum(x[i, n] * x[j, n] for n in range(offs[b], offs[b + 1]))
                assert abs(G[b, i, j] - ref) <= 1e-14 * max(1.0, abs(ref))


def test_gram_symmetric_psd_and_additive_over_splits():
    rng = np.random.default_rng(2)
    k, n = 6, 5000
    x = rand_grads(rng, k, n)
    G = oracle.gram(x, np.array([0, n]))[0]
    assert np.array_equal(G, G.T) or np.allclose(G, G.T, rtol=0, atol=1e-12 * np.abs(G).max())
    assert np.linalg.eigvalsh(G).min() > -1e-10 * np.abs(G).max()
    np.testing.assert_allclose(np.diag(G), [math.fsum(v * v for v in x[i]) for i in range(k)], rtol=1e-14)
    # inner products decompose additively over disjoint blocks (Eq. decomp)
    cuts = np.array([0, 17, 1000, 1001, 4096, n])
    parts = oracle.gram(x, cuts)
    np.testing.assert_allclose(parts.sum(0), G, rtol=1e-12, atol=1e-12 * np.abs(G).max())


def test_single_element_bucket_is_outer_product():
    x = np.array([[2.0], [-3.0], [0.5]])
    G = oracle.gram(x, np.array([0, 1]))[0]
    assert np.array_equal(G, np.outer(x[:, 0], x[:, 0]))


# ----------------------------------------------------------------------------
# MGDA
# ----------------------------------------------------------------------------


def _closed_form_k2(g1, g2):
    """Two-task min-norm weight on g1 from the vectors: clip(((g2-g1).g2)/|g1-g2|^2, 0, 1)."""
    diff = g1 - g2
    den = float(np.dot(diff, diff))
    if den == 0.0:
        return None
    return min(max(float(np.dot(g2 - g1, g2)) / den, 0.0), 1.0)


@pytest.mark.parametrize("seed", range(40))
def test_mgda_k2_closed_form(seed):
    rng = np.random.default_rng(100 + seed)
    n = 257
    rho = rng.uniform(-0.95, 0.95)
    scales = np.exp(rng.uniform(np.log(0.1), np.log(10.0), size=2))
    x = rand_grads(rng, 2, n, corr=np.array([[1, rho], [rho, 1]]), scales=scales)
    G = oracle.gram(x, np.array([0, n]))[0]
    want = _closed_form_k2(x[0], x[1])
    for iters in (0, 1, 20):
        a = oracle.mgda_fw(G, iters)
        assert abs(a[0] - want) <= 1e-10 and abs(a.sum() - 1) <= 1e-14 and a.min() >= 0


def test_mgda_k2_clip_branches_reached():
    rng = np.random.default_rng(7)
    hit = set()
    for _ in range(200):
        s = np.exp(rng.uniform(np.log(0.1), np.log(10.0), size=2))
        x = rand_grads(rng, 2, 33, scales=s)
        a = oracle.mgda_fw(oracle.gram(x, np.array([0, 33]))[0], 20)[0]
        hit.add("lo" if a == 0.0 else "hi" if a == 1.0 else "mid")
    assert hit == {"lo", "hi", "mid"}


def test_golden_hand_examples():
    cases = json.load(open(GOLD))["cases"]
    for c in cases:
        g = np.array(c["g"], dtype=np.float64)       # rows are task gradients
        G = g @ g.T
        if c["name"].startswith("mgda"):
            for a in (oracle.mgda_fw(G, 20), oracle.mgda_exact(G)):
                np.testing.assert_allclose(a, c["alpha"], atol=1e-12)
                np.testing.assert_allclose(a @ g, c["d"], atol=1e-12)
        elif c["name"].startswith("pcgrad"):
            w = oracle.pcgrad(G, np.array(c["order"]) if "order" in c else None)
            np.testing.assert_allclose(w, c["weights"], atol=1e-12)
            np.testing.assert_allclose(w @ g, c["d"], atol=1e-12)
        elif c["name"].startswith("cagrad"):
            runs = [oracle.cagrad_fw(G, c["c"], c.get("iters", 20))]
            if c.get("iters", 20) == 20:
                runs.append(oracle.cagrad_exact(G, c["c"]))    # the cases at 20 steps are optima
            for wts, w in runs:
                np.testing.assert_allclose(wts, c["weights"], atol=1e-9)
                np.testing.assert_allclose(wts @ g, c["d"], atol=1e-9)
                if "w" in c:
                    np.testing.assert_allclose(w, c["w"], atol=1e-12)


def _simplex_grid(k, step):
    m = int(round(1 / step))
    for idx in itertools.product(range(m + 1), repeat=k - 1):
        if sum(idx) <= m:
            yield np.array(list(idx) + [m - sum(idx)], dtype=np.float64) / m


@pytest.mark.parametrize("k,step", [(2, 1e-3), (3, 4e-3)])
@pytest.mark.parametrize("seed", range(6))
def test_mgda_exact_beats_simplex_grid(k, step, seed):
    rng = np.random.default_rng(200 + seed)
    n = 40
    x = rand_grads(rng, k, n, corr=rand_corr(rng, k, -0.8, 0.8),
                   scales=np.exp(rng.uniform(-1, 1, size=k)))
    G = oracle.gram(x, np.array([0, n]))[0]
    a = oracle.mgda_exact(G)
    best = min(float(np.sum((w @ x) ** 2)) for w in _simplex_grid(k, step))   # |sum w g|^2 from vectors
    val = float(np.sum((a @ x) ** 2))
    assert val <= best + 1e-9 * best
    # grid resolution bound: the optimum is within one grid cell of a grid point
    assert val >= best - 4 * step * float(np.abs(G).max())


@pytest.mark.parametrize("k", [2, 3, 4, 6, 8, 10])
def test_mgda_exact_kkt_and_fw_convergence(k):
    rng = np.random.default_rng(300 + k)
    for trial in range(5):
        n = 64
        x = rand_grads(rng, k, n, corr=rand_corr(rng, k, -0.6, 0.8))
        G = oracle.gram(x, np.array([0, n]))[0]
        a = oracle.mgda_exact(G)
        d = a @ x
        dn = float(d @ d)
        scale = float(np.max(np.diag(G)))
        # Eq. local_prop: <g_t, d> >= |d|^2 for every task t (normalised by max |g_t|^2)
        assert (x @ d).min() / scale >= dn / scale - 1e-9
        assert a.min() >= 0 and abs(a.sum() - 1) <= 1e-12
        # FW objective is non-increasing and approaches the exact optimum
        prev = math.inf
        for it in (0, 1, 2, 5, 20, 100):
            af = oracle.mgda_fw(G, it)
            assert af.min() >= 0 and abs(af.sum() - 1) <= 1e-12
            v = float(af @ G @ af)
            assert v <= prev + 1e-12 * scale
            prev = v
        assert oracle.mgda_fw(G, 4000) @ G @ oracle.mgda_fw(G, 4000) <= dn + 2e-4 * scale


def test_mgda_concatenation_is_common_descent():
    # Eq. global_bound: with exact per-bucket solutions, <g_t, d> >= |d|^2 globally
    rng = np.random.default_rng(11)
    k, lens = 4, [50, 80, 13, 200]
    offs = np.concatenate([[0], np.cumsum(lens)])
    x = rand_grads(rng, k, offs[-1], corr=rand_corr(rng, k, -0.7, 0.7))
    r = oracle.resolve(x.astype(np.float32), offs, "mgda", exact=True)
    d = r["out_f64"]
    assert (x @ d).min() >= float(d @ d) * (1 - 1e-9)


def test_mgda_stationary_bucket_gives_zero():
    # Appendix B case (a): 0 in the hull of a bucket's gradients => d_(k) = 0
    g = np.array([[1.0, 2.0, -1.0], [0.5, -1.0, 3.0], [-1.5, -1.0, -2.0]])   # rows sum to 0
    G = g @ g.T
    for a in (oracle.mgda_exact(G), oracle.mgda_fw(G, 200)):
        assert np.linalg.norm(a @ g) <= 1e-3 * np.abs(g).max()


# ----------------------------------------------------------------------------
# PCGrad
# ----------------------------------------------------------------------------


def vector_pcgrad(x, order):
    """Algorithm 1's PCGrad branch on the actual vectors."""
    k = x.shape[0]
    d = x.copy()
    for t in range(k):
        for j in order[t]:
            p = float(d[t] @ x[j])
            if p < 0:
                d[t] = d[t] - p / float(x[j] @ x[j]) * x[j]
    return d.sum(0), d


@pytest.mark.parametrize("k", [2, 3, 4, 6, 10])
def test_pcgrad_coefficients_equal_vector_projection(k):
    rng = np.random.default_rng(400 + k)
    for trial in range(10):
        n = 31
        x = rand_grads(rng, k, n, corr=rand_corr(rng, k, -0.8, 0.5),
                       scales=np.exp(rng.uniform(-2, 2, size=k)))
        order = np.array([rng.permutation([j for j in range(k) if j != t]) for t in range(k)])
        G = oracle.gram(x, np.array([0, n]))[0]
        w = oracle.pcgrad(G, order)
        d_ref, d_tasks = vector_pcgrad(x, order)
        np.testing.assert_allclose(w @ x, d_ref, rtol=1e-10, atol=1e-10 * np.abs(d_ref).max())


def test_pcgrad_no_conflict_means_plain_sum():
    rng = np.random.default_rng(5)
    x = np.abs(rand_grads(rng, 5, 40))            # all pairwise inner products > 0
    G = oracle.gram(x, np.array([0, 40]))[0]
    assert np.array_equal(oracle.pcgrad(G), np.ones(5))


def test_pcgrad_k2_closed_form_and_orthogonality():
    rng = np.random.default_rng(6)
    for _ in range(50):
        x = rand_grads(rng, 2, 20, corr=np.array([[1, -0.6], [-0.6, 1]]))
        g12 = float(x[0] @ x[1])
        assert g12 < 0
        w = oracle.pcgrad(oracle.gram(x, np.array([0, 20]))[0])
        np.testing.assert_allclose(w, [1 - g12 / float(x[0] @ x[0]), 1 - g12 / float(x[1] @ x[1])], rtol=1e-12)
        # each projected task gradient is orthogonal to the one it was projected off
        _, d = vector_pcgrad(x, [[1], [0]])
        assert abs(float(d[0] @ x[1])) <= 1e-12 * float(x[1] @ x[1]) * 10


# ----------------------------------------------------------------------------
# CAGrad
# ----------------------------------------------------------------------------


def _cagrad_primal(x, c):
    g0 = x.mean(0)
    return g0, c * float(np.linalg.norm(g0))


@pytest.mark.parametrize("k", [2, 3, 4, 8, 10])
@pytest.mark.parametrize("c", [0.0, 0.25, 0.5, 0.9])
def test_cagrad_exact_primal_dual(k, c):
    rng = np.random.default_rng(500 + k + int(100 * c))
    for trial in range(4):
        n = 48
        x = rand_grads(rng, k, n, corr=rand_corr(rng, k, -0.7, 0.7),
                       scales=np.exp(rng.uniform(-1, 1, size=k)))
        G = oracle.gram(x, np.array([0, n]))[0]
        wts, w = oracle.cagrad_exact(G, c)
        d = wts @ x
        g0, r = _cagrad_primal(x, c)
        gn2 = float(g0 @ g0)
        # trust region (Eq. cagrad), tight when the dual point is not degenerate
        assert np.linalg.norm(d - g0) <= r * (1 + 1e-9) + 1e-12
        # Theorem 3.2 (a): <g_avg, d> >= (1 - c^2)/2 |g_avg|^2
        assert float(g0 @ d) >= (1 - c * c) / 2 * gn2 * (1 - 1e-9)
        # zero duality gap: worst inner product at d equals the dual value
        gw = w @ x
        dual = float(gw @ g0) + r * float(np.linalg.norm(gw))
        primal = float((x @ d).min())
        assert abs(primal - dual) <= 1e-8 * max(1.0, abs(dual), gn2)
        # no feasible direction does better (random search on the sphere of radius r)
        u = rng.standard_normal((4000, n))
        u *= r / np.linalg.norm(u, axis=1, keepdims=True)
        trial_vals = ((g0 + u) @ x.T).min(1)
        assert trial_vals.max() <= primal + 1e-9 * max(1.0, gn2)
        if c == 0.0:
            np.testing.assert_allclose(wts, np.full(k, 1.0 / k), rtol=0, atol=0)


@pytest.mark.parametrize("k,step", [(2, 1e-3), (3, 4e-3)])
def test_cagrad_exact_beats_dual_grid(k, step):
    rng = np.random.default_rng(600 + k)
    for trial in range(4):
        n = 30
        x = rand_grads(rng, k, n, corr=rand_corr(rng, k, -0.8, 0.8),
                       scales=np.exp(rng.uniform(-1, 1, size=k)))
        g0, r = _cagrad_primal(x, 0.5)
        F = lambda w: float((w @ x) @ g0) + r * float(np.linalg.norm(w @ x))   # noqa: E731
        _, w = oracle.cagrad_exact(oracle.gram(x, np.array([0, n]))[0], 0.5)
        best = min(F(v) for v in _simplex_grid(k, step))
        assert F(w) <= best + 1e-12 * max(1.0, abs(best))


def test_cagrad_fw_k2_is_exact_and_fw_feasible():
    rng = np.random.default_rng(8)
    for k in (2, 3, 4, 8):
        for _ in range(20):
            n = 24
            x = rand_grads(rng, k, n, corr=rand_corr(rng, k, -0.8, 0.8),
                           scales=np.exp(rng.uniform(-1, 1, size=k)))
            G = oracle.gram(x, np.array([0, n]))[0]
            wts, w = oracle.cagrad_fw(G, 0.5, 20)
            assert w.min() >= 0 and abs(w.sum() - 1) <= 1e-12
            d = wts @ x
            g0, r = _cagrad_primal(x, 0.5)
            assert np.linalg.norm(d - g0) <= r * (1 + 1e-9) + 1e-12
            if k == 2:
                we, _ = oracle.cagrad_exact(G, 0.5)
                np.testing.assert_allclose(wts, we, rtol=1e-7, atol=1e-9)


def test_cagrad_zero_average_gives_zero_update():
    # Theorem 3.2 (b) direction: g_avg = 0 makes the ball a point, d = 0
    g = np.array([[1.0, -2.0, 0.5], [-1.0, 2.0, -0.5]])
    G = g @ g.T
    for wts, _ in (oracle.cagrad_fw(G, 0.5, 20), oracle.cagrad_exact(G, 0.5)):
        assert np.linalg.norm(wts @ g) <= 1e-12


# ----------------------------------------------------------------------------
# combine and resolve
# ----------------------------------------------------------------------------


def test_combine_uniform_weights_is_the_mean():
    rng = np.random.default_rng(9)
    x = rand_grads(rng, 6, 777)
    offs = np.array([0, 100, 101, 777])
    out = oracle.combine(x, offs, np.full((3, 6), 1 / 6))
    np.testing.assert_allclose(out, np.mean(x, axis=0), rtol=1e-14, atol=1e-16)


@pytest.mark.parametrize("dt", ["f32", "bf16"])
def test_combine_unit_weight_reproduces_a_task_bitwise(dt):
    rng = np.random.default_rng(10)
    x32 = rng.standard_normal((3, 500)).astype(np.float32)
    rows = x32 if dt == "f32" else oracle.f64_to_bf16_bits(x32.astype(np.float64))
    x = oracle.decode_rows(rows)
    offs = np.array([0, 123, 500])
    W = np.array([[0.0, 1.0, 0.0], [0.0, 0.0, 1.0]])
    r = oracle.round_to_dtype(oracle.combine(x, offs, W), dt)
    assert np.array_equal(r[:123], rows[1, :123]) and np.array_equal(r[123:], rows[2, 123:])


def test_combine_elementwise_brute_force():
    rng = np.random.default_rng(12)
    k, lens = 3, [5, 1, 9]
    offs = np.concatenate([[0], np.cumsum(lens)])
    x = rand_grads(rng, k, offs[-1])
    W = rng.standard_normal((3, k))
    out = oracle.combine(x, offs, W)
    for b in range(3):
        for n in range(offs[b], offs[b + 1]):
            assert abs(out[n] - math.fsum(W[b, i] * x[i, n] for i in range(k))) <= 1e-15 * 8


def test_resolve_is_bucketwise_concatenation():
    rng = np.random.default_rng(13)
    k, lens = 4, [64, 3, 100]
    offs = np.concatenate([[0], np.cumsum(lens)])
    rows = rand_grads(rng, k, offs[-1]).astype(np.float32)
    orders = np.array([[rng.permutation([j for j in range(k) if j != t]) for t in range(k)] for _ in lens])
    for m in ("mgda", "pcgrad", "cagrad", "mean"):
        whole = oracle.resolve(rows, offs, m, orders=orders)
        for b in range(3):
            part = oracle.resolve(rows[:, offs[b]:offs[b + 1]], np.array([0, lens[b]]), m,
                                  orders=orders[b:b + 1])
            assert np.array_equal(whole["out"][offs[b]:offs[b + 1]], part["out"])


# ----------------------------------------------------------------------------
# conflict diagnostics: cosines and counts from the vectors themselves
# ----------------------------------------------------------------------------


def _vector_conflicts(x, offs):
    """Cosines, (mean, population std, min), (argmin pair, count) computed
    from the gradient vectors with numpy norms and statistics routines."""
    import statistics
    k = x.shape[0]
    res = []
    for b in range(len(offs) - 1):
        xb = x[:, offs[b]:offs[b + 1]]
        cos, neg = {}, 0
        for i, j in itertools.combinations(range(k), 2):
            ni, nj = np.linalg.norm(xb[i]), np.linalg.norm(xb[j])
            d = math.fsum(xb[i] * xb[j])
            cos[(i, j)] = 0.0 if ni == 0 or nj == 0 else max(-1.0, min(1.0, d / (ni * nj)))
            neg += d < 0
        vals = list(cos.values())
        m = min(vals)
        first = next(pq for pq in itertools.combinations(range(k), 2) if cos[pq] == m)
        res.append((cos, statistics.fmean(vals), statistics.pstdev(vals), m, first, neg))
    return res


def check_conflicts(fn):
    rng = np.random.default_rng(21)
    lens = [40, 1, 17, 64]
    offs = np.concatenate([[0], np.cumsum(lens)])
    x = rand_grads(rng, 5, offs[-1], corr=rand_corr(rng, 5, -0.7, 0.7))
    x[3, offs[2]:offs[3]] = 0.0                 # a zero gradient in bucket 2
    grams = np.stack([x[:, offs[b]:offs[b + 1]] @ x[:, offs[b]:offs[b + 1]].T for b in range(4)])
    cos, summ, pairs = fn(grams)
    for b, (vc, mean, std, m, first, neg) in enumerate(_vector_conflicts(x, offs)):
        for (i, j), c in vc.items():
            assert abs(cos[b, i, j] - c) <= 1e-12 and abs(cos[b, j, i] - c) <= 1e-12
        norms = np.linalg.norm(x[:, offs[b]:offs[b + 1]], axis=1)
        assert np.array_equal(np.diag(cos[b]), (norms > 0).astype(float))
        assert abs(summ[b, 0] - mean) <= 1e-12 and abs(summ[b, 1] - std) <= 1e-12
        assert abs(summ[b, 2] - m) <= 1e-12
        assert tuple(pairs[b, :2]) == first and pairs[b, 2] == neg
    # exact ties (orthogonal unit vectors): the first pair wins, none conflicts
    e = np.eye(4)[:3]
    cos, summ, pairs = fn((e @ e.T)[None])
    assert tuple(pairs[0]) == (0, 1, 0) and summ[0, 0] == 0.0 and summ[0, 1] == 0.0


def test_conflicts_match_vector_cosines():
    check_conflicts(oracle.conflicts)
    check_slice_offsets(oracle.slice_offsets)
    check_gram_reduce(oracle.gram_reduce)


def test_conflicts_closed_forms():
    # e1, e2, e1+e2: cosines 0, 1/sqrt2, 1/sqrt2 -> mean sqrt2/3, std 1/3
    x = np.array([[1.0, 0.0], [0.0, 1.0], [1.0, 1.0]])
    _, summ, pairs = oracle.conflicts((x @ x.T)[None])
    assert abs(summ[0, 0] - math.sqrt(2) / 3) <= 1e-15 and abs(summ[0, 1] - 1 / 3) <= 1e-15
    assert summ[0, 2] == 0.0 and tuple(pairs[0]) == (0, 1, 0)
    # three unit vectors 120 degrees apart: every pair conflicts at cos -1/2
    ang = np.array([0.0, 2 * np.pi / 3, 4 * np.pi / 3])
    x = np.stack([np.cos(ang), np.sin(ang)], 1)
    _, summ, pairs = oracle.conflicts((x @ x.T)[None])
    assert abs(summ[0, 0] + 0.5) <= 1e-15 and summ[0, 1] <= 1e-15 and pairs[0, 2] == 3
    # opposite and parallel pairs
    x = np.array([[1.0, 2.0, -3.0], [-2.0, -4.0, 6.0], [0.5, 1.0, -1.5]])
    cos, summ, pairs = oracle.conflicts((x @ x.T)[None])
    assert cos[0, 0, 1] == -1.0 and cos[0, 0, 2] == 1.0 and pairs[0, 2] == 2
    assert tuple(pairs[0, :2]) == (0, 1)


def test_conflicts_invariances():
    rng = np.random.default_rng(22)
    x = rand_grads(rng, 4, 50, corr=rand_corr(rng, 4, -0.8, 0.8))
    cos, _, pairs = oracle.conflicts((x @ x.T)[None])
    s = np.array([3.0, 0.25, 7.0, 1.5])          # positive per-task scales
    xs = x * s[:, None]
    cos_s, _, pairs_s = oracle.conflicts((xs @ xs.T)[None])
    np.testing.assert_allclose(cos_s, cos, atol=1e-14)
    assert pairs_s[0, 2] == pairs[0, 2]
    xf = x.copy()
    xf[1] *= -1.0                                 # negating a task flips its row
    cos_f, _, _ = oracle.conflicts((xf @ xf.T)[None])
    sign = np.ones(4)
    sign[1] = -1.0
    np.testing.assert_allclose(cos_f[0], cos[0] * np.outer(sign, sign), atol=1e-14)


def test_conflicts_non_finite_bucket():
    G = np.stack([np.eye(3), np.full((3, 3), np.nan)])
    cos, summ, pairs = oracle.conflicts(G)
    assert np.all(np.isnan(cos[1])) and np.all(np.isnan(summ[1])) and np.all(pairs[1] == -1)
    assert tuple(pairs[0]) == (0, 1, 0)


# ----------------------------------------------------------------------------
# bucket slices and the slice-order Gram sum (Eq. decomp over slices)
# ----------------------------------------------------------------------------


def check_slice_offsets(fn):
    rng = np.random.default_rng(23)
    for T in (1, 2, 3, 7, 8):
        lens = [0, 1, 2, 5, 7, 64, 1000, int(rng.integers(1, 5000))]
        offs = np.concatenate([[0], np.cumsum(lens)])
        so = fn(offs, T)
        assert len(so) == len(lens) * T + 1 and so[0] == 0 and so[-1] == offs[-1]
        assert np.all(np.diff(so) >= 0)
        for b, n in enumerate(lens):
            assert so[b * T] == offs[b]
            sizes = np.diff(so[b * T:(b + 1) * T + 1])
            assert sizes.sum() == n and sizes.max() - sizes.min() <= 1
            # every element's slice, computed element by element: i lies in
            # slice t iff t n / T <= i < (t + 1) n / T rounded down, i.e.
            # t = ceil((i + 1) T / n) - 1
            for i in range(n):
                t = -((-(i + 1) * T) // n) - 1
                assert so[b * T + t] <= offs[b] + i < so[b * T + t + 1], (T, b, i)


def check_gram_reduce(fn):
    rng = np.random.default_rng(24)
    lens = [50, 1, 0, 33, 8]
    offs = np.concatenate([[0], np.cumsum(lens)])
    x = rng.integers(-8, 9, size=(4, offs[-1])).astype(np.float64)   # exact in fp64
    for T in (1, 2, 5):
        so = oracle.slice_offsets(offs, T)
        sub = np.stack([x[:, so[i]:so[i + 1]] @ x[:, so[i]:so[i + 1]].T for i in range(len(so) - 1)])
        parts = sub.reshape(len(lens), T, 4, 4).transpose(1, 0, 2, 3)   # [T, B, K, K]
        full = np.stack([x[:, offs[b]:offs[b + 1]] @ x[:, offs[b]:offs[b + 1]].T for b in range(len(lens))])
        assert np.array_equal(fn(parts), full)


def test_slice_offsets_partition_every_bucket():
    check_slice_offsets(oracle.slice_offsets)


def test_gram_reduce_is_additive_over_slices():
    check_gram_reduce(oracle.gram_reduce)
    # real-valued data: equal to the whole bucket's Gram to fp64 rounding
    rng = np.random.default_rng(25)
    x = rng.standard_normal((3, 1000))
    offs = np.array([0, 1000])
    so = oracle.slice_offsets(offs, 8)
    parts = np.stack([oracle.gram(x, so[t:t + 2] - 0) for t in range(8)])
    np.testing.assert_allclose(oracle.gram_reduce(parts)[0], x @ x.T, rtol=1e-13, atol=1e-12)


def test_global_moo_is_one_bucket():
    """B = 1 (the whole vector as one bucket, global MOO): the Gram is the
    plain matrix of inner products of the full gradients."""
    rng = np.random.default_rng(26)
    x = rng.standard_normal((4, 777))
    G = oracle.gram(x, np.array([0, 777]))[0]
    for i in range(4):
        for j in range(4):
            assert abs(G[i, j] - math.fsum(x[i] * x[j])) <= 1e-12


# ----------------------------------------------------------------------------
# the pins catch plausible mistakes planted in the oracle (on the CPU)
# ----------------------------------------------------------------------------


def check_gram(gram_fn):
    rng = np.random.default_rng(15)
    lens = [3, 1, 8]
    offs = np.concatenate([[0], np.cumsum(lens)])
    x = rand_grads(rng, 3, offs[-1])
    G = gram_fn(x, offs)
    for b in range(3):
        for i in range(3):
            for j in range(3):
                ref = math.fsum(x[i, n] * x[j, n] for n in range(offs[b], offs[b + 1]))
                assert abs(G[b, i, j] - ref) <= 1e-14 * max(1.0, abs(ref))


def check_mgda_k2(fw_fn):
    rng = np.random.default_rng(16)
    for _ in range(20):
        x = rand_grads(rng, 2, 50, corr=np.array([[1, -0.3], [-0.3, 1]]),
                       scales=np.exp(rng.uniform(-1, 1, size=2)))
        a = fw_fn(x @ x.T, 20)
        assert abs(a[0] - _closed_form_k2(x[0], x[1])) <= 1e-10


def _golden(*prefixes):
    for c in json.load(open(GOLD))["cases"]:
        if c["name"].startswith(prefixes):
            g = np.array(c["g"], dtype=np.float64)
            yield c, g @ g.T


def check_mgda_fw_k3(fw_fn):
    # the hand-derived three- and four-task Frank-Wolfe runs
    for c, G in _golden("mgda3", "mgda4", "mgda8"):
        np.testing.assert_allclose(fw_fn(G, 20), c["alpha"], rtol=0, atol=1e-12)


def check_cagrad_fw_k3(ca_fn):
    # the hand-derived runs: symmetric optima, an asymmetric optimum reached by
    # the first step, and the first two steps of an asymmetric run
    for c, G in _golden("cagrad3", "cagrad4", "cagrad8", "cagrad_vertex"):
        wts, w = ca_fn(G, c["c"], c.get("iters", 20))
        np.testing.assert_allclose(wts, c["weights"], rtol=0, atol=1e-12)
        if "w" in c:
            np.testing.assert_allclose(w, c["w"], rtol=0, atol=1e-12)


def _cagrad_dual(G, c, w):
    """F(w) = <g_w, g_avg> + c |g_avg| |g_w| from the vectors' Gram matrix:
    <g_w, g_avg> = w^T G 1 / K and |g|^2 = the quadratic forms."""
    k = G.shape[0]
    one = np.full(k, 1.0 / k)
    return float(w @ G @ one) + c * math.sqrt(max(float(one @ G @ one), 0.0)) * math.sqrt(max(float(w @ G @ w), 0.0))


def check_cagrad_fw_descent(ca_fn):
    """Frank-Wolfe with an exact line search never raises the dual objective,
    stays on the simplex and approaches the exact minimiser (whose optimality
    is pinned by the trust-region, duality-gap and grid checks above)."""
    for k in (3, 4, 6, 8, 10):
        rng = np.random.default_rng(700 + k)
        for trial in range(3):
            n = 64
            x = rand_grads(rng, k, n, corr=rand_corr(rng, k, -0.7, 0.7),
                           scales=np.exp(rng.uniform(-1, 1, size=k)))
            G = x @ x.T
            scale = float(np.max(np.diag(G)))
            for c in (0.25, 0.5, 0.9):
                f_opt = _cagrad_dual(G, c, oracle.cagrad_exact(G, c)[1])
                prev = math.inf
                for it in (0, 1, 2, 5, 20, 100):
                    w = ca_fn(G, c, it)[1]
                    assert w.min() >= 0 and abs(w.sum() - 1) <= 1e-12
                    f = _cagrad_dual(G, c, w)
                    assert f <= prev + 1e-12 * scale
                    prev = f
                f0 = _cagrad_dual(G, c, np.full(k, 1.0 / k))
                f_long = _cagrad_dual(G, c, ca_fn(G, c, 2000)[1])
                assert f_opt - 1e-12 * scale <= f_long <= f_opt + 1e-3 * scale
                assert f_long - f_opt <= 0.01 * (f0 - f_opt) + 1e-12 * scale


def check_pcgrad(pc_fn):
    rng = np.random.default_rng(17)
    for _ in range(10):
        x = rand_grads(rng, 4, 30, corr=rand_corr(rng, 4, -0.8, 0.3))
        order = np.array([rng.permutation([j for j in range(4) if j != t]) for t in range(4)])
        d_ref, _ = vector_pcgrad(x, order)
        np.testing.assert_allclose(pc_fn(x @ x.T, order) @ x, d_ref, rtol=1e-10,
                                   atol=1e-10 * np.abs(d_ref).max())


def check_cagrad(ca_fn):
    rng = np.random.default_rng(18)
    for _ in range(5):
        x = rand_grads(rng, 3, 30, corr=rand_corr(rng, 3, -0.8, 0.8))
        wts, w = ca_fn(x @ x.T, 0.5)
        d = wts @ x
        g0, r = _cagrad_primal(x, 0.5)
        assert np.linalg.norm(d - g0) <= r * (1 + 1e-9) + 1e-12
        gw = w @ x
        dual = float(gw @ g0) + r * float(np.linalg.norm(gw))
        assert abs(float((x @ d).min()) - dual) <= 1e-8 * max(1.0, abs(dual))


def check_combine(comb_fn):
    rng = np.random.default_rng(19)
    offs = np.array([0, 4, 9])
    x = rand_grads(rng, 3, 9)
    W = rng.standard_normal((2, 3))
    out = comb_fn(x, offs, W)
    for b in range(2):
        for n in range(offs[b], offs[b + 1]):
            assert abs(out[n] - math.fsum(W[b, i] * x[i, n] for i in range(3))) <= 1e-14


def test_checks_pass_on_the_oracle():
    check_gram(oracle.gram)
    check_mgda_k2(oracle.mgda_fw)
    check_pcgrad(oracle.pcgrad)
    check_cagrad(oracle.cagrad_exact)
    check_combine(oracle.combine)
    check_mgda_fw_k3(oracle.mgda_fw)
    check_mgda_fw_k3(_fw_copy())
    check_cagrad_fw_k3(oracle.cagrad_fw)
    check_cagrad_fw_k3(_cagrad_fw_copy())
    check_cagrad_fw_descent(oracle.cagrad_fw)
    check_cagrad_fw_descent(_cagrad_fw_copy())
    check_conflicts(oracle.conflicts)
    check_slice_offsets(oracle.slice_offsets)
    check_gram_reduce(oracle.gram_reduce)


def _gram_off_by_one(x, offs):
    out = np.empty((len(offs) - 1, x.shape[0], x.shape[0]))
    for b in range(len(offs) - 1):
        xb = x[:, offs[b]:offs[b + 1] + 1]
        out[b] = xb @ xb.T
    return out


def _fw_swapped_pair(G, iters):
    import oracle.reference as ref
    good = ref.pair_min_norm
    try:
        ref.pair_min_norm = lambda aa, ab, bb: good(bb, ab, aa)
        return ref.mgda_fw(G, iters)
    finally:
        ref.pair_min_norm = good


def _fw_copy(vertex=np.argmin, line=lambda aa, ab, bb: (aa, ab, bb)):
    """The oracle's MGDA Frank-Wolfe, restated so one step can be changed."""
    def fw(G, iters):
        k = G.shape[0]
        best = None
        for i in range(k):
            for j in range(i + 1, k):
                gamma, val = oracle.pair_min_norm(G[i, i], G[i, j], G[j, j])
                if best is None or val < best[0]:
                    best = (val, i, j, gamma)
        _, i, j, gamma = best
        a = np.zeros(k)
        a[i], a[j] = gamma, 1.0 - gamma
        for _ in range(iters):
            ga = G @ a
            t = int(vertex(ga))
            gamma, _ = oracle.pair_min_norm(*line(float(a @ ga), float(ga[t]), float(G[t, t])))
            a = gamma * a
            a[t] += 1.0 - gamma
        return a
    return fw


class _NumpyArgmax:
    """numpy with argmin replaced by argmax."""
    argmin = staticmethod(np.argmax)

    def __getattr__(self, name):
        return getattr(np, name)


def _cagrad_fw_argmax(G, c, iters):
    # mistake: the step vertex and the line-search candidate are maximisers
    import oracle.reference as ref
    good = ref.np
    try:
        ref.np = _NumpyArgmax()
        return ref.cagrad_fw(G, c, iters)
    finally:
        ref.np = good


def _cagrad_fw_copy(start=None, full_gradient=True, step_on_vertex=True):
    """The oracle's CAGrad Frank-Wolfe, restated so one step can be changed:
    the start point, the gradient's second term r G w/|g_w|, and which end of
    the segment the line-search variable weights."""
    def fw(G, c, iters):
        k = G.shape[0]
        b = G.sum(axis=1) / k
        r = c * math.sqrt(max(float(G.sum()) / (k * k), 0.0))
        w = np.full(k, 1.0 / k) if start is None else np.eye(k)[start]
        for _ in range(iters):
            gw = G @ w
            cq = float(w @ gw)
            nrm = math.sqrt(max(cq, 0.0))
            grad = b + (r * gw / nrm if (nrm > 1e-300 and full_gradient) else 0.0)
            s = int(np.argmin(grad))
            bw = float(b @ w)
            beta1 = float(b[s]) - bw
            A = float(G[s, s]) - 2.0 * float(gw[s]) + cq
            Bq = float(gw[s]) - cq
            cands = [0.0, 1.0]
            D = r * r * A - beta1 * beta1
            if A > 0.0 and D > 0.0 and (A * cq - Bq * Bq) / D >= 0.0:
                root = abs(beta1) * math.sqrt((A * cq - Bq * Bq) / D)
                cands += [g for g in ((-Bq - root) / A, (-Bq + root) / A) if 0.0 < g < 1.0]
            cands.sort()
            vals = [bw + beta1 * g + r * math.sqrt(max(A * g * g + 2.0 * Bq * g + cq, 0.0)) for g in cands]
            gamma = cands[int(np.argmin(vals))]
            if step_on_vertex:
                w = (1.0 - gamma) * w
                w[s] += gamma
            else:
                w = gamma * w
                w[s] += 1.0 - gamma
        nrm = math.sqrt(max(float(w @ G @ w), 0.0))
        if r == 0.0 or nrm <= 1e-12 * math.sqrt(max(float(np.max(np.diag(G))), 0.0)):
            return np.full(k, 1.0 / k), w
        return 1.0 / k + (r / nrm) * w, w
    return fw


def _pcgrad_projects_off_current(G, order):
    # mistake: projects d_t off the *current* d_j instead of the original g_j
    k = G.shape[0]
    C = np.eye(k)
    for t in range(k):
        for j in order[t]:
            p = float(C[t] @ G @ C[j])
            if p < 0:
                C[t] -= p / float(C[j] @ G @ C[j]) * C[j]
    return C.sum(0)


def _pcgrad_sign_flip(G, order):
    k = G.shape[0]
    C = np.eye(k)
    for t in range(k):
        for j in order[t]:
            p = float(C[t] @ G[:, j])
            if p < 0:
                C[t, j] += p / G[j, j]
    return C.sum(0)


def _cagrad_radius_squared(G, c):
    # mistake: trust-region radius c |g_avg|^2 instead of c |g_avg|
    import oracle.reference as ref
    good = ref._cagrad_terms
    try:
        ref._cagrad_terms = lambda G, c: (good(G, c)[0], c * float(G.sum()) / G.shape[0] ** 2)
        return ref.cagrad_exact(G, c)
    finally:
        ref._cagrad_terms = good


def _combine_first_bucket_weights(x, offs, W):
    # mistake: every bucket uses bucket 0's weights
    out = np.empty(x.shape[1])
    for b in range(len(offs) - 1):
        out[offs[b]:offs[b + 1]] = W[0] @ x[:, offs[b]:offs[b + 1]]
    return out


def _conflicts_mutant(**change):
    """The oracle's conflicts() with one plausible mistake planted."""
    def fn(grams):
        grams = np.asarray(grams, dtype=np.float64)
        nb, k, _ = grams.shape
        cos = np.zeros((nb, k, k))
        summ = np.empty((nb, 3))
        pairs = np.empty((nb, 3), dtype=np.int64)
        for b in range(nb):
            G = grams[b]
            vals, count, best = [], 0, None
            for i in range(k):
                cos[b, i, i] = 1.0 if G[i, i] > 0 else 0.0
                for j in range(i + 1, k):
                    den = G[i, i] * G[j, j] if change.get("no_sqrt") else math.sqrt(G[i, i] * G[j, j])
                    c = 0.0 if den == 0 else max(-1.0, min(1.0, G[i, j] / den))
                    cos[b, i, j] = cos[b, j, i] = c
                    vals.append(c)
                    count += (G[i, j] <= 0) if change.get("le") else (G[i, j] < 0)
                    ties_last = change.get("last_tie")
                    if best is None or c < best[0] or (ties_last and c == best[0]):
                        best = (c, i, j)
            v = np.array(vals)
            summ[b] = (v.mean(), v.std(ddof=1 if change.get("ddof1") else 0), best[0])
            pairs[b] = (best[1], best[2], count)
        return cos, summ, pairs
    return fn


def _slice_offsets_ceil(offs, T):
    # mistake: rounds the slice starts up
    out = []
    for b in range(len(offs) - 1):
        n = int(offs[b + 1] - offs[b])
        out += [int(offs[b]) + -((-t * n) // T) for t in range(T)]
    return np.array(out + [int(offs[-1])])


def _gram_reduce_drops_last(parts):
    # mistake: the last slice is not added
    acc = np.array(parts[0], dtype=np.float64)
    for t in range(1, len(parts) - 1):
        acc = acc + parts[t]
    return acc


@pytest.mark.parametrize("check,mutant", [
    (check_gram, _gram_off_by_one),
    (check_mgda_k2, _fw_swapped_pair),
    (check_mgda_fw_k3, _fw_copy(vertex=np.argmax)),
    (check_mgda_fw_k3, _fw_copy(line=lambda aa, ab, bb: (bb, ab, aa))),
    (check_cagrad_fw_k3, _cagrad_fw_argmax),
    (check_cagrad_fw_k3, _cagrad_fw_copy(start=0)),
    (check_cagrad_fw_k3, _cagrad_fw_copy(full_gradient=False)),
    (check_cagrad_fw_k3, _cagrad_fw_copy(step_on_vertex=False)),
    (check_cagrad_fw_descent, _cagrad_fw_copy(full_gradient=False)),
    (check_pcgrad, _pcgrad_projects_off_current),
    (check_pcgrad, _pcgrad_sign_flip),
    (check_cagrad, _cagrad_radius_squared),
    (check_combine, _combine_first_bucket_weights),
    (check_conflicts, _conflicts_mutant(no_sqrt=True)),
    (check_conflicts, _conflicts_mutant(le=True)),
    (check_conflicts, _conflicts_mutant(last_tie=True)),
    (check_conflicts, _conflicts_mutant(ddof1=True)),
    (check_slice_offsets, _slice_offsets_ceil),
    (check_gram_reduce, _gram_reduce_drops_last),
])
def test_planted_mistakes_are_caught(check, mutant):
    with pytest.raises(AssertionError):
        check(mutant)
