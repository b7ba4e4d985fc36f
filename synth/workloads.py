"""Model-shaped synthetic gradient workloads (inputs only; no method arithmetic).

The paper fine-tunes Llama-3-8B, Llama-3.1-8B and Qwen3-4B/8B with one
language per GPU (Section 4.1, Appendix E) and cuts the flattened gradient
into fixed-size buckets (Section 3.2, Figure 4).  Its gradients need models
and data that are not available, so each workload below stands in for them
with seeded Gaussian (or Student-t) gradients laid out over the parameter
list of a model of that shape, with a target correlation between the K
per-language gradients drawn per bucket.

Recipe for every workload (one bucket b at a time):

* C_b, the K x K target correlation, has off-diagonals drawn by the
  workload's rule; when C_b is not positive definite its eigenvalues are
  clipped to >= 1e-3, it is rebuilt and rescaled to a unit diagonal.
* z ~ N(0, 1) iid (or Student-t with 3 degrees of freedom), shape [K, n_b],
  from a torch generator keyed by (workload seed, bucket index).
* x = L_b z with L_b = chol(C_b), times an optional per-element scale that
  depends only on the tensor the element belongs to (shared by all tasks),
  times an optional per-(bucket, task) scale; then cast (RNE) to the
  workload's dtype.
"""

from __future__ import annotations

import dataclasses
import math
from typing import Callable, List, Optional, Sequence, Tuple

import numpy as np

MiB = 1 << 20

# ----------------------------------------------------------------------------
# parameter lists (name, numel) in module order
# ----------------------------------------------------------------------------


def gpt2_small_tensors() -> List[Tuple[str, int]]:
    """GPT-2 small: 12 layers, d=768, FFN 3072, vocab 50257, 1024 positions,
    tied output head.  148 tensors, 124,439,808 parameters."""
    d, vocab, layers, ctx, ff = 768, 50257, 12, 1024, 3072
    t = [("wte", vocab * d), ("wpe", ctx * d)]
    for i in range(layers):
        p = f"h.{i}."
        t += [
            (p + "ln_1.weight", d), (p + "ln_1.bias", d),
            (p + "attn.c_attn.weight", d * 3 * d), (p + "attn.c_attn.bias", 3 * d),
            (p + "attn.c_proj.weight", d * d), (p + "attn.c_proj.bias", d),
            (p + "ln_2.weight", d), (p + "ln_2.bias", d),
            (p + "mlp.c_fc.weight", d * ff), (p + "mlp.c_fc.bias", ff),
            (p + "mlp.c_proj.weight", ff * d), (p + "mlp.c_proj.bias", d),
        ]
    t += [("ln_f.weight", d), ("ln_f.bias", d)]
    return t


def llama_tensors(layers: int, d: int, ff: int, vocab: int, n_q: int, n_kv: int,
                  head_dim: int, tied: bool) -> List[Tuple[str, int]]:
    """Llama-style decoder (RMSNorm, GQA attention, SwiGLU MLP), no biases."""
    t = [("embed_tokens", vocab * d)]
    for i in range(layers):
        p = f"layers.{i}."
        t += [
            (p + "input_layernorm", d),
            (p + "self_attn.q_proj", n_q * head_dim * d),
            (p + "self_attn.k_proj", n_kv * head_dim * d),
            (p + "self_attn.v_proj", n_kv * head_dim * d),
            (p + "self_attn.o_proj", d * n_q * head_dim),
            (p + "post_attention_layernorm", d),
            (p + "mlp.gate_proj", ff * d),
            (p + "mlp.up_proj", ff * d),
            (p + "mlp.down_proj", d * ff),
        ]
    t += [("norm", d)]
    if not tied:
        t += [("lm_head", vocab * d)]
    return t


def llama3_8b_tensors():
    """Meta-Llama-3-8B shape: 32 layers, d=4096, FFN 14336, vocab 128256,
    32 query / 8 KV heads of 128, untied head.  291 tensors, 8,030,261,248."""
    return llama_tensors(32, 4096, 14336, 128256, 32, 8, 128, tied=False)


def qwen_1p7b_like_tensors():
    """Qwen3-1.7B-like: 28 layers, d=2048, FFN 6144, vocab 151936, 16 query /
    8 KV heads of 128, tied embeddings.  254 tensors, 1,720,567,808."""
    return llama_tensors(28, 2048, 6144, 151936, 16, 8, 128, tied=True)


# ----------------------------------------------------------------------------
# buckets
# ----------------------------------------------------------------------------


def fixed_bucket_offsets(n: int, bucket_elems: int) -> np.ndarray:
    """Contiguous fixed-size cuts [0, c, 2c, ..., n]; the last bucket takes the
    remainder.  Returns int64 offsets of length B+1."""
    if n < 1 or bucket_elems < 1:
        raise ValueError("n and bucket_elems must be >= 1")
    cuts = np.arange(0, n, bucket_elems, dtype=np.int64)
    return np.concatenate([cuts, np.array([n], dtype=np.int64)])


# ----------------------------------------------------------------------------
# per-bucket correlations
# ----------------------------------------------------------------------------


def _repair(c: np.ndarray, floor: float = 1e-3) -> np.ndarray:
    """Eigen-clip a symmetric matrix to >= floor and rescale to unit diagonal."""
    ev, vec = np.linalg.eigh(c)
    if ev.min() >= floor:
        return c
    ev = np.maximum(ev, floor)
    r = (vec * ev) @ vec.T
    s = 1.0 / np.sqrt(np.diag(r))
    r = r * s[:, None] * s[None, :]
    return 0.5 * (r + r.T)


def _uniform_offdiag(rng, k, lo, hi):
    c = np.eye(k)
    iu = np.triu_indices(k, 1)
    v = rng.uniform(lo, hi, size=len(iu[0]))
    c[iu] = v
    c[(iu[1], iu[0])] = v
    return c


@dataclasses.dataclass(frozen=True)
class CorrRule:
    """How the off-diagonal cosines of each bucket are drawn.

    kind = "uniform": every pair U[lo, hi].
    kind = "conflict": a seeded `frac` of the buckets each get one seeded pair
    with cosine U[c_lo, c_hi] (strongly negative) and every other pair
    U[lo, hi]; the remaining buckets draw every pair U[lo, hi].
    """
    kind: str = "uniform"
    lo: float = -0.5
    hi: float = 0.5
    frac: float = 0.0
    c_lo: float = -0.9
    c_hi: float = -0.5


def bucket_correlations(rule: CorrRule, k: int, b: int, seed: int) -> np.ndarray:
    """[B, K, K] float64 realised (repaired) correlation matrices."""
    rng = np.random.default_rng([seed, 0xC0])
    out = np.empty((b, k, k))
    conflict = np.zeros(b, dtype=bool)
    if rule.kind == "conflict":
        n_conf = int(round(rule.frac * b))
        conflict[rng.choice(b, size=n_conf, replace=False)] = True
    for i in range(b):
        c = _uniform_offdiag(rng, k, rule.lo, rule.hi)
        if conflict[i]:
            p, q = sorted(rng.choice(k, size=2, replace=False))
            c[p, q] = c[q, p] = rng.uniform(rule.c_lo, rule.c_hi)
        out[i] = _repair(c)
    return out


def per_task_scales(k: int, b: int, seed: int, lo: float, hi: float) -> np.ndarray:
    """[B, K] log-uniform per-(bucket, task) gradient scales."""
    rng = np.random.default_rng([seed, 0x5C])
    return np.exp(rng.uniform(math.log(lo), math.log(hi), size=(b, k)))


def pcgrad_orders(b: int, k: int, seed: int) -> np.ndarray:
    """[B, K, K-1] int8: for bucket b and task t, a seeded random permutation of
    the other tasks {j != t} (the order in which t is projected)."""
    rng = np.random.default_rng([seed, 0x9C])
    out = np.empty((b, k, k - 1), dtype=np.int8)
    for i in range(b):
        for t in range(k):
            others = np.array([j for j in range(k) if j != t], dtype=np.int8)
            out[i, t] = rng.permutation(others)
    return out


# ----------------------------------------------------------------------------
# workloads
# ----------------------------------------------------------------------------


@dataclasses.dataclass
class Workload:
    name: str
    K: int
    dtype: str                       # "f32" or "bf16"
    tensors: List[Tuple[str, int]]
    bucket_elems: Optional[int]      # fixed-size cuts; None -> explicit offsets
    method: str                      # "mgda" | "pcgrad" | "cagrad" | "mean"
    corr: CorrRule
    seed: int
    max_iter: int = 20
    cagrad_c: float = 0.5
    dist: str = "normal"             # "normal" | "student_t3"
    tensor_scale: Optional[Tuple[float, float]] = None   # log-uniform per tensor
    task_scale: Optional[Tuple[float, float]] = None     # log-uniform per (bucket, task)
    offsets_override: Optional[np.ndarray] = None

    @property
    def N(self) -> int:
        return int(sum(n for _, n in self.tensors))

    @property
    def elem_bytes(self) -> int:
        return 4 if self.dtype == "f32" else 2

    def offsets(self) -> np.ndarray:
        if self.offsets_override is not None:
            return np.asarray(self.offsets_override, dtype=np.int64)
        return fixed_bucket_offsets(self.N, self.bucket_elems)

    @property
    def B(self) -> int:
        return len(self.offsets()) - 1

    def correlations(self) -> np.ndarray:
        return bucket_correlations(self.corr, self.K, self.B, self.seed)

    def orders(self) -> np.ndarray:
        return pcgrad_orders(self.B, self.K, self.seed)

    def task_scales(self) -> Optional[np.ndarray]:
        if self.task_scale is None:
            return None
        return per_task_scales(self.K, self.B, self.seed, *self.task_scale)

    def tensor_scales(self) -> Optional[np.ndarray]:
        if self.tensor_scale is None:
            return None
        rng = np.random.default_rng([self.seed, 0x7E])
        lo, hi = self.tensor_scale
        return np.exp(rng.uniform(math.log(lo), math.log(hi), size=len(self.tensors)))

    def with_method(self, method: str) -> "Workload":
        return dataclasses.replace(self, method=method, name=f"{self.name.rsplit('-', 1)[0]}-{method}")


def _bucket_bytes_elems(nbytes: int, dtype: str) -> int:
    return nbytes // (4 if dtype == "f32" else 2)


def _make_workloads():
    w = {}
    # Two languages, 1 Mi fp32 elements, four buckets of 256 Ki: MGDA, whose
    # K=2 case has a closed form.
    w["k2-mgda-1m-f32"] = Workload(
        name="k2-mgda-1m-f32", K=2, dtype="f32", tensors=[("flat", 1 << 20)],
        bucket_elems=262_144, method="mgda",
        corr=CorrRule("uniform", -0.5, 0.5), seed=1001)
    # GPT-2 small (124M) fp32, 25 MiB buckets, per-tensor scales, PCGrad.
    w["gpt2-124m-k4-pcgrad-f32"] = Workload(
        name="gpt2-124m-k4-pcgrad-f32", K=4, dtype="f32", tensors=gpt2_small_tensors(),
        bucket_elems=_bucket_bytes_elems(25 * MiB, "f32"), method="pcgrad",
        corr=CorrRule("uniform", -0.6, 0.6), seed=1002, tensor_scale=(1e-4, 1e-1))
    # Llama-3-8B shape bf16, 25 MiB buckets, MGDA Frank-Wolfe 20 iterations.
    w["llama3-8b-k4-mgda-bf16"] = Workload(
        name="llama3-8b-k4-mgda-bf16", K=4, dtype="bf16", tensors=llama3_8b_tensors(),
        bucket_elems=_bucket_bytes_elems(25 * MiB, "bf16"), method="mgda",
        corr=CorrRule("uniform", -0.8, 0.8), seed=1003)
    # Same shape, eight languages (the paper's own deployment width), CAGrad c=0.5.
    w["llama3-8b-k8-cagrad-bf16"] = Workload(
        name="llama3-8b-k8-cagrad-bf16", K=8, dtype="bf16", tensors=llama3_8b_tensors(),
        bucket_elems=_bucket_bytes_elems(25 * MiB, "bf16"), method="cagrad",
        corr=CorrRule("conflict", 0.0, 0.6, frac=0.10, c_lo=-0.9, c_hi=-0.5), seed=1004)
    # Qwen3-1.7B-like fp32, K=10, heavy-tailed entries; bucket-size sweep x method.
    for mib in (1, 5, 25, 100):
        for m in ("mgda", "pcgrad", "cagrad"):
            nm = f"qwen-1.7b-k10-{mib}mib-{m}-f32"
            w[nm] = Workload(
                name=nm, K=10, dtype="f32", tensors=qwen_1p7b_like_tensors(),
                bucket_elems=_bucket_bytes_elems(mib * MiB, "f32"), method=m,
                corr=CorrRule("uniform", -0.6, 0.6), seed=1005, dist="student_t3")
    return w


WORKLOADS = _make_workloads()


def small_workload(base: Workload, n: int, bucket_lens: Optional[Sequence[int]] = None,
                   bucket_elems: Optional[int] = None, seed: Optional[int] = None,
                   **overrides) -> Workload:
    """A reduced copy of `base` (same K, dtype, method and recipe) over n
    elements.  The parameter list is `base`'s scaled down to n (each tensor
    keeps its share, at least 1 element) so per-tensor scales still vary
    inside a bucket.  Buckets: explicit lengths (ragged allowed) or fixed cuts.
    """
    sizes = np.array([s for _, s in base.tensors], dtype=np.float64)
    share = np.maximum(1, np.floor(sizes / sizes.sum() * n)).astype(np.int64)
    share[-1] += n - share.sum()
    if share[-1] < 1:  # pathological tiny n: fall back to one tensor
        share = np.array([n], dtype=np.int64)
    names = [nm for nm, _ in base.tensors][: len(share)]
    tensors = list(zip(names, (int(s) for s in share)))
    offs = None
    if bucket_lens is not None:
        assert sum(bucket_lens) == n
        offs = np.concatenate([[0], np.cumsum(bucket_lens)]).astype(np.int64)
    be = bucket_elems if bucket_elems is not None else (None if offs is not None else base.bucket_elems)
    kw = dict(name=f"{base.name}@{n}", tensors=tensors, bucket_elems=be, offsets_override=offs)
    if seed is not None:
        kw["seed"] = seed
    kw.update(overrides)
    return dataclasses.replace(base, **kw)


# ----------------------------------------------------------------------------
# gradient generation (torch; runs on the device that will hold the grads)
# ----------------------------------------------------------------------------


def _torch_dtype(dtype: str):
    import torch
    return torch.float32 if dtype == "f32" else torch.bfloat16


def fill_grads(wl: Workload, device="cpu", out=None, buckets: Optional[Sequence[int]] = None,
               progress: Optional[Callable[[int], None]] = None):
    """Draw the K gradients of `wl` as a contiguous [K, N] tensor on `device`.

    Bucket b is drawn from torch generator seed (wl.seed * 1_000_003 + b), so
    any subset of buckets can be regenerated on its own.  `out` may be a
    preallocated [K, N] tensor; `buckets` restricts which buckets are drawn.
    """
    import torch
    offs = wl.offsets()
    corr = wl.correlations()
    tscale = wl.tensor_scales()
    kscale = wl.task_scales()
    tdt = _torch_dtype(wl.dtype)
    if out is None:
        out = torch.empty((wl.K, wl.N), dtype=tdt, device=device)
    tens_off = np.concatenate([[0], np.cumsum([s for _, s in wl.tensors])]).astype(np.int64)
    gen = torch.Generator(device=device)
    todo = range(len(offs) - 1) if buckets is None else buckets
    for b in todo:
        lo, hi = int(offs[b]), int(offs[b + 1])
        n = hi - lo
        gen.manual_seed(wl.seed * 1_000_003 + b)
        z = torch.randn((wl.K, n), generator=gen, device=device, dtype=torch.float32)
        if wl.dist == "student_t3":
            chi = torch.randn((3, wl.K, n), generator=gen, device=device, dtype=torch.float32)
            z = z / torch.sqrt((chi * chi).sum(0) / 3.0)
            del chi
        L = torch.from_numpy(np.linalg.cholesky(corr[b]).astype(np.float32)).to(device)
        x = L @ z
        del z
        if tscale is not None:
            # per-element scale of the tensor each element belongs to
            t0 = int(np.searchsorted(tens_off, lo, side="right") - 1)
            t1 = int(np.searchsorted(tens_off, hi, side="left"))
            seg_lo = np.maximum(tens_off[t0:t1], lo)
            seg_hi = np.minimum(tens_off[t0 + 1:t1 + 1], hi)
            reps = torch.from_numpy((seg_hi - seg_lo).astype(np.int64)).to(device)
            vals = torch.from_numpy(tscale[t0:t1].astype(np.float32)).to(device)
            x *= torch.repeat_interleave(vals, reps)[None, :]
        if kscale is not None:
            x *= torch.from_numpy(kscale[b].astype(np.float32)).to(device)[:, None]
        out[:, lo:hi] = x.to(tdt)
        del x
        if progress is not None:
            progress(b)
    return out


def host_rows(grads, lo: int, hi: int) -> np.ndarray:
    """Copy columns [lo, hi) of a [K, N] gradient tensor to host memory as a
    numpy array: float32 for fp32 grads, uint16 bit patterns for bf16."""
    import torch
    sl = grads[:, lo:hi].contiguous().cpu()
    if sl.dtype == torch.bfloat16:
        return sl.view(torch.int16).numpy().view(np.uint16)
    return sl.numpy()
