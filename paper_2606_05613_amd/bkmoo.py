"""Python binding of libbkmoo (argument marshalling only).

Every step of the path runs in the HIP library; this module turns torch
tensors into the C ABI's pointers and sizes, allocates outputs and the
workspace with torch's caching allocator when the caller passes none, and
raises on any non-OK status.  There is no fallback: if the library is not
built, importing this module fails.

Names mirror include/bkmoo.h: workspace_size, gram, solve, combine, resolve,
resolve_noalloc, conflicts, slice_offsets, gram_reduce, resolve_path, resolve_traffic,
read_device_error, set_resolve_path, set_wait_limit, set_grid_override,
status_string.
"""

from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence, Union

import torch  # must be imported before the library so both share one HIP runtime

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libbkmoo.so")

F32, BF16 = 0, 1
METHODS = {"mgda": 0, "pcgrad": 1, "cagrad": 2, "mean": 3, "mgda-exact": 4, "cagrad-exact": 5}
DEVERR_OFFSETS = 0x1
DEVERR_TIMEOUT = 0x2
PATH_TWO_PASS, PATH_HYBRID, PATH_REFILL = 1, 3, 4


class BkmooError(RuntimeError):
    pass


class _Hparams(ctypes.Structure):
    _fields_ = [("max_iter", ctypes.c_int32), ("cagrad_c", ctypes.c_double),
                ("pcgrad_order", ctypes.c_void_p)]


def _load():
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built; run `python -m paper_2606_05613_amd.build`")
    lib = ctypes.CDLL(LIB_PATH)
    i32, i64, sz, vp, u32 = ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t, ctypes.c_void_p, ctypes.c_uint32
    vpp = ctypes.POINTER(ctypes.c_void_p)
    sig = {
        "bkmoo_workspace_size": [i32, i64, i32, ctypes.c_int, ctypes.POINTER(sz)],
        "bkmoo_gram": [i32, vpp, ctypes.c_int, i64, i32, vp, vp, vp, sz, vp],
        "bkmoo_solve": [i32, i32, vp, ctypes.c_int, ctypes.POINTER(_Hparams), vp, vp, vp],
        "bkmoo_combine": [i32, vpp, ctypes.c_int, i64, i32, vp, vp, vp, ctypes.c_int, vp, sz, vp],
        "bkmoo_resolve": [i32, vpp, ctypes.c_int, i64, i32, vp, ctypes.c_int, ctypes.POINTER(_Hparams),
                          vp, ctypes.c_int, vp, vp, vp, vp, sz, vp],
        "bkmoo_resolve_noalloc": [i32, vpp, ctypes.c_int, i64, i32, vp, ctypes.c_int, ctypes.POINTER(_Hparams),
                                  vp, ctypes.c_int, vp, vp, vp, vp],
        "bkmoo_conflicts": [i32, i32, vp, vp, vp, vp, vp],
        "bkmoo_slice_offsets": [i32, i32, vp, vp, vp],
        "bkmoo_resolve_traffic": [i32, i64, i32, vp, ctypes.c_int, ctypes.c_int, ctypes.c_int, i32, i32,
                                  ctypes.POINTER(ctypes.c_uint64)],
        "bkmoo_gram_reduce": [i32, i32, i32, vp, ctypes.c_int, vp, vp],
        "bkmoo_read_device_error": [vp, ctypes.POINTER(u32), vp],
        "bkmoo_set_grid_override": [i32],
        "bkmoo_resolve_path": [i32, i64, i32, ctypes.c_int, ctypes.c_int, i32, ctypes.c_int, i32,
                               ctypes.POINTER(i32)],
        "bkmoo_set_resolve_path": [i32],
        "bkmoo_set_wait_limit": [u32],
        "bkmoo_status_string": [ctypes.c_int],
    }
    for name, args in sig.items():
        fn = getattr(lib, name)
        fn.argtypes = args
        fn.restype = ctypes.c_char_p if name == "bkmoo_status_string" else ctypes.c_int
    return lib


_lib = _load()

EXPORTS = ("bkmoo_workspace_size", "bkmoo_gram", "bkmoo_solve", "bkmoo_combine", "bkmoo_resolve",
           "bkmoo_resolve_noalloc",
           "bkmoo_conflicts", "bkmoo_slice_offsets", "bkmoo_gram_reduce", "bkmoo_resolve_traffic",
           "bkmoo_read_device_error", "bkmoo_set_grid_override", "bkmoo_resolve_path",
           "bkmoo_set_resolve_path", "bkmoo_set_wait_limit", "bkmoo_status_string")


def status_string(st: int) -> str:
    return _lib.bkmoo_status_string(st).decode()


def _check(st: int, what: str):
    if st != 0:
        raise BkmooError(f"{what}: {status_string(st)} ({st})")


def _dt(t: torch.Tensor) -> int:
    if t.dtype == torch.float32:
        return F32
    if t.dtype == torch.bfloat16:
        return BF16
    raise TypeError(f"unsupported dtype {t.dtype} (float32 or bfloat16)")


def _torch_dt(code: int):
    return torch.float32 if code == F32 else torch.bfloat16


def _stream_ptr(device) -> int:
    return torch.cuda.current_stream(device).cuda_stream


Grads = Union[torch.Tensor, Sequence[torch.Tensor]]


def _rows(grads: Grads):
    """K row pointers (host array), dtype code, K, N, device."""
    if isinstance(grads, torch.Tensor):
        if grads.dim() != 2:
            raise ValueError("grads must be [K, N] or a list of K 1-D tensors")
        if not grads.is_contiguous():
            raise ValueError("a [K, N] grads tensor must be contiguous")
        rows = [grads[i] for i in range(grads.shape[0])]
    else:
        rows = list(grads)
    if not rows:
        raise ValueError("no gradient rows")
    dt = _dt(rows[0])
    n = rows[0].numel()
    dev = rows[0].device
    for r in rows:
        if r.dtype != rows[0].dtype or r.numel() != n or r.device != dev or r.dim() != 1 \
                or not r.is_contiguous():
            raise ValueError("rows must be contiguous 1-D tensors of one dtype, length and device")
        if dev.type != "cuda":
            raise ValueError("gradient rows must be on a GPU")
    arr = (ctypes.c_void_p * len(rows))(*[r.data_ptr() for r in rows])
    return arr, dt, len(rows), n, dev, rows


def _gpu(t: torch.Tensor, what: str):
    """The GPU device of t; host tensors are refused (the kernels would
    dereference their pointers on the GPU)."""
    if t.device.type != "cuda":
        raise ValueError(f"{what} must be on a GPU")
    return t.device


def _tensor(t: torch.Tensor, shape, dtype, dev, what: str) -> int:
    """Pointer of a caller-supplied tensor that must match exactly."""
    if t.dtype != dtype or tuple(t.shape) != tuple(shape) or not t.is_contiguous() or t.device != dev:
        raise ValueError(f"{what} must be a contiguous {dtype} tensor of shape {tuple(shape)} on {dev}")
    return t.data_ptr()


def _offsets(offsets: torch.Tensor, dev) -> torch.Tensor:
    if offsets.dtype != torch.int64 or offsets.dim() != 1 or offsets.device != dev \
            or not offsets.is_contiguous():
        raise ValueError("bucket_offsets must be a contiguous int64 1-D tensor on the grads' device")
    return offsets


def _hparams(max_iter: int, cagrad_c: float, pcgrad_order: Optional[torch.Tensor], K: int, B: int, dev):
    ptr = None
    if pcgrad_order is not None:
        ptr = _tensor(pcgrad_order, (B, K, K - 1), torch.int8, dev, "pcgrad_order")
    return _Hparams(int(max_iter), float(cagrad_c), ptr)


def workspace_size(K: int, N: int, B: int, dtype) -> int:
    code = dtype if isinstance(dtype, int) else (F32 if dtype in (torch.float32, "f32") else BF16)
    out = ctypes.c_size_t(0)
    _check(_lib.bkmoo_workspace_size(K, N, B, code, ctypes.byref(out)), "bkmoo_workspace_size")
    return out.value


def _workspace(ws: Optional[torch.Tensor], K, N, B, dt, dev) -> torch.Tensor:
    need = workspace_size(K, N, B, dt)
    if ws is None:
        return torch.empty(need, dtype=torch.uint8, device=dev)
    if ws.dtype != torch.uint8 or ws.device != dev or not ws.is_contiguous():
        raise ValueError("workspace must be a contiguous uint8 tensor on the grads' device")
    return ws


def gram(grads: Grads, bucket_offsets: torch.Tensor, gram_out: Optional[torch.Tensor] = None,
         workspace: Optional[torch.Tensor] = None) -> torch.Tensor:
    """Per-bucket Gram matrices, fp64 [B, K, K]."""
    arr, dt, K, N, dev, _ = _rows(grads)
    offs = _offsets(bucket_offsets, dev)
    B = offs.numel() - 1
    if gram_out is None:
        gram_out = torch.empty((B, K, K), dtype=torch.float64, device=dev)
    _tensor(gram_out, (B, K, K), torch.float64, dev, "gram_out")
    ws = _workspace(workspace, K, N, B, dt, dev)
    with torch.cuda.device(dev):
        _check(_lib.bkmoo_gram(K, arr, dt, N, B, offs.data_ptr(), gram_out.data_ptr(), ws.data_ptr(),
                               ws.numel(), _stream_ptr(dev)), "bkmoo_gram")
    return gram_out


def solve(gram_in: torch.Tensor, method: str, max_iter: int = 20, cagrad_c: float = 0.5,
          pcgrad_order: Optional[torch.Tensor] = None, weights: Optional[torch.Tensor] = None,
          aux: Optional[torch.Tensor] = None):
    """Per-bucket combine weights (fp32 [B, K]) and the method's variable (fp64 [B, K])."""
    if gram_in.dtype != torch.float64 or gram_in.dim() != 3 or not gram_in.is_contiguous():
        raise ValueError("gram must be a contiguous fp64 [B, K, K] tensor")
    B, K, _ = gram_in.shape
    dev = _gpu(gram_in, "gram")
    if weights is None:
        weights = torch.empty((B, K), dtype=torch.float32, device=dev)
    if aux is None:
        aux = torch.empty((B, K), dtype=torch.float64, device=dev)
    _tensor(weights, (B, K), torch.float32, dev, "weights")
    _tensor(aux, (B, K), torch.float64, dev, "aux")
    hp = _hparams(max_iter, cagrad_c, pcgrad_order, K, B, dev)
    with torch.cuda.device(dev):
        _check(_lib.bkmoo_solve(K, B, gram_in.data_ptr(), METHODS[method], ctypes.byref(hp),
                                weights.data_ptr(), aux.data_ptr(), _stream_ptr(dev)), "bkmoo_solve")
    return weights, aux


SLICES_RANK_MAJOR, SLICES_BUCKET_MAJOR = 0, 1


def slice_offsets(bucket_offsets: torch.Tensor, T: int) -> torch.Tensor:
    """Offsets (int64 [B*T+1], bucket-major) of T contiguous slices of every
    bucket: slice t of bucket b starts at o_b + floor(t n_b / T)."""
    offs = bucket_offsets
    if offs.dtype != torch.int64 or offs.dim() != 1 or not offs.is_contiguous() or offs.device.type != "cuda":
        raise ValueError("bucket_offsets must be a contiguous int64 GPU tensor")
    B = offs.numel() - 1
    out = torch.empty(B * T + 1, dtype=torch.int64, device=offs.device)
    with torch.cuda.device(offs.device):
        _check(_lib.bkmoo_slice_offsets(B, int(T), offs.data_ptr(), out.data_ptr(), _stream_ptr(offs.device)),
               "bkmoo_slice_offsets")
    return out


def gram_reduce(partial: torch.Tensor, layout: int = SLICES_RANK_MAJOR,
                gram_out: Optional[torch.Tensor] = None) -> torch.Tensor:
    """Sum per-slice partial Grams in slice order: partial fp64 [T, B, K, K]
    (rank-major) or [B, T, K, K] (bucket-major) -> [B, K, K]."""
    if partial.dtype != torch.float64 or partial.dim() != 4 or not partial.is_contiguous():
        raise ValueError("partial must be a contiguous fp64 4-d tensor")
    if layout == SLICES_RANK_MAJOR:
        T, B, K, _ = partial.shape
    else:
        B, T, K, _ = partial.shape
    dev = _gpu(partial, "partial")
    if gram_out is None:
        gram_out = torch.empty((B, K, K), dtype=torch.float64, device=dev)
    _tensor(gram_out, (B, K, K), torch.float64, dev, "gram_out")
    with torch.cuda.device(dev):
        _check(_lib.bkmoo_gram_reduce(K, B, T, partial.data_ptr(), int(layout), gram_out.data_ptr(),
                                      _stream_ptr(dev)), "bkmoo_gram_reduce")
    return gram_out


def conflicts(gram_in: torch.Tensor, cosines: bool = True, summary: bool = True,
              pairs: bool = True):
    """Per-bucket conflict diagnostics from fp64 [B, K, K] Gram matrices:
    (cosines fp64 [B, K, K], summary fp64 [B, 3] = mean / population std / min
    pairwise cosine, pairs int32 [B, 3] = argmin pair and the count of pairs
    with a negative inner product).  Outputs not asked for are None."""
    if gram_in.dtype != torch.float64 or gram_in.dim() != 3 or not gram_in.is_contiguous():
        raise ValueError("gram must be a contiguous fp64 [B, K, K] tensor")
    B, K, _ = gram_in.shape
    dev = _gpu(gram_in, "gram")
    cos = torch.empty((B, K, K), dtype=torch.float64, device=dev) if cosines else None
    summ = torch.empty((B, 3), dtype=torch.float64, device=dev) if summary else None
    prs = torch.empty((B, 3), dtype=torch.int32, device=dev) if pairs else None
    ptr = lambda t: t.data_ptr() if t is not None else None
    with torch.cuda.device(dev):
        _check(_lib.bkmoo_conflicts(K, B, gram_in.data_ptr(), ptr(cos), ptr(summ), ptr(prs),
                                    _stream_ptr(dev)), "bkmoo_conflicts")
    return cos, summ, prs


def combine(grads: Grads, bucket_offsets: torch.Tensor, weights: torch.Tensor,
            out: Optional[torch.Tensor] = None, out_dtype=None,
            workspace: Optional[torch.Tensor] = None) -> torch.Tensor:
    """The concatenated bucket updates, N elements of out_dtype (default: input dtype)."""
    arr, dt, K, N, dev, _ = _rows(grads)
    offs = _offsets(bucket_offsets, dev)
    B = offs.numel() - 1
    _tensor(weights, (B, K), torch.float32, dev, "weights")
    if out is None:
        out = torch.empty(N, dtype=out_dtype or _torch_dt(dt), device=dev)
    odt = _dt(out)
    _tensor(out, (N,), out.dtype, dev, "out")
    ws = _workspace(workspace, K, N, B, dt, dev)
    with torch.cuda.device(dev):
        _check(_lib.bkmoo_combine(K, arr, dt, N, B, offs.data_ptr(), weights.data_ptr(), out.data_ptr(),
                                  odt, ws.data_ptr(), ws.numel(), _stream_ptr(dev)), "bkmoo_combine")
    return out


def resolve(grads: Grads, bucket_offsets: torch.Tensor, method: str, max_iter: int = 20,
            cagrad_c: float = 0.5, pcgrad_order: Optional[torch.Tensor] = None,
            out: Optional[torch.Tensor] = None, out_dtype=None,
            gram_out: Optional[torch.Tensor] = None, weights: Optional[torch.Tensor] = None,
            aux: Optional[torch.Tensor] = None, workspace: Optional[torch.Tensor] = None,
            check_error: bool = False):
    """Gram -> solve -> combine on the current stream.  Returns `out`; gram,
    weights and aux are written to the tensors passed (if any).

    The device error word (invalid offsets, an expired wait of the hybrid
    path) lives in the workspace: pass `workspace` and read it with
    read_device_error(), or set check_error=True to wait for the call and
    raise BkmooError when the word is not zero."""
    arr, dt, K, N, dev, _ = _rows(grads)
    offs = _offsets(bucket_offsets, dev)
    B = offs.numel() - 1
    if out is None:
        out = torch.empty(N, dtype=out_dtype or _torch_dt(dt), device=dev)
    odt = _dt(out)
    _tensor(out, (N,), out.dtype, dev, "out")
    ws = _workspace(workspace, K, N, B, dt, dev)
    hp = _hparams(max_iter, cagrad_c, pcgrad_order, K, B, dev)

    def ptr(t, shape, dtype, what):
        return None if t is None else _tensor(t, shape, dtype, dev, what)

    with torch.cuda.device(dev):
        _check(_lib.bkmoo_resolve(K, arr, dt, N, B, offs.data_ptr(), METHODS[method], ctypes.byref(hp),
                                  out.data_ptr(), odt, ptr(gram_out, (B, K, K), torch.float64, "gram_out"),
                                  ptr(weights, (B, K), torch.float32, "weights"),
                                  ptr(aux, (B, K), torch.float64, "aux"),
                                  ws.data_ptr(), ws.numel(), _stream_ptr(dev)), "bkmoo_resolve")
    if check_error:
        err = read_device_error(ws)
        if err:
            what = [n for bit, n in ((DEVERR_OFFSETS, "invalid bucket offsets"),
                                     (DEVERR_TIMEOUT, "a bounded wait expired")) if err & bit]
            raise BkmooError(f"bkmoo_resolve: device error 0x{err:x} ({', '.join(what) or 'unknown'})")
    return out


def resolve_noalloc(grads: Grads, bucket_offsets: torch.Tensor, method: str, out: torch.Tensor,
                    max_iter: int = 20, cagrad_c: float = 0.5, pcgrad_order: Optional[torch.Tensor] = None,
                    gram_out: Optional[torch.Tensor] = None, weights: Optional[torch.Tensor] = None,
                    aux: Optional[torch.Tensor] = None):
    """resolve() on the library's own fixed device scratch (bkmoo_resolve_noalloc):
    nothing is allocated, so `out` must be given.  Calls that overlap on one
    device share that scratch and race.  Returns `out`."""
    arr, dt, K, N, dev, _ = _rows(grads)
    offs = _offsets(bucket_offsets, dev)
    B = offs.numel() - 1
    _tensor(out, (N,), out.dtype, dev, "out")
    hp = _hparams(max_iter, cagrad_c, pcgrad_order, K, B, dev)

    def ptr(t, shape, dtype, what):
        return None if t is None else _tensor(t, shape, dtype, dev, what)

    with torch.cuda.device(dev):
        _check(_lib.bkmoo_resolve_noalloc(K, arr, dt, N, B, offs.data_ptr(), METHODS[method], ctypes.byref(hp),
                                          out.data_ptr(), _dt(out),
                                          ptr(gram_out, (B, K, K), torch.float64, "gram_out"),
                                          ptr(weights, (B, K), torch.float32, "weights"),
                                          ptr(aux, (B, K), torch.float64, "aux"), _stream_ptr(dev)),
               "bkmoo_resolve_noalloc")
    return out


def read_device_error(workspace: torch.Tensor) -> int:
    v = ctypes.c_uint32(0)
    dev = _gpu(workspace, "workspace")
    with torch.cuda.device(dev):
        _check(_lib.bkmoo_read_device_error(workspace.data_ptr(), ctypes.byref(v), _stream_ptr(dev)),
               "bkmoo_read_device_error")
    return v.value


def set_grid_override(workgroups: int):
    _check(_lib.bkmoo_set_grid_override(int(workgroups)), "bkmoo_set_grid_override")


def resolve_path(grads: Grads, bucket_offsets_len: int, method: str = "mgda", max_iter: int = 20,
                 out_dtype=None) -> int:
    """PATH_TWO_PASS, PATH_HYBRID or PATH_REFILL: what resolve() would run for these
    grads and method (output assumed aligned like the rows)."""
    arr, dt, K, N, dev, rows = _rows(grads)
    B = bucket_offsets_len - 1
    odt = dt if out_dtype is None else _dt(torch.empty(0, dtype=out_dtype))
    phases = {r.data_ptr() % 16 for r in rows}
    out = ctypes.c_int32(0)
    _check(_lib.bkmoo_resolve_path(K, N, B, dt, odt, int(len(phases) == 1), METHODS[method],
                                   int(max_iter), ctypes.byref(out)), "bkmoo_resolve_path")
    return out.value


def resolve_traffic(K: int, bucket_offsets, dtype, path: int, out_dtype=None, method: str = "mgda",
                    max_iter: int = 20) -> int:
    """Bytes a resolve on `path` requests from memory for these offsets (a
    host int64 array-like of B+1 entries); on the hybrid path part of the
    re-read is served by the last-level cache."""
    import numpy as np
    offs = np.ascontiguousarray(np.asarray(bucket_offsets, dtype=np.int64))
    code = lambda d: d if isinstance(d, int) else (F32 if d in (torch.float32, "f32") else BF16)
    dt = code(dtype)
    odt = dt if out_dtype is None else code(out_dtype)
    out = ctypes.c_uint64(0)
    _check(_lib.bkmoo_resolve_traffic(K, int(offs[-1]), len(offs) - 1, offs.ctypes.data, dt, odt, METHODS[method],
                                      int(max_iter), int(path), ctypes.byref(out)), "bkmoo_resolve_traffic")
    return out.value


def set_resolve_path(path: int):
    """0 automatic, PATH_TWO_PASS, PATH_HYBRID or PATH_REFILL (process-wide)."""
    _check(_lib.bkmoo_set_resolve_path(int(path)), "bkmoo_set_resolve_path")


def set_wait_limit(polls: int):
    _check(_lib.bkmoo_set_wait_limit(int(polls)), "bkmoo_set_wait_limit")
