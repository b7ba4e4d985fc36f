"""The C-ABI library loads on a machine without a GPU, exports every entry
point include/bkmoo.h declares, and rejects bad arguments synchronously,
before anything is queued (no compute call is made here)."""

import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "bkmoo.h")


@pytest.fixture(scope="module")
def b():
    import torch  # noqa: F401  (shares its HIP runtime with the library)
    from paper_2606_05613_amd import bkmoo
    return bkmoo


def declared_functions():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"^\s*(?:const\s+char\s*\*\s*|bkmoo_status\s+)(bkmoo_\w+)\s*\(", text, re.M)))


def test_header_declares_the_boundary():
    names = declared_functions()
    for n in ("bkmoo_workspace_size", "bkmoo_gram", "bkmoo_solve", "bkmoo_combine", "bkmoo_resolve",
              "bkmoo_read_device_error", "bkmoo_status_string"):
        assert n in names


def test_library_exports_every_declared_symbol(b):
    lib = ctypes.CDLL(b.LIB_PATH)
    for n in declared_functions():
        assert hasattr(lib, n), n
    assert set(declared_functions()) <= set(b.EXPORTS)


def test_binding_argument_counts_match_the_header(b):
    """Every function the binding types has the header's number of
    parameters (a signature change in one and not the other would pass
    pointers in the wrong slots)."""
    text = open(HEADER).read()
    decls = re.findall(r"^(?:bkmoo_status|const char\s*\*)\s*(bkmoo_\w+)\s*\(([^;]*)\);", text, re.M)
    assert decls and {n for n, _ in decls} == set(declared_functions())
    for name, params in decls:
        n_header = len([p for p in params.split(",") if p.strip()])
        fn = getattr(b._lib, name)
        assert fn.argtypes is not None and len(fn.argtypes) == n_header, name


def test_status_strings(b):
    for code, word in ((0, "OK"), (-1, "EINVAL"), (-2, "EUNSUPPORTED"), (-3, "EWORKSPACE"), (-4, "EHIP")):
        assert word in b.status_string(code)
    assert "unknown" in b.status_string(7)


def test_workspace_size_rules(b):
    L = b._lib
    out = ctypes.c_size_t(0)
    assert L.bkmoo_workspace_size(4, 1000, 3, 1, ctypes.byref(out)) == 0 and out.value > 0
    small = out.value
    assert L.bkmoo_workspace_size(4, 10**9, 3, 1, ctypes.byref(out)) == 0 and out.value > small
    assert L.bkmoo_workspace_size(4, 0, 1, 0, ctypes.byref(out)) == 0
    assert L.bkmoo_workspace_size(1, 1000, 3, 1, ctypes.byref(out)) == -1
    assert L.bkmoo_workspace_size(17, 1000, 3, 1, ctypes.byref(out)) == -2
    assert L.bkmoo_workspace_size(4, -1, 3, 1, ctypes.byref(out)) == -1
    assert L.bkmoo_workspace_size(4, 1000, 0, 1, ctypes.byref(out)) == -1
    assert L.bkmoo_workspace_size(4, 1000, 3, 2, ctypes.byref(out)) == -1
    assert L.bkmoo_workspace_size(4, 1000, 3, 1, None) == -1
    # an upper bound on per-chunk slots: about 8 K(K+1)/2 bytes per few thousand elements
    assert b.workspace_size(4, 8_030_261_248, 613, "bf16") < 64 << 20


FAKE = 0x7F0000000000   # 256-aligned, never dereferenced: every call below fails validation first


def rows(k, base=FAKE, step=1 << 20):
    return (ctypes.c_void_p * k)(*[base + i * step for i in range(k)])


def test_gram_and_combine_argument_errors(b):
    L = b._lib
    ws_need = b.workspace_size(4, 4096, 2, "f32")
    r = rows(4)
    offs, out, ws, gram = FAKE + (64 << 20), FAKE + (80 << 20), FAKE + (96 << 20), FAKE + (128 << 20)
    assert L.bkmoo_gram(4, None, 0, 4096, 2, offs, gram, ws, ws_need, None) == -1
    assert L.bkmoo_gram(4, r, 0, 4096, 2, None, gram, ws, ws_need, None) == -1
    assert L.bkmoo_gram(4, r, 0, 4096, 2, offs, None, ws, ws_need, None) == -1
    assert L.bkmoo_gram(4, r, 0, 4096, 2, offs, gram, ws, ws_need - 1, None) == -3
    assert L.bkmoo_gram(4, r, 5, 4096, 2, offs, gram, ws, ws_need, None) == -1
    assert L.bkmoo_gram(17, r, 0, 4096, 2, offs, gram, ws, ws_need, None) == -2
    assert L.bkmoo_gram(4, rows(4, FAKE + 2), 0, 4096, 2, offs, gram, ws, ws_need, None) == -1  # misaligned fp32
    w = FAKE + (112 << 20)
    assert L.bkmoo_combine(4, r, 0, 4096, 2, offs, w, out, 0, ws, ws_need - 8, None) == -3
    assert L.bkmoo_combine(4, r, 0, 4096, 2, offs, None, out, 0, ws, ws_need, None) == -1
    # output overlapping a row but not equal to it
    assert L.bkmoo_combine(4, r, 0, 4096, 2, offs, w, FAKE + 64, 0, ws, ws_need, None) == -1
    # in place with a different element size overlaps too
    assert L.bkmoo_combine(4, r, 0, 4096, 2, offs, w, FAKE, 1, ws, ws_need, None) == -1


def test_solve_and_resolve_hparam_errors(b):
    L = b._lib
    g, w = FAKE, FAKE + (1 << 20)
    hp = b._Hparams(20, 0.5, None)
    assert L.bkmoo_solve(4, 3, g, 7, ctypes.byref(hp), w, None, None) == -1        # method
    assert L.bkmoo_solve(4, 3, g, 0, None, w, None, None) == -1                     # hp needed
    assert L.bkmoo_solve(4, 3, None, 0, ctypes.byref(hp), w, None, None) == -1
    assert L.bkmoo_solve(4, 3, g, 0, ctypes.byref(hp), None, None, None) == -1
    assert L.bkmoo_solve(1, 3, g, 0, ctypes.byref(hp), w, None, None) == -1
    assert L.bkmoo_solve(4, 0, g, 0, ctypes.byref(hp), w, None, None) == -1
    for bad in (b._Hparams(20, 1.0, None), b._Hparams(20, -0.1, None), b._Hparams(20, float("nan"), None),
                b._Hparams(-1, 0.5, None)):
        assert L.bkmoo_solve(4, 3, g, 2, ctypes.byref(bad), w, None, None) == -1
    r = rows(4)
    ws_need = b.workspace_size(4, 4096, 2, "bf16")
    out, ws, offs = FAKE + (80 << 20), FAKE + (96 << 20), FAKE + (64 << 20)
    bad = b._Hparams(20, 1.5, None)
    assert L.bkmoo_resolve(4, r, 1, 4096, 2, offs, 2, ctypes.byref(bad), out, 1, None, None, None, ws,
                           ws_need, None) == -1
    assert L.bkmoo_resolve(4, r, 1, 4096, 2, offs, 0, ctypes.byref(hp), out, 1, None, None, None, ws,
                           ws_need - 1, None) == -3


def test_conflicts_argument_errors(b):
    L = b._lib
    g, o = FAKE, FAKE + (1 << 20)
    assert L.bkmoo_conflicts(1, 3, g, o, None, None, None) == -1       # K < 2
    assert L.bkmoo_conflicts(17, 3, g, o, None, None, None) == -2      # K > 16
    assert L.bkmoo_conflicts(4, 0, g, o, None, None, None) == -1       # no bucket
    assert L.bkmoo_conflicts(4, 3, None, o, None, None, None) == -1    # no Gram
    assert L.bkmoo_conflicts(4, 3, g, None, None, None, None) == -1    # no output


def test_exact_method_argument_errors(b):
    L = b._lib
    g, w = FAKE, FAKE + (1 << 20)
    hp = b._Hparams(0, 0.5, None)
    assert L.bkmoo_solve(11, 3, g, 4, None, w, None, None) == -2                    # K > 10
    assert L.bkmoo_solve(11, 3, g, 5, ctypes.byref(hp), w, None, None) == -2
    assert L.bkmoo_solve(4, 3, g, 5, None, w, None, None) == -1                     # c needed
    bad = b._Hparams(0, 1.0, None)
    assert L.bkmoo_solve(4, 3, g, 5, ctypes.byref(bad), w, None, None) == -1        # c out of range
    assert L.bkmoo_solve(4, 3, g, 6, ctypes.byref(hp), w, None, None) == -1         # no such method
    path = ctypes.c_int32(0)
    assert L.bkmoo_resolve_path(11, 1 << 20, 2, 1, 1, 1, 4, 0, ctypes.byref(path)) == -2
    assert L.bkmoo_resolve_path(4, 1 << 20, 2, 1, 1, 1, 4, 0, ctypes.byref(path)) == 0
    assert path.value == b.PATH_TWO_PASS


def test_slice_argument_errors(b):
    L = b._lib
    o, so = FAKE, FAKE + (1 << 20)
    assert L.bkmoo_slice_offsets(0, 4, o, so, None) == -1
    assert L.bkmoo_slice_offsets(3, 0, o, so, None) == -1
    assert L.bkmoo_slice_offsets(1 << 20, 1 << 12, o, so, None) == -1    # B*T beyond int32
    assert L.bkmoo_slice_offsets(3, 4, None, so, None) == -1
    assert L.bkmoo_slice_offsets(3, 4, o, None, None) == -1
    p, g = FAKE, FAKE + (64 << 20)
    assert L.bkmoo_gram_reduce(1, 3, 2, p, 0, g, None) == -1
    assert L.bkmoo_gram_reduce(17, 3, 2, p, 0, g, None) == -2
    assert L.bkmoo_gram_reduce(4, 3, 0, p, 0, g, None) == -1
    assert L.bkmoo_gram_reduce(4, 3, 2, p, 2, g, None) == -1              # layout
    assert L.bkmoo_gram_reduce(4, 3, 2, p, 0, p + 64, None) == -1         # overlap
    assert L.bkmoo_gram_reduce(4, 3, 2, None, 0, g, None) == -1


def test_resolve_traffic_two_pass_and_errors(b):
    """The two-pass byte count needs no device: 2K reads and one write per
    element; bad offsets and unknown paths are rejected."""
    import numpy as np
    offs = np.array([0, 10, 25, 25, 40])
    assert b.resolve_traffic(4, offs, "bf16", b.PATH_TWO_PASS) == (2 * 4 * 2 + 2) * 40
    assert b.resolve_traffic(3, offs, "f32", b.PATH_TWO_PASS, out_dtype="bf16") == (2 * 3 * 4 + 2) * 40
    for bad in ([0, 10, 5, 40], [1, 10, 40]):
        with pytest.raises(b.BkmooError, match="EINVAL"):
            b.resolve_traffic(4, np.array(bad), "bf16", b.PATH_TWO_PASS)
    with pytest.raises(b.BkmooError, match="EINVAL"):
        b.resolve_traffic(4, offs, "bf16", 7)
    with pytest.raises(b.BkmooError, match="EINVAL"):
        b.resolve_traffic(4, offs, "bf16", b.PATH_TWO_PASS, max_iter=-1)
    L = b._lib
    out = ctypes.c_uint64(0)
    o = np.ascontiguousarray(offs, dtype=np.int64)
    assert L.bkmoo_resolve_traffic(4, 40, 4, o.ctypes.data, 1, 1, 9, 20, b.PATH_TWO_PASS, ctypes.byref(out)) == -1


def test_grid_override_rejects_negative(b):
    assert b._lib.bkmoo_set_grid_override(-1) == -1
    assert b._lib.bkmoo_set_grid_override(0) == 0


def test_binding_rejects_bad_tensors_on_cpu(b):
    import torch
    with pytest.raises(ValueError):
        b.gram(torch.zeros((2, 8)), torch.zeros(2, dtype=torch.int64))   # CPU rows
    with pytest.raises(TypeError):
        b.gram(torch.zeros((2, 8), dtype=torch.float16), torch.zeros(2, dtype=torch.int64))
    # host tensors are refused before any call reaches the library
    G = torch.zeros((3, 2, 2), dtype=torch.float64)
    for call in (lambda: b.solve(G, "mgda"), lambda: b.conflicts(G),
                 lambda: b.gram_reduce(torch.zeros((2, 3, 2, 2), dtype=torch.float64)),
                 lambda: b.read_device_error(torch.zeros(256, dtype=torch.uint8)),
                 lambda: b.slice_offsets(torch.zeros(4, dtype=torch.int64), 2),
                 lambda: b.combine(torch.zeros((2, 8)), torch.zeros(2, dtype=torch.int64),
                                   torch.zeros((1, 2))),
                 lambda: b.resolve(torch.zeros((2, 8)), torch.zeros(2, dtype=torch.int64), "mgda")):
        with pytest.raises(ValueError, match="GPU"):
            call()


def test_resolve_noalloc_rejects_before_queueing(b):
    """The no-allocation resolve checks its arguments like bkmoo_resolve, and
    a configuration whose workspace exceeds its fixed 96 MiB scratch, before
    it looks up the scratch or queues anything."""
    L = b._lib
    hp = b._Hparams(20, 0.5, None)
    offs, out = FAKE + (64 << 20), FAKE + (80 << 20)
    # K=16 bf16 over 2^33 elements needs far more than the scratch holds
    assert b.workspace_size(16, 1 << 33, 1, "bf16") > 96 << 20
    assert L.bkmoo_resolve_noalloc(16, rows(16, step=1 << 34), 1, 1 << 33, 1, offs, 0, ctypes.byref(hp),
                                   FAKE - (32 << 30), 1, None, None, None, None) == -3
    r = rows(4)
    assert L.bkmoo_resolve_noalloc(1, r, 1, 4096, 2, offs, 0, ctypes.byref(hp), out, 1, None, None, None,
                                   None) == -1                                              # K < 2
    assert L.bkmoo_resolve_noalloc(4, None, 1, 4096, 2, offs, 0, ctypes.byref(hp), out, 1, None, None, None,
                                   None) == -1                                              # no rows
    assert L.bkmoo_resolve_noalloc(4, r, 1, 4096, 2, None, 0, ctypes.byref(hp), out, 1, None, None, None,
                                   None) == -1                                              # no offsets
    bad = b._Hparams(20, 1.5, None)
    assert L.bkmoo_resolve_noalloc(4, r, 1, 4096, 2, offs, 2, ctypes.byref(bad), out, 1, None, None, None,
                                   None) == -1                                              # c >= 1
    assert L.bkmoo_resolve_noalloc(4, r, 1, 4096, 2, offs, 0, ctypes.byref(hp), FAKE + 64, 1, None, None, None,
                                   None) == -1                                              # overlapping out
